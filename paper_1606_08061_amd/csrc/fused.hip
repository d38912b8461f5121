// The factored minibatch step (Algorithm 3 for squared error, Algorithm 4 with
// dl/ds = 0 for the spherical softmax) as five launches on one stream.
//
// Notation (rows are examples: H is m x d, the paper's d x m H transposed):
//   H^ = H Q, H~ = H U^T, X = H U^{-T T}      (Alg. 3 steps 1, 5, 6; Alg. 4 rows 1, 5)
//   q_j = h_j . h^_j (eq. qvec), a_kj = h~_j . V_r (eq. gen-A-fact), the loss epilogue
//   l_j, dl/dq_j, dl/dA_kj, G_j = sum_k dl/dA_kj V_r (the V^T Yring of eq. gen-Zhat-fact)
//   Z^ = G U, grad_H = 2 diag(dl/dq) H^ + Z^ (eq. gen-grad-H-fact)
//   M = 4 D M^ D + Yring^T Yring + 2 D HZ + 2 HZ^T D (eq. gen-M; M^ = H H^^T,
//       HZ = H~ G^T, D = diag(dl/dq))
//   U <- U - 2 eta H~^T D H (eq. updateU / gen-updateU)
//   Q <- Q + H^T Zq + Zq^T H, Zq = (eta^2/2) M H - eta grad_H (eq. updateQ / gen-Qnew)
//   U^{-T} <- U^{-T} + (R X)^T H, R = 2 eta S C^{-1} S, C = I - 2 eta S N S,
//       S = D^(1/2), N = H H^T (the Woodbury form of section 4.7)
//   V_r <- V_r - eta sum dl/dA_kj P_j with P = U_new^{-T} H (eq. updateV, gen-updateV)
//
// The Woodbury inverse.  E = 2 eta S N S is symmetric positive semidefinite, and C
// is positive definite with C^{-1} = sum_k E^k when its spectral radius is below 1.
// The step takes C^{-1} as the degree-7 polynomial p(E) interpolating 1/(1 - x) at
// the Chebyshev points of [0, b], b = ||E^2||_inf^(1/2) >= rho(E): for every
// eigenvalue x of E, |1/(1 - x) - p(x)| <= 2 (b/4)^8 / (1 - b)^9 (the interpolation
// remainder with the node polynomial of the Chebyshev points), so a b for which
// that bound is below 2^-24 certifies both that C is positive definite and that
// p(E) equals C^{-1} to below fp32 rounding (b <= 0.3; the workloads of the paper's
// shapes have b of 0.05 to 0.25).  Otherwise (a large step, or a matrix that is not
// positive definite) one workgroup forms C^{-1} by exact Gauss-Jordan elimination,
// whose pivots also decide positive definiteness.  With Xs = S X:
//   R X = 2 eta S p(E) Xs,  p(E) Xs = sum_k c_k E^k Xs.
// P needs no product of its own: P = S^{-1} C^{-1} S X, i.e. P_j = (R X)_j /
// (2 eta dl/dq_j), and an example with dl/dq_j = 0 has dl/dA_kj = 0 (no V update).
//
// Launches (every product on v_mfma_f32_16x16x4_f32 or v_mfma_f32_32x32x2_f32):
//   1  H^ (with the row partials of q), H~, X, N; the step's target rows of V read
//      into the L2 of the XCD that gathers them in launch 2
//   2  gather + loss epilogue (one workgroup per example); M^ = H H^^T; E^2 (with
//      its absolute row sums); W1 = E Xs
//   3  Z^ with grad_H; HZ; P2 = E^2 Xs; P3 = E^2 W1; E^4; Yring^T Yring; L = sum l_j;
//      the certificate, the coefficients c_k, and (uncertified) the exact R
//   4  Zq; R X; the U update                                 [writes U]
//   5  the Q and U^{-T} updates; the V scatter                [writes Q, U^{-T}, V]
// Q, U, U^{-T} and V are read (launches 1-3) before any of them is written
// (launches 4-5), and every error is raised by launch 3 at the latest; launches 4
// and 5 read the error flag first and write nothing if it is set, so a failed step
// changes no state.
#include <cmath>

#include "gemm_tiles.h"
#include "scatter.h"

namespace lst {

namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__device__ __forceinline__ const float *rsv(const float *p, const float *H, float *gH) {
  const uintptr_t v = reinterpret_cast<uintptr_t>(p);
  return v == 16 ? H : (v == 32 ? gH : p);
}

// q_j from the row partials of launch 1's H^ tiles, summed in tile order (every
// workgroup that needs q_j forms the identical value).
__device__ __forceinline__ float q_of(const float *__restrict__ qpart, int T, int m, int j) {
  float q = 0.f;
  for (int t = 0; t < T; ++t) q += qpart[(int64_t)t * m + j];
  return q;
}

// dl/dq_j: 1 for squared error; for the spherical softmax (sum of the example's
// target weights over its valid slots, in slot order) / (q_j + D eps).
__device__ __forceinline__ float dq_of(int loss, float q, float tsum, float Deps) {
  return loss == LST_LOSS_SQUARED ? 1.f : tsum / (q + Deps);
}

__device__ __forceinline__ float tsum_of(const int *__restrict__ idx, const float *__restrict__ val,
                                         int K, int64_t D, int j) {
  float s = 0.f;
  for (int k = 0; k < K; ++k) {
    const int r = idx[(int64_t)j * K + k];
    if (r >= 0 && (int64_t)r < D) s += val[(int64_t)j * K + k];
  }
  return s;
}

__device__ __forceinline__ float scale_of(int mode, const float *dq, int i) {
  if (mode == SC_NONE || !dq) return 1.f;
  const float v = dq[i];
  return mode == SC_DQ ? v : sqrtf(v);  // sqrt of a negative dl/dq is NaN: never certified
}

// ---------------------------------------------------------------------------
// One 16 x 16 output tile of an Op16 (workgroup of 256 threads).  Lane
// l = c + 16 g of wavefront w supplies A[i0 + c][k] and B[k][j0 + c] for
// k = kb + 4 g + s in instruction s of the k-block kb = 16 (w + 4 u); accumulator
// register r holds C[i0 + 4 g + r][j0 + c].  The four wavefronts' sums are added
// through LDS in a fixed order.  Loads of up to kGroup k-blocks are issued before
// their products.
// ---------------------------------------------------------------------------
constexpr int kGroup = 8;

// Four consecutive k values of index idx of a source: tr = 0 -> p[idx ld + k]
// (contiguous, one 16-byte load when aligned), tr = 1 -> p[k ld + idx].  k >= kend
// reads as zero (address clamped).
__device__ __forceinline__ void ld4k(const float *__restrict__ p, int64_t ld, int tr, int idx,
                                     int k0, int kend, float (&o)[4]) {
  if (k0 + 3 < kend) {
    if (tr == 0) {
      const float *q = p + (int64_t)idx * ld + k0;
      if (((reinterpret_cast<uintptr_t>(q)) & 15) == 0) {
        const float4 v = *reinterpret_cast<const float4 *>(q);
        o[0] = v.x;
        o[1] = v.y;
        o[2] = v.z;
        o[3] = v.w;
      } else {
        o[0] = q[0];
        o[1] = q[1];
        o[2] = q[2];
        o[3] = q[3];
      }
    } else {
      const float *q = p + (int64_t)k0 * ld + idx;
      o[0] = q[0];
      o[1] = q[ld];
      o[2] = q[2 * ld];
      o[3] = q[3 * ld];
    }
    return;
  }
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const int k = min(k0 + s, kend - 1);
    const float v = tr == 0 ? p[(int64_t)idx * ld + k] : p[(int64_t)k * ld + idx];
    o[s] = (k0 + s < kend) ? v : 0.f;
  }
}

struct TileCtx {
  const float *H;
  float *gH;
  float lr;
  const float *dq;    // dl/dq for the scale modes (may be null when no term scales)
  const float *coef;  // polynomial coefficients (LDS), or null
};

__device__ __forceinline__ float coef_of(const TileCtx &x, int c) { return c < 0 ? 1.f : x.coef[c]; }

__device__ __forceinline__ void op16_tile(const Op16 &g, int local, const TileCtx &x) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = lane & 15, lg = lane >> 4;
  // column-major tile order: consecutive tiles share a B panel (and so an XCD's L2)
  const int tn = local / g.tiles_m, tm = local - tn * g.tiles_m;
  const int i0 = tm * 16, j0 = tn * 16;
  const int ia = min(i0 + c, g.M - 1), jb = min(j0 + c, g.N - 1);
  const int K = g.K;

  const float *A = rsv(g.A, x.H, x.gH);
  const float *Bp[kMaxTerms];
  float bco[kMaxTerms];
#pragma unroll
  for (int t = 0; t < kMaxTerms; ++t) {
    Bp[t] = t < g.nb ? rsv(g.b[t].p, x.H, x.gH) : nullptr;
    bco[t] = t < g.nb ? coef_of(x, g.b[t].coef) : 0.f;
  }
  // MASM: A(i,k) = 4 dq_i M^_ik dq_k + YY_ik + 2 dq_i HZ_ik + 2 dq_k HZ_ki
  const float dqi = (g.amode == AM_MASM && x.dq) ? x.dq[ia] : 1.f;

  floatx4 acc = {0.f, 0.f, 0.f, 0.f};
  const int nblk = (K + 15) >> 4;
  const int nw = nblk > wave ? (nblk - wave + 3) / 4 : 0;
  for (int u0 = 0; u0 < nw; u0 += kGroup) {
    float a[kGroup][4], b[kGroup][4];
#pragma unroll
    for (int u = 0; u < kGroup; ++u) {
      const int k0 = 16 * (wave + 4 * min(u0 + u, nw - 1)) + 4 * lg;
      if (g.amode == AM_MASM) {
        float mh[4], yy[4], hz[4], hzt[4], dk[4];
        ld4k(g.Mh, g.ldm, 0, ia, k0, K, mh);
        ld4k(g.YY, g.ldm, 0, ia, k0, K, yy);
        ld4k(g.HZ, g.ldm, 0, ia, k0, K, hz);
        ld4k(g.HZ, g.ldm, 1, ia, k0, K, hzt);
        if (x.dq) {
          ld4k(x.dq, 0, 0, 0, k0, K, dk);
        } else {
          dk[0] = dk[1] = dk[2] = dk[3] = 1.f;
        }
#pragma unroll
        for (int s = 0; s < 4; ++s)
          a[u][s] = 4.f * dqi * mh[s] * dk[s] + yy[s] + 2.f * dqi * hz[s] + 2.f * dk[s] * hzt[s];
      } else {
        ld4k(A, g.lda, g.tA, ia, k0, K, a[u]);
      }
#pragma unroll
      for (int s = 0; s < 4; ++s) b[u][s] = 0.f;
#pragma unroll
      for (int t = 0; t < kMaxTerms; ++t) {
        if (t >= g.nb) break;
        float v[4];
        ld4k(Bp[t], g.b[t].ld, g.b[t].tr, jb, k0, K, v);
        if (g.b[t].sc != SC_NONE) {
#pragma unroll
          for (int s = 0; s < 4; ++s) v[s] *= scale_of(g.b[t].sc, x.dq, min(k0 + s, K - 1));
        }
#pragma unroll
        for (int s = 0; s < 4; ++s) b[u][s] = fmaf(bco[t], v[s], b[u][s]);
      }
    }
#pragma unroll
    for (int u = 0; u < kGroup; ++u)
      if (u0 + u < nw) {
#pragma unroll
        for (int s = 0; s < 4; ++s)
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[u][s], b[u][s], acc, 0, 0, 0);
      }
  }

  __shared__ float red[4][4][64];
#pragma unroll
  for (int r = 0; r < 4; ++r) red[wave][r][lane] = acc[r];
  __syncthreads();
  // output of this thread: accumulator register `wave` of lane `lane`
  const int oi = i0 + 4 * lg + wave, oj = j0 + c;
  const bool ok = oi < g.M && oj < g.N;
  const int ci = min(oi, g.M - 1), cj = min(oj, g.N - 1);
  float v = (red[0][wave][lane] + red[1][wave][lane]) + (red[2][wave][lane] + red[3][wave][lane]);
  __syncthreads();  // red is reused by the next tile of this workgroup
#pragma unroll
  for (int t = 0; t < kMaxTerms; ++t) {
    if (t >= g.nadd) break;
    const OpTerm &ad = g.add[t];
    const float *p = rsv(ad.p, x.H, x.gH);
    v = fmaf(coef_of(x, ad.coef) * scale_of(ad.sc, x.dq, ci), p[(int64_t)ci * ad.ld + cj], v);
  }
  float al = g.alpha;
  for (int e = 0; e < g.alpha_lr; ++e) al *= x.lr;
  v *= al * scale_of(g.rs, x.dq, ci) * scale_of(g.cs, x.dq, cj);
  if (g.Cin) {
    float be = g.beta;
    for (int e = 0; e < g.beta_lr; ++e) be *= x.lr;
    v = fmaf(be, rsv(g.Cin, x.H, x.gH)[(int64_t)ci * g.ldcin + cj], v);
  }
  if (ok) {
    if (g.C) const_cast<float *>(rsv(g.C, x.H, x.gH))[(int64_t)oi * g.ldc + oj] = v;
    if (g.C2)
      const_cast<float *>(rsv(g.C2, x.H, x.gH))[(int64_t)oi * g.ldc2 + oj] =
          2.f * scale_of(g.rs2, x.dq, oi) * rsv(g.E, x.H, x.gH)[(int64_t)oi * g.lde + oj] + v;
  }
  if (g.rowred != RR_NONE) {
    float r = 0.f;
    if (ok) r = g.rowred == RR_DOT ? v * rsv(g.Rr, x.H, x.gH)[(int64_t)oi * g.ldrr + oj] : fabsf(v);
    // the 16 lanes of this row (same g, same wavefront), in a fixed order
    r += __shfl_xor(r, 1);
    r += __shfl_xor(r, 2);
    r += __shfl_xor(r, 4);
    r += __shfl_xor(r, 8);
    if (c == 0 && oi < g.M) g.rowout[(int64_t)tn * g.M + oi] = r;
  }
}

// Workgroup w of a section of 8 ceil(T / 8) workgroups (the section starting on a
// multiple of 8, so that w runs on XCD w % 8): the logical tile it owns, or -1.
// XCD x owns a contiguous range of tiles.
__device__ __forceinline__ int section_tile(int w, int T) {
  const int q = T >> 3, r = T & 7;
  const int x = w & 7, slot = w >> 3;
  if (slot >= (x < r ? q + 1 : q)) return -1;
  return x < r ? x * (q + 1) + slot : r * (q + 1) + (x - r) * q + slot;
}

// Tile `tile` of a batch of Op16 (the descriptor whose range holds it); alt
// descriptors replace theirs when the polynomial is not certified.
__device__ __forceinline__ void run_op(const OpBatch &ob, int tile, const TileCtx &x, bool cert) {
  int di = 0;
  for (int q = 1; q < ob.n; ++q)
    if (tile >= ob.op[q].tile_begin) di = q;
  if (di >= ob.n_main) return;  // alt descriptors own no tiles of their own
  const Op16 *g = &ob.op[di];
  const int local = tile - g->tile_begin;
  if (!cert && g->alt >= 0) g = &ob.op[g->alt];
  op16_tile(*g, local, x);
}

// ---------------------------------------------------------------------------
// Launch 1: contractions, N, prefetch of the target rows.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void step_contract_kernel(const StepPlan *__restrict__ pl,
                                                            const float *H, float lr,
                                                            const int *__restrict__ idx, int K,
                                                            const float *__restrict__ V,
                                                            int64_t ldv, int64_t D, int d, int m) {
  const OpBatch &ob = pl->ob[0];
  const int w = blockIdx.x;
  const int sec = (ob.total + 7) & ~7;
  if (w < sec) {
    const int tile = section_tile(w, ob.total);
    if (tile < 0) return;
    const TileCtx x{H, nullptr, lr, nullptr, nullptr};
    run_op(ob, tile, x, true);
    return;
  }
  // Prefetch workgroup of example j (XCD j % 8, that of its gather workgroup in
  // launch 2): the indices, then one load per 128-byte line of every target row.
  const int j = w - sec;
  if (j >= m) return;
  __shared__ int prow[LST_MAX_K];
  for (int k = threadIdx.x; k < K; k += 256) {
    const int r = idx[(int64_t)j * K + k];
    prow[k] = (r < 0 || (int64_t)r >= D) ? -1 : r;
  }
  __syncthreads();
  const int nl = (d + 31) >> 5;
  float sink = 0.f;
  for (int e = threadIdx.x; e < K * nl; e += 256) {
    const int k = e / nl, r = prow[k];
    if (r >= 0) sink += V[(int64_t)r * ldv + 32 * (e - k * nl)];
  }
  asm volatile("" ::"v"(sink));
}

// ---------------------------------------------------------------------------
// Launch 2: the gather and loss epilogue of one example per workgroup.
// ---------------------------------------------------------------------------
struct GatherArgs {
  int K, d, m, T;
  int64_t D;
  const float *H, *Htil, *qpart;
  const int *idx;
  const float *val;
  const float *V;
  int64_t ldv;
  int loss;
  float eps, lr;
  float *G, *Atil, *dq, *dA, *wA, *lvec;
  int *srow;
  float *sval;
  int *scnt;
  int *flag;
};

// Loss epilogue of one example (section 4, dl/ds = 0); r[k] < 0 marks an empty slot.
// l = q - 2 a.t + ||y||^2 (squared error, ||y||^2 by index equality) or
// l = sum_k t_k [log(q + D eps) - log(a_k^2 + eps)] (spherical softmax).
__device__ __forceinline__ void epilogue(int loss, float q, float gq, int K, const int *r,
                                         const float *t, const float *a, float Deps, float eps,
                                         float &l, float *g) {
  l = 0.f;
  if (loss == LST_LOSS_SQUARED) {
    float at = 0.f, yy = 0.f;
    for (int k = 0; k < K; ++k) {
      g[k] = 0.f;
      if (r[k] < 0) continue;
      at += t[k] * a[k];
      for (int kk = 0; kk < K; ++kk)
        if (r[kk] == r[k]) yy += t[k] * t[kk];
      g[k] = -2.f * t[k];
    }
    l = q - 2.f * at + yy;
  } else {
    const float lz = logf(q + Deps);
    for (int k = 0; k < K; ++k) {
      g[k] = 0.f;
      if (r[k] < 0) continue;
      const float den = a[k] * a[k] + eps;
      l += t[k] * (lz - logf(den));
      g[k] = -2.f * t[k] * a[k] / den;
    }
  }
  (void)gq;
}

// The sorted list of the example's target rows with their summed dl/dA (rows
// ascending; repeated rows merged, values added in slot order) for Yring^T Yring.
// All threads of the workgroup call it; threads k < K each place one slot.
__device__ __forceinline__ void sorted_slots(int j, int K, const int *sr, const float *sg,
                                             int *srow, float *sval, int *scnt) {
  __shared__ int first[LST_MAX_K];
  const int k = threadIdx.x;
  if (k < K) {
    const int r = sr[k];
    bool f = r >= 0;
    for (int k2 = 0; k2 < k; ++k2) f &= sr[k2] != r;
    first[k] = f ? 1 : 0;
  }
  __syncthreads();
  if (k < K && first[k]) {
    const int r = sr[k];
    float v = 0.f;
    int pos = 0;
    for (int k2 = 0; k2 < K; ++k2) {
      if (sr[k2] == r) v += sg[k2];
      pos += (first[k2] && sr[k2] < r) ? 1 : 0;
    }
    srow[(int64_t)j * K + pos] = r;
    sval[(int64_t)j * K + pos] = v;
  }
  if (threadIdx.x == 0) {
    int n = 0;
    for (int k2 = 0; k2 < K; ++k2) n += first[k2];
    scnt[j] = n;
  }
}

// Register-resident form for K <= 4 KPW and d <= 64 NV: wavefront w keeps the
// target rows k = w, w + 4, ... in registers from the dot products a_kj to the G
// sum, so V is read once and the index loads lead straight into the row loads.
template <int KPW, int NV>
__device__ __forceinline__ void gather_reg(const GatherArgs &ga, int j) {
  constexpr int W = 4;
  __shared__ int sr[W * KPW];
  __shared__ float sa[W * KPW], st[W * KPW], sg[W * KPW];
  __shared__ float s_dq;
  __shared__ int s_bad;
  __shared__ float gpart[W][64 * NV];
  const int K = ga.K, d = ga.d;
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  if (t == 0) s_bad = 0;
  int r[KPW];
  bool bad = false;
#pragma unroll
  for (int i = 0; i < KPW; ++i) {
    const int k = wave + W * i;
    int v = -1;
    if (k < K) {
      v = ga.idx[(int64_t)j * K + k];
      if (v < -1 || (int64_t)v >= ga.D) {
        bad = true;
        v = -1;
      }
    }
    r[i] = v;
  }
  float vr[KPW][NV];
#pragma unroll
  for (int i = 0; i < KPW; ++i) {
    const float *row = ga.V + (int64_t)max(r[i], 0) * ga.ldv;
#pragma unroll
    for (int n = 0; n < NV; ++n) {
      const int c = lane + 64 * n;
      const float xv = row[min(c, d - 1)];
      vr[i][n] = (r[i] >= 0 && c < d) ? xv : 0.f;
    }
  }
  float ht[NV];
  const float *htp = ga.Htil + (int64_t)j * d;
#pragma unroll
  for (int n = 0; n < NV; ++n) {
    const int c = lane + 64 * n;
    ht[n] = (c < d) ? htp[c] : 0.f;
  }
  float a[KPW];
#pragma unroll
  for (int i = 0; i < KPW; ++i) {
    float sacc = 0.f;
#pragma unroll
    for (int n = 0; n < NV; ++n) sacc += ht[n] * vr[i][n];
    a[i] = wave_sum(sacc);
  }
  __syncthreads();  // s_bad initialised
  if (lane == 0) {
#pragma unroll
    for (int i = 0; i < KPW; ++i) {
      const int k = wave + W * i;
      if (k < K) {
        sr[k] = r[i];
        sa[k] = a[i];
        st[k] = ga.val[(int64_t)j * K + k];
      }
    }
    if (bad) atomicOr(&s_bad, 1);
  }
  __syncthreads();
  if (t == 0) {
    if (s_bad) atomicOr(ga.flag, FLAG_INDEX);
    const float q = q_of(ga.qpart, ga.T, ga.m, j);
    const float Deps = (float)ga.D * ga.eps;
    const float gq = dq_of(ga.loss, q, tsum_of(ga.idx, ga.val, K, ga.D, j), Deps);
    float l;
    epilogue(ga.loss, q, gq, K, sr, st, sa, Deps, ga.eps, l, sg);
    ga.dq[j] = gq;
    ga.lvec[j] = l;
    s_dq = gq;
  }
  __syncthreads();
  const float gq = s_dq;
  for (int k = t; k < K; k += 256) {
    ga.dA[(int64_t)j * K + k] = sg[k];
    ga.wA[(int64_t)j * K + k] = gq != 0.f ? sg[k] / (2.f * gq) : 0.f;
  }
  sorted_slots(j, K, sr, sg, ga.srow, ga.sval, ga.scnt);
#pragma unroll
  for (int n = 0; n < NV; ++n) {
    float gv = 0.f;
#pragma unroll
    for (int i = 0; i < KPW; ++i) {
      const int k = wave + W * i;
      if (k < K) gv += sg[k] * vr[i][n];
    }
    gpart[wave][lane + 64 * n] = gv;
  }
  __syncthreads();
  const float s2 = 2.f * ga.lr * gq;
  for (int c = t; c < d; c += 256) {
    ga.G[(int64_t)j * d + c] = (gpart[0][c] + gpart[1][c]) + (gpart[2][c] + gpart[3][c]);
    ga.Atil[(int64_t)j * d + c] = s2 * htp[c];
  }
}

// General form (any K <= LST_MAX_K, any d): the K dot products spread over the
// wavefronts, then G column-parallel.
__device__ __forceinline__ void gather_gen(const GatherArgs &ga, int j) {
  __shared__ int sr[LST_MAX_K];
  __shared__ float sa[LST_MAX_K], st[LST_MAX_K], sg[LST_MAX_K];
  __shared__ float s_dq;
  __shared__ int s_bad;
  const int K = ga.K, d = ga.d;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const float *ht = ga.Htil + (int64_t)j * d;
  if (t == 0) s_bad = 0;
  __syncthreads();
  for (int k = t; k < K; k += 256) {
    int r = ga.idx[(int64_t)j * K + k];
    if (r < -1 || (int64_t)r >= ga.D) {
      atomicOr(&s_bad, 1);
      r = -1;
    }
    sr[k] = r;
    st[k] = ga.val[(int64_t)j * K + k];
  }
  __syncthreads();
  for (int k = wave; k < K; k += 4) {
    const int r = sr[k];
    float a = 0.f;
    if (r >= 0) {
      const float *vr = ga.V + (int64_t)r * ga.ldv;
      float s = 0.f;
      for (int c = lane; c < d; c += 64) s += ht[c] * vr[c];
      a = wave_sum(s);
    }
    if (lane == 0) sa[k] = a;
  }
  __syncthreads();
  if (t == 0) {
    if (s_bad) atomicOr(ga.flag, FLAG_INDEX);
    const float q = q_of(ga.qpart, ga.T, ga.m, j);
    const float Deps = (float)ga.D * ga.eps;
    const float gq = dq_of(ga.loss, q, tsum_of(ga.idx, ga.val, K, ga.D, j), Deps);
    float l;
    epilogue(ga.loss, q, gq, K, sr, st, sa, Deps, ga.eps, l, sg);
    ga.dq[j] = gq;
    ga.lvec[j] = l;
    s_dq = gq;
  }
  __syncthreads();
  const float gq = s_dq;
  for (int k = t; k < K; k += 256) {
    ga.dA[(int64_t)j * K + k] = sg[k];
    ga.wA[(int64_t)j * K + k] = gq != 0.f ? sg[k] / (2.f * gq) : 0.f;
  }
  sorted_slots(j, K, sr, sg, ga.srow, ga.sval, ga.scnt);
  const float s2 = 2.f * ga.lr * gq;
  for (int c = t; c < d; c += 256) {
    float s = 0.f;
    for (int k = 0; k < K; ++k) {
      const int r = sr[k];
      if (r >= 0) s += sg[k] * ga.V[(int64_t)r * ga.ldv + c];
    }
    ga.G[(int64_t)j * d + c] = s;
    ga.Atil[(int64_t)j * d + c] = s2 * ht[c];
  }
}

// dl/dq of every example into LDS (the spherical softmax's E products need all of
// them before the gather workgroups have written theirs; the same arithmetic).
__device__ __forceinline__ void dq_all(const GatherArgs &ga, float *sdq) {
  for (int i = threadIdx.x; i < ga.m; i += 256) {
    const float q = q_of(ga.qpart, ga.T, ga.m, i);
    sdq[i] = dq_of(ga.loss, q, tsum_of(ga.idx, ga.val, ga.K, ga.D, i), (float)ga.D * ga.eps);
  }
  __syncthreads();
}

template <int KPW, int NV>
__global__ __launch_bounds__(256) void step_gather_kernel(const StepPlan *__restrict__ pl,
                                                          const float *H, float lr,
                                                          const GatherArgs ga) {
  const int w = blockIdx.x;
  const int gsec = (ga.m + 7) & ~7;
  if (w < gsec) {
    if (w >= ga.m) return;
    if constexpr (NV > 0)
      gather_reg<KPW, NV>(ga, w);
    else
      gather_gen(ga, w);
    return;
  }
  const OpBatch &ob = pl->ob[1];
  const int tile = section_tile(w - gsec, ob.total);
  if (tile < 0) return;
  __shared__ float sdq[LST_MAX_M];
  const float *dq = nullptr;
  if (ga.loss != LST_LOSS_SQUARED) {
    dq_all(ga, sdq);
    dq = sdq;
  }
  const TileCtx x{H, nullptr, lr, dq, nullptr};
  run_op(ob, tile, x, true);
}

// ---------------------------------------------------------------------------
// Launch 3: Z^ and grad_H, HZ, the polynomial's products, Yring^T Yring, the loss,
// the certificate.
// ---------------------------------------------------------------------------
struct CertArgs {
  int m;
  const float *bpart;  // [ceil(m/16)][m] absolute row partial sums of E^2
  const float *N, *dq; // dq null for squared error
  float *Cwork, *R, *coef;
  int *cert;
  int *flag;
};

// Power-basis coefficients c_0..c_7 of the degree-7 interpolant of 1/(1 - x) at the
// Chebyshev points of [0, b] (fp64: divided differences in y = x / b on [0, 1], the
// Newton form expanded, c_k = d_k / b^k).  For b below 1e-3 the Neumann
// coefficients (all 1) are already exact to far below fp32 rounding.
__device__ void cheb_coeffs(double b, float *c) {
  if (!(b > 1e-3)) {
    for (int k = 0; k < 8; ++k) c[k] = 1.f;
    return;
  }
  double y[8], f[8];
  for (int i = 0; i < 8; ++i) {
    y[i] = 0.5 * (1.0 + cos((2.0 * i + 1.0) * M_PI / 16.0));
    f[i] = 1.0 / (1.0 - b * y[i]);
  }
  for (int k = 1; k < 8; ++k)
    for (int i = 7; i >= k; --i) f[i] = (f[i] - f[i - 1]) / (y[i] - y[i - k]);
  // p(y) = f0 + (y - y0)(f1 + (y - y1)(f2 + ...)): expand from the innermost factor
  double p[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  p[0] = f[7];
  int deg = 0;
  for (int k = 6; k >= 0; --k) {
    // p <- p * (y - y_k) + f_k
    for (int e = deg + 1; e >= 1; --e) p[e] = p[e - 1] - y[k] * p[e];
    p[0] = -y[k] * p[0] + f[k];
    ++deg;
  }
  double bk = 1.0;
  for (int k = 0; k < 8; ++k) {
    c[k] = (float)(p[k] / bk);
    bk *= b;
  }
}

// The bound of the interpolation error at b (see the top of the file).
__device__ __forceinline__ bool certified(double b) {
  if (!(b >= 0.0) || !(b < 0.5)) return false;
  const double r = b / 4.0, r2 = r * r, r4 = r2 * r2;
  const double om = 1.0 - b;
  const double om3 = om * om * om;
  return 2.0 * r4 * r4 <= 5.9604644775390625e-8 * (om3 * om3 * om3);  // 2^-24
}

// Exact R = 2 eta S C^{-1} S by Gauss-Jordan elimination without pivoting on one
// workgroup (C is symmetric; its pivots are all positive exactly when it is
// positive definite, else the error flag is raised).  C in Cwork, in place.
__device__ void exact_r(const CertArgs &ca, float lr) {
  const int m = ca.m, t = threadIdx.x;
  __shared__ float colp[LST_MAX_M], rowp[LST_MAX_M];
  __shared__ int s_bad;
  float *A = ca.Cwork;
  if (t == 0) s_bad = 0;
  __syncthreads();
  for (int i = t; i < m; i += 256) {
    const float v = ca.dq ? ca.dq[i] : 1.f;
    if (!(v >= 0.f)) s_bad = 1;  // no real square root: not positive definite
    colp[i] = sqrtf(fmaxf(v, 0.f));
  }
  __syncthreads();
  if (s_bad) {
    if (t == 0) atomicOr(ca.flag, FLAG_NOT_SPD);
    return;
  }
  for (int64_t e = t; e < (int64_t)m * m; e += 256) {
    const int i = (int)(e / m), j = (int)(e - (int64_t)i * m);
    A[e] = (i == j ? 1.f : 0.f) - 2.f * lr * colp[i] * ca.N[e] * colp[j];
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __syncthreads();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  for (int p = 0; p < m; ++p) {
    for (int i = t; i < m; i += 256) {
      colp[i] = A[(int64_t)i * m + p];
      rowp[i] = A[(int64_t)p * m + i];
    }
    __syncthreads();
    const float piv = colp[p];
    if (!(piv > 0.f)) {
      if (t == 0) atomicOr(ca.flag, FLAG_NOT_SPD);
      return;
    }
    const float ip = 1.f / piv;
    for (int64_t e = t; e < (int64_t)m * m; e += 256) {
      const int i = (int)(e / m), j = (int)(e - (int64_t)i * m);
      float v;
      if (i == p)
        v = (j == p) ? ip : rowp[j] * ip;
      else if (j == p)
        v = -colp[i] * ip;
      else
        v = A[e] - colp[i] * (rowp[j] * ip);
      A[e] = v;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __syncthreads();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  }
  for (int i = t; i < m; i += 256) colp[i] = ca.dq ? sqrtf(fmaxf(ca.dq[i], 0.f)) : 1.f;
  __syncthreads();
  for (int64_t e = t; e < (int64_t)m * m; e += 256) {
    const int i = (int)(e / m), j = (int)(e - (int64_t)i * m);
    ca.R[e] = 2.f * lr * colp[i] * A[e] * colp[j];
  }
}

__device__ void cert_task(const CertArgs &ca, float lr) {
  __shared__ float rmax[4];
  __shared__ int rbad[4];
  const int m = ca.m, T = (m + 15) >> 4;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  float mx = 0.f;
  int bad = 0;
  for (int i = t; i < m; i += 256) {
    float s = 0.f;
    for (int q = 0; q < T; ++q) s += ca.bpart[(int64_t)q * m + i];
    if (!isfinite(s)) bad = 1;
    mx = fmaxf(mx, s);
  }
  for (int o = 32; o > 0; o >>= 1) {
    mx = fmaxf(mx, __shfl_xor(mx, o));
    bad |= __shfl_xor(bad, o);
  }
  if (lane == 0) {
    rmax[wave] = mx;
    rbad[wave] = bad;
  }
  __syncthreads();
  const float b2 = fmaxf(fmaxf(rmax[0], rmax[1]), fmaxf(rmax[2], rmax[3]));
  const bool anybad = rbad[0] | rbad[1] | rbad[2] | rbad[3];
  const double b = sqrt((double)b2);
  const bool ok = !anybad && certified(b);
  if (t == 0) {
    float c[8];
    cheb_coeffs(ok ? b : 0.0, c);
    for (int k = 0; k < 8; ++k) ca.coef[k] = c[k];
    *ca.cert = ok ? 1 : 0;
  }
  if (!ok) exact_r(ca, lr);
}

// Yring^T Yring entry (i, j): the merge of the two examples' sorted slot lists.
__device__ __forceinline__ void yy_entry(int e, int m, int K, const int *__restrict__ srow,
                                         const float *__restrict__ sval,
                                         const int *__restrict__ scnt, float *__restrict__ YY) {
  if (e >= m * m) return;
  const int i = e / m, j = e - (e / m) * m;
  const int *ri = srow + (int64_t)i * K, *rj = srow + (int64_t)j * K;
  const float *vi = sval + (int64_t)i * K, *vj = sval + (int64_t)j * K;
  const int na = scnt[i], nb = scnt[j];
  float yy = 0.f;
  int a = 0, b = 0;
  while (a < na && b < nb) {
    const int ra = ri[a], rb = rj[b];
    if (ra == rb) {
      yy += vi[a] * vj[b];
      ++a;
      ++b;
    } else if (ra < rb) {
      ++a;
    } else {
      ++b;
    }
  }
  YY[e] = yy;
}

struct MidArgs {
  int m, K;
  const int *srow;
  const float *sval;
  const int *scnt;
  float *YY;
  const float *lvec;
  float *loss_out;
  int *flag;
};

__global__ __launch_bounds__(256) void step_zgrad_kernel(const StepPlan *__restrict__ pl,
                                                         const float *H, float *gH, float lr,
                                                         const float *dq, const MidArgs ma,
                                                         const CertArgs ca) {
  const OpBatch &ob = pl->ob[2];
  const int w = blockIdx.x;
  const int sec = (ob.total + 7) & ~7;
  if (w < sec) {
    const int tile = section_tile(w, ob.total);
    if (tile < 0) return;
    const TileCtx x{H, gH, lr, dq, nullptr};
    run_op(ob, tile, x, true);
    return;
  }
  const int nyy = (ma.m * ma.m + 255) / 256;
  const int u = w - sec;
  if (u < nyy) {
    if (ma.K > 0)
      yy_entry(u * 256 + threadIdx.x, ma.m, ma.K, ma.srow, ma.sval, ma.scnt, ma.YY);
    else if (u * 256 + (int)threadIdx.x < ma.m * ma.m)
      ma.YY[u * 256 + threadIdx.x] = 0.f;
    return;
  }
  if (u == nyy) {  // the loss, summed in a fixed order
    __shared__ float red[256];
    float s = 0.f;
    for (int j = threadIdx.x; j < ma.m; j += 256) s += ma.lvec[j];
    red[threadIdx.x] = s;
    __syncthreads();
    for (int h = 128; h > 0; h >>= 1) {
      if ((int)threadIdx.x < h) red[threadIdx.x] += red[threadIdx.x + h];
      __syncthreads();
    }
    if (threadIdx.x == 0) {
      const float L = red[0];
      *ma.loss_out = L;
      if (!isfinite(L)) atomicOr(ma.flag, FLAG_NONFINITE);
    }
    return;
  }
  if (u == nyy + 1) cert_task(ca, lr);
}

// ---------------------------------------------------------------------------
// Launch 4: Zq, R X and the U update.  Launch 5: the Q and U^{-T} updates and the
// V scatter.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void step_mid_kernel(const StepPlan *__restrict__ pl,
                                                       const float *H, float *gH, float lr,
                                                       const float *dq,
                                                       const float *__restrict__ coef,
                                                       const int *__restrict__ cert,
                                                       const int *__restrict__ flag) {
  const OpBatch &ob = pl->ob[3];
  const int w = blockIdx.x;
  const int sec = (ob.total + 7) & ~7;
  if (w < sec) {
    const int tile = section_tile(w, ob.total);
    if (tile < 0) return;
    __shared__ float sc[8];
    if (threadIdx.x < 8) sc[threadIdx.x] = coef[threadIdx.x];
    const bool ok = *cert != 0;
    __syncthreads();
    const TileCtx x{H, gH, lr, dq, sc};
    run_op(ob, tile, x, ok);
    return;
  }
  const GemmBatch &gb = pl->gb_mid;
  const int w2 = w - sec;
  if (w2 >= gb.total_tiles) return;
  gemm_body<4>(gb, H, gH, lr, flag, w2);
}

__global__ __launch_bounds__(256) void step_update_kernel(const StepPlan *__restrict__ pl,
                                                          const float *H, float *gH, float lr,
                                                          const int *__restrict__ flag, int n,
                                                          int K, int d,
                                                          const int *__restrict__ idx,
                                                          const float *__restrict__ wA,
                                                          const float *__restrict__ RX, float *V,
                                                          int64_t ldv) {
  const GemmBatch &gb = pl->gb_update;
  const int w = blockIdx.x;
  const int sec = (gb.total_tiles + 7) & ~7;
  if (w < sec) {
    if (w >= gb.total_tiles) return;
    gemm_body<4>(gb, H, gH, lr, flag, w);
    return;
  }
  extern __shared__ int sh[];
  if (*flag != 0) return;
  // V_r -= sum over the row's slots of (dl/dA_kj / (2 dl/dq_j)) (R X)_j
  scatter_slot<256>(w - sec, n, K, d, 1.f, idx, wA, RX, V, ldv, sh);
}

}  // namespace

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------
namespace {

Op16 op(int M, int N, int K, const float *A, int64_t lda, int tA, const float *B, int64_t ldb,
        int tB, float *C, int64_t ldc) {
  Op16 g{};
  g.M = M;
  g.N = N;
  g.K = K;
  g.amode = AM_PLAIN;
  g.A = A;
  g.lda = lda;
  g.tA = tA;
  g.nb = 1;
  g.b[0] = OpTerm{B, ldb, tB, SC_NONE, -1};
  g.alpha = 1.f;
  g.C = C;
  g.ldc = ldc;
  g.alt = -1;
  return g;
}

void finalize(OpBatch &ob, int n_main) {
  int total = 0;
  for (int q = 0; q < ob.n; ++q) {
    Op16 &g = ob.op[q];
    g.tiles_m = (g.M + 15) / 16;
    g.tiles_n = (g.N + 15) / 16;
    if (q < n_main) {
      g.tile_begin = total;
      if (g.M > 0 && g.N > 0) total += g.tiles_m * g.tiles_n;
    }
  }
  for (int q = 0; q < ob.n; ++q)
    if (q >= n_main || ob.op[q].M <= 0 || ob.op[q].N <= 0) ob.op[q].tile_begin = total;
  ob.total = total;
  ob.n_main = n_main;
}

}  // namespace

void build_step_plan(const StepBufs &sb, int m, StepPlan &pl) {
  pl = StepPlan{};
  const int d = sb.d, ldd = sb.ldd;
  const bool sq = sb.loss == LST_LOSS_SQUARED;
  const float *H = sym_H();
  float *gH = sym_gradH();
  const int T = (d + 15) / 16;
  (void)T;
  // Launch 1: H^ = H Q (row partials h . h^ -> qpart), H~ = H U^T, X = H U^{-T T}, N = H H^T
  {
    OpBatch &ob = pl.ob[0];
    ob.op[0] = op(m, d, d, H, d, 0, sb.Q, ldd, 0, sb.Hhat, d);
    ob.op[0].rowred = RR_DOT;
    ob.op[0].Rr = H;
    ob.op[0].ldrr = d;
    ob.op[0].rowout = sb.qpart;
    ob.op[1] = op(m, d, d, H, d, 0, sb.U, ldd, 0, sb.Htil, d);
    ob.op[2] = op(m, d, d, H, d, 0, sb.UinvT, ldd, 0, sb.X, d);
    ob.op[3] = op(m, m, d, H, d, 0, H, d, 0, sb.N, m);
    ob.n = 4;
    finalize(ob, 4);
  }
  // Launch 2: M^ = H H^^T; E^2 = 4 eta^2 S N D N S (|row| partials -> bpart);
  // W1 = E Xs = 2 eta S N D X
  {
    OpBatch &ob = pl.ob[1];
    ob.op[0] = op(m, m, d, H, d, 0, sb.Hhat, d, 0, sb.Mhat, m);
    ob.op[1] = op(m, m, m, sb.N, m, 0, sb.N, m, 0, sb.E2, m);
    ob.op[1].alpha = 4.f;
    ob.op[1].alpha_lr = 2;
    ob.op[1].rowred = RR_ABS;
    ob.op[1].rowout = sb.bpart;
    ob.op[2] = op(m, d, m, sb.N, m, 0, sb.X, d, 1, sb.W1, d);
    ob.op[2].alpha = 2.f;
    ob.op[2].alpha_lr = 1;
    if (!sq) {
      ob.op[1].b[0].sc = SC_DQ;
      ob.op[1].rs = ob.op[1].cs = SC_SQRT;
      ob.op[2].b[0].sc = SC_DQ;
      ob.op[2].rs = SC_SQRT;
    }
    ob.n = 3;
    finalize(ob, 3);
  }
  // Launch 3: Z^ = G U with grad_H = 2 D H^ + Z^; HZ = H~ G^T; E^4 = E^2 E^2;
  // P2 = E^2 Xs; P3 = E^2 W1
  {
    OpBatch &ob = pl.ob[2];
    Op16 z = op(m, d, d, sb.G, d, 0, sb.U, ldd, 1, nullptr, d);
    z.C2 = gH;
    z.ldc2 = d;
    z.E = sb.Hhat;
    z.lde = d;
    z.rs2 = sq ? SC_NONE : SC_DQ;
    ob.op[0] = z;
    ob.op[1] = op(m, m, d, sb.Htil, d, 0, sb.G, d, 0, sb.HZ, m);
    ob.op[2] = op(m, m, m, sb.E2, m, 0, sb.E2, m, 1, sb.E4, m);
    ob.op[3] = op(m, d, m, sb.E2, m, 0, sb.X, d, 1, sb.P2, d);
    if (!sq) ob.op[3].b[0].sc = SC_SQRT;
    ob.op[4] = op(m, d, m, sb.E2, m, 0, sb.W1, d, 1, sb.P3, d);
    ob.n = 5;
    finalize(ob, 5);
  }
  // Launch 4: Zq = (eta^2/2) M H - eta grad_H (M assembled as it is loaded);
  // R X = 2 eta S (c0 Xs + c1 W1 + c2 P2 + c3 P3 + E^4 (c4 Xs + c5 W1 + c6 P2 + c7 P3)),
  // or R X with the exact R when the polynomial is not certified.
  {
    OpBatch &ob = pl.ob[3];
    Op16 zq = op(m, d, m, nullptr, 0, 0, H, d, 1, sb.Zq, d);
    zq.amode = AM_MASM;
    zq.Mh = sb.Mhat;
    zq.HZ = sb.HZ;
    zq.YY = sb.YY;
    zq.ldm = m;
    zq.alpha = 0.5f;
    zq.alpha_lr = 2;
    zq.Cin = gH;
    zq.ldcin = d;
    zq.beta = -1.f;
    zq.beta_lr = 1;
    ob.op[0] = zq;
    const int xsc = sq ? SC_NONE : SC_SQRT;
    Op16 rx = op(m, d, m, sb.E4, m, 0, sb.X, d, 1, sb.RX, d);
    rx.nb = 4;
    rx.b[0] = OpTerm{sb.X, d, 1, xsc, 4};
    rx.b[1] = OpTerm{sb.W1, d, 1, SC_NONE, 5};
    rx.b[2] = OpTerm{sb.P2, d, 1, SC_NONE, 6};
    rx.b[3] = OpTerm{sb.P3, d, 1, SC_NONE, 7};
    rx.nadd = 4;
    rx.add[0] = OpTerm{sb.X, d, 0, xsc, 0};
    rx.add[1] = OpTerm{sb.W1, d, 0, SC_NONE, 1};
    rx.add[2] = OpTerm{sb.P2, d, 0, SC_NONE, 2};
    rx.add[3] = OpTerm{sb.P3, d, 0, SC_NONE, 3};
    rx.alpha = 2.f;
    rx.alpha_lr = 1;
    rx.rs = xsc;
    rx.alt = 2;
    ob.op[1] = rx;
    ob.op[2] = op(m, d, m, sb.R, m, 0, sb.X, d, 1, sb.RX, d);  // exact R
    ob.n = 3;
    finalize(ob, 2);
    GemmBatch &gb = pl.gb_mid;
    // U <- U - (2 eta D H~)^T H
    gb.d[0] = gemm_desc(d, d, m, sb.Atil, d, 1, H, d, 1, sb.U, ldd, -1.f, sb.U, ldd, 1.f);
    gb.n = 1;
    gemm_prepare(gb);
  }
  // Launch 5: Q <- Q + H^T Zq + Zq^T H; U^{-T} <- U^{-T} + (R X)^T H
  {
    GemmBatch &gb = pl.gb_update;
    GemmDesc qd = gemm_desc(d, d, m, H, d, 1, sb.Zq, d, 1, sb.Q, ldd, 1.f, sb.Q, ldd, 1.f);
    qd.A2 = sb.Zq;
    qd.lda2 = d;
    qd.B2 = H;
    qd.ldb2 = d;
    qd.K2 = m;
    gb.d[0] = gemm_desc(d, d, m, sb.RX, d, 1, H, d, 1, sb.UinvT, ldd, 1.f, sb.UinvT, ldd, 1.f);
    gb.d[1] = qd;
    gb.n = 2;
    gemm_prepare(gb);
  }
}

void step_launch_sizes(const StepPlan &pl, int m, int K, int (&grid)[5]) {
  auto sec = [](int n) { return (n + 7) & ~7; };
  grid[0] = sec(pl.ob[0].total) + m;
  grid[1] = sec(m) + sec(pl.ob[1].total);
  grid[2] = sec(pl.ob[2].total) + (m * m + 255) / 256 + 2;
  grid[3] = sec(pl.ob[3].total) + pl.gb_mid.total_tiles;
  grid[4] = sec(pl.gb_update.total_tiles) + m * K;
}

void enqueue_step_launch(int which, const StepBufs &sb, const StepPlan &host, const StepPlan *dev,
                         const StepArgs &a, hipStream_t s) {
  int grid[5];
  step_launch_sizes(host, a.m, a.K, grid);
  const float *dqp = sb.loss == LST_LOSS_SQUARED ? nullptr : sb.dq;
  switch (which) {
    case 0:
      LST_LAUNCH(step_contract_kernel, dim3(grid[0]), dim3(256), 0, s, dev, a.H, a.lr, a.idx, a.K,
                 sb.V, sb.ldv, sb.D, sb.d, a.m);
      break;
    case 1: {
      GatherArgs ga{};
      ga.K = a.K;
      ga.d = sb.d;
      ga.m = a.m;
      ga.T = (sb.d + 15) / 16;
      ga.D = sb.D;
      ga.H = a.H;
      ga.Htil = sb.Htil;
      ga.qpart = sb.qpart;
      ga.idx = a.idx;
      ga.val = a.val;
      ga.V = sb.V;
      ga.ldv = sb.ldv;
      ga.loss = sb.loss;
      ga.eps = sb.eps;
      ga.lr = a.lr;
      ga.G = sb.G;
      ga.Atil = sb.Atil;
      ga.dq = sb.dq;
      ga.dA = sb.dA;
      ga.wA = sb.wA;
      ga.lvec = sb.lvec;
      ga.srow = sb.srow;
      ga.sval = sb.sval;
      ga.scnt = sb.scnt;
      ga.flag = sb.flag;
      const int kpw = (a.K + 3) / 4;
      const int d = sb.d;
#define LST_GATHER(KPW, NV)                                                                        \
  if (kpw <= KPW && d <= 64 * NV) {                                                                \
    LST_LAUNCH((step_gather_kernel<KPW, NV>), dim3(grid[1]), dim3(256), 0, s, dev, a.H, a.lr, ga); \
    break;                                                                                         \
  }
      LST_GATHER(1, 8)
      LST_GATHER(2, 8)
      LST_GATHER(4, 8)
      LST_GATHER(1, 16)
      LST_GATHER(2, 16)
#undef LST_GATHER
      LST_LAUNCH((step_gather_kernel<0, 0>), dim3(grid[1]), dim3(256), 0, s, dev, a.H, a.lr, ga);
      break;
    }
    case 2: {
      MidArgs ma{a.m, a.K, sb.srow, sb.sval, sb.scnt, sb.YY, sb.lvec, a.loss, sb.flag};
      CertArgs ca{a.m, sb.bpart, sb.N, dqp, sb.Cwork, sb.R, sb.coef, sb.cert, sb.flag};
      LST_LAUNCH(step_zgrad_kernel, dim3(grid[2]), dim3(256), 0, s, dev, a.H, a.gH, a.lr, dqp, ma,
                 ca);
      break;
    }
    case 3:
      LST_LAUNCH(step_mid_kernel, dim3(grid[3]), dim3(256), 0, s, dev, a.H, a.gH, a.lr, dqp,
                 sb.coef, sb.cert, sb.flag);
      break;
    default:
      LST_LAUNCH(step_update_kernel, dim3(grid[4]), dim3(256), (size_t)(2 * a.m * a.K) * sizeof(int),
                 s, dev, a.H, a.gH, a.lr, sb.flag, a.m * a.K, a.K, sb.d, a.idx, sb.wA, sb.RX, sb.V,
                 sb.ldv);
  }
}

}  // namespace lst
