// The factored minibatch step (Algorithm 3 for squared error, Algorithm 4 for the
// spherical family: dl/ds = 0 for the spherical softmax, every row for the Taylor
// softmax) as five launches on one stream.
//
// Notation (rows are examples: H is m x d, the paper's d x m H transposed):
//   H^ = H Q, H~ = H U^T, X = H U^{-T T}      (Alg. 3 steps 1, 5, 6; Alg. 4 rows 1, 5)
//   q_j = h_j . h^_j (eq. qvec), a_kj = h~_j . V_r (eq. gen-A-fact), the loss epilogue
//   l_j, dl/dq_j, dl/dA_kj, G_j = sum_k dl/dA_kj V_r (the V^T Yring of eq. gen-Zhat-fact)
//   Z^ = G U, grad_H = 2 diag(dl/dq) H^ + Z^ (eq. gen-grad-H-fact)
//   M = 4 D M^ D + Yring^T Yring + 2 D HZ + 2 HZ^T D (eq. gen-M; M^ = H H^^T,
//       HZ = H~ G^T, D = diag(dl/dq))
// With dl/ds (the Taylor softmax; W = V U + 1 omega^T, eq. gen-Wfact): s_j = h_j . w_bar
// and h~_j = h_j . omega (eq. svec, gen-htilde; launch 1), a_kj gains h~_j, Z^ gains
// w_bar ds_j + omega y_bar_j (eq. gen-Zhat-fact; y_bar_j = sum_k dl/dA_kj), HZ gains
// s ds^T + h~ y_bar^T (HZ = H^T Z^), M gains D ds ds^T + ds y_bar^T + y_bar ds^T, and
// launch 5 updates omega and w_bar (eq. gen-update-omega, gen-update-wbar).
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
//   4  Zq; R X; the U update; the scatter's plan (each slot's rank in its row, the
//      slots ordered by row)                                   [writes U]
//   5  the Q, U^{-T} (and omega, w_bar) updates; the V scatter [writes Q, U^{-T}, V]
// Q, U, U^{-T}, V, omega and w_bar are read (launches 1-3) before any of them is
// written (launches 4-5), and every error is raised by launch 3 at the latest; launches 4
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

// dl/dq_j with T = the sum of the example's target weights over its valid slots (in
// slot order): 1 for squared error, T / (q_j + D eps) for the spherical softmax,
// T / (2 D + 2 s_j + q_j) for the Taylor softmax.
__device__ __forceinline__ float dq_of(int loss, float q, float s, float tsum, float Dn,
                                       float eps) {
  if (loss == LST_LOSS_SQUARED) return 1.f;
  if (loss == LST_LOSS_TAYLOR_SOFTMAX) return tsum / (2.f * Dn + 2.f * s + q);
  return tsum / (q + Dn * eps);
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
// through LDS in a fixed order.  Loads of up to eight k-blocks (the G of op16_kloop)
// are issued before their products.
// ---------------------------------------------------------------------------

struct TileCtx {
  const float *H;
  float *gH;
  float lr;
  const float *dq;    // dl/dq for the scale modes (may be null when no term scales)
  const float *coef;  // polynomial coefficients, or null
};

__device__ __forceinline__ float coef_of(const TileCtx &x, int c) { return c < 0 ? 1.f : x.coef[c]; }

// Four consecutive k values (k0 .. k0 + 3, all below the end of k) of index idx of
// a source, by operand access mode: LV contiguous in k and 16-byte aligned (one
// vector load), LS contiguous in k, LT k-major (p[k ld + idx]).
enum : int { LV = 0, LS = 1, LT = 2 };

template <int MODE>
__device__ __forceinline__ void ld4f(const float *__restrict__ p, int64_t ld, int idx, int k0,
                                     float (&o)[4]) {
  if constexpr (MODE == LV) {
    const float4 v = *reinterpret_cast<const float4 *>(p + (int64_t)idx * ld + k0);
    o[0] = v.x;
    o[1] = v.y;
    o[2] = v.z;
    o[3] = v.w;
  } else if constexpr (MODE == LS) {
    const float *q = p + (int64_t)idx * ld + k0;
    o[0] = q[0];
    o[1] = q[1];
    o[2] = q[2];
    o[3] = q[3];
  } else {
    const float *q = p + (int64_t)k0 * ld + idx;
    o[0] = q[0];
    o[1] = q[ld];
    o[2] = q[2 * ld];
    o[3] = q[3 * ld];
  }
}

template <int MODE>
__device__ __forceinline__ void ld4m(const float *__restrict__ p, int64_t ld, int idx, int k0,
                                     int kend, float (&o)[4]) {
  if (k0 + 3 < kend) {
    ld4f<MODE>(p, ld, idx, k0, o);
    return;
  }
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const int k = min(k0 + s, kend - 1);
    const float v = MODE == LT ? p[(int64_t)k * ld + idx] : p[(int64_t)idx * ld + k];
    o[s] = (k0 + s < kend) ? v : 0.f;
  }
}

// The operand values of one k-block for one lane: a (A row ia) and b (the B terms
// combined, column jb) at k = k0 .. k0 + 3; MASKED: the block may pass the end of k.
template <int AMODE, int NB, bool SC, int AMD, int BMD, bool MASKED>
__device__ __forceinline__ void op16_block(const Op16 &g, const float *A, const float *const *Bp,
                                           const float *bco, float dqi, float dsi, float ybi,
                                           int ia, int jb, int k0, const TileCtx &x,
                                           float (&a)[4], float (&b)[4]) {
  const int K = g.K;
  if constexpr (AMODE != AM_PLAIN) {
    // M_ik = 4 dq_i M^_ik dq_k + YY_ik + 2 dq_i HZ_ik + 2 dq_k HZ_ki
    float mh[4], yy[4], hz[4], hzt[4], dk[4];
    ld4m<LS>(g.Mh, g.ldm, ia, k0, K, mh);
    ld4m<LS>(g.YY, g.ldm, ia, k0, K, yy);
    ld4m<LS>(g.HZ, g.ldm, ia, k0, K, hz);
    ld4m<LT>(g.HZ, g.ldm, ia, k0, K, hzt);
    if (x.dq) {
      ld4m<LS>(x.dq, 0, 0, k0, K, dk);
    } else {
      dk[0] = dk[1] = dk[2] = dk[3] = 1.f;
    }
#pragma unroll
    for (int s = 0; s < 4; ++s)
      a[s] = 4.f * dqi * mh[s] * dk[s] + yy[s] + 2.f * dqi * hz[s] + 2.f * dk[s] * hzt[s];
    if constexpr (AMODE == AM_MASM_S) {
      // + D ds_i ds_k + ds_i yb_k + yb_i ds_k
      float sk[4], yk[4];
      ld4m<LS>(g.ds, 0, 0, k0, K, sk);
      ld4m<LS>(g.yb, 0, 0, k0, K, yk);
#pragma unroll
      for (int s = 0; s < 4; ++s) a[s] += dsi * fmaf(g.Dn, sk[s], yk[s]) + ybi * sk[s];
    }
  } else if constexpr (MASKED) {
    ld4m<AMD>(A, g.lda, ia, k0, K, a);
  } else {
    ld4f<AMD>(A, g.lda, ia, k0, a);
  }
#pragma unroll
  for (int t = 0; t < NB; ++t) {
    float v[4];
    if constexpr (MASKED)
      ld4m<BMD>(Bp[t], g.b[t].ld, jb, k0, K, v);
    else
      ld4f<BMD>(Bp[t], g.b[t].ld, jb, k0, v);
    if constexpr (SC) {
      if (g.b[t].sc != SC_NONE) {
        float sv[4];
        if constexpr (MASKED) {
#pragma unroll
          for (int s = 0; s < 4; ++s) sv[s] = x.dq[min(k0 + s, K - 1)];
        } else {
          ld4f<LV>(x.dq, 0, 0, k0, sv);
        }
#pragma unroll
        for (int s = 0; s < 4; ++s) v[s] *= g.b[t].sc == SC_DQ ? sv[s] : sqrtf(sv[s]);
      }
    }
#pragma unroll
    for (int s = 0; s < 4; ++s) b[s] = t == 0 ? bco[0] * v[s] : fmaf(bco[t], v[s], b[s]);
  }
}

// Row partial sums of a tile (v Rr_ij, or |v|) over its 16 columns into
// rowout[tile column][i]; with qout, the last tile of the row block to finish sums
// the row's partials into qout[i].
__device__ __forceinline__ void rowred_epilogue(const Op16 &g, float v, bool ok, float rrv, int oi,
                                                int c, int tm, int tn, int i0) {
  if (g.rowred != RR_NONE) {
    float r = 0.f;
    if (ok) r = g.rowred == RR_DOT ? v * rrv : fabsf(v);
    // the 16 lanes of this row (same g, same wavefront), in a fixed order
    r += __shfl_xor(r, 1);
    r += __shfl_xor(r, 2);
    r += __shfl_xor(r, 4);
    r += __shfl_xor(r, 8);
    if (c == 0 && oi < g.M) {
      float *dst = g.rowout + (int64_t)tn * g.M + oi;
      if (g.qout)  // read by another workgroup of this launch, possibly on another XCD
        __hip_atomic_store(dst, r, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      else
        *dst = r;
    }
    if (g.qout) {
      // Arrival after this workgroup's partials are complete (each thread waits for
      // its own stores); the last of the row block's tiles_n arrivals sums them.
      __shared__ int last;
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();
      if (threadIdx.x == 0)
        last = __hip_atomic_fetch_add(g.qcnt + tm, 1, __ATOMIC_RELAXED,
                                      __HIP_MEMORY_SCOPE_AGENT) == g.tiles_n - 1;
      __syncthreads();
      if (last) {
        // row i0 + threadIdx.x / 16: lane l sums the partials l, l + 16, ... in order,
        // then the 16 lanes are added pairwise in a fixed pattern
        const int i = i0 + (int)(threadIdx.x >> 4), l = threadIdx.x & 15;
        float q = 0.f;
        if (i < g.M)
          for (int t = l; t < g.tiles_n; t += 16)
            q += __hip_atomic_load(g.rowout + (int64_t)t * g.M + i, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
        q += __shfl_xor(q, 1);
        q += __shfl_xor(q, 2);
        q += __shfl_xor(q, 4);
        q += __shfl_xor(q, 8);
        if (l == 0 && i < g.M) g.qout[i] = q;
      }
    }
  }
}

// The k loop of one tile, specialised at compile time: AMODE (plain or assembled M),
// NB (B terms: 1 or kMaxTerms), SC (B terms scaled by dl/dq), G (k-blocks whose loads
// are issued before their products; smaller where a block needs more registers, so
// that the kernels keep four wavefronts per SIMD without spilling), AMD / BMD (the
// operands' access modes).  The four wavefronts take the whole k-blocks of 16 in turn;
// the ragged end of k (K mod 16) is one more masked block, taken by wavefront 3.
template <int AMODE, int NB, bool SC, int G, int AMD, int BMD>
__device__ __forceinline__ floatx4 op16_kloop(const Op16 &g, int ia, int jb, const TileCtx &x,
                                              int wave, int lg) {
  const int K = g.K;
  const float *A = rsv(g.A, x.H, x.gH);
  const float *Bp[NB];
  float bco[NB];
#pragma unroll
  for (int t = 0; t < NB; ++t) {
    Bp[t] = rsv(g.b[t].p, x.H, x.gH);
    bco[t] = NB > 1 ? coef_of(x, g.b[t].coef) : 1.f;
  }
  const float dqi = (AMODE != AM_PLAIN && x.dq) ? x.dq[ia] : 1.f;
  const float dsi = AMODE == AM_MASM_S ? g.ds[ia] : 0.f;
  const float ybi = AMODE == AM_MASM_S ? g.yb[ia] : 0.f;
  floatx4 acc = {0.f, 0.f, 0.f, 0.f};
  const int nfull = K >> 4;
  const int nw = nfull > wave ? (nfull - wave + 3) / 4 : 0;
  for (int u0 = 0; u0 < nw; u0 += G) {
    float a[G][4], b[G][4];
#pragma unroll
    for (int u = 0; u < G; ++u) {
      const int k0 = 16 * (wave + 4 * min(u0 + u, nw - 1)) + 4 * lg;
      op16_block<AMODE, NB, SC, AMD, BMD, false>(g, A, Bp, bco, dqi, dsi, ybi, ia, jb, k0, x,
                                                 a[u], b[u]);
    }
#pragma unroll
    for (int u = 0; u < G; ++u)
      if (u0 + u < nw) {
#pragma unroll
        for (int s = 0; s < 4; ++s)
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[u][s], b[u][s], acc, 0, 0, 0);
      }
  }
  if ((K & 15) && wave == 3) {
    float a[4], b[4];
    op16_block<AMODE, NB, SC, AMD, BMD, true>(g, A, Bp, bco, dqi, dsi, ybi, ia, jb,
                                               16 * nfull + 4 * lg, x, a, b);
#pragma unroll
    for (int s = 0; s < 4; ++s) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[s], b[s], acc, 0, 0, 0);
  }
  return acc;
}

template <int AMODE, int NB, bool SC, int G>
__device__ __forceinline__ floatx4 op16_dispatch(const Op16 &g, int ia, int jb, const TileCtx &x,
                                                 int wave, int lg) {
  if constexpr (AMODE != AM_PLAIN || NB > 1) {
    // assembled M or several B terms: every B term k-major (the plan builder's layout)
    return op16_kloop<AMODE, NB, SC, G, LS, LT>(g, ia, jb, x, wave, lg);
  } else {
    const bool av = vec_ok(rsv(g.A, x.H, x.gH), g.lda);
    const int bm = g.b[0].tr ? LT : (vec_ok(rsv(g.b[0].p, x.H, x.gH), g.b[0].ld) ? LV : LS);
    if (av) {
      if (bm == LV) return op16_kloop<AMODE, NB, SC, G, LV, LV>(g, ia, jb, x, wave, lg);
      if (bm == LS) return op16_kloop<AMODE, NB, SC, G, LV, LS>(g, ia, jb, x, wave, lg);
      return op16_kloop<AMODE, NB, SC, G, LV, LT>(g, ia, jb, x, wave, lg);
    }
    if (bm == LV) return op16_kloop<AMODE, NB, SC, G, LS, LV>(g, ia, jb, x, wave, lg);
    if (bm == LS) return op16_kloop<AMODE, NB, SC, G, LS, LS>(g, ia, jb, x, wave, lg);
    return op16_kloop<AMODE, NB, SC, G, LS, LT>(g, ia, jb, x, wave, lg);
  }
}

__device__ __forceinline__ void op16_tile(const Op16 &g, int local, const TileCtx &x) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = lane & 15, lg = lane >> 4;
  // column-major tile order: consecutive tiles share a B panel (and so an XCD's L2)
  const int tn = local / g.tiles_m, tm = local - tn * g.tiles_m;
  const int i0 = tm * 16, j0 = tn * 16;
  const int ia = min(i0 + c, g.M - 1), jb = min(j0 + c, g.N - 1);
  // Output of this thread after the reduction: accumulator register `wave` of lane
  // `lane`.  Its epilogue operands are loaded before the k loop, so that their
  // latency overlaps it.
  const int oi = i0 + 4 * lg + wave, oj = j0 + c;
  const bool ok = oi < g.M && oj < g.N;
  const int ci = min(oi, g.M - 1), cj = min(oj, g.N - 1);
  float addv[kMaxTerms];
#pragma unroll
  for (int t = 0; t < kMaxTerms; ++t)
    addv[t] = t < g.nadd ? rsv(g.add[t].p, x.H, x.gH)[(int64_t)ci * g.add[t].ld + cj] : 0.f;
  const float cinv = g.Cin ? rsv(g.Cin, x.H, x.gH)[(int64_t)ci * g.ldcin + cj] : 0.f;
  const float ev = g.C2 ? rsv(g.E, x.H, x.gH)[(int64_t)ci * g.lde + cj] : 0.f;
  const float rrv = g.rowred == RR_DOT ? rsv(g.Rr, x.H, x.gH)[(int64_t)ci * g.ldrr + cj] : 0.f;

  floatx4 acc;
  if (g.amode == AM_MASM)
    acc = op16_dispatch<AM_MASM, 1, false, 2>(g, ia, jb, x, wave, lg);
  else if (g.amode == AM_MASM_S)
    acc = op16_dispatch<AM_MASM_S, 1, false, 1>(g, ia, jb, x, wave, lg);
  else if (g.nb > 1)
    acc = op16_dispatch<AM_PLAIN, kMaxTerms, true, 2>(g, ia, jb, x, wave, lg);
  else if (g.b[0].sc != SC_NONE)
    acc = op16_dispatch<AM_PLAIN, 1, true, 4>(g, ia, jb, x, wave, lg);
  else
    acc = op16_dispatch<AM_PLAIN, 1, false, 8>(g, ia, jb, x, wave, lg);

  __shared__ float red[4][4][64];
#pragma unroll
  for (int r = 0; r < 4; ++r) red[wave][r][lane] = acc[r];
  __syncthreads();
  float v = (red[0][wave][lane] + red[1][wave][lane]) + (red[2][wave][lane] + red[3][wave][lane]);
  __syncthreads();  // red is reused by the next tile of this workgroup
#pragma unroll
  for (int t = 0; t < kMaxTerms; ++t) {
    if (t >= g.nadd) break;
    v = fmaf(coef_of(x, g.add[t].coef) * scale_of(g.add[t].sc, x.dq, ci), addv[t], v);
  }
  // the rank-nuv addend (only the dl/ds products have one: loaded here, not before the
  // k loop, to keep the other products' registers)
  for (int r = 0; r < g.nuv; ++r)
    v = fmaf(g.ux[r][(int64_t)ci * g.uxi[r]], g.uy[r][(int64_t)cj * g.uyi[r]], v);
  float al = g.alpha;
  for (int e = 0; e < g.alpha_lr; ++e) al *= x.lr;
  v *= al * scale_of(g.rs, x.dq, ci) * scale_of(g.cs, x.dq, cj);
  if (g.Cin) {
    float be = g.beta;
    for (int e = 0; e < g.beta_lr; ++e) be *= x.lr;
    v = fmaf(be, cinv, v);
  }
  if (ok) {
    if (g.C) const_cast<float *>(rsv(g.C, x.H, x.gH))[(int64_t)oi * g.ldc + oj] = v;
    if (g.C2)
      const_cast<float *>(rsv(g.C2, x.H, x.gH))[(int64_t)oi * g.ldc2 + oj] =
          2.f * scale_of(g.rs2, x.dq, oi) * ev + v;
  }
  rowred_epilogue(g, v, ok, rrv, oi, c, tm, tn, i0);
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

// The same with each product split over the XCDs on its own: XCD x owns a contiguous
// eighth of every product's tiles, so that products of different k lengths spread
// evenly over the chip.  section_by_op: the section's workgroups.
template <class B>  // OpBatch or OpHdr
__host__ __device__ __forceinline__ int section_by_op(const B &ob) {
  int n = 0;
  for (int q = 0; q < kMaxOps; ++q)
    if (q < ob.n_main) n += (ob.count[q] + 7) >> 3;
  return 8 * n;
}

template <class B>
__device__ __forceinline__ int tile_by_op(const B &ob, int w) {
  const int x = w & 7;
  int s = w >> 3;
#pragma unroll
  for (int q = 0; q < kMaxOps; ++q) {
    if (q >= ob.n_main) break;
    const int T = ob.count[q], c8 = T >> 3, r = T & 7;
    const int c = x < r ? c8 + 1 : c8;
    if (s < c) return ob.begin[q] + (x < r ? x * (c8 + 1) : r * (c8 + 1) + (x - r) * c8) + s;
    s -= c;
  }
  return -1;
}

// Tile `tile` of a batch of Op16 (the descriptor whose range holds it); alt
// descriptors replace theirs when the polynomial is not certified.
__device__ __forceinline__ void run_op(const OpHdr &hd, const Op16 *ops, int tile, const TileCtx &x,
                                       bool cert) {
  int di = 0;
#pragma unroll
  for (int q = 1; q < kMaxOps; ++q)
    if (q < hd.n_main && tile >= hd.begin[q]) di = q;
  const Op16 *g = &ops[di];
  const int local = tile - hd.begin[di];
  if (!cert && g->alt >= 0) g = &ops[g->alt];
  op16_tile(*g, local, x);
}

// The step's products on 32 x 32 tiles (GT = 32, KS k-blocks of 8 in flight per wave)
// or on LDS-staged 64 x 64 tiles (GT = 64, large shapes).
template <int GT, int KS, bool TERMS = false, class Hd>
__device__ __forceinline__ void step_gemm(const GemmBatch &bt, const Hd &hd, const float *H,
                                          float *gH, float lr, const int *gate, int w,
                                          const int *cert = nullptr) {
  if constexpr (GT == 64)
    gemm_body64<TERMS>(bt, hd, H, gH, lr, gate, w, cert);
  else
    gemm_body<4, KS>(bt, hd, H, gH, lr, gate, w);
}

// ---------------------------------------------------------------------------
// Launch 1: contractions, N, prefetch of the target rows.  GT: the tile edge of the
// products in gb_contract.
// ---------------------------------------------------------------------------
template <int GT>
__global__ __launch_bounds__(256, 4) void step_contract_kernel(
    const StepPlan *__restrict__ pl, const OpHdr hd, const GemmHdr gh, const float *H, float lr,
    const int *__restrict__ idx,
    const float *__restrict__ val, int K, const float *__restrict__ V, int64_t ldv, int64_t D,
    int d, int m, float *__restrict__ tsum) {
  int w = blockIdx.x;
  // the products on 32 x 32 or 64 x 64 tiles (large shapes) first: their workgroups are
  // the long ones, and dispatched after the 16 x 16 tiles they would start only as those
  // end
  const int gsec = gemm_section(gh, GT);
  if (w < gsec) {
    if (GT == 64 || w < gh.total_tiles)
      step_gemm<GT, 4>(pl->gb_contract, gh, H, nullptr, lr, nullptr, w);
    return;
  }
  w -= gsec;
  const int sec = (hd.total + 7) & ~7;
  if (w < sec) {
    const int tile = section_tile(w, hd.total);
    if (tile < 0) return;
    const TileCtx x{H, nullptr, lr, nullptr, nullptr};
    run_op(hd, pl->ob[0].op, tile, x, true);
    return;
  }
  w -= sec;
  // Prefetch workgroup of example j (XCD j % 8, that of its gather workgroup in
  // launch 2): the indices, then one load per 128-byte line of every target row;
  // also the sum of the example's target weights over its valid slots, in slot order.
  const int j = w;
  if (j >= m) return;
  __shared__ int prow[LST_MAX_K];
  __shared__ float pval[LST_MAX_K];
  for (int k = threadIdx.x; k < K; k += 256) {
    const int r = idx[(int64_t)j * K + k];
    prow[k] = (r < 0 || (int64_t)r >= D) ? -1 : r;
    pval[k] = val[(int64_t)j * K + k];
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float ts = 0.f;
    for (int k = 0; k < K; ++k)
      if (prow[k] >= 0) ts += pval[k];
    tsum[j] = ts;
  }
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
  int K, d, m;
  int64_t D;
  const float *H, *Hhat, *Htil, *q, *tsum;
  int *qcnt;
  int nqcnt;
  const int *idx;
  const float *val;
  const float *V;
  int64_t ldv;
  int loss;
  float eps, lr;
  float *G, *Atil, *dq, *wA, *lvec;
  int *ticket;  // the V scatter's partial-sum ticket (launch 5), zeroed here
  int *srow;
  float *sval;
  int *scnt;
  const float *SW;         // Taylor softmax: s_j, h~_j (launch 1)
  float *ds, *yb, *cwo;    // Taylor softmax: dl/ds, y_bar, the omega / w_bar coefficients
  int *flag;
};

// The Taylor softmax's per-example outputs besides dl/dq and dl/dA: dl/ds_j = 2 dl/dq_j
// (= T / Z), y_bar_j = sum_k dl/dA_kj, and the coefficients of the launch-5 products
// w_bar -= H^T c_w, omega -= H^T c_o: c_w = eta (2 dq s + D ds + y_bar) (eq.
// gen-update-wbar), c_o = eta (2 dq h~ + ds) (eq. gen-update-omega).
__device__ __forceinline__ void taylor_outputs(const GatherArgs &ga, int j, float gq, float sj,
                                               float hw, float ybar) {
  const float gs = 2.f * gq;
  ga.ds[j] = gs;
  ga.yb[j] = ybar;
  ga.cwo[j] = ga.lr * (2.f * gq * sj + (float)ga.D * gs + ybar);
  ga.cwo[ga.m + j] = ga.lr * (2.f * gq * hw + gs);
}

// Loss epilogue of one example (section 4); r[k] < 0 marks an empty slot; a holds
// h~_j . V_r, to which the Taylor softmax adds h~_j = h_j . omega (eq. gen-A-fact).
// l = q - 2 a.t + ||y||^2 (squared error, ||y||^2 by index equality),
// l = sum_k t_k [log(q + D eps) - log(a_k^2 + eps)] (spherical softmax) or
// l = sum_k t_k [log(D + s + q/2) - log(1 + a_k + a_k^2/2)] (Taylor softmax).
__device__ __forceinline__ void epilogue(int loss, float q, float sj, float hw, int K,
                                         const int *r, const float *t, const float *a, float Dn,
                                         float eps, float &l, float *g) {
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
  } else if (loss == LST_LOSS_TAYLOR_SOFTMAX) {
    const float lz = logf(Dn + sj + 0.5f * q);
    for (int k = 0; k < K; ++k) {
      g[k] = 0.f;
      if (r[k] < 0) continue;
      const float ak = a[k] + hw;
      const float f = 1.f + ak + 0.5f * ak * ak;
      l += t[k] * (lz - logf(f));
      g[k] = -t[k] * (1.f + ak) / f;
    }
  } else {
    const float lz = logf(q + Dn * eps);
    for (int k = 0; k < K; ++k) {
      g[k] = 0.f;
      if (r[k] < 0) continue;
      const float den = a[k] * a[k] + eps;
      l += t[k] * (lz - logf(den));
      g[k] = -2.f * t[k] * a[k] / den;
    }
  }
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

// sorted_slots with the example's KM slots in registers (K <= KM).
template <int KM>
__device__ __forceinline__ void sorted_slots_reg(int j, int K, const int *sr, const float *sg,
                                                 int *srow, float *sval, int *scnt) {
  int rr[KM];
  float vv[KM];
#pragma unroll
  for (int k = 0; k < KM; ++k) {
    rr[k] = k < K ? sr[k] : -1;
    vv[k] = k < K ? sg[k] : 0.f;
  }
  bool first[KM];
  int n = 0;
#pragma unroll
  for (int k = 0; k < KM; ++k) {
    bool f = rr[k] >= 0;
#pragma unroll
    for (int k2 = 0; k2 < k; ++k2) f &= rr[k2] != rr[k];
    first[k] = f;
    n += f ? 1 : 0;
  }
  const int k = threadIdx.x;
  if (k < K) {
    int me = -1;
    bool fk = false;
#pragma unroll
    for (int u = 0; u < KM; ++u)
      if (u == k) {
        me = rr[u];
        fk = first[u];
      }
    if (fk) {
      float v = 0.f;
      int pos = 0;
#pragma unroll
      for (int u = 0; u < KM; ++u) {
        if (rr[u] == me) v += vv[u];
        pos += (first[u] && rr[u] < me) ? 1 : 0;
      }
      srow[(int64_t)j * K + pos] = me;
      sval[(int64_t)j * K + pos] = v;
    }
  }
  if (threadIdx.x == 0) scnt[j] = n;
}

// Register-resident form for K <= 4 KPW and d <= 64 NV: wavefront w keeps the
// target rows k = w, w + 4, ... in registers from the dot products a_kj to the G
// sum, so V is read once and the index loads lead straight into the row loads.
// A slot's dl/dA depends on its own a_kj only, so every wavefront forms the
// derivatives of its slots and its share of G_j = sum_k dl/dA_kj V_r without
// waiting for the others (squared error: dl/dA = -2 t, known with the indices);
// the loss, dl/dq and the slot lists follow after the one workgroup barrier.
// The loss is summed per wavefront (slots w, w + 4, ...), then over the wavefronts
// in a fixed order.
template <int KPW, int NV>
__device__ __forceinline__ void gather_reg(const GatherArgs &ga, int j) {
  constexpr int W = 4, KM = W * KPW;
  __shared__ int sr[KM];
  __shared__ float st[KM], sg[KM];
  __shared__ float gpart[W][64 * NV];
  __shared__ float sred[W], slp[W];  // q partials (squared error), loss partials
  __shared__ int sbad[W];
  const int K = ga.K, d = ga.d;
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const bool sq = ga.loss == LST_LOSS_SQUARED, tay = ga.loss == LST_LOSS_TAYLOR_SOFTMAX;
  const float Dn = (float)ga.D;
  // q_j: for squared error h_j . h^_j here (its operands loaded first, used after the
  // target rows' dot products); for the spherical family reduced in launch 1 (its E
  // products need every q_j), loaded with T, s_j and h~_j as uniform values.
  // Also h~_j at the columns this thread writes 2 eta dl/dq_j h~_j to (loaded here: in the
  // loop of those stores, the compiler could not move a load of h~ above the previous
  // column's stores, one round trip per 256 columns).
  constexpr int NQ = (64 * NV + 255) / 256;
  const float *htp = ga.Htil + (int64_t)j * d;
  float qh[NQ], qhh[NQ], hv[NQ];
#pragma unroll
  for (int u = 0; u < NQ; ++u) {
    const int c = t + 256 * u;
    qh[u] = (sq && c < d) ? ga.H[(int64_t)j * d + c] : 0.f;
    qhh[u] = (sq && c < d) ? ga.Hhat[(int64_t)j * d + c] : 0.f;
    hv[u] = c < d ? htp[c] : 0.f;
  }
  // h~_j in the layout of the target rows (lane + 64 n), before the rows' loads, which
  // wait for the indices
  float ht[NV];
#pragma unroll
  for (int n = 0; n < NV; ++n) {
    const int c = lane + 64 * n;
    ht[n] = (c < d) ? htp[c] : 0.f;
  }
  float qv = 0.f, tsv = 0.f, sj = 0.f, hw = 0.f;
  if (!sq) {
    qv = ga.q[j];
    tsv = ga.tsum[j];
    if (tay) {
      sj = ga.SW[2 * j];
      hw = ga.SW[2 * j + 1];
    }
  }
  int r[KPW];
  float tv[KPW];  // the slots' target values, loaded with the indices
  bool bad = false;
#pragma unroll
  for (int i = 0; i < KPW; ++i) {
    const int k = wave + W * i;
    int v = -1;
    tv[i] = 0.f;
    if (k < K) {
      v = ga.idx[(int64_t)j * K + k];
      tv[i] = ga.val[(int64_t)j * K + k];
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
  // the loss's log of the normaliser (spherical family)
  float lz = 0.f;
  if (tay)
    lz = logf(Dn + sj + 0.5f * qv);
  else if (!sq)
    lz = logf(qv + Dn * ga.eps);
  // a_kj, dl/dA_kj and this wavefront's part of the loss (squared error: of sum t a)
  float g[KPW];
  float lpart = 0.f;
#pragma unroll
  for (int i = 0; i < KPW; ++i) {
    float sacc = 0.f;
#pragma unroll
    for (int n = 0; n < NV; ++n) sacc += ht[n] * vr[i][n];
    const float a = wave_sum(sacc) + hw;
    const bool ok = wave + W * i < K && r[i] >= 0;
    float gi = 0.f;
    if (ok) {
      if (sq) {
        gi = -2.f * tv[i];
        lpart += tv[i] * a;
      } else if (tay) {
        const float f = 1.f + a + 0.5f * a * a;
        lpart += tv[i] * (lz - logf(f));
        gi = -tv[i] * (1.f + a) / f;
      } else {
        const float den = a * a + ga.eps;
        lpart += tv[i] * (lz - logf(den));
        gi = -2.f * tv[i] * a / den;
      }
    }
    g[i] = gi;
  }
#pragma unroll
  for (int n = 0; n < NV; ++n) {
    float gv = 0.f;
#pragma unroll
    for (int i = 0; i < KPW; ++i) gv += g[i] * vr[i][n];
    gpart[wave][lane + 64 * n] = gv;
  }
  if (sq) {
    float qs = 0.f;
#pragma unroll
    for (int u = 0; u < NQ; ++u) qs += qh[u] * qhh[u];
    qs = wave_sum(qs);
    if (lane == 0) sred[wave] = qs;
  }
  if (lane == 0) {
#pragma unroll
    for (int i = 0; i < KPW; ++i) {
      const int k = wave + W * i;
      if (k < K) {
        sr[k] = r[i];
        st[k] = tv[i];
        sg[k] = g[i];
      }
    }
    slp[wave] = lpart;
    sbad[wave] = bad ? 1 : 0;
  }
  __syncthreads();
  // G_j and 2 eta dl/dq_j h~_j
  const float gq = dq_of(ga.loss, qv, sj, tsv, Dn, ga.eps);
  const float s2 = 2.f * ga.lr * gq;
#pragma unroll
  for (int u = 0; u < NQ; ++u) {
    const int c = t + 256 * u;
    if (c < d) {
      ga.G[(int64_t)j * d + c] = (gpart[0][c] + gpart[1][c]) + (gpart[2][c] + gpart[3][c]);
      ga.Atil[(int64_t)j * d + c] = s2 * hv[u];
    }
  }
  if (t == 0) {
    if (sbad[0] | sbad[1] | sbad[2] | sbad[3]) atomicOr(ga.flag, FLAG_INDEX);
    float l = (slp[0] + slp[1]) + (slp[2] + slp[3]);
    if (sq) {  // l = q - 2 a.t + ||y||^2, ||y||^2 by index equality
      const float q = (sred[0] + sred[1]) + (sred[2] + sred[3]);
      int rr[KM];
      float tt[KM];
#pragma unroll
      for (int k = 0; k < KM; ++k) {
        rr[k] = k < K ? sr[k] : -1;
        tt[k] = k < K ? st[k] : 0.f;
      }
      float yy = 0.f;
#pragma unroll
      for (int k = 0; k < KM; ++k) {
        if (rr[k] < 0) continue;
#pragma unroll
        for (int kk = 0; kk < KM; ++kk)
          if (rr[kk] == rr[k]) yy += tt[k] * tt[kk];
      }
      l = q - 2.f * l + yy;
    }
    ga.lvec[j] = l;
    ga.dq[j] = gq;
    if (tay) {
      float ybar = 0.f;
#pragma unroll
      for (int k = 0; k < KM; ++k)
        if (k < K) ybar += sg[k];
      taylor_outputs(ga, j, gq, sj, hw, ybar);
    }
  }
  for (int k = t; k < K; k += 256) ga.wA[(int64_t)j * K + k] = gq != 0.f ? sg[k] / (2.f * gq) : 0.f;
  sorted_slots_reg<KM>(j, K, sr, sg, ga.srow, ga.sval, ga.scnt);
}

// General form (any K <= LST_MAX_K, any d): the K dot products spread over the
// wavefronts, then G column-parallel.
__device__ __forceinline__ void gather_gen(const GatherArgs &ga, int j) {
  __shared__ int sr[LST_MAX_K];
  __shared__ float sa[LST_MAX_K], st[LST_MAX_K], sg[LST_MAX_K];
  __shared__ float s_dq;
  __shared__ int s_bad;
  __shared__ float sred[4];
  const int K = ga.K, d = ga.d;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const float *ht = ga.Htil + (int64_t)j * d;
  if (t == 0) s_bad = 0;
  float qv = 0.f, tsv = 0.f;
  if (ga.loss == LST_LOSS_SQUARED) {
    float qs = 0.f;
    for (int c = t; c < d; c += 256) qs += ga.H[(int64_t)j * d + c] * ga.Hhat[(int64_t)j * d + c];
    qs = wave_sum(qs);
    if (lane == 0) sred[wave] = qs;
  } else if (t == 0) {
    qv = ga.q[j];
    tsv = ga.tsum[j];
  }
  const bool tay = ga.loss == LST_LOSS_TAYLOR_SOFTMAX;
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
    const float q = ga.loss == LST_LOSS_SQUARED ? (sred[0] + sred[1]) + (sred[2] + sred[3]) : qv;
    const float sj = tay ? ga.SW[2 * j] : 0.f, hw = tay ? ga.SW[2 * j + 1] : 0.f;
    const float gq = dq_of(ga.loss, q, sj, tsv, (float)ga.D, ga.eps);
    float l;
    epilogue(ga.loss, q, sj, hw, K, sr, st, sa, (float)ga.D, ga.eps, l, sg);
    if (tay) {
      float ybar = 0.f;
      for (int k = 0; k < K; ++k) ybar += sg[k];
      taylor_outputs(ga, j, gq, sj, hw, ybar);
    }
    ga.dq[j] = gq;
    ga.lvec[j] = l;
    s_dq = gq;
  }
  __syncthreads();
  const float gq = s_dq;
  for (int k = t; k < K; k += 256) ga.wA[(int64_t)j * K + k] = gq != 0.f ? sg[k] / (2.f * gq) : 0.f;
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
  const bool tay = ga.loss == LST_LOSS_TAYLOR_SOFTMAX;
  for (int i = threadIdx.x; i < ga.m; i += 256)
    sdq[i] = dq_of(ga.loss, ga.q[i], tay ? ga.SW[2 * i] : 0.f, ga.tsum[i], (float)ga.D, ga.eps);
  __syncthreads();
}

template <int KPW, int NV>
__global__ __launch_bounds__(256, 4) void step_gather_kernel(const StepPlan *__restrict__ pl,
                                                          const OpHdr hd, const float *H, float lr,
                                                          const GatherArgs ga) {
  const int w = blockIdx.x;
  const int gsec = (ga.m + 7) & ~7;
  if (w < gsec) {
    // launch 1 is complete: its q-reduction counters start the next step at zero; the
    // scatter's ticket starts launch 5 at zero
    if (w == 0 && (int)threadIdx.x < ga.nqcnt) ga.qcnt[threadIdx.x] = 0;
    if (w == 0 && threadIdx.x == 0) *ga.ticket = 0;
    if (w >= ga.m) return;
    if constexpr (NV > 0)
      gather_reg<KPW, NV>(ga, w);
    else
      gather_gen(ga, w);
    return;
  }
  const int tile = tile_by_op(hd, w - gsec);
  if (tile < 0) return;
  __shared__ __align__(16) float sdq[LST_MAX_M];
  const float *dq = nullptr;
  if (ga.loss != LST_LOSS_SQUARED) {
    dq_all(ga, sdq);
    dq = sdq;
  }
  const TileCtx x{H, nullptr, lr, dq, nullptr};
  run_op(hd, pl->ob[1].op, tile, x, true);
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
  // (1 + cos((2i + 1) pi / 16)) / 2, i = 0..7: the Chebyshev points of [0, 1]
  const double y[8] = {0.9903926402016152, 0.9157348061512727, 0.7777851165098011, 0.5975451610080642, 0.4024548389919359, 0.22221488349019902, 0.08426519384872733, 0.009607359798384785};
  double f[8];
  for (int i = 0; i < 8; ++i) f[i] = 1.0 / (1.0 - b * y[i]);
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

// Yring^T Yring entry (i, j) = sum over common rows r of (summed dl/dA of i at r) x
// (summed dl/dA of j at r), from the two examples' merged slot lists: chunks of 16
// entries of each list in registers (all loads of a chunk in flight together), every
// pair compared.  The products of a matching pair meet in the same order for (i, j)
// and (j, i) (rows ascending), so the matrix is exactly symmetric.
__device__ __forceinline__ void yy_entry(int e, int m, int K, const int *__restrict__ srow,
                                         const float *__restrict__ sval,
                                         const int *__restrict__ scnt, float *__restrict__ YY) {
  if (e >= m * m) return;
  const int i = e / m, j = e - (e / m) * m;
  const int *ri = srow + (int64_t)i * K, *rj = srow + (int64_t)j * K;
  const float *vi = sval + (int64_t)i * K, *vj = sval + (int64_t)j * K;
  const int na = scnt[i], nb = scnt[j];
  float yy = 0.f;
  for (int a0 = 0; a0 < na; a0 += 16) {
    int ra[16];
    float va[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const bool in = a0 + u < na;
      ra[u] = in ? ri[a0 + u] : -1;
      va[u] = in ? vi[a0 + u] : 0.f;
    }
    for (int b0 = 0; b0 < nb; b0 += 16) {
      int rb[16];
      float vb[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const bool in = b0 + u < nb;
        rb[u] = in ? rj[b0 + u] : -2;
        vb[u] = in ? vj[b0 + u] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < 16; ++u)
#pragma unroll
        for (int v = 0; v < 16; ++v)
          if (ra[u] == rb[v]) yy = fmaf(va[u], vb[v], yy);
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

// GT: the tile edge of the products in gb_zgrad, 0 when it is empty (a separate
// instantiation, so that the other shapes keep the smaller kernel: with the 32 x 32
// section compiled in, the registers and LDS it takes made the step 5 us slower at
// m = 128, d = 500, section empty or not).
template <int GT>
__global__ __launch_bounds__(256, 4) void step_zgrad_kernel(const StepPlan *__restrict__ pl,
                                                         const OpHdr hd, const GemmHdr gh,
                                                         const float *H, float *gH, float lr,
                                                         const float *dq, const MidArgs ma,
                                                         const CertArgs ca) {
  int w = blockIdx.x;
  if constexpr (GT != 0) {  // the long workgroups first, as in launch 1
    const int gsec = gemm_section(gh, GT);
    if (w < gsec) {
      if (GT == 64 || w < gh.total_tiles) step_gemm<GT, 4>(pl->gb_zgrad, gh, H, gH, lr, nullptr, w);
      return;
    }
    w -= gsec;
  }
  // Y^T Y, the loss and the certificate next (a section padded to a multiple of 8, so
  // that the 16 x 16 tiles' section keeps its XCD alignment)
  const int nyy = (ma.m * ma.m + 255) / 256;
  const int nsmall = (nyy + 2 + 7) & ~7;
  if (w >= nsmall) {
    w -= nsmall;
    const int tile = tile_by_op(hd, w);
    if (tile < 0) return;
    const TileCtx x{H, gH, lr, dq, nullptr};
    run_op(hd, pl->ob[2].op, tile, x, true);
    return;
  }
  const int u = w;
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
// Launch 4: Zq, R X, the U update and the V scatter's plan.  Launch 5: the Q and U^{-T}
// updates and the V scatter.  GT: the tile edge of gb_mid's and gb_update's products.
// ---------------------------------------------------------------------------
// (three workgroups per CU with the 64 x 64 tiles, for the registers of Zq's and R X's
// operand terms)
template <int GT>
__global__ __launch_bounds__(256, GT == 64 ? 3 : 4) void step_mid_kernel(const StepPlan *__restrict__ pl,
                                                       const OpHdr hd, const GemmHdr gh,
                                                       const float *H, float *gH, float lr,
                                                       const float *dq,
                                                       const float *__restrict__ coef,
                                                       const int *__restrict__ cert,
                                                       const int *__restrict__ flag, int n,
                                                       const int *__restrict__ idx, int *splan) {
  int w = blockIdx.x;
  // The U update (k = m) first, as in launch 1 (on 32 x 32 tiles this saved 0.65 us per
  // step at m = 128, d = 500 and 3 us at m = 512, d = 256); on 32 x 32 tiles four
  // k-blocks of 8 per wavefront at m = 128, all loaded before the first product (the
  // launch bound of four workgroups per CU leaves the registers for that).
  const int gsec = gemm_section(gh, GT);
  if (w < gsec) {
    if (GT == 64 || w < gh.total_tiles)
      step_gemm<GT, 4, true>(pl->gb_mid, gh, H, gH, lr, flag, w, cert);
    return;
  }
  w -= gsec;
  const int sec = (hd.total + 7) & ~7;
  if (w < sec) {
    const int tile = section_tile(w, hd.total);
    if (tile < 0) return;
    // the coefficients and the certificate are read where they are used (uniform loads)
    const TileCtx x{H, gH, lr, dq, coef};
    run_op(hd, pl->ob[3].op, tile, x, *cert != 0);
    return;
  }
  w -= sec;
  // the V scatter's plan for launch 5, 16 slots per workgroup
  if (w * 16 < n) scatter_plan(w, n, idx, splan);
}

// (five workgroups per CU on 32 x 32 tiles; four with the 64 x 64 tiles' LDS)
template <int GT>
__global__ __launch_bounds__(256, GT == 64 ? 4 : 5) void step_update_kernel(const StepPlan *__restrict__ pl,
                                                          const GemmHdr gh, const float *H,
                                                          float *gH, float lr,
                                                          const int *__restrict__ flag, int n,
                                                          int K, int d,
                                                          const int *__restrict__ idx,
                                                          const float *__restrict__ wA,
                                                          const float *__restrict__ RX, float *V,
                                                          int64_t ldv, const ScatterChunks ch) {
  // the products first (their workgroups are the long ones), then the scatter
  const int gsec = gemm_section(gh, GT);
  if ((int)blockIdx.x < gsec) {
    if (GT == 64 || (int)blockIdx.x < gh.total_tiles)
      step_gemm<GT, 2>(pl->gb_update, gh, H, gH, lr, flag, blockIdx.x);
    return;
  }
  const int w = blockIdx.x - gsec;
  if (w >= n) return;
  if (*flag != 0) return;
  // V_r -= sum over the row's slots of (dl/dA_kj / (2 dl/dq_j)) (R X)_j
  scatter_planned<256>(w, n, K, d, 1.f, idx, wA, RX, V, ldv, ch);
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

constexpr int kContract32MinTiles = 128;  // 32 x 32 tiles of one m x d product

// Launch 1's m x d products on 32 x 32 tiles once a product has 128 of them (measured:
// slower at m = 128, d = 500, where 16 x 16 tiles fill the chip better; 2-6 % faster
// per step at m = 256, d = 512 and at m = 512, d = 256 to 1024).
bool contract_on_32(int m, int d) {
  return ((m + 31) / 32) * ((d + 31) / 32) >= kContract32MinTiles;
}

// The tile edge of the large-shape batches: LDS-staged 64 x 64 tiles where they were
// measured faster than 32 x 32 tiles (m = 512: launches 1 and 3 at d = 256 to 1024,
// launches 4 and 5 at d = 1024; slower at m = 256, d = 512 and in launches 4 and 5 at
// d = 512, where the products have too few 64 x 64 tiles to fill the chip).
constexpr int kT64Contract = 32, kT64Zgrad = 64, kT64Update = 256, kT64MinK = 256;
int tiles64(int M, int N) { return ((M + 63) / 64) * ((N + 63) / 64); }
// launch 1 (m x d outputs, k = d; N, m x m, joins them)
int tile_contract(int m, int d) {
  return tiles64(m, d) >= kT64Contract && tiles64(m, m) >= kT64Zgrad ? 64 : 32;
}
// launch 3 (m x m and m x d outputs, k = d or m); on 64 x 64 tiles Z^ joins the batch
// with its grad_H epilogue (d = 1024: the launch 76 -> 50 us)
int tile_zgrad(int m, int d) { return tiles64(m, m) >= kT64Zgrad ? 64 : 32; }
// launches 4 and 5 (d x d outputs, k = m)
int tile_update(int m, int d) {
  return tiles64(d, d) >= kT64Update && m >= kT64MinK ? 64 : 32;
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
  for (int q = 0; q < kMaxOps; ++q) ob.begin[q] = q < ob.n ? ob.op[q].tile_begin : total;
  for (int q = 0; q < kMaxOps; ++q)
    ob.count[q] = q < n_main && ob.op[q].M > 0 && ob.op[q].N > 0
                      ? ob.op[q].tiles_m * ob.op[q].tiles_n
                      : 0;
  ob.total = total;
  ob.n_main = n_main;
}

}  // namespace

void build_step_plan(const StepBufs &sb, int m, StepPlan &pl) {
  pl = StepPlan{};
  const int d = sb.d, ldd = sb.ldd;
  const bool sq = sb.loss == LST_LOSS_SQUARED;
  const bool tay = sb.loss == LST_LOSS_TAYLOR_SOFTMAX;
  const float *H = sym_H();
  float *gH = sym_gradH();
  // Launch 1: H^ = H Q (row partials h . h^ -> qpart), H~ = H U^T, X = H U^{-T T}, N = H H^T.
  // At large shapes the m x d products go to 32 x 32 tiles, which read half the operand
  // bytes per output (H^ stays on 16 x 16 tiles for the spherical family, whose epilogue
  // reduces q_j); on 64 x 64 tiles N joins them.
  {
    OpBatch &ob = pl.ob[0];
    GemmBatch &gb = pl.gb_contract;
    const bool big = contract_on_32(m, d);
    ob.n = 0;
    gb.n = 0;
    if (!sq || !big) {
      Op16 h = op(m, d, d, H, d, 0, sb.Q, ldd, 0, sb.Hhat, d);
      if (!sq) {  // the spherical softmax's launch 2 needs every q_j at its start
        h.rowred = RR_DOT;
        h.Rr = H;
        h.ldrr = d;
        h.rowout = sb.qpart;
        h.qout = sb.q;
        h.qcnt = sb.qcnt;
      }
      ob.op[ob.n++] = h;
    } else {
      gb.d[gb.n++] = gemm_desc(m, d, d, H, d, 0, sb.Q, ldd, 0, sb.Hhat, d);
    }
    const int tc = tile_contract(m, d);
    if (big) {
      gb.d[gb.n++] = gemm_desc(m, d, d, H, d, 0, sb.U, ldd, 0, sb.Htil, d);
      gb.d[gb.n++] = gemm_desc(m, d, d, H, d, 0, sb.UinvT, ldd, 0, sb.X, d);
    } else {
      ob.op[ob.n++] = op(m, d, d, H, d, 0, sb.U, ldd, 0, sb.Htil, d);
      ob.op[ob.n++] = op(m, d, d, H, d, 0, sb.UinvT, ldd, 0, sb.X, d);
    }
    if (big && tc == 64)
      gb.d[gb.n++] = gemm_desc(m, m, d, H, d, 0, H, d, 0, sb.N, m);
    else
      ob.op[ob.n++] = op(m, m, d, H, d, 0, H, d, 0, sb.N, m);
    if (tay)  // [s h~] = H [w_bar omega] (eq. svec, gen-htilde)
      ob.op[ob.n++] = op(m, 2, d, H, d, 0, sb.WO, ldd, 0, sb.SW, 2);
    finalize(ob, ob.n);
    if (gb.n) gemm_prepare(gb, tc);
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
    Op16 hz = op(m, m, d, sb.Htil, d, 0, sb.G, d, 0, sb.HZ, m);
    if (tay) {
      // Z^ += ds w_bar^T + y_bar omega^T; HZ += s ds^T + h~ y_bar^T
      z.nuv = 2;
      z.ux[0] = sb.ds;
      z.uxi[0] = 1;
      z.uy[0] = sb.WO;
      z.uyi[0] = 1;
      z.ux[1] = sb.yb;
      z.uxi[1] = 1;
      z.uy[1] = sb.WO + ldd;
      z.uyi[1] = 1;
      hz.nuv = 2;
      hz.ux[0] = sb.SW;
      hz.uxi[0] = 2;
      hz.uy[0] = sb.ds;
      hz.uyi[0] = 1;
      hz.ux[1] = sb.SW + 1;
      hz.uxi[1] = 2;
      hz.uy[1] = sb.yb;
      hz.uyi[1] = 1;
    }
    // at large shapes the products without a fused epilogue or operand scaling go to
    // 32 x 32 tiles (as in launch 1)
    GemmBatch &gb = pl.gb_zgrad;
    const bool big = contract_on_32(m, d);
    const int tz = tile_zgrad(m, d);
    ob.n = 0;
    gb.n = 0;
    if (big && tz == 64 && !tay) {
      // Z^ itself is not stored: its grad_H epilogue writes 2 D H^ + Z^
      GemmDesc zd = gemm_desc(m, d, d, sb.G, d, 0, sb.U, ldd, 1, nullptr, d);
      zd.epi = EPI_GRADH;
      zd.C2 = gH;
      zd.ldc2 = d;
      zd.E = sb.Hhat;
      zd.lde = d;
      zd.rs = sq ? nullptr : sb.dq;
      gb.d[gb.n++] = zd;
    } else {
      ob.op[ob.n++] = z;
    }
    if (big && !tay)
      gb.d[gb.n++] = gemm_desc(m, m, d, sb.Htil, d, 0, sb.G, d, 0, sb.HZ, m);
    else
      ob.op[ob.n++] = hz;
    if (big) {
      gb.d[gb.n++] = gemm_desc(m, m, m, sb.E2, m, 0, sb.E2, m, 1, sb.E4, m);
      gb.d[gb.n++] = gemm_desc(m, d, m, sb.E2, m, 0, sb.W1, d, 1, sb.P3, d);
    } else {
      ob.op[ob.n++] = op(m, m, m, sb.E2, m, 0, sb.E2, m, 1, sb.E4, m);
      ob.op[ob.n++] = op(m, d, m, sb.E2, m, 0, sb.W1, d, 1, sb.P3, d);
    }
    if (big && sq) {
      gb.d[gb.n++] = gemm_desc(m, d, m, sb.E2, m, 0, sb.X, d, 1, sb.P2, d);
    } else {
      ob.op[ob.n] = op(m, d, m, sb.E2, m, 0, sb.X, d, 1, sb.P2, d);
      if (!sq) ob.op[ob.n].b[0].sc = SC_SQRT;
      ++ob.n;
    }
    finalize(ob, ob.n);
    if (gb.n) gemm_prepare(gb, tz);
  }
  // Launch 4: Zq = (eta^2/2) M H - eta grad_H (M assembled as it is loaded);
  // R X = 2 eta S (c0 Xs + c1 W1 + c2 P2 + c3 P3 + E^4 (c4 Xs + c5 W1 + c6 P2 + c7 P3)),
  // or R X with the exact R when the polynomial is not certified.
  {
    OpBatch &ob = pl.ob[3];
    Op16 zq = op(m, d, m, nullptr, 0, 0, H, d, 1, sb.Zq, d);
    zq.amode = AM_MASM;
    if (tay) {
      zq.amode = AM_MASM_S;
      zq.ds = sb.ds;
      zq.yb = sb.yb;
      zq.Dn = (float)sb.D;
    }
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
    // On 64 x 64 tiles (d = 1024) the squared error's Zq and R X join the U update: M
    // and R X's B assembled from their terms as they are staged, R X's addends in the
    // epilogue, and the exact R X as its alternative.
    const bool mid64 = sq && tile_update(m, d) == 64;
    if (!mid64) ob.op[0] = zq;
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
    GemmBatch &gb = pl.gb_mid;
    // U <- U - (2 eta D H~)^T H
    gb.d[0] = gemm_desc(d, d, m, sb.Atil, d, 1, H, d, 1, sb.U, ldd, -1.f, sb.U, ldd, 1.f);
    gb.n = 1;
    if (mid64) {
      // Zq = (eta^2 / 2) (4 M^ + Yring^T Yring + 2 HZ + 2 HZ^T) H - eta grad_H
      GemmDesc zd = gemm_desc(m, d, m, sb.Mhat, m, 0, H, d, 1, sb.Zq, d, 0.5f, gH, d, -1.f);
      zd.lr_scaled = 1;
      zd.nat = 3;
      zd.aw[0] = 4.f;
      zd.At[0] = sb.YY;
      zd.aw[1] = 1.f;
      zd.At[1] = sb.HZ;
      zd.aw[2] = 2.f;
      zd.Atr = sb.HZ;
      zd.awt = 2.f;
      gb.d[gb.n++] = zd;
      // R X = 2 eta (E^4 (c4 X + c5 W1 + c6 P2 + c7 P3) + c0 X + c1 W1 + c2 P2 + c3 P3)
      GemmDesc rd = gemm_desc(m, d, m, sb.E4, m, 0, sb.X, d, 1, sb.RX, d, 2.f);
      rd.lr_scaled = 2;
      rd.coef = sb.coef;
      rd.nbt = 4;
      rd.nadd = 4;
      rd.ldadd = d;
      const float *term[4] = {sb.X, sb.W1, sb.P2, sb.P3};
      for (int t = 0; t < 4; ++t) {
        rd.bcoef[t] = 4 + t;
        if (t > 0) rd.Bt[t - 1] = term[t];
        rd.acoef[t] = t;
        rd.addp[t] = term[t];
      }
      rd.alt1 = 4;  // d[3], below
      gb.d[gb.n++] = rd;
      ob.n = 0;
      finalize(ob, 0);
    } else {
      ob.op[1] = rx;
      ob.op[2] = op(m, d, m, sb.R, m, 0, sb.X, d, 1, sb.RX, d);  // exact R
      ob.n = 3;
      finalize(ob, 2);
    }
    gemm_prepare(gb, tile_update(m, d));
    if (mid64) {  // R X's alternative with the exact R, outside the batch's tile ranges
      GemmDesc &alt = gb.d[3];
      alt = gemm_desc(m, d, m, sb.R, m, 0, sb.X, d, 1, sb.RX, d);
      alt.tiles_m = gb.d[2].tiles_m;
      alt.tiles_n = gb.d[2].tiles_n;
      alt.tile_begin = gb.total_tiles;
    }
  }
  // Launch 5: Q <- Q + H^T Zq + Zq^T H; U^{-T} <- U^{-T} + (R X)^T H; omega, w_bar
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
    if (tay)  // [w_bar; omega] -= [c_w; c_o] H (eta folded into the coefficients)
      gb.d[gb.n++] = gemm_desc(2, d, m, sb.cwo, m, 0, H, d, 1, sb.WO, ldd, -1.f, sb.WO, ldd, 1.f);
    gemm_prepare(gb, tile_update(m, d));
  }
}

void step_launch_sizes(const StepPlan &pl, int m, int K, int (&grid)[5]) {
  auto sec = [](int n) { return (n + 7) & ~7; };
  auto gsec = [](const GemmBatch &b) { return gemm_section(gemm_hdr(b), b.tile); };
  grid[0] = sec(pl.ob[0].total) + gsec(pl.gb_contract) + m;
  grid[1] = sec(m) + section_by_op(pl.ob[1]);
  grid[2] = section_by_op(pl.ob[2]) + gsec(pl.gb_zgrad) + (((m * m + 255) / 256 + 2 + 7) & ~7);
  grid[3] = sec(pl.ob[3].total) + gsec(pl.gb_mid) + (m * K + 15) / 16;
  grid[4] = gsec(pl.gb_update) + m * K;
}

void enqueue_step_launch(int which, const StepBufs &sb, const StepPlan &host, const StepPlan *dev,
                         const StepArgs &a, hipStream_t s) {
  int grid[5];
  step_launch_sizes(host, a.m, a.K, grid);
  const float *dqp = sb.loss == LST_LOSS_SQUARED ? nullptr : sb.dq;
  switch (which) {
    case 0:
#define LST_CONTRACT(GT)                                                                          \
  LST_LAUNCH(step_contract_kernel<GT>, dim3(grid[0]), dim3(256), 0, s, dev, op_hdr(host.ob[0]),    \
             gemm_hdr(host.gb_contract), a.H, a.lr, a.idx, a.val, a.K, sb.V, sb.ldv, sb.D, sb.d, a.m, \
             sb.tsum)
      if (host.gb_contract.tile == 64)
        LST_CONTRACT(64);
      else
        LST_CONTRACT(32);
#undef LST_CONTRACT
      break;
    case 1: {
      GatherArgs ga{};
      ga.K = a.K;
      ga.d = sb.d;
      ga.m = a.m;
      ga.Hhat = sb.Hhat;
      ga.q = sb.q;
      ga.tsum = sb.tsum;
      ga.qcnt = sb.qcnt;
      ga.nqcnt = (a.m + 15) / 16;
      ga.D = sb.D;
      ga.H = a.H;
      ga.Htil = sb.Htil;
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
      ga.ticket = sb.ticket;
      ga.wA = sb.wA;
      ga.lvec = sb.lvec;
      ga.srow = sb.srow;
      ga.sval = sb.sval;
      ga.scnt = sb.scnt;
      ga.SW = sb.SW;
      ga.ds = sb.ds;
      ga.yb = sb.yb;
      ga.cwo = sb.cwo;
      ga.flag = sb.flag;
      const int kpw = (a.K + 3) / 4;
      const int d = sb.d;
      const OpHdr hd1 = op_hdr(host.ob[1]);
#define LST_GATHER(KPW, NV)                                                                        \
  if (kpw <= KPW && d <= 64 * NV) {                                                                \
    LST_LAUNCH((step_gather_kernel<KPW, NV>), dim3(grid[1]), dim3(256), 0, s, dev, hd1, a.H, a.lr, \
               ga);                                                                                \
    break;                                                                                         \
  }
      LST_GATHER(1, 8)
      LST_GATHER(2, 8)
      LST_GATHER(4, 8)
      LST_GATHER(1, 16)
      LST_GATHER(2, 16)
#undef LST_GATHER
      LST_LAUNCH((step_gather_kernel<0, 0>), dim3(grid[1]), dim3(256), 0, s, dev, hd1, a.H, a.lr,
                 ga);
      break;
    }
    case 2: {
      MidArgs ma{a.m, a.K, sb.srow, sb.sval, sb.scnt, sb.YY, sb.lvec, a.loss, sb.flag};
      CertArgs ca{a.m, sb.bpart, sb.N, dqp, sb.Cwork, sb.R, sb.coef, sb.cert, sb.flag};
#define LST_ZGRAD(GT)                                                                          \
  LST_LAUNCH(step_zgrad_kernel<GT>, dim3(grid[2]), dim3(256), 0, s, dev, op_hdr(host.ob[2]), \
             gemm_hdr(host.gb_zgrad), a.H, a.gH, a.lr, dqp, ma, ca)
      if (host.gb_zgrad.n == 0)
        LST_ZGRAD(0);
      else if (host.gb_zgrad.tile == 64)
        LST_ZGRAD(64);
      else
        LST_ZGRAD(32);
#undef LST_ZGRAD
      break;
    }
    case 3:
#define LST_MID(GT)                                                                             \
  LST_LAUNCH(step_mid_kernel<GT>, dim3(grid[3]), dim3(256), 0, s, dev, op_hdr(host.ob[3]),       \
             gemm_hdr(host.gb_mid), a.H, a.gH, a.lr, dqp, sb.coef, sb.cert, sb.flag, a.m * a.K, \
             a.idx, sb.splan)
      if (host.gb_mid.tile == 64)
        LST_MID(64);
      else
        LST_MID(32);
#undef LST_MID
      break;
    default: {
      // rows of more than C slots summed in chunks; the partial sums in P2 and P3, which
      // launch 4 has finished reading
      ScatterChunks ch{};
      ch.C = a.K > 32 ? a.K : 32;
      ch.half = a.m;
      ch.part0 = sb.P2;
      ch.part1 = sb.P3;
      ch.plan = sb.splan;
      ch.rcnt = sb.rcnt;
      ch.ticket = sb.ticket;
#define LST_UPDATE(GT)                                                                          \
  LST_LAUNCH(step_update_kernel<GT>, dim3(grid[4]), dim3(256), 0, s, dev,                        \
             gemm_hdr(host.gb_update), a.H, a.gH, a.lr, sb.flag, a.m * a.K, a.K, sb.d, a.idx, sb.wA, \
             sb.RX, sb.V, sb.ldv, ch)
      if (host.gb_update.tile == 64)
        LST_UPDATE(64);
      else
        LST_UPDATE(32);
#undef LST_UPDATE
    }
  }
}

}  // namespace lst
