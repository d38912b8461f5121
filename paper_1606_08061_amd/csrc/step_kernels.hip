// Non-GEMM kernels of the factored step and of the naive comparison path.
//
//   gather   -- the sparse part of Algorithm 4: A_kj = H~_j . V_{K_kj} (eq.
//               gen-A-fact), q_j = h_j . H^_j (eq. qvec), the loss epilogue
//               (l_j, dl/dq_j, dl/dA_kj) and G_j = sum_k dl/dA_kj V_{K_kj}
//               (the V^T Yring of eq. gen-Zhat-fact; Algorithm 3 step 2's V^T Y
//               up to the factor -2).
//   woodbury -- the m x m Woodbury matrix C = I - 2 eta S H^T H S and its
//               inverse (Gauss-Jordan without pivoting: C is symmetric positive
//               definite exactly when the step is admissible), giving
//               R = 2 eta S C^{-1} S for the U^{-T} update (Algorithm 3 step 6,
//               the Woodbury form of section 4.7).
//   mblock   -- L = sum_j l_j and the Q-update matrix M of eq. gen-M, with the
//               sparse Yring^T Yring by index equality.
//   scatter  -- eq. updateV / gen-updateV: V_r -= eta sum_{slots of row r}
//               dl/dA P_j, one writer per distinct row (its lowest slot), slots
//               summed in ascending order, so repeated rows never race and
//               results are reproducible bit for bit.
//   naive    -- column norms of O, the loss epilogue over the explicit output
//               and grad_O = 2 O diag(dl/dq) + Yring (eq. gen-grad-O).
#include <algorithm>

#include "lst_internal.h"
#include "scatter.h"
#include "woodbury_gj.h"

namespace lst {

namespace {

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Loss epilogue of one example (section 4: l(q, K, a, t) with dl/ds = 0).
// r[k] < 0 marks an empty slot.  Writes the example's loss, dl/dq and dl/da_k.
__device__ __forceinline__ void loss_epilogue(int loss, float q, int K, const int *r,
                                              const float *t, const float *a, float Deps,
                                              float eps, float &l, float &gq, float *g) {
  l = 0.f;
  gq = 0.f;
  if (loss == LST_LOSS_SQUARED) {
    // l = q - 2 a.t + ||y||^2 with ||y||^2 over equal indices (repeated slots add)
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
    gq = 1.f;
  } else {
    // l = sum_k t_k [log(q + D eps) - log(a_k^2 + eps)]
    const float z = q + Deps;
    const float lz = logf(z);
    for (int k = 0; k < K; ++k) {
      g[k] = 0.f;
      if (r[k] < 0) continue;
      const float den = a[k] * a[k] + eps;
      l += t[k] * (lz - logf(den));
      gq += t[k] / z;
      g[k] = -2.f * t[k] * a[k] / den;
    }
  }
}

// The same epilogue on register arrays (K <= KMAX slots, fully unrolled), so the
// serial part of a gather workgroup does no dependent LDS reads.
template <int KMAX>
__device__ __forceinline__ void loss_epilogue_reg(int loss, float q, int K, const int (&r)[KMAX],
                                                  const float (&t)[KMAX], const float (&a)[KMAX],
                                                  float Deps, float eps, float &l, float &gq,
                                                  float (&g)[KMAX]) {
  l = 0.f;
  gq = 0.f;
  if (loss == LST_LOSS_SQUARED) {
    float at = 0.f, yy = 0.f;
#pragma unroll
    for (int k = 0; k < KMAX; ++k) {
      const bool ok = k < K && r[k] >= 0;
      g[k] = ok ? -2.f * t[k] : 0.f;
      if (!ok) continue;
      at += t[k] * a[k];
#pragma unroll
      for (int kk = 0; kk < KMAX; ++kk)
        if (kk < K && r[kk] == r[k]) yy += t[k] * t[kk];
    }
    l = q - 2.f * at + yy;
    gq = 1.f;
  } else {
    const float z = q + Deps;
    const float lz = logf(z);
#pragma unroll
    for (int k = 0; k < KMAX; ++k) {
      g[k] = 0.f;
      if (k >= K || r[k] < 0) continue;
      const float den = a[k] * a[k] + eps;
      l += t[k] * (lz - logf(den));
      gq += t[k] / z;
      g[k] = -2.f * t[k] * a[k] / den;
    }
  }
}

constexpr int kGatherThreads = 256;

// One workgroup (four wavefronts) per example j.  The K row dot products
// A_kj = H~_j . V_r are spread over the wavefronts, and G_j = sum_k dl/dA_kj V_r
// is formed column-parallel, so the loads of the K target rows are in flight
// together rather than one row after another.
__global__ __launch_bounds__(kGatherThreads) void gather_kernel(
    int K, int d, int64_t D, const float *__restrict__ H, const float *__restrict__ Hhat,
    const float *__restrict__ Htil, const int *__restrict__ idx, const float *__restrict__ val,
    const float *__restrict__ V, int64_t ldv, int loss, float eps, float lr, float *__restrict__ G,
    float *__restrict__ Atil, float *__restrict__ dq, float *__restrict__ dA,
    float *__restrict__ lvec, int *__restrict__ flag) {
  __shared__ int sr[LST_MAX_K];
  __shared__ float sa[LST_MAX_K], st[LST_MAX_K], sg[LST_MAX_K];
  __shared__ float sred[kGatherThreads / 64];
  __shared__ float s_gq;
  __shared__ int s_bad;
  const int j = blockIdx.x;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const float *h = H + (int64_t)j * d;
  const float *hh = Hhat + (int64_t)j * d;
  const float *ht = Htil + (int64_t)j * d;

  if (t == 0) s_bad = 0;
  __syncthreads();
  for (int k = t; k < K; k += kGatherThreads) {
    int r = idx[(int64_t)j * K + k];
    if (r < -1 || (int64_t)r >= D) {
      atomicOr(&s_bad, 1);
      r = -1;
    }
    sr[k] = r;
    st[k] = val[(int64_t)j * K + k];
  }
  float qs = 0.f;
  for (int c = t; c < d; c += kGatherThreads) qs += h[c] * hh[c];
  qs = wave_sum(qs);
  if (lane == 0) sred[wave] = qs;
  __syncthreads();
  const float q = (sred[0] + sred[1]) + (sred[2] + sred[3]);
  if (t == 0 && s_bad) atomicOr(flag, FLAG_INDEX);

  for (int k = wave; k < K; k += kGatherThreads / 64) {
    const int r = sr[k];
    float a = 0.f;
    if (r >= 0) {
      const float *vr = V + (int64_t)r * ldv;
      float s = 0.f;
#pragma unroll 8
      for (int c = lane; c < d; c += 64) s += ht[c] * vr[c];
      a = wave_sum(s);
    }
    if (lane == 0) sa[k] = a;
  }
  __syncthreads();

  if (t == 0) {
    float l, gq;
    loss_epilogue(loss, q, K, sr, st, sa, (float)D * eps, eps, l, gq, sg);
    dq[j] = gq;
    lvec[j] = l;
    s_gq = gq;
  }
  __syncthreads();
  for (int k = t; k < K; k += kGatherThreads) dA[(int64_t)j * K + k] = sg[k];

  const float s2 = 2.f * lr * s_gq;
  for (int c = t; c < d; c += kGatherThreads) {
    float s = 0.f;
#pragma unroll 4
    for (int k = 0; k < K; ++k) {
      const int r = sr[k];
      if (r >= 0) s += sg[k] * V[(int64_t)r * ldv + c];
    }
    G[(int64_t)j * d + c] = s;
    Atil[(int64_t)j * d + c] = s2 * ht[c];
  }
}

// Register-resident variant for K <= 4 KPW and d <= 64 NV: wavefront w keeps the
// target rows k = w, w + 4, ... (64 NV columns per row) in registers from the
// dot products A_kj to the G sum, so V is read once and the index loads lead
// straight into the row loads.  G_j is summed per wavefront, then over the four
// wavefronts in a fixed order.
template <int KPW, int NV>
__global__ __launch_bounds__(kGatherThreads) void gather_reg_kernel(
    int K, int d, int64_t D, const float *__restrict__ H, const float *__restrict__ Hhat,
    const float *__restrict__ Htil, const int *__restrict__ idx, const float *__restrict__ val,
    const float *__restrict__ V, int64_t ldv, int loss, float eps, float lr, float *__restrict__ G,
    float *__restrict__ Atil, float *__restrict__ dq, float *__restrict__ dA,
    float *__restrict__ lvec, int *__restrict__ flag) {
  constexpr int W = kGatherThreads / 64;
  __shared__ int sr[W * KPW];
  __shared__ float sa[W * KPW], st[W * KPW], sg[W * KPW];
  __shared__ float sred[W];
  __shared__ float s_gq;
  __shared__ int s_bad;
  __shared__ float gpart[W][64 * NV];
  const int j = blockIdx.x;
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  if (t == 0) s_bad = 0;

  // Target rows of this wavefront (uniform loads), then the rows themselves.
  int r[KPW];
  bool bad = false;
#pragma unroll
  for (int i = 0; i < KPW; ++i) {
    const int k = wave + W * i;
    int v = -1;
    if (k < K) {
      v = idx[(int64_t)j * K + k];
      if (v < -1 || (int64_t)v >= D) {
        bad = true;
        v = -1;
      }
    }
    r[i] = v;
  }
  float vr[KPW][NV];
#pragma unroll
  for (int i = 0; i < KPW; ++i) {
    const float *row = V + (int64_t)max(r[i], 0) * ldv;
#pragma unroll
    for (int n = 0; n < NV; ++n) {
      const int c = lane + 64 * n;
      const float x = row[min(c, d - 1)];
      vr[i][n] = (r[i] >= 0 && c < d) ? x : 0.f;
    }
  }
  float ht[NV];
  const float *htp = Htil + (int64_t)j * d;
#pragma unroll
  for (int n = 0; n < NV; ++n) {
    const int c = lane + 64 * n;
    ht[n] = (c < d) ? htp[c] : 0.f;
  }
  // q_j = h_j . H^_j over all threads
  float qs = 0.f;
  for (int c = t; c < d; c += kGatherThreads) qs += H[(int64_t)j * d + c] * Hhat[(int64_t)j * d + c];
  qs = wave_sum(qs);
  // A_kj = H~_j . V_r for this wavefront's rows
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
    sred[wave] = qs;
#pragma unroll
    for (int i = 0; i < KPW; ++i) {
      const int k = wave + W * i;
      if (k < K) {
        sr[k] = r[i];
        sa[k] = a[i];
        st[k] = val[(int64_t)j * K + k];
      }
    }
    if (bad) atomicOr(&s_bad, 1);
  }
  __syncthreads();
  if (t == 0) {
    if (s_bad) atomicOr(flag, FLAG_INDEX);
    const float q = (sred[0] + sred[1]) + (sred[2] + sred[3]);
    constexpr int KM = W * KPW;
    int rr[KM];
    float tt[KM], aa[KM], gg[KM];
#pragma unroll
    for (int k = 0; k < KM; ++k) {
      rr[k] = k < K ? sr[k] : -1;
      tt[k] = k < K ? st[k] : 0.f;
      aa[k] = k < K ? sa[k] : 0.f;
    }
    float l, gq;
    loss_epilogue_reg<KM>(loss, q, K, rr, tt, aa, (float)D * eps, eps, l, gq, gg);
#pragma unroll
    for (int k = 0; k < KM; ++k)
      if (k < K) sg[k] = gg[k];
    dq[j] = gq;
    lvec[j] = l;
    s_gq = gq;
  }
  __syncthreads();
  for (int k = t; k < K; k += kGatherThreads) dA[(int64_t)j * K + k] = sg[k];
  // G_j = sum_k dl/dA_kj V_r: this wavefront's rows, then the four partials in order
#pragma unroll
  for (int n = 0; n < NV; ++n) {
    float g = 0.f;
#pragma unroll
    for (int i = 0; i < KPW; ++i) {
      const int k = wave + W * i;
      if (k < K) g += sg[k] * vr[i][n];
    }
    gpart[wave][lane + 64 * n] = g;
  }
  __syncthreads();
  const float s2 = 2.f * lr * s_gq;
  for (int c = t; c < d; c += kGatherThreads) {
    G[(int64_t)j * d + c] = (gpart[0][c] + gpart[1][c]) + (gpart[2][c] + gpart[3][c]);
    Atil[(int64_t)j * d + c] = s2 * htp[c];
  }
}

constexpr int kMaxSortKeys = 8192;

// The whole inverse on one workgroup (m <= 32 NBK); releases *done at the end,
// whether or not the matrix was accepted.
template <int NBK>
__global__ __launch_bounds__(64 * wb_waves<NBK>()) void woodbury_blocked_kernel(
    int m, float lr, int unit_dq, const float *__restrict__ dq, const float *__restrict__ N,
    float *__restrict__ R, int *__restrict__ flag, const StepSync wait, int *__restrict__ done) {
  step_sync_begin(wait);
  woodbury_blocked<NBK>(m, lr, unit_dq, dq, N, R, flag);
  if (done) release_count(done);
}

__global__ void step_sync_kernel(const StepSync wait, int *__restrict__ done) {
  step_sync_begin(wait);
  if (done) release_count(done);
}

// ---------------------------------------------------------------------------
// Larger m: the same block step with kBigBlock-row pivot blocks on the m x m
// matrix A (= C) in global memory, three launches per block b:
//   pivot kernel   P = A_bb^{-1} (the blocked elimination on one workgroup), PI = P + I;
//   row launch     Rp_:,j = P A_b,j for the columns j outside b, Rp_:,b = P + I,
//                  and the column panel copy Cp = A_:,b;
//   trailing launch A_i,: += -Cp_i Rp for the rows i outside b, A_b,: = Rp.
// Column b of a row outside b becomes A_ib - A_ib (P + I) = -A_ib P, as the block
// step requires; the diagonal block becomes P + I, and the next pivot kernel (or
// the final scaling) subtracts the I.
// ---------------------------------------------------------------------------

// A = C = I - 2 eta S N S (m x m); a negative or NaN dl/dq raises the error flag.
__global__ void form_c_kernel(int m, float lr, int unit_dq, const float *__restrict__ dq,
                              const float *__restrict__ N, float *__restrict__ A,
                              int *__restrict__ flag) {
  const int64_t total = (int64_t)m * m;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int i = (int)(e / m), j = (int)(e - (int64_t)i * m);
    const float qi = unit_dq ? 1.f : dq[i], qj = unit_dq ? 1.f : dq[j];
    if (i == j && !(qi >= 0.f)) atomicOr(flag, FLAG_NOT_SPD);
    const float si = sqrtf(fmaxf(qi, 0.f)), sj = sqrtf(fmaxf(qj, 0.f));
    A[e] = ((i == j) ? 1.f : 0.f) - 2.f * lr * si * N[e] * sj;
  }
}

// R = 2 eta S A S from the inverse held in A, less the I left on the last
// diagonal block (rows lb0 .. m-1).
__global__ void scale_r_kernel(int m, int lb0, float lr, int unit_dq, const float *__restrict__ dq,
                               const float *__restrict__ A, float *__restrict__ R) {
  const int64_t total = (int64_t)m * m;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int i = (int)(e / m), j = (int)(e - (int64_t)i * m);
    const float qi = unit_dq ? 1.f : dq[i], qj = unit_dq ? 1.f : dq[j];
    const float a = A[e] - ((i == j && i >= lb0) ? 1.f : 0.f);
    R[e] = 2.f * lr * sqrtf(fmaxf(qi, 0.f)) * a * sqrtf(fmaxf(qj, 0.f));
  }
}

// For m > d the branch inverts the d x d matrix B = I - 2 eta Hs^T Hs instead of the
// m x m C = I - 2 eta Hs Hs^T (Hs = S H, rows of H scaled by (dl/dq)^(1/2)): by the
// push-through identity C^{-1} = I + Hs R' Hs^T with R' = 2 eta B^{-1}, so
// R = 2 eta S C^{-1} S = 2 eta S (I + Hs R' Hs^T) S.  B and C share their nonzero
// eigenvalues, so B's pivots answer the same positive-definiteness question.
// Hs = S H; dl/dq < 0 has no real square root: flagged as not positive definite.
__global__ void scale_rows_sqrt_kernel(int m, int d, const float *__restrict__ H,
                                       const float *__restrict__ dq, float *__restrict__ Hs,
                                       int *__restrict__ flag) {
  const int64_t total = (int64_t)m * d;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int i = (int)(e / d);
    const float q = dq[i];
    if (e - (int64_t)i * d == 0 && !(q >= 0.f)) atomicOr(flag, FLAG_NOT_SPD);
    Hs[e] = sqrtf(fmaxf(q, 0.f)) * H[e];
  }
}

// R = 2 eta S (R0 + I) S in place, R0 = Hs R' Hs^T.
__global__ void push_through_r_kernel(int m, float lr, int unit_dq, const float *__restrict__ dq,
                                      float *__restrict__ R) {
  const int64_t total = (int64_t)m * m;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int i = (int)(e / m), j = (int)(e - (int64_t)i * m);
    const float si = unit_dq ? 1.f : sqrtf(fmaxf(dq[i], 0.f));
    const float sj = unit_dq ? 1.f : sqrtf(fmaxf(dq[j], 0.f));
    R[e] = 2.f * lr * si * (R[e] + (i == j ? 1.f : 0.f)) * sj;
  }
}

// Pivot block b0 .. b0+nb-1 (nb <= kBigBlock) of A: P and PI = P + I
// (kBigBlock^2 each, identity-padded).  First removes the I left on the
// previous diagonal block (rows pb0 .. pb0+pnb-1; pnb = 0 for none).
constexpr int kPivotNbk = kBigBlock / 32;

__global__ __launch_bounds__(64 * wb_waves<kPivotNbk>()) void pivot_block_kernel(
    int m, int b0, int nb, int pb0, int pnb, float *__restrict__ A, float *__restrict__ P,
    float *__restrict__ PI, int *__restrict__ flag) {
  constexpr int NBK = kPivotNbk;
  __shared__ GjLds<NBK> sh;
  if (threadIdx.x == 0) sh.bad[0] = sh.bad[1] = 0;
  for (int i = threadIdx.x; i < pnb; i += blockDim.x) A[(int64_t)(pb0 + i) * m + pb0 + i] -= 1.f;
  __syncthreads();
  const int lane = threadIdx.x & 63, j = lane & 31, h = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // All loads issued first and pinned (none moved under the padding conditions).
  constexpr int NW = wb_workers<NBK>(), NS = wb_sets<NBK>();
  const float *ab = A + (int64_t)b0 * m + b0;
  if (wave == NW) {  // the inverting wavefront: the pivot block A_00
    float raw[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) raw[r] = ab[(int64_t)min(acc_row(h, r), nb - 1) * m + min(j, nb - 1)];
#pragma unroll
    for (int r = 0; r < 16; ++r) asm volatile("" : "+v"(raw[r]));
    floatx16 a00;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = acc_row(h, r);
      a00[r] = (row < nb && j < nb) ? raw[r] : ((row == j) ? 1.f : 0.f);
    }
    if (!gj_inverter<NBK>(a00, sh, lane)) return;
    const int col = 32 * (NBK - 1) + j;
    last_column<NBK>(sh, lane, [&](int s, const floatx16 &v) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = 32 * s + acc_row(h, r);
        P[row * kBigBlock + col] = v[r];
        PI[row * kBigBlock + col] = v[r] + ((row == col) ? 1.f : 0.f);
      }
    });
    return;
  }
  floatx16 acc[NS][NBK];
  {
    float raw[NS][NBK][16];
#pragma unroll
    for (int t = 0; t < NS; ++t) {
      if (wave + NW * t >= NBK) continue;  // no such tile column
      const float *ap = ab + min(32 * (wave + NW * t) + j, nb - 1);
#pragma unroll
      for (int s = 0; s < NBK; ++s)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          raw[t][s][r] = ap[(int64_t)min(32 * s + acc_row(h, r), nb - 1) * m];
    }
#pragma unroll
    for (int t = 0; t < NS; ++t)
#pragma unroll
      for (int s = 0; s < NBK; ++s)
#pragma unroll
        for (int r = 0; r < 16; ++r) asm volatile("" : "+v"(raw[t][s][r]));
#pragma unroll
    for (int t = 0; t < NS; ++t) {
      const int col = 32 * (wave + NW * t) + j;
#pragma unroll
      for (int s = 0; s < NBK; ++s)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = 32 * s + acc_row(h, r);
          acc[t][s][r] = (row < nb && col < nb) ? raw[t][s][r] : ((row == col) ? 1.f : 0.f);
        }
    }
  }
  if (!gj_workers<NBK>(acc, sh, wave, lane)) {
    if (threadIdx.x == 0) atomicOr(flag, FLAG_NOT_SPD);
    return;
  }
#pragma unroll
  for (int t = 0; t < NS; ++t) {
    if (wave + NW * t >= NBK - 1) continue;  // column NBK - 1: the inverting wavefront's
    const int col = 32 * (wave + NW * t) + j;
#pragma unroll
    for (int s = 0; s < NBK; ++s)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = 32 * s + acc_row(h, r);
        P[row * kBigBlock + col] = acc[t][s][r];
        PI[row * kBigBlock + col] = acc[t][s][r] + ((row == col) ? 1.f : 0.f);
      }
  }
}

// Loss L = sum_j l_j (fixed order; non-finite -> error flag) and the Q-update
// matrix M of eq. gen-M (dl/ds = 0):
//   M_ij = 4 dq_i M^_ij dq_j + (Yring^T Yring)_ij + 2 dq_i (H~^T G)_ij + 2 dq_j (H~^T G)_ji
// Each workgroup stages the m x K targets in LDS and fills kMblockThreads
// entries of M; workgroup 0 also forms the loss.  For K <= kMblockDirectK the
// sparse term compares the two examples' targets directly (K^2 compares); for
// larger K column j of the sparse Yring is kept as a sorted list of (row,
// value) pairs and (Yring^T Yring)_ij is a merge of two lists in ascending row
// order.
constexpr int kMblockThreads = 256;
constexpr int kMblockDirectK = 16;  // K up to this: direct K x K compare, else sorted lists

__global__ __launch_bounds__(kMblockThreads) void mblock_kernel(
    int m, int K, const int *__restrict__ idx, const float *__restrict__ lvec,
    const float *__restrict__ dq, const float *__restrict__ dA, const float *__restrict__ Mhat,
    const float *__restrict__ HZ, float *__restrict__ M, float *__restrict__ loss_out,
    int *__restrict__ flag) {
  __shared__ int lrow[kMaxSortKeys];
  __shared__ float lval[kMaxSortKeys];
  __shared__ int lcnt[LST_MAX_M];
  __shared__ float red[kMblockThreads];
  const int t = threadIdx.x;
  const int e = blockIdx.x * kMblockThreads + t;

  // Prefetch this thread's dense terms before building the lists.
  const bool has = e < m * m;
  const int i = has ? e / m : 0, j = has ? e - (e / m) * m : 0;
  float mh = 0.f, hz = 0.f, hzt = 0.f, di = 0.f, dj = 0.f;
  if (has) {
    mh = Mhat[e];
    hz = HZ[e];
    hzt = HZ[(int64_t)j * m + i];
    di = dq[i];
    dj = dq[j];
  }

  if (blockIdx.x == 0) {
    float ls = 0.f;
    for (int q = t; q < m; q += kMblockThreads) ls += lvec[q];
    red[t] = ls;
    __syncthreads();
    for (int s = kMblockThreads / 2; s > 0; s >>= 1) {
      if (t < s) red[t] += red[t + s];
      __syncthreads();
    }
    if (t == 0) {
      const float L = red[0];
      *loss_out = L;
      if (!isfinite(L)) atomicOr(flag, FLAG_NONFINITE);
    }
  }

  // Index and value matrices into LDS with all loads in flight at once; each list
  // is then sorted in place (entry k is read before any insertion reaches it).
  for (int q = t; q < m * K; q += kMblockThreads) {
    lrow[q] = idx[q];
    lval[q] = dA[q];
  }
  __syncthreads();
  if (K <= kMblockDirectK) {
    // (Yring^T Yring)_ij = sum_a sum_b [idx_ia = idx_jb >= 0] dl/dA_ia dl/dA_jb: the
    // same bilinear sum as the merge of the two lists below (repeated rows add up
    // either way), straight from the staged rows, K^2 compares in registers.
    if (!has) return;
    int rj[kMblockDirectK];
    float vj[kMblockDirectK];
#pragma unroll
    for (int b = 0; b < kMblockDirectK; ++b) {
      rj[b] = b < K ? lrow[j * K + b] : -1;
      vj[b] = b < K ? lval[j * K + b] : 0.f;
    }
    float yy = 0.f;
#pragma unroll
    for (int a = 0; a < kMblockDirectK; ++a) {
      if (a >= K) break;
      const int r = lrow[i * K + a];
      float sb = 0.f;
#pragma unroll
      for (int b = 0; b < kMblockDirectK; ++b) sb += (rj[b] == r) ? vj[b] : 0.f;
      yy += (r >= 0) ? lval[i * K + a] * sb : 0.f;
    }
    M[e] = 4.f * di * mh * dj + yy + 2.f * di * hz + 2.f * dj * hzt;
    return;
  }
  for (int q = t; q < m; q += kMblockThreads) {
    int *lr = lrow + q * K;
    float *lv = lval + q * K;
    int c = 0;
    for (int k = 0; k < K; ++k) {
      const int r = lr[k];
      if (r < 0) continue;
      const float g = lv[k];
      int p = c;
      while (p > 0 && lr[p - 1] > r) {
        lr[p] = lr[p - 1];
        lv[p] = lv[p - 1];
        --p;
      }
      lr[p] = r;
      lv[p] = g;
      ++c;
    }
    int w = 0;
    for (int u = 0; u < c; ++u) {
      if (w > 0 && lr[w - 1] == lr[u]) {
        lv[w - 1] += lv[u];
      } else {
        lr[w] = lr[u];
        lv[w] = lv[u];
        ++w;
      }
    }
    lcnt[q] = w;
  }
  __syncthreads();
  if (!has) return;

  const int *ri = lrow + i * K, *rj = lrow + j * K;
  const float *vi = lval + i * K, *vj = lval + j * K;
  const int na = lcnt[i], nb = lcnt[j];
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
  M[e] = 4.f * di * mh * dj + yy + 2.f * di * hz + 2.f * dj * hzt;
}

constexpr int kScatterThreads = 512;

// The V update: one workgroup per target slot (scatter_slot).
__global__ __launch_bounds__(kScatterThreads) void scatter_kernel(
    int n, int K, int d, float lr, const int *__restrict__ idx, const float *__restrict__ dA,
    const float *__restrict__ P, float *__restrict__ V, int64_t ldv, const int *__restrict__ gate) {
  extern __shared__ int sh[];
  if (*gate != 0) return;
  scatter_slot<kScatterThreads>(blockIdx.x, n, K, d, lr, idx, dA, P, V, ldv, sh);
}

__global__ void identity_kernel(float *A, int d, int64_t ld) {
  const int64_t total = (int64_t)d * d;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int i = (int)(e / d), j = (int)(e % d);
    A[(int64_t)i * ld + j] = (i == j) ? 1.f : 0.f;
  }
}

__global__ void fill_kernel(float *p, float v) { *p = v; }

// ---- naive path ----

__global__ __launch_bounds__(256) void colnorm_kernel(const float *__restrict__ O, int64_t D, int m,
                                                      float *__restrict__ partial) {
  const int64_t rows = (D + gridDim.x - 1) / gridDim.x;
  const int64_t r0 = (int64_t)blockIdx.x * rows;
  const int64_t r1 = min(D, r0 + rows);
  for (int j = threadIdx.x; j < m; j += blockDim.x) {
    float s = 0.f;
    for (int64_t i = r0; i < r1; ++i) {
      const float o = O[i * m + j];
      s += o * o;
    }
    partial[(int64_t)blockIdx.x * m + j] = s;
  }
}

// One workgroup per example j: q_j from the partial column sums (fixed order),
// then the loss epilogue on the K target entries of column j of O.
__global__ __launch_bounds__(256) void naive_epilogue_kernel(int m, int K, int64_t D, int nparts,
                                                             const float *__restrict__ partial,
                                                             const float *__restrict__ O,
                                                             const int *__restrict__ idx,
                                                             const float *__restrict__ val, int loss,
                                                             float eps, float *__restrict__ dq,
                                                             float *__restrict__ dA,
                                                             float *__restrict__ lvec,
                                                             int *__restrict__ flag) {
  __shared__ float red[256];
  __shared__ int sr[LST_MAX_K];
  __shared__ float st[LST_MAX_K], sa[LST_MAX_K];
  __shared__ int s_bad;
  const int j = blockIdx.x, t = threadIdx.x;
  if (t == 0) s_bad = 0;
  float q = 0.f;
  for (int p = t; p < nparts; p += 256) q += partial[(int64_t)p * m + j];
  red[t] = q;
  __syncthreads();
  if (t < K) {
    int rr = idx[(int64_t)j * K + t];
    if (rr < -1 || (int64_t)rr >= D) {
      atomicOr(&s_bad, 1);
      rr = -1;
    }
    sr[t] = rr;
    st[t] = val[(int64_t)j * K + t];
    sa[t] = rr >= 0 ? O[(int64_t)rr * m + j] : 0.f;
  }
  for (int w = 128; w > 0; w >>= 1) {
    if (t < w) red[t] += red[t + w];
    __syncthreads();
  }
  if (t == 0) {
    float l, gq, g[LST_MAX_K];
    loss_epilogue(loss, red[0], K, sr, st, sa, (float)D * eps, eps, l, gq, g);
    dq[j] = gq;
    for (int k = 0; k < K; ++k) dA[(int64_t)j * K + k] = g[k];
    lvec[j] = l;
    if (s_bad) atomicOr(flag, FLAG_INDEX);
  }
}

// O <- 2 O diag(dq): n4 groups of four columns per row when m % 4 == 0.
__global__ __launch_bounds__(256) void scale_cols4_kernel(float4 *__restrict__ O, int64_t total4,
                                                          int n4, const float4 *__restrict__ dq) {
  const int64_t f0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int step = (int)(stride % n4);
  int c = (int)(f0 % n4);
  for (int64_t f = f0; f < total4; f += stride) {
    const float4 s = dq[c], o = O[f];
    O[f] = make_float4(2.f * s.x * o.x, 2.f * s.y * o.y, 2.f * s.z * o.z, 2.f * s.w * o.w);
    c += step;
    if (c >= n4) c -= n4;
  }
}

__global__ __launch_bounds__(256) void scale_cols_kernel(float *__restrict__ O, int64_t total, int m,
                                                         const float *__restrict__ dq) {
  const int64_t e0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int step = (int)(stride % m);
  int c = (int)(e0 % m);
  for (int64_t e = e0; e < total; e += stride) {
    O[e] = 2.f * dq[c] * O[e];
    c += step;
    if (c >= m) c -= m;
  }
}

// Adds dA at the targets of each column (one thread per column, so repeated
// targets within a column add in order) and sums the per-example losses.
__global__ __launch_bounds__(1024) void sparse_add_kernel(float *__restrict__ O, int64_t D, int m, int K,
                                                          const int *__restrict__ idx,
                                                          const float *__restrict__ dA,
                                                          const float *__restrict__ lvec,
                                                          float *__restrict__ loss_out,
                                                          int *__restrict__ flag) {
  __shared__ float red[1024];
  const int t = threadIdx.x;
  float l = 0.f;
  for (int j = t; j < m; j += 1024) {
    for (int k = 0; k < K; ++k) {
      const int r = idx[(int64_t)j * K + k];
      if (r >= 0 && (int64_t)r < D) O[(int64_t)r * m + j] += dA[(int64_t)j * K + k];
    }
    l += lvec[j];
  }
  red[t] = l;
  __syncthreads();
  for (int w = 512; w > 0; w >>= 1) {
    if (t < w) red[t] += red[t + w];
    __syncthreads();
  }
  if (t == 0) {
    *loss_out = red[0];
    if (!isfinite(red[0])) atomicOr(flag, FLAG_NONFINITE);
  }
}

}  // namespace

hipError_t launch_gather(hipStream_t s, int m, int K, int d, int64_t D, const float *H,
                         const float *Hhat, const float *Htil, const int *idx, const float *val,
                         const float *V, int64_t ldv, int loss, float eps, float lr, float *G,
                         float *Atil, float *dq, float *dA, float *lvec, int *flag) {
  const int kpw = (K + 3) / 4;
#define LST_GATHER_REG(KPW, NV)                                                               \
  if (kpw <= KPW && d <= 64 * NV) {                                                           \
    LST_LAUNCH((gather_reg_kernel<KPW, NV>), dim3(m), dim3(kGatherThreads), 0, s, K, d, D, H, \
               Hhat, Htil, idx, val, V, ldv, loss, eps, lr, G, Atil, dq, dA, lvec, flag);     \
    return hipSuccess;                                                                        \
  }
  LST_GATHER_REG(1, 8)
  LST_GATHER_REG(2, 8)
  LST_GATHER_REG(4, 8)
  LST_GATHER_REG(1, 16)
  LST_GATHER_REG(2, 16)
#undef LST_GATHER_REG
  LST_LAUNCH(gather_kernel, dim3(m), dim3(kGatherThreads), 0, s, K, d, D, H, Hhat, Htil, idx, val, V,
             ldv, loss, eps, lr, G, Atil, dq, dA, lvec, flag);
  return hipSuccess;  // checked once per step by the caller
}

hipError_t launch_step_sync(hipStream_t s, const StepSync &wait, int *done) {
  LST_LAUNCH(step_sync_kernel, dim3(1), dim3(64), 0, s, wait, done);
  return hipGetLastError();
}

// Dynamic LDS that brings a one-workgroup kernel's allocation to the whole
// per-workgroup limit, so that no workgroup of another kernel that uses LDS is
// placed on its compute unit: the elimination keeps all four SIMDs busy, and a
// workgroup sharing the unit (a gather or GEMM tile of the main stream) ran
// more than twice as long, holding up its whole launch.  0 if the sizes cannot
// be queried.
size_t exclusive_lds_pad(const void *kernel) {
  int dev = 0, limit = 0;
  hipFuncAttributes fa{};
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&limit, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess ||
      hipFuncGetAttributes(&fa, kernel) != hipSuccess || (size_t)limit <= fa.sharedSizeBytes)
    return 0;
  return (size_t)limit - fa.sharedSizeBytes;
}

template <auto Kernel>
size_t exclusive_lds_pad_cached() {  // one value per kernel
  static const size_t pad = exclusive_lds_pad(reinterpret_cast<const void *>(Kernel));
  return pad;
}

hipError_t launch_woodbury(hipStream_t s, int m, float lr, int unit_dq, const float *dq,
                           const float *N, float *R, float *Cwork, float *Pbig, float *Cp,
                           float *Rp, int *flag, const StepSync &wait, int *done) {
  switch (m <= kWoodburyOneWG ? (m + 31) / 32 : 0) {
#define LST_WB_CASE(NB)                                                                       \
  case NB:                                                                                    \
    LST_LAUNCH((woodbury_blocked_kernel<NB>), dim3(1), dim3(64 * wb_waves<NB>()),             \
               exclusive_lds_pad_cached<woodbury_blocked_kernel<NB>>(), s, m, lr, unit_dq, dq, N, R, \
               flag, wait, done);                                                             \
    break;
    LST_WB_CASE(1)
    LST_WB_CASE(2)
    LST_WB_CASE(3)
    LST_WB_CASE(4)
#undef LST_WB_CASE
    default: {
      if (wait.wx) LST_LAUNCH(step_sync_kernel, dim3(1), dim3(64), 0, s, wait, nullptr);
      const int blocks = (int)std::min<int64_t>(((int64_t)m * m + 255) / 256, 2048);
      float *PI = Pbig + kBigBlock * kBigBlock;
      LST_LAUNCH(form_c_kernel, dim3(blocks), dim3(256), 0, s, m, lr, unit_dq, dq, N, Cwork, flag);
      int pb0 = 0, pnb = 0;
      for (int b0 = 0; b0 < m; b0 += kBigBlock) {
        const int nb = std::min(kBigBlock, m - b0), e0 = b0 + nb;
        LST_LAUNCH(pivot_block_kernel, dim3(1), dim3(64 * wb_waves<kPivotNbk>()),
                   exclusive_lds_pad_cached<pivot_block_kernel>(), s, m, b0, nb, pb0, pnb, Cwork,
                   Pbig, PI, flag);
        float *Ab = Cwork + (int64_t)b0 * m;
        GemmBatch r{};
        int n = 0;
        if (b0 > 0) r.d[n++] = gemm_desc(nb, b0, nb, Pbig, kBigBlock, 0, Ab, m, 1, Rp, m);
        if (e0 < m)
          r.d[n++] = gemm_desc(nb, m - e0, nb, Pbig, kBigBlock, 0, Ab + e0, m, 1, Rp + e0, m);
        r.d[n++] = gemm_desc(nb, nb, 0, PI, kBigBlock, 0, PI, kBigBlock, 1, Rp + b0, m, 0.f, PI,
                             kBigBlock, 1.f);  // Rp_:,b = P + I
        r.d[n++] = gemm_desc(m, nb, 0, Cp, kBigBlock, 0, Cp, kBigBlock, 1, Cp, kBigBlock, 0.f,
                             Cwork + b0, m, 1.f);  // Cp = A_:,b
        r.n = n;
        gemm_prepare(r);
        gemm_enqueue(r, nullptr, s, GEMM_OTHER);
        GemmBatch t{};
        n = 0;
        if (b0 > 0)
          t.d[n++] = gemm_desc(b0, m, nb, Cp, kBigBlock, 0, Rp, m, 1, Cwork, m, -1.f, Cwork, m, 1.f);
        if (e0 < m) {
          float *Al = Cwork + (int64_t)e0 * m;
          t.d[n++] = gemm_desc(m - e0, m, nb, Cp + (int64_t)e0 * kBigBlock, kBigBlock, 0, Rp, m, 1,
                               Al, m, -1.f, Al, m, 1.f);
        }
        t.d[n++] = gemm_desc(nb, m, 0, Rp, m, 0, Rp, m, 1, Ab, m, 0.f, Rp, m, 1.f);  // A_b,: = Rp
        t.n = n;
        gemm_prepare(t);
        gemm_enqueue(t, nullptr, s, GEMM_OTHER);
        pb0 = b0;
        pnb = nb;
      }
      LST_LAUNCH(scale_r_kernel, dim3(blocks), dim3(256), 0, s, m, pb0, lr, unit_dq, dq, Cwork, R);
      if (done) LST_LAUNCH(step_sync_kernel, dim3(1), dim3(64), 0, s, StepSync{}, done);
    }
  }
  return hipSuccess;  // checked once per step by the caller
}

hipError_t launch_scale_rows_sqrt(hipStream_t s, int m, int d, const float *H, const float *dq,
                                  float *Hs, int *flag) {
  const int blocks = (int)std::min<int64_t>(((int64_t)m * d + 255) / 256, 2048);
  LST_LAUNCH(scale_rows_sqrt_kernel, dim3(blocks), dim3(256), 0, s, m, d, H, dq, Hs, flag);
  return hipSuccess;  // checked once per step by the caller
}

hipError_t launch_push_through_r(hipStream_t s, int m, float lr, int unit_dq, const float *dq,
                                 float *R) {
  const int blocks = (int)std::min<int64_t>(((int64_t)m * m + 255) / 256, 2048);
  LST_LAUNCH(push_through_r_kernel, dim3(blocks), dim3(256), 0, s, m, lr, unit_dq, dq, R);
  return hipSuccess;  // checked once per step by the caller
}

hipError_t launch_mblock(hipStream_t s, int m, int K, const int *idx, const float *lvec,
                         const float *dq, const float *dA, const float *Mhat, const float *HZ,
                         float *M, float *loss_out, int *flag) {
  const int blocks = (m * m + kMblockThreads - 1) / kMblockThreads;
  LST_LAUNCH(mblock_kernel, dim3(blocks), dim3(kMblockThreads), 0, s, m, K, idx, lvec, dq,
                     dA, Mhat, HZ, M, loss_out, flag);
  return hipSuccess;  // checked once per step by the caller
}

hipError_t launch_scatter(hipStream_t s, int m, int K, int d, float lr, const int *idx,
                          const float *dA, const float *P, float *V, int64_t ldv, const int *flag) {
  const int n = m * K;
  if (n == 0) return hipSuccess;
  LST_LAUNCH(scatter_kernel, dim3(n), dim3(kScatterThreads), 2 * n * sizeof(int), s, n, K,
                     d, lr, idx, dA, P, V, ldv, flag);
  return hipSuccess;  // checked once per step by the caller
}

hipError_t launch_identity(hipStream_t s, float *A, int d, int64_t ld) {
  int blocks = (int)(((int64_t)d * d + 255) / 256);
  if (blocks > 4096) blocks = 4096;
  LST_LAUNCH(identity_kernel, dim3(blocks), dim3(256), 0, s, A, d, ld);
  return hipGetLastError();
}

hipError_t launch_fill(hipStream_t s, float *p, float v) {
  LST_LAUNCH(fill_kernel, dim3(1), dim3(1), 0, s, p, v);
  return hipGetLastError();
}

hipError_t launch_colnorm(hipStream_t s, const float *O, int64_t D, int m, float *partial,
                          int nblk) {
  LST_LAUNCH(colnorm_kernel, dim3(nblk), dim3(256), 0, s, O, D, m, partial);
  return hipGetLastError();
}

hipError_t launch_naive_epilogue(hipStream_t s, int m, int K, int64_t D, int nparts,
                                 const float *partial, const float *O, const int *idx,
                                 const float *val, int loss, float eps, float *dq, float *dA,
                                 float *lvec, int *flag) {
  LST_LAUNCH(naive_epilogue_kernel, dim3(m), dim3(256), 0, s, m, K, D, nparts, partial, O, idx,
             val, loss, eps, dq, dA, lvec, flag);
  return hipGetLastError();
}

hipError_t launch_grad_o(hipStream_t s, float *O, int64_t D, int m, int K, const float *dq,
                         const int *idx, const float *dA, const float *lvec, float *loss_out,
                         int *flag) {
  const int64_t total = D * m;
  const bool v4 = (m & 3) == 0 && (reinterpret_cast<uintptr_t>(O) & 15) == 0 &&
                  (reinterpret_cast<uintptr_t>(dq) & 15) == 0;
  const int64_t units = v4 ? total / 4 : total;
  int blocks = (int)((units + 255) / 256);
  if (blocks > 8192) blocks = 8192;
  if (v4)
    LST_LAUNCH(scale_cols4_kernel, dim3(blocks), dim3(256), 0, s, reinterpret_cast<float4 *>(O),
               units, m / 4, reinterpret_cast<const float4 *>(dq));
  else
    LST_LAUNCH(scale_cols_kernel, dim3(blocks), dim3(256), 0, s, O, total, m, dq);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  LST_LAUNCH(sparse_add_kernel, dim3(1), dim3(1024), 0, s, O, D, m, K, idx, dA, lvec, loss_out,
             flag);
  return hipGetLastError();
}

}  // namespace lst
