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
#include "lst_internal.h"

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

constexpr int kMaxSortKeys = 8192;

// Gauss-Jordan inversion in place, matrix held in registers: thread (ti, tj)
// of a T x T grid owns the B x B block at rows ti*B.., cols tj*B...  Entries
// outside m x m are the identity and take no part.  Returns false (uniformly)
// if a pivot is not positive and finite.
//
// One elimination step on pivot k (p = A_kk) is written as
//   A' = X - f g^T,  X = A with column k replaced by e_k,
//   f_i = A_ik (i != k), f_k = p - 1,   g_j = A_kj / p (j != k), g_k = 1 / p,
// which gives A'_kj = A_kj / p, A'_ik = -A_ik / p, A'_kk = 1 / p and
// A'_ij = A_ij - A_ik A_kj / p elsewhere.  The pivot's position inside a block
// (KR) is a compile-time index of the unrolled inner loop, so the register
// block is never indexed at run time.  Lookahead: right after reading pivot k,
// the owners of row and column k+1 compute their updated values and publish
// them, so the one barrier per pivot waits only for the bulk of the update.
template <int B, int KR>
__device__ __forceinline__ float gj_new(const float (&a)[B][B], int r, int c, bool own_row,
                                        bool own_col, const float (&f)[B], const float (&g)[B]) {
  float x = a[r][c];
  if (c == KR) x = own_col ? ((r == KR && own_row) ? 1.f : 0.f) : x;
  return x - f[r] * g[c];
}

template <int T, int B, int KR>
__device__ __forceinline__ bool gj_step(float (&a)[B][B], int kb, int m, float *srow, float *scol) {
  const int t = threadIdx.x;
  const int ti = t / T, tj = t % T;
  const int k = kb * B + KR;
  const float *rowk = srow + (k & 1) * (T * B);
  const float *colk = scol + (k & 1) * (T * B);
  __syncthreads();
  const float p = rowk[k];
  if (!(p > 0.f) || !isfinite(p)) return false;
  const float ip = 1.f / p;
  const bool own_row = (ti == kb), own_col = (tj == kb);
  float f[B], g[B];
#pragma unroll
  for (int r = 0; r < B; ++r) f[r] = colk[ti * B + r];
#pragma unroll
  for (int c = 0; c < B; ++c) g[c] = rowk[tj * B + c] * ip;
  if (own_row) f[KR] = p - 1.f;
  if (own_col) g[KR] = ip;
  if (k + 1 < m) {
    constexpr int KR1 = (KR + 1 < B) ? KR + 1 : 0;
    const int kb1 = (KR + 1 < B) ? kb : kb + 1;
    float *rown = srow + ((k + 1) & 1) * (T * B);
    float *coln = scol + ((k + 1) & 1) * (T * B);
    if (ti == kb1) {
#pragma unroll
      for (int c = 0; c < B; ++c) rown[tj * B + c] = gj_new<B, KR>(a, KR1, c, own_row, own_col, f, g);
    }
    if (tj == kb1) {
#pragma unroll
      for (int r = 0; r < B; ++r) coln[ti * B + r] = gj_new<B, KR>(a, r, KR1, own_row, own_col, f, g);
    }
  }
#pragma unroll
  for (int r = 0; r < B; ++r)
#pragma unroll
    for (int c = 0; c < B; ++c) a[r][c] = gj_new<B, KR>(a, r, c, own_row, own_col, f, g);
  return true;
}

template <int T, int B, int KR>
__device__ __forceinline__ bool gj_block(float (&a)[B][B], int kb, int m, float *srow, float *scol) {
  if constexpr (KR < B) {
    if (kb * B + KR >= m) return true;
    if (!gj_step<T, B, KR>(a, kb, m, srow, scol)) return false;
    return gj_block<T, B, KR + 1>(a, kb, m, srow, scol);
  } else {
    return true;
  }
}

template <int T, int B>
__device__ bool gj_invert_regs(float (&a)[B][B], int m, float *srow, float *scol) {
  // publish pivot 0
  const int t = threadIdx.x;
  const int ti = t / T, tj = t % T;
  if (ti == 0) {
#pragma unroll
    for (int c = 0; c < B; ++c) srow[tj * B + c] = a[0][c];
  }
  if (tj == 0) {
#pragma unroll
    for (int r = 0; r < B; ++r) scol[ti * B + r] = a[r][0];
  }
  const int nb = (m + B - 1) / B;
  for (int kb = 0; kb < nb; ++kb)
    if (!gj_block<T, B, 0>(a, kb, m, srow, scol)) return false;
  return true;
}

// Gauss-Jordan inversion in place of an m x m matrix in global memory (large m).
__device__ bool gj_invert_global(float *A, int m, float *srow, float *scol) {
  for (int k = 0; k < m; ++k) {
    for (int t = threadIdx.x; t < m; t += blockDim.x) {
      srow[t] = A[(int64_t)k * m + t];
      scol[t] = A[(int64_t)t * m + k];
    }
    __syncthreads();
    const float p = srow[k];
    if (!(p > 0.f) || !isfinite(p)) return false;
    const float ip = 1.f / p;
    for (int e = threadIdx.x; e < m * m; e += blockDim.x) {
      const int i = e / m, j = e - i * m;
      float v;
      if (i == k)
        v = (j == k) ? ip : srow[j] * ip;
      else if (j == k)
        v = -scol[i] * ip;
      else
        v = A[e] - scol[i] * (srow[j] * ip);
      A[e] = v;
    }
    __syncthreads();
  }
  return true;
}

// Woodbury matrix C = I - 2 eta S N S with S = diag(dl/dq)^{1/2} and N = H^T H,
// its inverse, and R = 2 eta S C^{-1} S (U_new^{-T} = U^{-T} + (U^{-T} H) R H^T).
// unit_dq: dl/dq = 1 for every example (squared error), dq is not read.
template <int T, int B>
__global__ __launch_bounds__(T *T) void woodbury_kernel(int m, float lr, int unit_dq,
                                                       const float *__restrict__ dq,
                                                       const float *__restrict__ N,
                                                       float *__restrict__ R, float *__restrict__ Cwork,
                                                       int *__restrict__ flag) {
  __shared__ float sbuf[4096];
  __shared__ float sq[LST_MAX_M];
  __shared__ int s_bad;
  const int t = threadIdx.x;
  if (t == 0) s_bad = 0;
  __syncthreads();
  for (int i = t; i < m; i += T * T) {
    const float v = unit_dq ? 1.f : dq[i];
    if (!(v >= 0.f)) atomicOr(&s_bad, 1);  // negative or NaN dl/dq: no real square root
    sq[i] = sqrtf(fmaxf(v, 0.f));
  }
  __syncthreads();
  if (s_bad) {
    if (t == 0) atomicOr(flag, FLAG_NOT_SPD);
    return;
  }
  bool ok;
  if constexpr (B > 0) {
    float a[B][B];
    const int ti = t / T, tj = t % T;
#pragma unroll
    for (int r = 0; r < B; ++r)
#pragma unroll
      for (int c = 0; c < B; ++c) {
        const int i = ti * B + r, j = tj * B + c;
        float v = (i == j) ? 1.f : 0.f;
        if (i < m && j < m) v -= 2.f * lr * sq[i] * N[(int64_t)i * m + j] * sq[j];
        a[r][c] = v;
      }
    ok = gj_invert_regs<T, B>(a, m, sbuf, sbuf + 2048);
    if (ok) {
#pragma unroll
      for (int r = 0; r < B; ++r)
#pragma unroll
        for (int c = 0; c < B; ++c) {
          const int i = ti * B + r, j = tj * B + c;
          if (i < m && j < m) R[(int64_t)i * m + j] = 2.f * lr * sq[i] * a[r][c] * sq[j];
        }
    }
  } else {
    for (int e = t; e < m * m; e += T * T) {
      const int i = e / m, j = e - i * m;
      Cwork[e] = ((i == j) ? 1.f : 0.f) - 2.f * lr * sq[i] * N[e] * sq[j];
    }
    __syncthreads();
    ok = gj_invert_global(Cwork, m, sbuf, sbuf + 2048);
    if (ok) {
      for (int e = t; e < m * m; e += T * T) {
        const int i = e / m, j = e - i * m;
        R[e] = 2.f * lr * sq[i] * Cwork[e] * sq[j];
      }
    }
  }
  if (!ok && t == 0) atomicOr(flag, FLAG_NOT_SPD);
}

// Loss L = sum_j l_j (fixed order; non-finite -> error flag) and the Q-update
// matrix M of eq. gen-M (dl/ds = 0):
//   M_ij = 4 dq_i M^_ij dq_j + (Yring^T Yring)_ij + 2 dq_i (H~^T G)_ij + 2 dq_j (H~^T G)_ji
// Column j of the sparse Yring is kept as a sorted list of (row, value) pairs,
// so (Yring^T Yring)_ij is a merge of two lists in ascending row order.  Each
// workgroup builds the m lists in LDS and fills kMblockThreads entries of M;
// workgroup 0 also forms the loss.
constexpr int kMblockThreads = 256;

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

  for (int q = t; q < m; q += kMblockThreads) {
    int *lr = lrow + q * K;
    float *lv = lval + q * K;
    int c = 0;
    for (int k = 0; k < K; ++k) {
      const int r = idx[(int64_t)q * K + k];
      if (r < 0) continue;
      const float g = dA[(int64_t)q * K + k];
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

constexpr int kScatterThreads = 256;

// One workgroup per target slot s (slot = j*K + k of the m x K index matrix).
// The lowest slot of each V row does the row's update: it lists, in ascending
// slot order, every slot with the same row and applies
//   V_r -= eta sum_{slots s' of row r} dl/dA_s' P_{j(s')},
// so each distinct row has exactly one writer and a fixed summation order.
__global__ __launch_bounds__(kScatterThreads) void scatter_kernel(
    int n, int K, int d, float lr, const int *__restrict__ idx, const float *__restrict__ dA,
    const float *__restrict__ P, float *__restrict__ V, int64_t ldv, const int *__restrict__ gate) {
  extern __shared__ int sh[];
  int *sidx = sh;        // n target rows
  int *slist = sh + n;   // slots of this row, ascending
  __shared__ int swcnt[kScatterThreads / 64];
  if (*gate != 0) return;
  const int s = blockIdx.x;
  const int r = idx[s];
  if (r < 0) return;
  int dup = 0;
  for (int q = threadIdx.x; q < n; q += kScatterThreads) {
    const int v = idx[q];
    sidx[q] = v;
    dup |= (q < s && v == r);
  }
  if (__syncthreads_or(dup)) return;  // an earlier slot owns this row

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int total = 0;
  for (int base = s; base < n; base += kScatterThreads) {
    const int q = base + threadIdx.x;
    const bool match = q < n && sidx[q] == r;
    const unsigned long long mask = __ballot(match);
    if (lane == 0) swcnt[w] = __popcll(mask);
    __syncthreads();
    int before = total;
    for (int x = 0; x < w; ++x) before += swcnt[x];
    if (match) slist[before + __popcll(mask & ((1ull << lane) - 1ull))] = q;
    for (int x = 0; x < kScatterThreads / 64; ++x) total += swcnt[x];
    __syncthreads();
  }

  float *vr = V + (int64_t)r * ldv;
  for (int c = threadIdx.x; c < d; c += kScatterThreads) {
    float acc = 0.f;
    for (int t = 0; t < total; ++t) {
      const int q = slist[t];
      acc += dA[q] * P[(int64_t)(q / K) * d + c];
    }
    vr[c] -= lr * acc;
  }
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

__global__ __launch_bounds__(1024) void naive_epilogue_kernel(int m, int K, int64_t D, int nblk,
                                                              const float *__restrict__ partial,
                                                              const float *__restrict__ O,
                                                              const int *__restrict__ idx,
                                                              const float *__restrict__ val, int loss,
                                                              float eps, float *__restrict__ dq,
                                                              float *__restrict__ dA,
                                                              float *__restrict__ loss_out,
                                                              int *__restrict__ flag) {
  __shared__ float red[1024];
  __shared__ int s_flag;
  const int t = threadIdx.x;
  if (t == 0) s_flag = 0;
  __syncthreads();
  float lsum = 0.f;
  for (int j = t; j < m; j += blockDim.x) {
    float q = 0.f;
    for (int b = 0; b < nblk; ++b) q += partial[(int64_t)b * m + j];
    int r[LST_MAX_K];
    float tv[LST_MAX_K], a[LST_MAX_K], g[LST_MAX_K];
    for (int k = 0; k < K; ++k) {
      int rr = idx[(int64_t)j * K + k];
      if (rr < -1 || (int64_t)rr >= D) {
        atomicOr(&s_flag, FLAG_INDEX);
        rr = -1;
      }
      r[k] = rr;
      tv[k] = val[(int64_t)j * K + k];
      a[k] = rr >= 0 ? O[(int64_t)rr * m + j] : 0.f;
    }
    float l, gq;
    loss_epilogue(loss, q, K, r, tv, a, (float)D * eps, eps, l, gq, g);
    dq[j] = gq;
    for (int k = 0; k < K; ++k) dA[(int64_t)j * K + k] = g[k];
    lsum += l;
  }
  red[t] = lsum;
  __syncthreads();
  for (int s = 512; s > 0; s >>= 1) {
    if (t < s) red[t] += red[t + s];
    __syncthreads();
  }
  if (t == 0) {
    *loss_out = red[0];
    int f = s_flag;
    if (!isfinite(red[0])) f |= FLAG_NONFINITE;
    if (f) atomicOr(flag, f);
  }
}

__global__ __launch_bounds__(256) void scale_cols_kernel(float *__restrict__ O, int64_t total, int m,
                                                         const float *__restrict__ dq) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    O[e] = 2.f * dq[e % m] * O[e];
  }
}

__global__ __launch_bounds__(256) void sparse_add_kernel(float *__restrict__ O, int64_t D, int m, int K,
                                                         const int *__restrict__ idx,
                                                         const float *__restrict__ dA) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= m) return;
  for (int k = 0; k < K; ++k) {
    const int r = idx[(int64_t)j * K + k];
    if (r >= 0 && (int64_t)r < D) O[(int64_t)r * m + j] += dA[(int64_t)j * K + k];
  }
}

}  // namespace

hipError_t launch_gather(hipStream_t s, int m, int K, int d, int64_t D, const float *H,
                         const float *Hhat, const float *Htil, const int *idx, const float *val,
                         const float *V, int64_t ldv, int loss, float eps, float lr, float *G,
                         float *Atil, float *dq, float *dA, float *lvec, int *flag) {
  hipLaunchKernelGGL(gather_kernel, dim3(m), dim3(kGatherThreads), 0, s, K, d, D, H, Hhat, Htil, idx, val, V,
                     ldv, loss, eps, lr, G, Atil, dq, dA, lvec, flag);
  return hipSuccess;  // checked once per step by the caller
}

hipError_t launch_woodbury(hipStream_t s, int m, float lr, int unit_dq, const float *dq,
                           const float *N, float *R, float *Cwork, int *flag) {
  if (m <= 32)
    hipLaunchKernelGGL((woodbury_kernel<16, 2>), dim3(1), dim3(256), 0, s, m, lr, unit_dq, dq, N, R,
                       Cwork, flag);
  else if (m <= 64)
    hipLaunchKernelGGL((woodbury_kernel<16, 4>), dim3(1), dim3(256), 0, s, m, lr, unit_dq, dq, N, R,
                       Cwork, flag);
  else if (m <= 128)
    hipLaunchKernelGGL((woodbury_kernel<32, 4>), dim3(1), dim3(1024), 0, s, m, lr, unit_dq, dq, N,
                       R, Cwork, flag);
  else if (m <= 256)
    hipLaunchKernelGGL((woodbury_kernel<32, 8>), dim3(1), dim3(1024), 0, s, m, lr, unit_dq, dq, N,
                       R, Cwork, flag);
  else
    hipLaunchKernelGGL((woodbury_kernel<32, 0>), dim3(1), dim3(1024), 0, s, m, lr, unit_dq, dq, N,
                       R, Cwork, flag);
  return hipSuccess;  // checked once per step by the caller
}

hipError_t launch_mblock(hipStream_t s, int m, int K, const int *idx, const float *lvec,
                         const float *dq, const float *dA, const float *Mhat, const float *HZ,
                         float *M, float *loss_out, int *flag) {
  const int blocks = (m * m + kMblockThreads - 1) / kMblockThreads;
  hipLaunchKernelGGL(mblock_kernel, dim3(blocks), dim3(kMblockThreads), 0, s, m, K, idx, lvec, dq,
                     dA, Mhat, HZ, M, loss_out, flag);
  return hipSuccess;  // checked once per step by the caller
}

hipError_t launch_scatter(hipStream_t s, int m, int K, int d, float lr, const int *idx,
                          const float *dA, const float *P, float *V, int64_t ldv, const int *flag) {
  const int n = m * K;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(scatter_kernel, dim3(n), dim3(kScatterThreads), 2 * n * sizeof(int), s, n, K,
                     d, lr, idx, dA, P, V, ldv, flag);
  return hipSuccess;  // checked once per step by the caller
}

hipError_t launch_identity(hipStream_t s, float *A, int d, int64_t ld) {
  int blocks = (int)(((int64_t)d * d + 255) / 256);
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(identity_kernel, dim3(blocks), dim3(256), 0, s, A, d, ld);
  return hipGetLastError();
}

hipError_t launch_fill(hipStream_t s, float *p, float v) {
  hipLaunchKernelGGL(fill_kernel, dim3(1), dim3(1), 0, s, p, v);
  return hipGetLastError();
}

hipError_t launch_colnorm(hipStream_t s, const float *O, int64_t D, int m, float *partial,
                          int nblk) {
  hipLaunchKernelGGL(colnorm_kernel, dim3(nblk), dim3(256), 0, s, O, D, m, partial);
  return hipGetLastError();
}

hipError_t launch_naive_epilogue(hipStream_t s, int m, int K, int64_t D, int nblk,
                                 const float *partial, const float *O, const int *idx,
                                 const float *val, int loss, float eps, float *dq, float *dA,
                                 float *loss_out, int *flag) {
  hipLaunchKernelGGL(naive_epilogue_kernel, dim3(1), dim3(1024), 0, s, m, K, D, nblk, partial, O,
                     idx, val, loss, eps, dq, dA, loss_out, flag);
  return hipGetLastError();
}

hipError_t launch_grad_o(hipStream_t s, float *O, int64_t D, int m, int K, const float *dq,
                         const int *idx, const float *dA) {
  const int64_t total = D * m;
  int blocks = (int)((total + 255) / 256);
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(scale_cols_kernel, dim3(blocks), dim3(256), 0, s, O, total, m, dq);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(sparse_add_kernel, dim3((m + 255) / 256), dim3(256), 0, s, O, D, m, K, idx,
                     dA);
  return hipGetLastError();
}

}  // namespace lst
