// Non-GEMM kernels of the factored step and of the naive comparison path.
//
//   gather   -- the sparse part of Algorithm 4: A_kj = H~_j . V_{K_kj} (eq.
//               gen-A-fact), q_j = h_j . H^_j (eq. qvec), the loss epilogue
//               (l_j, dl/dq_j, dl/dA_kj) and G_j = sum_k dl/dA_kj V_{K_kj}
//               (the V^T Yring of eq. gen-Zhat-fact; Algorithm 3 step 2's V^T Y
//               up to the factor -2).  One wavefront per example.
//   small    -- the m x m block: L = sum_j l_j, M of eq. gen-M (with the sparse
//               Yring^T Yring by index equality), the Woodbury matrix
//               C = I - 2 eta S H^T H S and its inverse (Gauss-Jordan, no
//               pivoting: C is symmetric positive definite exactly when the
//               step is admissible), R = 2 eta S C^{-1} S, and the sort of the
//               (row, slot) keys that makes the V scatter conflict free.
//   scatter  -- eq. updateV / gen-updateV: V_r -= eta sum_{slots of row r}
//               dl/dA P_j, one wavefront per distinct row, slots in a fixed
//               order, so repeated rows never race and results are
//               reproducible bit for bit.
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

__global__ __launch_bounds__(64) void gather_kernel(int K, int d, int64_t D, const float *__restrict__ H,
                                                    const float *__restrict__ Hhat,
                                                    const float *__restrict__ Htil,
                                                    const int *__restrict__ idx,
                                                    const float *__restrict__ val,
                                                    const float *__restrict__ V, int64_t ldv, int loss,
                                                    float eps, float lr, float *__restrict__ G,
                                                    float *__restrict__ Atil, float *__restrict__ dq,
                                                    float *__restrict__ dA, float *__restrict__ lvec,
                                                    int *__restrict__ flag) {
  __shared__ int sr[LST_MAX_K];
  __shared__ float sa[LST_MAX_K], st[LST_MAX_K], sg[LST_MAX_K];
  const int j = blockIdx.x;
  const int lane = threadIdx.x;
  const float *h = H + (int64_t)j * d;
  const float *hh = Hhat + (int64_t)j * d;
  const float *ht = Htil + (int64_t)j * d;

  float qs = 0.f;
  for (int c = lane; c < d; c += 64) qs += h[c] * hh[c];
  const float q = wave_sum(qs);

  int bad = 0;
  for (int k = 0; k < K; ++k) {
    int r = idx[(int64_t)j * K + k];
    if (r < -1 || (int64_t)r >= D) {
      bad = 1;
      r = -1;
    }
    float a = 0.f;
    if (r >= 0) {
      const float *vr = V + (int64_t)r * ldv;
      float s = 0.f;
      for (int c = lane; c < d; c += 64) s += ht[c] * vr[c];
      a = wave_sum(s);
    }
    if (lane == 0) {
      sr[k] = r;
      sa[k] = a;
      st[k] = val[(int64_t)j * K + k];
    }
  }
  if (bad && lane == 0) atomicOr(flag, FLAG_INDEX);
  __syncthreads();

  float l, gq;
  if (lane == 0) {
    loss_epilogue(loss, q, K, sr, st, sa, (float)D * eps, eps, l, gq, sg);
    dq[j] = gq;
    lvec[j] = l;
    sa[0] = gq;  // broadcast dl/dq (sa no longer needed)
  }
  __syncthreads();
  gq = sa[0];
  for (int k = lane; k < K; k += 64) dA[(int64_t)j * K + k] = sg[k];

  const float s2 = 2.f * lr * gq;
  for (int c = lane; c < d; c += 64) {
    float s = 0.f;
    for (int k = 0; k < K; ++k) {
      const int r = sr[k];
      if (r >= 0) s += sg[k] * V[(int64_t)r * ldv + c];
    }
    G[(int64_t)j * d + c] = s;
    Atil[(int64_t)j * d + c] = s2 * ht[c];
  }
}

constexpr int kSmallThreads = 1024;
constexpr int kMaxSortKeys = 8192;

// Bitonic sort of n (power of two) 64-bit keys in LDS, ascending.
__device__ void bitonic_sort(unsigned long long *key, int n) {
  for (int size = 2; size <= n; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int t = threadIdx.x; t < (n >> 1); t += blockDim.x) {
        const int lo = 2 * t - (t & (stride - 1));
        const int hi = lo + stride;
        const bool up = ((lo & size) == 0);
        const unsigned long long a = key[lo], b = key[hi];
        if ((a > b) == up) {
          key[lo] = b;
          key[hi] = a;
        }
      }
      __syncthreads();
    }
  }
}

// Gauss-Jordan inversion in place, matrix held in registers: thread (ti, tj)
// of a 32 x 32 grid owns the B x B block at rows ti*B.., cols tj*B...  Entries
// outside m x m are the identity and take no part.  Returns false (uniformly)
// if a pivot is not positive and finite.
template <int B>
__device__ bool gj_invert_regs(float (&a)[B][B], int m, float *srow, float *scol) {
  const int t = threadIdx.x;
  const int ti = t >> 5, tj = t & 31;
  for (int k = 0; k < m; ++k) {
    float *rowk = srow + (k & 1) * (32 * B);
    float *colk = scol + (k & 1) * (32 * B);
    const int kb = k / B, kr = k - kb * B;
    if (ti == kb) {
#pragma unroll
      for (int c = 0; c < B; ++c) rowk[tj * B + c] = a[kr][c];
    }
    if (tj == kb) {
#pragma unroll
      for (int r = 0; r < B; ++r) colk[ti * B + r] = a[r][kr];
    }
    __syncthreads();
    const float p = rowk[k];
    if (!(p > 0.f) || !isfinite(p)) return false;
    const float ip = 1.f / p;
    float cr[B], rc[B];
#pragma unroll
    for (int r = 0; r < B; ++r) cr[r] = colk[ti * B + r];
#pragma unroll
    for (int c = 0; c < B; ++c) rc[c] = rowk[tj * B + c];
#pragma unroll
    for (int r = 0; r < B; ++r) {
      const int i = ti * B + r;
#pragma unroll
      for (int c = 0; c < B; ++c) {
        const int j = tj * B + c;
        if (i == k) {
          a[r][c] = (j == k) ? ip : rc[c] * ip;
        } else if (j == k) {
          a[r][c] = -cr[r] * ip;
        } else {
          a[r][c] -= cr[r] * (rc[c] * ip);
        }
      }
    }
  }
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

// Entry (i, j) of M (eq. gen-M, dl/ds = 0):
//   4 dq_i M^_ij dq_j + Yring^T Yring_ij + 2 dq_i (H~^T G)_ij + 2 dq_j (H~^T G)_ji
__device__ __forceinline__ float m_entry(int i, int j, int m, int K, const int *idx,
                                         const float *dq, const float *dA, const float *Mhat,
                                         const float *HZ) {
  float yy = 0.f;
  for (int k = 0; k < K; ++k) {
    const int ri = idx[(int64_t)i * K + k];
    if (ri < 0) continue;
    const float gi = dA[(int64_t)i * K + k];
    for (int kk = 0; kk < K; ++kk)
      if (idx[(int64_t)j * K + kk] == ri) yy += gi * dA[(int64_t)j * K + kk];
  }
  return 4.f * dq[i] * Mhat[(int64_t)i * m + j] * dq[j] + yy +
         2.f * dq[i] * HZ[(int64_t)i * m + j] + 2.f * dq[j] * HZ[(int64_t)j * m + i];
}

template <int B>
__global__ __launch_bounds__(kSmallThreads) void small_kernel(
    int m, int K, float lr, const int *__restrict__ idx, const float *__restrict__ lvec,
    const float *__restrict__ dq, const float *__restrict__ dA, const float *__restrict__ N,
    const float *__restrict__ Mhat, const float *__restrict__ HZ, float *__restrict__ M,
    float *__restrict__ R, float *__restrict__ Cwork, int *__restrict__ srow_out,
    int *__restrict__ sslot_out, int *__restrict__ nvalid, float *__restrict__ loss_out,
    int *__restrict__ flag) {
  __shared__ unsigned long long skey[kMaxSortKeys];
  __shared__ float red[kSmallThreads];
  __shared__ int s_abort;
  const int t = threadIdx.x;

  // Loss: fixed-order sum of the per-example losses; dl/dq must be >= 0.
  float ls = 0.f;
  int neg = 0;
  for (int j = t; j < m; j += kSmallThreads) {
    ls += lvec[j];
    if (!(dq[j] >= 0.f)) neg = 1;
  }
  red[t] = ls;
  if (t == 0) s_abort = *flag;
  __syncthreads();
  if (neg) atomicOr(&s_abort, FLAG_NOT_SPD);
  for (int s = kSmallThreads / 2; s > 0; s >>= 1) {
    if (t < s) red[t] += red[t + s];
    __syncthreads();
  }
  if (t == 0) {
    const float L = red[0];
    *loss_out = L;
    if (!isfinite(L)) s_abort |= FLAG_NONFINITE;
    if (s_abort) atomicOr(flag, s_abort);
  }
  __syncthreads();
  if (s_abort) return;

  // Sort (row, slot) keys of the valid target slots.
  const int n = m * K;
  int np = 1;
  while (np < n) np <<= 1;
  for (int e = t; e < np; e += kSmallThreads) {
    unsigned long long key = ~0ull;
    if (e < n) {
      const int r = idx[e];
      if (r >= 0) key = ((unsigned long long)(unsigned)r << 32) | (unsigned)e;
    }
    skey[e] = key;
  }
  __syncthreads();
  bitonic_sort(skey, np);
  int cnt = 0;
  for (int e = t; e < n; e += kSmallThreads) {
    const unsigned long long key = skey[e];
    if (key != ~0ull) {
      srow_out[e] = (int)(key >> 32);
      sslot_out[e] = (int)(key & 0xffffffffu);
      ++cnt;
    }
  }
  red[t] = (float)cnt;
  __syncthreads();
  for (int s = kSmallThreads / 2; s > 0; s >>= 1) {
    if (t < s) red[t] += red[t + s];
    __syncthreads();
  }
  if (t == 0) *nvalid = (int)red[0];

  // M (for the Q update) over all m x m entries.
  for (int e = t; e < m * m; e += kSmallThreads) {
    const int i = e / m, j = e - i * m;
    M[e] = m_entry(i, j, m, K, idx, dq, dA, Mhat, HZ);
  }

  // C = I - 2 eta S N S, inverted in place; R = 2 eta S C^{-1} S.
  float *srow = reinterpret_cast<float *>(skey);
  float *scol = srow + 2048;
  bool ok;
  if constexpr (B > 0) {
    float a[B][B];
    const int ti = t >> 5, tj = t & 31;
#pragma unroll
    for (int r = 0; r < B; ++r)
#pragma unroll
      for (int c = 0; c < B; ++c) {
        const int i = ti * B + r, j = tj * B + c;
        float v = (i == j) ? 1.f : 0.f;
        if (i < m && j < m)
          v -= 2.f * lr * sqrtf(dq[i]) * N[(int64_t)i * m + j] * sqrtf(dq[j]);
        a[r][c] = v;
      }
    __syncthreads();  // skey reuse as srow/scol
    ok = gj_invert_regs<B>(a, m, srow, scol);
    if (ok) {
#pragma unroll
      for (int r = 0; r < B; ++r)
#pragma unroll
        for (int c = 0; c < B; ++c) {
          const int i = ti * B + r, j = tj * B + c;
          if (i < m && j < m) R[(int64_t)i * m + j] = 2.f * lr * sqrtf(dq[i]) * a[r][c] * sqrtf(dq[j]);
        }
    }
  } else {
    for (int e = t; e < m * m; e += kSmallThreads) {
      const int i = e / m, j = e - i * m;
      Cwork[e] = ((i == j) ? 1.f : 0.f) - 2.f * lr * sqrtf(dq[i]) * N[e] * sqrtf(dq[j]);
    }
    __syncthreads();
    ok = gj_invert_global(Cwork, m, srow, scol);
    if (ok) {
      for (int e = t; e < m * m; e += kSmallThreads) {
        const int i = e / m, j = e - i * m;
        R[e] = 2.f * lr * sqrtf(dq[i]) * Cwork[e] * sqrtf(dq[j]);
      }
    }
  }
  if (!ok && t == 0) atomicOr(flag, FLAG_NOT_SPD);
}

__global__ __launch_bounds__(256) void scatter_kernel(int K, int d, float lr, const int *__restrict__ srow,
                                                      const int *__restrict__ sslot,
                                                      const int *__restrict__ nvalid,
                                                      const float *__restrict__ dA,
                                                      const float *__restrict__ P, float *__restrict__ V,
                                                      int64_t ldv, const int *__restrict__ gate) {
  if (*gate != 0) return;
  const int p = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int n = *nvalid;
  if (p >= n) return;
  const int r = srow[p];
  if (p > 0 && srow[p - 1] == r) return;  // not the first slot of its row
  int e = p + 1;
  while (e < n && srow[e] == r) ++e;
  float *vr = V + (int64_t)r * ldv;
  for (int c = lane; c < d; c += 64) {
    float acc = 0.f;
    for (int s = p; s < e; ++s) {
      const int slot = sslot[s];
      acc += dA[slot] * P[(int64_t)(slot / K) * d + c];
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
  hipLaunchKernelGGL(gather_kernel, dim3(m), dim3(64), 0, s, K, d, D, H, Hhat, Htil, idx, val, V,
                     ldv, loss, eps, lr, G, Atil, dq, dA, lvec, flag);
  return hipGetLastError();
}

hipError_t launch_small(hipStream_t s, int m, int K, float lr, const int *idx, const float *lvec,
                        const float *dq, const float *dA, const float *N, const float *Mhat,
                        const float *HZ, float *M, float *R, float *Cwork, int *srow, int *sslot,
                        int *nvalid, float *loss_out, int *flag) {
  if (m <= 32)
    hipLaunchKernelGGL(small_kernel<1>, dim3(1), dim3(kSmallThreads), 0, s, m, K, lr, idx, lvec,
                       dq, dA, N, Mhat, HZ, M, R, Cwork, srow, sslot, nvalid, loss_out, flag);
  else if (m <= 64)
    hipLaunchKernelGGL(small_kernel<2>, dim3(1), dim3(kSmallThreads), 0, s, m, K, lr, idx, lvec,
                       dq, dA, N, Mhat, HZ, M, R, Cwork, srow, sslot, nvalid, loss_out, flag);
  else if (m <= 128)
    hipLaunchKernelGGL(small_kernel<4>, dim3(1), dim3(kSmallThreads), 0, s, m, K, lr, idx, lvec,
                       dq, dA, N, Mhat, HZ, M, R, Cwork, srow, sslot, nvalid, loss_out, flag);
  else if (m <= 256)
    hipLaunchKernelGGL(small_kernel<8>, dim3(1), dim3(kSmallThreads), 0, s, m, K, lr, idx, lvec,
                       dq, dA, N, Mhat, HZ, M, R, Cwork, srow, sslot, nvalid, loss_out, flag);
  else
    hipLaunchKernelGGL(small_kernel<0>, dim3(1), dim3(kSmallThreads), 0, s, m, K, lr, idx, lvec,
                       dq, dA, N, Mhat, HZ, M, R, Cwork, srow, sslot, nvalid, loss_out, flag);
  return hipGetLastError();
}

hipError_t launch_scatter(hipStream_t s, int m, int K, int d, float lr, const int *srow,
                          const int *sslot, const int *nvalid, const float *dA, const float *P,
                          float *V, int64_t ldv, const int *flag) {
  const int n = m * K;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(scatter_kernel, dim3((n + 3) / 4), dim3(256), 0, s, K, d, lr, srow, sslot,
                     nvalid, dA, P, V, ldv, flag);
  return hipGetLastError();
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
