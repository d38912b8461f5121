// Non-GEMM kernels outside the factored step: identity and fill, and the naive
// comparison path's column norms of O, loss epilogue over the explicit output and
// grad_O = 2 O diag(dl/dq) + Yring (eq. gen-grad-O).
#include <algorithm>

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
