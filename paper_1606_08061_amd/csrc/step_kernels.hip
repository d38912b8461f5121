// Non-GEMM kernels outside the factored step: identity and fill, w_bar and the omega
// part of Q at initialisation, and the naive comparison path's column norms (and
// sums) of O, loss epilogue over the explicit output and
// grad_O = 2 O diag(dl/dq) + 1_D (dl/ds)^T + Yring (eq. gen-grad-O).
#include <algorithm>

#include "lst_internal.h"

namespace lst {

namespace {

// Loss epilogue of one example (section 4: l(q, s, K, a, t)).  r[k] < 0 marks an
// empty slot.  Writes the example's loss, dl/dq, dl/ds and dl/da_k.
__device__ __forceinline__ void loss_epilogue(int loss, float q, float s, int K, const int *r,
                                              const float *t, const float *a, float Dn,
                                              float eps, float &l, float &gq, float &gs,
                                              float *g) {
  l = 0.f;
  gq = 0.f;
  gs = 0.f;
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
  } else if (loss == LST_LOSS_TAYLOR_SOFTMAX) {
    // l = sum_k t_k [log(D + s + q/2) - log(f(a_k))], f(x) = 1 + x + x^2/2
    const float z = Dn + s + 0.5f * q;
    const float lz = logf(z);
    float ts = 0.f;
    for (int k = 0; k < K; ++k) {
      g[k] = 0.f;
      if (r[k] < 0) continue;
      const float f = 1.f + a[k] + 0.5f * a[k] * a[k];
      l += t[k] * (lz - logf(f));
      ts += t[k];
      g[k] = -t[k] * (1.f + a[k]) / f;
    }
    gq = ts / (2.f * z);
    gs = ts / z;
  } else {
    // l = sum_k t_k [log(q + D eps) - log(a_k^2 + eps)]
    const float z = q + Dn * eps;
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
                                                      float *__restrict__ partial,
                                                      float *__restrict__ psum) {
  const int64_t rows = (D + gridDim.x - 1) / gridDim.x;
  const int64_t r0 = (int64_t)blockIdx.x * rows;
  const int64_t r1 = min(D, r0 + rows);
  for (int j = threadIdx.x; j < m; j += blockDim.x) {
    float s = 0.f, u = 0.f;
    for (int64_t i = r0; i < r1; ++i) {
      const float o = O[i * m + j];
      s += o * o;
      u += o;
    }
    partial[(int64_t)blockIdx.x * m + j] = s;
    if (psum) psum[(int64_t)blockIdx.x * m + j] = u;
  }
}

// Column sums of V over a block of rows, partial[b][c] (block b of gridDim.x).
__global__ __launch_bounds__(256) void vcolsum_kernel(const float *__restrict__ V, int64_t ldv,
                                                      int64_t D, int d, float *__restrict__ part) {
  const int64_t rows = (D + gridDim.x - 1) / gridDim.x;
  const int64_t r0 = (int64_t)blockIdx.x * rows;
  const int64_t r1 = min(D, r0 + rows);
  for (int c = threadIdx.x; c < d; c += blockDim.x) {
    float u = 0.f;
    for (int64_t i = r0; i < r1; ++i) u += V[i * ldv + c];
    part[(int64_t)blockIdx.x * d + c] = u;
  }
}

// out[c] = sum_r U[r][c] v[r] + D omega[c], v = the reduced column sums (one workgroup).
__global__ __launch_bounds__(256) void wbar_finish_kernel(const float *__restrict__ part, int nblk,
                                                          int d, const float *__restrict__ U,
                                                          int ldd, int64_t D,
                                                          const float *__restrict__ omega,
                                                          float *__restrict__ out) {
  extern __shared__ float v[];
  for (int c = threadIdx.x; c < d; c += blockDim.x) {
    float u = 0.f;
    for (int b = 0; b < nblk; ++b) u += part[(int64_t)b * d + c];
    v[c] = u;
  }
  __syncthreads();
  for (int c = threadIdx.x; c < d; c += blockDim.x) {
    float w;
    if (U) {
      w = 0.f;
      for (int r = 0; r < d; ++r) w += U[(int64_t)r * ldd + c] * v[r];
    } else {
      w = v[c];
    }
    out[c] = w + (float)D * omega[c];
  }
}

__global__ __launch_bounds__(256) void q_omega_kernel(float *__restrict__ Q, int ldd, int d,
                                                      int64_t D, const float *__restrict__ wbar,
                                                      const float *__restrict__ omega) {
  const int64_t total = (int64_t)d * d;
  const float Dn = (float)D;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int i = (int)(e / d), j = (int)(e - (int64_t)i * d);
    const float ui = wbar[i] - Dn * omega[i], uj = wbar[j] - Dn * omega[j];
    Q[(int64_t)i * ldd + j] += ui * omega[j] + omega[i] * uj + Dn * omega[i] * omega[j];
  }
}

// One workgroup per example j: q_j from the partial column sums (fixed order),
// then the loss epilogue on the K target entries of column j of O.
__global__ __launch_bounds__(256) void naive_epilogue_kernel(int m, int K, int64_t D, int nparts,
                                                             const float *__restrict__ partial,
                                                             const float *__restrict__ psum,
                                                             const float *__restrict__ O,
                                                             const int *__restrict__ idx,
                                                             const float *__restrict__ val, int loss,
                                                             float eps, float *__restrict__ dq,
                                                             float *__restrict__ ds,
                                                             float *__restrict__ dA,
                                                             float *__restrict__ lvec,
                                                             int *__restrict__ flag) {
  __shared__ float red[256], red2[256];
  __shared__ int sr[LST_MAX_K];
  __shared__ float st[LST_MAX_K], sa[LST_MAX_K];
  __shared__ int s_bad;
  const int j = blockIdx.x, t = threadIdx.x;
  if (t == 0) s_bad = 0;
  float q = 0.f, u = 0.f;
  for (int p = t; p < nparts; p += 256) {
    q += partial[(int64_t)p * m + j];
    if (psum) u += psum[(int64_t)p * m + j];
  }
  red[t] = q;
  red2[t] = u;
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
    if (t < w) {
      red[t] += red[t + w];
      red2[t] += red2[t + w];
    }
    __syncthreads();
  }
  if (t == 0) {
    float l, gq, gs, g[LST_MAX_K];
    loss_epilogue(loss, red[0], red2[0], K, sr, st, sa, (float)D, eps, l, gq, gs, g);
    dq[j] = gq;
    if (ds) ds[j] = gs;
    for (int k = 0; k < K; ++k) dA[(int64_t)j * K + k] = g[k];
    lvec[j] = l;
    if (s_bad) atomicOr(flag, FLAG_INDEX);
  }
}

// O <- 2 O diag(dq) (+ 1_D ds^T when ds is not null): n4 groups of four columns per
// row when m % 4 == 0.
__global__ __launch_bounds__(256) void scale_cols4_kernel(float4 *__restrict__ O, int64_t total4,
                                                          int n4, const float4 *__restrict__ dq,
                                                          const float4 *__restrict__ ds) {
  const int64_t f0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int step = (int)(stride % n4);
  int c = (int)(f0 % n4);
  for (int64_t f = f0; f < total4; f += stride) {
    const float4 s = dq[c], o = O[f];
    const float4 a = ds ? ds[c] : make_float4(0.f, 0.f, 0.f, 0.f);
    O[f] = make_float4(fmaf(2.f * s.x, o.x, a.x), fmaf(2.f * s.y, o.y, a.y),
                       fmaf(2.f * s.z, o.z, a.z), fmaf(2.f * s.w, o.w, a.w));
    c += step;
    if (c >= n4) c -= n4;
  }
}

__global__ __launch_bounds__(256) void scale_cols_kernel(float *__restrict__ O, int64_t total, int m,
                                                         const float *__restrict__ dq,
                                                         const float *__restrict__ ds) {
  const int64_t e0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int step = (int)(stride % m);
  int c = (int)(e0 % m);
  for (int64_t e = e0; e < total; e += stride) {
    O[e] = fmaf(2.f * dq[c], O[e], ds ? ds[c] : 0.f);
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
                          float *psum, int nblk) {
  LST_LAUNCH(colnorm_kernel, dim3(nblk), dim3(256), 0, s, O, D, m, partial, psum);
  return hipGetLastError();
}

hipError_t launch_wbar(hipStream_t s, const float *V, int64_t ldv, int64_t D, int d,
                       const float *U, int ldd, const float *omega, float *part, int nblk,
                       float *out) {
  LST_LAUNCH(vcolsum_kernel, dim3(nblk), dim3(256), 0, s, V, ldv, D, d, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  LST_LAUNCH(wbar_finish_kernel, dim3(1), dim3(256), (size_t)d * sizeof(float), s, part, nblk, d,
             U, ldd, D, omega, out);
  return hipGetLastError();
}

hipError_t launch_q_omega(hipStream_t s, float *Q, int ldd, int d, int64_t D, const float *wbar,
                          const float *omega) {
  int blocks = (int)(((int64_t)d * d + 255) / 256);
  if (blocks > 4096) blocks = 4096;
  LST_LAUNCH(q_omega_kernel, dim3(blocks), dim3(256), 0, s, Q, ldd, d, D, wbar, omega);
  return hipGetLastError();
}

hipError_t launch_naive_epilogue(hipStream_t s, int m, int K, int64_t D, int nparts,
                                 const float *partial, const float *psum, const float *O,
                                 const int *idx, const float *val, int loss, float eps, float *dq,
                                 float *ds, float *dA, float *lvec, int *flag) {
  LST_LAUNCH(naive_epilogue_kernel, dim3(m), dim3(256), 0, s, m, K, D, nparts, partial, psum, O,
             idx, val, loss, eps, dq, ds, dA, lvec, flag);
  return hipGetLastError();
}

hipError_t launch_grad_o(hipStream_t s, float *O, int64_t D, int m, int K, const float *dq,
                         const float *ds, const int *idx, const float *dA, const float *lvec,
                         float *loss_out, int *flag) {
  const int64_t total = D * m;
  const bool v4 = (m & 3) == 0 && (reinterpret_cast<uintptr_t>(O) & 15) == 0 &&
                  (reinterpret_cast<uintptr_t>(dq) & 15) == 0 &&
                  (reinterpret_cast<uintptr_t>(ds) & 15) == 0;
  const int64_t units = v4 ? total / 4 : total;
  int blocks = (int)((units + 255) / 256);
  if (blocks > 8192) blocks = 8192;
  if (v4)
    LST_LAUNCH(scale_cols4_kernel, dim3(blocks), dim3(256), 0, s, reinterpret_cast<float4 *>(O),
               units, m / 4, reinterpret_cast<const float4 *>(dq),
               reinterpret_cast<const float4 *>(ds));
  else
    LST_LAUNCH(scale_cols_kernel, dim3(blocks), dim3(256), 0, s, O, total, m, dq, ds);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  LST_LAUNCH(sparse_add_kernel, dim3(1), dim3(1024), 0, s, O, D, m, K, idx, dA, lvec, loss_out,
             flag);
  return hipGetLastError();
}

}  // namespace lst
