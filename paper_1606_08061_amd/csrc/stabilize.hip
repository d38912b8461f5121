// Numerical stabilisation of section 5: the pristine restore V <- V U (5.1),
// Algorithm 5's fix-singular-value, the power iteration for the extreme singular
// values of U and the recomputation of U^{-T} (5.3).  None of these runs inside a
// training step; each is enqueued on the context's stream between steps.
#include <algorithm>

#include "lst_internal.h"

namespace lst {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));

// ---------------------------------------------------------------------------
// V <- V U in place (section 5.1), O(D d^2) on the matrix cores.  A workgroup owns
// 32 rows of V: it stages them in LDS (k-major, row stride 33 so that both the
// transposing stores and the MFMA operand reads are free of bank conflicts)
// before any of its waves writes, and no other workgroup reads them, so the
// in-place update is safe.  Wave w of four computes columns
// [32 NB w, 32 NB (w + 1)) as NB 32 x 32 blocks of v_mfma_f32_32x32x2f32; U (the
// B operand, d x d, L2-resident) streams from global memory, KS k-pairs per
// group, the next group's loads issued before the current group's MFMAs.
// ---------------------------------------------------------------------------
constexpr int kRestoreRows = 32, kRestoreLd = 33, kRestoreMaxd = 1024;

template <int NB, int KS>
__global__ __launch_bounds__(256) void restore_kernel(float *__restrict__ V, int64_t ldv,
                                                      int64_t D, const float *__restrict__ U,
                                                      int ldd, int d) {
  extern __shared__ float As[];  // [dk][kRestoreLd]
  constexpr int KG = 2 * KS;     // k per group
  const int dk = (d + KG - 1) / KG * KG;
  const int64_t r0 = (int64_t)blockIdx.x * kRestoreRows;
  const int t = threadIdx.x;
  constexpr int kPer = kRestoreMaxd / 256;
#pragma unroll
  for (int i0 = 0; i0 < kRestoreRows; i0 += 8) {
    float v[8][kPer];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int p = 0; p < kPer; ++p) {
        const int k = t + 256 * p;
        const int64_t r = r0 + i0 + i;
        v[i][p] = (r < D && k < d) ? V[r * ldv + k] : 0.f;
      }
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int p = 0; p < kPer; ++p) {
        const int k = t + 256 * p;
        if (k < dk) As[k * kRestoreLd + i0 + i] = v[i][p];
      }
  }
  __syncthreads();

  const int lane = t & 63, wave = t >> 6, li = lane & 31, lh = lane >> 5;
  const int cbase = wave * NB * 32 + li;
  floatx16 acc[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[b][r] = 0.f;
  auto load = [&](int g, float(&bv)[KS][NB]) {
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int k = g * KG + 2 * s + lh;
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const int c = cbase + 32 * b;
        bv[s][b] = (k < d && c < d) ? U[(int64_t)k * ldd + c] : 0.f;
      }
    }
  };
  auto compute = [&](int g, const float(&bv)[KS][NB]) {
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const float a = As[(g * KG + 2 * s + lh) * kRestoreLd + li];
#pragma unroll
      for (int b = 0; b < NB; ++b)
        acc[b] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, bv[s][b], acc[b], 0, 0, 0);
    }
  };
  const int ng = dk / KG;
  float b0[KS][NB], b1[KS][NB];
  load(0, b0);
  int g = 0;
  for (; g + 1 < ng; g += 2) {
    load(g + 1, b1);
    compute(g, b0);
    if (g + 2 < ng) load(g + 2, b0);
    compute(g + 1, b1);
  }
  if (g < ng) compute(g, b0);

  // acc[b][r] is row 8 (r / 4) + 4 lh + r % 4 of the block, column li
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const int c = cbase + 32 * b;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int64_t row = r0 + 8 * (r >> 2) + 4 * lh + (r & 3);
      if (c < d && row < D) V[row * ldv + c] = acc[b][r];
    }
  }
}

// ---------------------------------------------------------------------------
// y = A^T x for d x d row-major matrices, spread over the chip: workgroup
// (column block cb of 64, row slice r of kMvSlices, matrix z) sums its slice's rows
// (wave w of four takes the rows = w mod 4, lane j = 64 cb + lane) and writes the
// partial sums part[z][r][j]; a second kernel adds the slices in a fixed order, so
// the result does not depend on scheduling.  Two products (z = 0, 1) share a launch.
// ---------------------------------------------------------------------------
constexpr int kMvSlices = 16;

__global__ __launch_bounds__(256) void tmatvec_part_kernel(const float *__restrict__ A0,
                                                           const float *__restrict__ A1, int lda,
                                                           int d, const float *__restrict__ x0,
                                                           const float *__restrict__ x1,
                                                           float *__restrict__ part) {
  __shared__ float red[4][64];
  const float *A = blockIdx.z ? A1 : A0;
  const float *x = blockIdx.z ? x1 : x0;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int j = blockIdx.x * 64 + lane;
  const int rows = (d + kMvSlices - 1) / kMvSlices;
  const int i0 = blockIdx.y * rows, i1 = min(d, i0 + rows);
  float s0 = 0.f, s1 = 0.f;
  if (j < d) {
    int i = i0 + wave;
    for (; i + 4 < i1; i += 8) {
      s0 = fmaf(A[(int64_t)i * lda + j], x[i], s0);
      s1 = fmaf(A[(int64_t)(i + 4) * lda + j], x[i + 4], s1);
    }
    if (i < i1) s0 = fmaf(A[(int64_t)i * lda + j], x[i], s0);
  }
  red[wave][lane] = s0 + s1;
  __syncthreads();
  if (wave == 0 && j < d)
    part[((int64_t)blockIdx.z * kMvSlices + blockIdx.y) * d + j] =
        (red[0][lane] + red[1][lane]) + (red[2][lane] + red[3][lane]);
}

// y_z[j] = sum over the slices of part[z][r][j], in slice order.
__global__ __launch_bounds__(256) void tmatvec_sum_kernel(const float *__restrict__ part, int d,
                                                          float *__restrict__ y0,
                                                          float *__restrict__ y1) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= d) return;
  const float *p = part + (int64_t)blockIdx.y * kMvSlices * d;
  float s = 0.f;
  for (int r = 0; r < kMvSlices; ++r) s += p[(int64_t)r * d + j];
  (blockIdx.y ? y1 : y0)[j] = s;
}

// Sum over the workgroup (1024 threads) of v; every thread gets the result.
__device__ float block_sum_1024(float v, float *red) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  float s = 0.f;
  for (int w = 0; w < 16; ++w) s += red[w];
  return s;
}

// ---------------------------------------------------------------------------
// Algorithm 5, fix-singular-value.  alpha = (target - sigma) / sigma and
// beta = -alpha / (1 + alpha) are formed on the device from *sigma.
//   state: U[i, j] += alpha u_i a_j, U^{-T}[i, j] += beta u_i b_j with a = U^T u and
//          b = U^{-1} u = (U^{-T})^T u taken before the update.
//   V:     V_r += beta (V_r . u) u^T, one pass over V (a wavefront per row, the row
//          held in registers between its dot product and its update).
// ---------------------------------------------------------------------------
// false (the update is skipped) unless sigma is positive and finite
__device__ __forceinline__ bool fix_coefs(const float *sigma, float target, float &alpha,
                                          float &beta) {
  const float s = *sigma;
  alpha = (target - s) / s;
  beta = -alpha / (1.f + alpha);
  return s > 0.f && s < INFINITY && isfinite(beta);
}

__global__ __launch_bounds__(256) void fix_state_kernel(float *__restrict__ U,
                                                        float *__restrict__ UinvT, int ldd, int d,
                                                        const float *__restrict__ u,
                                                        const float *__restrict__ a,
                                                        const float *__restrict__ b,
                                                        const float *__restrict__ sigma,
                                                        float target, int *__restrict__ flag) {
  float alpha, beta;
  if (!fix_coefs(sigma, target, alpha, beta)) {
    if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(flag, FLAG_NONFINITE);
    return;
  }
  const int64_t n = (int64_t)d * d;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < n; e += (int64_t)gridDim.x * 256) {
    const int i = (int)(e / d), j = (int)(e - (int64_t)i * d);
    const int64_t o = (int64_t)i * ldd + j;
    U[o] = fmaf(alpha * u[i], a[j], U[o]);
    UinvT[o] = fmaf(beta * u[i], b[j], UinvT[o]);
  }
}

template <int NPL>  // row elements per lane: d <= 64 NPL
__global__ __launch_bounds__(256) void fix_v_kernel(float *__restrict__ V, int64_t ldv, int64_t D,
                                                    int d, const float *__restrict__ u,
                                                    const float *__restrict__ sigma,
                                                    float target) {
  float alpha, beta;
  if (!fix_coefs(sigma, target, alpha, beta)) return;
  const int lane = threadIdx.x & 63;
  float uu[NPL];
#pragma unroll
  for (int p = 0; p < NPL; ++p) {
    const int k = lane + 64 * p;
    uu[p] = k < d ? u[k] : 0.f;
  }
  // two rows per wave per iteration (r and r + waves), so that 2 NPL loads are in flight
  const int64_t waves = (int64_t)gridDim.x * 4;
  for (int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); r < D; r += 2 * waves) {
    const bool two = r + waves < D;
    float *row0 = V + r * ldv, *row1 = V + (two ? r + waves : r) * ldv;
    float v0[NPL], v1[NPL];
#pragma unroll
    for (int p = 0; p < NPL; ++p) {
      const int k = lane + 64 * p;
      v0[p] = k < d ? row0[k] : 0.f;
      v1[p] = (two && k < d) ? row1[k] : 0.f;
    }
    float s0 = 0.f, s1 = 0.f;
#pragma unroll
    for (int p = 0; p < NPL; ++p) {
      s0 = fmaf(v0[p], uu[p], s0);
      s1 = fmaf(v1[p], uu[p], s1);
    }
    for (int o = 32; o > 0; o >>= 1) {
      s0 += __shfl_xor(s0, o);
      s1 += __shfl_xor(s1, o);
    }
    const float b0 = beta * s0, b1 = beta * s1;
#pragma unroll
    for (int p = 0; p < NPL; ++p) {
      const int k = lane + 64 * p;
      if (k < d) {
        row0[k] = fmaf(b0, uu[p], v0[p]);
        if (two) row1[k] = fmaf(b1, uu[p], v1[p]);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Power iteration (section 5.3) as repeated squaring: 2^s rounds of u <- G u / ||G u||
// with G = A A^T give u = G^(2^s) u0 / ||G^(2^s) u0||.  G^(2^s) comes from s
// matrix-core squarings; before each one the matrix is divided by its trace (the
// sum of its eigenvalues, all >= 0), which keeps every entry within [-1, 1] without
// changing the direction of the result.  The division reads the diagonal of one
// buffer and writes the scaled copy to another, so no workgroup sees a
// half-scaled diagonal.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void trace_scale_kernel(const float *__restrict__ S, int d,
                                                          float *__restrict__ out) {
  __shared__ float red[4];
  float tr = 0.f;
  for (int i = threadIdx.x; i < d; i += 256) tr += S[(int64_t)i * d + i];
  for (int o = 32; o > 0; o >>= 1) tr += __shfl_xor(tr, o);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = tr;
  __syncthreads();
  const float inv = 1.f / ((red[0] + red[1]) + (red[2] + red[3]));
  const int64_t n = (int64_t)d * d;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < n; e += (int64_t)gridDim.x * 256)
    out[e] = S[e] * inv;
}

// One workgroup of 1024 adding the slices of an A^T x product (tmatvec_part_kernel),
// then: mode 0 -- u = y / ||y|| into u_out; mode 1 -- *sigma_out = ||y|| (which = 0)
// or 1 / ||y|| (which = 1).
__global__ __launch_bounds__(1024) void power_norm_kernel(const float *__restrict__ part, int d,
                                                          int mode, int which,
                                                          float *__restrict__ u_out,
                                                          float *__restrict__ sigma_out) {
  extern __shared__ float sy[];  // d floats
  __shared__ float red[16];
  float sq = 0.f;
  for (int j = threadIdx.x; j < d; j += 1024) {
    float s = 0.f;
    for (int r = 0; r < kMvSlices; ++r) s += part[(int64_t)r * d + j];
    sy[j] = s;
    sq = fmaf(s, s, sq);
  }
  const float n = sqrtf(block_sum_1024(sq, red));
  if (mode == 0) {
    const float inv = 1.f / n;
    for (int j = threadIdx.x; j < d; j += 1024) u_out[j] = sy[j] * inv;
  } else if (threadIdx.x == 0) {
    *sigma_out = which ? 1.f / n : n;
  }
}

// ---------------------------------------------------------------------------
// Recomputing U^{-T} (section 5.3) by Newton-Schulz rounds Y <- Y + E Y with
// E = I - Y U^T, which converge quadratically to U^{-T} once ||E|| < 1.  From
// scratch the start is Y0 = U / (||U||_1 ||U||_inf) (the transpose of the classical
// X0 = U^T / (...)), for which the iteration converges for any invertible U.  E is
// accumulated in fp64: its entries are sums of d terms of size |Y| |U| that cancel
// to the residual, and an fp32 sum would leave noise of order cond(U) eps32 in E,
// which the correction E Y then spreads over all of Y (a relative error of 3e-2 at
// cond(U) = 4e6).  With E exact to fp32 rounding the fp32 correction converges to
// the fp32 rounding of U^{-T} while cond(U) eps32 < 1 (mixed-precision refinement).
// ---------------------------------------------------------------------------
// 32 x 32 entries of E per workgroup of four wavefronts, each a 16 x 16 block on the
// fp64 matrix cores (v_mfma_f64_16x16x4_f64: lane l holds A[l % 16][l / 16] and
// B[l / 16][l % 16] of a k-step of 4, and register r of the result is row
// l / 16 + 4 r, column l % 16 of the block -- rows interleaved, unlike the fp32
// 16 x 16 x 4 form; checked on the device); k in chunks of 32 staged in LDS as
// doubles (rows of Y and rows of U, both k-contiguous).
typedef double doublex4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void residual64_kernel(const float *__restrict__ Y, int ldy,
                                                         const float *__restrict__ U, int ldu,
                                                         int d, float *__restrict__ E) {
  __shared__ double Ys[32][33], Us[32][33];
  const int i0 = blockIdx.y * 32, j0 = blockIdx.x * 32;
  const int ti = threadIdx.x >> 5, tj = threadIdx.x & 31;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int bi = 16 * (wave >> 1), bj = 16 * (wave & 1);
  const int li = lane & 15, lk = lane >> 4;
  doublex4 acc = {0.0, 0.0, 0.0, 0.0};
  for (int k0 = 0; k0 < d; k0 += 32) {
    const int k = k0 + tj;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int r = ti + 8 * q;
      Ys[r][tj] = (i0 + r < d && k < d) ? (double)Y[(int64_t)(i0 + r) * ldy + k] : 0.0;
      Us[r][tj] = (j0 + r < d && k < d) ? (double)U[(int64_t)(j0 + r) * ldu + k] : 0.0;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 32; kk += 4)
      acc = __builtin_amdgcn_mfma_f64_16x16x4f64(Ys[bi + li][kk + lk], Us[bj + li][kk + lk], acc,
                                                 0, 0, 0);
    __syncthreads();
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int i = i0 + bi + lk + 4 * r, j = j0 + bj + li;
    if (i < d && j < d) E[(int64_t)i * d + j] = (float)((i == j ? 1.0 : 0.0) - acc[r]);
  }
}

// One workgroup of 1024: c = 1 / (max column abs sum * max row abs sum).
__global__ __launch_bounds__(1024) void ns_norms_kernel(const float *__restrict__ U, int ldd, int d,
                                                        float *__restrict__ c) {
  __shared__ float red[16];
  float cmax = 0.f, rmax = 0.f;
  for (int j = threadIdx.x; j < d; j += 1024) {
    float cs = 0.f, rs = 0.f;
    for (int i = 0; i < d; ++i) {
      cs += fabsf(U[(int64_t)i * ldd + j]);
      rs += fabsf(U[(int64_t)j * ldd + i]);
    }
    cmax = fmaxf(cmax, cs);
    rmax = fmaxf(rmax, rs);
  }
  for (int o = 32; o > 0; o >>= 1) {
    cmax = fmaxf(cmax, __shfl_xor(cmax, o));
    rmax = fmaxf(rmax, __shfl_xor(rmax, o));
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) red[wave] = cmax;
  __syncthreads();
  float cm = 0.f;
  for (int w = 0; w < 16; ++w) cm = fmaxf(cm, red[w]);
  __syncthreads();
  if (lane == 0) red[wave] = rmax;
  __syncthreads();
  float rm = 0.f;
  for (int w = 0; w < 16; ++w) rm = fmaxf(rm, red[w]);
  if (threadIdx.x == 0) *c = 1.f / (cm * rm);
}

__global__ __launch_bounds__(256) void scaled_copy_kernel(const float *__restrict__ A, int lda,
                                                          int d, const float *__restrict__ c,
                                                          float *__restrict__ out, int ldo) {
  const float s = *c;
  const int64_t n = (int64_t)d * d;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < n; e += (int64_t)gridDim.x * 256) {
    const int i = (int)(e / d), j = (int)(e - (int64_t)i * d);
    out[(int64_t)i * ldo + j] = s * A[(int64_t)i * lda + j];
  }
}

// *amax = max_ij |E_ij| (non-negative floats compare as their bit patterns, NaN counting
// as infinite; *amax starts at 0).  One atomic per workgroup.
constexpr int kAbsmaxBlocks = 64;
__global__ __launch_bounds__(256) void absmax_kernel(const float *__restrict__ E, int d,
                                                     float *__restrict__ amax) {
  __shared__ float red[4];
  float m = 0.f;
  const int64_t n = (int64_t)d * d;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < n; e += (int64_t)gridDim.x * 256) {
    const float a = fabsf(E[e]);
    m = fmaxf(m, a == a ? a : INFINITY);
  }
  for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0)
    atomicMax(reinterpret_cast<int *>(amax),
              __float_as_int(fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]))));
}

int elementwise_blocks(int d) {
  return (int)std::min<int64_t>(((int64_t)d * d + 255) / 256, 4096);
}

}  // namespace

hipError_t launch_restore(hipStream_t s, float *V, int64_t ldv, int64_t D, const float *U, int ldd,
                          int d) {
  if (d > kRestoreMaxd) return hipErrorInvalidValue;
  const dim3 grid((unsigned)((D + kRestoreRows - 1) / kRestoreRows));
  const int nb = d <= 128 ? 1 : d <= 256 ? 2 : d <= 512 ? 4 : 8;
  const int ks = nb == 8 ? 4 : 8;
  const size_t lds = (size_t)((d + 2 * ks - 1) / (2 * ks) * (2 * ks)) * kRestoreLd * sizeof(float);
  switch (nb) {
    case 1: LST_LAUNCH((restore_kernel<1, 8>), grid, dim3(256), lds, s, V, ldv, D, U, ldd, d); break;
    case 2: LST_LAUNCH((restore_kernel<2, 8>), grid, dim3(256), lds, s, V, ldv, D, U, ldd, d); break;
    case 4: LST_LAUNCH((restore_kernel<4, 8>), grid, dim3(256), lds, s, V, ldv, D, U, ldd, d); break;
    default: LST_LAUNCH((restore_kernel<8, 4>), grid, dim3(256), lds, s, V, ldv, D, U, ldd, d);
  }
  return hipGetLastError();
}

hipError_t launch_tmatvec2(hipStream_t s, const float *A0, const float *A1, int lda, int d,
                           const float *x0, const float *x1, float *y0, float *y1, float *part) {
  const int nz = A1 ? 2 : 1;
  LST_LAUNCH(tmatvec_part_kernel, dim3((d + 63) / 64, kMvSlices, nz), dim3(256), 0, s, A0, A1, lda,
             d, x0, x1, part);
  LST_LAUNCH(tmatvec_sum_kernel, dim3((d + 255) / 256, nz), dim3(256), 0, s, part, d, y0, y1);
  return hipGetLastError();
}

hipError_t launch_fix_state(hipStream_t s, float *U, float *UinvT, int ldd, int d, const float *u,
                            const float *a, const float *b, const float *sigma, float target,
                            int *flag) {
  LST_LAUNCH(fix_state_kernel, dim3(elementwise_blocks(d)), dim3(256), 0, s, U, UinvT, ldd, d, u, a,
             b, sigma, target, flag);
  return hipGetLastError();
}

hipError_t launch_fix_v(hipStream_t s, float *V, int64_t ldv, int64_t D, int d, const float *u,
                        const float *sigma, float target) {
  const dim3 grid((unsigned)std::min<int64_t>((D + 3) / 4, 8192));
  if (d <= 256)
    LST_LAUNCH(fix_v_kernel<4>, grid, dim3(256), 0, s, V, ldv, D, d, u, sigma, target);
  else if (d <= 512)
    LST_LAUNCH(fix_v_kernel<8>, grid, dim3(256), 0, s, V, ldv, D, d, u, sigma, target);
  else if (d <= 1024)
    LST_LAUNCH(fix_v_kernel<16>, grid, dim3(256), 0, s, V, ldv, D, d, u, sigma, target);
  else if (d <= 2048)
    LST_LAUNCH(fix_v_kernel<32>, grid, dim3(256), 0, s, V, ldv, D, d, u, sigma, target);
  else
    LST_LAUNCH(fix_v_kernel<64>, grid, dim3(256), 0, s, V, ldv, D, d, u, sigma, target);
  return hipGetLastError();
}

hipError_t launch_trace_scale(hipStream_t s, const float *S, int d, float *out) {
  LST_LAUNCH(trace_scale_kernel, dim3(elementwise_blocks(d)), dim3(256), 0, s, S, d, out);
  return hipGetLastError();
}

hipError_t launch_power_finish(hipStream_t s, const float *S, int d, const float *u0,
                               const float *A, int lda, int which, float *u_out,
                               float *sigma_out, float *part) {
  const dim3 grid((d + 63) / 64, kMvSlices, 1);
  const size_t lds = (size_t)d * sizeof(float);
  // u = S u0 / ||S u0|| (S symmetric: S u0 = S^T u0)
  LST_LAUNCH(tmatvec_part_kernel, grid, dim3(256), 0, s, S, S, d, d, u0, u0, part);
  LST_LAUNCH(power_norm_kernel, dim3(1), dim3(1024), lds, s, part, d, 0, which, u_out, sigma_out);
  // sigma from ||A^T u||
  LST_LAUNCH(tmatvec_part_kernel, grid, dim3(256), 0, s, A, A, lda, d, u_out, u_out, part);
  LST_LAUNCH(power_norm_kernel, dim3(1), dim3(1024), lds, s, part, d, 1, which, u_out, sigma_out);
  return hipGetLastError();
}

hipError_t launch_ns_start(hipStream_t s, const float *U, int ldd, int d, float *c, float *Y,
                           int ldy) {
  LST_LAUNCH(ns_norms_kernel, dim3(1), dim3(1024), 0, s, U, ldd, d, c);
  LST_LAUNCH(scaled_copy_kernel, dim3(elementwise_blocks(d)), dim3(256), 0, s, U, ldd, d, c, Y,
             ldy);
  return hipGetLastError();
}

hipError_t launch_residual64(hipStream_t s, const float *Y, int ldy, const float *U, int ldu, int d,
                             float *E) {
  const dim3 grid((d + 31) / 32, (d + 31) / 32);
  LST_LAUNCH(residual64_kernel, grid, dim3(256), 0, s, Y, ldy, U, ldu, d, E);
  return hipGetLastError();
}

hipError_t launch_absmax(hipStream_t s, const float *E, int d, float *amax) {
  LST_LAUNCH(absmax_kernel, dim3(std::min(elementwise_blocks(d), kAbsmaxBlocks)), dim3(256), 0, s, E,
             d, amax);
  return hipGetLastError();
}

}  // namespace lst
