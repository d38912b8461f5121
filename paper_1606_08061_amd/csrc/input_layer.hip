// The sparse input layer of section 2.2: with a K-sparse input x (indices u, values
// v), the forward pass W1^T x visits only the K rows of W1 that x names, and the
// update W1 <- W1 - eta x grad_a^T changes only those rows.  Minibatch form: A = X W1
// (one row per example) and W1 <- W1 - eta X^T grad_A, the update through the same
// per-row owner scatter as the V update of the factored step (one writer per row,
// a row named by several slots of the minibatch summed in slot order).
#include <algorithm>

#include "lst_internal.h"
#include "scatter.h"

namespace lst {
namespace {

constexpr int kInputThreads = 256;

// One workgroup per example: the example's slots in LDS (an index outside [-1, D_in)
// sets bit 0 of *status and its slot is skipped), then A_j = sum_k v_k W1[u_k] in
// slot order, columns spread over the threads.
__global__ __launch_bounds__(kInputThreads) void input_forward_kernel(
    const float *__restrict__ W1, int64_t ldw, int64_t D_in, int d, const int *__restrict__ idx,
    const float *__restrict__ val, int K, float *__restrict__ A, int *__restrict__ status) {
  __shared__ int su[LST_MAX_K];
  __shared__ float sv[LST_MAX_K];
  const int j = blockIdx.x, t = threadIdx.x;
  if (t < K) {
    int u = idx[(int64_t)j * K + t];
    if (u < -1 || u >= D_in) {
      atomicOr(status, FLAG_INDEX);
      u = -1;
    }
    su[t] = u;
    sv[t] = val[(int64_t)j * K + t];
  }
  __syncthreads();
  for (int c = t; c < d; c += kInputThreads) {
    float a = 0.f;
    for (int k = 0; k < K; ++k)
      if (su[k] >= 0) a = fmaf(sv[k], W1[(int64_t)su[k] * ldw + c], a);
    A[(int64_t)j * d + c] = a;
  }
}

// One workgroup: bit 0 of *status if any of the n indices lies outside [-1, D_in).
__global__ __launch_bounds__(256) void input_check_kernel(const int *__restrict__ idx, int n,
                                                          int64_t D_in, int *__restrict__ status) {
  int bad = 0;
  for (int q = threadIdx.x; q < n; q += 256) bad |= (idx[q] < -1 || idx[q] >= D_in) ? 1 : 0;
  if (__syncthreads_or(bad) && threadIdx.x == 0) atomicOr(status, FLAG_INDEX);
}

// W1[u] -= eta sum over the slots naming u of v_slot grad_A[example(slot)]; nothing is
// written while *status is non-zero (an invalid index in this call or an earlier one).
__global__ __launch_bounds__(kInputThreads) void input_update_kernel(
    int n, int K, int d, float lr, const int *__restrict__ idx, const float *__restrict__ val,
    const float *__restrict__ gA, float *__restrict__ W1, int64_t ldw,
    const int *__restrict__ status) {
  extern __shared__ int sh[];
  if (*status != 0) return;
  scatter_slot<kInputThreads>(blockIdx.x, n, K, d, lr, idx, val, gA, W1, ldw, sh);
}

}  // namespace

hipError_t launch_input_forward(hipStream_t s, const float *W1, int64_t ldw, int64_t D_in, int d,
                                const int *idx, const float *val, int m, int K, float *A,
                                int *status) {
  if (m == 0) return hipSuccess;
  LST_LAUNCH(input_forward_kernel, dim3(m), dim3(kInputThreads), 0, s, W1, ldw, D_in, d, idx, val,
             K, A, status);
  return hipGetLastError();
}

hipError_t launch_input_update(hipStream_t s, float *W1, int64_t ldw, int64_t D_in, int d,
                               const int *idx, const float *val, int m, int K, const float *gA,
                               float lr, int *status) {
  const int n = m * K;
  if (n == 0) return hipSuccess;
  LST_LAUNCH(input_check_kernel, dim3(1), dim3(256), 0, s, idx, n, D_in, status);
  LST_LAUNCH(input_update_kernel, dim3(n), dim3(kInputThreads), 2 * n * sizeof(int), s, n, K, d,
             lr, idx, val, gA, W1, ldw, status);
  return hipGetLastError();
}

}  // namespace lst
