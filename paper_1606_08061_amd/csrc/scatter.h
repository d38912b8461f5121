// V update of the factored step (eq. updateV): the per-row owner scatter, as a
// device function of one workgroup of T threads (device code shared by the HIP
// sources of liblst; not part of the C ABI).
#pragma once

#include "lst_internal.h"

namespace lst {

namespace {

// One workgroup of T threads per target slot s (slot = j*K + k of the m x K index
// matrix); sh: 2n ints of dynamic LDS.
// The lowest slot of each V row does the row's update: it lists, in ascending
// slot order, every slot with the same row and applies
//   V_r -= eta sum_{slots s' of row r} dl/dA_s' P_{j(s')},
// so each distinct row has exactly one writer and a fixed summation order.
template <int T>
__device__ __forceinline__ void scatter_slot(int s, int n, int K, int d, float lr,
                                             const int *__restrict__ idx,
                                             const float *__restrict__ dA,
                                             const float *__restrict__ P, float *__restrict__ V,
                                             int64_t ldv, int *sh) {
  int *sidx = sh;        // n target rows
  int *slist = sh + n;   // slots of this row, ascending
  __shared__ int swcnt[T / 64];
  const int r = idx[s];
  if (r < 0) return;
  int dup = 0;
  for (int q = threadIdx.x; q < n; q += T) {
    const int v = idx[q];
    sidx[q] = v;
    dup |= (q < s && v == r);
  }
  if (__syncthreads_or(dup)) return;  // an earlier slot owns this row

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int total = 0;
  for (int base = s; base < n; base += T) {
    const int q = base + threadIdx.x;
    const bool match = q < n && sidx[q] == r;
    const unsigned long long mask = __ballot(match);
    if (lane == 0) swcnt[w] = __popcll(mask);
    __syncthreads();
    int before = total;
    for (int x = 0; x < w; ++x) before += swcnt[x];
    if (match) slist[before + __popcll(mask & ((1ull << lane) - 1ull))] = q;
    for (int x = 0; x < T / 64; ++x) total += swcnt[x];
    __syncthreads();
  }

  // The row's sum over its `total` slots: columns in groups of four where the
  // layout allows; the slots split into np interleaved parts (np a power of two,
  // as many as the threads left over by the columns allow), each part summed in
  // slot order, the parts then added in a fixed order through LDS.  Rows with many slots (frequent targets) are so spread
  // over the workgroup instead of running one slot after another.
  float *vr = V + (int64_t)r * ldv;
  const bool v4 = (d & 3) == 0 && (ldv & 3) == 0 && (reinterpret_cast<uintptr_t>(V) & 15) == 0 &&
                  (reinterpret_cast<uintptr_t>(P) & 15) == 0;
  const int width = v4 ? 4 : 1;
  const int ng = (d + width - 1) / width;  // column groups
  int np = 1;
  while (np < 16 && 2 * np * ng <= T) np *= 2;
  __shared__ float4 spart[T];
  for (int g0 = 0; g0 < ng; g0 += T / np) {
    const int gl = threadIdx.x % (T / np), part = threadIdx.x / (T / np);
    const int g = g0 + gl;
    const bool active = g < ng;
    // kIlp slots' rows loaded before any is accumulated (the loads all in flight), then
    // added in slot order
    constexpr int kIlp = 8;
    float4 sum = make_float4(0.f, 0.f, 0.f, 0.f);
    auto row = [&](int q) {
      const float *pr = P + (int64_t)(q / K) * d + g * width;
      return v4 ? *reinterpret_cast<const float4 *>(pr) : make_float4(pr[0], 0.f, 0.f, 0.f);
    };
    auto add = [&](float w, const float4 &x) {
      sum.x += w * x.x;
      sum.y += w * x.y;
      sum.z += w * x.z;
      sum.w += w * x.w;
    };
    if (active) {
      int t = part;
      for (; t + (kIlp - 1) * np < total; t += kIlp * np) {
        float w[kIlp];
        float4 x[kIlp];
#pragma unroll
        for (int u = 0; u < kIlp; ++u) {
          const int q = slist[t + u * np];
          w[u] = dA[q];
          x[u] = row(q);
        }
#pragma unroll
        for (int u = 0; u < kIlp; ++u) add(w[u], x[u]);
      }
      for (; t < total; t += np) {  // fewer than kIlp left
        const int q = slist[t];
        add(dA[q], row(q));
      }
    }
    spart[threadIdx.x] = sum;
    __syncthreads();
    if (part == 0 && active) {
      float4 tot = spart[gl];
      for (int p2 = 1; p2 < np; ++p2) {
        const float4 x = spart[gl + p2 * (T / np)];
        tot.x += x.x;
        tot.y += x.y;
        tot.z += x.z;
        tot.w += x.w;
      }
      if (v4) {
        float4 *dst = reinterpret_cast<float4 *>(vr) + g;
        float4 v = *dst;
        v.x -= lr * tot.x;
        v.y -= lr * tot.y;
        v.z -= lr * tot.z;
        v.w -= lr * tot.w;
        *dst = v;
      } else {
        vr[g] -= lr * tot.x;
      }
    }
    __syncthreads();
  }
}

}  // namespace

}  // namespace lst
