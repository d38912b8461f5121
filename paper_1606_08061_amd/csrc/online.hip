// The online step (one example, squared error; Algorithm 2) as one kernel
// launch.  Every product reads the pre-update Q, U, U^{-T} (Algorithm 2 steps 1, 2,
// 5, 6) before any of them is written (steps 5, 6, 8), so the whole step is two
// phases around a single grid-wide barrier:
//   A. rows r of Q, U, U^{-T} (one wavefront per row): h^ = Q h, U h and X = U^{-T} h;
//      y^ = U^T g with g = V^T y (g_i for the rows of a slice from the K target rows
//      of V), as partial sums over (64-column block, row slice) tasks.
//   B. every workgroup adds the slices of y^ and forms the same scalars in the same
//      order: ||h||^2, L = h^T h^ - 2 h^T y^ + y^T y (step 4), grad_h = 2 (h^ - y^)
//      (step 3); then the rank-one updates of its rows of U (step 5), U^{-T} (step 6,
//      Sherman-Morrison) and Q (step 8), and workgroup 0 the K rows of V with
//      U_new^{-T} h = X / (1 - 2 eta ||h||^2) (step 7: the fresh U^{-T}).
// A target index outside [-1, D), an earlier sticky error, 1 - 2 eta ||h||^2 <= 0 or
// a non-finite L leave the state untouched (every workgroup takes the same decision
// from the same values).
#include <algorithm>

#include "lst_internal.h"

namespace lst {
namespace {

constexpr int kOnlineWGs = 128;   // workgroups: 128 x 256 threads fit on the GPU at once
constexpr int kOnlineSlices = 8;  // row slices of the y^ = U^T g partial sums

__device__ __forceinline__ float wave_sum(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// The vectors handed from phase A to phase B go through agent-scope atomic stores and
// loads, which are coherent across the chip's separate L2 caches by themselves; so the
// barrier needs no agent-scope fences (a release there writes back, an acquire
// invalidates, the whole L2 of the workgroup's XCD, and with every workgroup doing
// both the step took 33 us).
__device__ __forceinline__ void put(float *p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float get(const float *p) {
  return __hip_atomic_load(const_cast<float *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Grid-wide barrier with one go/abort decision per launch.
//
// bar[0] counts arrivals (unsigned, wrapping; each launch adds exactly gridDim.x, a
// divisor of 2^32, since every workgroup arrives once even when late), so launch
// number gen = ticket / gridDim.x.  bar[1] holds the decision of the latest decided
// launch as (gen << 2) | state, state 1 = go, 2 = abort; any other content means the
// current launch is still pending.  The last arriver moves pending to go, a waiter
// whose bounded spin expires moves pending to abort (both by compare-and-swap, so the
// first decision stands), and every workgroup then acts on the one decision: either
// all of them write their part of the step, or none does.
//
// Ordering: every thread waits for its own hand-off stores to complete (s_waitcnt
// vmcnt(0): agent-scope atomic stores are complete once they have reached the
// memory side, where the other XCDs read them) before the workgroup barrier, and
// thread 0 arrives after that barrier, so the arrival is ordered after all of the
// workgroup's phase-A results.  Phase B reads them with agent-scope loads issued
// after the decision was seen.
__device__ __forceinline__ unsigned decided(unsigned w, unsigned gen) {
  return ((w >> 2) == (gen & 0x3FFFFFFFu) && (w & 3u) != 0u) ? (w & 3u) : 0u;
}

__device__ bool grid_barrier(unsigned *bar, int spin_limit, int *flag) {
  __shared__ int ok;
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned ticket =
        __hip_atomic_fetch_add(bar, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const unsigned gen = ticket / gridDim.x;
    const unsigned tag = (gen & 0x3FFFFFFFu) << 2;
    unsigned *dec = bar + 1;
    unsigned w = __hip_atomic_load(dec, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (ticket % gridDim.x == gridDim.x - 1u) {  // last arriver: pending -> go
      while (!decided(w, gen) &&
             !__hip_atomic_compare_exchange_strong(dec, &w, tag | 1u, __ATOMIC_RELAXED,
                                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
      }
    }
    for (int it = 0; !decided(w, gen); ++it) {
      if (it >= spin_limit) {  // expired: pending -> abort, unless decided meanwhile
        if (__hip_atomic_compare_exchange_strong(dec, &w, tag | 2u, __ATOMIC_RELAXED,
                                                 __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
          w = tag | 2u;
          atomicOr(flag, FLAG_SYNC);
        }
        continue;  // w now holds the current word
      }
      __builtin_amdgcn_s_sleep(1);
      w = __hip_atomic_load(dec, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    ok = decided(w, gen) == 1u ? 1 : 0;
  }
  __syncthreads();
  return ok != 0;
}

__global__ __launch_bounds__(256) void online_step_kernel(
    int64_t D, int d, int K, const float *__restrict__ h, const int *__restrict__ idx,
    const float *__restrict__ val, float lr, float *V, int64_t ldv, float *U, float *UinvT,
    float *Q, int ldd, float *__restrict__ loss_out, float *__restrict__ grad_h,
    float *__restrict__ work, unsigned *__restrict__ bar, int spin_limit, int *__restrict__ flag) {
  extern __shared__ float lds[];  // h, y^, h^, g, X (d each)
  __shared__ float red[4][64];
  __shared__ int bad_idx;
  float *sh = lds, *sy = lds + d, *shh = lds + 2 * d, *sg = lds + 3 * d, *sx = lds + 4 * d;
  float *ypart = work;                        // [kOnlineSlices][d]
  float *hhat = work + kOnlineSlices * d;     // Q h
  float *uh = hhat + d;                       // U h
  float *xv = uh + d;                         // U^{-T} h
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int gwave = blockIdx.x * 4 + wave, nwaves = gridDim.x * 4;
  const int closed = *flag;  // an earlier error: compute nothing into the state

  // g = V^T y from the K target rows (empty and invalid slots add nothing), all loads of
  // the workgroup in flight together
  for (int i = t; i < d; i += 256) {
    sh[i] = h[i];
    float g = 0.f;
    for (int k = 0; k < K; ++k) {
      const int ck = idx[k];
      if (ck >= 0 && ck < D) g = fmaf(val[k], V[(int64_t)ck * ldv + i], g);
    }
    sg[i] = g;
  }
  if (t == 0) {
    int b = 0;
    for (int k = 0; k < K; ++k) b |= (idx[k] < -1 || idx[k] >= D) ? 1 : 0;
    bad_idx = b;
  }
  __syncthreads();
  if (blockIdx.x == 0 && t == 0 && bad_idx) atomicOr(flag, FLAG_INDEX);

  // ---- phase A ----
  for (int r = gwave; r < d; r += nwaves) {
    const float *q = Q + (int64_t)r * ldd, *u = U + (int64_t)r * ldd, *x = UinvT + (int64_t)r * ldd;
    float a = 0.f, b = 0.f, c = 0.f;
#pragma unroll 8
    for (int k = lane; k < d; k += 64) {
      const float hk = sh[k];
      a = fmaf(q[k], hk, a);
      b = fmaf(u[k], hk, b);
      c = fmaf(x[k], hk, c);
    }
    a = wave_sum(a);
    b = wave_sum(b);
    c = wave_sum(c);
    if (lane == 0) {
      put(hhat + r, a);
      put(uh + r, b);
      put(xv + r, c);
    }
  }
  const int ncb = (d + 63) / 64;
  const int rows = (d + kOnlineSlices - 1) / kOnlineSlices;
  for (int task = blockIdx.x; task < ncb * kOnlineSlices; task += gridDim.x) {
    const int cb = task % ncb, sl = task / ncb;
    const int j = cb * 64 + lane;
    const int i0 = sl * rows, i1 = min(d, i0 + rows);
    float s = 0.f;
    if (j < d) {
      float s1 = 0.f;
      int i = i0 + wave;
#pragma unroll 4
      for (; i + 4 < i1; i += 8) {
        s = fmaf(U[(int64_t)i * ldd + j], sg[i], s);
        s1 = fmaf(U[(int64_t)(i + 4) * ldd + j], sg[i + 4], s1);
      }
      if (i < i1) s = fmaf(U[(int64_t)i * ldd + j], sg[i], s);
      s += s1;
    }
    red[wave][lane] = s;
    __syncthreads();
    if (wave == 0 && j < d)
      put(ypart + (int64_t)sl * d + j, (red[0][lane] + red[1][lane]) + (red[2][lane] + red[3][lane]));
    __syncthreads();
  }

  const bool met = grid_barrier(bar, spin_limit, flag);

  // ---- phase B ----
  for (int j = t; j < d; j += 256) {
    // all of this thread's handoff loads in flight before any is used
    float v[kOnlineSlices + 2];
#pragma unroll
    for (int sl = 0; sl < kOnlineSlices; ++sl) v[sl] = get(ypart + (int64_t)sl * d + j);
    v[kOnlineSlices] = get(hhat + j);
    v[kOnlineSlices + 1] = get(xv + j);
    float s = 0.f;
#pragma unroll
    for (int sl = 0; sl < kOnlineSlices; ++sl) s += v[sl];
    sy[j] = s;
    shh[j] = v[kOnlineSlices];
    sx[j] = v[kOnlineSlices + 1];
  }
  __syncthreads();
  // ||h||^2, h^T h^, h^T y^ (fixed-order reduction: wave partials, then in order)
  float p0 = 0.f, p1 = 0.f, p2 = 0.f;
  for (int j = t; j < d; j += 256) {
    p0 = fmaf(sh[j], sh[j], p0);
    p1 = fmaf(sh[j], shh[j], p1);
    p2 = fmaf(sh[j], sy[j], p2);
  }
  p0 = wave_sum(p0);
  p1 = wave_sum(p1);
  p2 = wave_sum(p2);
  if (lane == 0) {
    red[0][wave] = p0;
    red[1][wave] = p1;
    red[2][wave] = p2;
  }
  __syncthreads();
  const float hh = (red[0][0] + red[0][1]) + (red[0][2] + red[0][3]);
  const float hhh = (red[1][0] + red[1][1]) + (red[1][2] + red[1][3]);
  const float hy = (red[2][0] + red[2][1]) + (red[2][2] + red[2][3]);
  // y^T y by index equality (repeated indices add their values)
  float yy = 0.f;
  for (int a = 0; a < K; ++a) {
    if (idx[a] < 0) continue;
    for (int b = 0; b < K; ++b)
      if (idx[b] == idx[a]) yy = fmaf(val[a], val[b], yy);
  }
  const float L = hhh - 2.f * hy + yy;
  const float den = 1.f - 2.f * lr * hh;
  const bool spd = den > 0.f;
  const bool finite = isfinite(L);
  if (blockIdx.x == 0 && t == 0) {
    *loss_out = L;
    if (!spd) atomicOr(flag, FLAG_NOT_SPD);
    if (!finite) atomicOr(flag, FLAG_NONFINITE);
  }
  if (grad_h && blockIdx.x == 0)
    for (int j = t; j < d; j += 256) grad_h[j] = 2.f * (shh[j] - sy[j]);
  if (closed || bad_idx || !met || !spd || !finite) return;

  const float cu = 2.f * lr / den;  // Sherman-Morrison coefficient of step 6
  const float c4 = 4.f * lr * lr * L;
  for (int r = gwave; r < d; r += nwaves) {
    float *q = Q + (int64_t)r * ldd, *u = U + (int64_t)r * ldd, *x = UinvT + (int64_t)r * ldd;
    const float hr = sh[r], gr = 2.f * (shh[r] - sy[r]);
    const float ur = -2.f * lr * get(uh + r), xr = cu * sx[r];
    // eight columns per lane of the three rows loaded before any of them is stored (the
    // rows may not overlap, but the compiler cannot know that)
    constexpr int kCols = 8;
    for (int k0 = lane; k0 < d; k0 += 64 * kCols) {
      float uv[kCols], xv2[kCols], qv[kCols];
#pragma unroll
      for (int e = 0; e < kCols; ++e) {
        const int k = min(k0 + 64 * e, d - 1);
        uv[e] = u[k];
        xv2[e] = x[k];
        qv[e] = q[k];
      }
#pragma unroll
      for (int e = 0; e < kCols; ++e) {
        const int k = k0 + 64 * e;
        if (k < d) {
          const float hk = sh[k], gk = 2.f * (shh[k] - sy[k]);
          u[k] = fmaf(ur, hk, uv[e]);
          x[k] = fmaf(xr, hk, xv2[e]);
          q[k] = fmaf(c4 * hr, hk, qv[e] - lr * (hr * gk + gr * hk));
        }
      }
    }
  }
  // step 7: V_c += 2 eta (sum of t over the slots of row c) P, P = U_new^{-T} h =
  // X / (1 - 2 eta ||h||^2).  Slot k goes to workgroup k mod gridDim; the first slot of
  // each distinct row owns it (one writer per row), its coefficient summed in slot order.
  const float pv = 2.f * lr / den;
  for (int k = blockIdx.x; k < K; k += gridDim.x) {
    const int ck = idx[k];
    bool owner = ck >= 0;
    float tsum = 0.f;
    for (int k2 = 0; k2 < K; ++k2) {
      if (idx[k2] != ck) continue;
      if (k2 < k) owner = false;
      tsum += val[k2];
    }
    if (!owner) continue;
    float *row = V + (int64_t)ck * ldv;
    const float sc = pv * tsum;
    for (int j = t; j < d; j += 256) row[j] = fmaf(sc, sx[j], row[j]);
  }
}

}  // namespace

size_t online_work_floats(int d) { return (size_t)(kOnlineSlices + 3) * d; }

hipError_t launch_online_step(hipStream_t s, int64_t D, int d, int K, const float *h,
                              const int *idx, const float *val, float lr, float *V, int64_t ldv,
                              float *U, float *UinvT, float *Q, int ldd, float *loss_out,
                              float *grad_h, float *work, unsigned *bar, int spin_limit,
                              int *flag) {
  LST_LAUNCH(online_step_kernel, dim3(kOnlineWGs), dim3(256), (size_t)(5 * d * sizeof(float)), s,
             D, d, K, h, idx, val, lr, V, ldv, U, UinvT, Q, ldd, loss_out, grad_h, work, bar,
             spin_limit, flag);
  return hipGetLastError();
}

}  // namespace lst
