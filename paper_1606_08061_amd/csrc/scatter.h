// V update of the factored step (eq. updateV): the per-row owner scatter, as device
// functions of one workgroup of T threads (device code shared by the HIP sources of
// liblst; not part of the C ABI).
#pragma once

#include "lst_internal.h"

namespace lst {

namespace {

// Device-coherent (agent-scope) accesses, for values that cross workgroups, and
// XCDs, within one launch.
__device__ __forceinline__ void st_dev_f(float *p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_dev_f(const float *p) {
  return __hip_atomic_load(const_cast<float *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Four consecutive floats at base + off bytes (16-byte aligned) by one device-coherent
// buffer load (the agent-scope cache policy, sc1); bytes at or beyond `bytes` read as
// zero.
__device__ __forceinline__ float4 ld_dev4(const float *base, uint32_t off, uint32_t bytes) {
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(base), (short)0, (int)bytes, 0x00020000);
  return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 16));
}

// The row sum  sum_{t < cnt} dA[list[t]] P_{j(list[t])}  for one V row of d columns:
// columns in groups of four where the layout allows (v4); the slots split into np
// interleaved parts (np a power of two, as many as the threads left over by the
// columns allow), each part summed in slot order with kIlp rows' loads in flight, the
// parts then added in a fixed order through LDS.  emit(g, tot) receives column group
// g's total (from one thread per group).
template <int T, class Emit>
__device__ __forceinline__ void row_sum(const int *list, int cnt, int K, int d, bool v4,
                                        const float *__restrict__ dA, const float *__restrict__ P,
                                        const Emit &emit) {
  const int width = v4 ? 4 : 1;
  const int ng = (d + width - 1) / width;  // column groups
  int np = 1;
  while (np < 16 && 2 * np * ng <= T) np *= 2;
  __shared__ float4 spart[T];
  for (int g0 = 0; g0 < ng; g0 += T / np) {
    const int gl = threadIdx.x % (T / np), prt = threadIdx.x / (T / np);
    const int g = g0 + gl;
    const bool active = g < ng;
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
      int t = prt;
      for (; t + (kIlp - 1) * np < cnt; t += kIlp * np) {
        float w[kIlp];
        float4 x[kIlp];
#pragma unroll
        for (int u = 0; u < kIlp; ++u) {
          const int q = list[t + u * np];
          w[u] = dA[q];
          x[u] = row(q);
        }
#pragma unroll
        for (int u = 0; u < kIlp; ++u) add(w[u], x[u]);
      }
      for (; t < cnt; t += np) {  // fewer than kIlp left
        const int q = list[t];
        add(dA[q], row(q));
      }
    }
    spart[threadIdx.x] = sum;
    __syncthreads();
    if (prt == 0 && active) {
      float4 tot = spart[gl];
      for (int p2 = 1; p2 < np; ++p2) {
        const float4 x = spart[gl + p2 * (T / np)];
        tot.x += x.x;
        tot.y += x.y;
        tot.z += x.z;
        tot.w += x.w;
      }
      emit(g, tot);
    }
    __syncthreads();
  }
}

// V_r[g] -= lr tot (column group g of width 4 or 1).
__device__ __forceinline__ void sub_row(float *vr, int g, bool v4, float lr, const float4 &tot) {
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
  float *vr = V + (int64_t)r * ldv;
  const bool v4 = (d & 3) == 0 && (ldv & 3) == 0 && (reinterpret_cast<uintptr_t>(V) & 15) == 0 &&
                  (reinterpret_cast<uintptr_t>(P) & 15) == 0;
  row_sum<T>(slist, total, K, d, v4, dA, P,
             [&](int g, const float4 &tot) { sub_row(vr, g, v4, lr, tot); });
}

// The step's form.  A workgroup per slot again, but the rows' slot lists come from a
// plan made in the previous launch (scatter_plan below), so that a slot that leads
// nothing exits after one load.  A row with more than C slots (a frequent target under
// a skewed index distribution) is summed in chunks of C slots by as many workgroups:
// each stores its chunk's partial sum and counts itself in the row's counter, and the
// last to arrive adds the partials in chunk order and writes the row, so the row still
// has one writer and a fixed summation order.
//
// The plan (4 n words): meta[s] = (rank of s among its row's slots) | (the row's slot
// count << 14), or -1 for an empty slot; pos[s] = the position of s in the slots
// ordered by (row, slot); sorted[pos] = s; tbl[pos] = the partial id of the chunk that
// starts at pos.  Partial id p (taken from *ticket) is row p of part0 for p < half,
// else row p - half of part1 (row stride d); C >= K keeps the ids below 2 half = 2 m (a
// row of more than C slots has at most total / C + 1 chunks, and there are fewer than
// n / C such rows).  rcnt (n words, indexed by a row's first position) is zero before
// the launch and left zero by each row's last arriver; *ticket is zero at the launch's
// start.
struct ScatterChunks {
  int C;
  int half;
  float *part0, *part1;
  int *plan;  // meta, pos, sorted, tbl: n words each
  int *rcnt, *ticket;
};

constexpr int kListMax = 64;       // a chunk's slots: C = max(32, K) <= LST_MAX_K
constexpr int kChunkMax = 257;     // a row's chunks: n / 32 + 1 (n = m K <= 8192)
constexpr int kPlanTile = 2048;    // indices staged in LDS per pass of the plan

// The plan for slots [16 b, 16 b + 16) of n: sixteen threads per slot, each comparing
// a sixteenth of every staged tile of indices (four at a time); their counts added by
// lane shuffles.
__device__ __forceinline__ void scatter_plan(int b, int n, const int *__restrict__ idx,
                                             int *__restrict__ plan) {
  __shared__ __align__(16) int tile[kPlanTile];
  const int s = 16 * b + ((int)threadIdx.x >> 4), part = threadIdx.x & 15;
  const int r = s < n ? idx[s] : -1;
  int below = 0, total = 0, less = 0;
  for (int t0 = 0; t0 < n; t0 += kPlanTile) {
    const int tn = min(kPlanTile, n - t0), tn4 = (tn + 3) >> 2;
    __syncthreads();  // the previous tile has been read
    for (int i = threadIdx.x; i < 4 * tn4; i += 256) tile[i] = i < tn ? idx[t0 + i] : -1;
    __syncthreads();
    if (r >= 0) {
      const int4 *t4 = reinterpret_cast<const int4 *>(tile);
#pragma unroll 4
      for (int i = part; i < tn4; i += 16) {
        const int4 v = t4[i];
        const int q = t0 + 4 * i;
        total += (v.x == r) + (v.y == r) + (v.z == r) + (v.w == r);
        below += ((v.x == r) & (q < s)) + ((v.y == r) & (q + 1 < s)) + ((v.z == r) & (q + 2 < s)) +
                 ((v.w == r) & (q + 3 < s));
        less += ((v.x >= 0) & (v.x < r)) + ((v.y >= 0) & (v.y < r)) + ((v.z >= 0) & (v.z < r)) +
                ((v.w >= 0) & (v.w < r));
      }
    }
  }
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) {
    below += __shfl_xor(below, o);
    total += __shfl_xor(total, o);
    less += __shfl_xor(less, o);
  }
  if (part == 0 && s < n) {
    plan[s] = r >= 0 ? below | (total << 14) : -1;
    if (r >= 0) {
      plan[n + s] = less + below;
      plan[2 * n + less + below] = s;
    }
  }
}

template <int T>
__device__ __forceinline__ void scatter_planned(int s, int n, int K, int d, float lr,
                                                const int *__restrict__ idx,
                                                const float *__restrict__ dA,
                                                const float *__restrict__ P,
                                                float *__restrict__ V, int64_t ldv,
                                                const ScatterChunks &ch) {
  __shared__ int slist[kListMax];
  __shared__ int spid[kChunkMax];
  __shared__ int sid, slast;
  const int *meta = ch.plan, *spos = ch.plan + n, *sorted = ch.plan + 2 * n;
  int *tbl = ch.plan + 3 * n;
  const int mt = meta[s];
  const int C = ch.C;
  // the row's first slot leads; a row of more than C slots has a leader every C slots
  if (mt < 0 || (mt & 0x3FFF) % C != 0) return;
  const int rank = mt & 0x3FFF, total = mt >> 14;
  const int pos = spos[s], pos0 = pos - rank;
  const int nch = (total + C - 1) / C;
  const int mine = min(total - rank, C);  // this workgroup's slots: sorted[pos, pos + mine)
  for (int t = threadIdx.x; t < mine; t += T) slist[t] = sorted[pos + t];
  __syncthreads();

  float *vr = V + (int64_t)idx[s] * ldv;
  const bool v4 = (d & 3) == 0 && (ldv & 3) == 0 && (reinterpret_cast<uintptr_t>(V) & 15) == 0 &&
                  (reinterpret_cast<uintptr_t>(P) & 15) == 0;
  const int width = v4 ? 4 : 1;
  if (nch == 1) {
    row_sum<T>(slist, mine, K, d, v4, dA, P,
               [&](int g, const float4 &tot) { sub_row(vr, g, v4, lr, tot); });
    return;
  }
  if (threadIdx.x == 0)
    sid = __hip_atomic_fetch_add(ch.ticket, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  const int id = sid;
  if (id >= 2 * ch.half) return;  // cannot happen with C >= K (see ScatterChunks)
  float *part = id < ch.half ? ch.part0 + (int64_t)id * d : ch.part1 + (int64_t)(id - ch.half) * d;
  row_sum<T>(slist, mine, K, d, v4, dA, P, [&](int g, const float4 &tot) {
    float *pp = part + g * width;
    st_dev_f(pp, tot.x);
    if (v4) {
      st_dev_f(pp + 1, tot.y);
      st_dev_f(pp + 2, tot.z);
      st_dev_f(pp + 3, tot.w);
    }
  });

  // Arrival after every thread's partial stores have completed (each waits for its
  // own), so that the row's last arriver reads complete partials.
  if (threadIdx.x == 0)
    __hip_atomic_store(tbl + pos, id, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (threadIdx.x == 0) {
    slast = __hip_atomic_fetch_add(ch.rcnt + pos0, 1, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT) == nch - 1;
    if (slast)  // every chunk has arrived: the counter returns to zero for the next step
      __hip_atomic_store(ch.rcnt + pos0, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
  if (!slast) return;

  // The last arriver adds the chunks' partials in chunk order (eight chunks' loads in
  // flight), their ids read from the chunks' first positions.
  for (int c = threadIdx.x; c < nch; c += T)
    spid[c] = __hip_atomic_load(tbl + pos0 + c * C, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  const int ng = (d + width - 1) / width;
  const uint32_t pbytes = (uint32_t)((size_t)ch.half * d * sizeof(float));
  auto partial = [&](int c, int g) {
    const int pid = spid[c];
    const float *base = pid < ch.half ? ch.part0 : ch.part1;
    const uint32_t off =
        (uint32_t)(((size_t)(pid < ch.half ? pid : pid - ch.half) * d + g * width) * sizeof(float));
    if (v4) return ld_dev4(base, off, pbytes);
    return make_float4(ld_dev_f(base + off / sizeof(float)), 0.f, 0.f, 0.f);
  };
  for (int g = threadIdx.x; g < ng; g += T) {
    float4 tot = make_float4(0.f, 0.f, 0.f, 0.f);
    constexpr int kCh = 8;
    for (int c0 = 0; c0 < nch; c0 += kCh) {
      float4 x[kCh];
#pragma unroll
      for (int u = 0; u < kCh; ++u) x[u] = partial(min(c0 + u, nch - 1), g);
#pragma unroll
      for (int u = 0; u < kCh; ++u)
        if (c0 + u < nch) {
          tot.x += x[u].x;
          tot.y += x[u].y;
          tot.z += x[u].z;
          tot.w += x[u].w;
        }
    }
    sub_row(vr, g, v4, lr, tot);
  }
}

}  // namespace

}  // namespace lst
