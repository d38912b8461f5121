// Batched fp32 GEMM on the CDNA4 matrix cores (v_mfma_f32_32x32x2_f32).
//
// Every d x d and d x m contraction of the factored step (Algorithm 3 steps
// 1, 2, 5, 6, 8 and the matching rows of Algorithm 4), the m x m products
// (H^T H, H^T H^, H~^T G) and the naive path's D x d products go through this
// one kernel template.  A workgroup owns a 32 x 32 output tile; its NW
// wavefronts split the k range and their accumulators are summed through LDS
// in a fixed order, so results do not depend on scheduling.
//
// MFMA operand mapping (one 32x32x2 instruction, 64 lanes): lane l supplies
// A[i = l%32][kk = l/32] and B[kk = l/32][j = l%32]; the 16 accumulator values
// of lane l hold C[8*(r/4) + 4*(l/32) + r%4][l%32], r = 0..15.  A k-block of 8
// is consumed by four instructions; in instruction s lane-half h feeds
// k = kb + 4h + s for both operands, so each lane reads 4 consecutive k values
// of its row (one 16-byte load when k is the contiguous dimension).
//
// Loads are branch free: a lane whose output row (column) lies beyond M (N)
// reads the last valid row instead, since that output is never stored; only
// the ragged end of the k range is masked.  Operands are fetched kStage
// k-blocks ahead of the matrix cores.
#include "lst_internal.h"
#include "scatter.h"

namespace lst {

namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kStage = 4;

// Operand access modes.  VEC: k contiguous and 16-byte aligned, one float4 per
// lane; STRIDED: four scalars at p[idx*si + (k0+s)*sk] (k contiguous with an
// unaligned stride, or the index contiguous).
enum : int { VEC = 0, STRIDED = 1 };

template <int MODE>
__device__ __forceinline__ void ld4(const float *__restrict__ p, int64_t si, int64_t sk, int idx,
                                    int k0, float (&o)[4]) {
  if constexpr (MODE == VEC) {
    const float4 v = *reinterpret_cast<const float4 *>(p + (int64_t)idx * si + k0);
    o[0] = v.x;
    o[1] = v.y;
    o[2] = v.z;
    o[3] = v.w;
  } else {
    const float *q = p + (int64_t)idx * si + (int64_t)k0 * sk;
    o[0] = q[0];
    o[1] = q[sk];
    o[2] = q[2 * sk];
    o[3] = q[3 * sk];
  }
}

// Ragged end of the k range: k >= kend reads as zero (address clamped).
__device__ __forceinline__ void ld4_tail(const float *__restrict__ p, int64_t si, int64_t sk,
                                         int idx, int k0, int kend, float (&o)[4]) {
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const int kk = k0 + s;
    const float v = p[(int64_t)idx * si + (int64_t)min(kk, kend - 1) * sk];
    o[s] = (kk < kend) ? v : 0.f;
  }
}

// One wavefront's share of the k blocks of 8: blocks wave, wave + NW, ... of
// the first segment (k in [kbeg, kbeg + len1)) followed by the second (k in
// [0, len2) of A2, B2), so that the loads of both are in flight together.  The
// last block of a segment may be ragged (masked loads).
template <int NW, int AM, int BM>
__device__ __forceinline__ void kloop(floatx16 &acc, const float *A, int64_t asi, int64_t ask,
                                      const float *B, int64_t bsi, int64_t bsk, int len1,
                                      const float *A2, int64_t asi2, int64_t ask2, const float *B2,
                                      int64_t bsi2, int64_t bsk2, int len2, int ia, int jb,
                                      int kbeg, int wave, int lh) {
  const int nb1 = (len1 + 7) >> 3;
  const int nb = nb1 + ((len2 + 7) >> 3);
  const int nw = nb > wave ? (nb - wave + NW - 1) / NW : 0;
  auto load = [&](int s, float(&a)[4], float(&b)[4]) {
    const int bi = wave + NW * min(s, nw - 1);
    if (bi < nb1) {
      const int k0 = kbeg + 8 * bi + 4 * lh;
      if (8 * bi + 8 <= len1) {
        ld4<AM>(A, asi, ask, ia, k0, a);
        ld4<BM>(B, bsi, bsk, jb, k0, b);
      } else {
        ld4_tail(A, asi, ask, ia, k0, kbeg + len1, a);
        ld4_tail(B, bsi, bsk, jb, k0, kbeg + len1, b);
      }
    } else {
      const int k0 = 8 * (bi - nb1) + 4 * lh;
      if (8 * (bi - nb1) + 8 <= len2) {
        ld4<AM>(A2, asi2, ask2, ia, k0, a);
        ld4<BM>(B2, bsi2, bsk2, jb, k0, b);
      } else {
        ld4_tail(A2, asi2, ask2, ia, k0, len2, a);
        ld4_tail(B2, bsi2, bsk2, jb, k0, len2, b);
      }
    }
  };
  if (nw == 0) return;
  float a[kStage][4], b[kStage][4];
#pragma unroll
  for (int u = 0; u < kStage; ++u) load(u, a[u], b[u]);
  for (int s0 = 0; s0 < nw; s0 += kStage) {
    float an[kStage][4], bn[kStage][4];
#pragma unroll
    for (int u = 0; u < kStage; ++u)
      if (s0 + kStage + u < nw) load(s0 + kStage + u, an[u], bn[u]);
#pragma unroll
    for (int u = 0; u < kStage; ++u) {
      if (s0 + u < nw) {
#pragma unroll
        for (int s = 0; s < 4; ++s)
          acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[u][s], b[u][s], acc, 0, 0, 0);
      }
    }
#pragma unroll
    for (int u = 0; u < kStage; ++u)
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        a[u][s] = an[u][s];
        b[u][s] = bn[u][s];
      }
  }
}

__device__ __forceinline__ bool vec_ok(const float *p, int64_t ld) {
  return ((reinterpret_cast<uintptr_t>(p) & 15) == 0) && ((ld & 3) == 0);
}

// opA(i,k): tA = 0 -> A[i*lda + k] (index stride lda, k stride 1); tA = 1 -> A[k*lda + i].
// opB(k,j): tB = 0 -> B[j*ldb + k];                                 tB = 1 -> B[k*ldb + j].
// k runs over [kbeg, kend) of (A, B) and then over [0, K2) of (A2, B2).
template <int NW>
__device__ __forceinline__ void segment(floatx16 &acc, const float *A, int64_t lda, int tA,
                                        const float *B, int64_t ldb, int tB, const float *A2,
                                        int64_t lda2, const float *B2, int64_t ldb2, int K2,
                                        int ia, int jb, int kbeg, int kend, int wave, int lh) {
  const int64_t asi = tA ? 1 : lda, ask = tA ? lda : 1;
  const int64_t bsi = tB ? 1 : ldb, bsk = tB ? ldb : 1;
  const int64_t asi2 = tA ? 1 : lda2, ask2 = tA ? lda2 : 1;
  const int64_t bsi2 = tB ? 1 : ldb2, bsk2 = tB ? ldb2 : 1;
  const bool av = !tA && vec_ok(A, lda) && (K2 == 0 || vec_ok(A2, lda2));
  const bool bv = !tB && vec_ok(B, ldb) && (K2 == 0 || vec_ok(B2, ldb2));
#define LST_KLOOP(AMODE, BMODE)                                                                    \
  kloop<NW, AMODE, BMODE>(acc, A, asi, ask, B, bsi, bsk, kend - kbeg, A2, asi2, ask2, B2, bsi2, \
                          bsk2, K2, ia, jb, kbeg, wave, lh)
  if (av && bv)
    LST_KLOOP(VEC, VEC);
  else if (av)
    LST_KLOOP(VEC, STRIDED);
  else if (bv)
    LST_KLOOP(STRIDED, VEC);
  else
    LST_KLOOP(STRIDED, STRIDED);
#undef LST_KLOOP
}

__device__ __forceinline__ void finish(const GemmDesc &g, int i, int j, float v) {
  float out = g.alpha * v;
  if (g.Cin) out += g.beta * g.Cin[(int64_t)i * g.ldcin + j];
  g.C[(int64_t)i * g.ldc + j] = out;
  if (g.epi == EPI_GRADH) g.C2[(int64_t)i * g.ldc2 + j] = 2.f * g.rs[i] * g.E[(int64_t)i * g.lde + j] + out;
}

// Workgroup w runs on XCD w % 8; consecutive logical tiles are given to the same
// XCD so that tiles sharing an operand panel share that XCD's L2.
__device__ __forceinline__ int xcd_tile(int wg, int T) {
  const int q = T >> 3, r = T & 7;
  const int x = wg & 7, slot = wg >> 3;
  return x < r ? x * (q + 1) + slot : r * (q + 1) + (x - r) * q + slot;
}

__device__ __forceinline__ const float *resolve(const float *p, const float *H, float *gH) {
  const uintptr_t v = reinterpret_cast<uintptr_t>(p);
  return v == 16 ? H : (v == 32 ? gH : p);
}

template <int NW>
__device__ __forceinline__ void gemm_body(const GemmBatch &bt, const float *H, float *gH, float lr,
                                          const int *__restrict__ gate) {
  // The gate only suppresses writes, so its load is waited for at the end.
  const int closed = gate ? *gate : 0;
  const int tile = xcd_tile(blockIdx.x, bt.total_tiles);
  int di = 0;
#pragma unroll
  for (int q = 1; q < kMaxBatch; ++q)
    if (q < bt.n && tile >= bt.d[q].tile_begin) di = q;
  GemmDesc g = bt.d[di];
  g.A = resolve(g.A, H, gH);
  g.B = resolve(g.B, H, gH);
  g.A2 = resolve(g.A2, H, gH);
  g.B2 = resolve(g.B2, H, gH);
  g.Cin = resolve(g.Cin, H, gH);
  g.C2 = const_cast<float *>(resolve(g.C2, H, gH));
  if (g.lr_scaled) {
    g.alpha *= lr * lr;
    g.beta *= lr;
  }

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int li = lane & 31, lh = lane >> 5;
  const int local = tile - g.tile_begin;
  const int per_split = g.tiles_m * g.tiles_n;
  const int split = local / per_split;
  const int t2 = local - split * per_split;
  const int tm = t2 / g.tiles_n;
  const int tn = t2 - tm * g.tiles_n;
  const int i0 = tm * 32, j0 = tn * 32;
  const int ia = min(i0 + li, g.M - 1), jb = min(j0 + li, g.N - 1);

  // Epilogue operands (C_in, and E of the grad_H epilogue) are fetched before the
  // k loop so that their latency overlaps it.  Thread o of the tile's 1024
  // outputs holds output (r, ln) = (o / 64, o % 64) after the reduction below.
  constexpr int kPer = 1024 / (64 * NW);
  float cin[kPer], ein[kPer];
  const bool use_cin = g.Cin != nullptr && g.splits == 1;
  const bool use_e = g.epi == EPI_GRADH && g.splits == 1;
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int o = threadIdx.x + u * 64 * NW;
    const int r = o >> 6, ln = o & 63;
    const int i = min(i0 + (r >> 2) * 8 + (ln >> 5) * 4 + (r & 3), g.M - 1);
    const int j = min(j0 + (ln & 31), g.N - 1);
    cin[u] = use_cin ? g.Cin[(int64_t)i * g.ldcin + j] : 0.f;
    ein[u] = use_e ? g.E[(int64_t)i * g.lde + j] : 0.f;
  }

  floatx16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.f;

  if (g.splits > 1) {
    const int kbeg = split * g.kchunk;
    const int kend = min(g.K, kbeg + g.kchunk);
    segment<NW>(acc, g.A, g.lda, g.tA, g.B, g.ldb, g.tB, nullptr, 0, nullptr, 0, 0, ia, jb, kbeg,
                kend, wave, lh);
  } else {
    segment<NW>(acc, g.A, g.lda, g.tA, g.B, g.ldb, g.tB, g.A2, g.lda2, g.B2, g.ldb2, g.K2, ia, jb,
                0, g.K, wave, lh);
  }

  __shared__ float red[NW][16][64];
#pragma unroll
  for (int r = 0; r < 16; ++r) red[wave][r][lane] = acc[r];
  __syncthreads();
  if (closed) return;  // after the last barrier
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int o = threadIdx.x + u * 64 * NW;
    const int r = o >> 6, ln = o & 63;
    float v = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) v += red[w][r][ln];
    const int i = i0 + (r >> 2) * 8 + (ln >> 5) * 4 + (r & 3);
    const int j = j0 + (ln & 31);
    if (i < g.M && j < g.N) {
      if (g.splits > 1) {
        g.partial[((int64_t)split * g.M + i) * g.N + j] = v;
      } else {
        const float out = g.alpha * v + g.beta * cin[u];
        g.C[(int64_t)i * g.ldc + j] = out;
        if (use_e) g.C2[(int64_t)i * g.ldc2 + j] = 2.f * g.rs[i] * ein[u] + out;
      }
    }
  }
}

// PHASE only names the instantiation, so profilers report each step phase separately.
template <int PHASE, int NW>
__global__ __launch_bounds__(64 * NW, 12 / NW) void gemm_kernel(const GemmBatch bt, const int *__restrict__ gate) {
  gemm_body<NW>(bt, nullptr, nullptr, 1.f, gate);
}

// The batch read from device memory (a plan), with the step's H, grad_H and lr.
template <int PHASE, int NW>
__global__ __launch_bounds__(64 * NW, 12 / NW) void gemm_plan_kernel(const GemmBatch *__restrict__ bt,
                                                            const float *H, float *gH, float lr,
                                                            const int *__restrict__ gate,
                                                            const StepSync sync) {
  step_sync_begin(sync);
  gemm_body<NW>(*bt, H, gH, lr, gate);
}

// The squared-error update launch with the V update in it: workgroups below
// ntiles run the update plan's tiles, each of the others one target slot of the
// scatter (256 threads).  Both only read the mid launch's outputs (Yw, dl/dA),
// and they write disjoint state (U^-T and Q; the target rows of V), so the
// scatter needs no launch of its own after the update.
__global__ __launch_bounds__(256, 4) void update_scatter_kernel(
    const GemmBatch *__restrict__ bt, int ntiles, const float *H, float *gH, float lr,
    const int *__restrict__ gate, int n, int K, int d, float slr, const int *__restrict__ idx,
    const float *__restrict__ dA, const float *__restrict__ P, float *__restrict__ V,
    int64_t ldv) {
  if ((int)blockIdx.x < ntiles) {
    gemm_body<4>(*bt, H, gH, lr, gate);
    return;
  }
  extern __shared__ int sh[];
  if (*gate != 0) return;
  scatter_slot<256>((int)blockIdx.x - ntiles, n, K, d, slr, idx, dA, P, V, ldv, sh);
}

__global__ __launch_bounds__(256) void splitk_reduce_kernel(const GemmDesc g, const int *__restrict__ gate) {
  if (gate && *gate != 0) return;
  const int64_t total = (int64_t)g.M * g.N;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    // eight interleaved partial sums (loads in flight together), added in a fixed order
    float v[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    int s = 0;
    for (; s + 8 <= g.splits; s += 8)
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] += g.partial[(int64_t)(s + u) * total + e];
    for (; s < g.splits; ++s) v[0] += g.partial[(int64_t)s * total + e];
    const float sum = ((v[0] + v[1]) + (v[2] + v[3])) + ((v[4] + v[5]) + (v[6] + v[7]));
    const int i = (int)(e / g.N), j = (int)(e % g.N);
    finish(g, i, j, sum);
  }
}

// ---------------------------------------------------------------------------
// 16 x 16 output tiles (v_mfma_f32_16x16x4f32) for the step's plans: four times
// the workgroups of the 32 x 32 form on these small products, and each
// wavefront's share of k loaded in one round.  Lane l = c + 16 g supplies
// A[i = c][k] and B[k][j = c] for k = kb + 4g + s in instruction s of a k-block
// of 16 (four consecutive k of its row: one 16-byte load when k is contiguous);
// accumulator register r holds C[4g + r][c].  The four wavefronts take the
// k-blocks w, w + 4, ...; their sums are added through LDS in a fixed order.
// ---------------------------------------------------------------------------
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kT16Group = 8;  // k-blocks of 16 loaded per round

template <int AM, int BM>
__device__ __forceinline__ void kloop16(floatx4 &acc, const float *A, int64_t asi, int64_t ask,
                                        const float *B, int64_t bsi, int64_t bsk, int ia, int jb,
                                        int K, int wave, int g) {
  const int nfull = K >> 4;
  const int nw = nfull > wave ? (nfull - wave + 3) / 4 : 0;
  for (int b0 = 0; b0 < nw; b0 += kT16Group) {
    float a[kT16Group][4], b[kT16Group][4];
#pragma unroll
    for (int u = 0; u < kT16Group; ++u) {
      const int kb = 16 * (wave + 4 * min(b0 + u, nw - 1)) + 4 * g;
      ld4<AM>(A, asi, ask, ia, kb, a[u]);
      ld4<BM>(B, bsi, bsk, jb, kb, b[u]);
    }
#pragma unroll
    for (int u = 0; u < kT16Group; ++u)
      if (b0 + u < nw) {
#pragma unroll
        for (int s = 0; s < 4; ++s)
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[u][s], b[u][s], acc, 0, 0, 0);
      }
  }
  if ((K & 15) && wave == 3) {
    const int k0 = 16 * nfull + 4 * g;
    float a[4], b[4];
    ld4_tail(A, asi, ask, ia, k0, K, a);
    ld4_tail(B, bsi, bsk, jb, k0, K, b);
#pragma unroll
    for (int s = 0; s < 4; ++s) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[s], b[s], acc, 0, 0, 0);
  }
}

__device__ __forceinline__ void segment16(floatx4 &acc, const float *A, int64_t lda, int tA,
                                          const float *B, int64_t ldb, int tB, int ia, int jb,
                                          int K, int wave, int g) {
  const int64_t asi = tA ? 1 : lda, ask = tA ? lda : 1;
  const int64_t bsi = tB ? 1 : ldb, bsk = tB ? ldb : 1;
  const bool av = !tA && vec_ok(A, lda);
  const bool bv = !tB && vec_ok(B, ldb);
  if (av && bv)
    kloop16<VEC, VEC>(acc, A, asi, ask, B, bsi, bsk, ia, jb, K, wave, g);
  else if (av)
    kloop16<VEC, STRIDED>(acc, A, asi, ask, B, bsi, bsk, ia, jb, K, wave, g);
  else if (bv)
    kloop16<STRIDED, VEC>(acc, A, asi, ask, B, bsi, bsk, ia, jb, K, wave, g);
  else
    kloop16<STRIDED, STRIDED>(acc, A, asi, ask, B, bsi, bsk, ia, jb, K, wave, g);
}

// One 16 x 16 tile per workgroup of 256 threads; thread t finishes output
// (4 (t / 16 % 4) + ..., see below) after the reduction.  No split-k.
// One 16 x 16 output tile of a plan batch (workgroup blockIdx.x).
__device__ __forceinline__ void gemm16_tile(const GemmBatch &bt_, const float *H, float *gH,
                                            float lr, const int *__restrict__ gate) {
  const GemmBatch *bt = &bt_;
  const int closed = gate ? *gate : 0;  // waited for at the end: it only suppresses writes
  const int tile = xcd_tile(blockIdx.x, bt->total_tiles);
  int di = 0;
#pragma unroll
  for (int q = 1; q < kMaxBatch; ++q)
    if (q < bt->n && tile >= bt->d[q].tile_begin) di = q;
  GemmDesc g = bt->d[di];
  g.A = resolve(g.A, H, gH);
  g.B = resolve(g.B, H, gH);
  g.A2 = resolve(g.A2, H, gH);
  g.B2 = resolve(g.B2, H, gH);
  g.Cin = resolve(g.Cin, H, gH);
  g.C2 = const_cast<float *>(resolve(g.C2, H, gH));
  if (g.lr_scaled) {
    g.alpha *= lr * lr;
    g.beta *= lr;
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = lane & 15, lg = lane >> 4;
  const int local = tile - g.tile_begin;
  const int tm = local / g.tiles_n, tn = local - tm * g.tiles_n;
  const int i0 = tm * 16, j0 = tn * 16;
  const int ia = min(i0 + c, g.M - 1), jb = min(j0 + c, g.N - 1);

  // Output of thread t after the reduction: accumulator register r = wave of
  // lane lane: row 4 lg + wave, column c (each wavefront finishes one register).
  const int oi = i0 + 4 * lg + wave, oj = j0 + c;
  const int ci = min(oi, g.M - 1), cj = min(oj, g.N - 1);
  const bool use_e = g.epi == EPI_GRADH;
  const float cin = g.Cin ? g.Cin[(int64_t)ci * g.ldcin + cj] : 0.f;
  const float ein = use_e ? g.E[(int64_t)ci * g.lde + cj] : 0.f;

  floatx4 acc = {0.f, 0.f, 0.f, 0.f};
  segment16(acc, g.A, g.lda, g.tA, g.B, g.ldb, g.tB, ia, jb, g.K, wave, lg);
  if (g.K2 > 0) segment16(acc, g.A2, g.lda2, g.tA, g.B2, g.ldb2, g.tB, ia, jb, g.K2, wave, lg);

  __shared__ float red[4][4][64];
#pragma unroll
  for (int r = 0; r < 4; ++r) red[wave][r][lane] = acc[r];
  __syncthreads();
  if (closed) return;  // after the last barrier
  const float v = (red[0][wave][lane] + red[1][wave][lane]) + (red[2][wave][lane] + red[3][wave][lane]);
  if (oi < g.M && oj < g.N) {
    const float out = g.alpha * v + g.beta * cin;
    g.C[(int64_t)oi * g.ldc + oj] = out;
    if (use_e) g.C2[(int64_t)oi * g.ldc2 + oj] = 2.f * g.rs[oi] * ein + out;
  }
}

template <int PHASE>
__global__ __launch_bounds__(256) void gemm16_plan_kernel(const GemmBatch *__restrict__ bt,
                                                           const float *H, float *gH, float lr,
                                                           const int *__restrict__ gate,
                                                           const int *__restrict__ pf_idx,
                                                           int pf_K, const StepSync sync) {
  step_sync_begin(sync);
  if ((int)blockIdx.x >= bt->total_tiles) {
    // Prefetch workgroup: the target rows of example j (indices outside [0, D) skipped).
    // The indices first (one load each, through LDS), then one load per 128-byte
    // line of every row, all at once.
    const int j = (int)blockIdx.x - bt->pf_base;
    if (j < 0 || j >= bt->pf_m) return;
    __shared__ int prow[LST_MAX_K];
    for (int k = threadIdx.x; k < pf_K; k += 256) {
      const int r = pf_idx[(int64_t)j * pf_K + k];
      prow[k] = (r < 0 || (int64_t)r >= bt->pf_D) ? -1 : r;
    }
    __syncthreads();
    const int nl = (bt->pf_d + 31) >> 5;  // 128-byte lines per row (one load touches each)
    float sink = 0.f;
    for (int e = threadIdx.x; e < pf_K * nl; e += 256) {
      const int k = e / nl, r = prow[k];
      if (r >= 0) sink += bt->pf_V[(int64_t)r * bt->pf_ldv + 32 * (e - k * nl)];
    }
    asm volatile("" ::"v"(sink));
    return;
  }
  gemm16_tile(*bt, H, gH, lr, gate);
}

// ---------------------------------------------------------------------------
// Large products (the naive path's D x m, D x d and split-D m x d GEMMs): a
// 128 x 128 output tile per workgroup of four wavefronts (2 x 2, each 64 x 64 =
// 2 x 2 blocks of v_mfma_f32_32x32x2f32), k in steps of 16 staged through two
// LDS buffers.  The global loads of step s + 2 are issued before step s runs on
// the matrix cores (two register sets), so each load has two steps of MFMA work
// to arrive in.  LDS holds both operands k-major ([k][i], [k][j]) so the MFMA
// operand reads are consecutive across lanes.  Requires 16-byte aligned operands
// with leading dimensions that are multiples of 4 (checked by the host).
// ---------------------------------------------------------------------------
constexpr int kBigT = 128, kBigK = 16, kBigLd = kBigT + 4, kBigU = kBigK / 8;

// Global -> registers for one k-step: 2048 floats of each operand per workgroup,
// two float4 per thread.  KCONT: k is the contiguous dimension of the operand.
// MASK: the step may run past kend (the last step of a k range).
template <bool KCONT, bool MASK>
__device__ __forceinline__ void big_load(const float *__restrict__ p, int64_t ld, int idx0, int nidx,
                                         int k0, int kend, float4 (&v)[kBigU]) {
  const int t = threadIdx.x;
#pragma unroll
  for (int u = 0; u < kBigU; ++u) {
    if constexpr (KCONT) {  // thread t: row t / 2, k chunk (t % 2) U + u
      const float *row = p + (int64_t)min(idx0 + (t >> 1), nidx - 1) * ld;
      const int k = k0 + ((t & 1) * kBigU + u) * 4;
      if constexpr (!MASK) {
        v[u] = *reinterpret_cast<const float4 *>(row + k);
      } else {
        const float4 x = *reinterpret_cast<const float4 *>(row + (k + 3 < kend ? k : 0));
        v[u] = (k + 3 < kend) ? x
                              : make_float4(k < kend ? row[k] : 0.f, k + 1 < kend ? row[k + 1] : 0.f,
                                            k + 2 < kend ? row[k + 2] : 0.f, 0.f);
      }
    } else {  // thread t: k row t / 32 + 8 u, index (t % 32) * 4 .. + 3
      const int k = k0 + (t >> 5) + 8 * u;
      const int i = min(idx0 + (t & 31) * 4, nidx - 4);
      const float4 x =
          *reinterpret_cast<const float4 *>(p + (int64_t)(MASK ? min(k, kend - 1) : k) * ld + i);
      v[u] = (!MASK || k < kend) ? x : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  }
}

template <bool KCONT>
__device__ __forceinline__ void big_store(float (*lds)[kBigLd], const float4 (&v)[kBigU]) {
  const int t = threadIdx.x;
#pragma unroll
  for (int u = 0; u < kBigU; ++u) {
    if constexpr (KCONT) {
      const int i = t >> 1, k = ((t & 1) * kBigU + u) * 4;
      lds[k][i] = v[u].x;
      lds[k + 1][i] = v[u].y;
      lds[k + 2][i] = v[u].z;
      lds[k + 3][i] = v[u].w;
    } else {
      *reinterpret_cast<float4 *>(&lds[(t >> 5) + 8 * u][(t & 31) * 4]) = v[u];
    }
  }
}

__device__ __forceinline__ void big_mfma(float (*As)[kBigLd], float (*Bs)[kBigLd], floatx16 (&acc)[2][2],
                                         int wr, int wc, int li, int lh) {
#pragma unroll
  for (int kk = 0; kk < kBigK; kk += 2) {
    float a[2], b[2];
#pragma unroll
    for (int x = 0; x < 2; ++x) {
      a[x] = As[kk + lh][64 * wr + 32 * x + li];
      b[x] = Bs[kk + lh][64 * wc + 32 * x + li];
    }
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
      for (int y = 0; y < 2; ++y)
        acc[x][y] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[x], b[y], acc[x][y], 0, 0, 0);
  }
}

// Epilogues: C = alpha acc; C = alpha acc + beta Cin; or the split's partial sums.
enum : int { BIG_STORE = 0, BIG_AXPBY = 1, BIG_PARTIAL = 2 };

// TA: opA(i,k) = A[k*lda + i] (else A[i*lda + k]); TB: opB(k,j) = B[k*ldb + j] (else B[j*ldb + k]).
template <int PHASE, bool TA, bool TB, int EPI>
__global__ __launch_bounds__(256) void gemm_big_kernel(const GemmDesc g, const int *__restrict__ gate) {
  const int closed = gate ? *gate : 0;
  const int tiles_per_split = g.tiles_m * g.tiles_n;
  const int tile = xcd_tile(blockIdx.x, tiles_per_split * g.splits);
  const int split = tile / tiles_per_split;
  const int t2 = tile - split * tiles_per_split;
  const int tm = t2 / g.tiles_n, tn = t2 - tm * g.tiles_n;
  const int i0 = tm * kBigT, j0 = tn * kBigT;
  const int kbeg = split * g.kchunk, kend = min(g.K, kbeg + g.kchunk);

  __shared__ float As[2][kBigK][kBigLd];
  __shared__ float Bs[2][kBigK][kBigLd];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int li = lane & 31, lh = lane >> 5;
  const int wr = wave >> 1, wc = wave & 1;

  floatx16 acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;

  const int nsteps = (kend - kbeg + kBigK - 1) / kBigK;
  const int nfull = (kend - kbeg) / kBigK;  // steps entirely below kend
  auto load = [&](int st, float4(&ra)[kBigU], float4(&rb)[kBigU]) {
    const int k0 = kbeg + st * kBigK;
    if (st < nfull) {
      big_load<!TA, false>(g.A, g.lda, i0, g.M, k0, kend, ra);
      big_load<!TB, false>(g.B, g.ldb, j0, g.N, k0, kend, rb);
    } else {
      big_load<!TA, true>(g.A, g.lda, i0, g.M, k0, kend, ra);
      big_load<!TB, true>(g.B, g.ldb, j0, g.N, k0, kend, rb);
    }
  };
  float4 ra0[kBigU], rb0[kBigU], ra1[kBigU], rb1[kBigU];
  if (nsteps > 0) {
    load(0, ra0, rb0);
    big_store<!TA>(As[0], ra0);
    big_store<!TB>(Bs[0], rb0);
  }
  if (nsteps > 1) load(1, ra1, rb1);
  __syncthreads();
  // Step st runs on LDS buffer st % 2, with the loads of step st + 2 in flight in
  // register set st % 2; step st + 1 goes from register set (st + 1) % 2 to LDS.
  int st = 0;
  for (; st + 1 < nsteps; st += 2) {
    if (st + 2 < nsteps) load(st + 2, ra0, rb0);
    big_mfma(As[0], Bs[0], acc, wr, wc, li, lh);
    big_store<!TA>(As[1], ra1);
    big_store<!TB>(Bs[1], rb1);
    __syncthreads();
    if (st + 3 < nsteps) load(st + 3, ra1, rb1);
    big_mfma(As[1], Bs[1], acc, wr, wc, li, lh);
    if (st + 2 < nsteps) {
      big_store<!TA>(As[0], ra0);
      big_store<!TB>(Bs[0], rb0);
    }
    __syncthreads();
  }
  if (st < nsteps) big_mfma(As[0], Bs[0], acc, wr, wc, li, lh);
  if (closed) return;

  if (g.colsq) {
    // lane (li, lh) of wave (wr, wc) holds, for each column j, the rows
    // 64 wr + 32 x + 8 (r / 4) + 4 lh + r % 4 of the tile: a fixed 32-row subset.
#pragma unroll
    for (int y = 0; y < 2; ++y) {
      float sq = 0.f;
#pragma unroll
      for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int i = i0 + 64 * wr + 32 * x + 8 * (r >> 2) + 4 * lh + (r & 3);
          const float v = acc[x][y][r];
          sq += i < g.M ? v * v : 0.f;
        }
      const int j = j0 + 64 * wc + 32 * y + li;
      if (j < g.N) g.colsq[(int64_t)(kBigColsqRows * tm + 2 * wr + lh) * g.N + j] = sq;
    }
  }
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y) {
      const int j = j0 + 64 * wc + 32 * y + li;
      // C may be Cin (an in-place update): all 16 reads of the block precede its writes.
      float cin[16];
      if constexpr (EPI == BIG_AXPBY) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int i = i0 + 64 * wr + 32 * x + 8 * (r >> 2) + 4 * lh + (r & 3);
          cin[r] = (i < g.M && j < g.N) ? g.Cin[(int64_t)i * g.ldcin + j] : 0.f;
        }
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int i = i0 + 64 * wr + 32 * x + 8 * (r >> 2) + 4 * lh + (r & 3);
        if (i < g.M && j < g.N) {
          if constexpr (EPI == BIG_PARTIAL)
            g.partial[((int64_t)split * g.M + i) * g.N + j] = acc[x][y][r];
          else if constexpr (EPI == BIG_AXPBY)
            g.C[(int64_t)i * g.ldc + j] = g.alpha * acc[x][y][r] + g.beta * cin[r];
          else
            g.C[(int64_t)i * g.ldc + j] = g.alpha * acc[x][y][r];
        }
      }
    }
}

template <int P, int NW>
void launch_phase(int total, hipStream_t s, const GemmBatch &b, const int *gate) {
  LST_LAUNCH((gemm_kernel<P, NW>), dim3(total), dim3(64 * NW), 0, s, b, gate);
}

}  // namespace

GemmDesc gemm_desc(int M, int N, int K, const float *A, int64_t lda, int tA, const float *B,
                   int64_t ldb, int tB, float *C, int64_t ldc, float alpha, const float *Cin,
                   int64_t ldcin, float beta) {
  GemmDesc g{};
  g.M = M;
  g.N = N;
  g.K = K;
  g.K2 = 0;
  g.A = A;
  g.lda = lda;
  g.tA = tA;
  g.B = B;
  g.ldb = ldb;
  g.tB = tB;
  g.C = C;
  g.ldc = ldc;
  g.alpha = alpha;
  g.Cin = Cin;
  g.ldcin = ldcin;
  g.beta = beta;
  g.epi = EPI_NONE;
  g.splits = 1;
  g.kchunk = K;
  return g;
}

size_t gemm_plan_split(GemmDesc &g, int target_wgs, float *partial) {
  const int tiles = ((g.M + 31) / 32) * ((g.N + 31) / 32);
  int splits = (target_wgs + tiles - 1) / tiles;
  const int max_splits = (g.K + 255) / 256;  // at least 256 k per split
  if (splits > max_splits) splits = max_splits;
  if (splits < 2) {
    g.splits = 1;
    g.kchunk = g.K;
    return 0;
  }
  int chunk = (g.K + splits - 1) / splits;
  chunk = (chunk + 7) / 8 * 8;
  splits = (g.K + chunk - 1) / chunk;
  g.splits = splits;
  g.kchunk = chunk;
  g.partial = partial;
  return (size_t)splits * g.M * g.N;
}

int gemm_prepare(GemmBatch &b) {
  int total = 0;
  int kmax = 0;
  const int ts = b.t16 ? 16 : 32;
  for (int q = 0; q < b.n; ++q) {
    GemmDesc &g = b.d[q];
    g.tiles_m = (g.M + ts - 1) / ts;
    g.tiles_n = (g.N + ts - 1) / ts;
    g.tile_begin = total;
    if (g.M > 0 && g.N > 0) {
      total += g.tiles_m * g.tiles_n * (g.splits > 1 ? g.splits : 1);
      const int kk = g.splits > 1 ? g.kchunk : g.K + g.K2;
      if (kk > kmax) kmax = kk;
    }
  }
  // Empty descriptors (M or N == 0) own no tiles; give them tile_begin past the end.
  for (int q = 0; q < b.n; ++q)
    if (b.d[q].M <= 0 || b.d[q].N <= 0) b.d[q].tile_begin = total;
  b.total_tiles = total;
  b.wide = kmax >= 384 ? 1 : 0;  // waves per tile: enough to keep each wave's share of k short
  return total;
}

void gemm_enqueue(const GemmBatch &b, const int *gate, hipStream_t s, int phase) {
  const int total = b.total_tiles;
  if (total == 0) return;
  const bool wide = b.wide != 0;
  switch (phase) {
#define LST_GEMM_CASE(P)                          \
  case P:                                         \
    if (wide)                                     \
      launch_phase<P, 8>(total, s, b, gate); \
    else                                          \
      launch_phase<P, 4>(total, s, b, gate); \
    break;
    LST_GEMM_CASE(GEMM_CONTRACT)
    LST_GEMM_CASE(GEMM_ZGRAD)
    LST_GEMM_CASE(GEMM_MID)
    LST_GEMM_CASE(GEMM_UPDATE)
    LST_GEMM_CASE(GEMM_NAIVE_FWD)
    LST_GEMM_CASE(GEMM_NAIVE_GRAD)
    LST_GEMM_CASE(GEMM_NAIVE_UPDATE)
#undef LST_GEMM_CASE
    default:
      if (wide)
        launch_phase<GEMM_OTHER, 8>(total, s, b, gate);
      else
        launch_phase<GEMM_OTHER, 4>(total, s, b, gate);
  }
  for (int q = 0; q < b.n; ++q) {
    const GemmDesc &g = b.d[q];
    if (g.splits > 1 && g.M > 0 && g.N > 0) {
      const int64_t tot = (int64_t)g.M * g.N;
      int blocks = (int)((tot + 255) / 256);
      if (blocks > 2048) blocks = 2048;
      LST_LAUNCH(splitk_reduce_kernel, dim3(blocks), dim3(256), 0, s, g, gate);
    }
  }
}

void gemm_enqueue_plan(const GemmBatch &host, const GemmBatch *dev, const float *H,
                       float *gradH, float lr, const int *gate, hipStream_t s, int phase,
                       const int *pf_idx, int pf_K, const StepSync &sync) {
  const int total = host.total_tiles;
  if (total == 0) return;
  if (host.t16) {
    const int grid = (pf_idx && host.pf_m > 0) ? host.pf_base + host.pf_m : total;
    switch (phase) {
#define LST_PLAN16_CASE(P)                                                                     \
  case P:                                                                                      \
    LST_LAUNCH((gemm16_plan_kernel<P>), dim3(grid), dim3(256), 0, s, dev, H, gradH, lr, gate, \
               pf_idx, pf_K, sync);                                                             \
    break;
      LST_PLAN16_CASE(GEMM_CONTRACT)
      LST_PLAN16_CASE(GEMM_ZGRAD)
      LST_PLAN16_CASE(GEMM_MID)
      LST_PLAN16_CASE(GEMM_UPDATE)
#undef LST_PLAN16_CASE
      default:
        LST_LAUNCH((gemm16_plan_kernel<GEMM_OTHER>), dim3(grid), dim3(256), 0, s, dev, H, gradH,
                   lr, gate, pf_idx, pf_K, sync);
    }
    return;
  }
  const bool wide = host.wide != 0;
  switch (phase) {
#define LST_PLAN_CASE(P)                                                                       \
  case P:                                                                                      \
    if (wide)                                                                                  \
      LST_LAUNCH((gemm_plan_kernel<P, 8>), dim3(total), dim3(512), 0, s, dev, H, gradH, lr,     \
                 gate, sync);                                                                   \
    else                                                                                       \
      LST_LAUNCH((gemm_plan_kernel<P, 4>), dim3(total), dim3(256), 0, s, dev, H, gradH, lr,     \
                 gate, sync);                                                                   \
    break;
    LST_PLAN_CASE(GEMM_CONTRACT)
    LST_PLAN_CASE(GEMM_ZGRAD)
    LST_PLAN_CASE(GEMM_MID)
    LST_PLAN_CASE(GEMM_UPDATE)
#undef LST_PLAN_CASE
    default:
      if (wide)
        LST_LAUNCH((gemm_plan_kernel<GEMM_OTHER, 8>), dim3(total), dim3(512), 0, s, dev, H, gradH,
                   lr, gate, sync);
      else
        LST_LAUNCH((gemm_plan_kernel<GEMM_OTHER, 4>), dim3(total), dim3(256), 0, s, dev, H, gradH,
                   lr, gate, sync);
  }
}

bool gemm_enqueue_plan_scatter(const GemmBatch &host, const GemmBatch *dev, const float *H,
                               float *gradH, float lr, const int *gate, hipStream_t s, int n,
                               int K, int d, float slr, const int *idx, const float *dA,
                               const float *P, float *V, int64_t ldv) {
  if (host.wide || host.t16) return false;
  for (int i = 0; i < host.n; ++i)
    if (host.d[i].splits > 1) return false;
  LST_LAUNCH(update_scatter_kernel, dim3(host.total_tiles + n), dim3(256), 2 * n * sizeof(int), s,
             dev, host.total_tiles, H, gradH, lr, gate, n, K, d, slr, idx, dA, P, V, ldv);
  return true;
}

bool gemm_big_ok(const GemmDesc &g) {
  auto al = [](const void *p, int64_t ld) {
    return (reinterpret_cast<uintptr_t>(p) & 15) == 0 && (ld & 3) == 0;
  };
  // the index dimension of a k-major operand is read four at a time
  const bool dims = (!g.tA || (g.M & 3) == 0) && (!g.tB || (g.N & 3) == 0);
  return g.K2 == 0 && g.epi == EPI_NONE && dims && al(g.A, g.lda) && al(g.B, g.ldb) &&
         g.M >= 4 && g.N >= 4 && g.K >= 4;
}

size_t gemm_big_plan(GemmDesc &g, int target_wgs, size_t partial_floats, float *partial) {
  g.tiles_m = (g.M + kBigT - 1) / kBigT;
  g.tiles_n = (g.N + kBigT - 1) / kBigT;
  const int tiles = g.tiles_m * g.tiles_n;
  int splits = (target_wgs + tiles - 1) / tiles;
  const int by_k = (g.K + 1023) / 1024;  // at least 1024 k per split
  if (splits > by_k) splits = by_k;
  if (partial_floats / ((size_t)g.M * g.N) < (size_t)splits)
    splits = (int)(partial_floats / ((size_t)g.M * g.N));
  if (splits < 2 || !partial) {
    g.splits = 1;
    g.kchunk = g.K;
    g.partial = nullptr;
    return 0;
  }
  int chunk = (g.K + splits - 1) / splits;
  chunk = (chunk + kBigK - 1) / kBigK * kBigK;
  g.splits = (g.K + chunk - 1) / chunk;
  g.kchunk = chunk;
  g.partial = partial;
  return (size_t)g.splits * g.M * g.N;
}

template <int P, bool TA, bool TB>
void big_launch(const GemmDesc &g, const int *gate, hipStream_t s, dim3 grid) {
  if (g.splits > 1)
    LST_LAUNCH((gemm_big_kernel<P, TA, TB, BIG_PARTIAL>), grid, dim3(256), 0, s, g, gate);
  else if (g.Cin)
    LST_LAUNCH((gemm_big_kernel<P, TA, TB, BIG_AXPBY>), grid, dim3(256), 0, s, g, gate);
  else
    LST_LAUNCH((gemm_big_kernel<P, TA, TB, BIG_STORE>), grid, dim3(256), 0, s, g, gate);
}

hipError_t gemm_big_launch(GemmDesc g, const int *gate, hipStream_t s, int phase) {
  const int total = g.tiles_m * g.tiles_n * g.splits;
  if (total == 0) return hipSuccess;
  if (g.colsq && g.splits > 1) return hipErrorInvalidValue;  // column sums need whole k
  const dim3 grid(total);
  if (phase == GEMM_NAIVE_FWD && !g.tA && !g.tB)
    big_launch<GEMM_NAIVE_FWD, false, false>(g, gate, s, grid);
  else if (phase == GEMM_NAIVE_GRAD && g.tA && g.tB)
    big_launch<GEMM_NAIVE_GRAD, true, true>(g, gate, s, grid);
  else if (phase == GEMM_NAIVE_UPDATE && !g.tA && g.tB)
    big_launch<GEMM_NAIVE_UPDATE, false, true>(g, gate, s, grid);
  else if (g.tA && g.tB)
    big_launch<GEMM_OTHER, true, true>(g, gate, s, grid);
  else if (g.tA)
    big_launch<GEMM_OTHER, true, false>(g, gate, s, grid);
  else if (g.tB)
    big_launch<GEMM_OTHER, false, true>(g, gate, s, grid);
  else
    big_launch<GEMM_OTHER, false, false>(g, gate, s, grid);
  if (g.splits > 1) {
    const int64_t tot = (int64_t)g.M * g.N;
    int blocks = (int)((tot + 255) / 256);
    if (blocks > 2048) blocks = 2048;
    LST_LAUNCH(splitk_reduce_kernel, dim3(blocks), dim3(256), 0, s, g, gate);
  }
  return hipGetLastError();
}

hipError_t gemm_launch(GemmBatch &b, const int *gate, hipStream_t s, int phase) {
  gemm_prepare(b);
  gemm_enqueue(b, gate, s, phase);
  return hipGetLastError();
}

}  // namespace lst
