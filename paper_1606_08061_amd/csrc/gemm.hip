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

// One wavefront's share of the k range [kbeg, kend): full blocks of 8 with
// index wave, wave + NW, ...; the ragged tail block goes to wave NW-1.
template <int NW, int AM, int BM>
__device__ __forceinline__ void kloop(floatx16 &acc, const float *A, int64_t asi, int64_t ask,
                                      const float *B, int64_t bsi, int64_t bsk, int ia, int jb,
                                      int kbeg, int kend, int wave, int lh) {
  const int nfull = (kend - kbeg) >> 3;
  const int nw = nfull > wave ? (nfull - wave + NW - 1) / NW : 0;
  if (nw > 0) {
    auto kof = [&](int s) { return kbeg + 8 * (wave + NW * min(s, nw - 1)) + 4 * lh; };
    float a[kStage][4], b[kStage][4];
#pragma unroll
    for (int u = 0; u < kStage; ++u) {
      ld4<AM>(A, asi, ask, ia, kof(u), a[u]);
      ld4<BM>(B, bsi, bsk, jb, kof(u), b[u]);
    }
    for (int s0 = 0; s0 < nw; s0 += kStage) {
      float an[kStage][4], bn[kStage][4];
#pragma unroll
      for (int u = 0; u < kStage; ++u) {
        ld4<AM>(A, asi, ask, ia, kof(s0 + kStage + u), an[u]);
        ld4<BM>(B, bsi, bsk, jb, kof(s0 + kStage + u), bn[u]);
      }
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
  if (((kend - kbeg) & 7) && wave == NW - 1) {
    const int k0 = kbeg + 8 * nfull + 4 * lh;
    float a[4], b[4];
    ld4_tail(A, asi, ask, ia, k0, kend, a);
    ld4_tail(B, bsi, bsk, jb, k0, kend, b);
#pragma unroll
    for (int s = 0; s < 4; ++s) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[s], b[s], acc, 0, 0, 0);
  }
}

__device__ __forceinline__ bool vec_ok(const float *p, int64_t ld) {
  return ((reinterpret_cast<uintptr_t>(p) & 15) == 0) && ((ld & 3) == 0);
}

// opA(i,k): tA = 0 -> A[i*lda + k] (index stride lda, k stride 1); tA = 1 -> A[k*lda + i].
// opB(k,j): tB = 0 -> B[j*ldb + k];                                 tB = 1 -> B[k*ldb + j].
template <int NW>
__device__ __forceinline__ void segment(floatx16 &acc, const float *A, int64_t lda, int tA,
                                        const float *B, int64_t ldb, int tB, int ia, int jb,
                                        int kbeg, int kend, int wave, int lh) {
  const int64_t asi = tA ? 1 : lda, ask = tA ? lda : 1;
  const int64_t bsi = tB ? 1 : ldb, bsk = tB ? ldb : 1;
  const bool av = !tA && vec_ok(A, lda);
  const bool bv = !tB && vec_ok(B, ldb);
  if (av && bv)
    kloop<NW, VEC, VEC>(acc, A, asi, ask, B, bsi, bsk, ia, jb, kbeg, kend, wave, lh);
  else if (av)
    kloop<NW, VEC, STRIDED>(acc, A, asi, ask, B, bsi, bsk, ia, jb, kbeg, kend, wave, lh);
  else if (bv)
    kloop<NW, STRIDED, VEC>(acc, A, asi, ask, B, bsi, bsk, ia, jb, kbeg, kend, wave, lh);
  else
    kloop<NW, STRIDED, STRIDED>(acc, A, asi, ask, B, bsi, bsk, ia, jb, kbeg, kend, wave, lh);
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
    segment<NW>(acc, g.A, g.lda, g.tA, g.B, g.ldb, g.tB, ia, jb, kbeg, kend, wave, lh);
  } else {
    segment<NW>(acc, g.A, g.lda, g.tA, g.B, g.ldb, g.tB, ia, jb, 0, g.K, wave, lh);
    if (g.K2 > 0) segment<NW>(acc, g.A2, g.lda2, g.tA, g.B2, g.ldb2, g.tB, ia, jb, 0, g.K2, wave, lh);
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
__global__ __launch_bounds__(64 * NW) void gemm_kernel(const GemmBatch bt, const int *__restrict__ gate) {
  gemm_body<NW>(bt, nullptr, nullptr, 1.f, gate);
}

// The batch read from device memory (a plan), with the step's H, grad_H and lr.
template <int PHASE, int NW>
__global__ __launch_bounds__(64 * NW) void gemm_plan_kernel(const GemmBatch *__restrict__ bt,
                                                            const float *H, float *gH, float lr,
                                                            const int *__restrict__ gate) {
  gemm_body<NW>(*bt, H, gH, lr, gate);
}

__global__ __launch_bounds__(256) void splitk_reduce_kernel(const GemmDesc g, const int *__restrict__ gate) {
  if (gate && *gate != 0) return;
  const int64_t total = (int64_t)g.M * g.N;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    float v = 0.f;
    for (int s = 0; s < g.splits; ++s) v += g.partial[(int64_t)s * total + e];
    const int i = (int)(e / g.N), j = (int)(e % g.N);
    finish(g, i, j, v);
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
template <int PHASE>
__global__ __launch_bounds__(256) void gemm16_plan_kernel(const GemmBatch *__restrict__ bt,
                                                           const float *H, float *gH, float lr,
                                                           const int *__restrict__ gate,
                                                           const int *__restrict__ pf_idx,
                                                           int pf_K) {
  if ((int)blockIdx.x >= bt->total_tiles) {
    // Prefetch workgroup: the target rows of example j (indices outside [0, D) skipped).
    const int j = (int)blockIdx.x - bt->pf_base;
    if (j < 0 || j >= bt->pf_m) return;
    float sink = 0.f;
    for (int k = 0; k < pf_K; ++k) {
      const int r = pf_idx[(int64_t)j * pf_K + k];
      if (r < 0 || (int64_t)r >= bt->pf_D) continue;
      const float *row = bt->pf_V + (int64_t)r * bt->pf_ldv;
      for (int c = threadIdx.x; c < bt->pf_d; c += 256) sink += row[c];
    }
    asm volatile("" ::"v"(sink));
    return;
  }
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
                       const int *pf_idx, int pf_K) {
  const int total = host.total_tiles;
  if (total == 0) return;
  if (host.t16) {
    const int grid = (pf_idx && host.pf_m > 0) ? host.pf_base + host.pf_m : total;
    switch (phase) {
#define LST_PLAN16_CASE(P)                                                                     \
  case P:                                                                                      \
    LST_LAUNCH((gemm16_plan_kernel<P>), dim3(grid), dim3(256), 0, s, dev, H, gradH, lr, gate, \
               pf_idx, pf_K);                                                                  \
    break;
      LST_PLAN16_CASE(GEMM_CONTRACT)
      LST_PLAN16_CASE(GEMM_ZGRAD)
      LST_PLAN16_CASE(GEMM_MID)
      LST_PLAN16_CASE(GEMM_UPDATE)
#undef LST_PLAN16_CASE
      default:
        LST_LAUNCH((gemm16_plan_kernel<GEMM_OTHER>), dim3(grid), dim3(256), 0, s, dev, H, gradH,
                   lr, gate, pf_idx, pf_K);
    }
    return;
  }
  const bool wide = host.wide != 0;
  switch (phase) {
#define LST_PLAN_CASE(P)                                                                       \
  case P:                                                                                      \
    if (wide)                                                                                  \
      LST_LAUNCH((gemm_plan_kernel<P, 8>), dim3(total), dim3(512), 0, s, dev, H, gradH, lr,     \
                 gate);                                                                        \
    else                                                                                       \
      LST_LAUNCH((gemm_plan_kernel<P, 4>), dim3(total), dim3(256), 0, s, dev, H, gradH, lr,     \
                 gate);                                                                        \
    break;
    LST_PLAN_CASE(GEMM_CONTRACT)
    LST_PLAN_CASE(GEMM_ZGRAD)
    LST_PLAN_CASE(GEMM_MID)
    LST_PLAN_CASE(GEMM_UPDATE)
#undef LST_PLAN_CASE
    default:
      if (wide)
        LST_LAUNCH((gemm_plan_kernel<GEMM_OTHER, 8>), dim3(total), dim3(512), 0, s, dev, H, gradH,
                   lr, gate);
      else
        LST_LAUNCH((gemm_plan_kernel<GEMM_OTHER, 4>), dim3(total), dim3(256), 0, s, dev, H, gradH,
                   lr, gate);
  }
}

hipError_t gemm_launch(GemmBatch &b, const int *gate, hipStream_t s, int phase) {
  gemm_prepare(b);
  gemm_enqueue(b, gate, s, phase);
  return hipGetLastError();
}

}  // namespace lst
