// Batched fp32 GEMM on the CDNA4 matrix cores (v_mfma_f32_32x32x2_f32) outside
// the step's own launches: the initial Q = V^T V, materialize_W = V U, the
// section 5 products, and the naive path's D x d products (128 x 128 tiles).  A
// workgroup owns a 32 x 32 output tile (gemm_tiles.h); its NW wavefronts split the
// k range and their accumulators are summed through LDS in a fixed order, so
// results do not depend on scheduling.
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
#include <algorithm>
#include "gemm_tiles.h"

namespace lst {

namespace {

// PHASE only names the instantiation, so profilers report each step phase separately.
template <int PHASE, int NW>
__global__ __launch_bounds__(64 * NW, 12 / NW) void gemm_kernel(const GemmBatch bt, const int *__restrict__ gate) {
  gemm_body<NW>(bt, bt, nullptr, nullptr, 1.f, gate, blockIdx.x);
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
  // (k arithmetic in 64 bits: K may be D, up to 2^31 - 1)
  const int max_splits = (int)(((int64_t)g.K + 255) / 256);  // at least 256 k per split
  if (splits > max_splits) splits = max_splits;
  if (splits < 2) {
    g.splits = 1;
    g.kchunk = g.K;
    return 0;
  }
  int chunk = (int)(((int64_t)g.K + splits - 1) / splits);
  chunk = (chunk + 7) / 8 * 8;
  splits = (int)(((int64_t)g.K + chunk - 1) / chunk);
  g.splits = splits;
  g.kchunk = chunk;
  g.partial = partial;
  return (size_t)splits * g.M * g.N;
}

int gemm_prepare(GemmBatch &b, int ts) {
  int total = 0;
  int kmax = 0;
  b.tile = ts;
  for (int q = 0; q < b.n; ++q) {
    GemmDesc &g = b.d[q];
    g.tiles_m = (g.M + ts - 1) / ts;
    g.tiles_n = (g.N + ts - 1) / ts;
    g.tile_begin = total;
    if (g.M > 0 && g.N > 0) {
      total += g.tiles_m * g.tiles_n * (g.splits > 1 ? g.splits : 1);
      const int64_t kk = g.splits > 1 ? (int64_t)g.kchunk : (int64_t)g.K + g.K2;
      if (kk > kmax) kmax = (int)std::min<int64_t>(kk, 1 << 30);
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
