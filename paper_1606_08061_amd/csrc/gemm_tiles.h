// The 32 x 32-tile fp32 GEMM body on the CDNA4 matrix cores (v_mfma_f32_32x32x2_f32),
// shared by the batched GEMM launches and by the state-update launches of the step
// (device code of liblst; not part of the C ABI).
//
// A workgroup owns a 32 x 32 output tile; its NW wavefronts split the k range and
// their accumulators are summed through LDS in a fixed order, so results do not
// depend on scheduling.
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
// the ragged end of the k range is masked.  Operands are fetched KS k-blocks
// ahead of the matrix cores (kStage unless a launch needs fewer registers).
#pragma once

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

// One wavefront's share of the k blocks of 8: blocks wave, wave + NW, ... of
// the first segment (k in [kbeg, kbeg + len1)) followed by the second (k in
// [0, len2) of A2, B2), so that the loads of both are in flight together.  The
// last block of a segment may be ragged (masked loads).
template <int NW, int AM, int BM, int KS>
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
  float a[KS][4], b[KS][4];
#pragma unroll
  for (int u = 0; u < KS; ++u) load(u, a[u], b[u]);
  for (int s0 = 0; s0 < nw; s0 += KS) {
    float an[KS][4], bn[KS][4];
#pragma unroll
    for (int u = 0; u < KS; ++u)
      if (s0 + KS + u < nw) load(s0 + KS + u, an[u], bn[u]);
#pragma unroll
    for (int u = 0; u < KS; ++u) {
      if (s0 + u < nw) {
#pragma unroll
        for (int s = 0; s < 4; ++s)
          acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[u][s], b[u][s], acc, 0, 0, 0);
      }
    }
#pragma unroll
    for (int u = 0; u < KS; ++u)
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
template <int NW, int KS>
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
  kloop<NW, AMODE, BMODE, KS>(acc, A, asi, ask, B, bsi, bsk, kend - kbeg, A2, asi2, ask2, B2, bsi2, \
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

// hd: the batch's tile ranges (the batch itself, or a GemmHdr passed by value).
template <int NW, int KS = kStage, class Hd>
__device__ __forceinline__ void gemm_body(const GemmBatch &bt, const Hd &hd, const float *H,
                                          float *gH, float lr, const int *__restrict__ gate,
                                          int wg) {
  // The gate only suppresses writes, so its load is waited for at the end.
  const int closed = gate ? *gate : 0;
  const int tile = xcd_tile(wg, hd.total_tiles);
  int di = 0;
#pragma unroll
  for (int q = 1; q < kMaxBatch; ++q)
    if (q < hd.n && tile >= hdr_begin(hd, q)) di = q;
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
    segment<NW, KS>(acc, g.A, g.lda, g.tA, g.B, g.ldb, g.tB, nullptr, 0, nullptr, 0, 0, ia, jb, kbeg,
                kend, wave, lh);
  } else {
    segment<NW, KS>(acc, g.A, g.lda, g.tA, g.B, g.ldb, g.tB, g.A2, g.lda2, g.B2, g.ldb2, g.K2, ia, jb,
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

}  // namespace

}  // namespace lst
