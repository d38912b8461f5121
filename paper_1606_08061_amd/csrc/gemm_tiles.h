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


// ---------------------------------------------------------------------------
// 64 x 64 tiles staged through LDS (the step's products at large shapes).
//
// The workgroup's 256 threads load each 16-wide k step of the two 64-index operand
// panels once: every row's 64 bytes by 4 consecutive lanes when k is contiguous, every
// k row's 256 bytes by 16 lanes when the index is.  The panels are stored k-major in
// LDS ([k][index], padded rows) and wave (wr, wc) runs the 32 x 32 quadrant (wr, wc) of
// the tile over the whole k range from there, 8 MFMAs a k step into two accumulators
// (even and odd k pairs).  Against the 32 x 32 tiles above, whose waves read 32-byte
// pieces of each row straight from memory, an operand element crosses the L2 once per
// 64 outputs instead of once per 32.
// LDS is double buffered; the loads of the next kT64P steps are in flight in registers
// while a step runs on the matrix cores.
// ---------------------------------------------------------------------------
constexpr int kT64 = 64, kT64K = 16, kT64Ld = kT64 + 4;
// per thread and k step: kT64U 16-byte pieces of each operand; k contiguous: kT64Lpr
// lanes a row, kT64Rpu rows a piece
constexpr int kT64U = kT64K / 16, kT64Lpr = kT64K / 4, kT64Rpu = 256 / kT64Lpr;
constexpr int kT64P = 2;  // k steps in flight in registers (even: LDS buffer = step % 2)
static_assert(kT64P % 2 == 0, "the LDS buffer of a step is its register slot's parity");

// One operand of one k segment: element (index i, k) at p[i ld + k] (k contiguous) or
// p[k ld + i] (index contiguous); n indices, k in [0, kend).
struct Panel {
  const float *p;
  int64_t ld;
  int n, kend;
};

// Load modes: KCV: k contiguous, 16-byte loads (aligned p, ld and kend multiples of 4);
// IXV: index contiguous, 16-byte loads (aligned p, ld and n multiples of 4); GEN: either
// layout (kc), scalar loads.
enum : int { KCV = 0, IXV = 1, GEN = 2 };

template <int MODE>
__device__ __forceinline__ void p64_load(const Panel &q, bool kc, int idx0, int k0,
                                         float4 (&v)[kT64U]) {
  const int t = threadIdx.x;
#pragma unroll
  for (int u = 0; u < kT64U; ++u) {
    if constexpr (MODE == IXV) {  // thread t: k row t / 16 + 16 u, indices 4 (t % 16) ..
      const int k = k0 + (t >> 4) + 16 * u;
      const float *row = q.p + (int64_t)min(k, q.kend - 1) * q.ld;
      const float4 x = *reinterpret_cast<const float4 *>(row + min(idx0 + (t & 15) * 4, q.n - 4));
      v[u] = k < q.kend ? x : make_float4(0.f, 0.f, 0.f, 0.f);
    } else {  // thread t: index t / kT64Lpr + kT64Rpu u, k 4 (t % kT64Lpr) ..
      const int i = min(idx0 + t / kT64Lpr + kT64Rpu * u, q.n - 1);
      const int k = k0 + (t % kT64Lpr) * 4;
      if constexpr (MODE == KCV) {
        const float4 x =
            *reinterpret_cast<const float4 *>(q.p + (int64_t)i * q.ld + min(k, q.kend - 4));
        v[u] = k < q.kend ? x : make_float4(0.f, 0.f, 0.f, 0.f);
      } else {
        const int64_t si = kc ? q.ld : 1, sk = kc ? 1 : q.ld;
        float e[4];
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          const float x = q.p[(int64_t)i * si + (int64_t)min(k + s, q.kend - 1) * sk];
          e[s] = k + s < q.kend ? x : 0.f;
        }
        v[u] = make_float4(e[0], e[1], e[2], e[3]);
      }
    }
  }
}

template <int MODE>
__device__ __forceinline__ void p64_store(float (*lds)[kT64Ld], const float4 (&v)[kT64U]) {
  const int t = threadIdx.x;
#pragma unroll
  for (int u = 0; u < kT64U; ++u) {
    if constexpr (MODE == IXV) {
      *reinterpret_cast<float4 *>(&lds[(t >> 4) + 16 * u][(t & 15) * 4]) = v[u];
    } else {
      const int i = t / kT64Lpr + kT64Rpu * u, k = (t % kT64Lpr) * 4;
      lds[k][i] = v[u].x;
      lds[k + 1][i] = v[u].y;
      lds[k + 2][i] = v[u].z;
      lds[k + 3][i] = v[u].w;
    }
  }
}

__device__ __forceinline__ void p64_mfma(float (*As)[kT64Ld], float (*Bs)[kT64Ld],
                                         floatx16 (&acc)[2], int ai, int bj, int lh) {
#pragma unroll
  for (int kk = 0; kk < kT64K; kk += 2) {
    const float a = As[kk + lh][ai];
    const float b = Bs[kk + lh][bj];
    acc[(kk >> 1) & 1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc[(kk >> 1) & 1], 0, 0, 0);
  }
}

// Extra operand terms of a k step (one k segment): NA terms of opA in its layout (the
// first from the panel, the others from a[]), with ATR one more read transposed
// (element (i, k) at at[k lda + i], in the k-contiguous thread mapping), and NB terms
// of opB; each operand's terms are combined with their weights as it is stored to LDS.
template <int NA, bool ATR, int NB>
struct Terms {
  const float *a[NA > 1 ? NA - 1 : 1];
  const float *b[NB > 1 ? NB - 1 : 1];
  const float *at;
  float wa[NA], wb[NB], wt;
};

template <int MODE, int N, bool TR>
__device__ __forceinline__ void p64_store_terms(float (*lds)[kT64Ld], const float4 (&v)[N][kT64U],
                                                const float4 (&vt)[kT64U], const float (&w)[N],
                                                float wt) {
  if constexpr (N == 1 && !TR) {
    p64_store<MODE>(lds, v[0]);
  } else {
    float4 c[kT64U];
#pragma unroll
    for (int u = 0; u < kT64U; ++u) {
      c[u] = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int t = 0; t < N + (TR ? 1 : 0); ++t) {
        const float4 x = t < N ? v[t < N ? t : 0][u] : vt[u];
        const float y = t < N ? w[t < N ? t : 0] : wt;
        c[u].x = fmaf(y, x.x, c[u].x);
        c[u].y = fmaf(y, x.y, c[u].y);
        c[u].z = fmaf(y, x.z, c[u].z);
        c[u].w = fmaf(y, x.w, c[u].w);
      }
    }
    p64_store<MODE>(lds, c);
  }
}

// k steps 0 .. ns1 - 1 run over segment 0 (pa0, pb0), the rest over segment 1.
template <int AM, int BM, int NA, bool ATR, int NB>
__device__ __forceinline__ void k64(const Panel &pa0, const Panel &pb0, const Panel &pa1,
                                    const Panel &pb1, const Terms<NA, ATR, NB> &tm, bool akc,
                                    bool bkc, int ns1, int ns, int i0, int j0,
                                    float (*As)[kT64K][kT64Ld], float (*Bs)[kT64K][kT64Ld],
                                    floatx16 (&acc)[2], int ai, int bj, int lh) {
  auto load = [&](int st, float4(&ra)[NA][kT64U], float4(&rt)[kT64U], float4(&rb)[NB][kT64U]) {
    const bool s1 = st >= ns1;
    const int k0 = (s1 ? st - ns1 : st) * kT64K;
    const Panel &A = s1 ? pa1 : pa0, &B = s1 ? pb1 : pb0;
    p64_load<AM>(A, akc, i0, k0, ra[0]);
#pragma unroll
    for (int t = 1; t < NA; ++t) {
      Panel q = A;
      q.p = tm.a[t - 1];
      p64_load<AM>(q, akc, i0, k0, ra[t]);
    }
    if constexpr (ATR) {
      Panel q = A;
      q.p = tm.at;
      p64_load<GEN>(q, false, i0, k0, rt);
    }
    p64_load<BM>(B, bkc, j0, k0, rb[0]);
#pragma unroll
    for (int t = 1; t < NB; ++t) {
      Panel q = B;
      q.p = tm.b[t - 1];
      p64_load<BM>(q, bkc, j0, k0, rb[t]);
    }
  };
  constexpr int AS = AM == IXV ? IXV : KCV, BS = BM == IXV ? IXV : KCV;  // LDS store layout
  // Register slot u % kT64P holds step u from its load until its store to LDS buffer
  // u % 2, one step before its products; the slot then takes step u + kT64P.
  float4 ra[kT64P][NA][kT64U], rt[kT64P][kT64U], rb[kT64P][NB][kT64U];
  auto store = [&](int buf, int slot) {
    p64_store_terms<AS, NA, ATR>(As[buf], ra[slot], rt[slot], tm.wa, tm.wt);
    const float4 none[kT64U] = {};
    p64_store_terms<BS, NB, false>(Bs[buf], rb[slot], none, tm.wb, 0.f);
  };
#pragma unroll
  for (int u = 0; u < kT64P; ++u)
    if (u < ns) load(u, ra[u], rt[u], rb[u]);
  if (ns > 0) store(0, 0);
  __syncthreads();
  for (int st = 0; st < ns; st += kT64P) {
#pragma unroll
    for (int u = 0; u < kT64P; ++u) {
      const int s = st + u;
      if (s < ns) {
        if (s + kT64P < ns) load(s + kT64P, ra[u], rt[u], rb[u]);
        p64_mfma(As[u & 1], Bs[u & 1], acc, ai, bj, lh);
        if (s + 1 < ns) store((u + 1) & 1, (u + 1) % kT64P);
        __syncthreads();
      }
    }
  }
}

__device__ __forceinline__ bool p64_vec(const float *p, int64_t ld, int ext) {
  return ((reinterpret_cast<uintptr_t>(p) & 15) == 0) && ((ld & 3) == 0) && ((ext & 3) == 0) &&
         ext >= 4;
}

// A batch on 64 x 64 tiles (GemmBatch::tile == 64): C = alpha opA opB + beta C_in, with
// the second k segment (A2, B2, K2) when K2 > 0, and the grad_H epilogue (C2 = 2 rs E
// + C, rs = 1 when null; C may then be null).  No split k (the host plans none).  Tiles
// of one product run column by column, so that the tiles one XCD takes share B's
// panels.  TERMS: the batch may also hold operand terms, addends and alternatives
// (GemmDesc::nat ... alt1; a separate instantiation, for the registers they take).
// wg: the workgroup's index in the batch's section (gemm_section(hd, 64) of them);
// cert: the certificate flag that selects alternatives (null: certified).
template <bool TERMS>
__device__ __forceinline__ void gemm_body64(const GemmBatch &bt, const GemmHdr &hd,
                                            const float *H, float *gH, float lr,
                                            const int *__restrict__ gate, int wg,
                                            const int *__restrict__ cert = nullptr) {
  const int tile = gemm_tile64(hd, wg);
  if (tile < 0) return;
  const int closed = gate ? *gate : 0;
  int di = 0;
#pragma unroll
  for (int q = 1; q < kMaxBatch; ++q)
    if (q < hd.n && tile >= hdr_begin(hd, q)) di = q;
  const int local = tile - hd.tile_begin[di];
  GemmDesc g = bt.d[di];
  const int tn = local / g.tiles_m, tm = local - tn * g.tiles_m;
  if (TERMS && g.alt1 > 0 && cert && *cert == 0) g = bt.d[g.alt1 - 1];  // same shape
  g.A = resolve(g.A, H, gH);
  g.B = resolve(g.B, H, gH);
  g.A2 = resolve(g.A2, H, gH);
  g.B2 = resolve(g.B2, H, gH);
  g.Cin = resolve(g.Cin, H, gH);
  g.C2 = const_cast<float *>(resolve(g.C2, H, gH));
  if (g.lr_scaled == 1) {
    g.alpha *= lr * lr;
    g.beta *= lr;
  } else if (g.lr_scaled == 2) {
    g.alpha *= lr;
  }
  const bool epi = g.epi == EPI_GRADH;
  const int i0 = tm * kT64, j0 = tn * kT64;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int li = lane & 31, lh = lane >> 5;
  const int ai = 32 * (wave >> 1) + li, bj = 32 * (wave & 1) + li;

  // The epilogue operand (E with the grad_H epilogue, else C_in) before the k loop, so
  // that its latency overlaps it; lane (li, lh) of the wave holds rows
  // 8 (r / 4) + 4 lh + r % 4 of the quadrant, column li.
  const int ib = i0 + 32 * (wave >> 1) + 4 * lh;
  const int j = j0 + bj, jc = min(j, g.N - 1);
  const float *pre = epi ? g.E : g.Cin;
  const int64_t ldpre = epi ? g.lde : g.ldcin;
  float pv[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int i = min(ib + 8 * (r >> 2) + (r & 3), g.M - 1);
    pv[r] = pre ? pre[(int64_t)i * ldpre + jc] : 0.f;
  }

  const bool akc = g.tA == 0, bkc = g.tB == 0;
  const Panel pa0{g.A, g.lda, g.M, g.K}, pb0{g.B, g.ldb, g.N, g.K};
  const Panel pa1{g.K2 > 0 ? g.A2 : g.A, g.K2 > 0 ? g.lda2 : g.lda, g.M, g.K2};
  const Panel pb1{g.K2 > 0 ? g.B2 : g.B, g.K2 > 0 ? g.ldb2 : g.ldb, g.N, g.K2};
  const int ns1 = (g.K + kT64K - 1) / kT64K;
  const int ns = ns1 + (g.K2 + kT64K - 1) / kT64K;
  auto vec = [&](const Panel &p0, const Panel &p1, bool kc) {
    const int e0 = kc ? p0.kend : p0.n, e1 = kc ? p1.kend : p1.n;
    return p64_vec(p0.p, p0.ld, e0) && (g.K2 == 0 || p64_vec(p1.p, p1.ld, e1));
  };
  bool av = vec(pa0, pa1, akc), bv = vec(pb0, pb1, bkc);

  floatx16 acc[2];
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[x][r] = 0.f;
  // one LDS allocation for every load mode (the k loop's instantiations share it)
  __shared__ float As[2][kT64K][kT64Ld];
  __shared__ float Bs[2][kT64K][kT64Ld];
#define LST_K64(AM, BM, NA, ATR, NB, TM)                                                       \
  k64<AM, BM, NA, ATR, NB>(pa0, pb0, pa1, pb1, TM, akc, bkc, ns1, ns, i0, j0, As, Bs, acc, ai, \
                           bj, lh)
  int nadd = 0;
  bool done = false;
  if constexpr (TERMS) {
    nadd = g.nadd;
    if (g.nat > 1 || g.Atr) {  // Zq: M assembled from its terms as it is staged
      Terms<3, true, 1> t3{};
#pragma unroll
      for (int t = 0; t < 3; ++t) {
        t3.wa[t] = t < g.nat ? g.aw[t] : 0.f;
        if (t > 0) {
          t3.a[t - 1] = t < g.nat ? g.At[t - 1] : g.A;
          av = av && p64_vec(t3.a[t - 1], g.lda, g.K);
        }
      }
      t3.at = g.Atr ? g.Atr : g.A;
      t3.wt = g.Atr ? g.awt : 0.f;
      t3.wb[0] = 1.f;
      if (av && bv && akc && !bkc)
        LST_K64(KCV, IXV, 3, true, 1, t3);
      else
        LST_K64(GEN, GEN, 3, true, 1, t3);
      done = true;
    } else if (g.nbt > 1) {  // R X: the B terms combined as they are staged
      Terms<1, false, 4> t4{};
      t4.wa[0] = 1.f;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        t4.wb[t] = t < g.nbt ? g.coef[g.bcoef[t]] : 0.f;
        if (t > 0) {
          t4.b[t - 1] = t < g.nbt ? g.Bt[t - 1] : g.B;
          bv = bv && p64_vec(t4.b[t - 1], g.ldb, bkc ? g.K : g.N);
        }
      }
      if (av && bv && akc && !bkc)
        LST_K64(KCV, IXV, 1, false, 4, t4);
      else
        LST_K64(GEN, GEN, 1, false, 4, t4);
      done = true;
    }
  }
  if (!done) {
    const Terms<1, false, 1> t1{};
    if (av && bv) {
      if (akc && bkc)
        LST_K64(KCV, KCV, 1, false, 1, t1);
      else if (akc)
        LST_K64(KCV, IXV, 1, false, 1, t1);
      else if (bkc)
        LST_K64(IXV, KCV, 1, false, 1, t1);
      else
        LST_K64(IXV, IXV, 1, false, 1, t1);
    } else {
      LST_K64(GEN, GEN, 1, false, 1, t1);
    }
  }
#undef LST_K64
  if (closed || j >= g.N) return;  // after the k loop's last barrier
  float adw[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) adw[t] = t < nadd ? g.coef[g.acoef[t]] : 0.f;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int i = ib + 8 * (r >> 2) + (r & 3);
    if (i < g.M) {
      float v = acc[0][r] + acc[1][r];
#pragma unroll
      for (int t = 0; t < 4; ++t)
        if (t < nadd) v = fmaf(adw[t], g.addp[t][(int64_t)i * g.ldadd + j], v);
      float out = g.alpha * v;
      if (g.Cin) out += g.beta * (epi ? g.Cin[(int64_t)i * g.ldcin + j] : pv[r]);
      if (g.C) g.C[(int64_t)i * g.ldc + j] = out;
      if (epi) g.C2[(int64_t)i * g.ldc2 + j] = 2.f * (g.rs ? g.rs[i] : 1.f) * pv[r] + out;
    }
  }
}

}  // namespace

}  // namespace lst
