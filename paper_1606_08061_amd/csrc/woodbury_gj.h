// Blocked Gauss-Jordan inverse of the m x m Woodbury matrix on one workgroup
// (device code shared by the HIP sources of liblst; not part of the C ABI).
#pragma once

#include "lst_internal.h"

namespace lst {

namespace {

// ---------------------------------------------------------------------------
// Blocked Gauss-Jordan inverse on the matrix cores.
//
// The mp x mp matrix (mp = 32 NBK >= m, padded with the identity) lives in
// MFMA accumulator registers as NBK x NBK tiles of 32 x 32, each tile column
// held by one column wavefront (acc[i] = tile (i, c); at most three of them,
// so one holds two columns when NBK = 4), and one more wavefront forms and
// inverts the pivot blocks (see gj_workers).  In accumulator layout lane
// l = j + 32 h holds column j of a tile and register r holds row acc_row(h, r).
// Block step kb with pivot block
// P = A_kb,kb^{-1} is, in place,
//   A_kb,j <- P A_kb,j,   A_ij <- A_ij - A_i,kb (P A_kb,j),
//   A_i,kb <- -A_i,kb P,  A_kb,kb <- P                          (i, j != kb),
// the block form of the scalar step below; after NBK block steps the tiles hold
// the inverse.  The products run on v_mfma_f32_32x32x2f32 with the k index of
// instruction r taken as acc_row(h, r) in lane-half h, so a tile held in
// registers is directly the B operand of a product: a column owner needs from
// LDS only P and the column panel -A_i,kb.  Since every pivot block is a Schur
// complement of C, the pivots met inside the 32 x 32 inversions are exactly
// those of unblocked elimination: all are positive iff C is positive definite.
// ---------------------------------------------------------------------------
typedef float floatx16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ int acc_row(int h, int r) { return 4 * h + (r & 3) + 8 * (r >> 2); }

constexpr int kTileLd = 36;  // LDS row stride (floats) of a staged 32 x 32 tile: 16-byte rows
constexpr int kTileSz = 32 * kTileLd;

// One scalar Gauss-Jordan step on pivot K (p = A_KK) of a 16 x 16 block:
//   A' = A - (f - e_K) g^T,   f = A_:K (column K),
//   g_j = A_Kj / p (j != K), g_K = 1 + 1/p,
// i.e. A'_Kj = A_Kj / p, A'_iK = -A_iK / p, A'_KK = 1 / p, A'_ij = A_ij - A_iK A_Kj / p.
// Since A_KK = p, g_j = (A_Kj + [j = K]) / p needs no separate case.  A lane
// applies -f g_c to its rows with the column-K value taken straight from the
// lane of its 16-lane row that holds column K (a DPP operand of the multiply-add),
// then adds g_c on row K.  A bad pivot sets `bad`; the caller discards the block.
__device__ __forceinline__ float lane_read(float v, int lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

// Orders LDS writes of some lanes of a wavefront before later LDS reads of other
// lanes of the same wavefront (the hardware keeps one wavefront's LDS accesses in
// order; the fence stops the compiler from moving a read above the write).
__device__ __forceinline__ void wave_lds_sync() { __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront"); }

// Cross-lane moves of the 16 x 16 Gauss-Jordan steps below: DPP row_newbcast
// (one lane of each 16-lane row to the whole row) and two permlane swaps (one
// 16-lane row to all four).
template <int N>
__device__ __forceinline__ float row_newbcast(float v) {  // lane N of each 16-lane row
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x150 + N, 0xF, 0xF, false));
}

template <int Q>
__device__ __forceinline__ float row16_broadcast(float v) {  // 16-lane row Q to all four rows
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                  false);
  const unsigned y = (Q >> 1) ? a[1] : a[0];  // rows (2(Q>>1), 2(Q>>1)+1) in both halves
  const auto b = __builtin_amdgcn_permlane16_swap(y, y, false, false);
  return __uint_as_float((Q & 1) ? b[1] : b[0]);
}

// Inversion of a 32 x 32 pivot block as four 16 x 16 blocks, [A11 A12; A21 A22]^{-1}
// by the Schur complement S = A22 - A21 A11^{-1} A12: two 16 x 16 Gauss-Jordan
// inversions (the first 16 pivots, then the 16 pivots of S: exactly the 32
// pivots of the unblocked elimination) and six 16 x 16 products on
// v_mfma_f32_16x16x4_f32.  A 16 x 16 block sits in the accumulator layout of that
// instruction: lane c + 16 g holds rows 4g .. 4g+3 of column c, so a pivot step
// costs four multiply-adds per lane instead of sixteen.  Column K reaches the
// lane's 16-lane row by DPP row_newbcast, row K the whole wavefront by two
// permlane swaps, the pivot by readlane.  `scr` holds three staged 16 x 16
// matrices (row stride kS16) for the products' left operands.
typedef float floatx4 __attribute__((ext_vector_type(4)));
constexpr int kS16 = 20;  // LDS row stride (floats) of a staged 16 x 16 matrix: 16-byte rows

// eg[q] = 1 in the lanes of 16-lane row q, else 0.
template <int K>
__device__ __forceinline__ void gj16_step(float (&t)[4], int c, const float (&eg)[4], bool &bad) {
  constexpr int QK = K >> 2, RK = K & 3;
  const float p = lane_read(t[RK], 16 * QK + K);
  bad |= !(p > 0.f && p < INFINITY);              // checked once after the 16 steps
  const float rw = row16_broadcast<QK>(t[RK]);    // row K at column c (p at c = K)
  const float ng = -((c == K ? rw + 1.f : rw) * __builtin_amdgcn_rcpf(p));  // -g_c
#pragma unroll
  for (int r = 0; r < 4; ++r) t[r] = fmaf(row_newbcast<K>(t[r]), ng, t[r]);  // rows 4g + r
  t[RK] = fmaf(-eg[QK], ng, t[RK]);               // + g_c on row K
}

template <int K>
__device__ __forceinline__ void gj16_from(float (&t)[4], int c, const float (&eg)[4], bool &bad) {
  if constexpr (K < 16) {
    gj16_step<K>(t, c, eg, bad);
    gj16_from<K + 1>(t, c, eg, bad);
  }
}

// Row-major 16 x 16 (stride ld) <-> accumulator layout.
__device__ __forceinline__ void ld16(const float *m, int ld, float (&x)[4], int g, int c) {
#pragma unroll
  for (int r = 0; r < 4; ++r) x[r] = m[(4 * g + r) * ld + c];
}
__device__ __forceinline__ void st16(float *m, int ld, const float (&x)[4], int g, int c) {
#pragma unroll
  for (int r = 0; r < 4; ++r) m[(4 * g + r) * ld + c] = x[r];
}

// x (accumulator layout) += sgn * A B, A row-major in LDS (stride lda, a multiple
// of 4), B in accumulator layout: k = 4g + s in instruction s.
__device__ __forceinline__ void mm16(float (&x)[4], const float *A, int lda, const float (&b)[4],
                                     int g, int c, float sgn) {
  const float4 a = *reinterpret_cast<const float4 *>(A + c * lda + 4 * g);
  floatx4 acc = {x[0], x[1], x[2], x[3]};
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(sgn * a.x, b[0], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(sgn * a.y, b[1], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(sgn * a.z, b[2], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(sgn * a.w, b[3], acc, 0, 0, 0);
#pragma unroll
  for (int r = 0; r < 4; ++r) x[r] = acc[r];
}

// Transposed store of a block in accumulator layout: T[c][4g + r] = x[r].
__device__ __forceinline__ void st16t(float *m, int ld, const float (&x)[4], int g, int c) {
  *reinterpret_cast<float4 *>(m + c * ld + 4 * g) = make_float4(x[0], x[1], x[2], x[3]);
}

// Inverts the 32 x 32 block staged row-major (stride kTileLd) in `in` by one
// wavefront: X11 = A11^{-1}, T1 = A21 X11, T2 = X11 A12, X22 = (A22 - T1 A12)^{-1},
// X12 = -T2 X22, X21 = -X22 T1, X11' = X11 - T2 X21 (= X11 + T2 X22 T1).  Writes
// the inverse row-major to pa and transposed to pb (both stride kTileLd); false
// (uniformly, nothing written) on a bad pivot.
__device__ __forceinline__ bool gj32_invert(const float *in, float *pa, float *pb, float *scr,
                                            int lane) {
  const int c = lane & 15, g = lane >> 4;
  float *s0 = scr, *s1 = scr + 16 * kS16, *s2 = scr + 32 * kS16;
  bool bad = false;
  float eg[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) eg[q] = g == q ? 1.f : 0.f;
  float x11[4], a12[4], x22[4];
  ld16(in, kTileLd, x11, g, c);                      // A11
  ld16(in + 16, kTileLd, a12, g, c);                 // A12
  ld16(in + 16 * kTileLd + 16, kTileLd, x22, g, c);  // A22
  gj16_from<0>(x11, c, eg, bad);                      // X11 = A11^{-1}
  float t1[4] = {0.f, 0.f, 0.f, 0.f}, t2[4] = {0.f, 0.f, 0.f, 0.f};
  mm16(t1, in + 16 * kTileLd, kTileLd, x11, g, c, 1.f);  // T1 = A21 X11
  st16(s0, kS16, t1, g, c);
  st16(s1, kS16, x11, g, c);
  wave_lds_sync();
  mm16(x22, s0, kS16, a12, g, c, -1.f);  // S = A22 - T1 A12
  mm16(t2, s1, kS16, a12, g, c, 1.f);    // T2 = X11 A12
  st16(s2, kS16, t2, g, c);
  gj16_from<0>(x22, c, eg, bad);          // X22 = S^{-1}
  wave_lds_sync();
  st16(s1, kS16, x22, g, c);
  float x12[4] = {0.f, 0.f, 0.f, 0.f}, x21[4] = {0.f, 0.f, 0.f, 0.f};
  mm16(x12, s2, kS16, x22, g, c, -1.f);  // X12 = -T2 X22
  wave_lds_sync();
  mm16(x21, s1, kS16, t1, g, c, -1.f);   // X21 = -X22 T1
  mm16(x11, s2, kS16, x21, g, c, -1.f);  // X11' = X11 - T2 X21
  if (bad) return false;
  st16(pa, kTileLd, x11, g, c);
  st16(pa + 16, kTileLd, x12, g, c);
  st16(pa + 16 * kTileLd, kTileLd, x21, g, c);
  st16(pa + 16 * kTileLd + 16, kTileLd, x22, g, c);
  st16t(pb, kTileLd, x11, g, c);
  st16t(pb + 16 * kTileLd, kTileLd, x12, g, c);
  st16t(pb + 16, kTileLd, x21, g, c);
  st16t(pb + 16 * kTileLd + 16, kTileLd, x22, g, c);
  return true;
}

// Operand fetch of a staged tile: lane (i or j, h) reads its 16 values at
// column (row) offsets acc_row(h, 0..15), four 16-byte reads.
__device__ __forceinline__ void lds_operand(const float *tile, int idx, int h, float (&o)[16]) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float4 v = *reinterpret_cast<const float4 *>(tile + idx * kTileLd + 4 * h + 8 * q);
    o[4 * q] = v.x;
    o[4 * q + 1] = v.y;
    o[4 * q + 2] = v.z;
    o[4 * q + 3] = v.w;
  }
}

// Stage a register tile for use as an A operand later (row-major: T[row][col]).
__device__ __forceinline__ void stage_a(float *tile, const floatx16 &v, int j, int h) {
#pragma unroll
  for (int r = 0; r < 16; ++r) tile[acc_row(h, r) * kTileLd + j] = v[r];
}

// The same, negated.
__device__ __forceinline__ void stage_a_neg(float *tile, const floatx16 &v, int j, int h) {
#pragma unroll
  for (int r = 0; r < 16; ++r) tile[acc_row(h, r) * kTileLd + j] = -v[r];
}

// acc += A B over one 32-wide k block, k of instruction r = acc_row(h, r).
__device__ __forceinline__ floatx16 mfma32(const float (&a)[16], const float (&b)[16], floatx16 acc) {
#pragma unroll
  for (int r = 0; r < 16; ++r) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[r], b[r], acc, 0, 0, 0);
  return acc;
}


// Woodbury matrix C = I - 2 eta S N S with S = diag(dl/dq)^{1/2} and N = H^T H,
// its inverse, and R = 2 eta S C^{-1} S (U_new^{-T} = U^{-T} + (U^{-T} H) R H^T).
// unit_dq: dl/dq = 1 for every example (squared error), dq is not read.
// Returns false after raising the error flag when some dl/dq is negative or NaN.
__device__ __forceinline__ bool woodbury_scales(int m, int unit_dq, const float *__restrict__ dq,
                                                float *sq, int *s_bad, int *flag) {
  const int t = threadIdx.x;
  if (t == 0) *s_bad = 0;
  __syncthreads();
  for (int i = t; i < m; i += blockDim.x) {
    const float v = unit_dq ? 1.f : dq[i];
    if (!(v >= 0.f)) atomicOr(s_bad, 1);  // negative or NaN dl/dq: no real square root
    sq[i] = sqrtf(fmaxf(v, 0.f));
  }
  __syncthreads();
  if (__builtin_amdgcn_readfirstlane(*s_bad)) {
    if (t == 0) atomicOr(flag, FLAG_NOT_SPD);
    return false;
  }
  return true;
}

// Stage a register tile for use as a B operand later (transposed: T[col][row]);
// lds_operand of the copy gives the tile back in accumulator layout.
__device__ __forceinline__ void stage_b(float *tile, const floatx16 &v, int j, int h) {
#pragma unroll
  for (int q = 0; q < 4; ++q)
    *reinterpret_cast<float4 *>(tile + j * kTileLd + 4 * h + 8 * q) =
        make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
}

// Wavefronts of the elimination: wb_workers own the tile columns (column c
// belongs to wavefront c % wb_workers, as its tile set c / wb_workers) and one
// more inverts the pivot blocks, one wavefront per SIMD: the inversion is a
// chain of dependent vector instructions that slows down several times over
// beside a wavefront issuing matrix instructions on the same SIMD.
template <int NBK>
constexpr int wb_workers() { return NBK < 3 ? NBK : 3; }
template <int NBK>
constexpr int wb_waves() { return wb_workers<NBK>() + 1; }
template <int NBK>
constexpr int wb_sets() { return (NBK + wb_workers<NBK>() - 1) / wb_workers<NBK>(); }

// LDS of the blocked elimination.  Everything a block step reads is written in
// the step before it (or before the first), so it is double-buffered by
// block-step parity.
template <int NBK>
struct alignas(16) GjLds {
  float cpan[2][NBK][kTileSz];  // -A_i,kb (row-major: A operand)
  float pa[2][kTileSz];         // P_kb row-major (A operand)
  float pb[2][kTileSz];         // P_kb transposed (B operand, accumulator-layout reads)
  float nb[2][kTileSz];         // A_kb,kb+1 transposed
  float nd[2][kTileSz];         // A_kb+1,kb+1 transposed
  float pin[kTileSz];           // the pivot block being inverted, row-major
  float scr[3 * 16 * kS16];     // left operands of the inversion's 16 x 16 products
  int bad[2];                   // bad pivot block, by block-step parity (0 on entry)
};

// Block step kb on tile column col (acc[i] = tile (i, col)); see gj_workers.
template <int NBK>
__device__ __forceinline__ void column_step(floatx16 (&acc)[NBK], GjLds<NBK> &sh, int col, int kb,
                                            int j, int h) {
  const int buf = kb & 1;
  if (col == kb) {
    float b[16];
    lds_operand(sh.pb[buf], j, h, b);  // P at (acc_row(h, r), j): B operand and own layout
#pragma unroll
    for (int s = 0; s < NBK; ++s) {
      if (s == kb) continue;
      float a[16];
      lds_operand(sh.cpan[buf][s], j, h, a);
      floatx16 z;
#pragma unroll
      for (int r = 0; r < 16; ++r) z[r] = 0.f;
      acc[s] = mfma32(a, b, z);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int s = 0; s < NBK; ++s)
      if (s == kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[s][r] = b[r];
    return;
  }
  float rp[16];  // P A_kb,col: the B operand of the column's trailing products
#pragma unroll
  for (int s = 0; s < NBK; ++s) {
    if (s != kb) continue;
    float a[16], b[16];
    lds_operand(sh.pa[buf], j, h, a);
#pragma unroll
    for (int r = 0; r < 16; ++r) b[r] = acc[s][r];
    floatx16 z;
#pragma unroll
    for (int r = 0; r < 16; ++r) z[r] = 0.f;
    acc[s] = mfma32(a, b, z);
#pragma unroll
    for (int r = 0; r < 16; ++r) rp[r] = acc[s][r];
  }
  const bool next = col == kb + 1;
#pragma unroll
  for (int s = 0; s < NBK; ++s) {
    if (s == kb || (next && s == kb + 1)) continue;
    float a[16];
    lds_operand(sh.cpan[buf][s], j, h, a);
    acc[s] = mfma32(a, rp, acc[s]);
    __builtin_amdgcn_sched_barrier(0);  // one tile's operands live at a time
  }
  if (next) {
#pragma unroll
    for (int s = 0; s < NBK; ++s)
      if (s != kb + 1) stage_a_neg(sh.cpan[buf ^ 1][s], acc[s], j, h);
  } else if (col == kb + 2) {
#pragma unroll
    for (int s = 0; s < NBK; ++s) {
      if (s == kb + 1) stage_b(sh.nb[buf ^ 1], acc[s], j, h);
      if (s == kb + 2) stage_b(sh.nd[buf ^ 1], acc[s], j, h);
    }
  }
}

// The NBK block steps with look-ahead, split by role: gj_workers runs on the
// wb_workers column owners, gj_inverter on the one inverting wavefront; both
// pass the same barriers (one per block step).  Each step kb opens with a
// barrier after which P_kb is in pa/pb[kb & 1], -A_i,kb (i != kb) in
// cpan[kb & 1] and the tiles A_kb,kb+1 and A_kb+1,kb+1 in nb/nd[kb & 1] (values
// after step kb - 1).  Each tile column is updated by its owner: column kb
// gives A_i,kb <- -A_i,kb P and A_kb,kb <- P; any other column c the row-panel
// tile P A_kb,c and the trailing tiles A_i,c - A_i,kb (P A_kb,c).  Meanwhile the
// inverting wavefront forms the next pivot block, A_kb+1,kb+1 - A_kb+1,kb
// (P A_kb,kb+1), from the staged tiles and inverts it, so the inversion of
// P_kb+1 runs beside the rest of step kb (the owner of column kb + 1 skips that
// tile, which P_kb+1 replaces).  The owners of columns kb + 1 and kb + 2 stage
// the next step's column panel and nb/nd.  A bad pivot block is flagged in
// bad[its step's parity], which no wavefront writes between the barrier that
// opens that step and the next one, so every wavefront reads the same value
// and all leave at the same step.

// acc[t][i] is tile (i, wave + wb_workers t).  Returns false (uniformly) if a
// pivot is not positive and finite; the tiles are then meaningless.  Column
// NBK - 1 is left at its values before the last block step: the inverting
// wavefront finishes it (last_column).
template <int NBK>
__device__ __forceinline__ bool gj_workers(floatx16 (&acc)[wb_sets<NBK>()][NBK], GjLds<NBK> &sh,
                                           int wave, int lane) {
  constexpr int NW = wb_workers<NBK>(), NS = wb_sets<NBK>();
  const int j = lane & 31, h = lane >> 5;
#pragma unroll
  for (int t = 0; t < NS; ++t) {
    const int col = wave + NW * t;
    if (col == 0) {
#pragma unroll
      for (int s = 1; s < NBK; ++s) stage_a_neg(sh.cpan[0][s], acc[t][s], j, h);
    } else if (col == 1) {
      stage_b(sh.nb[0], acc[t][0], j, h);
      stage_b(sh.nd[0], acc[t][1], j, h);
    }
  }
  for (int kb = 0; kb < NBK; ++kb) {
    __syncthreads();
    if (__builtin_amdgcn_readfirstlane(sh.bad[kb & 1])) return false;
#pragma unroll
    for (int t = 0; t < NS; ++t) {
      const int col = wave + NW * t;
      // the last pivot column is the inverting wavefront's (last_column)
      if (col < NBK && !(kb == NBK - 1 && col == kb)) column_step<NBK>(acc[t], sh, col, kb, j, h);
    }
  }
  return true;
}

// a00: the pivot block A_00 in accumulator layout.  Returns false (uniformly,
// at the same step as gj_workers) if a pivot is not positive and finite.
template <int NBK>
__device__ __forceinline__ bool gj_inverter(const floatx16 &a00, GjLds<NBK> &sh, int lane) {
  const int j = lane & 31, h = lane >> 5;
  stage_a(sh.pin, a00, j, h);
  // kb = -1 inverts A_00 into buffer 0; block step kb >= 0 forms and inverts the next
  // pivot block.  One call site of the inversion: a single copy of its code.
  for (int kb = -1; kb < NBK - 1; ++kb) {
    const int dst = (kb + 1) & 1;
    if (kb >= 0) {
      const int buf = kb & 1;
      __syncthreads();
      if (__builtin_amdgcn_readfirstlane(sh.bad[buf])) return false;
      float a[16], b[16];
      lds_operand(sh.pa[buf], j, h, a);
      lds_operand(sh.nb[buf], j, h, b);
      floatx16 z;
#pragma unroll
      for (int r = 0; r < 16; ++r) z[r] = 0.f;
      const floatx16 t = mfma32(a, b, z);  // P A_kb,kb+1
      float d[16];
      lds_operand(sh.cpan[buf][kb + 1], j, h, a);
      lds_operand(sh.nd[buf], j, h, d);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        b[r] = t[r];
        z[r] = d[r];
      }
      stage_a(sh.pin, mfma32(a, b, z), j, h);
    }
    wave_lds_sync();
    if (!gj32_invert(sh.pin, sh.pa[dst], sh.pb[dst], sh.scr, lane) && lane == 0) sh.bad[dst] = 1;
  }
  __syncthreads();  // the barrier that opens the last block step
  return !__builtin_amdgcn_readfirstlane(sh.bad[(NBK - 1) & 1]);
}

// The last block step's pivot column (kb = NBK - 1), by the inverting wavefront
// after gj_inverter: tile (i, kb) of the inverse is -A_i,kb P = cpan[kb & 1][i] P
// for i != kb and P itself for i = kb, all from LDS the last step left in place
// (nothing writes those buffers after its opening barrier).  This takes the
// column's three products and its stores off its owner, which in the last step
// would otherwise hold two columns.  out(i, tile) receives each tile.  Every lane
// of the wavefront must call it (the products read all lanes' operands).
template <int NBK, typename Out>
__device__ __forceinline__ void last_column(const GjLds<NBK> &sh, int lane, Out out) {
  constexpr int kb = NBK - 1, buf = kb & 1;
  const int j = lane & 31, h = lane >> 5;
  float b[16];
  lds_operand(sh.pb[buf], j, h, b);  // P at (acc_row(h, r), j)
#pragma unroll
  for (int s = 0; s < NBK; ++s) {
    floatx16 v;
    if (s == kb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) v[r] = b[r];
    } else {
      float a[16];
      lds_operand(sh.cpan[buf][s], j, h, a);
      floatx16 z;
#pragma unroll
      for (int r = 0; r < 16; ++r) z[r] = 0.f;
      v = mfma32(a, b, z);
    }
    out(s, v);
    __builtin_amdgcn_sched_barrier(0);
  }
}

// The whole inverse on one workgroup of 64 wb_waves<NBK>() threads (m <= 32 NBK):
// C = I - 2 eta S N S from N, its inverse, R = 2 eta S C^{-1} S.  A rejected
// matrix (non-positive pivot, negative or NaN dl/dq) raises FLAG_NOT_SPD.
template <int NBK>
__device__ __forceinline__ void woodbury_blocked(int m, float lr, int unit_dq,
                                                 const float *__restrict__ dq,
                                                 const float *__restrict__ N,
                                                 float *__restrict__ R, int *__restrict__ flag) {
  __shared__ GjLds<NBK> sh;
  __shared__ __align__(16) float sq[32 * NBK];
  if (threadIdx.x == 0) sh.bad[1] = 0;  // published by the barriers in woodbury_scales
  if (!woodbury_scales(m, unit_dq, dq, sq, &sh.bad[0], flag)) return;
  const int lane = threadIdx.x & 63, j = lane & 31, h = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const float tl = 2.f * lr;
  // Load C: lane (j, h) reads column col of rows 32 s + acc_row(h, 0..15); the
  // scales come from LDS, sq[row] as four 16-byte reads.  Entries outside m x m
  // read a clamped in-range address and are replaced by the identity.  All loads
  // are issued first and pinned by empty asm statements, so that none is moved
  // under the (row, col) < m conditions and they overlap in flight.
  constexpr int NW = wb_workers<NBK>(), NS = wb_sets<NBK>();
  if (wave == NW) {  // the inverting wavefront: the pivot block A_00
    float raw[16];
    const float *np = N + min(j, m - 1);
#pragma unroll
    for (int r = 0; r < 16; ++r) raw[r] = np[min(acc_row(h, r), m - 1) * m];
#pragma unroll
    for (int r = 0; r < 16; ++r) asm volatile("" : "+v"(raw[r]));
    const float sc = tl * sq[min(j, m - 1)];
    float sr[16];
    lds_operand(sq, 0, h, sr);
    floatx16 a00;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = acc_row(h, r);
      const float c = (row < m && j < m) ? -(sr[r] * raw[r] * sc) : 0.f;
      a00[r] = (row == j) ? 1.f + c : c;
    }
    if (!gj_inverter<NBK>(a00, sh, lane)) return;
    // the whole wavefront takes part in the products; only the stores are masked
    const int lcol = 32 * (NBK - 1) + j;
    const float lsc = tl * sq[min(lcol, m - 1)];
    last_column<NBK>(sh, lane, [&](int s, const floatx16 &v) {
      if (lcol >= m) return;
      float sr[16];
      lds_operand(sq + 32 * s, 0, h, sr);
      const int base = (32 * s + 4 * h) * m + lcol;
      if (32 * s + 32 <= m) {
#pragma unroll
        for (int r = 0; r < 16; ++r) R[base + ((r & 3) + 8 * (r >> 2)) * m] = sr[r] * v[r] * lsc;
      } else {
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (32 * s + acc_row(h, r) < m) R[base + ((r & 3) + 8 * (r >> 2)) * m] = sr[r] * v[r] * lsc;
      }
    });
    return;
  }
  floatx16 acc[NS][NBK];
  {
    float raw[NS][NBK][16];
#pragma unroll
    for (int t = 0; t < NS; ++t) {
      if (wave + NW * t >= NBK) continue;  // no such tile column
      const float *np = N + min(32 * (wave + NW * t) + j, m - 1);
#pragma unroll
      for (int s = 0; s < NBK; ++s)
#pragma unroll
        for (int r = 0; r < 16; ++r) raw[t][s][r] = np[min(32 * s + acc_row(h, r), m - 1) * m];
    }
#pragma unroll
    for (int t = 0; t < NS; ++t)
#pragma unroll
      for (int s = 0; s < NBK; ++s)
#pragma unroll
        for (int r = 0; r < 16; ++r) asm volatile("" : "+v"(raw[t][s][r]));
#pragma unroll
    for (int t = 0; t < NS; ++t) {
      const int col = 32 * (wave + NW * t) + j;
      const float sc = tl * sq[min(col, m - 1)];
#pragma unroll
      for (int s = 0; s < NBK; ++s) {
        float sr[16];
        lds_operand(sq + 32 * s, 0, h, sr);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = 32 * s + acc_row(h, r);
          const float c = (row < m && col < m) ? -(sr[r] * raw[t][s][r] * sc) : 0.f;
          acc[t][s][r] = (row == col) ? 1.f + c : c;
        }
      }
    }
  }

  if (!gj_workers<NBK>(acc, sh, wave, lane)) {
    if (threadIdx.x == 0) atomicOr(flag, FLAG_NOT_SPD);
    return;
  }
  // R row-major; tiles inside m x m (all of them when m is a multiple of 32)
  // store without per-row checks, at 32-bit offsets from R.
#pragma unroll
  for (int t = 0; t < NS; ++t) {
    const int col = 32 * (wave + NW * t) + j;
    if (wave + NW * t >= NBK - 1 || col >= m) continue;  // column NBK - 1: the inverting wavefront's
    const float sc = tl * sq[col];
#pragma unroll
    for (int s = 0; s < NBK; ++s) {
      float sr[16];
      lds_operand(sq + 32 * s, 0, h, sr);
      const int base = (32 * s + 4 * h) * m + col;
      if (32 * s + 32 <= m) {
#pragma unroll
        for (int r = 0; r < 16; ++r)
          R[base + ((r & 3) + 8 * (r >> 2)) * m] = sr[r] * acc[t][s][r] * sc;
      } else {
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (32 * s + acc_row(h, r) < m)
            R[base + ((r & 3) + 8 * (r >> 2)) * m] = sr[r] * acc[t][s][r] * sc;
      }
    }
  }
}


}  // namespace

}  // namespace lst
