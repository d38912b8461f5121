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
// MFMA accumulator registers as NBK x NBK tiles of 32 x 32, tile t owned by
// wavefront t % W.  In accumulator layout lane l = j + 32 h holds column j of a
// tile and register r holds row acc_row(h, r).  Block step kb with pivot block
// P = A_kb,kb^{-1} is, in place,
//   A_kb,j <- P A_kb,j,   A_ij <- A_ij - A_i,kb (P A_kb,j),
//   A_i,kb <- -A_i,kb P,  A_kb,kb <- P                          (i, j != kb),
// the block form of the scalar step below; after NBK block steps the tiles hold
// the inverse.  The products run on v_mfma_f32_32x32x2f32 with the k index of
// instruction r taken as acc_row(h, r) in lane-half h, so a tile held in
// registers is directly the B operand of a product; the other operands come
// from LDS copies of the column panel, the new row panel and P.  Since every
// pivot block is a Schur complement of C, the pivots met inside the 32 x 32
// inversions are exactly those of unblocked elimination: all are positive iff
// C is positive definite.
// ---------------------------------------------------------------------------
typedef float floatx16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ int acc_row(int h, int r) { return 4 * h + (r & 3) + 8 * (r >> 2); }

constexpr int kTileLd = 36;  // LDS row stride (floats) of a staged 32 x 32 tile: 16-byte rows
constexpr int kTileSz = 32 * kTileLd;

// One scalar Gauss-Jordan step on pivot K (p = A_KK) of a 32 x 32 block:
//   A' = X - f g^T,  X = A with column K replaced by e_K,
//   f_i = A_iK (i != K), f_K = p - 1,   g_j = A_Kj / p (j != K), g_K = 1 / p,
// i.e. A'_Kj = A_Kj / p, A'_iK = -A_iK / p, A'_KK = 1 / p, A'_ij = A_ij - A_iK A_Kj / p.
// Column K needs no separate case: there t_i = f_i (and t_K = p), so
// A' = t - f (1 + 1/p) gives -f_i / p and 1 / p.  A bad pivot sets `bad`; the
// caller discards the block.
__device__ __forceinline__ float lane_read(float v, int lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

// Orders LDS writes of some lanes of a wavefront before later LDS reads of other
// lanes of the same wavefront (the hardware keeps one wavefront's LDS accesses in
// order; the fence stops the compiler from moving a read above the write).
__device__ __forceinline__ void wave_lds_sync() { __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront"); }

// The pivot-block inversion runs in the layout the cross-lane moves favour:
// lane 16 q + c holds rows 8q .. 8q+7 of columns 2c and 2c+1, t[8e + r] = T[8q + r][2c + e].
// Column K at the lane's rows sits in lane c = K/2 of the lane's own 16-lane row
// (DPP row_newbcast); row K at the lane's columns sits in 16-lane row K/8 (two
// permlane swaps broadcast it to all four rows); the pivot comes from readlane.
// No LDS round trip is on the serial path.
template <int N>
__device__ __forceinline__ float row_newbcast(float v) {  // lane N of each 16-lane row
  return __int_as_float(
      __builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x150 + N, 0xF, 0xF, false));
}

template <int Q>
__device__ __forceinline__ float row16_broadcast(float v) {  // 16-lane row Q to all four rows
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                  false);
  const unsigned y = (Q >> 1) ? a[1] : a[0];  // rows (2(Q>>1), 2(Q>>1)+1) in both halves
  const auto b = __builtin_amdgcn_permlane16_swap(y, y, false, false);
  return __uint_as_float((Q & 1) ? b[1] : b[0]);
}

template <int K>
__device__ __forceinline__ void gjr_step(float (&t)[16], int q, int c, bool &bad) {
  constexpr int QK = K >> 3, RK = K & 7, CK = K >> 1, EK = K & 1;
  const float p = lane_read(t[8 * EK + RK], 16 * QK + CK);
  bad |= !(p > 0.f && p < INFINITY);  // checked once after the 32 steps
  float f[8];                          // column K at rows 8q + r
#pragma unroll
  for (int r = 0; r < 8; ++r) f[r] = row_newbcast<CK>(t[8 * EK + r]);
  float rw[2];  // row K at columns 2c + e
#pragma unroll
  for (int e = 0; e < 2; ++e) rw[e] = row16_broadcast<QK>(t[8 * e + RK]);
  float ip = __builtin_amdgcn_rcpf(p);
  ip = fmaf(ip, fmaf(-p, ip, 1.f), ip);  // one Newton step on the hardware reciprocal
  float g[2];
#pragma unroll
  for (int e = 0; e < 2; ++e) g[e] = (e == EK && c == CK) ? 1.f + ip : rw[e] * ip;
#pragma unroll
  for (int e = 0; e < 2; ++e)
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const float fr = (r == RK && q == QK) ? p - 1.f : f[r];
      t[8 * e + r] = fmaf(-fr, g[e], t[8 * e + r]);
    }
}

template <int K>
__device__ __forceinline__ void gjr_from(float (&t)[16], int q, int c, bool &bad) {
  if constexpr (K < 32) {
    gjr_step<K>(t, q, c, bad);
    gjr_from<K + 1>(t, q, c, bad);
  }
}

// Inverts the 32 x 32 block staged row-major (stride kTileLd) in `tile` by one
// wavefront and leaves the inverse there; false (uniformly) on a bad pivot.
__device__ __forceinline__ bool gj32_invert_staged(float *tile, int lane) {
  const int q = lane >> 4, c = lane & 15;
  float t[16];
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    const float2 v = *reinterpret_cast<const float2 *>(tile + (8 * q + r) * kTileLd + 2 * c);
    t[r] = v.x;
    t[8 + r] = v.y;
  }
  bool bad = false;
  gjr_from<0>(t, q, c, bad);
  if (bad) return false;
#pragma unroll
  for (int r = 0; r < 8; ++r)
    *reinterpret_cast<float2 *>(tile + (8 * q + r) * kTileLd + 2 * c) = make_float2(t[r], t[8 + r]);
  return true;
}

// The same inversion as four 16 x 16 blocks, [A11 A12; A21 A22]^{-1} by the
// Schur complement S = A22 - A21 A11^{-1} A12: two 16 x 16 Gauss-Jordan
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

template <int K>
__device__ __forceinline__ void gj16_step(float (&t)[4], int g, int c, bool &bad) {
  constexpr int QK = K >> 2, RK = K & 3;
  const float p = lane_read(t[RK], 16 * QK + K);
  bad |= !(p > 0.f && p < INFINITY);  // checked once after the 16 steps
  float f[4];                          // column K at rows 4g + r
#pragma unroll
  for (int r = 0; r < 4; ++r) f[r] = row_newbcast<K>(t[r]);
  const float rw = row16_broadcast<QK>(t[RK]);  // row K at column c
  float ip = __builtin_amdgcn_rcpf(p);
  ip = fmaf(ip, fmaf(-p, ip, 1.f), ip);  // one Newton step on the hardware reciprocal
  const float gc = (c == K) ? 1.f + ip : rw * ip;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const float fr = (r == RK && g == QK) ? p - 1.f : f[r];
    t[r] = fmaf(-fr, gc, t[r]);
  }
}

template <int K>
__device__ __forceinline__ void gj16_from(float (&t)[4], int g, int c, bool &bad) {
  if constexpr (K < 16) {
    gj16_step<K>(t, g, c, bad);
    gj16_from<K + 1>(t, g, c, bad);
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

// Inverts the 32 x 32 block staged row-major (stride kTileLd) in `tile` by one
// wavefront and leaves the inverse there; false (uniformly) on a bad pivot.
__device__ __forceinline__ bool gj32_invert_schur(float *tile, float *scr, int lane) {
  const int c = lane & 15, g = lane >> 4;
  float *s0 = scr, *s1 = scr + 16 * kS16, *s2 = scr + 32 * kS16;
  bool bad = false;
  float x11[4], a12[4], t1[4], x22[4];
  ld16(tile, kTileLd, x11, g, c);                        // A11
  ld16(tile + 16, kTileLd, a12, g, c);                   // A12
  ld16(tile + 16 * kTileLd + 16, kTileLd, x22, g, c);    // A22
  gj16_from<0>(x11, g, c, bad);                          // X11 = A11^{-1}
#pragma unroll
  for (int r = 0; r < 4; ++r) t1[r] = 0.f;
  mm16(t1, tile + 16 * kTileLd, kTileLd, x11, g, c, 1.f);  // T1 = A21 X11
  st16(s0, kS16, t1, g, c);
  st16(s1, kS16, x11, g, c);
  wave_lds_sync();
  mm16(x22, s0, kS16, a12, g, c, -1.f);                 // S = A22 - T1 A12
  gj16_from<0>(x22, g, c, bad);                          // X22 = S^{-1}
  float t2[4] = {0.f, 0.f, 0.f, 0.f};
  mm16(t2, s1, kS16, a12, g, c, 1.f);                    // T2 = X11 A12
  st16(s2, kS16, t2, g, c);
  wave_lds_sync();
  float x12[4] = {0.f, 0.f, 0.f, 0.f};
  mm16(x12, s2, kS16, x22, g, c, -1.f);                  // X12 = -T2 X22
  st16(s1, kS16, x22, g, c);                             // (X11 staged copy no longer needed)
  st16(s0, kS16, x12, g, c);
  wave_lds_sync();
  float x21[4] = {0.f, 0.f, 0.f, 0.f};
  mm16(x21, s1, kS16, t1, g, c, -1.f);                   // X21 = -X22 T1
  mm16(x11, s0, kS16, t1, g, c, -1.f);                   // X11' = X11 - X12 T1
  if (bad) return false;
  wave_lds_sync();
  st16(tile, kTileLd, x11, g, c);
  st16(tile + 16, kTileLd, x12, g, c);
  st16(tile + 16 * kTileLd, kTileLd, x21, g, c);
  st16(tile + 16 * kTileLd + 16, kTileLd, x22, g, c);
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

// Stage a register tile for use as a B operand later (transposed: T[col][row]).
__device__ __forceinline__ void stage_b(float *tile, const floatx16 &v, int j, int h) {
#pragma unroll
  for (int q = 0; q < 4; ++q)
    *reinterpret_cast<float4 *>(tile + j * kTileLd + 4 * h + 8 * q) =
        make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
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

template <int NBK>
constexpr int wb_waves() { return 4; }  // NBK <= 4: at most 4 tiles per wavefront

// LDS of the blocked elimination.  Column panel and P are double-buffered by
// block-step parity, so a block step needs two barriers: after the pivot block
// is inverted and the column panel staged, and after the new row panel is staged.
template <int NBK>
struct alignas(16) GjLds {
  float cpan[2][NBK][kTileSz];  // A_i,kb        (A operand)
  float rpan[NBK][kTileSz];     // P A_kb,j      (B operand)
  float pa[2][kTileSz];         // P             (A operand)
  float pb[2][kTileSz];         // P             (B operand)
  int bad;
};

// The NBK block steps on the register-resident tiles (tile t = wave + W s).
// sh.bad must be 0 on entry.  Returns false (uniformly) if a pivot is not
// positive and finite; the tiles are then meaningless.
template <int NBK, int W, int TPW>
__device__ __forceinline__ bool blocked_gj(floatx16 (&acc)[TPW], GjLds<NBK> &sh, int wave,
                                           int lane) {
  constexpr int NT = NBK * NBK;
  const int j = lane & 31, h = lane >> 5;
  for (int kb = 0; kb < NBK; ++kb) {
    const int buf = kb & 1;
    // (a) invert the pivot block (its owner), stage P and the column panel
    const int td = kb * NBK + kb;
    if (wave == td % W) {
      const int sd = td / W;  // slot of the pivot block; copied out by value so that
      float p[16];            // the register tiles are never indexed at run time
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float v = acc[0][r];
#pragma unroll
        for (int s = 1; s < TPW; ++s) v = (s == sd) ? acc[s][r] : v;
        p[r] = v;
      }
      floatx16 pv;
#pragma unroll
      for (int r = 0; r < 16; ++r) pv[r] = p[r];
      stage_a(sh.pa[buf], pv, j, h);  // the pivot block, row-major
      wave_lds_sync();
      if (gj32_invert_schur(sh.pa[buf], sh.pb[buf], lane)) {  // P replaces it (A-operand layout)
        wave_lds_sync();
#pragma unroll
        for (int r = 0; r < 16; ++r) pv[r] = sh.pa[buf][acc_row(h, r) * kTileLd + j];
#pragma unroll
        for (int s = 0; s < TPW; ++s)
          if (s == sd) acc[s] = pv;
        stage_b(sh.pb[buf], pv, j, h);
      } else if (lane == 0) {
        sh.bad = 1;
      }
    }
#pragma unroll
    for (int s = 0; s < TPW; ++s) {
      const int t = wave + W * s;
      if (t < NT && t % NBK == kb && t / NBK != kb) stage_a(sh.cpan[buf][t / NBK], acc[s], j, h);
    }
    __syncthreads();
    if (__builtin_amdgcn_readfirstlane(sh.bad)) return false;
    // (b) row panel A_kb,j <- P A_kb,j, staged for the trailing update
#pragma unroll
    for (int s = 0; s < TPW; ++s) {
      const int t = wave + W * s;
      if (t >= NT) continue;
      const int ti = t / NBK, tj = t % NBK;
      if (ti != kb || tj == kb) continue;
      float a[16], b[16];
      lds_operand(sh.pa[buf], j, h, a);
#pragma unroll
      for (int r = 0; r < 16; ++r) b[r] = acc[s][r];
      floatx16 z;
#pragma unroll
      for (int r = 0; r < 16; ++r) z[r] = 0.f;
      acc[s] = mfma32(a, b, z);
      stage_b(sh.rpan[tj], acc[s], j, h);
      __builtin_amdgcn_sched_barrier(0);
    }
    __syncthreads();
    // (c) trailing tiles and the column panel
#pragma unroll
    for (int s = 0; s < TPW; ++s) {
      const int t = wave + W * s;
      if (t >= NT) continue;
      const int ti = t / NBK, tj = t % NBK;
      if (ti == kb) continue;
      float a[16], b[16];
      lds_operand(sh.cpan[buf][ti], j, h, a);
#pragma unroll
      for (int r = 0; r < 16; ++r) a[r] = -a[r];
      if (tj != kb) {
        lds_operand(sh.rpan[tj], j, h, b);
        acc[s] = mfma32(a, b, acc[s]);
      } else {
        lds_operand(sh.pb[buf], j, h, b);
        floatx16 z;
#pragma unroll
        for (int r = 0; r < 16; ++r) z[r] = 0.f;
        acc[s] = mfma32(a, b, z);
      }
      __builtin_amdgcn_sched_barrier(0);  // one tile's operands live at a time
    }
  }
  return true;
}

// The whole inverse on one workgroup of 64 wb_waves threads (m <= 32 NBK):
// C = I - 2 eta S N S from N, its inverse, R = 2 eta S C^{-1} S.  A rejected
// matrix (non-positive pivot, negative or NaN dl/dq) raises FLAG_NOT_SPD.
template <int NBK>
__device__ __forceinline__ void woodbury_blocked(int m, float lr, int unit_dq,
                                                 const float *__restrict__ dq,
                                                 const float *__restrict__ N,
                                                 float *__restrict__ R, int *__restrict__ flag) {
  constexpr int W = wb_waves<NBK>();
  constexpr int NT = NBK * NBK;
  constexpr int TPW = (NT + W - 1) / W;  // tiles per wavefront
  __shared__ GjLds<NBK> sh;
  __shared__ __align__(16) float sq[32 * NBK];
  if (!woodbury_scales(m, unit_dq, dq, sq, &sh.bad, flag)) return;
  const int lane = threadIdx.x & 63, j = lane & 31, h = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const float tl = 2.f * lr;

  // Load C tile by tile: lane (j, h) reads column col of rows acc_row(h, 0..15);
  // the scales come from LDS, sq[row] as four 16-byte reads.  Entries outside
  // m x m read a clamped in-range address and are replaced by the identity.
  // All loads are issued first and pinned by empty asm statements, so that none
  // is moved under the (row, col) < m conditions and they overlap in flight.
  float raw[TPW][16];
#pragma unroll
  for (int s = 0; s < TPW; ++s) {
    const int t = min(wave + W * s, NT - 1);
    const int col = (t % NBK) * 32 + j, r0 = (t / NBK) * 32;
    const float *np = N + min(col, m - 1);
#pragma unroll
    for (int r = 0; r < 16; ++r) raw[s][r] = np[min(r0 + acc_row(h, r), m - 1) * m];
  }
#pragma unroll
  for (int s = 0; s < TPW; ++s)
#pragma unroll
    for (int r = 0; r < 16; ++r) asm volatile("" : "+v"(raw[s][r]));
  floatx16 acc[TPW];
#pragma unroll
  for (int s = 0; s < TPW; ++s) {
    const int t = min(wave + W * s, NT - 1);
    const int r0 = (t / NBK) * 32, col = (t % NBK) * 32 + j;
    const float sc = tl * sq[min(col, m - 1)];
    float sr[16];
    lds_operand(sq + r0, 0, h, sr);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = r0 + acc_row(h, r);
      const float c = (row < m && col < m) ? -(sr[r] * raw[s][r] * sc) : 0.f;
      acc[s][r] = (row == col) ? 1.f + c : c;
    }
  }

  if (!blocked_gj<NBK, W, TPW>(acc, sh, wave, lane)) {
    if (threadIdx.x == 0) atomicOr(flag, FLAG_NOT_SPD);
    return;
  }
#pragma unroll
  for (int s = 0; s < TPW; ++s) {
    const int t = wave + W * s;
    if (t >= NT) continue;
    const int r0 = (t / NBK) * 32, col = (t % NBK) * 32 + j;
    if (col >= m) continue;
    const float sc = tl * sq[col];
    float sr[16];
    lds_operand(sq + r0, 0, h, sr);
    float *rp = R + col;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = r0 + acc_row(h, r);
      if (row < m) rp[row * m] = sr[r] * acc[s][r] * sc;
    }
  }
}


}  // namespace

}  // namespace lst
