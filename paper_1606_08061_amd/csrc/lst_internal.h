// Internal declarations shared by the HIP sources of liblst (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>

#include <cstddef>
#include <cstdint>

#include "lst.h"

namespace lst {

// Kernel timing hook.  While a phase is being timed, the launch macro attaches
// g_prof.start to the next kernel launched (the phase's first) and g_prof.stop
// to every launch (the last one records the phase's end).
struct ProfHook {
  hipEvent_t start = nullptr, stop = nullptr;
};
extern thread_local ProfHook g_prof;

#define LST_LAUNCH(KERNEL, GRID, BLOCK, SHMEM, STREAM, ...)                                     \
  do {                                                                                          \
    hipEvent_t lst_ev_a_ = ::lst::g_prof.start;                                                \
    ::lst::g_prof.start = nullptr;                                                             \
    if (lst_ev_a_ || ::lst::g_prof.stop)                                                       \
      hipExtLaunchKernelGGL(KERNEL, GRID, BLOCK, SHMEM, STREAM, lst_ev_a_, ::lst::g_prof.stop, \
                            0, __VA_ARGS__);                                                   \
    else                                                                                       \
      hipLaunchKernelGGL(KERNEL, GRID, BLOCK, SHMEM, STREAM, __VA_ARGS__);                     \
  } while (0)


// Sticky device error bits (mapped to lst_status by lst_sync_status).
enum : int { FLAG_INDEX = 1, FLAG_NOT_SPD = 2, FLAG_NONFINITE = 4, FLAG_SYNC = 8 };

// ---------------------------------------------------------------------------
// Batched fp32 MFMA GEMM.
//
// One descriptor computes  C[i,j] = alpha * sum_k opA(i,k) opB(k,j) + beta * Cin[i,j]
// for i < M, j < N, with the k sum running over one or two segments
// (k in [0,K) with A,B then k in [0,K2) with A2,B2).  Operand layouts:
//   tA = 0: opA(i,k) = A[i*lda + k]      tA = 1: opA(i,k) = A[k*lda + i]
//   tB = 0: opB(k,j) = B[j*ldb + k]      tB = 1: opB(k,j) = B[k*ldb + j]
// Epilogue EPI_GRADH additionally writes C2[i,j] = 2 rs[i] E[i,j] + C[i,j].
// splits > 1 splits the single segment's k range across workgroups; partial
// sums go to `partial` ([splits][M][N]) and a second kernel reduces them in a
// fixed order before applying the epilogue.
// ---------------------------------------------------------------------------
enum : int { EPI_NONE = 0, EPI_GRADH = 1 };

struct GemmDesc {
  const float *A, *B, *A2, *B2;
  float *C;
  const float *Cin;
  const float *rs;
  const float *E;
  float *C2;
  float *partial;
  int64_t lda, ldb, lda2, ldb2, ldc, ldcin, lde, ldc2;
  int M, N, K, K2;
  int tA, tB;
  float alpha, beta;
  int epi;
  int splits;
  int kchunk;  // k per split (multiple of 8) when splits > 1
  int tiles_m, tiles_n;
  int tile_begin;
  int lr_scaled;  // 1: alpha *= lr^2 and beta *= lr at launch; 2: alpha *= lr (plans shared
                  // across lr)
  // 128 x 128-tile kernel without split: when set, also writes per-column partial
  // sums of squares of the product, colsq[p][j] for p < 4 * tiles_m (each the sum
  // over 32 of the tile's rows of C[i,j]^2 before alpha/beta).
  float *colsq;
  // Operand terms (64 x 64 tiles of launch 4, one k segment, opA with k contiguous and
  // opB with the index contiguous):
  //   opA = sum over t < nat of aw[t] A_t (A_0 = A, the others At[t - 1], same lda)
  //         + awt opAt, opAt(i,k) = Atr[k lda + i] when Atr is set;
  //   opB = sum over t < nbt of coef[bcoef[t]] B_t (B_0 = B, the others Bt[t - 1]);
  //   the product gains sum over t < nadd of coef[acoef[t]] addp[t][i ldadd + j]
  //   before alpha;
  //   alt1 > 0: descriptor alt1 - 1 of the batch (same shape, plain) replaces this one
  //   while *cert == 0.
  int nat, nbt, nadd, alt1;
  const float *At[2], *Atr, *Bt[3], *addp[4];
  float aw[3], awt;
  int bcoef[4], acoef[4];
  int64_t ldadd;
  const float *coef;
};

// Operand placeholders of plans kept in device memory: a plan is built once per
// minibatch size m and refers to the step's H and grad_H through these values,
// which the kernels replace by the pointers passed at launch.
inline const float *sym_H() { return reinterpret_cast<const float *>(uintptr_t{16}); }
inline float *sym_gradH() { return reinterpret_cast<float *>(uintptr_t{32}); }

constexpr int kMaxBatch = 5;

struct GemmBatch {
  GemmDesc d[kMaxBatch];
  int n;
  int total_tiles;
  int wide;  // 8 wavefronts per tile (long k) instead of 4
  int tile;  // output tile edge: 32 (the batched launches, the step's default) or 64 (the
             // step's LDS-staged tiles at large shapes)
};

// A GemmBatch's tile ranges, passed to the step's kernels by value (as OpHdr below):
// descriptor q owns tiles [tile_begin[q], tile_begin[q] + count[q]).
struct GemmHdr {
  int n, total_tiles;
  int tile_begin[kMaxBatch];
  int count[kMaxBatch];
};
inline GemmHdr gemm_hdr(const GemmBatch &b) {
  GemmHdr h{};
  h.n = b.n;
  h.total_tiles = b.total_tiles;
  for (int q = 0; q < kMaxBatch; ++q) {
    const GemmDesc &g = b.d[q];
    h.tile_begin[q] = g.tile_begin;
    h.count[q] = q < b.n && g.M > 0 && g.N > 0 ? g.tiles_m * g.tiles_n * (g.splits > 1 ? g.splits : 1) : 0;
  }
  return h;
}

// The workgroups of a step launch's section for a batch: 32 x 32 tiles in one range
// (8 ceil(T / 8) workgroups for T tiles, each XCD a contiguous eighth); 64 x 64 tiles
// product by product, 8 ceil(T_q / 8) workgroups for product q, its T_q tiles spread
// evenly over the 8 XCDs (measured at m = 512: launch 3, whose products differ in k,
// 7 us faster at d = 1024; launch 5 6 us).
__host__ __device__ inline int gemm_section(const GemmHdr &h, int tile_edge) {
  if (tile_edge != 64) return (h.total_tiles + 7) & ~7;
  int n = 0;
  for (int q = 0; q < kMaxBatch; ++q)
    if (q < h.n) n += (h.count[q] + 7) >> 3;
  return 8 * n;
}

// Workgroup w of a 64 x 64 tiles' section (w % 8 its XCD): the tile it owns, or -1.
// XCD x owns a contiguous eighth of every product's tiles.
__host__ __device__ inline int gemm_tile64(const GemmHdr &h, int w) {
  const int x = w & 7;
  int s = w >> 3;
  for (int q = 0; q < kMaxBatch; ++q) {
    if (q >= h.n) break;
    const int T = h.count[q], c8 = T >> 3, r = T & 7;
    const int c = x < r ? c8 + 1 : c8;
    if (s < c) return h.tile_begin[q] + (x < r ? x * (c8 + 1) : r * (c8 + 1) + (x - r) * c8) + s;
    s -= c;
  }
  return -1;
}
__host__ __device__ inline int hdr_begin(const GemmBatch &b, int q) { return b.d[q].tile_begin; }
__host__ __device__ inline int hdr_begin(const GemmHdr &h, int q) { return h.tile_begin[q]; }

GemmDesc gemm_desc(int M, int N, int K, const float *A, int64_t lda, int tA, const float *B,
                   int64_t ldb, int tB, float *C, int64_t ldc, float alpha = 1.f,
                   const float *Cin = nullptr, int64_t ldcin = 0, float beta = 0.f);

// Kernel instantiations (distinct symbols per phase for profilers).
enum : int {
  GEMM_OTHER = 0,
  GEMM_NAIVE_FWD = 5,
  GEMM_NAIVE_GRAD = 6,
  GEMM_NAIVE_UPDATE = 7
};

// Enqueue every descriptor of the batch (one main launch plus one reduce launch
// per split descriptor).  When gate is not null the kernels skip all writes if
// *gate != 0 at kernel start.
hipError_t gemm_launch(GemmBatch &b, const int *gate, hipStream_t s, int phase = GEMM_OTHER);

// Two-part form: gemm_prepare fills the tile bookkeeping (returns the tile
// count); gemm_enqueue launches without checking for errors.
int gemm_prepare(GemmBatch &b, int tile = 32);
void gemm_enqueue(const GemmBatch &b, const int *gate, hipStream_t s, int phase);

// Large single products on 128 x 128 tiles (the naive path).  gemm_big_ok: the
// operands meet the kernel's alignment needs (else use gemm_launch).  gemm_big_plan
// fills the tile counts and splits k over workgroups when the tiles are few, with
// at most partial_floats of partial sums.  gemm_big_launch also runs the reduce.
bool gemm_big_ok(const GemmDesc &g);
constexpr int kBigColsqRows = 4;  // colsq rows per 128-row tile
size_t gemm_big_plan(GemmDesc &g, int target_wgs, size_t partial_floats, float *partial);
hipError_t gemm_big_launch(GemmDesc g, const int *gate, hipStream_t s, int phase);

// Choose a split count for a long-k descriptor and attach its partial buffer.
// Returns the number of floats the partial buffer needs.
size_t gemm_plan_split(GemmDesc &g, int target_wgs, float *partial);

// ---------------------------------------------------------------------------
// The factored step (fused.hip): five launches on one stream.
//
// Op16: one product C = post(A opB) on 16 x 16 output tiles, k = K.  A is a plain
// operand (A(i,k) = A[i lda + k], or A[k lda + i] with tA) or, for the Q update's
// M, assembled as it is loaded (AM_MASM: 4 dq_i M^_ik dq_k + YY_ik + 2 dq_i HZ_ik +
// 2 dq_k HZ_ki; AM_MASM_S adds the dl/ds terms D ds_i ds_k + ds_i yb_k + yb_i ds_k).
// opB(k,j) = sum_t coef_t scale_t(k) B_t(k,j) over up to four terms
// (tr = 0: B_t[j ld + k]; tr = 1: B_t[k ld + j]).  Epilogue:
//   v = alpha lr^alpha_lr rs(i) cs(j) (acc + sum_t coef_t scale_t(i) Add_t[i ld + j]
//       + sum_r ux_r[i uxi_r] uy_r[j uyi_r]) + beta lr^beta_lr Cin_ij,
// stored to C (if any), C2 = 2 rs2(i) E_ij + v (if any), and the row partial sums
// (v Rr_ij, or |v|) of the tile's 16 columns to rowout[tile column][i].  The scale
// modes take dl/dq (SC_DQ) or its square root (SC_SQRT) of the index; coefficient
// indices select one of the Woodbury polynomial's c_k (-1: 1).
// ---------------------------------------------------------------------------
enum : int { SC_NONE = 0, SC_DQ = 1, SC_SQRT = 2 };
enum : int { RR_NONE = 0, RR_DOT = 1, RR_ABS = 2 };
enum : int { AM_PLAIN = 0, AM_MASM = 1, AM_MASM_S = 2 };
constexpr int kMaxTerms = 4;
constexpr int kMaxOps = 6;
constexpr int kMaxRank = 2;

struct OpTerm {
  const float *p;
  int64_t ld;
  int tr;
  int sc;
  int coef;
};

struct Op16 {
  int M, N, K;
  int tiles_m, tiles_n, tile_begin;
  int amode;
  const float *A;
  int64_t lda;
  int tA;
  const float *Mh, *HZ, *YY;
  int64_t ldm;
  int nb;
  OpTerm b[kMaxTerms];
  int nadd;
  OpTerm add[kMaxTerms];
  // rank-nuv addend sum_r ux_r[i uxi_r] uy_r[j uyi_r] (the dl/ds terms of Z^ and HZ)
  int nuv;
  const float *ux[kMaxRank], *uy[kMaxRank];
  int uxi[kMaxRank], uyi[kMaxRank];
  // AM_MASM_S: dl/ds (ds), y_bar (yb) and D of M's dl/ds terms
  const float *ds, *yb;
  float Dn;
  float alpha;
  int alpha_lr;
  int rs, cs;
  const float *Cin;
  int64_t ldcin;
  float beta;
  int beta_lr;
  float *C;
  int64_t ldc;
  float *C2;
  int64_t ldc2;
  const float *E;
  int64_t lde;
  int rs2;
  int rowred;
  const float *Rr;
  int64_t ldrr;
  float *rowout;
  // With qout: the last tile of each row block to finish (counted in qcnt[tile row],
  // which the next launch resets) sums the row partials into qout[i].
  float *qout;
  int *qcnt;
  int alt;  // >= 0: the descriptor used instead when the Woodbury polynomial is not certified
};

// The header fields come first and the tile ranges are repeated there, so that a
// workgroup finds its descriptor from one cache line.
struct OpBatch {
  int n;                 // descriptors (including alternates)
  int n_main;            // descriptors that own tiles (the first n_main)
  int total;             // tiles
  int begin[kMaxOps];    // op[q].tile_begin
  int count[kMaxOps];    // op[q]'s tiles
  Op16 op[kMaxOps];
};

// An OpBatch's tile ranges, passed to the kernels by value so that a workgroup finds its
// descriptor with one dependent load (of the descriptor itself) instead of two.
struct OpHdr {
  int n_main, total;
  int begin[kMaxOps], count[kMaxOps];
};
inline OpHdr op_hdr(const OpBatch &ob) {
  OpHdr h{};
  h.n_main = ob.n_main;
  h.total = ob.total;
  for (int q = 0; q < kMaxOps; ++q) {
    h.begin[q] = ob.begin[q];
    h.count[q] = ob.count[q];
  }
  return h;
}

// The products of one step for one minibatch size m (kept in device memory):
// ob[l] for launches 1..4 (16 x 16 tiles), gb_mid (the U update, launch 4) and
// gb_update (the Q and U^{-T} updates, launch 5) on 32 x 32 tiles.
struct StepPlan {
  OpBatch ob[4];
  // gb_contract, gb_zgrad: products of launches 1 and 3 on 32 x 32 tiles at large
  // shapes (else empty)
  GemmBatch gb_contract, gb_zgrad, gb_mid, gb_update;
};

// The context's state and workspace pieces the step uses.
struct StepBufs {
  int64_t D;
  int d, ldd, loss;
  float eps;
  float *V;
  int64_t ldv;
  float *U, *UinvT, *Q;
  float *WO;             // 2 x ldd: w_bar, omega (Taylor softmax; else null)
  float *Hhat, *Htil, *X, *G, *Atil, *W1, *P2, *P3, *RX, *Zq;  // m x d
  float *N, *Mhat, *HZ, *YY, *E2, *E4, *R, *Cwork;             // m x m
  float *qpart, *bpart;  // row partials: [ceil(d/16)][m], [ceil(m/16)][m]
  float *q, *tsum;       // m: q_j = h_j . h^_j, the sum of example j's valid target weights
  int *qcnt;             // ceil(m/16) arrival counters of the q reduction
  float *dq, *lvec;      // m
  float *dA, *wA, *sval; // m x K (dA: the naive path's only)
  int *srow, *scnt;      // m x K, m
  int *rcnt;             // m x K: the V scatter's per-row arrival counters (zero between steps)
  int *splan;            // 4 m x K: the V scatter's plan (meta, pos, sorted, tbl; launch 4)
  float *coef;           // 8
  int *cert;
  int *ticket;           // the V scatter's next partial-sum id (zeroed by launch 2)
  float *SW;             // m x 2: s_j = h_j . w_bar, h~_j = h_j . omega
  float *ds, *yb;        // m: dl/ds_j, y_bar_j = sum_k dl/dA_kj
  float *cwo;            // 2 x m: eta (2 dq s + D ds + y_bar), eta (2 dq h~ + ds)
  int *flag;
};

struct StepArgs {
  const float *H;
  int m;
  const int *idx;
  const float *val;
  int K;
  float lr;
  float *loss;
  float *gH;
};

void build_step_plan(const StepBufs &sb, int m, StepPlan &pl);

// Device memory carved in 256-byte aligned pieces (a null base only measures).
constexpr size_t kWsAlign = 256;
struct Carver {
  char *base;
  size_t off = 0;
  template <class T>
  T *take(size_t n) {
    off = (off + kWsAlign - 1) & ~(kWsAlign - 1);
    T *p = base ? reinterpret_cast<T *>(base + off) : nullptr;
    off += n * sizeof(T);
    return p;
  }
};
// The step's intermediates for up to m examples of up to K slots (api.hip).
void carve_step(StepBufs &b, float *&gradH, size_t m, size_t d, size_t K, Carver &cv);
// which = 0..4: launch which + 1 of the step.
void enqueue_step_launch(int which, const StepBufs &sb, const StepPlan &host, const StepPlan *dev,
                         const StepArgs &a, hipStream_t s);

// ---------------------------------------------------------------------------
// Non-step kernels (step_kernels.hip)
// ---------------------------------------------------------------------------
hipError_t launch_identity(hipStream_t s, float *A, int d, int64_t ld);
hipError_t launch_fill(hipStream_t s, float *p, float v);

// Naive-path kernels.  Column norms come as nparts partial sums partial[p][j]
// (from the forward product's epilogue, or from launch_colnorm, which also writes the
// partial column sums to psum when it is not null).
hipError_t launch_colnorm(hipStream_t s, const float *O, int64_t D, int m, float *partial,
                          float *psum, int nblk);
// w_bar = U^T (V^T 1_D) + D omega: nblk row blocks of V summed into part (nblk x d),
// then reduced and multiplied by U^T (U null: identity).  out must not alias part.
hipError_t launch_wbar(hipStream_t s, const float *V, int64_t ldv, int64_t D, int d,
                       const float *U, int ldd, const float *omega, float *part, int nblk,
                       float *out);
// Q += u omega^T + omega u^T + D omega omega^T with u = w_bar - D omega (the omega part
// of W^T W for W = V U + 1_D omega^T, given Q = (V U)^T (V U)).
hipError_t launch_q_omega(hipStream_t s, float *Q, int ldd, int d, int64_t D, const float *wbar,
                          const float *omega);
// psum (Taylor softmax): partial column sums of O (nparts x m, from launch_colnorm),
// giving s_j; dl/ds_j goes to ds.  Both null for the other losses.
hipError_t launch_naive_epilogue(hipStream_t s, int m, int K, int64_t D, int nparts,
                                 const float *partial, const float *psum, const float *O,
                                 const int *idx, const float *val, int loss, float eps, float *dq,
                                 float *ds, float *dA, float *lvec, int *flag);
// grad_O = 2 O diag(dq) + 1_D ds^T (ds may be null) + sum of dA at the targets, in place
// over O; also loss_out = sum_j lvec[j].
hipError_t launch_grad_o(hipStream_t s, float *O, int64_t D, int m, int K, const float *dq,
                         const float *ds, const int *idx, const float *dA, const float *lvec,
                         float *loss_out, int *flag);

// ---------------------------------------------------------------------------
// The sparse input layer of section 2.2 (input_layer.hip): A = X W1 and
// W1 -= eta X^T grad_A for m examples of K slots; status: a device int whose bit
// FLAG_INDEX is set for an index outside [-1, D_in) (the update then writes nothing).
// ---------------------------------------------------------------------------
hipError_t launch_input_forward(hipStream_t s, const float *W1, int64_t ldw, int64_t D_in, int d,
                                const int *idx, const float *val, int m, int K, float *A,
                                int *status);
hipError_t launch_input_update(hipStream_t s, float *W1, int64_t ldw, int64_t D_in, int d,
                               const int *idx, const float *val, int m, int K, const float *gA,
                               float lr, int *status);

// ---------------------------------------------------------------------------
// The online step (m = 1, squared error; Algorithm 2) as one launch
// (online.hip).  work: online_work_floats(d) floats; bar: a grid-barrier counter
// and its decision word (bar[0], bar[1]) that start at 0; spin_limit bounds the barrier's
// wait (polls) before the step is abandoned.
// ---------------------------------------------------------------------------
size_t online_work_floats(int d);
hipError_t launch_online_step(hipStream_t s, int64_t D, int d, int K, const float *h,
                              const int *idx, const float *val, float lr, float *V, int64_t ldv,
                              float *U, float *UinvT, float *Q, int ldd, float *loss_out,
                              float *grad_h, float *work, unsigned *bar, int spin_limit,
                              int *flag);

// ---------------------------------------------------------------------------
// Numerical stabilisation kernels (stabilize.hip), enqueued between steps.
// ---------------------------------------------------------------------------
// V <- V U in place (d <= 1024, else hipErrorInvalidValue).
hipError_t launch_restore(hipStream_t s, float *V, int64_t ldv, int64_t D, const float *U, int ldd,
                          int d);
// y0 = A0^T x0 and, if A1 is not null, y1 = A1^T x1, for d x d row-major matrices
// with row stride lda; part: 2 * 16 * d floats of partial sums.  y must not alias x.
hipError_t launch_tmatvec2(hipStream_t s, const float *A0, const float *A1, int lda, int d,
                           const float *x0, const float *x1, float *y0, float *y1, float *part);
// Algorithm 5's rank-one updates of U and U^{-T} (a = U^T u, b = (U^{-T})^T u) and
// of V, with the coefficients formed from the device scalar *sigma; a sigma that
// is not positive and finite skips both and sets FLAG_NONFINITE.
hipError_t launch_fix_state(hipStream_t s, float *U, float *UinvT, int ldd, int d, const float *u,
                            const float *a, const float *b, const float *sigma, float target,
                            int *flag);
hipError_t launch_fix_v(hipStream_t s, float *V, int64_t ldv, int64_t D, int d, const float *u,
                        const float *sigma, float target);
// out = S / trace(S) for a d x d S (row stride d); out must not alias S.
hipError_t launch_trace_scale(hipStream_t s, const float *S, int d, float *out);
// u_out = S u0 / ||S u0|| (S symmetric, row stride d), *sigma_out = ||A^T u_out||
// (which = 0) or its inverse; part: 16 * d floats.  u_out may alias u0.
hipError_t launch_power_finish(hipStream_t s, const float *S, int d, const float *u0,
                               const float *A, int lda, int which, float *u_out,
                               float *sigma_out, float *part);
// Y = U / (||U||_1 ||U||_inf), the from-scratch start of the Newton-Schulz
// iteration (*c receives the factor).
hipError_t launch_ns_start(hipStream_t s, const float *U, int ldd, int d, float *c, float *Y,
                           int ldy);
// E = I - Y U^T (d x d, row stride d) with fp64 accumulation.
hipError_t launch_residual64(hipStream_t s, const float *Y, int ldy, const float *U, int ldu, int d,
                             float *E);
// *amax = max_ij |E_ij| (E d x d, row stride d); *amax must be 0 on entry.
hipError_t launch_absmax(hipStream_t s, const float *E, int d, float *amax);

}  // namespace lst
