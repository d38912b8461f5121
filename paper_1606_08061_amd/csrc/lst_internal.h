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
// Ordering between the step's two streams without host events: monotone
// progress counters in device memory.  A kernel given a StepSync adds 1 to
// *sig from its workgroup 0 on entry ("every kernel before me on my stream has
// completed") and, if wx is set, waits until *wx - *wy >= wd (thread 0 polls,
// then the workgroup acquires).  Waits are placed in single-workgroup kernels
// only.  A producer publishes its results with release_count at its end.
// The wait is bounded (a few tenths of a second); when it expires it sets
// FLAG_SYNC, which also closes the gated state updates, and the kernel goes on,
// so no wave waits forever.
// ---------------------------------------------------------------------------
struct StepSync {
  const int *wx = nullptr, *wy = nullptr;
  int wd = 0;
  int *sig = nullptr;
  int *flag = nullptr;
};

constexpr int kSyncSpinLimit = 1 << 18;

__device__ inline void step_sync_begin(const StepSync &s) {
  if (s.sig && blockIdx.x == 0 && threadIdx.x == 0)
    __hip_atomic_fetch_add(s.sig, 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
  if (!s.wx) return;
  if (threadIdx.x == 0) {
    // relaxed polls (coherent loads, no cache invalidation per poll), one acquire after
    for (int it = 0;; ++it) {
      const int x = __hip_atomic_load(s.wx, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const int y = __hip_atomic_load(s.wy, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if ((int)((unsigned)x - (unsigned)y) >= s.wd) break;
      if (it >= kSyncSpinLimit) {
        atomicOr(s.flag, FLAG_SYNC);
        break;
      }
      __builtin_amdgcn_s_sleep(2);
    }
  }
  __syncthreads();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
}

// Called by every thread of the (single) producing workgroup after its last write.
__device__ inline void release_count(int *cnt) {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
  __syncthreads();
  if (threadIdx.x == 0) __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}

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
  int lr_scaled;  // alpha *= lr^2 and beta *= lr at launch (plans shared across lr)
  // 128 x 128-tile kernel without split: when set, also writes per-column partial
  // sums of squares of the product, colsq[p][j] for p < 4 * tiles_m (each the sum
  // over 32 of the tile's rows of C[i,j]^2 before alpha/beta).
  float *colsq;
};

// Operand placeholders of plans kept in device memory: a plan is built once per
// minibatch size m and refers to the step's H and grad_H through these values,
// which the kernel replaces by the pointers passed at launch.
inline const float *sym_H() { return reinterpret_cast<const float *>(uintptr_t{16}); }
inline float *sym_gradH() { return reinterpret_cast<float *>(uintptr_t{32}); }

constexpr int kMaxBatch = 4;

struct GemmBatch {
  GemmDesc d[kMaxBatch];
  int n;
  int total_tiles;
  int wide;  // 8 wavefronts per tile (long k) instead of 4
  int t16;   // 16 x 16 output tiles (plans): set before gemm_prepare
  // Optional prefetch (16 x 16 plans): pf_m extra workgroups after the tiles
  // (whose count is padded to pf_base, a multiple of 8, so that workgroup
  // pf_base + j shares an XCD with workgroup j of the next launch) read the K
  // target rows of example j of V (D x ldv) into the caches.
  const float *pf_V;
  int64_t pf_D, pf_ldv;
  int pf_m, pf_d, pf_base;
};

GemmDesc gemm_desc(int M, int N, int K, const float *A, int64_t lda, int tA, const float *B,
                   int64_t ldb, int tB, float *C, int64_t ldc, float alpha = 1.f,
                   const float *Cin = nullptr, int64_t ldcin = 0, float beta = 0.f);

// Kernel instantiations (distinct symbols per step phase for profilers).
enum : int {
  GEMM_OTHER = 0,
  GEMM_CONTRACT = 1,
  GEMM_ZGRAD = 2,
  GEMM_MID = 3,
  GEMM_UPDATE = 4,
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
int gemm_prepare(GemmBatch &b);
void gemm_enqueue(const GemmBatch &b, const int *gate, hipStream_t s, int phase);

// Launch of a prepared batch whose identical copy `dev` lives in device memory
// (no split-k): the kernel reads its descriptors from there and takes H, grad_H
// and lr for the placeholders, so the launch carries a few dozen bytes of
// arguments instead of the whole batch.
void gemm_enqueue_plan(const GemmBatch &host, const GemmBatch *dev, const float *H,
                       float *gradH, float lr, const int *gate, hipStream_t s, int phase,
                       const int *pf_idx = nullptr, int pf_K = 0, const StepSync &sync = {});

// The same launch for a plan of 32 x 32 tiles without split-k, with n more
// workgroups that each run one target slot of the V scatter (V_r -= slr sum
// dl/dA P_j over the row's slots).  Returns false, launching nothing, if the
// plan does not qualify.
bool gemm_enqueue_plan_scatter(const GemmBatch &host, const GemmBatch *dev, const float *H,
                               float *gradH, float lr, const int *gate, hipStream_t s, int n,
                               int K, int d, float slr, const int *idx, const float *dA,
                               const float *P, float *V, int64_t ldv);

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
// Step kernels (step_kernels.hip)
// ---------------------------------------------------------------------------
hipError_t launch_gather(hipStream_t s, int m, int K, int d, int64_t D, const float *H,
                         const float *Hhat, const float *Htil, const int *idx, const float *val,
                         const float *V, int64_t ldv, int loss, float eps, float lr, float *G,
                         float *Atil, float *dq, float *dA, float *lvec, int *flag);

// m <= kWoodburyOneWG: one workgroup.  Larger m: blocked in kBigBlock-row steps
// through Cwork (m x m), Pbig (2 kBigBlock^2), Cp (m x kBigBlock) and Rp (kBigBlock x m).
constexpr int kWoodburyOneWG = 128;
constexpr int kBigBlock = 128;
// wait: ordering before the first kernel reads dq; done: counter released after
// R is written (also when the matrix was rejected).
hipError_t launch_woodbury(hipStream_t s, int m, float lr, int unit_dq, const float *dq,
                           const float *N, float *R, float *Cwork, float *Pbig, float *Cp,
                           float *Rp, int *flag, const StepSync &wait, int *done);

// The m > d form of the branch (push-through identity): Hs = diag(dq)^(1/2) H (m x d,
// flagging dq < 0), and R = 2 eta S (R0 + I) S in place over R0 = Hs R' Hs^T (m x m).
hipError_t launch_scale_rows_sqrt(hipStream_t s, int m, int d, const float *H, const float *dq,
                                  float *Hs, int *flag);
hipError_t launch_push_through_r(hipStream_t s, int m, float lr, int unit_dq, const float *dq,
                                 float *R);

// One workgroup: waits as `wait` says, then releases *done (if not null).
hipError_t launch_step_sync(hipStream_t s, const StepSync &wait, int *done);

hipError_t launch_mblock(hipStream_t s, int m, int K, const int *idx, const float *lvec,
                         const float *dq, const float *dA, const float *Mhat, const float *HZ,
                         float *M, float *loss_out, int *flag);

hipError_t launch_scatter(hipStream_t s, int m, int K, int d, float lr, const int *idx,
                          const float *dA, const float *P, float *V, int64_t ldv, const int *flag);

hipError_t launch_identity(hipStream_t s, float *A, int d, int64_t ld);
hipError_t launch_fill(hipStream_t s, float *p, float v);

// Naive-path kernels.  Column norms come as nparts partial sums partial[p][j]
// (from the forward product's epilogue, or from launch_colnorm).
hipError_t launch_colnorm(hipStream_t s, const float *O, int64_t D, int m, float *partial,
                          int nblk);
hipError_t launch_naive_epilogue(hipStream_t s, int m, int K, int64_t D, int nparts,
                                 const float *partial, const float *O, const int *idx,
                                 const float *val, int loss, float eps, float *dq, float *dA,
                                 float *lvec, int *flag);
// grad_O = 2 O diag(dq) + sum of dA at the targets, in place over O; also
// loss_out = sum_j lvec[j].
hipError_t launch_grad_o(hipStream_t s, float *O, int64_t D, int m, int K, const float *dq,
                         const int *idx, const float *dA, const float *lvec, float *loss_out,
                         int *flag);

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
// that starts at 0 and is reset together with the step's progress counters.
// ---------------------------------------------------------------------------
size_t online_work_floats(int d);
hipError_t launch_online_step(hipStream_t s, int64_t D, int d, int K, const float *h,
                              const int *idx, const float *val, float lr, float *V, int64_t ldv,
                              float *U, float *UinvT, float *Q, int ldd, float *loss_out,
                              float *grad_h, float *work, unsigned *bar, int *flag);

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
