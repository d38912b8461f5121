/*
 * lst.h -- exact output-layer training step for very large sparse targets on gfx950.
 *
 * Method: Vincent, de Brebisson, Bouthillier, "Exact gradient updates in time
 * independent of output size for the spherical loss family" (arXiv 1606.08061).
 * The D x d output weights are kept factored as W = V U (section 3.2), or
 * W = V U + 1_D omega^T for losses that use s = sum(o) (eq. gen-Wfact), with the
 * bookkeeping matrices Q = W^T W (section 3.4), U^{-T} (eq. updateU-T, Woodbury
 * for minibatches, section 3.6 / 4.7) and w_bar = W^T 1_D (section 4.1.2).  One step (Algorithm 3 for
 * squared error, Algorithm 4 for the spherical family) computes the exact
 * minibatch loss, its gradient with respect to the hidden layer H and the full
 * gradient update of the implicit W in O(m d^2 + m^2 d + m^3 + m K d), touching
 * only the m*K target rows of V.  A naive O(D d) path with the same step
 * contract (sections 2.3 and 4.3) is provided for comparison.
 *
 * Conventions shared by every entry point
 *   - Memory: every float / int pointer is a DEVICE pointer owned by the caller
 *     (allocated with the HIP runtime, e.g. through PyTorch), except where a
 *     parameter says "host".  The library never allocates or frees device
 *     memory: a context works in a caller-owned workspace of
 *     lst_workspace_bytes (lst_naive_workspace_bytes) bytes, 256-byte aligned,
 *     that must stay allocated and untouched by the caller until lst_destroy.
 *     The context itself is a small host object.
 *   - Layout: row-major.  A minibatch H is m x d, one example per row (the same
 *     bytes as the paper's d x m H with one example per column).  V and W are
 *     D x d with row stride ldv / ldw >= d (floats); U, U^{-T} and Q are d x d
 *     with row stride ldd >= d; WO is 2 x d with row stride ldd, row 0 holding
 *     w_bar and row 1 omega.
 *   - Targets: idx and val are m x K (row stride K).  idx holds 0-based row
 *     indices in [0, D); -1 marks an empty slot (the paper's "at most K"
 *     non-zeros).  An index repeated inside one example adds its values
 *     (y = sum_k val_k onehot(idx_k)); repeated indices across examples are
 *     allowed and their V updates are summed in a fixed order.
 *   - Streams: every call is enqueued on the stream given at creation (a
 *     hipStream_t passed as void*; NULL = the null stream) and returns without
 *     synchronising, except lst_sync_status and lst_init_factored.  A context
 *     must not be used from two host threads at once.
 *   - Errors: every call returns an lst_status.  Argument errors detectable on
 *     the host are returned at once and nothing is enqueued.  Data-dependent
 *     errors found on the device (an index outside [-1, D), a Woodbury matrix
 *     that is not positive definite, a non-finite loss) set a sticky device
 *     flag: all later state writes of that step and of every following step
 *     are skipped, so V, U, U^{-T}, Q and WO keep the values they had before
 *     the failing step.  lst_sync_status reports and clears the flag.
 */
#ifndef LST_H
#define LST_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct lst_ctx lst_ctx;

/* Loss functions of the spherical family (section 4) implemented by the step. */
enum lst_loss {
  /* l = ||o - y||^2 (section 2.1); as a spherical loss q - 2 a.t + ||y||^2. */
  LST_LOSS_SQUARED = 0,
  /* l = -sum_k t_k log((o_{c_k}^2 + eps) / sum_i (o_i^2 + eps)), the spherical
     softmax named in section 4 (no definition is printed there; this is the
     reading used by the library, independent of sum(o)). */
  LST_LOSS_SPHERICAL_SOFTMAX = 1,
  /* l = -sum_k t_k log(f(o_{c_k}) / sum_i f(o_i)), f(x) = 1 + x + x^2/2: the
     Taylor softmax, also named in section 4 without a definition; read as the
     softmax with exp replaced by its second-order Taylor polynomial.  Since
     sum_i f(o_i) = D + s + q/2 it depends on s = sum(o): the step keeps omega and
     w_bar (eq. gen-Wfact, gen-update-omega, gen-update-wbar) and needs WO.  The
     target weights of an example must not sum to a negative value (dl/dq >= 0,
     which the Woodbury update needs). */
  LST_LOSS_TAYLOR_SOFTMAX = 2
};

enum lst_status {
  LST_OK = 0,
  LST_E_ARG = -1,       /* null pointer, bad enum, lr <= 0 or not finite, ... */
  LST_E_SHAPE = -2,     /* m > m_max, K > K_max, ld < d, D or d out of range   */
  LST_E_INDEX = -3,     /* (device) a target index outside [-1, D)             */
  LST_E_NOT_SPD = -4,   /* (device) the m x m Woodbury matrix is not positive
                           definite: the step is too large for the batch
                           (m = 1: 1 - 2 eta ||h||^2 <= 0, eq. updateU-T);
                           (host) U is numerically singular (section 5)       */
  LST_E_NONFINITE = -5, /* (device) the loss is NaN or infinite, or a singular
                           value given to fix-singular-value is not positive
                           and finite                                          */
  LST_E_HIP = -6,       /* a HIP runtime call failed                           */
  LST_E_STATE = -7,     /* wrong context kind for this call                    */
  LST_E_SYNC = -8       /* (device) the online step's bounded grid barrier
                           expired (its workgroups were not all resident); the
                           step wrote nothing                                  */
};

/* Limits of one context. */
#define LST_MAX_D ((int64_t)2147483647)
#define LST_MAX_d 4096
#define LST_MAX_M 1024
#define LST_MAX_K 64

/*
 * lst_workspace_bytes -- size in bytes of the device workspace lst_create needs for
 * these dimensions (the step's m x d, m x m and per-example intermediates, the
 * products' descriptors for up to 16 minibatch sizes, the section 5 scratch and the
 * split-k partial sums of the initial Q = V^T V).  0 if the arguments are invalid
 * (the checks of lst_create).
 */
size_t lst_workspace_bytes(int64_t D, int32_t d, int32_t m_max, int32_t K_max, int32_t loss);

/*
 * lst_create -- context for the factored step (Algorithm 3 / Algorithm 4).
 *   D, d         output size and hidden size (1 <= d <= LST_MAX_d, 1 <= D <= LST_MAX_D).
 *   m_max, K_max largest minibatch and largest number of target slots per
 *                example that lst_step will be given (<= LST_MAX_M, LST_MAX_K,
 *                m_max * K_max <= 8192).
 *   loss         an lst_loss value.
 *   eps          spherical softmax epsilon (> 0); ignored for squared error.
 *   V            D x ldv device buffer holding V (updated in place by lst_step).
 *   U, UinvT, Q  d x ldd device buffers (updated in place by lst_step).
 *   WO           2 x ldd device buffer: w_bar (row 0) and omega (row 1), updated
 *                in place by lst_step; needed by LST_LOSS_TAYLOR_SOFTMAX (else
 *                LST_E_ARG), unused by the other losses (may be NULL).
 *   workspace    device buffer of ws_bytes >= lst_workspace_bytes(D, d, m_max,
 *                K_max, loss) bytes, 256-byte aligned (LST_E_ARG if NULL or
 *                misaligned, LST_E_SHAPE if too small); cleared on the stream here.
 *   stream       hipStream_t as void*; every call is enqueued on it.
 * The buffers are borrowed: they must stay allocated until lst_destroy.  The
 * state they hold is not read here; call lst_init_factored before the first
 * step.  On success *out receives the context.
 */
int lst_create(lst_ctx **out, int64_t D, int32_t d, int32_t m_max, int32_t K_max, int32_t loss,
               float eps, float *V, int64_t ldv, float *U, float *UinvT, float *Q, float *WO,
               int32_t ldd, void *workspace, size_t ws_bytes, void *stream);

/* Options of a context (lst_set_option). */
enum lst_option {
  /* 1 (default for squared error): m = 1 squared-error steps run as the one-launch
     online step of Algorithm 2; 0: they take the general minibatch path. */
  LST_OPT_ONLINE_KERNEL = 0,
  /* Polls (0 .. 2^30, default 2^20) a workgroup of the online step waits at its
     grid barrier before the step is abandoned (nothing written, LST_E_SYNC at the
     next lst_sync_status).  Small values force that outcome, for testing it. */
  LST_OPT_SPIN_LIMIT = 1
};

/* lst_set_option -- sets an lst_option; LST_E_ARG for an unknown option or value. */
int lst_set_option(lst_ctx *c, int32_t option, int64_t value);

/*
 * lst_init_factored -- Algorithm 1 (and the general initialisation of section 4.8).
 *   V0 (D x ldv0, device) is copied into V when not NULL; NULL keeps V as it is.
 *   U0 (d x ldu0, device) is copied into U when not NULL; NULL sets U = I.
 * Then U^{-T} = inv(U)^T and Q = W^T W are computed (Q = V^T V when U = I), and
 * the sticky error flag is cleared.  For the Taylor softmax W = V U + 1_D omega^T
 * with omega read from row 1 of WO as the caller left it (zero for a fresh start,
 * as section 4.8 initialises it), and w_bar = W^T 1_D is written to row 0.  With U0 given, U is inverted
 * in fp64 on the host (LST_E_NOT_SPD if it is singular).  V^T V is split over D
 * into the workspace's partial sums.  Synchronises the stream.  Passing the current (V, U) re-derives the bookkeeping from scratch,
 * which is also how a run resumes from a (V, U) checkpoint.
 */
int lst_init_factored(lst_ctx *c, const float *V0, int64_t ldv0, const float *U0, int32_t ldu0);

/*
 * lst_step -- one minibatch step (Algorithm 3 for squared error, Algorithm 4
 * with dl/ds = 0 and omega = 0 for the spherical softmax).
 *   H        m x d device buffer, row stride d (one example per row).
 *   m        number of examples, 0 <= m <= m_max (m = 0 writes loss 0).
 *   idx, val m x K device buffers (int32 indices, float values), see above.
 *   K        slots per example, 0 <= K <= K_max.
 *   lr       learning rate eta > 0: W <- W - eta dL/dW.
 *   loss_dev device float receiving L = sum over the m examples.
 *   grad_H   m x d device buffer receiving dL/dH (row stride d); may be NULL.
 * State V, U, U^{-T}, Q is updated in place so that V U equals
 * W - eta dL/dW (eq. updateU / updateV, eq. gen-updateU / gen-updateV), Q equals
 * the new W^T W (eq. updateQ / gen-Qnew) and U^{-T} the new inverse transpose
 * (Woodbury, section 4.7: C = I - 2 eta S H^T H S is inverted as a certified
 * degree-7 Chebyshev polynomial in 2 eta S H^T H S on the matrix cores when the
 * bound ||(2 eta S H^T H S)^2||_inf^(1/2) proves it exact to below fp32 rounding,
 * else by exact elimination, whose pivots decide LST_E_NOT_SPD).  Five kernel
 * launches on the stream; returns once they are enqueued (the first call with a
 * new m also copies that m's product descriptors into the workspace, ordered on
 * the stream); device-side errors surface at the next lst_sync_status.
 * With m = 1 and squared error (the online case, Algorithm 2) the step runs as
 * one launch of 128 workgroups (its products read the old Q, U, U^{-T}, one
 * bounded grid-wide barrier with a single go/abort decision, then the rank-one
 * updates; 128 workgroups of 256 threads fit on the GPU at once), unless graphs
 * are on or LST_OPT_ONLINE_KERNEL is 0; same results to fp32 rounding.  Should the
 * barrier ever expire (workgroups kept from running by other work on the GPU),
 * the step writes nothing and lst_sync_status reports LST_E_SYNC.
 */
int lst_step(lst_ctx *c, const float *H, int32_t m, const int32_t *idx, const float *val,
             int32_t K, float lr, float *loss_dev, float *grad_H);

/*
 * lst_use_graphs -- off (default) or on.  When on, lst_step records the five
 * launches of a step as one HIP graph the first time it sees a given (H, idx,
 * val, loss_dev, grad_H, m, K, lr) and replays it whenever the same arguments
 * recur (up to 256 per context, least recently used evicted); the kernels and
 * results are the same as without graphs.  While the profiling hook is on, steps
 * are enqueued kernel by kernel.
 */
int lst_use_graphs(lst_ctx *c, int32_t on);

/*
 * lst_step_noalloc -- for callers that cannot allocate device memory (code under
 * stream capture, tight serving loops, hosts that forbid allocation): lst_step
 * without a context or workspace, on the same kernels.  The state (V, U, UinvT, Q,
 * as in lst_create) and the step's arguments (as in lst_step) are passed directly;
 * WO is needed for the Taylor softmax as in lst_create.  The step's descriptors
 * and intermediates live in a device array of 16 MiB that
 * the library holds on each GPU it runs on until the process ends.  The call
 * allocates and frees nothing.
 *   m, K         0 <= m <= LST_MAX_M, 0 <= K <= LST_MAX_K, m K <= 8192, and the
 *                step must fit the array: 4 (11 m d + 8 m^2) bytes plus about
 *                4 (m (d + m) / 16 + 8 m K + 13 m) + 22 KiB (with K = 5: m = 128 fits up
 *                to d = 2860, m = 256 up to d = 1287, m = 512 up to d = 361);
 *                LST_E_SHAPE beyond it.
 *   status_dev   device int32, set to 0 by the call, then ORed by the kernels with
 *                1 (a target index outside [-1, D)), 2 (the Woodbury matrix is not
 *                positive definite) or 4 (the loss is not finite); a nonzero value
 *                means the step changed no state.  Read it after the stream is done.
 *   stream       hipStream_t as void*; it must belong to the current device
 *                (LST_E_ARG otherwise), as must every buffer.
 * Every call on one GPU shares that GPU's array, which keeps the last call's
 * contents: calls that overlap on one GPU (different streams or host threads
 * without ordering between them) race and give wrong results; calls ordered on
 * one stream do not.  The first call on a device looks up the array's address
 * there; a call whose descriptors differ from the previous call's (another m, d,
 * K, loss or state buffers) rewrites them with a few extra small launches.
 * Results equal lst_step's on the same state (m = 1 takes the five-launch path).
 */
int lst_step_noalloc(int64_t D, int32_t d, int32_t loss, float eps, float *V, int64_t ldv, float *U,
                     float *UinvT, float *Q, float *WO, int32_t ldd, const float *H, int32_t m,
                     const int32_t *idx, const float *val, int32_t K, float lr, float *loss_dev,
                     float *grad_H, int32_t *status_dev, void *stream);

/*
 * lst_materialize_W -- W = V U (+ 1_D omega^T for the Taylor softmax) into a D x ldw
 * device buffer (section 5.1: the explicit weights, an O(D d^2) product).  For a
 * naive context, copies its W.
 */
int lst_materialize_W(lst_ctx *c, float *W, int64_t ldw);

/*
 * The sparse input layer (section 2.2), no context needed.  A minibatch of m inputs,
 * each K-sparse: idx, val are m x K device arrays (index -1 = empty slot; repeated
 * indices add their values), W1 is D_in x ldw (device, row-major), status_dev one
 * device int32 that the caller sets to 0 and the calls OR with LST_E_INDEX's device
 * bit (1) when an index lies outside [-1, D_in).  Both are enqueued on stream.
 *
 * lst_input_forward -- A = X W1: row j of A (m x d, row stride d) is
 * sum_k val[j,k] W1[idx[j,k]], an O(K d) gather per example; an invalid slot adds
 * nothing.
 */
int lst_input_forward(const float *W1, int64_t ldw, int64_t D_in, int32_t d, const int32_t *idx,
                      const float *val, int32_t m, int32_t K, float *A, int32_t *status_dev,
                      void *stream);

/*
 * lst_input_update -- W1 <- W1 - lr X^T grad_A (grad_A m x d, row stride d): only the
 * rows the inputs name change, each by one writer that sums its slots in slot order
 * (bit-reproducible).  Writes nothing if *status_dev is non-zero after the index
 * check (an invalid index in this call, or an error left in it by an earlier call).
 */
int lst_input_update(float *W1, int64_t ldw, int64_t D_in, int32_t d, const int32_t *idx,
                     const float *val, int32_t m, int32_t K, const float *grad_A, float lr,
                     int32_t *status_dev, void *stream);

/*
 * Numerical stabilisation (section 5), on a factored context, between steps.
 * Each call is enqueued on the context's stream after the steps before it
 * (lst_singular_stabilize synchronises it); none changes W = V U or Q = W^T W
 * beyond fp32 rounding.  Device-side errors surface at lst_sync_status.
 *
 * lst_restore_pristine -- section 5.1: V <- V U (in place, an O(D d^2) product on
 * the matrix cores), then U <- I and U^{-T} <- I (omega and w_bar unchanged).  Needs d <= 1024 (LST_E_SHAPE
 * otherwise).
 */
int lst_restore_pristine(lst_ctx *c);

/*
 * lst_refresh_uinvt -- section 5.3: U^{-T} recomputed from U, so that the drift
 * the rank-m updates accumulate in it is discarded.  Runs iters (1..100) rounds of
 * the Newton-Schulz iteration Y <- Y + E Y, E = I - Y U^T, with E accumulated in
 * fp64 and E Y an fp32 product on the matrix cores (mixed-precision refinement: the
 * result is the fp32 rounding of U^{-T} while cond(U) is below about 1e7).  Starts
 * from the carried U^{-T} (from_scratch = 0; converges if max |E| < 1, then each
 * round squares the error) or from U / (||U||_1 ||U||_inf) (from_scratch = 1:
 * converges for any invertible U, in about 2 log2(cond U) + 5 rounds).  resid_dev:
 * one device float receiving max_ij |(I - U^{-T} U^T)_ij| after the last round, or
 * NULL.  The paper recomputes by Gaussian elimination; the result is the same
 * inverse.
 */
int lst_refresh_uinvt(lst_ctx *c, int32_t iters, int32_t from_scratch, float *resid_dev);

/*
 * lst_power_iteration -- section 5.3: an extreme singular value of U and its left
 * singular vector by 2^log2_iters (0..30) power iterations u <- A A^T u / ||A A^T u||
 * from u0: A = U for the largest (which = 0), A = U^{-T} for the smallest (which =
 * 1; sigma = 1 / ||U^{-1} u||).  The iterations are carried out as log2_iters
 * squarings of A A^T on the matrix cores.  u0, u_out: d device floats (may alias);
 * u_out receives the unit vector, sigma_out (one device float) the singular value.
 * which = 1 uses the carried U^{-T}: refresh it first if it may have drifted.
 */
int lst_power_iteration(lst_ctx *c, int32_t which, int32_t log2_iters, const float *u0,
                        float *u_out, float *sigma_out);

/*
 * lst_fix_singular_value -- Algorithm 5, fix-singular-value: the singular value
 * s = *sigma_dev (device float) of U along its left singular vector u (d device
 * floats, unit norm) becomes target (> 0): with a = (target - s) / s and
 * b = -a / (1 + a), U <- U + a u (U^T u)^T, V <- V + b (V u) u^T (one pass over V)
 * and U^{-T} <- U^{-T} + b u (U^{-1} u)^T.  If *sigma_dev is not positive and
 * finite, nothing changes and lst_sync_status reports LST_E_NONFINITE.
 */
int lst_fix_singular_value(lst_ctx *c, const float *u, const float *sigma_dev, float target);

/*
 * lst_singular_stabilize -- the procedure of section 5.3 around Algorithm 5:
 * U^{-T} recomputed first (lst_refresh_uinvt: two rounds from the carried value if
 * its residual max |I - U^{-T} U^T| is below 1/4, else rounds from scratch until it
 * is, then two more; LST_E_NOT_SPD if 96 rounds do not get there, U being
 * numerically singular), then, while the smallest singular value of U
 * (lst_power_iteration, which = 1) is below lo and fewer than max_fixes corrections
 * have been made, it is set to 1; then the same for the largest (which = 0) above
 * hi.  Every search starts from u0 (d device floats) with 2^log2_iters iterations.
 * Host outputs: n_fixed[0], n_fixed[1] the corrections of the smallest and of the
 * largest; sigmas[0], sigmas[1] the last smallest and largest singular values
 * found.  Synchronises the stream after each search; LST_E_NONFINITE if a search
 * returns a value that is not positive and finite.  The paper suggests a safe
 * range of [0.001, 100] checked every 100 steps.
 */
int lst_singular_stabilize(lst_ctx *c, float lo, float hi, int32_t log2_iters, const float *u0,
                           int32_t max_fixes, int32_t *n_fixed, float *sigmas);

/*
 * lst_sync_status -- synchronises the context's stream, returns the sticky
 * device error (LST_OK if none) and clears it.  Also returns LST_E_HIP if a
 * kernel launch or the synchronisation failed.  After LST_E_SYNC it also resets
 * the online step's barrier counter.
 */
int lst_sync_status(lst_ctx *c);

/* lst_status_string -- static, human-readable name of a status code. */
const char *lst_status_string(int status);

/* lst_destroy -- synchronises the stream and frees the context (the caller then
   owns its workspace again). */
void lst_destroy(lst_ctx *c);

/* lst_naive_workspace_bytes -- workspace bytes of lst_naive_create (the D x m
   output and its column-norm and split-k partial sums); 0 for invalid arguments. */
size_t lst_naive_workspace_bytes(int64_t D, int32_t d, int32_t m_max, int32_t K_max,
                                 int32_t loss);

/*
 * lst_naive_create -- context for the naive O(D d) step of sections 2.3 / 4.3:
 * O = W H^T (D x m) on MFMA, the loss over the full output, grad_H = W^T grad_O
 * and W <- W - eta grad_O H, with W held explicitly.
 *   W      D x ldw device buffer, updated in place by lst_naive_step.
 *   workspace, ws_bytes  as in lst_create, sized by lst_naive_workspace_bytes.
 *   Other arguments as in lst_create.
 */
int lst_naive_create(lst_ctx **out, int64_t D, int32_t d, int32_t m_max, int32_t K_max,
                     int32_t loss, float eps, float *W, int64_t ldw, void *workspace,
                     size_t ws_bytes, void *stream);

/* lst_naive_step -- same contract as lst_step, on a naive context. */
int lst_naive_step(lst_ctx *c, const float *H, int32_t m, const int32_t *idx, const float *val,
                   int32_t K, float lr, float *loss_dev, float *grad_H);

/* Phases of a step, as timed by the profiling hook below: the five launches of a
   factored step, the naive step's parts and the online step. */
enum lst_phase {
  LST_PHASE_CONTRACT = 0,      /* H^ = Q H, H~ = U H, X = U^{-T} H, N = H^T H (matrix cores)  */
  LST_PHASE_GATHER = 1,        /* gather of the K target rows of V, loss epilogue, G; H^T H^,
                                  E^2 and E Xs of the Woodbury polynomial                    */
  LST_PHASE_ZGRAD = 2,         /* Z^ = U^T G, grad_H, H~^T G, E^2 Xs, E^3 Xs, E^4, Yring^T
                                  Yring, the loss sum, the certificate (or exact inverse)    */
  LST_PHASE_MID = 3,           /* (eta^2/2) M H - eta grad_H, R X, the U update              */
  LST_PHASE_UPDATE = 4,        /* the U^{-T} and Q updates and the V scatter                 */
  LST_PHASE_NAIVE_FWD = 5,     /* naive: O = W H^T                                           */
  LST_PHASE_NAIVE_LOSS = 6,    /* naive: column norms of O, loss, grad_O                     */
  LST_PHASE_NAIVE_GRAD = 7,    /* naive: grad_H = grad_O^T W                                 */
  LST_PHASE_NAIVE_UPDATE = 8,  /* naive: W <- W - eta grad_O H                               */
  LST_PHASE_ONLINE = 9,        /* m = 1, squared error: the whole step in one launch         */
  LST_NUM_PHASES = 10
};

/*
 * lst_profile_enable -- tracing hook.  While on (on != 0), steps are enqueued
 * without HIP graphs and each phase's kernels are launched with a pair of HIP
 * events attached to the launches themselves (start of the phase's first kernel,
 * end of its last kernel), so the recorded time is the phases' GPU execution time
 * without launch gaps.  Turning it on clears earlier records.
 */
int lst_profile_enable(lst_ctx *c, int32_t on);

/*
 * lst_profile_read -- synchronises the stream and, for phases 0..n-1 (n <=
 * LST_NUM_PHASES), writes to host arrays counts[p] = number of timed launches
 * and ms[p] = their summed duration in milliseconds since the last enable/read;
 * then clears the records.  At most 65536 launches per phase are recorded.
 */
int lst_profile_read(lst_ctx *c, int32_t *counts, double *ms, int32_t n);

#ifdef __cplusplus
}
#endif

#endif /* LST_H */
