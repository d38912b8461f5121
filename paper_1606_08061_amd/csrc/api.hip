// C ABI of liblst: argument validation, workspace carving and the enqueue order
// of the factored step (Algorithm 3 / Algorithm 4) and of the naive step.
#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <memory>
#include <mutex>
#include <new>
#include <vector>

#include "lst_internal.h"

using namespace lst;

namespace lst {
thread_local ProfHook g_prof;

// The step's intermediates for minibatches of up to m examples with up to K slots
// each (m x d, m x m, per-example and per-slot pieces), and grad_H's stand-in for
// steps given no grad_H buffer.
void carve_step(StepBufs &b, float *&gradH, size_t m, size_t d, size_t K, Carver &cv) {
  const size_t md = m * d, mm = m * m, mk = m * (K > 0 ? K : 1);
  b.Hhat = cv.take<float>(md);
  b.Htil = cv.take<float>(md);
  b.X = cv.take<float>(md);
  b.G = cv.take<float>(md);
  b.Atil = cv.take<float>(md);
  b.W1 = cv.take<float>(md);
  b.P2 = cv.take<float>(md);
  b.P3 = cv.take<float>(md);
  b.RX = cv.take<float>(md);
  b.Zq = cv.take<float>(md);
  gradH = cv.take<float>(md);
  b.N = cv.take<float>(mm);
  b.Mhat = cv.take<float>(mm);
  b.HZ = cv.take<float>(mm);
  b.YY = cv.take<float>(mm);
  b.E2 = cv.take<float>(mm);
  b.E4 = cv.take<float>(mm);
  b.R = cv.take<float>(mm);
  b.Cwork = cv.take<float>(mm);
  b.qpart = cv.take<float>((d + 15) / 16 * m);
  b.bpart = cv.take<float>((m + 15) / 16 * m);
  b.q = cv.take<float>(m);
  b.tsum = cv.take<float>(m);
  b.qcnt = cv.take<int>((m + 15) / 16);
  b.dq = cv.take<float>(m);
  b.lvec = cv.take<float>(m);
  b.rcnt = cv.take<int>(mk);
  b.splan = cv.take<int>(4 * mk);
  b.wA = cv.take<float>(mk);
  b.sval = cv.take<float>(mk);
  b.srow = cv.take<int>(mk);
  b.scnt = cv.take<int>(m);
  b.coef = cv.take<float>(8);
  b.cert = cv.take<int>(2);  // the certificate, then the scatter's ticket
  b.ticket = b.cert ? b.cert + 1 : nullptr;
  b.SW = cv.take<float>(2 * m);
  b.ds = cv.take<float>(m);
  b.yb = cv.take<float>(m);
  b.cwo = cv.take<float>(2 * m);
}
}  // namespace lst

namespace {

enum : int { KIND_FACTORED = 1, KIND_NAIVE = 2 };
constexpr int kTargetWGs = 1024;  // workgroups a split-k GEMM aims for
constexpr int kColnormBlocks = 1024;
constexpr size_t kInitPartialCap = size_t(8) << 20;  // floats of split-k partials for Q = V^T V
constexpr int kWbarBlocks = 256;                    // row blocks of the column sums V^T 1_D
constexpr int kDefaultSpin = 1 << 20;               // polls of the online step's barrier


// A factored step recorded as a HIP graph, replayed when the same arguments recur.
struct GraphEntry {
  const void *H, *idx, *val;
  void *loss, *grad;
  int m, K;
  uint32_t lr_bits;
  hipGraphExec_t exec;
  uint64_t last_use;
};
constexpr size_t kGraphCap = 256;

// The step's products for one minibatch size m: host copy and its device slot.
constexpr size_t kPlanCap = 16;
struct PlanEntry {
  int m;
  std::unique_ptr<StepPlan> host;
  StepPlan *dev;
  uint64_t last_use;
};

}  // namespace

struct lst_ctx {
  int kind;
  int64_t D;
  int d, m_max, K_max, loss;
  float eps;
  hipStream_t stream;
  // factored state (borrowed)
  float *V;
  int64_t ldv;
  float *U, *UinvT, *Q;
  float *WO;  // w_bar, omega (Taylor softmax)
  int ldd;
  // naive state (borrowed)
  float *W;
  int64_t ldw;
  // workspace (borrowed from the caller)
  void *ws;
  size_t ws_bytes;
  StepBufs sb;
  float *gradH;  // grad_H when the caller passes none
  // section 5 stabilisation: two d x d scratch matrices (row stride d), four
  // d-vectors, the partial sums of two matrix-vector products (32 d; also the
  // online step's work vectors) and eight scalars
  float *Sd0, *Sd1, *svec, *spart, *sscal;
  float *initpart;  // split-k partial sums of Q = V^T V (lst_init_factored)
  size_t initpart_floats;
  float *wpart;     // row-block column sums of V for w_bar (Taylor softmax)
  int *flag;
  int *cnt;  // [0] the online step's grid-barrier counter, [1] its decision word
  float *O, *colpart, *colsum, *splitpart;
  hipError_t last_err;
  hipStream_t cap;  // stream a step is captured on when it is recorded as a HIP graph
  bool have_cap;
  // tracing: event pairs per phase
  bool prof_on;
  std::vector<hipEvent_t> prof_ev[LST_NUM_PHASES];
  int prof_used[LST_NUM_PHASES];
  std::vector<PlanEntry> plans;
  StepPlan *plan_pool;
  uint64_t plan_tick;
  bool use_graphs;
  std::vector<GraphEntry> graphs;
  uint64_t graph_tick;
  // options (lst_set_option)
  bool online;     // m = 1 squared-error steps as one launch
  int spin_limit;  // bound of the online step's barrier wait
};

namespace {

bool finite_pos(float x) { return std::isfinite(x) && x > 0.f; }

// Floats of split-k partials for Q = V^T V: as many splits as the GEMM would take,
// capped at kInitPartialCap floats (fewer splits beyond it).
size_t init_partial_floats(int64_t D, int d) {
  GemmDesc g = gemm_desc(d, d, (int)D, nullptr, d, 1, nullptr, d, 1, nullptr, d);
  const size_t want = gemm_plan_split(g, kTargetWGs, nullptr);
  return std::min(want, kInitPartialCap / ((size_t)d * d) * ((size_t)d * d));
}

void carve_factored(lst_ctx *c, Carver &cv) {
  const size_t d = (size_t)c->d;
  carve_step(c->sb, c->gradH, (size_t)c->m_max, d, (size_t)c->K_max, cv);
  c->Sd0 = cv.take<float>(d * d);
  c->Sd1 = cv.take<float>(d * d);
  c->svec = cv.take<float>(4 * d);
  c->spart = cv.take<float>(std::max<size_t>(32 * d, online_work_floats(c->d)));
  c->sscal = cv.take<float>(8);
  c->initpart_floats = init_partial_floats(c->D, c->d);
  c->initpart = cv.take<float>(c->initpart_floats);
  c->wpart = c->loss == LST_LOSS_TAYLOR_SOFTMAX ? cv.take<float>((size_t)kWbarBlocks * d) : nullptr;
  c->flag = cv.take<int>(1);
  c->cnt = cv.take<int>(4);
  c->plan_pool = cv.take<StepPlan>(kPlanCap);
  c->sb.flag = c->flag;
}

// Upper bound of the split-k partial buffer of grad_H = grad_O^T W for any m <= m_max:
// gemm_plan_split keeps splits <= ceil(kTargetWGs / tiles), and m * d <= tiles * 1024.
// The 128 x 128-tile kernel's bound is the same with 128^2 floats per tile.
size_t naive_split_floats(const lst_ctx *c) {
  const size_t tiles = (size_t)((c->m_max + 31) / 32) * ((c->d + 31) / 32);
  const size_t tiles128 = (size_t)((c->m_max + 127) / 128) * ((c->d + 127) / 128);
  const size_t a = (kTargetWGs + tiles) * 1024, b = (kTargetWGs + tiles128) * 16384;
  return a > b ? a : b;
}

// One naive-path product: the 128 x 128-tile kernel when the operands allow it,
// else the general one.  split: spread k over workgroups (grad_H's k = D).
hipError_t naive_gemm(lst_ctx *c, GemmDesc g, bool split, const int *gate, hipStream_t s,
                      int phase) {
  if (gemm_big_ok(g)) {
    gemm_big_plan(g, kTargetWGs, split ? naive_split_floats(c) : 0, split ? c->splitpart : nullptr);
    return gemm_big_launch(g, gate, s, phase);
  }
  if (split) gemm_plan_split(g, kTargetWGs, c->splitpart);
  GemmBatch b{};
  b.d[0] = g;
  b.n = 1;
  return gemm_launch(b, gate, s, phase);
}

void carve_naive(lst_ctx *c, Carver &cv) {
  const size_t md = (size_t)c->m_max * c->d;
  const size_t mk = (size_t)c->m_max * (c->K_max > 0 ? c->K_max : 1);
  c->O = cv.take<float>((size_t)c->D * c->m_max);
  const size_t parts128 = (size_t)kBigColsqRows * ((c->D + 127) / 128);
  c->colpart = cv.take<float>((parts128 > kColnormBlocks ? parts128 : kColnormBlocks) * c->m_max);
  c->splitpart = cv.take<float>(naive_split_floats(c));
  c->gradH = cv.take<float>(md);
  c->sb.dq = cv.take<float>(c->m_max);
  c->sb.lvec = cv.take<float>(c->m_max);
  c->sb.dA = cv.take<float>(mk);
  if (c->loss == LST_LOSS_TAYLOR_SOFTMAX) {  // column sums of O for s_j, and dl/ds
    c->colsum = cv.take<float>((size_t)kColnormBlocks * c->m_max);
    c->sb.ds = cv.take<float>(c->m_max);
  }
  c->flag = cv.take<int>(1);
}

int common_args(int64_t D, int32_t d, int32_t m_max, int32_t K_max, int32_t loss, float eps) {
  if (loss != LST_LOSS_SQUARED && loss != LST_LOSS_SPHERICAL_SOFTMAX &&
      loss != LST_LOSS_TAYLOR_SOFTMAX)
    return LST_E_ARG;
  if (loss == LST_LOSS_SPHERICAL_SOFTMAX && !finite_pos(eps)) return LST_E_ARG;
  if (D < 1 || D > LST_MAX_D || d < 1 || d > LST_MAX_d) return LST_E_SHAPE;
  if (m_max < 1 || m_max > LST_MAX_M || K_max < 0 || K_max > LST_MAX_K) return LST_E_SHAPE;
  if ((int64_t)m_max * K_max > 8192) return LST_E_SHAPE;
  return LST_OK;
}

// The bytes a context's carve takes (plus alignment slack for an aligned base).
size_t ws_size(int kind, int64_t D, int32_t d, int32_t m_max, int32_t K_max, int32_t loss) {
  lst_ctx probe{};
  probe.kind = kind;
  probe.D = D;
  probe.d = d;
  probe.m_max = m_max;
  probe.K_max = K_max;
  probe.loss = loss;
  Carver cv{nullptr};
  if (kind == KIND_FACTORED)
    carve_factored(&probe, cv);
  else
    carve_naive(&probe, cv);
  return (cv.off + kWsAlign - 1) & ~(kWsAlign - 1);
}

// Takes the caller's workspace: checks its size and alignment, carves it and clears
// it on the stream (the error flag and counters start at zero).
int take_ws(lst_ctx *c, void *ws, size_t ws_bytes, void (*carve)(lst_ctx *, Carver &)) {
  const size_t need = ws_size(c->kind, c->D, c->d, c->m_max, c->K_max, c->loss);
  if (!ws) return LST_E_ARG;
  if ((reinterpret_cast<uintptr_t>(ws) & (kWsAlign - 1)) != 0) return LST_E_ARG;
  if (ws_bytes < need) return LST_E_SHAPE;
  c->ws = ws;
  c->ws_bytes = need;
  Carver real{static_cast<char *>(ws)};
  carve(c, real);
  if (hipMemsetAsync(ws, 0, need, c->stream) != hipSuccess) return LST_E_HIP;
  return LST_OK;
}

int step_args(const lst_ctx *c, const float *H, int32_t m, const int32_t *idx, const float *val,
              int32_t K, float lr, const float *loss_dev) {
  if (!loss_dev) return LST_E_ARG;
  if (m < 0 || m > c->m_max || K < 0 || K > c->K_max) return LST_E_SHAPE;
  if (m > 0 && !H) return LST_E_ARG;
  if (m > 0 && K > 0 && (!idx || !val)) return LST_E_ARG;
  if (!finite_pos(lr)) return LST_E_ARG;
  return LST_OK;
}

int record(lst_ctx *c, hipError_t e) {
  if (e != hipSuccess) {
    c->last_err = e;
    return LST_E_HIP;
  }
  return LST_OK;
}

constexpr int kProfCap = 65536;

// Records the start (begin=true) or the end of a phase when profiling is on.
// Phase timing: begin hands a fresh event pair to the launch hook (see
// LST_LAUNCH); end withdraws it and keeps the pair if a kernel consumed it.
void prof(lst_ctx *c, int phase, bool begin) {
  if (!c->prof_on) return;
  int &used = c->prof_used[phase];
  if (!begin) {
    const bool launched = g_prof.stop != nullptr && g_prof.start == nullptr;
    g_prof = ProfHook{};
    if (launched) ++used;
    return;
  }
  g_prof = ProfHook{};
  if (used >= kProfCap) return;
  std::vector<hipEvent_t> &ev = c->prof_ev[phase];
  while (ev.size() < 2 * (size_t)used + 2) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) {
      c->prof_on = false;
      return;
    }
    ev.push_back(e);
  }
  g_prof.start = ev[2 * (size_t)used];
  g_prof.stop = ev[2 * (size_t)used + 1];
}

void graphs_free(lst_ctx *c) {
  for (GraphEntry &g : c->graphs)
    if (g.exec) (void)hipGraphExecDestroy(g.exec);
  c->graphs.clear();
}

void prof_free(lst_ctx *c) {
  for (int p = 0; p < LST_NUM_PHASES; ++p) {
    for (hipEvent_t e : c->prof_ev[p]) (void)hipEventDestroy(e);
    c->prof_ev[p].clear();
    c->prof_used[p] = 0;
  }
}

// fp64 Gauss-Jordan with partial pivoting (init only): returns false if singular.
bool invert_host(std::vector<double> &a, int n, std::vector<double> &inv) {
  inv.assign((size_t)n * n, 0.0);
  for (int i = 0; i < n; ++i) inv[(size_t)i * n + i] = 1.0;
  for (int k = 0; k < n; ++k) {
    int p = k;
    double best = std::fabs(a[(size_t)k * n + k]);
    for (int i = k + 1; i < n; ++i)
      if (std::fabs(a[(size_t)i * n + k]) > best) {
        best = std::fabs(a[(size_t)i * n + k]);
        p = i;
      }
    if (!(best > 0.0) || !std::isfinite(best)) return false;
    if (p != k)
      for (int j = 0; j < n; ++j) {
        std::swap(a[(size_t)k * n + j], a[(size_t)p * n + j]);
        std::swap(inv[(size_t)k * n + j], inv[(size_t)p * n + j]);
      }
    const double ip = 1.0 / a[(size_t)k * n + k];
    for (int j = 0; j < n; ++j) {
      a[(size_t)k * n + j] *= ip;
      inv[(size_t)k * n + j] *= ip;
    }
    for (int i = 0; i < n; ++i) {
      if (i == k) continue;
      const double f = a[(size_t)i * n + k];
      if (f == 0.0) continue;
      for (int j = 0; j < n; ++j) {
        a[(size_t)i * n + j] -= f * a[(size_t)k * n + j];
        inv[(size_t)i * n + j] -= f * inv[(size_t)k * n + j];
      }
    }
  }
  return true;
}

lst_ctx *new_ctx(int kind, int64_t D, int32_t d, int32_t m_max, int32_t K_max, int32_t loss,
                 float eps, void *stream) {
  lst_ctx *c = new (std::nothrow) lst_ctx{};
  if (!c) return nullptr;
  c->kind = kind;
  c->D = D;
  c->d = d;
  c->m_max = m_max;
  c->K_max = K_max;
  c->loss = loss;
  c->eps = eps;
  c->stream = static_cast<hipStream_t>(stream);
  c->last_err = hipSuccess;
  c->online = loss == LST_LOSS_SQUARED;
  c->spin_limit = kDefaultSpin;
  return c;
}

}  // namespace

extern "C" {

const char *lst_status_string(int status) {
  switch (status) {
    case LST_OK: return "LST_OK";
    case LST_E_ARG: return "LST_E_ARG";
    case LST_E_SHAPE: return "LST_E_SHAPE";
    case LST_E_INDEX: return "LST_E_INDEX";
    case LST_E_NOT_SPD: return "LST_E_NOT_SPD";
    case LST_E_NONFINITE: return "LST_E_NONFINITE";
    case LST_E_HIP: return "LST_E_HIP";
    case LST_E_STATE: return "LST_E_STATE";
    case LST_E_SYNC: return "LST_E_SYNC";
    default: return "LST_E_UNKNOWN";
  }
}

size_t lst_workspace_bytes(int64_t D, int32_t d, int32_t m_max, int32_t K_max, int32_t loss) {
  if (common_args(D, d, m_max, K_max, loss, 1.f) != LST_OK) return 0;
  return ws_size(KIND_FACTORED, D, d, m_max, K_max, loss);
}

size_t lst_naive_workspace_bytes(int64_t D, int32_t d, int32_t m_max, int32_t K_max,
                                 int32_t loss) {
  if (common_args(D, d, m_max, K_max, loss, 1.f) != LST_OK) return 0;
  return ws_size(KIND_NAIVE, D, d, m_max, K_max, loss);
}

int lst_create(lst_ctx **out, int64_t D, int32_t d, int32_t m_max, int32_t K_max, int32_t loss,
               float eps, float *V, int64_t ldv, float *U, float *UinvT, float *Q, float *WO,
               int32_t ldd, void *workspace, size_t ws_bytes, void *stream) {
  if (!out) return LST_E_ARG;
  *out = nullptr;
  int st = common_args(D, d, m_max, K_max, loss, eps);
  if (st != LST_OK) return st;
  if (!V || !U || !UinvT || !Q) return LST_E_ARG;
  if (loss == LST_LOSS_TAYLOR_SOFTMAX && !WO) return LST_E_ARG;
  if (ldv < d || ldd < d) return LST_E_SHAPE;
  lst_ctx *c = new_ctx(KIND_FACTORED, D, d, m_max, K_max, loss, eps, stream);
  if (!c) return LST_E_ARG;
  c->V = V;
  c->ldv = ldv;
  c->U = U;
  c->UinvT = UinvT;
  c->Q = Q;
  c->WO = loss == LST_LOSS_TAYLOR_SOFTMAX ? WO : nullptr;
  c->ldd = ldd;
  st = take_ws(c, workspace, ws_bytes, carve_factored);
  if (st == LST_OK) {
    StepBufs &b = c->sb;
    b.D = D;
    b.d = d;
    b.ldd = ldd;
    b.loss = loss;
    b.eps = eps;
    b.V = V;
    b.ldv = ldv;
    b.U = U;
    b.UinvT = UinvT;
    b.Q = Q;
    b.WO = c->WO;
    c->plans.reserve(kPlanCap);
    if (hipStreamCreateWithFlags(&c->cap, hipStreamNonBlocking) != hipSuccess) st = LST_E_HIP;
    else c->have_cap = true;
  }
  if (st != LST_OK) {
    lst_destroy(c);
    return st;
  }
  *out = c;
  return LST_OK;
}

int lst_naive_create(lst_ctx **out, int64_t D, int32_t d, int32_t m_max, int32_t K_max,
                     int32_t loss, float eps, float *W, int64_t ldw, void *workspace,
                     size_t ws_bytes, void *stream) {
  if (!out) return LST_E_ARG;
  *out = nullptr;
  int st = common_args(D, d, m_max, K_max, loss, eps);
  if (st != LST_OK) return st;
  if (!W) return LST_E_ARG;
  if (ldw < d) return LST_E_SHAPE;
  lst_ctx *c = new_ctx(KIND_NAIVE, D, d, m_max, K_max, loss, eps, stream);
  if (!c) return LST_E_ARG;
  c->W = W;
  c->ldw = ldw;
  st = take_ws(c, workspace, ws_bytes, carve_naive);
  if (st != LST_OK) {
    lst_destroy(c);
    return st;
  }
  *out = c;
  return LST_OK;
}

void lst_destroy(lst_ctx *c) {
  if (!c) return;
  if (c->ws) (void)hipStreamSynchronize(c->stream);
  graphs_free(c);
  if (c->have_cap) (void)hipStreamDestroy(c->cap);
  prof_free(c);
  delete c;
}

int lst_set_option(lst_ctx *c, int32_t option, int64_t value) {
  if (!c) return LST_E_ARG;
  switch (option) {
    case LST_OPT_ONLINE_KERNEL:
      if (c->kind != KIND_FACTORED) return LST_E_STATE;
      if (value != 0 && value != 1) return LST_E_ARG;
      c->online = value == 1 && c->loss == LST_LOSS_SQUARED;
      return LST_OK;
    case LST_OPT_SPIN_LIMIT:
      if (value < 0 || value > (int64_t)1 << 30) return LST_E_ARG;
      c->spin_limit = (int)value;
      return LST_OK;
    default:
      return LST_E_ARG;
  }
}

int lst_profile_enable(lst_ctx *c, int32_t on) {
  if (!c) return LST_E_ARG;
  if (record(c, hipStreamSynchronize(c->stream))) return LST_E_HIP;
  for (int p = 0; p < LST_NUM_PHASES; ++p) c->prof_used[p] = 0;
  c->prof_on = on != 0;
  return LST_OK;
}

int lst_profile_read(lst_ctx *c, int32_t *counts, double *ms, int32_t n) {
  if (!c || !counts || !ms || n < 0 || n > LST_NUM_PHASES) return LST_E_ARG;
  if (record(c, hipStreamSynchronize(c->stream))) return LST_E_HIP;
  for (int p = 0; p < n; ++p) {
    double tot = 0.0;
    for (int i = 0; i < c->prof_used[p]; ++i) {
      float t = 0.f;
      if (record(c, hipEventElapsedTime(&t, c->prof_ev[p][2 * i], c->prof_ev[p][2 * i + 1])))
        return LST_E_HIP;
      tot += t;
    }
    counts[p] = c->prof_used[p];
    ms[p] = tot;
  }
  for (int p = 0; p < LST_NUM_PHASES; ++p) c->prof_used[p] = 0;
  return LST_OK;
}

int lst_sync_status(lst_ctx *c) {
  if (!c) return LST_E_ARG;
  if (hipStreamSynchronize(c->stream) != hipSuccess) return LST_E_HIP;
  if (c->last_err != hipSuccess) {
    c->last_err = hipSuccess;
    return LST_E_HIP;
  }
  int f = 0;
  if (hipMemcpy(&f, c->flag, sizeof(int), hipMemcpyDeviceToHost) != hipSuccess) return LST_E_HIP;
  if (f != 0) {
    const int zero = 0;
    if (hipMemcpy(c->flag, &zero, sizeof(int), hipMemcpyHostToDevice) != hipSuccess)
      return LST_E_HIP;
  }
  if (f & FLAG_INDEX) return LST_E_INDEX;
  if (f & FLAG_NONFINITE) return LST_E_NONFINITE;
  if (f & FLAG_NOT_SPD) return LST_E_NOT_SPD;
  if (f & FLAG_SYNC) {
    // The stream is idle: restart the online step's barrier counter and decision word.
    if (c->cnt && hipMemset(c->cnt, 0, 4 * sizeof(int)) != hipSuccess) return LST_E_HIP;
    return LST_E_SYNC;
  }
  return LST_OK;
}

int lst_init_factored(lst_ctx *c, const float *V0, int64_t ldv0, const float *U0, int32_t ldu0) {
  if (!c) return LST_E_ARG;
  if (c->kind != KIND_FACTORED) return LST_E_STATE;
  if ((V0 && ldv0 < c->d) || (U0 && ldu0 < c->d)) return LST_E_SHAPE;
  hipStream_t s = c->stream;
  const int d = c->d;
  const size_t row = (size_t)d * sizeof(float);
  if (V0 && V0 != c->V) {
    if (record(c, hipMemcpy2DAsync(c->V, c->ldv * sizeof(float), V0, ldv0 * sizeof(float), row,
                                   (size_t)c->D, hipMemcpyDeviceToDevice, s)))
      return LST_E_HIP;
  }
  if (U0) {
    if (U0 != c->U &&
        record(c, hipMemcpy2DAsync(c->U, c->ldd * sizeof(float), U0, ldu0 * sizeof(float), row,
                                   (size_t)d, hipMemcpyDeviceToDevice, s)))
      return LST_E_HIP;
    std::vector<float> hu((size_t)d * d);
    if (record(c, hipMemcpy2DAsync(hu.data(), row, c->U, c->ldd * sizeof(float), row, (size_t)d,
                                   hipMemcpyDeviceToHost, s)) ||
        record(c, hipStreamSynchronize(s)))
      return LST_E_HIP;
    std::vector<double> a(hu.begin(), hu.end()), inv;
    if (!invert_host(a, d, inv)) return LST_E_NOT_SPD;
    std::vector<float> hut((size_t)d * d);
    for (int i = 0; i < d; ++i)
      for (int j = 0; j < d; ++j) hut[(size_t)i * d + j] = (float)inv[(size_t)j * d + i];
    if (record(c, hipMemcpy2DAsync(c->UinvT, c->ldd * sizeof(float), hut.data(), row, row,
                                   (size_t)d, hipMemcpyHostToDevice, s)) ||
        record(c, hipStreamSynchronize(s)))
      return LST_E_HIP;
  } else {
    if (record(c, launch_identity(s, c->U, d, c->ldd)) ||
        record(c, launch_identity(s, c->UinvT, d, c->ldd)))
      return LST_E_HIP;
  }
  // Q = U^T (V^T V) U  (Q = V^T V when U = I), V^T V split over D into the workspace's
  // partial sums (as many splits as they hold).
  GemmDesc g = gemm_desc(d, d, (int)c->D, c->V, c->ldv, 1, c->V, c->ldv, 1, nullptr, d);
  if (gemm_plan_split(g, kTargetWGs, c->initpart) > c->initpart_floats) {
    const int fit = (int)(c->initpart_floats / ((size_t)d * d));
    if (fit >= 2) {
      int chunk = (int)((c->D + fit - 1) / fit);
      chunk = (chunk + 7) / 8 * 8;
      g.kchunk = chunk;
      g.splits = (int)((c->D + chunk - 1) / chunk);
    } else {
      g.splits = 1;
      g.kchunk = (int)c->D;
      g.partial = nullptr;
    }
  }
  GemmBatch b{};
  int st = LST_OK;
  if (!U0) {
    g.C = c->Q;
    g.ldc = c->ldd;
    b.d[0] = g;
    b.n = 1;
    if (record(c, gemm_launch(b, nullptr, s))) st = LST_E_HIP;
  } else {
    float *Gm = c->Sd0, *Tm = c->Sd1;
    g.C = Gm;
    g.ldc = d;
    b.d[0] = g;
    b.n = 1;
    if (record(c, gemm_launch(b, nullptr, s))) st = LST_E_HIP;
    GemmBatch b2{};
    b2.d[0] = gemm_desc(d, d, d, Gm, d, 0, c->U, c->ldd, 1, Tm, d);  // T = G U
    b2.n = 1;
    if (st == LST_OK && record(c, gemm_launch(b2, nullptr, s))) st = LST_E_HIP;
    GemmBatch b3{};
    b3.d[0] = gemm_desc(d, d, d, c->U, c->ldd, 1, Tm, d, 1, c->Q, c->ldd);  // Q = U^T T
    b3.n = 1;
    if (st == LST_OK && record(c, gemm_launch(b3, nullptr, s))) st = LST_E_HIP;
  }
  if (st == LST_OK && c->WO) {
    // W = V U + 1_D omega^T with the caller's omega: w_bar = U^T (V^T 1_D) + D omega,
    // and Q gains the omega part of W^T W
    const float *omega = c->WO + c->ldd;
    if (record(c, launch_wbar(s, c->V, c->ldv, c->D, d, U0 ? c->U : nullptr, c->ldd, omega,
                              c->wpart, kWbarBlocks, c->WO)) ||
        record(c, launch_q_omega(s, c->Q, c->ldd, d, c->D, c->WO, omega)))
      st = LST_E_HIP;
  }
  const int zero = 0;
  if (record(c, hipStreamSynchronize(s))) st = LST_E_HIP;
  if (record(c, hipMemcpy(c->flag, &zero, sizeof(int), hipMemcpyHostToDevice))) st = LST_E_HIP;
  return st;
}

}  // extern "C"

namespace {

// The plan for m, built and copied to its device slot on first use (an ordered copy
// on the context's stream).  Replacing the least recently used plan first drains the
// stream and drops the recorded graphs that launch it.
PlanEntry *get_plan(lst_ctx *c, int m) {
  for (PlanEntry &e : c->plans)
    if (e.m == m) {
      e.last_use = ++c->plan_tick;
      return &e;
    }
  StepPlan *slot;
  if (c->plans.size() < kPlanCap) {
    slot = c->plan_pool + c->plans.size();
    c->plans.push_back(PlanEntry{});
  } else {
    size_t v = 0;
    for (size_t i = 1; i < c->plans.size(); ++i)
      if (c->plans[i].last_use < c->plans[v].last_use) v = i;
    if (record(c, hipStreamSynchronize(c->stream))) return nullptr;
    const int old_m = c->plans[v].m;
    for (size_t i = c->graphs.size(); i-- > 0;)
      if (c->graphs[i].m == old_m) {
        (void)hipGraphExecDestroy(c->graphs[i].exec);
        c->graphs.erase(c->graphs.begin() + i);
      }
    slot = c->plans[v].dev;
    c->plans.erase(c->plans.begin() + v);
    c->plans.push_back(PlanEntry{});
  }
  PlanEntry &e = c->plans.back();
  e.m = m;
  e.dev = slot;
  e.host.reset(new (std::nothrow) StepPlan);
  if (!e.host) {
    c->plans.pop_back();
    return nullptr;
  }
  build_step_plan(c->sb, m, *e.host);
  if (record(c, hipMemcpyAsync(e.dev, e.host.get(), sizeof(StepPlan), hipMemcpyHostToDevice,
                               c->stream))) {
    c->plans.pop_back();
    return nullptr;
  }
  e.last_use = ++c->plan_tick;
  return &e;
}

constexpr int kStepPhase[5] = {LST_PHASE_CONTRACT, LST_PHASE_GATHER, LST_PHASE_ZGRAD,
                               LST_PHASE_MID, LST_PHASE_UPDATE};

// The five launches of a factored step on stream s.
int enqueue_factored_step(lst_ctx *c, hipStream_t s, const PlanEntry &pl, const StepArgs &a) {
  for (int l = 0; l < 5; ++l) {
    prof(c, kStepPhase[l], true);
    enqueue_step_launch(l, c->sb, *pl.host, pl.dev, a, s);
    prof(c, kStepPhase[l], false);
  }
  // launch errors are not checked one by one: one stays pending and is reported here
  return record(c, hipGetLastError()) ? LST_E_HIP : LST_OK;
}

// Replays (capturing first if needed) the graph of a step with these arguments.
int graph_step(lst_ctx *c, const PlanEntry &pl, const StepArgs &a, const float *grad_arg) {
  uint32_t lr_bits;
  std::memcpy(&lr_bits, &a.lr, sizeof(lr_bits));
  GraphEntry *hit = nullptr;
  for (GraphEntry &g : c->graphs)
    if (g.H == a.H && g.idx == a.idx && g.val == a.val && g.loss == a.loss &&
        g.grad == grad_arg && g.m == a.m && g.K == a.K && g.lr_bits == lr_bits) {
      hit = &g;
      break;
    }
  if (!hit) {
    if (c->graphs.size() >= kGraphCap) {  // evict the least recently used graph
      size_t v = 0;
      for (size_t i = 1; i < c->graphs.size(); ++i)
        if (c->graphs[i].last_use < c->graphs[v].last_use) v = i;
      if (record(c, hipStreamSynchronize(c->stream))) return LST_E_HIP;
      (void)hipGraphExecDestroy(c->graphs[v].exec);
      c->graphs.erase(c->graphs.begin() + v);
    }
    if (record(c, hipStreamBeginCapture(c->cap, hipStreamCaptureModeThreadLocal)))
      return LST_E_HIP;
    const int st = enqueue_factored_step(c, c->cap, pl, a);
    hipGraph_t graph = nullptr;
    const hipError_t ec = hipStreamEndCapture(c->cap, &graph);
    if (st != LST_OK || ec != hipSuccess || !graph) {
      if (graph) (void)hipGraphDestroy(graph);
      if (ec != hipSuccess) c->last_err = ec;
      return st != LST_OK ? st : LST_E_HIP;
    }
    GraphEntry e{a.H, a.idx, a.val, a.loss, const_cast<float *>(grad_arg), a.m, a.K, lr_bits,
                 nullptr, 0};
    const hipError_t ei = hipGraphInstantiate(&e.exec, graph, nullptr, nullptr, 0);
    (void)hipGraphDestroy(graph);
    if (record(c, ei)) return LST_E_HIP;
    c->graphs.push_back(e);
    hit = &c->graphs.back();
  }
  hit->last_use = ++c->graph_tick;
  return record(c, hipGraphLaunch(hit->exec, c->stream));
}

}  // namespace

extern "C" {

int lst_step(lst_ctx *c, const float *H, int32_t m, const int32_t *idx, const float *val, int32_t K,
             float lr, float *loss_dev, float *grad_H) {
  if (!c) return LST_E_ARG;
  if (c->kind != KIND_FACTORED) return LST_E_STATE;
  int st = step_args(c, H, m, idx, val, K, lr, loss_dev);
  if (st != LST_OK) return st;
  if (m == 0) return record(c, launch_fill(c->stream, loss_dev, 0.f));
  const bool graphs = c->use_graphs && !c->prof_on;
  if (m == 1 && c->online && !graphs) {
    // the online step of Algorithm 2 in one launch (its work vectors share the section 5
    // scratch, which is only used between steps on this stream)
    prof(c, LST_PHASE_ONLINE, true);
    const hipError_t e = launch_online_step(
        c->stream, c->D, c->d, K, H, idx, val, lr, c->V, c->ldv, c->U, c->UinvT, c->Q, c->ldd,
        loss_dev, grad_H, c->spart, reinterpret_cast<unsigned *>(c->cnt), c->spin_limit, c->flag);
    prof(c, LST_PHASE_ONLINE, false);
    return record(c, e);
  }
  const PlanEntry *pl = get_plan(c, m);
  if (!pl) return LST_E_HIP;
  StepArgs a{H, m, idx, val, K, lr, loss_dev, grad_H ? grad_H : c->gradH};
  if (graphs) return graph_step(c, *pl, a, grad_H);
  return enqueue_factored_step(c, c->stream, *pl, a);
}

int lst_use_graphs(lst_ctx *c, int32_t on) {
  if (!c) return LST_E_ARG;
  if (c->kind != KIND_FACTORED) return LST_E_STATE;
  c->use_graphs = on != 0;
  return LST_OK;
}

int lst_materialize_W(lst_ctx *c, float *W, int64_t ldw) {
  if (!c || !W) return LST_E_ARG;
  if (ldw < c->d) return LST_E_SHAPE;
  if (c->kind == KIND_NAIVE) {
    return record(c, hipMemcpy2DAsync(W, ldw * sizeof(float), c->W, c->ldw * sizeof(float),
                                      (size_t)c->d * sizeof(float), (size_t)c->D,
                                      hipMemcpyDeviceToDevice, c->stream));
  }
  GemmBatch b{};
  b.d[0] = gemm_desc((int)c->D, c->d, c->d, c->V, c->ldv, 0, c->U, c->ldd, 1, W, ldw);
  if (c->WO) {  // + 1_D omega^T: omega as a C input of row stride 0
    b.d[0].Cin = c->WO + c->ldd;
    b.d[0].ldcin = 0;
    b.d[0].beta = 1.f;
  }
  b.n = 1;
  return record(c, gemm_launch(b, nullptr, c->stream));
}

int lst_naive_step(lst_ctx *c, const float *H, int32_t m, const int32_t *idx, const float *val,
                   int32_t K, float lr, float *loss_dev, float *grad_H) {
  if (!c) return LST_E_ARG;
  if (c->kind != KIND_NAIVE) return LST_E_STATE;
  int st = step_args(c, H, m, idx, val, K, lr, loss_dev);
  if (st != LST_OK) return st;
  hipStream_t s = c->stream;
  if (m == 0) return record(c, launch_fill(s, loss_dev, 0.f));
  const int d = c->d;
  const int64_t D = c->D;
  float *gH = grad_H ? grad_H : c->gradH;
  // O = W H^T  (D x m), the O(D d) forward product of section 2.3, with the
  // partial column sums of squares for q_j = ||o_j||^2 when the tiled kernel runs.
  prof(c, LST_PHASE_NAIVE_FWD, true);
  GemmDesc fwd = gemm_desc((int)D, m, d, c->W, c->ldw, 0, H, d, 0, c->O, m);
  int nparts = kColnormBlocks;
  const bool tay = c->loss == LST_LOSS_TAYLOR_SOFTMAX;
  if (gemm_big_ok(fwd) && !tay) {
    fwd.colsq = c->colpart;
    gemm_big_plan(fwd, kTargetWGs, 0, nullptr);
    nparts = kBigColsqRows * fwd.tiles_m;
    if (record(c, gemm_big_launch(fwd, nullptr, s, GEMM_NAIVE_FWD))) return LST_E_HIP;
  } else {
    if (record(c, naive_gemm(c, fwd, false, nullptr, s, GEMM_NAIVE_FWD)) ||
        record(c, launch_colnorm(s, c->O, D, m, c->colpart, tay ? c->colsum : nullptr,
                                 kColnormBlocks)))
      return LST_E_HIP;
  }
  prof(c, LST_PHASE_NAIVE_FWD, false);
  // The loss and dl/dq, dl/da from the explicit O.
  prof(c, LST_PHASE_NAIVE_LOSS, true);
  if (record(c, launch_naive_epilogue(s, m, K, D, nparts, c->colpart, tay ? c->colsum : nullptr,
                                      c->O, idx, val, c->loss, c->eps, c->sb.dq,
                                      tay ? c->sb.ds : nullptr, c->sb.dA, c->sb.lvec, c->flag)))
    return LST_E_HIP;
  // grad_O = 2 O diag(dl/dq) + 1_D (dl/ds)^T + Yring, in place over O.
  if (record(c, launch_grad_o(s, c->O, D, m, K, c->sb.dq, tay ? c->sb.ds : nullptr, idx,
                              c->sb.dA, c->sb.lvec, loss_dev, c->flag)))
    return LST_E_HIP;
  prof(c, LST_PHASE_NAIVE_LOSS, false);
  // grad_H = grad_O^T W (split over D), then W <- W - eta grad_O H.
  prof(c, LST_PHASE_NAIVE_GRAD, true);
  if (record(c, naive_gemm(c, gemm_desc(m, d, (int)D, c->O, m, 1, c->W, c->ldw, 1, gH, d), true,
                           nullptr, s, GEMM_NAIVE_GRAD)))
    return LST_E_HIP;
  prof(c, LST_PHASE_NAIVE_GRAD, false);
  prof(c, LST_PHASE_NAIVE_UPDATE, true);
  if (record(c, naive_gemm(c,
                           gemm_desc((int)D, d, m, c->O, m, 0, H, d, 1, c->W, c->ldw, -lr, c->W,
                                     c->ldw, 1.f),
                           false, c->flag, s, GEMM_NAIVE_UPDATE)))
    return LST_E_HIP;
  prof(c, LST_PHASE_NAIVE_UPDATE, false);
  return LST_OK;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Section 5: numerical stabilisation between steps.
// ---------------------------------------------------------------------------
namespace {

int factored_ctx(const lst_ctx *c) {
  if (!c) return LST_E_ARG;
  return c->kind == KIND_FACTORED ? LST_OK : LST_E_STATE;
}

hipError_t square_gemm(lst_ctx *c, const float *A, int lda, int tA, const float *B, int ldb,
                       int tB, float *C, int ldc, float alpha = 1.f, const float *Cin = nullptr,
                       int ldcin = 0, float beta = 0.f) {
  const int d = c->d;
  GemmBatch b{};
  b.d[0] = gemm_desc(d, d, d, A, lda, tA, B, ldb, tB, C, ldc, alpha, Cin, ldcin, beta);
  b.n = 1;
  return gemm_launch(b, nullptr, c->stream);
}

// Newton-Schulz rounds Y <- Y + (I - Y U^T) Y ending in U^{-T}; see lst_refresh_uinvt.
int refresh_uinvt(lst_ctx *c, int iters, bool from_scratch, float *resid) {
  const int d = c->d, ldd = c->ldd;
  hipStream_t s = c->stream;
  float *Y = c->UinvT;
  int ldy = ldd;
  if (from_scratch) {
    if (record(c, launch_ns_start(s, c->U, ldd, d, c->sscal, c->Sd0, d))) return LST_E_HIP;
    Y = c->Sd0;
    ldy = d;
  }
  for (int it = 0; it < iters; ++it) {
    float *Yn = Y == c->UinvT ? c->Sd0 : c->UinvT;
    const int ldn = Yn == c->UinvT ? ldd : d;
    if (record(c, launch_residual64(s, Y, ldy, c->U, ldd, d, c->Sd1)) ||            // E = I - Y U^T
        record(c, square_gemm(c, c->Sd1, d, 0, Y, ldy, 1, Yn, ldn, 1.f, Y, ldy, 1.f)))  // Y + E Y
      return LST_E_HIP;
    Y = Yn;
    ldy = ldn;
  }
  if (Y != c->UinvT &&
      record(c, hipMemcpy2DAsync(c->UinvT, (size_t)ldd * sizeof(float), Y, (size_t)d * sizeof(float),
                                 (size_t)d * sizeof(float), (size_t)d, hipMemcpyDeviceToDevice, s)))
    return LST_E_HIP;
  if (resid && (record(c, launch_residual64(s, c->UinvT, ldd, c->U, ldd, d, c->Sd1)) ||
                record(c, launch_fill(s, resid, 0.f)) || record(c, launch_absmax(s, c->Sd1, d, resid))))
    return LST_E_HIP;
  return LST_OK;
}

// max |I - U^{-T} U^T| of the current U^{-T}, on the host (synchronises the stream).
int uinvt_residual(lst_ctx *c, float *r) {
  float *dev = c->sscal + 2;
  if (record(c, launch_residual64(c->stream, c->UinvT, c->ldd, c->U, c->ldd, c->d, c->Sd1)) ||
      record(c, launch_fill(c->stream, dev, 0.f)) ||
      record(c, launch_absmax(c->stream, c->Sd1, c->d, dev)) ||
      record(c, hipMemcpyAsync(r, dev, sizeof(float), hipMemcpyDeviceToHost, c->stream)) ||
      record(c, hipStreamSynchronize(c->stream)))
    return LST_E_HIP;
  return LST_OK;
}

// U^{-T} recomputed before a stabilisation check: two rounds from the carried value
// when its residual is small enough for the iteration to converge from it, else from
// scratch in groups of eight rounds until the residual is small, then two more.
constexpr float kWarmResidual = 0.25f;
int refresh_for_check(lst_ctx *c) {
  float r = 0.f;
  int st = uinvt_residual(c, &r);
  if (st != LST_OK) return st;
  if (!(r < kWarmResidual)) {
    bool scratch = true;
    for (int rounds = 0; !(r < kWarmResidual); rounds += 8) {
      if (rounds >= 96) return LST_E_NOT_SPD;  // U is numerically singular
      if ((st = refresh_uinvt(c, 8, scratch, nullptr)) != LST_OK ||
          (st = uinvt_residual(c, &r)) != LST_OK)
        return st;
      scratch = false;
    }
  }
  return refresh_uinvt(c, 2, false, nullptr);
}

int power_iteration(lst_ctx *c, int which, int log2_iters, const float *u0, float *u_out,
                    float *sigma_out) {
  const int d = c->d, ldd = c->ldd;
  hipStream_t s = c->stream;
  const float *A = which ? c->UinvT : c->U;
  if (record(c, square_gemm(c, A, ldd, 0, A, ldd, 0, c->Sd0, d))) return LST_E_HIP;  // G = A A^T
  for (int it = 0; it < log2_iters; ++it)
    if (record(c, launch_trace_scale(s, c->Sd0, d, c->Sd1)) ||
        record(c, square_gemm(c, c->Sd1, d, 0, c->Sd1, d, 1, c->Sd0, d)))
      return LST_E_HIP;
  return record(c, launch_power_finish(s, c->Sd0, d, u0, A, ldd, which, u_out, sigma_out, c->spart));
}

int fix_singular_value(lst_ctx *c, const float *u, const float *sigma, float target) {
  const int d = c->d, ldd = c->ldd;
  hipStream_t s = c->stream;
  float *a = c->svec, *b = c->svec + d;
  if (record(c, launch_tmatvec2(s, c->U, c->UinvT, ldd, d, u, u, a, b, c->spart)) ||
      record(c, launch_fix_state(s, c->U, c->UinvT, ldd, d, u, a, b, sigma, target, c->flag)) ||
      record(c, launch_fix_v(s, c->V, c->ldv, c->D, d, u, sigma, target)))
    return LST_E_HIP;
  return LST_OK;
}

bool in_svec(const lst_ctx *c, const float *p) {
  return p >= c->svec && p < c->svec + 4 * (size_t)c->d;
}

}  // namespace

extern "C" {

int lst_restore_pristine(lst_ctx *c) {
  int st = factored_ctx(c);
  if (st != LST_OK) return st;
  if (c->d > 1024) return LST_E_SHAPE;
  hipStream_t s = c->stream;
  if (record(c, launch_restore(s, c->V, c->ldv, c->D, c->U, c->ldd, c->d)) ||
      record(c, launch_identity(s, c->U, c->d, c->ldd)) ||
      record(c, launch_identity(s, c->UinvT, c->d, c->ldd)))
    return LST_E_HIP;
  return LST_OK;
}

int lst_refresh_uinvt(lst_ctx *c, int32_t iters, int32_t from_scratch, float *resid_dev) {
  int st = factored_ctx(c);
  if (st != LST_OK) return st;
  if (iters < 1 || iters > 100) return LST_E_ARG;
  return refresh_uinvt(c, iters, from_scratch != 0, resid_dev);
}

int lst_power_iteration(lst_ctx *c, int32_t which, int32_t log2_iters, const float *u0,
                        float *u_out, float *sigma_out) {
  int st = factored_ctx(c);
  if (st != LST_OK) return st;
  if ((which != 0 && which != 1) || log2_iters < 0 || log2_iters > 30 || !u0 || !u_out ||
      !sigma_out)
    return LST_E_ARG;
  return power_iteration(c, which, log2_iters, u0, u_out, sigma_out);
}

int lst_fix_singular_value(lst_ctx *c, const float *u, const float *sigma_dev, float target) {
  int st = factored_ctx(c);
  if (st != LST_OK) return st;
  if (!u || !sigma_dev || !finite_pos(target) || in_svec(c, u)) return LST_E_ARG;
  return fix_singular_value(c, u, sigma_dev, target);
}

int lst_singular_stabilize(lst_ctx *c, float lo, float hi, int32_t log2_iters, const float *u0,
                           int32_t max_fixes, int32_t *n_fixed, float *sigmas) {
  int st = factored_ctx(c);
  if (st != LST_OK) return st;
  if (!finite_pos(lo) || !finite_pos(hi) || hi < lo || log2_iters < 0 || log2_iters > 30 || !u0 ||
      max_fixes < 0 || !n_fixed || !sigmas)
    return LST_E_ARG;
  hipStream_t s = c->stream;
  if ((st = refresh_for_check(c)) != LST_OK) return st;
  float *u = c->svec + 2 * (size_t)c->d, *sig = c->sscal + 1;
  for (int which = 1; which >= 0; --which) {  // the smallest singular value first
    int n = 0;
    float sv = 0.f;
    for (;;) {
      if ((st = power_iteration(c, which, log2_iters, u0, u, sig)) != LST_OK) return st;
      if (record(c, hipMemcpyAsync(&sv, sig, sizeof(float), hipMemcpyDeviceToHost, s)) ||
          record(c, hipStreamSynchronize(s)))
        return LST_E_HIP;
      if (!std::isfinite(sv) || !(sv > 0.f)) return LST_E_NONFINITE;
      if ((which ? sv >= lo : sv <= hi) || n >= max_fixes) break;
      if ((st = fix_singular_value(c, u, sig, 1.f)) != LST_OK) return st;
      ++n;
    }
    n_fixed[1 - which] = n;
    sigmas[1 - which] = sv;
  }
  return LST_OK;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Section 2.2: the sparse input layer (no context).
// ---------------------------------------------------------------------------
namespace {
int input_args(int64_t D_in, int32_t d, int64_t ldw, const void *W1, const int32_t *idx,
               const float *val, int32_t m, int32_t K, const int32_t *status) {
  if (!W1 || !status) return LST_E_ARG;
  if (D_in < 1 || D_in > LST_MAX_D || d < 1 || d > LST_MAX_d || ldw < d) return LST_E_SHAPE;
  if (m < 0 || K < 0 || K > LST_MAX_K || (int64_t)m * K > 8192) return LST_E_SHAPE;
  if (m > 0 && K > 0 && (!idx || !val)) return LST_E_ARG;
  return LST_OK;
}
}  // namespace

extern "C" {

int lst_input_forward(const float *W1, int64_t ldw, int64_t D_in, int32_t d, const int32_t *idx,
                      const float *val, int32_t m, int32_t K, float *A, int32_t *status_dev,
                      void *stream) {
  int st = input_args(D_in, d, ldw, W1, idx, val, m, K, status_dev);
  if (st != LST_OK) return st;
  if (m > 0 && !A) return LST_E_ARG;
  const hipError_t e = launch_input_forward(static_cast<hipStream_t>(stream), W1, ldw, D_in, d, idx,
                                            val, m, K, A, status_dev);
  return e == hipSuccess ? LST_OK : LST_E_HIP;
}

int lst_input_update(float *W1, int64_t ldw, int64_t D_in, int32_t d, const int32_t *idx,
                     const float *val, int32_t m, int32_t K, const float *grad_A, float lr,
                     int32_t *status_dev, void *stream) {
  int st = input_args(D_in, d, ldw, W1, idx, val, m, K, status_dev);
  if (st != LST_OK) return st;
  if (m > 0 && K > 0 && !grad_A) return LST_E_ARG;
  if (!finite_pos(lr)) return LST_E_ARG;
  const hipError_t e = launch_input_update(static_cast<hipStream_t>(stream), W1, ldw, D_in, d, idx,
                                           val, m, K, grad_A, lr, status_dev);
  return e == hipSuccess ? LST_OK : LST_E_HIP;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// lst_step_noalloc: the factored step with its intermediates in a fixed device array
// ---------------------------------------------------------------------------

namespace {

constexpr size_t kScratchBytes = size_t(16) << 20;
constexpr int kScratchDevices = 16;

}  // namespace

// The step's descriptors and intermediates of lst_step_noalloc.  Each device holds its
// own copy at its own address, obtained once per device with hipGetSymbolAddress; host
// code uses that address only (the symbol's name is not a device address on the host).
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

struct ScratchDev {
  char *base;        // this device's copy of scratch, null until set up
  bool plan_valid;   // plan holds the descriptors last written to the array
  StepPlan plan;
};
ScratchDev g_scratch[kScratchDevices];
std::mutex g_scratch_mu;

constexpr int kChunkWords = 512;  // 2 KiB of kernel arguments per launch
struct WordChunk {
  uint32_t w[kChunkWords];
};

__global__ void __launch_bounds__(256) put_words_kernel(uint32_t *dst, WordChunk c, int n) {
  for (int i = (int)threadIdx.x; i < n; i += 256) dst[i] = c.w[i];
}

__global__ void __launch_bounds__(256) clear_words_kernel(int *a, int na, int *b, int nb, int *c,
                                                           int nc) {
  for (int i = (int)threadIdx.x; i < na; i += 256) a[i] = 0;
  for (int i = (int)threadIdx.x; i < nb; i += 256) b[i] = 0;
  for (int i = (int)threadIdx.x; i < nc; i += 256) c[i] = 0;
}

// Bytes of the array a step of m examples, K slots and hidden size d takes: the
// descriptors first, then the intermediates.
size_t noalloc_bytes(int m, int d, int K) {
  Carver cv{nullptr};
  cv.take<StepPlan>(1);
  StepBufs b{};
  float *g = nullptr;
  carve_step(b, g, (size_t)m, (size_t)d, (size_t)K, cv);
  return cv.off;
}

// Writes the descriptors into the array with kernel arguments (no host buffer has to
// outlive the call), unless the array already holds these exact descriptors.
hipError_t put_plan(ScratchDev &sd, const StepPlan &pl, hipStream_t s) {
  static_assert(sizeof(StepPlan) % sizeof(uint32_t) == 0, "plan is copied in words");
  if (sd.plan_valid && std::memcmp(&sd.plan, &pl, sizeof(StepPlan)) == 0) return hipSuccess;
  sd.plan_valid = false;
  const uint32_t *src = reinterpret_cast<const uint32_t *>(&pl);
  uint32_t *dst = reinterpret_cast<uint32_t *>(sd.base);
  const int words = (int)(sizeof(StepPlan) / sizeof(uint32_t));
  for (int o = 0; o < words; o += kChunkWords) {
    WordChunk c;
    const int n = std::min(kChunkWords, words - o);
    std::memcpy(c.w, src + o, (size_t)n * sizeof(uint32_t));
    hipLaunchKernelGGL(put_words_kernel, dim3(1), dim3(256), 0, s, dst + o, c, n);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  std::memcpy(&sd.plan, &pl, sizeof(StepPlan));
  sd.plan_valid = true;
  return hipSuccess;
}

}  // namespace

extern "C" {

int lst_step_noalloc(int64_t D, int32_t d, int32_t loss, float eps, float *V, int64_t ldv, float *U,
                     float *UinvT, float *Q, float *WO, int32_t ldd, const float *H, int32_t m,
                     const int32_t *idx, const float *val, int32_t K, float lr, float *loss_dev,
                     float *grad_H, int32_t *status_dev, void *stream) {
  const int mm = m < 1 ? 1 : m;
  int st = common_args(D, d, mm, K, loss, eps);
  if (st != LST_OK) return st;
  if (!V || !U || !UinvT || !Q || !loss_dev || !status_dev) return LST_E_ARG;
  if (loss == LST_LOSS_TAYLOR_SOFTMAX && !WO) return LST_E_ARG;
  if (ldv < d || ldd < d) return LST_E_SHAPE;
  if (m < 0) return LST_E_SHAPE;
  if (m > 0 && !H) return LST_E_ARG;
  if (m > 0 && K > 0 && (!idx || !val)) return LST_E_ARG;
  if (!finite_pos(lr)) return LST_E_ARG;
  if (noalloc_bytes(mm, d, K) > kScratchBytes) return LST_E_SHAPE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return LST_E_HIP;
  if (dev < 0 || dev >= kScratchDevices) return LST_E_ARG;
  if (s) {
    int sdev = -1;
    if (hipStreamGetDevice(s, &sdev) != hipSuccess) return LST_E_HIP;
    if (sdev != dev) return LST_E_ARG;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  ScratchDev &sd = g_scratch[dev];
  if (!sd.base) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return LST_E_HIP;
    sd.base = static_cast<char *>(p);
  }
  if (m == 0) {
    hipLaunchKernelGGL(clear_words_kernel, dim3(1), dim3(256), 0, s, status_dev, 1, nullptr, 0,
                       nullptr, 0);
    if (hipGetLastError() != hipSuccess) return LST_E_HIP;
    return launch_fill(s, loss_dev, 0.f) == hipSuccess ? LST_OK : LST_E_HIP;
  }
  StepBufs b{};
  float *gradH = nullptr;
  Carver cv{sd.base};
  StepPlan *dev_plan = cv.take<StepPlan>(1);
  carve_step(b, gradH, (size_t)m, (size_t)d, (size_t)K, cv);
  b.D = D;
  b.d = d;
  b.ldd = ldd;
  b.loss = loss;
  b.eps = eps;
  b.V = V;
  b.ldv = ldv;
  b.U = U;
  b.UinvT = UinvT;
  b.Q = Q;
  b.WO = loss == LST_LOSS_TAYLOR_SOFTMAX ? WO : nullptr;
  b.flag = status_dev;
  static StepPlan host;  // built under the lock; copied into the array by put_plan
  build_step_plan(b, m, host);
  if (put_plan(sd, host, s) != hipSuccess) return LST_E_HIP;
  // the error word and the arrival counters of this layout start at zero
  hipLaunchKernelGGL(clear_words_kernel, dim3(1), dim3(256), 0, s, status_dev, 1, b.qcnt,
                     (m + 15) / 16, b.rcnt, m * (K > 0 ? K : 1));
  if (hipGetLastError() != hipSuccess) return LST_E_HIP;
  StepArgs a{H, m, idx, val, K, lr, loss_dev, grad_H ? grad_H : gradH};
  for (int l = 0; l < 5; ++l) enqueue_step_launch(l, b, host, dev_plan, a, s);
  return hipGetLastError() == hipSuccess ? LST_OK : LST_E_HIP;
}

}  // extern "C"
