// C ABI of liblst: argument validation, workspace carving and the enqueue order
// of the factored step (Algorithm 3 / Algorithm 4) and of the naive step.
#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <new>
#include <vector>

#include "lst_internal.h"

using namespace lst;

namespace lst {
thread_local ProfHook g_prof;
}  // namespace lst

namespace {

enum : int { KIND_FACTORED = 1, KIND_NAIVE = 2 };
constexpr int kTargetWGs = 1024;   // workgroups a split-k GEMM aims for
constexpr int kColnormBlocks = 1024;

// Device workspace carved in 256-byte aligned pieces.
struct Carver {
  char *base;
  size_t off = 0;
  template <class T>
  T *take(size_t n) {
    off = (off + 255) & ~size_t(255);
    T *p = base ? reinterpret_cast<T *>(base + off) : nullptr;
    off += n * sizeof(T);
    return p;
  }
};

// A factored step recorded as a HIP graph, replayed when the same arguments recur.
struct GraphEntry {
  const void *H, *idx, *val;
  void *loss, *grad;
  int m, K;
  uint32_t lr_bits;
  // the step's parts in launch order: main stream up to M, side stream (Woodbury
  // branch), main stream state updates
  hipGraphExec_t exec_a, exec_side, exec_b;
  uint64_t last_use;
};
constexpr size_t kGraphCap = 256;

// The five GEMM batches of a factored step for one m: Gram product, contractions,
// Z^/grad_H, mid and state updates.
constexpr int kPlanBatches = 5;
constexpr size_t kPlanCap = 16;
struct PlanEntry {
  int m;
  GemmBatch b[kPlanBatches];
  GemmBatch *dev;
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
  int ldd;
  // naive state (borrowed)
  float *W;
  int64_t ldw;
  // workspace (owned)
  void *ws;
  size_t ws_bytes;
  float *Hhat, *Htil, *X, *G, *Atil, *Zhat, *gradH, *Yw, *Zq, *P;
  float *N, *Mhat, *HZ, *M, *R, *Cwork;
  float *Pbig, *Cp, *Rp;  // blocked Woodbury inverse for m > kWoodburyOneWG
  float *dq, *lvec, *dA;
  // section 5 stabilisation: two d x d scratch matrices (row stride d), four
  // d-vectors, the partial sums of two matrix-vector products (32 d) and eight scalars
  float *Sd0, *Sd1, *svec, *spart, *sscal;
  int *flag;
  // progress counters ordering the two streams of a factored step: [0] contraction
  // launches started, [1] Woodbury inverses completed, [2] Z^ launches started; [3]
  // the grid barrier of the online step's single launch
  int *cnt;
  float *O, *colpart, *splitpart;
  hipError_t last_err;
  // side stream of a factored step (Woodbury inverse); cap is the stream a step
  // is captured on when it is recorded as HIP graphs
  hipStream_t side[1];
  hipStream_t cap;
  bool have_side;
  // tracing: event pairs per phase
  bool prof_on;
  std::vector<hipEvent_t> prof_ev[LST_NUM_PHASES];
  int prof_used[LST_NUM_PHASES];
  // GEMM plans of the factored step, one per minibatch size m (host copies and
  // their device slots in plan_pool)
  std::vector<PlanEntry> plans;
  GemmBatch *plan_pool;
  uint64_t plan_tick;
  // captured steps, one per distinct (inputs, m, K, lr)
  bool use_graphs;
  // test hook (environment variable LST_TEST_WITHHOLD_WOODBURY_RELEASE at creation):
  // the Woodbury branch never releases its counter, so the state-update wait of
  // every step expires (bounded) and reports LST_E_SYNC
  bool withhold_release;
  // environment variable LST_ONE_STREAM at creation: the side stream's work is
  // enqueued on the context's stream instead, after the main chain up to M (the
  // waits are then met on arrival).  For tools that run one dispatch at a time,
  // such as hardware counter collection, under which a wait on another stream's
  // progress could not be met.
  bool one_stream;
  // m = 1 squared-error steps as one launch (see lst_step)
  bool online;
  std::vector<GraphEntry> graphs;
  uint64_t graph_tick;
};

namespace {

bool finite_pos(float x) { return std::isfinite(x) && x > 0.f; }

void carve_factored(lst_ctx *c, Carver &cv) {
  const size_t md = (size_t)c->m_max * c->d, mm = (size_t)c->m_max * c->m_max;
  const size_t mk = (size_t)c->m_max * (c->K_max > 0 ? c->K_max : 1);
  c->Hhat = cv.take<float>(md);
  c->Htil = cv.take<float>(md);
  c->X = cv.take<float>(md);
  c->G = cv.take<float>(md);
  c->Atil = cv.take<float>(md);
  c->Zhat = cv.take<float>(md);
  c->gradH = cv.take<float>(md);
  c->Yw = cv.take<float>(md);
  c->Zq = cv.take<float>(md);
  c->P = cv.take<float>(md);
  c->N = cv.take<float>(mm);
  c->Mhat = cv.take<float>(mm);
  c->HZ = cv.take<float>(mm);
  c->M = cv.take<float>(mm);
  c->R = cv.take<float>(mm);
  c->Cwork = cv.take<float>(mm);
  const size_t big = c->m_max > kWoodburyOneWG ? kBigBlock : 0;
  c->Pbig = cv.take<float>(2 * big * big);  // P and P + I
  c->Cp = cv.take<float>((size_t)c->m_max * big);
  c->Rp = cv.take<float>(big * c->m_max);
  c->dq = cv.take<float>(c->m_max);
  c->lvec = cv.take<float>(c->m_max);
  c->dA = cv.take<float>(mk);
  c->Sd0 = cv.take<float>((size_t)c->d * c->d);
  c->Sd1 = cv.take<float>((size_t)c->d * c->d);
  c->svec = cv.take<float>(4 * (size_t)c->d);
  c->spart = cv.take<float>(std::max<size_t>(32 * (size_t)c->d, online_work_floats(c->d)));
  c->sscal = cv.take<float>(8);
  c->flag = cv.take<int>(1);
  c->cnt = cv.take<int>(4);
  c->plan_pool = cv.take<GemmBatch>(kPlanCap * kPlanBatches);
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
  c->dq = cv.take<float>(c->m_max);
  c->lvec = cv.take<float>(c->m_max);
  c->dA = cv.take<float>(mk);
  c->flag = cv.take<int>(1);
}

int common_args(int64_t D, int32_t d, int32_t m_max, int32_t K_max, int32_t loss, float eps) {
  if (loss != LST_LOSS_SQUARED && loss != LST_LOSS_SPHERICAL_SOFTMAX) return LST_E_ARG;
  if (loss == LST_LOSS_SPHERICAL_SOFTMAX && !finite_pos(eps)) return LST_E_ARG;
  if (D < 1 || D > LST_MAX_D || d < 1 || d > LST_MAX_d) return LST_E_SHAPE;
  if (m_max < 1 || m_max > LST_MAX_M || K_max < 0 || K_max > LST_MAX_K) return LST_E_SHAPE;
  if ((int64_t)m_max * K_max > 8192) return LST_E_SHAPE;
  return LST_OK;
}

int alloc_ws(lst_ctx *c, void (*carve)(lst_ctx *, Carver &)) {
  Carver probe{nullptr};
  carve(c, probe);
  c->ws_bytes = probe.off + 256;
  if (hipMalloc(&c->ws, c->ws_bytes) != hipSuccess) return LST_E_HIP;
  Carver real{static_cast<char *>(c->ws)};
  carve(c, real);
  if (hipMemsetAsync(c->ws, 0, c->ws_bytes, c->stream) != hipSuccess) return LST_E_HIP;
  if (hipStreamSynchronize(c->stream) != hipSuccess) return LST_E_HIP;
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

void graph_entry_free(GraphEntry &g) {
  hipGraphExec_t ex[3] = {g.exec_a, g.exec_side, g.exec_b};
  for (hipGraphExec_t e : ex)
    if (e) (void)hipGraphExecDestroy(e);
}

int side_create(lst_ctx *c) {
  for (int i = 0; i < 1; ++i)
    if (hipStreamCreateWithFlags(&c->side[i], hipStreamNonBlocking) != hipSuccess) return LST_E_HIP;
  if (hipStreamCreateWithFlags(&c->cap, hipStreamNonBlocking) != hipSuccess) return LST_E_HIP;
  c->have_side = true;
  return LST_OK;
}

void side_free(lst_ctx *c) {
  if (!c->have_side) return;
  for (int i = 0; i < 1; ++i)
    if (c->side[i]) (void)hipStreamDestroy(c->side[i]);
  if (c->cap) (void)hipStreamDestroy(c->cap);
  for (GraphEntry &g : c->graphs) graph_entry_free(g);
  c->graphs.clear();
  c->have_side = false;
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

int lst_create(lst_ctx **out, int64_t D, int32_t d, int32_t m_max, int32_t K_max, int32_t loss,
               float eps, float *V, int64_t ldv, float *U, float *UinvT, float *Q, int32_t ldd,
               void *stream) {
  if (!out) return LST_E_ARG;
  *out = nullptr;
  int st = common_args(D, d, m_max, K_max, loss, eps);
  if (st != LST_OK) return st;
  if (!V || !U || !UinvT || !Q) return LST_E_ARG;
  if (ldv < d || ldd < d) return LST_E_SHAPE;
  lst_ctx *c = new (std::nothrow) lst_ctx{};
  if (!c) return LST_E_ARG;
  c->kind = KIND_FACTORED;
  c->D = D;
  c->d = d;
  c->m_max = m_max;
  c->K_max = K_max;
  c->loss = loss;
  c->eps = eps;
  c->stream = static_cast<hipStream_t>(stream);
  c->V = V;
  c->ldv = ldv;
  c->U = U;
  c->UinvT = UinvT;
  c->Q = Q;
  c->ldd = ldd;
  c->last_err = hipSuccess;
  c->use_graphs = false;
  c->withhold_release = std::getenv("LST_TEST_WITHHOLD_WOODBURY_RELEASE") != nullptr;
  c->one_stream = std::getenv("LST_ONE_STREAM") != nullptr;
  {
    const char *ok = std::getenv("LST_ONLINE_KERNEL");
    c->online = loss == LST_LOSS_SQUARED && !(ok && std::strcmp(ok, "0") == 0);
  }
  st = alloc_ws(c, carve_factored);
  if (st == LST_OK) st = side_create(c);
  if (st != LST_OK) {
    lst_destroy(c);
    return st;
  }
  *out = c;
  return LST_OK;
}

int lst_naive_create(lst_ctx **out, int64_t D, int32_t d, int32_t m_max, int32_t K_max,
                     int32_t loss, float eps, float *W, int64_t ldw, void *stream) {
  if (!out) return LST_E_ARG;
  *out = nullptr;
  int st = common_args(D, d, m_max, K_max, loss, eps);
  if (st != LST_OK) return st;
  if (!W) return LST_E_ARG;
  if (ldw < d) return LST_E_SHAPE;
  lst_ctx *c = new (std::nothrow) lst_ctx{};
  if (!c) return LST_E_ARG;
  c->kind = KIND_NAIVE;
  c->D = D;
  c->d = d;
  c->m_max = m_max;
  c->K_max = K_max;
  c->loss = loss;
  c->eps = eps;
  c->stream = static_cast<hipStream_t>(stream);
  c->W = W;
  c->ldw = ldw;
  c->last_err = hipSuccess;
  st = alloc_ws(c, carve_naive);
  if (st != LST_OK) {
    lst_destroy(c);
    return st;
  }
  *out = c;
  return LST_OK;
}

void lst_destroy(lst_ctx *c) {
  if (!c) return;
  if (c->ws) {
    (void)hipStreamSynchronize(c->stream);
    (void)hipFree(c->ws);
  }
  if (c->have_side)
    for (int i = 0; i < 1; ++i) (void)hipStreamSynchronize(c->side[i]);
  side_free(c);
  prof_free(c);
  delete c;
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
  if (c->have_side)
    for (int i = 0; i < 1; ++i)
      if (hipStreamSynchronize(c->side[i]) != hipSuccess) return LST_E_HIP;
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
    // Both streams are idle: restart the progress counters from a consistent state.
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
  // Q = U^T (V^T V) U  (Q = V^T V when U = I), V^T V split over D.
  GemmDesc g = gemm_desc(d, d, (int)c->D, c->V, c->ldv, 1, c->V, c->ldv, 1, nullptr, d);
  const size_t pf = gemm_plan_split(g, kTargetWGs, nullptr);
  float *tmp = nullptr;
  const size_t tmp_floats = pf + 2 * (size_t)d * d + 64;
  if (record(c, hipMalloc(&tmp, tmp_floats * sizeof(float)))) return LST_E_HIP;
  float *part = tmp, *Gm = tmp + ((pf + 63) / 64) * 64, *Tm = Gm + (size_t)d * d;
  gemm_plan_split(g, kTargetWGs, part);
  GemmBatch b{};
  int st = LST_OK;
  if (!U0) {
    g.C = c->Q;
    g.ldc = c->ldd;
    b.d[0] = g;
    b.n = 1;
    if (record(c, gemm_launch(b, nullptr, s))) st = LST_E_HIP;
  } else {
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
  const int zero = 0;
  if (record(c, hipStreamSynchronize(s))) st = LST_E_HIP;
  (void)hipFree(tmp);
  if (record(c, hipMemcpy(c->flag, &zero, sizeof(int), hipMemcpyHostToDevice))) st = LST_E_HIP;
  return st;
}

}  // extern "C"

namespace {

// Enqueues one factored step on stream s (and the context's side streams).
void gemm_run(GemmBatch &b, const int *gate, hipStream_t s, int phase = GEMM_OTHER) {
  gemm_prepare(b);
  gemm_enqueue(b, gate, s, phase);
}

// The step's GEMM batches for minibatch size m, with H and grad_H as placeholders.
void build_plan(const lst_ctx *c, int m, GemmBatch (&b)[kPlanBatches]) {
  const int d = c->d, ldd = c->ldd;
  const float *H = sym_H();
  float *gH = sym_gradH();
  for (GemmBatch &x : b) x = GemmBatch{};
  // N = H^T H (Woodbury branch)
  b[0].d[0] = gemm_desc(m, m, d, H, d, 0, H, d, 0, c->N, m);
  b[0].n = 1;
  // H^ = Q H, H~ = U H, X = U^{-T} H (Algorithm 3 steps 1, 5, 6; Algorithm 4 rows 1, 5)
  b[1].d[0] = gemm_desc(m, d, d, H, d, 0, c->Q, ldd, 0, c->Hhat, d);
  b[1].d[1] = gemm_desc(m, d, d, H, d, 0, c->U, ldd, 0, c->Htil, d);
  b[1].d[2] = gemm_desc(m, d, d, H, d, 0, c->UinvT, ldd, 0, c->X, d);
  b[1].n = 3;
  // Z^ = U^T G with grad_H = 2 H^ diag(dl/dq) + Z^; M^ = H^T H^; H^T Z^ = H~^T G
  GemmDesc z = gemm_desc(m, d, d, c->G, d, 0, c->U, ldd, 1, c->Zhat, d);
  z.epi = EPI_GRADH;
  z.rs = c->dq;
  z.E = c->Hhat;
  z.lde = d;
  z.C2 = gH;
  z.ldc2 = d;
  b[2].d[0] = z;
  b[2].d[1] = gemm_desc(m, m, d, H, d, 0, c->Hhat, d, 0, c->Mhat, m);
  b[2].d[2] = gemm_desc(m, m, d, c->Htil, d, 0, c->G, d, 0, c->HZ, m);
  b[2].n = 3;
  // Yw = R X; Zq = (eta^2/2) M H - eta grad_H; U <- U - 2 eta H~ diag(dl/dq) H^T
  // (eq. updateU / gen-updateU).  Zq's alpha and beta scale with eta at launch.
  b[3].d[0] = gemm_desc(m, d, m, c->R, m, 0, c->X, d, 1, c->Yw, d);
  GemmDesc zq = gemm_desc(m, d, m, c->M, m, 0, H, d, 1, c->Zq, d, 0.5f, gH, d, -1.f);
  zq.lr_scaled = 1;
  b[3].d[1] = zq;
  b[3].d[2] = gemm_desc(d, d, m, c->Atil, d, 1, H, d, 1, c->U, ldd, -1.f, c->U, ldd, 1.f);
  b[3].n = 3;
  // U^{-T} += (2 eta X S C^{-1} S) H^T (Woodbury); Q += H Zq^T + Zq H^T (eq. updateQ /
  // gen-Qnew); P = U_new^{-T} H = X + (2 eta X S C^{-1} S)(H^T H).
  b[4].d[0] = gemm_desc(d, d, m, c->Yw, d, 1, H, d, 1, c->UinvT, ldd, 1.f, c->UinvT, ldd, 1.f);
  GemmDesc qd = gemm_desc(d, d, m, H, d, 1, c->Zq, d, 1, c->Q, ldd, 1.f, c->Q, ldd, 1.f);
  qd.A2 = c->Zq;
  qd.lda2 = d;
  qd.B2 = H;
  qd.ldb2 = d;
  qd.K2 = m;
  b[4].d[1] = qd;
  // P is needed for the spherical softmax only: for squared error S = I, and with
  // 2 eta N = I - C one has I + N R = I + (I - C) C^{-1} = C^{-1}, so P = C^{-1} X
  // = Yw / (2 eta) and the V update (eq. updateV) uses Yw with the factor 1/2.
  b[4].d[2] = gemm_desc(m, d, m, c->N, m, 0, c->Yw, d, 1, c->P, d, 1.f, c->X, d, 1.f);
  b[4].n = c->loss == LST_LOSS_SQUARED ? 2 : 3;
  // 16 x 16 tiles where the outputs are m x m or m x d with long k (Gram product,
  // contractions, Z^): four times the workgroups of 32 x 32 tiles.  The d x d
  // updates (short k = m, read-modify-write of the state) keep 32 x 32 tiles.
  for (int i = 0; i < kPlanBatches; ++i) {
    b[i].t16 = i <= 2 ? 1 : 0;
    gemm_prepare(b[i]);
  }
  // The contraction launch also reads the step's target rows of V into the caches
  // (one workgroup per example, on the XCD of that example's gather workgroup).
  b[1].pf_V = c->V;
  b[1].pf_D = c->D;
  b[1].pf_ldv = c->ldv;
  b[1].pf_d = d;
  b[1].pf_m = m;
  b[1].pf_base = (b[1].total_tiles + 7) / 8 * 8;
}

// The plan for m, built and copied to its device slot on first use.  Replacing
// the least recently used plan first drains the streams and drops the recorded
// graphs that launch it.
PlanEntry *get_plan(lst_ctx *c, int m) {
  for (PlanEntry &e : c->plans)
    if (e.m == m) {
      e.last_use = ++c->plan_tick;
      return &e;
    }
  GemmBatch *slot;
  if (c->plans.size() < kPlanCap) {
    slot = c->plan_pool + c->plans.size() * kPlanBatches;
    c->plans.push_back(PlanEntry{});
  } else {
    size_t v = 0;
    for (size_t i = 1; i < c->plans.size(); ++i)
      if (c->plans[i].last_use < c->plans[v].last_use) v = i;
    if (record(c, hipStreamSynchronize(c->stream)) || record(c, hipStreamSynchronize(c->side[0])))
      return nullptr;
    const int old_m = c->plans[v].m;
    for (size_t i = c->graphs.size(); i-- > 0;)
      if (c->graphs[i].m == old_m) {
        graph_entry_free(c->graphs[i]);
        c->graphs.erase(c->graphs.begin() + i);
      }
    slot = c->plans[v].dev;
    c->plans.erase(c->plans.begin() + v);
    c->plans.push_back(PlanEntry{});
  }
  PlanEntry &e = c->plans.back();
  e.m = m;
  e.dev = slot;
  build_plan(c, m, e.b);
  if (record(c, hipMemcpy(e.dev, e.b, sizeof(e.b), hipMemcpyHostToDevice))) {
    c->plans.pop_back();
    return nullptr;
  }
  e.last_use = ++c->plan_tick;
  return &e;
}

// A step runs on two streams ordered by the progress counters c->cnt (no host
// events): the main stream signals when its contraction launch starts (the
// step's inputs are ready and the previous step has consumed N and R); the side
// stream then forms N = H^T H and the Woodbury inverse and releases R; the main
// stream waits for that before the state updates.  Each wait is a kernel of one
// workgroup (many polling workgroups slow the step down).
// The parts are launched in the order main (to M), side, main (updates), so that
// every wait's producer is launched before it even where the two streams share
// a hardware queue.

// Main stream up to M: contractions, gather and loss epilogue, Z^ and grad_H, M.
int enqueue_main_a(lst_ctx *c, hipStream_t s, const PlanEntry &pl, const float *H, int32_t m,
                   const int32_t *idx, const float *val, int32_t K, float lr, float *loss_dev,
                   float *gH) {
  const bool unit_dq = (c->loss == LST_LOSS_SQUARED);
  auto gemm = [&](int i, int phase, int *sig) {
    StepSync sy;
    sy.sig = sig;
    gemm_enqueue_plan(pl.b[i], pl.dev + i, H, gH, lr, nullptr, s, phase, i == 1 ? idx : nullptr,
                      K, sy);
  };
  prof(c, LST_PHASE_CONTRACT, true);
  gemm(1, GEMM_CONTRACT, c->cnt + 0);
  prof(c, LST_PHASE_CONTRACT, false);

  // Sparse gather of the K target rows of the pre-update V and the loss epilogue.
  prof(c, LST_PHASE_GATHER, true);
  launch_gather(s, m, K, c->d, c->D, H, c->Hhat, c->Htil, idx, val, c->V, c->ldv, c->loss, c->eps,
                lr, c->G, c->Atil, c->dq, c->dA, c->lvec, c->flag);
  prof(c, LST_PHASE_GATHER, false);

  // Z^ and grad_H; its start tells the spherical softmax's Woodbury branch that
  // dl/dq is ready.
  prof(c, LST_PHASE_ZGRAD, true);
  gemm(2, GEMM_ZGRAD, unit_dq ? nullptr : c->cnt + 2);
  prof(c, LST_PHASE_ZGRAD, false);

  // Loss and M; sets the error flag on a non-finite loss.
  prof(c, LST_PHASE_MBLOCK, true);
  launch_mblock(s, m, K, idx, c->lvec, c->dq, c->dA, c->Mhat, c->HZ, c->M, loss_dev, c->flag);
  prof(c, LST_PHASE_MBLOCK, false);
  return record(c, hipGetLastError()) ? LST_E_HIP : LST_OK;
}

// Side stream: N = H^T H, then C = I - 2 eta S N S and R = 2 eta S C^{-1} S (for
// m > d, through the d x d inverse of I - 2 eta (SH)^T (SH): the m >= d variant the
// paper suggests after Algorithm 3, here as the same Woodbury R).  For squared error
// dl/dq = 1; the spherical softmax waits for the gather's dl/dq = T / (q + D eps).
int enqueue_side(lst_ctx *c, hipStream_t s, const PlanEntry &pl, const float *H, int32_t m,
                 float lr, float *gH) {
  const bool unit_dq = (c->loss == LST_LOSS_SQUARED);
  StepSync started;  // the main stream has reached this step's contraction
  started.wx = c->cnt + 0;
  started.wy = c->cnt + 1;
  started.wd = 1;
  started.flag = c->flag;
  launch_step_sync(s, started, nullptr);
  prof(c, LST_PHASE_GRAM, true);
  gemm_enqueue_plan(pl.b[0], pl.dev + 0, H, gH, lr, nullptr, s, GEMM_OTHER);
  prof(c, LST_PHASE_GRAM, false);
  StepSync gathered;
  if (!unit_dq) {
    gathered.wx = c->cnt + 2;
    gathered.wy = c->cnt + 1;
    gathered.wd = 1;
    gathered.flag = c->flag;
  }
  prof(c, LST_PHASE_WOODBURY, true);
  int *done = c->withhold_release ? nullptr : c->cnt + 1;
  const int d = c->d;
  if (m > kWoodburyOneWG && d < m) {
    // m > d: the d x d inverse of B = I - 2 eta Hs^T Hs instead of the m x m one (see
    // push_through_r_kernel): R' = 2 eta B^{-1} into Sd0, then R = 2 eta S (I + Hs R' Hs^T) S.
    const float *Hs = H;
    if (!unit_dq) {
      launch_step_sync(s, gathered, nullptr);
      launch_scale_rows_sqrt(s, m, d, H, c->dq, c->P, c->flag);
      Hs = c->P;
    }
    GemmBatch b{};
    b.d[0] = gemm_desc(d, d, m, Hs, d, 1, Hs, d, 1, c->Sd1, d);  // Hs^T Hs
    b.n = 1;
    gemm_run(b, nullptr, s);
    launch_woodbury(s, d, lr, 1, c->dq, c->Sd1, c->Sd0, c->Cwork, c->Pbig, c->Cp, c->Rp, c->flag,
                    StepSync{}, nullptr);
    b = GemmBatch{};
    b.d[0] = gemm_desc(m, d, d, Hs, d, 0, c->Sd0, d, 1, c->Zq, d);  // T = Hs R'
    b.n = 1;
    gemm_run(b, nullptr, s);
    b = GemmBatch{};
    b.d[0] = gemm_desc(m, m, d, c->Zq, d, 0, Hs, d, 0, c->R, m);  // R0 = T Hs^T
    b.n = 1;
    gemm_run(b, nullptr, s);
    launch_push_through_r(s, m, lr, unit_dq ? 1 : 0, c->dq, c->R);
    if (done) launch_step_sync(s, StepSync{}, done);
  } else {
    launch_woodbury(s, m, lr, unit_dq ? 1 : 0, c->dq, c->N, c->R, c->Cwork, c->Pbig, c->Cp, c->Rp,
                    c->flag, gathered, done);
  }
  prof(c, LST_PHASE_WOODBURY, false);
  return record(c, hipGetLastError()) ? LST_E_HIP : LST_OK;
}

// Main stream: the gated state updates (see build_plan) once the side stream has
// released this step's R (and its error flag), then the scatter into V.
int enqueue_main_b(lst_ctx *c, hipStream_t s, const PlanEntry &pl, const float *H, int32_t m,
                   const int32_t *idx, int32_t K, float lr, float *gH) {
  StepSync joined;
  joined.wx = c->cnt + 1;
  joined.wy = c->cnt + 0;
  joined.wd = 0;
  joined.flag = c->flag;
  launch_step_sync(s, joined, nullptr);
  prof(c, LST_PHASE_MID, true);
  gemm_enqueue_plan(pl.b[3], pl.dev + 3, H, gH, lr, c->flag, s, GEMM_MID);
  prof(c, LST_PHASE_MID, false);
  // V_r -= eta sum dl/dA P_j over the slots of each distinct target row (eq. updateV).
  // For squared error eta P = Yw / 2 (see build_plan): the scatter needs nothing
  // from the update launch and runs in it; the spherical softmax's P comes from it.
  const bool squared = c->loss == LST_LOSS_SQUARED;
  prof(c, LST_PHASE_UPDATE, true);
  const bool fused =
      squared && m * K > 0 &&
      gemm_enqueue_plan_scatter(pl.b[4], pl.dev + 4, H, gH, lr, c->flag, s, m * K, K, c->d, 0.5f,
                                idx, c->dA, c->Yw, c->V, c->ldv);
  if (!fused) gemm_enqueue_plan(pl.b[4], pl.dev + 4, H, gH, lr, c->flag, s, GEMM_UPDATE);
  prof(c, LST_PHASE_UPDATE, false);
  if (!fused) {
    prof(c, LST_PHASE_SCATTER, true);
    launch_scatter(s, m, K, c->d, squared ? 0.5f : lr, idx, c->dA, squared ? c->Yw : c->P, c->V,
                   c->ldv, c->flag);
    prof(c, LST_PHASE_SCATTER, false);
  }
  // Kernel launches above are not checked one by one: a launch error stays pending
  // and is reported here.
  return record(c, hipGetLastError()) ? LST_E_HIP : LST_OK;
}

int enqueue_factored_step(lst_ctx *c, const PlanEntry &pl, const float *H, int32_t m,
                          const int32_t *idx, const float *val, int32_t K, float lr,
                          float *loss_dev, float *grad_H) {
  float *gH = grad_H ? grad_H : c->gradH;
  int st = enqueue_main_a(c, c->stream, pl, H, m, idx, val, K, lr, loss_dev, gH);
  if (st == LST_OK) st = enqueue_side(c, c->one_stream ? c->stream : c->side[0], pl, H, m, lr, gH);
  if (st == LST_OK) st = enqueue_main_b(c, c->stream, pl, H, m, idx, K, lr, gH);
  return st;
}

// Replays (capturing first if needed) the graph of a step with these arguments.
int graph_step(lst_ctx *c, const PlanEntry &pl, const float *H, int32_t m, const int32_t *idx,
               const float *val, int32_t K, float lr, float *loss_dev, float *grad_H) {
  uint32_t lr_bits;
  std::memcpy(&lr_bits, &lr, sizeof(lr_bits));
  GraphEntry *hit = nullptr;
  for (GraphEntry &g : c->graphs)
    if (g.H == H && g.idx == idx && g.val == val && g.loss == loss_dev && g.grad == grad_H &&
        g.m == m && g.K == K && g.lr_bits == lr_bits) {
      hit = &g;
      break;
    }
  if (!hit) {
    if (c->graphs.size() >= kGraphCap) {  // evict the least recently used graph
      size_t v = 0;
      for (size_t i = 1; i < c->graphs.size(); ++i)
        if (c->graphs[i].last_use < c->graphs[v].last_use) v = i;
      if (record(c, hipStreamSynchronize(c->stream)) || record(c, hipStreamSynchronize(c->side[0])))
        return LST_E_HIP;
      graph_entry_free(c->graphs[v]);
      c->graphs.erase(c->graphs.begin() + v);
    }
    float *gH = grad_H ? grad_H : c->gradH;
    // The step's three parts are captured one after the other on the capture stream.
    auto capture = [&](int part, hipGraphExec_t *exec) -> int {
      if (record(c, hipStreamBeginCapture(c->cap, hipStreamCaptureModeThreadLocal)))
        return LST_E_HIP;
      const int st =
          part == 0   ? enqueue_main_a(c, c->cap, pl, H, m, idx, val, K, lr, loss_dev, gH)
          : part == 1 ? enqueue_side(c, c->cap, pl, H, m, lr, gH)
                      : enqueue_main_b(c, c->cap, pl, H, m, idx, K, lr, gH);
      hipGraph_t graph = nullptr;
      const hipError_t ec = hipStreamEndCapture(c->cap, &graph);
      if (st != LST_OK || ec != hipSuccess || !graph) {
        if (graph) (void)hipGraphDestroy(graph);
        if (ec != hipSuccess) c->last_err = ec;
        return st != LST_OK ? st : LST_E_HIP;
      }
      const hipError_t ei = hipGraphInstantiate(exec, graph, nullptr, nullptr, 0);
      (void)hipGraphDestroy(graph);
      return record(c, ei) ? LST_E_HIP : LST_OK;
    };
    GraphEntry e{H, idx, val, loss_dev, grad_H, m, K, lr_bits, nullptr, nullptr, nullptr, 0};
    int st = capture(0, &e.exec_a);
    if (st == LST_OK) st = capture(1, &e.exec_side);
    if (st == LST_OK) st = capture(2, &e.exec_b);
    if (st != LST_OK) {
      graph_entry_free(e);
      return st;
    }
    c->graphs.push_back(e);
    hit = &c->graphs.back();
  }
  hit->last_use = ++c->graph_tick;
  if (record(c, hipGraphLaunch(hit->exec_a, c->stream)) ||
      record(c, hipGraphLaunch(hit->exec_side, c->one_stream ? c->stream : c->side[0])))
    return LST_E_HIP;
  return record(c, hipGraphLaunch(hit->exec_b, c->stream));
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
        loss_dev, grad_H, c->spart, reinterpret_cast<unsigned *>(c->cnt + 3), c->flag);
    prof(c, LST_PHASE_ONLINE, false);
    return record(c, e);
  }
  const PlanEntry *pl = get_plan(c, m);
  if (!pl) return LST_E_HIP;
  if (graphs) return graph_step(c, *pl, H, m, idx, val, K, lr, loss_dev, grad_H);
  return enqueue_factored_step(c, *pl, H, m, idx, val, K, lr, loss_dev, grad_H);
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
  if (gemm_big_ok(fwd)) {
    fwd.colsq = c->colpart;
    gemm_big_plan(fwd, kTargetWGs, 0, nullptr);
    nparts = kBigColsqRows * fwd.tiles_m;
    if (record(c, gemm_big_launch(fwd, nullptr, s, GEMM_NAIVE_FWD))) return LST_E_HIP;
  } else {
    if (record(c, naive_gemm(c, fwd, false, nullptr, s, GEMM_NAIVE_FWD)) ||
        record(c, launch_colnorm(s, c->O, D, m, c->colpart, kColnormBlocks)))
      return LST_E_HIP;
  }
  prof(c, LST_PHASE_NAIVE_FWD, false);
  // The loss and dl/dq, dl/da from the explicit O.
  prof(c, LST_PHASE_NAIVE_LOSS, true);
  if (record(c, launch_naive_epilogue(s, m, K, D, nparts, c->colpart, c->O, idx, val, c->loss,
                                      c->eps, c->dq, c->dA, c->lvec, c->flag)))
    return LST_E_HIP;
  // grad_O = 2 O diag(dl/dq) + Yring, in place over O.
  if (record(c, launch_grad_o(s, c->O, D, m, K, c->dq, idx, c->dA, c->lvec, loss_dev, c->flag)))
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
