// Host-side checks of liblst built without device code under AddressSanitizer and
// UndefinedBehaviorSanitizer (no GPU is touched):
//  * every entry point's argument and workspace validation, with the status it returns;
//  * the step's product descriptors (build_step_plan over many shapes, every loss): each
//    operand a descriptor names lies, at the largest index a kernel forms from it, inside
//    the one buffer the pointer starts in (the carved intermediates, H, grad_H or the
//    state), tile ranges cover each batch exactly, and a fallback descriptor has the
//    shape of the one it replaces.
// Exit status 0 when every check holds; the sanitizers abort on the first report.
#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "lst.h"
#include "lst_internal.h"

using namespace lst;

namespace {

int g_fail = 0;
#define CHECK(c, ...)                           \
  do {                                          \
    if (!(c)) {                                 \
      std::fprintf(stderr, "FAIL: " __VA_ARGS__); \
      std::fprintf(stderr, "\n");               \
      ++g_fail;                                 \
    }                                           \
  } while (0)

struct Range {
  uintptr_t lo, hi;  // [lo, hi) bytes
  const char *name;
};

// Address ranges of the buffers a plan may name; pointers are never dereferenced.
struct Space {
  std::vector<Range> r;
  uintptr_t H = 0, gH = 0;
  void add(const char *n, uintptr_t lo, size_t bytes) { r.push_back({lo, lo + bytes, n}); }
  uintptr_t res(const void *p) const {
    const uintptr_t v = reinterpret_cast<uintptr_t>(p);
    return v == 16 ? H : (v == 32 ? gH : v);
  }
  // Elements [first, last] (floats or ints) from p stay inside p's buffer.
  void in(const char *what, const void *p, int64_t last, size_t elem = 4) const {
    const uintptr_t a = res(p);
    CHECK(a != 0, "%s: null operand", what);
    if (!a) return;
    const Range *hit = nullptr;
    for (const Range &x : r)
      if (a >= x.lo && a < x.hi) hit = &x;
    CHECK(hit != nullptr, "%s: pointer outside every buffer", what);
    if (!hit) return;
    CHECK(last >= 0, "%s: negative extent", what);
    CHECK(a + (uintptr_t)(last + 1) * elem <= hit->hi, "%s: extent %lld past the end of %s",
          what, (long long)last, hit->name);
  }
};

int64_t last2(int rows, int cols, int ld, int tr) {  // largest index of a rows x cols operand
  return tr ? (int64_t)(cols - 1) * ld + (rows - 1) : (int64_t)(rows - 1) * ld + (cols - 1);
}

void check_op(const Space &sp, const Op16 &g, const char *tag) {
  if (g.M <= 0 || g.N <= 0) return;
  char w[160];
  if (g.amode == AM_PLAIN) {
    std::snprintf(w, sizeof w, "%s A", tag);
    sp.in(w, g.A, last2(g.M, g.K, g.lda, g.tA));
  } else {
    std::snprintf(w, sizeof w, "%s M^", tag);
    sp.in(w, g.Mh, last2(g.M, g.K, (int)g.ldm, 0));
    sp.in(w, g.YY, last2(g.M, g.K, (int)g.ldm, 0));
    sp.in(w, g.HZ, last2(g.M, g.K, (int)g.ldm, 0));
    sp.in(w, g.HZ, last2(g.M, g.K, (int)g.ldm, 1));
    if (g.amode == AM_MASM_S) {
      sp.in(w, g.ds, g.K - 1);
      sp.in(w, g.yb, g.K - 1);
      sp.in(w, g.ds, g.M - 1);
    }
  }
  for (int t = 0; t < g.nb; ++t) {
    std::snprintf(w, sizeof w, "%s B%d", tag, t);
    // B(k, j): tr = 0 -> p[j ld + k], tr = 1 -> p[k ld + j]
    sp.in(w, g.b[t].p, g.b[t].tr ? (int64_t)(g.K - 1) * g.b[t].ld + (g.N - 1)
                                  : (int64_t)(g.N - 1) * g.b[t].ld + (g.K - 1));
  }
  for (int t = 0; t < g.nadd; ++t) {
    std::snprintf(w, sizeof w, "%s add%d", tag, t);
    sp.in(w, g.add[t].p, last2(g.M, g.N, (int)g.add[t].ld, 0));
  }
  for (int r = 0; r < g.nuv; ++r) {
    std::snprintf(w, sizeof w, "%s uv%d", tag, r);
    sp.in(w, g.ux[r], (int64_t)(g.M - 1) * g.uxi[r]);
    sp.in(w, g.uy[r], (int64_t)(g.N - 1) * g.uyi[r]);
  }
  std::snprintf(w, sizeof w, "%s C", tag);
  if (g.C) sp.in(w, g.C, last2(g.M, g.N, (int)g.ldc, 0));
  if (g.Cin) sp.in(w, g.Cin, last2(g.M, g.N, (int)g.ldcin, 0));
  if (g.C2) {
    sp.in(w, g.C2, last2(g.M, g.N, (int)g.ldc2, 0));
    sp.in(w, g.E, last2(g.M, g.N, (int)g.lde, 0));
  }
  if (g.rowred != RR_NONE) {
    std::snprintf(w, sizeof w, "%s rowred", tag);
    if (g.rowred == RR_DOT) sp.in(w, g.Rr, last2(g.M, g.N, (int)g.ldrr, 0));
    sp.in(w, g.rowout, (int64_t)g.tiles_n * g.M - 1);
    if (g.qout) {
      sp.in(w, g.qout, g.M - 1);
      sp.in(w, g.qcnt, g.tiles_m - 1);
    }
  }
  CHECK(g.tiles_m == (g.M + 15) / 16 && g.tiles_n == (g.N + 15) / 16, "%s: tile counts", tag);
}

void check_batch(const Space &sp, const OpBatch &ob, const char *tag) {
  CHECK(ob.n >= ob.n_main && ob.n <= kMaxOps, "%s: descriptor counts", tag);
  int total = 0;
  for (int q = 0; q < ob.n_main; ++q) {
    const Op16 &g = ob.op[q];
    const int t = (g.M > 0 && g.N > 0) ? g.tiles_m * g.tiles_n : 0;
    CHECK(t == 0 || g.tile_begin == total, "%s op %d: tile_begin %d, expected %d", tag, q,
          g.tile_begin, total);
    total += t;
    if (g.alt >= 0) {
      CHECK(g.alt >= ob.n_main && g.alt < ob.n, "%s op %d: alt index", tag, q);
      if (g.alt < ob.n)
        CHECK(ob.op[g.alt].M == g.M && ob.op[g.alt].N == g.N, "%s op %d: alt shape", tag, q);
    }
  }
  CHECK(total == ob.total, "%s: total %d, tiles %d", tag, ob.total, total);
  for (int q = 0; q < ob.n; ++q) {
    char w[96];
    std::snprintf(w, sizeof w, "%s op %d", tag, q);
    check_op(sp, ob.op[q], w);
  }
}

void check_gemm(const Space &sp, const GemmBatch &gb, const char *tag) {
  CHECK(gb.n >= 0 && gb.n <= kMaxBatch, "%s: batch size", tag);
  for (int i = 0; i < gb.n; ++i) {
    const GemmDesc &g = gb.d[i];
    char w[96];
    std::snprintf(w, sizeof w, "%s desc %d", tag, i);
    // opA(i,k): tA = 0 -> A[i lda + k]; opB(k,j): tB = 0 -> B[j ldb + k], tB = 1 -> B[k ldb + j]
    sp.in(w, g.A, g.tA ? (int64_t)(g.K - 1) * g.lda + (g.M - 1) : (int64_t)(g.M - 1) * g.lda + (g.K - 1));
    sp.in(w, g.B, g.tB ? (int64_t)(g.K - 1) * g.ldb + (g.N - 1) : (int64_t)(g.N - 1) * g.ldb + (g.K - 1));
    if (g.A2 && g.K2 > 0) {  // the second k segment, same transpositions
      sp.in(w, g.A2, g.tA ? (int64_t)(g.K2 - 1) * g.lda2 + (g.M - 1)
                          : (int64_t)(g.M - 1) * g.lda2 + (g.K2 - 1));
      sp.in(w, g.B2, g.tB ? (int64_t)(g.K2 - 1) * g.ldb2 + (g.N - 1)
                          : (int64_t)(g.N - 1) * g.ldb2 + (g.K2 - 1));
    }
    // C may be null under the grad_H epilogue (the product itself not kept)
    CHECK(g.C || g.epi == EPI_GRADH, "%s: no output", w);
    if (g.C) sp.in(w, g.C, (int64_t)(g.M - 1) * g.ldc + (g.N - 1));
    if (g.Cin) sp.in(w, g.Cin, (int64_t)(g.M - 1) * g.ldcin + (g.N - 1));
    // the 32 x 32 body scales by lr only in mode 1
    CHECK(g.lr_scaled != 2 || gb.tile == 64, "%s: lr scaling mode 2 on 32 x 32 tiles", w);
    // operand terms, addends, alternatives (64 x 64 tiles, one k segment)
    if (g.nat > 1 || g.Atr || g.nbt > 1 || g.nadd > 0 || g.alt1 > 0)
      CHECK(gb.tile == 64 && g.K2 == 0 && g.tA == 0 && g.tB == 1 && g.nat <= 3 && g.nbt <= 4 &&
                g.nadd <= 4,
            "%s: operand terms", w);
    for (int t = 1; t < g.nat && t < 3; ++t)
      sp.in(w, g.At[t - 1], (int64_t)(g.M - 1) * g.lda + (g.K - 1));
    if (g.Atr) sp.in(w, g.Atr, (int64_t)(g.K - 1) * g.lda + (g.M - 1));
    for (int t = 1; t < g.nbt && t < 4; ++t)
      sp.in(w, g.Bt[t - 1], (int64_t)(g.K - 1) * g.ldb + (g.N - 1));
    for (int t = 0; t < g.nadd && t < 4; ++t)
      sp.in(w, g.addp[t], (int64_t)(g.M - 1) * g.ldadd + (g.N - 1));
    if (g.nbt > 1 || g.nadd > 0) {
      CHECK(g.coef != nullptr, "%s: coefficients", w);
      if (g.coef) sp.in(w, g.coef, 7);
      for (int t = 0; t < 4; ++t)
        CHECK((t >= g.nbt || (g.bcoef[t] >= 0 && g.bcoef[t] < 8)) &&
                  (t >= g.nadd || (g.acoef[t] >= 0 && g.acoef[t] < 8)),
              "%s: coefficient index", w);
    }
    if (g.alt1 > 0) {  // outside the batch, same shape, plain, its operands in range
      CHECK(g.alt1 - 1 >= gb.n && g.alt1 - 1 < kMaxBatch, "%s: alternative index", w);
      if (g.alt1 - 1 >= gb.n && g.alt1 - 1 < kMaxBatch) {
        const GemmDesc &a = gb.d[g.alt1 - 1];
        CHECK(a.M == g.M && a.N == g.N && a.tiles_m == g.tiles_m && a.tiles_n == g.tiles_n &&
                  a.nat <= 1 && !a.Atr && a.nbt <= 1 && a.nadd == 0 && a.alt1 == 0 && a.K2 == 0,
              "%s: alternative shape", w);
        sp.in(w, a.A, a.tA ? (int64_t)(a.K - 1) * a.lda + (a.M - 1)
                           : (int64_t)(a.M - 1) * a.lda + (a.K - 1));
        sp.in(w, a.B, a.tB ? (int64_t)(a.K - 1) * a.ldb + (a.N - 1)
                           : (int64_t)(a.N - 1) * a.ldb + (a.K - 1));
        sp.in(w, a.C, (int64_t)(a.M - 1) * a.ldc + (a.N - 1));
      }
    }
    if (g.epi == EPI_GRADH) {
      CHECK(gb.tile == 64 || g.C, "%s: the 32 x 32 grad_H epilogue stores C", w);
      sp.in(w, g.C2, (int64_t)(g.M - 1) * g.ldc2 + (g.N - 1));
      sp.in(w, g.E, (int64_t)(g.M - 1) * g.lde + (g.N - 1));
      if (g.rs) sp.in(w, g.rs, g.M - 1);
    }
    CHECK(g.splits == 1, "%s: split descriptors in a step plan", w);
    // the tile bookkeeping the kernels decode (32 x 32 tiles, or the 64 x 64 tiles,
    // which have no fused epilogue)
    CHECK(gb.tile == 32 || gb.tile == 64, "%s: tile edge %d", w, gb.tile);
    CHECK(g.tiles_m == (g.M + gb.tile - 1) / gb.tile && g.tiles_n == (g.N + gb.tile - 1) / gb.tile,
          "%s: tile counts", w);
    CHECK(gb.tile == 32 || g.colsq == nullptr, "%s: column sums on 64 x 64 tiles", w);
  }
  int total = 0;
  for (int i = 0; i < gb.n; ++i) {
    const GemmDesc &g = gb.d[i];
    const int t = (g.M > 0 && g.N > 0) ? g.tiles_m * g.tiles_n : 0;
    CHECK(t == 0 || g.tile_begin == total, "%s desc %d: tile_begin %d, expected %d", tag, i,
          g.tile_begin, total);
    total += t;
  }
  CHECK(gb.n == 0 || total == gb.total_tiles, "%s: total %d, tiles %d", tag, gb.total_tiles, total);
  // the header's per-product counts, and the section covering every tile exactly once
  const GemmHdr h = gemm_hdr(gb);
  int sum = 0;
  for (int i = 0; i < kMaxBatch; ++i) sum += h.count[i];
  CHECK(gb.n == 0 || sum == gb.total_tiles, "%s: header counts %d, tiles %d", tag, sum, gb.total_tiles);
  if (gb.n > 0 && gb.tile == 64) {
    std::vector<int> seen(gb.total_tiles, 0);
    const int ns = gemm_section(h, 64);
    for (int w = 0; w < ns; ++w) {
      const int t = gemm_tile64(h, w);
      CHECK(t >= -1 && t < gb.total_tiles, "%s: section tile %d out of range", tag, t);
      if (t >= 0 && t < gb.total_tiles) ++seen[t];
    }
    for (int t = 0; t < gb.total_tiles; ++t)
      CHECK(seen[t] == 1, "%s: 64 x 64 tile %d owned %d times", tag, t, seen[t]);
  }
}

void plans() {
  const int ms[] = {1, 2, 15, 16, 17, 100, 128, 257, 512};
  const int ds[] = {1, 7, 32, 500, 513, 1024};
  const int Ks[] = {0, 1, 5, 16};
  int n = 0;
  for (int loss = 0; loss < 3; ++loss)
    for (int m : ms)
      for (int d : ds)
        for (int K : Ks)
          for (int pad : {0, 3}) {
            if (m * K > 8192) continue;
            const int ldd = d + pad;
            const uintptr_t base = uintptr_t(1) << 40;
            StepBufs b{};
            float *gradH = nullptr;
            Carver cv{reinterpret_cast<char *>(base)};
            carve_step(b, gradH, (size_t)m, (size_t)d, (size_t)K, cv);
            Space sp;
            // every carved piece ends where the next begins (or at the end of the carve)
            std::vector<std::pair<uintptr_t, const char *>> p = {
                {(uintptr_t)b.Hhat, "H^"}, {(uintptr_t)b.Htil, "H~"}, {(uintptr_t)b.X, "X"},
                {(uintptr_t)b.G, "G"}, {(uintptr_t)b.Atil, "2 eta D H~"}, {(uintptr_t)b.W1, "W1"},
                {(uintptr_t)b.P2, "P2"}, {(uintptr_t)b.P3, "P3"}, {(uintptr_t)b.RX, "RX"},
                {(uintptr_t)b.Zq, "Zq"}, {(uintptr_t)gradH, "grad_H stand-in"},
                {(uintptr_t)b.N, "N"}, {(uintptr_t)b.Mhat, "M^"}, {(uintptr_t)b.HZ, "HZ"},
                {(uintptr_t)b.YY, "YY"}, {(uintptr_t)b.E2, "E2"}, {(uintptr_t)b.E4, "E4"},
                {(uintptr_t)b.R, "R"}, {(uintptr_t)b.Cwork, "Cwork"}, {(uintptr_t)b.qpart, "qpart"},
                {(uintptr_t)b.bpart, "bpart"}, {(uintptr_t)b.q, "q"}, {(uintptr_t)b.tsum, "tsum"},
                {(uintptr_t)b.qcnt, "qcnt"}, {(uintptr_t)b.dq, "dq"}, {(uintptr_t)b.lvec, "lvec"},
                {(uintptr_t)b.rcnt, "rcnt"}, {(uintptr_t)b.splan, "splan"}, {(uintptr_t)b.wA, "wA"}, {(uintptr_t)b.sval, "sval"},
                {(uintptr_t)b.srow, "srow"}, {(uintptr_t)b.scnt, "scnt"}, {(uintptr_t)b.coef, "coef"},
                {(uintptr_t)b.cert, "cert"}, {(uintptr_t)b.SW, "SW"}, {(uintptr_t)b.ds, "ds"},
                {(uintptr_t)b.yb, "yb"}, {(uintptr_t)b.cwo, "cwo"}};
            std::sort(p.begin(), p.end());
            for (size_t i = 0; i < p.size(); ++i) {
              const uintptr_t hi = i + 1 < p.size() ? p[i + 1].first : base + cv.off;
              CHECK(p[i].first < hi, "carve: empty piece %s", p[i].second);
              sp.add(p[i].second, p[i].first, hi - p[i].first);
            }
            // the caller's arrays, each in its own address range
            const uintptr_t st = uintptr_t(1) << 44, gap = uintptr_t(1) << 36;
            sp.H = st;
            sp.add("H", sp.H, (size_t)m * d * 4);
            sp.gH = st + gap;
            sp.add("grad_H", sp.gH, (size_t)m * d * 4);
            b.U = reinterpret_cast<float *>(st + 2 * gap);
            sp.add("U", (uintptr_t)b.U, (size_t)d * ldd * 4);
            b.UinvT = reinterpret_cast<float *>(st + 3 * gap);
            sp.add("U^-T", (uintptr_t)b.UinvT, (size_t)d * ldd * 4);
            b.Q = reinterpret_cast<float *>(st + 4 * gap);
            sp.add("Q", (uintptr_t)b.Q, (size_t)d * ldd * 4);
            b.WO = loss == LST_LOSS_TAYLOR_SOFTMAX ? reinterpret_cast<float *>(st + 5 * gap) : nullptr;
            if (b.WO) sp.add("WO", (uintptr_t)b.WO, (size_t)2 * ldd * 4);
            b.D = 200000;
            b.d = d;
            b.ldd = ldd;
            b.loss = loss;
            b.eps = 1e-3f;
            StepPlan pl;
            build_step_plan(b, m, pl);
            char tag[96];
            for (int l = 0; l < 4; ++l) {
              std::snprintf(tag, sizeof tag, "loss %d m %d d %d K %d ldd %d launch %d", loss, m, d, K,
                            ldd, l + 1);
              check_batch(sp, pl.ob[l], tag);
            }
            std::snprintf(tag, sizeof tag, "loss %d m %d d %d K %d ldd %d contraction", loss, m, d,
                          K, ldd);
            check_gemm(sp, pl.gb_contract, tag);
            std::snprintf(tag, sizeof tag, "loss %d m %d d %d K %d ldd %d launch 3 32 x 32", loss, m,
                          d, K, ldd);
            check_gemm(sp, pl.gb_zgrad, tag);
            std::snprintf(tag, sizeof tag, "loss %d m %d d %d K %d ldd %d U update", loss, m, d, K, ldd);
            check_gemm(sp, pl.gb_mid, tag);
            std::snprintf(tag, sizeof tag, "loss %d m %d d %d K %d ldd %d Q/U^-T update", loss, m, d,
                          K, ldd);
            check_gemm(sp, pl.gb_update, tag);
            ++n;
          }
  std::printf("plans checked: %d\n", n);
}

void abi() {
  void *P = reinterpret_cast<void *>(uintptr_t{0x1000});
  float *F = static_cast<float *>(P);
  void *WS = reinterpret_cast<void *>(uintptr_t{0x100000});
  lst_ctx *c = nullptr;
  const size_t nb = lst_workspace_bytes(1000, 32, 16, 3, 0);
  CHECK(nb > 0 && nb % 256 == 0, "workspace bytes %zu", nb);
  CHECK(lst_workspace_bytes(0, 32, 16, 3, 0) == 0, "D = 0 sized");
  CHECK(lst_workspace_bytes(1000, 0, 16, 3, 0) == 0, "d = 0 sized");
  CHECK(lst_workspace_bytes(1000, 32, 2000, 3, 0) == 0, "m above the limit sized");
  CHECK(lst_workspace_bytes(1000, 32, 512, 64, 0) == 0, "m K above the limit sized");
  CHECK(lst_naive_workspace_bytes(1000, 32, 16, 3, 0) >= (size_t)1000 * 16 * 4, "naive bytes");
  for (int d = 1; d <= 4096; d *= 4)
    for (int m = 1; m <= 1024; m *= 4)
      for (int loss = 0; loss < 3; ++loss)
        CHECK(lst_workspace_bytes(2147483647LL, d, m, 8, loss) > 0, "large D sizes");
  CHECK(lst_create(nullptr, 1000, 32, 16, 3, 0, 1e-3f, F, 32, F, F, F, F, 32, WS, nb, nullptr) ==
            LST_E_ARG, "null out");
  struct Case {
    int64_t D;
    int d, m, K, loss;
    float eps;
    float *V;
    int64_t ldv;
    float *WO;
    int ldd;
    void *ws;
    size_t wsb;
    int want;
  } cases[] = {
      {0, 32, 16, 3, 0, 1e-3f, F, 32, F, 32, WS, nb, LST_E_SHAPE},
      {1000, 32, 16, 3, 5, 1e-3f, F, 32, F, 32, WS, nb, LST_E_ARG},
      {1000, 32, 16, 3, 1, 0.f, F, 32, F, 32, WS, nb, LST_E_ARG},
      {1000, 32, 16, 3, 1, -1.f, F, 32, F, 32, WS, nb, LST_E_ARG},
      {1000, 32, 16, 3, 0, 1e-3f, nullptr, 32, F, 32, WS, nb, LST_E_ARG},
      {1000, 32, 16, 3, 0, 1e-3f, F, 31, F, 32, WS, nb, LST_E_SHAPE},
      {1000, 32, 16, 3, 0, 1e-3f, F, 32, F, 31, WS, nb, LST_E_SHAPE},
      {1000, 32, 16, 3, 2, 1e-3f, F, 32, nullptr, 32, WS, nb, LST_E_ARG},
      {1000, 5000, 16, 3, 0, 1e-3f, F, 5000, F, 5000, WS, nb, LST_E_SHAPE},
      {1000, 32, 16, 3, 0, 1e-3f, F, 32, F, 32, nullptr, nb, LST_E_ARG},
      {1000, 32, 16, 3, 0, 1e-3f, F, 32, F, 32, static_cast<char *>(WS) + 4, nb, LST_E_ARG},
      {1000, 32, 16, 3, 0, 1e-3f, F, 32, F, 32, WS, nb - 256, LST_E_SHAPE},
  };
  for (const Case &k : cases) {
    c = reinterpret_cast<lst_ctx *>(P);
    const int st = lst_create(&c, k.D, k.d, k.m, k.K, k.loss, k.eps, k.V, k.ldv, F, F, F, k.WO,
                              k.ldd, k.ws, k.wsb, nullptr);
    CHECK(st == k.want && c == nullptr, "lst_create case D %lld d %d: %d, expected %d",
          (long long)k.D, k.d, st, k.want);
  }
  CHECK(lst_naive_create(&c, 1000, 32, 16, 3, 0, 1e-3f, F, 32, WS,
                         lst_naive_workspace_bytes(1000, 32, 16, 3, 0) - 256, nullptr) == LST_E_SHAPE,
        "naive workspace too small");
  CHECK(lst_step(nullptr, F, 1, nullptr, nullptr, 0, 0.1f, F, nullptr) == LST_E_ARG, "lst_step null");
  CHECK(lst_naive_step(nullptr, F, 1, nullptr, nullptr, 0, 0.1f, F, nullptr) == LST_E_ARG, "naive null");
  CHECK(lst_sync_status(nullptr) == LST_E_ARG, "sync null");
  CHECK(lst_set_option(nullptr, 0, 1) == LST_E_ARG, "option null");
  CHECK(lst_materialize_W(nullptr, F, 8) == LST_E_ARG, "materialize null");
  CHECK(lst_init_factored(nullptr, nullptr, 0, nullptr, 0) == LST_E_ARG, "init null");
  CHECK(lst_use_graphs(nullptr, 1) == LST_E_ARG, "graphs null");
  CHECK(lst_profile_enable(nullptr, 1) == LST_E_ARG, "profile null");
  CHECK(lst_restore_pristine(nullptr) == LST_E_ARG, "restore null");
  CHECK(lst_refresh_uinvt(nullptr, 2, 0, nullptr) == LST_E_ARG, "refresh null");
  CHECK(lst_input_forward(nullptr, 8, 10, 8, nullptr, nullptr, 1, 1, F, reinterpret_cast<int32_t *>(P),
                          nullptr) == LST_E_ARG, "input forward null");
  CHECK(lst_input_update(F, 8, 10, 8, nullptr, nullptr, 1, 65, F, 0.1f, reinterpret_cast<int32_t *>(P),
                         nullptr) == LST_E_SHAPE, "input update K");
  int32_t *S = reinterpret_cast<int32_t *>(P);
  CHECK(lst_step_noalloc(200000, 500, 0, 1e-3f, nullptr, 500, F, F, F, nullptr, 500, F, 128, S, F, 5,
                         0.1f, F, F, S, nullptr) == LST_E_ARG, "noalloc null V");
  CHECK(lst_step_noalloc(200000, 500, 2, 1e-3f, F, 500, F, F, F, nullptr, 500, F, 128, S, F, 5, 0.1f,
                         F, F, S, nullptr) == LST_E_ARG, "noalloc Taylor without WO");
  CHECK(lst_step_noalloc(200000, 3000, 0, 1e-3f, F, 3000, F, F, F, nullptr, 3000, F, 128, S, F, 5,
                         0.1f, F, F, S, nullptr) == LST_E_SHAPE, "noalloc beyond the array");
  CHECK(lst_step_noalloc(200000, 500, 0, 1e-3f, F, 500, F, F, F, nullptr, 500, F, -1, S, F, 5, 0.1f,
                         F, F, S, nullptr) == LST_E_SHAPE, "noalloc m < 0");
  for (int s = -9; s <= 1; ++s) CHECK(lst_status_string(s) != nullptr, "status string %d", s);
  lst_destroy(nullptr);
}

}  // namespace

int main() {
  abi();
  plans();
  if (g_fail) {
    std::fprintf(stderr, "%d checks failed\n", g_fail);
    return 1;
  }
  std::printf("all host checks passed\n");
  return 0;
}
