// C-ABI of the library: argument validation, search-space layout, workspace carving,
// and the orchestration of the kernels for gp_fit / gp_score (declared in baco_gp.h).
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <memory>
#include <mutex>
#include <string>
#include <vector>

#include "common.h"

using namespace bgp;

namespace {

thread_local std::string g_err;

gp_status fail(gp_status st, const std::string &msg) {
  g_err = msg;
  return st;
}

#define HIPCHK(expr)                                                                    \
  do {                                                                                  \
    hipError_t e_ = (expr);                                                             \
    if (e_ != hipSuccess)                                                               \
      return fail(GP_E_HIP, std::string(#expr) + " failed: " + hipGetErrorString(e_));  \
  } while (0)

inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

// Bump allocator over the caller's workspace; with base == nullptr it only measures.
struct Carver {
  char *base = nullptr;
  size_t size = SIZE_MAX;
  size_t off = 0;
  bool ok = true;
  template <class T>
  T *take(int64_t count) {
    const size_t bytes = (size_t)round_up((int64_t)std::max<int64_t>(count, 1) * (int64_t)sizeof(T), 256);
    if (off + bytes > size) ok = false;
    T *p = base ? reinterpret_cast<T *>(base + off) : nullptr;
    off += bytes;
    return p;
  }
};

// ------------------------------------------------------------------ space layout
struct Layout {
  int d = 0, R = 0;
  int R_bound = 0;  // R for any lengthscales (each categorical in its own word)
  int n_num = 0, n_bits = 0, n_eq = 0, n_dot = 0;
  int w_bits0 = 0, w_eq0 = 0, w_dot0 = 0;
  std::vector<ParamEnc> penc;   // encode order
  std::vector<double> table;    // transformed ordinal values
  std::vector<TermDesc> tdesc;  // space order
  std::vector<double> num_scale; // 1 / l per NUM word
  Weights64 w64{};
  std::vector<float> bits_w, eq_w, dot_w2;
  std::vector<int32_t> dot_s2;
};

gp_status build_layout(const gp_space *sp, const double *ls, Layout &L) {
  if (!sp) return fail(GP_E_INVALID, "space is NULL");
  const int d = sp->d;
  if (d < 1) return fail(GP_E_INVALID, "space.d must be >= 1");
  if (d > kMaxD) return fail(GP_E_UNSUPPORTED, "space.d must be <= 64");
  if (!sp->type) return fail(GP_E_INVALID, "space.type is NULL");
  L = Layout();
  L.d = d;
  std::vector<double> l(d, 1.0);
  if (ls) {
    for (int p = 0; p < d; ++p) {
      if (!(ls[p] > 0.0) || !std::isfinite(ls[p]))
        return fail(GP_E_INVALID, "lengthscale[" + std::to_string(p) + "] must be finite and > 0");
      l[p] = ls[p];
    }
  }
  auto levels = [&](int p) { return sp->n_levels ? sp->n_levels[p] : 0; };
  auto islog = [&](int p) { return sp->log2 && sp->log2[p] != 0; };

  struct CatItem { int p; double w; int lv; };
  std::vector<CatItem> cats;
  std::vector<int> nums, kend, hamm, spear, eqs;
  for (int p = 0; p < d; ++p) {
    const int t = sp->type[p];
    const std::string where = "parameter " + std::to_string(p) + ": ";
    if (t == GP_REAL || t == GP_INT) {
      if (!sp->lo || !sp->hi) return fail(GP_E_INVALID, where + "lo/hi required");
      const double lo = sp->lo[p], hi = sp->hi[p];
      if (!std::isfinite(lo) || !std::isfinite(hi) || !(lo <= hi))
        return fail(GP_E_INVALID, where + "need finite lo <= hi");
      if (islog(p) && !(lo > 0.0)) return fail(GP_E_INVALID, where + "log2 needs lo > 0");
      if (t == GP_INT && (lo != std::floor(lo) || hi != std::floor(hi) || lo < -2147483648.0 ||
                          hi > 2147483647.0))
        return fail(GP_E_INVALID, where + "integer bounds must be int32 values");
      nums.push_back(p);
    } else if (t == GP_ORD) {
      const int lv = levels(p);
      if (lv < 1 || lv > 4096) return fail(GP_E_INVALID, where + "ordinal needs 1..4096 values");
      if (!sp->ord_values || !sp->ord_values[p]) return fail(GP_E_INVALID, where + "ord_values missing");
      for (int k = 0; k < lv; ++k) {
        const double v = sp->ord_values[p][k];
        if (!std::isfinite(v)) return fail(GP_E_INVALID, where + "ordinal value not finite");
        if (k && !(v > sp->ord_values[p][k - 1]))
          return fail(GP_E_INVALID, where + "ordinal values must be strictly ascending");
        if (islog(p) && !(v > 0.0)) return fail(GP_E_INVALID, where + "log2 needs values > 0");
      }
      nums.push_back(p);
    } else if (t == GP_CAT) {
      const int lv = levels(p);
      if (lv < 1 || lv > 65536) return fail(GP_E_INVALID, where + "categorical needs 1..65536 levels");
      if (islog(p)) return fail(GP_E_INVALID, where + "log2 is for numeric parameters");
      if (lv <= 32) cats.push_back({p, 1.0 / (2.0 * l[p] * l[p]), lv});
      else eqs.push_back(p);
    } else if (t == GP_PERM) {
      const int m = levels(p);
      if (m < 2 || m > 8) return fail(GP_E_UNSUPPORTED, where + "permutations need 2..8 items");
      if (islog(p)) return fail(GP_E_INVALID, where + "log2 is for numeric parameters");
      const int dist = sp->perm_dist ? sp->perm_dist[p] : GP_PERM_SPEARMAN;
      if (dist == GP_PERM_KENDALL) kend.push_back(p);
      else if (dist == GP_PERM_HAMMING) hamm.push_back(p);
      else if (dist == GP_PERM_SPEARMAN) spear.push_back(p);
      else if (dist == GP_PERM_NAIVE) eqs.push_back(p);
      else return fail(GP_E_INVALID, where + "unknown permutation distance");
    } else {
      return fail(GP_E_INVALID, where + "unknown parameter type");
    }
  }
  L.tdesc.resize(d);
  // NUM words
  L.n_num = (int)nums.size();
  for (int q = 0; q < L.n_num; ++q) {
    const int p = nums[q];
    const int t = sp->type[p];
    ParamEnc e{};
    e.kind = t;
    e.col = p;
    e.word = q;
    e.bit = -1;
    e.flags = islog(p) ? 1 : 0;
    e.num_index = q;
    e.table = -1;
    double t_lo, t_hi;
    if (t == GP_ORD) {
      const int lv = levels(p);
      e.levels = lv;
      e.table = (int)L.table.size();
      for (int k = 0; k < lv; ++k) {
        const double v = sp->ord_values[p][k];
        L.table.push_back(islog(p) ? std::log2(v) : v);
      }
      t_lo = L.table[e.table];
      t_hi = L.table[e.table + lv - 1];
    } else {
      e.lo = sp->lo[p];
      e.hi = sp->hi[p];
      t_lo = islog(p) ? std::log2(e.lo) : e.lo;
      t_hi = islog(p) ? std::log2(e.hi) : e.hi;
    }
    e.t_lo = t_lo;
    e.den = t_hi - t_lo;
    L.penc.push_back(e);
    L.num_scale.push_back(1.0 / l[p]);
    L.w64.num_w[q] = 1.0 / (l[p] * l[p]);
    L.tdesc[p] = TermDesc{t, q, -1, 0, 0};
  }
  // BITS words: categorical one-hot fields grouped by weight, Kendall, Hamming
  L.w_bits0 = L.n_num;
  auto bits_word = [&](double w) {
    L.bits_w.push_back((float)w);
    L.w64.bits_w[L.bits_w.size() - 1] = w;
    return L.w_bits0 + (int)L.bits_w.size() - 1;
  };
  std::stable_sort(cats.begin(), cats.end(), [](const CatItem &a, const CatItem &b) { return a.w < b.w; });
  int cur_word = -1, used = 0;
  double curw = -1.0;
  for (const CatItem &c : cats) {
    if (cur_word < 0 || c.w != curw || used + c.lv > 32) {
      cur_word = bits_word(c.w);
      used = 0;
      curw = c.w;
    }
    ParamEnc e{};
    e.kind = GP_CAT;
    e.col = c.p;
    e.word = cur_word;
    e.bit = used;
    e.levels = c.lv;
    e.num_index = -1;
    e.table = -1;
    L.penc.push_back(e);
    L.tdesc[c.p] = TermDesc{GP_CAT, cur_word, used, c.lv, 0};
    used += c.lv;
  }
  for (int p : kend) {
    const int m = levels(p);
    const int wd = bits_word(1.0 / (l[p] * l[p] * (m * (m - 1) / 2.0)));
    ParamEnc e{};
    e.kind = GP_PERM; e.col = p; e.word = wd; e.bit = -1; e.levels = m;
    e.flags = GP_PERM_KENDALL << 8; e.num_index = -1; e.table = -1;
    L.penc.push_back(e);
    L.tdesc[p] = TermDesc{GP_PERM, wd, -1, m, GP_PERM_KENDALL};
  }
  for (int p : hamm) {
    const int m = levels(p);
    const double w = 1.0 / (2.0 * l[p] * l[p] * m);
    const int wd = bits_word(w);
    bits_word(w);
    ParamEnc e{};
    e.kind = GP_PERM; e.col = p; e.word = wd; e.bit = -1; e.levels = m;
    e.flags = GP_PERM_HAMMING << 8; e.num_index = -1; e.table = -1;
    L.penc.push_back(e);
    L.tdesc[p] = TermDesc{GP_PERM, wd, -1, m, GP_PERM_HAMMING};
  }
  L.n_bits = (int)L.bits_w.size();
  // EQ words: categoricals above 32 levels, naive permutations
  L.w_eq0 = L.w_bits0 + L.n_bits;
  for (int p : eqs) {
    const int wd = L.w_eq0 + (int)L.eq_w.size();
    const double w = 1.0 / (l[p] * l[p]);
    L.eq_w.push_back((float)w);
    L.w64.eq_w[L.eq_w.size() - 1] = w;
    ParamEnc e{};
    e.kind = sp->type[p]; e.col = p; e.word = wd; e.bit = -1; e.levels = levels(p);
    e.num_index = -1; e.table = -1;
    if (sp->type[p] == GP_PERM) {
      e.flags = GP_PERM_NAIVE << 8;
      L.tdesc[p] = TermDesc{GP_PERM, wd, -1, levels(p), GP_PERM_NAIVE};
    } else {
      L.tdesc[p] = TermDesc{GP_CAT, wd, -1, levels(p), 0};
    }
    L.penc.push_back(e);
  }
  L.n_eq = (int)L.eq_w.size();
  // DOT words: Spearman permutations (2 words each)
  L.w_dot0 = L.w_eq0 + L.n_eq;
  for (int p : spear) {
    const int m = levels(p);
    const int q = (int)L.dot_w2.size();
    const int wd = L.w_dot0 + 2 * q;
    const double w = 1.0 / (l[p] * l[p] * ((double)m * m * m - m) / 3.0);
    L.dot_w2.push_back((float)(2.0 * w));
    L.dot_s2.push_back((m - 1) * m * (2 * m - 1) / 6);
    L.w64.dot_w2[q] = 2.0 * w;
    L.w64.dot_s2[q] = (m - 1) * m * (2 * m - 1) / 6;
    ParamEnc e{};
    e.kind = GP_PERM; e.col = p; e.word = wd; e.bit = -1; e.levels = m;
    e.flags = GP_PERM_SPEARMAN << 8; e.num_index = -1; e.table = -1;
    L.penc.push_back(e);
    L.tdesc[p] = TermDesc{GP_PERM, wd, -1, m, GP_PERM_SPEARMAN};
  }
  L.n_dot = (int)L.dot_w2.size();
  L.R = L.w_dot0 + 2 * L.n_dot;
  L.R_bound = L.n_num + (int)cats.size() + (int)kend.size() + 2 * (int)hamm.size() +
              (int)eqs.size() + 2 * (int)spear.size();
  if (L.n_bits > kMaxBitsWords || L.n_eq > kMaxEqWords || L.n_dot > kMaxDot || L.R > kMaxWords)
    return fail(GP_E_UNSUPPORTED, "search space needs too many code words");
  L.w64.n_num = L.n_num;
  L.w64.n_bits = L.n_bits;
  L.w64.n_eq = L.n_eq;
  L.w64.n_dot = L.n_dot;
  L.w64.w_bits0 = L.w_bits0;
  L.w64.w_eq0 = L.w_eq0;
  L.w64.w_dot0 = L.w_dot0;
  return GP_OK;
}

// ------------------------------------------------------------------ profiling
// Per scoring call: events 0..GP_STAGE_COUNT bound the stages in order. A scoring fused
// with a fit contracts in two launches on two streams: events S+1, S+2 bound the early
// one (value tiles) and event S+3 marks the start of the late one, whose end is event 3;
// its encoding runs on a stream of its own, ended by event S+4 (event 1 then marks the
// cross-kernel's start). The epilogue and the fp64 recomputation each run in two parts
// (the value model's, which a fused scoring runs early on the value stream, and the
// rest): events S+5 .. S+7 mark the value epilogue's start and end and the end of the
// recomputation's block path, S+8 the start of the classifier's epilogue (whose end is
// event 4).
constexpr int kProfEvents = GP_STAGE_COUNT + 9;
constexpr int kProfEarly = GP_STAGE_COUNT + 1, kProfLate = GP_STAGE_COUNT + 3;
constexpr int kProfEncEnd = GP_STAGE_COUNT + 4;
constexpr int kProfValEpi = GP_STAGE_COUNT + 5, kProfClsEpi = GP_STAGE_COUNT + 8;
struct Profiler {
  std::mutex mu;
  bool on = false;
  std::vector<hipEvent_t> pool;
  std::vector<std::pair<int, bool>> calls;  // first event index per call; split contraction
  int next = 0;
} g_prof;

constexpr int kProfMaxCalls = 4096;

// Events for one scoring call, or nullptr when not recording.
hipEvent_t *prof_begin(bool split_contraction = false) {
  std::lock_guard<std::mutex> lk(g_prof.mu);
  if (!g_prof.on || (int)g_prof.calls.size() >= kProfMaxCalls) return nullptr;
  while ((int)g_prof.pool.size() < g_prof.next + kProfEvents) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    g_prof.pool.push_back(e);
  }
  hipEvent_t *ev = &g_prof.pool[g_prof.next];
  g_prof.calls.push_back({g_prof.next, split_contraction});
  g_prof.next += kProfEvents;
  return ev;
}

}  // namespace

// ------------------------------------------------------------------ model handle
struct gp_model {
  Layout lay;
  int n = 0, n_f = 0, lda = 0, variant = -1;
  XObsLayout xl{};
  double sv = 1.0, nv = 0.0, csv = 0.0, fstar = 0.0;
  bool has_cls = false;
  int cls_iters = 0;
  mutable bool inv_ready = false;  // d_Linv, d_Kinv formed (on first export)
  std::vector<int32_t> order;  // model row -> original observation index
  ParamEnc *d_penc = nullptr;
  double *d_table = nullptr;
  TermDesc *d_tdesc = nullptr;
  uint32_t *d_codes = nullptr;
  double *d_xa = nullptr;     // cross-kernel observation operands
  uint32_t *d_xr = nullptr;   // and records
  double *d_K = nullptr, *d_L = nullptr, *d_Linv = nullptr, *d_B64 = nullptr, *d_Kinv = nullptr;
  double *d_alpha = nullptr;
  uint16_t *d_Bt = nullptr;   // split fp16 packed B^T
  float *d_cscale = nullptr;  // its column unscaling factors
  int kexp = 0;               // K* is split after scaling by 2^kexp
  double *d_cf = nullptr, *d_cgrad = nullptr, *d_csw = nullptr, *d_cL = nullptr;
  int n_reg_tiles = 0, ntiles = 0;
  CTile tiles[kMaxTiles];
  XArgs xa{};  // template of the cross-kernel arguments
  double refine_var = 1e-2, refine_sens = 300.0;
};

namespace {

struct FitPlan {
  ParamEnc *penc; double *table; TermDesc *tdesc; double *num_scale;
  int32_t *order; uint8_t *valid; int32_t *info;
  uint32_t *codes, *xr;
  double *xa;
  double *yf, *K, *Aw, *L, *Dv, *Linv, *B64, *Kinv, *beta, *alpha, *fstar;
  uint16_t *Bt;
  float *cscale;
  // classifier
  double *Kc, *Bm, *LB, *LE, *Dc, *t, *f, *fnew, *grad, *W, *sw, *b, *v, *z2;
  NewtonScratch *nscr;
};

FitPlan plan_fit(Carver &cv, const Layout &L, int n, bool cls) {
  FitPlan P{};
  const int lda = (int)round_up(n, kKChunk);
  P.penc = cv.take<ParamEnc>(L.d);
  P.table = cv.take<double>((int64_t)L.table.size());
  P.tdesc = cv.take<TermDesc>(L.d);
  P.num_scale = cv.take<double>(kMaxD);
  P.order = cv.take<int32_t>(n);
  P.valid = cv.take<uint8_t>(n);
  P.info = cv.take<int32_t>(4);
  P.codes = cv.take<uint32_t>((int64_t)n * L.R_bound);
  // cross-kernel observation side, sized for the largest variant (the variant depends
  // on the lengthscales through the grouping of categoricals)
  P.xa = cv.take<double>((int64_t)xobs_a_doubles_max(n));
  P.xr = cv.take<uint32_t>((int64_t)xobs_r_words_max(n));
  P.yf = cv.take<double>(n);
  const int64_t nn = (int64_t)n * n;
  const int64_t nblk = (n + kNB - 1) / kNB;
  P.K = cv.take<double>(nn);
  P.Aw = cv.take<double>(2 * nn);  // [K; I]
  P.L = cv.take<double>(nn);
  P.Dv = cv.take<double>(nblk * kNB * kNB);
  P.Linv = cv.take<double>(nn);
  P.B64 = cv.take<double>(nn);
  P.Kinv = cv.take<double>(nn);
  P.beta = cv.take<double>(n);
  P.alpha = cv.take<double>(n);
  P.fstar = cv.take<double>(1);
  // value and classifier column tiles, and one more for the classifier's dense column
  // when neither last tile has a spare sub-tile for it
  const int64_t bcols = round_up(n, kColTile) * (cls ? 2 : 1) + (cls ? kColTile : 0);
  P.Bt = cv.take<uint16_t>(bcols * 2 * lda);
  P.cscale = cv.take<float>(bcols);
  if (cls) {
    P.Kc = cv.take<double>(nn);
    // [B ; I] and the identity rows' panels (L_B^-T)
    P.Bm = cv.take<double>(2 * nn);
    P.LB = cv.take<double>(nn);
    P.LE = cv.take<double>(nn);
    P.Dc = cv.take<double>(nblk * kNB * kNB);
    P.t = cv.take<double>(n);
    P.f = cv.take<double>(n);
    P.fnew = cv.take<double>(n);
    P.grad = cv.take<double>(n);
    P.W = cv.take<double>(n);
    P.sw = cv.take<double>(n);
    P.b = cv.take<double>(n);
    P.v = cv.take<double>(n);
    P.z2 = cv.take<double>((int64_t)kGemvSlices * n);
    P.nscr = cv.take<NewtonScratch>(1);
  }
  return P;
}

struct ScorePlan {
  uint32_t *cand; uint8_t *valid; uint16_t *Kstar; double *mu64; float *sens, *fbar, *part, *pwork;
  int32_t *rlist, *rcount; float *amax_v; int64_t *amax_i;
  double *rpart, *rmup;
  double *rpart64, *rmu64;  // block path of the refinement ([tiles][rows], [rows])
  XSplit xs;
};
constexpr int kArgmaxBlocks = 1024;

// Scoring buffers for rows candidate rows; every size grows with each argument, so a plan
// for upper bounds of them (used before a fit has fixed them) covers the actual plan.
ScorePlan plan_score(Carver &cv, int R, int lda, int ntiles, int n_f, int n, int64_t rows) {
  ScorePlan P{};
  P.rcount = cv.take<int32_t>(64);
  P.cand = cv.take<uint32_t>((int64_t)R * rows);
  P.valid = cv.take<uint8_t>(rows);
  P.Kstar = cv.take<uint16_t>(rows * 2 * lda);
  P.mu64 = cv.take<double>(rows);
  P.sens = cv.take<float>(rows);
  P.fbar = cv.take<float>(rows);
  P.part = cv.take<float>((int64_t)ntiles * rows);
  P.pwork = cv.take<float>(rows);
  P.rlist = cv.take<int32_t>(rows);
  const int64_t nr = (n_f + kRefineColRange - 1) / kRefineColRange;
  P.rpart = cv.take<double>((int64_t)kRefineSplitGroups * nr * 8);
  P.rmup = cv.take<double>((int64_t)kRefineSplitGroups * 8);
  if (rows > kRefineBlockMin) {
    P.rpart64 = cv.take<double>((int64_t)((n_f + kRefineBlockCols - 1) / kRefineBlockCols) * rows);
    P.rmu64 = cv.take<double>(rows);
  }
  P.amax_v = cv.take<float>(kArgmaxBlocks);
  P.amax_i = cv.take<int64_t>(kArgmaxBlocks);
  P.xs.nsplit = xkernel_splits(rows, n);
  if (P.xs.nsplit > 1) {
    P.xs.mu = cv.take<double>(P.xs.nsplit * rows);
    P.xs.sens = cv.take<float>(P.xs.nsplit * rows);
  }
  return P;
}
ScorePlan plan_score(Carver &cv, const gp_model &m, int64_t rows) {
  return plan_score(cv, m.lay.R, m.lda, m.ntiles, m.n_f, m.n, rows);
}
// Column tiles of the contraction at most: value and classifier tiles and one for the
// classifier's dense column.
int max_tiles(int n, bool cls) {
  const int t = (int)((n + kColTile - 1) / kColTile);
  return cls ? 2 * t + 1 : t;
}

gp_status check_ws(const void *ws, size_t have, size_t need) {
  if (!ws) return fail(GP_E_WORKSPACE, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(ws) % 256) return fail(GP_E_WORKSPACE, "workspace must be 256-byte aligned");
  if (have < need)
    return fail(GP_E_WORKSPACE, "workspace too small: need " + std::to_string(need) + " bytes, have " +
                                    std::to_string(have));
  return GP_OK;
}

gp_status check_cols(const void *const *cols, int d) {
  if (!cols) return fail(GP_E_INVALID, "column array is NULL");
  for (int p = 0; p < d; ++p)
    if (!cols[p]) return fail(GP_E_INVALID, "column " + std::to_string(p) + " is NULL");
  return GP_OK;
}

// Encode launcher bound to a layout uploaded at (penc, table).
hipError_t encode_into(const Layout &L, const void *const *cols, const ParamEnc *penc,
                       const double *table, int64_t count, int64_t rows, const int32_t *rowmap,
                       uint32_t *out, int64_t s_word, int64_t s_row, uint8_t *valid, float *num_out,
                       int32_t *clear, hipStream_t s);

}  // namespace

namespace {
hipError_t encode_into(const Layout &L, const void *const *cols, const ParamEnc *penc,
                       const double *table, int64_t count, int64_t rows, const int32_t *rowmap,
                       uint32_t *out, int64_t s_word, int64_t s_row, uint8_t *valid, float *num_out,
                       int32_t *clear, hipStream_t s) {
  return launch_encode(cols, L.d, penc, table, count, rows, rowmap, out, s_word, s_row, valid,
                       num_out, L.n_num, clear, s);
}

gp_status upload_layout(const Layout &L, ParamEnc *penc, double *table, TermDesc *tdesc,
                        hipStream_t s) {
  HIPCHK(hipMemcpyAsync(penc, L.penc.data(), sizeof(ParamEnc) * L.penc.size(), hipMemcpyHostToDevice, s));
  if (!L.table.empty())
    HIPCHK(hipMemcpyAsync(table, L.table.data(), sizeof(double) * L.table.size(), hipMemcpyHostToDevice, s));
  if (tdesc)
    HIPCHK(hipMemcpyAsync(tdesc, L.tdesc.data(), sizeof(TermDesc) * L.tdesc.size(), hipMemcpyHostToDevice, s));
  return GP_OK;
}

#define HIPRET(expr)              \
  do {                              \
    hipError_t e_ = (expr);         \
    if (e_ != hipSuccess) return e_; \
  } while (0)

// Scoring outputs (the gp_score arguments after the candidates).
struct ScoreOut {
  const uint8_t *mask;
  float eps_f;
  float *mu, *sigma, *ei, *p_feas, *acq;
  int64_t *argmax;
};

gp_status check_score_args(const Layout &L, const void *const *C_cols, int64_t M, const ScoreOut &o) {
  if (M < 0 || M > INT32_MAX) return fail(GP_E_INVALID, "M must be in 0..2^31-1");
  if (!(o.eps_f >= 0.f && o.eps_f <= 1.f)) return fail(GP_E_INVALID, "eps_f must be in [0, 1]");
  if (M == 0) return GP_OK;
  if (!o.mu || !o.sigma || !o.ei || !o.acq)
    return fail(GP_E_INVALID, "mu, sigma, ei and acq are required");
  return check_cols(C_cols, L.d);
}

// Candidate encoding (needs the space layout only).
hipError_t score_encode(const gp_model &m, const ScorePlan &P, const void *const *C_cols,
                        int64_t M, int64_t rows, hipStream_t s) {
  return encode_into(m.lay, C_cols, m.d_penc, m.d_table, M, rows, nullptr, P.cand, rows, 1,
                     P.valid, nullptr, P.rcount, s);
}

// The cross-kernel (K*, mu, sens) of encoded candidates, which needs the value model only
// (kstar false: the means only, K* not written).
hipError_t score_xkernel(const gp_model &m, const ScorePlan &P, int64_t rows, hipStream_t s,
                         bool kstar = true);

// First half of scoring: candidate encoding and the cross-kernel. ev: optional profiling
// events (stages 0..2).
hipError_t score_front(const gp_model &m, const ScorePlan &P, const void *const *C_cols, int64_t M,
                       int64_t rows, hipStream_t s, hipEvent_t *ev) {
  if (ev) HIPRET(hipEventRecord(ev[0], s));
  HIPRET(score_encode(m, P, C_cols, M, rows, s));
  if (ev) HIPRET(hipEventRecord(ev[1], s));
  HIPRET(score_xkernel(m, P, rows, s));
  if (ev) HIPRET(hipEventRecord(ev[2], s));
  return hipSuccess;
}

hipError_t score_xkernel(const gp_model &m, const ScorePlan &P, int64_t rows, hipStream_t s,
                         bool kstar) {
  XArgs xa = m.xa;
  xa.cand = P.cand;
  xa.ldc = rows;
  xa.Kstar = kstar ? P.Kstar : nullptr;
  xa.mu = P.mu64;
  xa.sens = P.sens;
  xa.rows = rows;
  return launch_xkernel(xa, m.variant, P.xs, s, false, false);  // the epilogue sums splits
}

// The contraction over the column tiles [t0, t1) of the model.
hipError_t contract_tiles(const gp_model &m, const ScorePlan &P, int64_t rows, int t0, int t1,
                          hipStream_t s) {
  if (t1 <= t0) return hipSuccess;
  CArgs ca{};
  ca.A = P.Kstar;
  ca.Bt = m.d_Bt;
  ca.cscale = m.d_cscale;
  ca.lda = m.lda;
  ca.ntiles = t1 - t0;
  ca.nrowtiles = (int)(rows / kRowTile);
  ca.part = P.part + (int64_t)t0 * rows;
  ca.lin = P.fbar;
  ca.rows = rows;
  for (int t = t0; t < t1; ++t) ca.tiles[t - t0] = m.tiles[t];
  return launch_contract(ca, s);
}

int stream_cus(hipStream_t s);

EArgs make_eargs(const gp_model &m, const ScorePlan &P, int64_t M, int64_t rows,
                 const ScoreOut &o) {
  EArgs ea{};
  ea.part = P.part;
  ea.rows = rows;
  ea.M = M;
  ea.ntiles = m.ntiles;
  ea.n_reg_tiles = m.n_reg_tiles;
  ea.has_cls = m.has_cls ? 1 : 0;
  ea.mu64 = P.mu64;
  ea.sens = P.sens;
  ea.nsplit = xkernel_splits(rows, m.xa.n);  // > 1: score_xkernel left the partials
  if (ea.nsplit > 1) {
    ea.pmu = P.xs.mu;
    ea.psens = P.xs.sens;
  }
  ea.fbar = P.fbar;
  ea.valid = P.valid;
  ea.mask = o.mask;
  ea.eps_f = o.eps_f;
  ea.sv = (float)m.sv;
  ea.cls_sv = (float)m.csv;
  ea.fstar = (float)m.fstar;
  ea.refine_var = (float)m.refine_var;
  ea.refine_sens = (float)m.refine_sens;
  ea.mu = o.mu;
  ea.sigma = o.sigma;
  ea.ei = o.ei;
  ea.p_feas = o.p_feas;
  ea.acq = o.acq;
  ea.refine_list = P.rlist;
  ea.refine_count = P.rcount;
  return ea;
}

RArgs make_rargs(const gp_model &m, const ScorePlan &P, int64_t rows, const ScoreOut &o) {
  RArgs ra{};
  ra.cand = P.cand;
  ra.ldc = rows;
  ra.obs = m.d_codes;
  ra.R = m.lay.R;
  ra.n_f = m.n_f;
  ra.cb = refine_candidates_per_block(m.n_f);
  ra.ldb = m.n_f;
  ra.B64 = m.d_B64;
  ra.alpha = m.d_alpha;
  ra.list = P.rlist;
  ra.count = P.rcount;
  ra.sv = m.sv;
  ra.fstar = m.fstar;
  ra.mask = o.mask;
  ra.eps_f = o.eps_f;
  ra.mu = o.mu;
  ra.sigma = o.sigma;
  ra.ei = o.ei;
  ra.acq = o.acq;
  ra.part = P.rpart;
  ra.mup = P.rmup;
  ra.part64 = P.rpart64;
  ra.mu64 = P.rmu64;
  ra.cap = P.rpart64 ? rows : 0;
  return ra;
}

// The value model's half of the scoring's tail: its epilogue (mu, sigma, EI of the
// candidates kept in fp32, the list of the others) and the fp64 recomputation's block
// path. fstar_dev: f* on the device, for a scoring that runs before the host knows it.
// Needs the value tiles' contraction done on s.
hipError_t score_value_tail(const gp_model &m, const ScorePlan &P, int64_t M, int64_t rows,
                            const ScoreOut &o, const double *fstar_dev, hipStream_t s,
                            hipEvent_t *ev) {
  EArgs ea = make_eargs(m, P, M, rows, o);
  ea.fstar_dev = fstar_dev;
  if (ev) HIPRET(hipEventRecord(ev[kProfValEpi], s));
  HIPRET(launch_epilogue_value(ea, s));
  if (ev) HIPRET(hipEventRecord(ev[kProfValEpi + 1], s));
  HIPRET(launch_refine_block(make_rargs(m, P, rows, o), m.lay.w64, stream_cus(s), s));
  if (ev) HIPRET(hipEventRecord(ev[kProfValEpi + 2], s));
  return hipSuccess;
}

// Second half: the variance contraction (and the classifier's latent mean) over the
// tiles from tile0 on (the ones before were contracted earlier), the value model's tail
// unless a fused scoring runs it on the value model's stream (value_done: its event), the
// classifier's epilogue (p, acq), the rest of the fp64 recomputation and the arg-max.
hipError_t score_back(const gp_model &m, const ScorePlan &P, int64_t M, int64_t rows,
                      const ScoreOut &o, int tile0, hipStream_t s, hipEvent_t *ev,
                      hipEvent_t value_done = nullptr) {
  if (ev && tile0 > 0) HIPRET(hipEventRecord(ev[kProfLate], s));
  HIPRET(contract_tiles(m, P, rows, tile0, m.ntiles, s));
  if (ev) HIPRET(hipEventRecord(ev[3], s));
  const EArgs ea = make_eargs(m, P, M, rows, o);
  float *pwork = o.p_feas ? o.p_feas : P.pwork;
  if (value_done) {
    HIPRET(hipStreamWaitEvent(s, value_done, 0));
    if (ev) HIPRET(hipEventRecord(ev[kProfClsEpi], s));
    HIPRET(launch_epilogue_cls(ea, pwork, s));
  } else {  // one stream: both epilogues in one pass, then the block recomputation
    if (ev) HIPRET(hipEventRecord(ev[kProfValEpi], s));
    HIPRET(launch_epilogue(ea, pwork, s));
    if (ev) HIPRET(hipEventRecord(ev[kProfValEpi + 1], s));
    HIPRET(launch_refine_block(make_rargs(m, P, rows, o), m.lay.w64, stream_cus(s), s));
    if (ev) HIPRET(hipEventRecord(ev[kProfValEpi + 2], s));
    if (ev) HIPRET(hipEventRecord(ev[kProfClsEpi], s));
  }
  if (ev) HIPRET(hipEventRecord(ev[4], s));
  const RArgs ra = make_rargs(m, P, rows, o);
  const int64_t rgrid = std::min<int64_t>((M + ra.cb - 1) / ra.cb, 1024);
  HIPRET(launch_refine_rest(ra, m.lay.w64, pwork, (int)rgrid, s));
  if (ev) HIPRET(hipEventRecord(ev[5], s));
  if (o.argmax) HIPRET(launch_argmax(o.acq, M, P.amax_v, P.amax_i, kArgmaxBlocks, o.argmax, s));
  if (ev) HIPRET(hipEventRecord(ev[6], s));
  return hipSuccess;
}

// Library-owned host resources: pinned host buffers (per host thread) and streams (per
// device), created on first use. gp_release frees all of them; a generation counter
// tells each thread that its buffers were released, so they are allocated again.
struct Owned {
  std::mutex mu;
  std::vector<void *> pinned;
  std::vector<hipStream_t> streams;
  std::vector<hipStream_t> side;                               // per device
  std::vector<std::pair<hipStream_t, hipStream_t>> split;      // per device
  uint64_t gen = 1;
} g_owned;

uint64_t owned_gen() {
  std::lock_guard<std::mutex> lk(g_owned.mu);
  return g_owned.gen;
}

hipError_t pinned_alloc(void **p, size_t bytes, unsigned flags) {
  hipError_t e = hipHostMalloc(p, bytes, flags);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lk(g_owned.mu);
  g_owned.pinned.push_back(*p);
  return hipSuccess;
}

void pinned_free(void *p) {
  if (!p) return;
  {
    std::lock_guard<std::mutex> lk(g_owned.mu);
    auto it = std::find(g_owned.pinned.begin(), g_owned.pinned.end(), p);
    if (it == g_owned.pinned.end()) return;  // already released
    g_owned.pinned.erase(it);
  }
  (void)hipHostFree(p);
}

// Pinned host memory per host thread for gp_fit (synchronous, so one call per thread
// uses it at a time), allocated on first use: the classifier's status ring (written by
// the device, coherent), the end-of-fit readback, and a staging area for the uploads,
// grown when a larger fit needs it.
constexpr int kStatusRing = 4;
struct FitReadback {
  int32_t info[4];
  double fstar;
  uint8_t valid[kMaxN];
  uint8_t feasible[kMaxN];
};
struct FitHost {
  NewtonStatus *ring = nullptr, *ring_dev = nullptr;  // host pointer, device pointer
  FitReadback *rb = nullptr;
  char *stage = nullptr;
  size_t stage_cap = 0;
  uint64_t gen = 0;
};
FitHost *fit_host(size_t stage_bytes) {
  thread_local FitHost h;
  const uint64_t g = owned_gen();
  if (h.gen != g) h = FitHost{nullptr, nullptr, nullptr, nullptr, 0, g};
  if (!h.ring) {
    void *p = nullptr;
    if (pinned_alloc(&p, sizeof(NewtonStatus) * kStatusRing, hipHostMallocCoherent) != hipSuccess)
      return nullptr;
    void *d = nullptr;
    if (hipHostGetDevicePointer(&d, p, 0) != hipSuccess) {
      pinned_free(p);
      return nullptr;
    }
    h.ring = static_cast<NewtonStatus *>(p);
    h.ring_dev = static_cast<NewtonStatus *>(d);
  }
  if (!h.rb) {
    void *p = nullptr;
    if (pinned_alloc(&p, sizeof(FitReadback), hipHostMallocDefault) != hipSuccess) return nullptr;
    h.rb = static_cast<FitReadback *>(p);
  }
  if (h.stage_cap < stage_bytes) {
    pinned_free(h.stage);
    h.stage = nullptr;
    h.stage_cap = 0;
    void *p = nullptr;
    const size_t cap = std::max<size_t>(stage_bytes, 64 * 1024);
    if (pinned_alloc(&p, cap, hipHostMallocDefault) != hipSuccess) return nullptr;
    h.stage = static_cast<char *>(p);
    h.stage_cap = cap;
  }
  return &h;
}

// A library-owned stream per device (default priority) for fit work that runs
// concurrently with the caller's stream; always joined back before gp_fit returns.
hipError_t side_stream(hipStream_t *out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lk(g_owned.mu);
  auto &streams = g_owned.side;
  if ((int)streams.size() <= dev) streams.resize(dev + 1, nullptr);
  if (!streams[dev]) {
    e = hipStreamCreateWithFlags(&streams[dev], hipStreamNonBlocking);
    if (e != hipSuccess) return e;
    g_owned.streams.push_back(streams[dev]);
  }
  *out = streams[dev];
  return hipSuccess;
}

// Two library-owned streams per device for a fit fused with scoring (default priority):
// the classifier's latency-bound Newton iterations get a quarter of the compute units,
// the value model and the first half of scoring the other three quarters, so neither
// queues behind the other's workgroups.
hipError_t split_streams(hipStream_t *cls, hipStream_t *val) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lk(g_owned.mu);
  auto &streams = g_owned.split;
  if ((int)streams.size() <= dev) streams.resize(dev + 1, {nullptr, nullptr});
  if (!streams[dev].first) {
    int ncu = 0;
    if ((e = hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess)
      return e;
    if (ncu < 2) return hipErrorInvalidDevice;
    const int split = std::max(1, ncu / 4);
    std::vector<uint32_t> a((ncu + 31) / 32, 0u), b(a.size(), 0u);
    for (int c = 0; c < ncu; ++c) (c < split ? a : b)[c / 32] |= 1u << (c % 32);
    hipStream_t sa = nullptr, sb = nullptr;
    if ((e = hipExtStreamCreateWithCUMask(&sa, (uint32_t)a.size(), a.data())) != hipSuccess) return e;
    if ((e = hipExtStreamCreateWithCUMask(&sb, (uint32_t)b.size(), b.data())) != hipSuccess) {
      (void)hipStreamDestroy(sa);
      return e;
    }
    streams[dev] = {sa, sb};
    g_owned.streams.push_back(sa);
    g_owned.streams.push_back(sb);
  }
  *cls = streams[dev].first;
  *val = streams[dev].second;
  return hipSuccess;
}

// Compute units a stream's work can occupy: the shares of the split streams, else all.
int stream_cus(hipStream_t s) {
  int dev = 0, ncu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      ncu < 1)
    return 1;
  std::lock_guard<std::mutex> lk(g_owned.mu);
  if (s && dev < (int)g_owned.split.size()) {
    const int split = std::max(1, ncu / 4);
    if (g_owned.split[dev].first == s) return split;
    if (g_owned.split[dev].second == s) return ncu - split;
  }
  return ncu;
}

// Scoring fused with a fit: the candidates, the gp_score outputs and the workspace
// region that the scoring buffers take.
struct ScoreJob {
  const void *const *C_cols;
  int64_t M;
  ScoreOut o;
  char *ws;
  size_t ws_bytes;
};

// The fit, and with `job` the scoring of its candidates by the fitted model.
gp_status fit_impl(const gp_space *space, const void *const *X_cols, int32_t n, const double *y,
                   const uint8_t *feasible, const gp_hyper *reg, const gp_hyper *cls,
                   void *workspace, size_t ws_bytes, hipStream_t s, const ScoreJob *job,
                   gp_model **out) {
  {
    if (!out) return fail(GP_E_INVALID, "out is NULL");
    *out = nullptr;
    if (!reg || !reg->lengthscale) return fail(GP_E_INVALID, "reg hyperparameters missing");
    if (!y) return fail(GP_E_INVALID, "y is NULL");
    if (n < 1 || n > kMaxN) return fail(GP_E_INVALID, "n must be in 1..4096");
    if (!(reg->signal_var > 0.0) || !std::isfinite(reg->signal_var))
      return fail(GP_E_INVALID, "signal_var must be finite and > 0");
    if (!(reg->noise_var >= 0.0) || !std::isfinite(reg->noise_var))
      return fail(GP_E_INVALID, "noise_var must be finite and >= 0");
    if (cls && (!(cls->signal_var > 0.0) || !std::isfinite(cls->signal_var)))
      return fail(GP_E_INVALID, "classifier signal_var must be finite and > 0");
    std::unique_ptr<gp_model> m(new gp_model());
    gp_status st = build_layout(space, reg->lengthscale, m->lay);
    if (st != GP_OK) return st;
    const Layout &L = m->lay;
    if (cls && cls->lengthscale)
      for (int p = 0; p < L.d; ++p)
        if (cls->lengthscale[p] != reg->lengthscale[p])
          return fail(GP_E_UNSUPPORTED, "the classifier shares the value model's lengthscales");
    if ((st = check_cols(X_cols, L.d)) != GP_OK) return st;
    if (job && (st = check_score_args(L, job->C_cols, job->M, job->o)) != GP_OK) return st;
    if (job && job->M > 0) {
      // the scoring region as it will be carved below, with this fit's code words
      Carver need;
      plan_score(need, L.R, (int)round_up(n, kKChunk), max_tiles(n, cls != nullptr), n, n,
                 round_up(job->M, kRowTile));
      if (need.off > job->ws_bytes)
        return fail(GP_E_WORKSPACE, "scoring workspace too small: need " + std::to_string(need.off) +
                                        " bytes, have " + std::to_string(job->ws_bytes));
    }
    m->variant = xkernel_variant(L.n_num, L.n_bits, L.n_eq, L.n_dot);
    if (m->variant < 0) return fail(GP_E_UNSUPPORTED, "no cross-kernel variant for this space");
    Carver meas;
    plan_fit(meas, L, n, cls != nullptr);
    if ((st = check_ws(workspace, ws_bytes, meas.off)) != GP_OK) return st;
    Carver cv;
    cv.base = static_cast<char *>(workspace);
    cv.size = ws_bytes;
    FitPlan P = plan_fit(cv, L, n, cls != nullptr);

    m->n = n;
    m->sv = reg->signal_var;
    m->nv = reg->noise_var;
    m->has_cls = cls != nullptr;
    m->csv = cls ? cls->signal_var : 0.0;
    m->lda = (int)round_up(n, kKChunk);
    m->d_penc = P.penc;
    m->d_table = P.table;
    m->d_tdesc = P.tdesc;
    m->d_codes = P.codes;
    m->d_xa = P.xa;
    m->d_xr = P.xr;
    // The layout tables, numeric scales and model order occupy consecutive workspace
    // regions: they go up in one copy from a pinned image of that span.
    char *dev0 = reinterpret_cast<char *>(P.penc);
    const size_t o_table = reinterpret_cast<char *>(P.table) - dev0;
    const size_t o_tdesc = reinterpret_cast<char *>(P.tdesc) - dev0;
    const size_t o_scale = reinterpret_cast<char *>(P.num_scale) - dev0;
    const size_t o_order = reinterpret_cast<char *>(P.order) - dev0;
    const size_t span = o_order + sizeof(int32_t) * n;
    FitHost *hb = fit_host(span);
    if (!hb) return fail(GP_E_HIP, "pinned host allocation failed");
    FitReadback *rb = hb->rb;

    // model order: feasible observations first (value model), then infeasible
    if (feasible) {
      HIPCHK(hipMemcpyAsync(rb->feasible, feasible, n, hipMemcpyDeviceToHost, s));
      HIPCHK(hipStreamSynchronize(s));
    } else {
      std::memset(rb->feasible, 1, n);
    }
    m->order.clear();
    for (int i = 0; i < n; ++i)
      if (rb->feasible[i]) m->order.push_back(i);
    m->n_f = (int)m->order.size();
    for (int i = 0; i < n; ++i)
      if (!rb->feasible[i]) m->order.push_back(i);
    const int nf = m->n_f;
    if (nf == 0) return fail(GP_E_INVALID, "no feasible observation: the value model needs at least one");
    char *img = hb->stage;
    std::memset(img, 0, span);
    std::memcpy(img, L.penc.data(), sizeof(ParamEnc) * L.penc.size());
    if (!L.table.empty()) std::memcpy(img + o_table, L.table.data(), sizeof(double) * L.table.size());
    std::memcpy(img + o_tdesc, L.tdesc.data(), sizeof(TermDesc) * L.tdesc.size());
    std::copy(L.num_scale.begin(), L.num_scale.end(), reinterpret_cast<double *>(img + o_scale));
    std::memcpy(img + o_order, m->order.data(), sizeof(int32_t) * n);
    HIPCHK(hipMemcpyAsync(dev0, img, span, hipMemcpyHostToDevice, s));
    HIPCHK(hipMemsetAsync(P.info, 0, 4 * sizeof(int32_t), s));  // infos and the Newton halt word

    // encode observations (AoS, model order); their validity flags are read back with
    // the end-of-fit status (an invalid observation is reported before any other failure)
    HIPCHK(encode_into(L, X_cols, P.penc, P.table, n, n, P.order, P.codes, 1, L.R, P.valid, nullptr,
                       nullptr, s));
    auto first_invalid = [&]() -> int {  // synchronises; -1 if every observation is valid
      if (hipMemcpyAsync(rb->valid, P.valid, n, hipMemcpyDeviceToHost, s) != hipSuccess ||
          hipStreamSynchronize(s) != hipSuccess)
        return -1;
      for (int i = 0; i < n; ++i)
        if (!rb->valid[i]) return i;
      return -1;
    };
    auto invalid_error = [&](int i) {
      return fail(GP_E_INVALID, "observation " + std::to_string(m->order[i]) +
                                    " is not a valid configuration of the space");
    };

    // The value model (stream sv) and the classifier (stream sc) are independent until
    // the classifier's columns join the value model's in the packed B^T: fork, then join.
    // Alone, the classifier runs on the caller's stream and the value model on a side
    // stream. With a scoring job, each gets a stream restricted to its own share of the
    // compute units, and the first half of scoring (candidate encoding and the
    // cross-kernel, which need the value model only) follows the value model on its
    // stream while the host still drives the classifier's Newton iterations.
    // (Without a classifier there is nothing to share the compute units with: the value
    // model and all of the scoring run on the unmasked side stream.)
    hipStream_t sc = s, sv = nullptr;
    if (job && cls) HIPCHK(split_streams(&sc, &sv));
    else HIPCHK(side_stream(&sv));
    // With a scoring job the classifier's tail and the second half of scoring run on the
    // library's non-blocking side stream, which the caller's stream joins at the end: the
    // split streams are blocking ones (a CU mask takes no stream flags), so work on a
    // caller's legacy default stream would wait for all of their earlier work.
    hipStream_t stail = s;
    if (job) HIPCHK(side_stream(&stail));
    constexpr int kEvs = 8 + kStatusRing;
    hipEvent_t evs[kEvs] = {};
    struct EvGuard {  // on an error exit: no enqueued work still uses the workspace
      hipEvent_t *e;
      hipStream_t q4[4];
      bool ok = false;
      ~EvGuard() {
        if (!ok)
          for (hipStream_t q : q4) (void)hipStreamSynchronize(q);
        for (int i = 0; i < kEvs; ++i)
          if (e[i]) (void)hipEventDestroy(e[i]);
      }
    } evg{evs, {sv, sc, s, stail}};
    for (auto &e : evs) HIPCHK(hipEventCreateWithFlags(&e, hipEventDisableTiming));
    hipEvent_t ev_fork = evs[0], ev_join = evs[1], ev_vcon = evs[2], ev_front = evs[3];
    hipEvent_t ev_done = evs[4], ev_rehome = evs[5], ev_vfit = evs[6], ev_vaux = evs[7];
    hipEvent_t *ev_it = evs + 8;
    HIPCHK(hipEventRecord(ev_fork, s));
    HIPCHK(hipStreamWaitEvent(sv, ev_fork, 0));
    if (sc != s) HIPCHK(hipStreamWaitEvent(sc, ev_fork, 0));

    // With a scoring job the candidates are encoded on the caller's stream (idle until
    // the join) while the value model is fitted; the buffers are planned for the largest
    // tile count and n_f the fit could give.
    ScorePlan SP{};
    int64_t rows = 0;
    hipEvent_t *pev = nullptr;  // stage profiling of the scoring
    const bool fused = job && job->M > 0;
    if (fused) {
      rows = round_up(job->M, kRowTile);
      Carver cs;
      cs.base = job->ws;
      cs.size = job->ws_bytes;
      SP = plan_score(cs, L.R, m->lda, max_tiles(n, cls != nullptr), n, n, rows);
      if (!cs.ok) return fail(GP_E_WORKSPACE, "scoring workspace too small");
      pev = prof_begin(true);
      if (pev) HIPCHK(hipEventRecord(pev[0], s));
      HIPCHK(score_encode(*m, SP, job->C_cols, job->M, rows, s));
      HIPCHK(hipEventRecord(ev_front, s));
      if (pev) HIPCHK(hipEventRecord(pev[kProfEncEnd], s));
    }

    int32_t info = 0;
    const double rho = cls ? m->csv / m->sv : 0.0;
    // Laplace probit classifier on all n observations (labels +1 feasible / -1 not),
    // Newton's method in the B = I + W^1/2 K W^1/2 form. The prediction uses W, grad and
    // chol(B) of the last Newton iterate, which differs from the returned mode by less
    // than the 1e-10 convergence tolerance. Iteration it+1 is already enqueued while the
    // host waits for the status of iteration it (it+2 follows once that status is read),
    // so the GPU does not wait on the host; once the device sets the halt word, the
    // iteration already enqueued does nothing, and the work that uses the classifier
    // waits for the converged iteration only (the caller's stream is ordered after the
    // idle one at the end of the fit, before a later call can clear the halt word).
    // Each factorisation carries the identity below B: its panels are Y = L^-T, with which
    // the step's two triangular solves are products, and the last one leaves L_B^-1 for
    // the prediction without a separate triangular inverse.
    constexpr double kNewtonTol = 1e-10;
    constexpr int kNewtonMax = 100;
    int32_t *halt = P.info + 2;
    NewtonStatus *hst = hb->ring;
    double *fbuf[2] = {P.f, P.fnew};
    auto enqueue_iteration = [&](int it) -> hipError_t {
      const double *f = fbuf[(it - 1) & 1];
      double *fn = fbuf[it & 1];
      hipError_t e;
      // probit terms, v = W^1/2 K b, [B ; I] and B's first diagonal block factored
      if ((e = launch_newton_setup(P.Kc, f, P.t, P.grad, P.W, P.sw, P.b, P.v, P.Bm, n, P.LB, P.Dc,
                                   P.info, halt, sc)) != hipSuccess)
        return e;
      // f_new = K a, a = b - W^1/2 L^-T L^-1 v, both solves as products with Y = L^-T
      // from the identity rows' panels: z = Y^T v, a = b - W^1/2 (Y z) (in place of b)
      if ((e = chol_factor(P.Bm, n, P.LB, n, P.Dc, n, P.info, sc, n, P.LE, n, halt, false, n,
                           true)) != hipSuccess)
        return e;
      if ((e = launch_gemv_cols(P.LE, n, P.v, P.z2, n, n, halt, sc)) != hipSuccess) return e;
      if ((e = launch_newton_a(P.LE, P.z2, P.b, P.sw, P.b, n, halt, sc)) != hipSuccess) return e;
      if ((e = launch_gemv_newton(P.Kc, P.b, fn, f, n, n, kNewtonTol, P.info, halt, P.nscr,
                                  hb->ring_dev + it % kStatusRing, sc)) != hipSuccess)
        return e;
      return hipEventRecord(ev_it[it % kStatusRing], sc);
    };
    // the classifier's Gram matrix, labels and cleared buffers, then its first iteration
    auto start_classifier = [&]() -> hipError_t {
      hipError_t e;
      if ((e = launch_gram(P.codes, L.R, n, L.w64, m->csv, 0.0, P.Kc, n, sc)) != hipSuccess) return e;
      if ((e = launch_labels(feasible, P.order, P.t, n, sc)) != hipSuccess) return e;
      if ((e = hipMemsetAsync(P.f, 0, sizeof(double) * n, sc)) != hipSuccess) return e;
      if ((e = hipMemsetAsync(P.nscr, 0, sizeof(NewtonScratch), sc)) != hipSuccess) return e;
      // L's upper triangle, and the identity rows' panels below their diagonal blocks,
      // are never written
      if ((e = hipMemsetAsync(P.LB, 0, sizeof(double) * (size_t)n * n, sc)) != hipSuccess) return e;
      if ((e = hipMemsetAsync(P.LE, 0, sizeof(double) * (size_t)n * n, sc)) != hipSuccess) return e;
      return enqueue_iteration(1);
    };
    bool cls_started = false;
    if (cls && !fused) {
      HIPCHK(start_classifier());
      cls_started = true;
    }
    // The host reads the Newton statuses in order and keeps two iterations ahead of the
    // last one read. Enqueueing the value model and the first half of scoring takes the
    // host longer than several iterations take the device, so it polls between those
    // launches (block = false) and only blocks once they are all enqueued.
    int it_read = 1, last_enqueued = cls ? 1 : 0;
    bool converged = !cls;
    auto newton_poll = [&](bool block) -> gp_status {
      while (!converged && cls_started) {
        if (last_enqueued < std::min(it_read + 1, kNewtonMax)) {
          HIPCHK(enqueue_iteration(last_enqueued + 1));
          ++last_enqueued;
          continue;
        }
        hipEvent_t e = ev_it[it_read % kStatusRing];
        if (block) {
          HIPCHK(hipEventSynchronize(e));
        } else {
          const hipError_t q = hipEventQuery(e);
          if (q == hipErrorNotReady) return GP_OK;
          HIPCHK(q);
        }
        const NewtonStatus h = hst[it_read % kStatusRing];
        if (h.halt == 3 || h.halt == 2) {
          const int bad = first_invalid();
          if (bad >= 0) return invalid_error(bad);
        }
        if (h.halt == 3)
          return fail(GP_E_NOT_SPD, "classifier matrix B not positive definite at pivot " +
                                        std::to_string(h.info - 1));
        if (h.halt == 2) return fail(GP_E_NOT_CONVERGED, "classifier Newton step not finite");
        if (h.halt == 1) {
          converged = true;
          break;
        }
        if (it_read == kNewtonMax) {
          const int bad = first_invalid();
          if (bad >= 0) return invalid_error(bad);
          return fail(GP_E_NOT_CONVERGED, "classifier Newton iteration did not converge in 100 steps");
        }
        ++it_read;
      }
      return GP_OK;
    };
#define NEWTON_POLL()                                  \
  do {                                                 \
    const gp_status st_ = newton_poll(false);          \
    if (st_ != GP_OK) return st_;                      \
  } while (0)

    // value model: K, L, B = L^-T, alpha, f*  (stream sv). The factorisation carries
    // identity rows below K, whose panels are L^-T (no separate triangular inverse);
    // L^-1 and K^-1 are formed only when exported.
    HIPCHK(launch_gather_f64(y, P.order, P.yf, nf, sv));
    HIPCHK(launch_gram(P.codes, L.R, nf, L.w64, m->sv, m->nv, P.K, nf, sv));
    HIPCHK(launch_copy_ident(P.K, nf, P.Aw, nf, sv));
    HIPCHK(hipMemsetAsync(P.B64, 0, sizeof(double) * (size_t)nf * nf, sv));  // L^-T's lower part
    HIPCHK(chol_factor(P.Aw, nf, P.L, nf, P.Dv, nf, P.info + 1, sv, nf, P.B64, nf, nullptr, true,
                       nf));
    NEWTON_POLL();
    HIPCHK(launch_gemv_t_upper(P.B64, nf, P.yf, P.beta, nf, sv));       // beta = L^-1 y
    HIPCHK(launch_gemv_rows(P.B64, nf, P.beta, P.alpha, nf, 0, sv));   // alpha = L^-T beta
    // With a scoring job f*, the value columns' packed B^T and the status readback are
    // made on the tail's stream (idle until the classifier converges), off the value
    // model's path to the cross-kernel; the value tiles' contraction waits for them.
    hipStream_t sx = fused ? stail : sv;
    if (sx != sv) {
      HIPCHK(hipEventRecord(ev_vfit, sv));
      HIPCHK(hipStreamWaitEvent(sx, ev_vfit, 0));
    }
    HIPCHK(launch_reduce_min(P.yf, nf, P.fstar, sx));
    m->d_K = P.K;
    m->d_L = P.L;
    m->d_Linv = P.Linv;
    m->d_B64 = P.B64;
    m->d_Kinv = P.Kinv;
    m->d_alpha = P.alpha;

    // packed B^T for the fp32 contraction, column tiles of 128
    const int nreg_pad = (int)round_up(nf, kColTile);
    const int ncls_pad = cls ? (int)round_up(n, kColTile) : 0;
    m->d_Bt = P.Bt;
    m->d_cscale = P.cscale;
    // k* <= s, so the scaled K* lies below 2^(kSplitTop+1); the clamp keeps 2^kexp a
    // normal fp32 number for any signal variance
    m->kexp = std::min(std::max(kSplitTop - std::ilogb(m->sv), -100), 100);
    HIPCHK(launch_pack_bt(P.B64, nf, nf, true, nullptr, 1.0, m->kexp, P.Bt, P.cscale, m->lda,
                          nreg_pad, sx));
    // observation x-records for the cross-kernel variant
    XObsLayout &xl = m->xl;
    xl = xobs_layout(m->variant, L.n_num, L.n_bits, L.n_eq, L.n_dot, L.w_bits0, L.w_eq0, L.w_dot0);
    if (xobs_a_doubles(n, xl.ks) > xobs_a_doubles_max(n) || xobs_r_words(n, xl.rw) > xobs_r_words_max(n))
      return fail(GP_E_INVALID, "internal error: cross-kernel observation arrays exceed their bound");
    HIPCHK(launch_make_xobs(P.codes, L.R, n, xl, P.num_scale, P.alpha, nf, P.xa, P.xr, sv));
    NEWTON_POLL();

    XArgs &xa = m->xa;
    xa = XArgs{};
    xa.xa64 = P.xa;
    xa.xr = P.xr;
    xa.n = n;
    xa.lda = m->lda;
    xa.n_num = L.n_num; xa.n_bits = L.n_bits; xa.n_eq = L.n_eq; xa.n_dot = L.n_dot;
    xa.w_bits0 = L.w_bits0; xa.w_eq0 = L.w_eq0; xa.w_dot0 = L.w_dot0;
    for (int q = 0; q < L.n_num; ++q) xa.num_scale64[q] = L.num_scale[q];
    for (int q = 0; q < L.n_bits; ++q) xa.bits_w[q] = L.bits_w[q];
    for (int q = 0; q < L.n_eq; ++q) xa.eq_w[q] = L.eq_w[q];
    for (int q = 0; q < L.n_dot; ++q) {
      xa.dot_w2[q] = L.dot_w2[q];
      xa.dot_s2[q] = L.dot_s2[q];
    }
    // Matern-5/2 polynomial coefficients times 2^kexp: an exact rescaling of every
    // kernel value, so K* leaves the cross-kernel already scaled for its fp16 split
    xa.A0 = (float)std::ldexp(m->sv, m->kexp);
    xa.A1 = (float)std::ldexp(m->sv * std::sqrt(5.0), m->kexp);
    xa.A2 = (float)std::ldexp(m->sv * 5.0 / 3.0, m->kexp);
    xa.kinv = std::ldexp(1.0f, -m->kexp);

    // the value model's status for the end-of-fit checks: validity of the observations
    // (encoded before the fork), its factorisation info, f*
    if (sx != sv) HIPCHK(hipEventRecord(ev_vaux, sx));
    HIPCHK(hipMemcpyAsync(rb->valid, P.valid, n, hipMemcpyDeviceToHost, sx));
    HIPCHK(hipMemcpyAsync(rb->info + 1, P.info + 1, sizeof(int32_t), hipMemcpyDeviceToHost, sx));
    HIPCHK(hipMemcpyAsync(&rb->fstar, P.fstar, sizeof(double), hipMemcpyDeviceToHost, sx));
    HIPCHK(hipEventRecord(ev_join, sx));
    m->ntiles = 0;
    for (int c0 = 0; c0 < nf; c0 += kColTile)
      m->tiles[m->ntiles++] = CTile{c0, (int)round_up(std::min(c0 + kColTile, nf), kKChunk),
                                    (int16_t)c0, (int16_t)std::min(kColTile, nf - c0), -1};
    m->n_reg_tiles = m->ntiles;
    if (fused) {
      // the cross-kernel and the value model's column tiles of the contraction behind
      // the value model (and the encoding)
      m->fstar = 0.0;  // not read by the first half
      HIPCHK(hipStreamWaitEvent(sv, ev_front, 0));
      if (pev) HIPCHK(hipEventRecord(pev[1], sv));
      HIPCHK(score_xkernel(*m, SP, rows, sv));
      // The classifier's first iteration is enqueued once the value model and the
      // cross-kernel are: the host's launches (about twenty per Newton iteration) would
      // otherwise hold back the value model's chain, the longer one. (A fit alone starts
      // the classifier first.)
      if (cls) {
        HIPCHK(start_classifier());
        cls_started = true;
      }
      NEWTON_POLL();
      if (pev) HIPCHK(hipEventRecord(pev[2], sv));
      if (sx != sv) HIPCHK(hipStreamWaitEvent(sv, ev_vaux, 0));  // packed B^T and f*
      if (pev) HIPCHK(hipEventRecord(pev[kProfEarly], sv));
      HIPCHK(contract_tiles(*m, SP, rows, 0, m->n_reg_tiles, sv));
      if (pev) HIPCHK(hipEventRecord(pev[kProfEarly + 1], sv));
      HIPCHK(hipEventRecord(ev_vcon, sv));
      HIPCHK(score_value_tail(*m, SP, job->M, rows, job->o, P.fstar, sv, pev));
      HIPCHK(hipEventRecord(ev_front, sv));
    }

#undef NEWTON_POLL
    int rehome_lin = 0;  // > 0: the classifier's dense column moves to this value-tile column
    if (cls) {
      {
        const gp_status st = newton_poll(true);
        if (st != GP_OK) return st;
      }
      const int it = it_read;
      m->cls_iters = it;
      // the classifier's results are those of iteration it; the one enqueued after it
      // still sits on sc and changes nothing
      HIPCHK(hipStreamWaitEvent(stail, ev_it[it % kStatusRing], 0));
      // L_B^-1 = (the identity rows' panels of the last factorisation)^T
      HIPCHK(launch_pack_bt(P.LE, n, n, true, P.sw, rho, m->kexp,
                            P.Bt + (int64_t)nreg_pad * 2 * m->lda,
                            P.cscale + nreg_pad, m->lda, ncls_pad, stail));
      for (int c0 = 0; c0 < n; c0 += kColTile)
        m->tiles[m->ntiles++] =
            CTile{nreg_pad + c0, (int)round_up(std::min(c0 + kColTile, n), kKChunk), (int16_t)c0,
                  (int16_t)std::min(kColTile, n - c0), -1};
      m->d_cf = fbuf[it & 1];
      m->d_cgrad = P.grad;
      m->d_csw = P.sw;
      m->d_cL = P.LB;
    }
    if (cls) {
      HIPCHK(hipStreamWaitEvent(stail, ev_join, 0));
      // The classifier's latent mean at a candidate is k_c*^T grad = K* (rho grad): a dense
      // column of B, placed in a spare 16-column sub-tile of the last value tile (not when
      // the value tiles are contracted ahead of the classifier), else of the last
      // classifier tile, else in a tile of its own. (After the join: the value columns'
      // packing wrote zeros over the spare columns.)
      const int rlast = nf % kColTile, clast = n % kColTile;
      int t = -1, lin = 0, ncols = 1;
      if (!fused && rlast > 0 && round_up(rlast, 16) < kColTile) {
        t = m->n_reg_tiles - 1;
        lin = (int)round_up(rlast, 16);
      } else if (clast > 0 && round_up(clast, 16) < kColTile) {
        t = m->ntiles - 1;
        lin = (int)round_up(clast, 16);
      } else {
        t = m->ntiles++;
        m->tiles[t] = CTile{nreg_pad + ncls_pad, 0, 0, 0, 0};
        ncols = kColTile;  // the dense column, then zero columns
      }
      m->tiles[t].lin = lin;
      m->tiles[t].kend = (int)round_up(n, kKChunk);
      const int64_t c = m->tiles[t].bcol + lin;
      HIPCHK(launch_pack_vec(P.grad, n, rho, m->kexp, P.Bt + c * 2 * m->lda, P.cscale + c, m->lda,
                             ncols, stail));
      // For later scoring calls with this model the dense column moves into the last value
      // tile's spare sub-tile, where an unfused fit puts it (one full-length tile less per
      // call): packed on the value model's stream after its tail, the tile list changed
      // once this step's tiles are enqueued.
      if (fused && ncols == kColTile && rlast > 0 && round_up(rlast, 16) < kColTile) {
        rehome_lin = (int)round_up(rlast, 16);
        const int64_t cv = m->tiles[m->n_reg_tiles - 1].bcol + rehome_lin;
        HIPCHK(hipStreamWaitEvent(sv, ev_it[m->cls_iters % kStatusRing], 0));
        HIPCHK(launch_pack_vec(P.grad, n, rho, m->kexp, P.Bt + cv * 2 * m->lda, P.cscale + cv,
                               m->lda, 1, sv));
        HIPCHK(hipEventRecord(ev_rehome, sv));
      }
    }
    HIPCHK(hipStreamWaitEvent(stail, ev_join, 0));
    // the classifier's contraction follows the value tiles' (it needs K* only, but would
    // only compete with them for the compute units); its epilogue waits for the value
    // model's tail
    if (fused) HIPCHK(hipStreamWaitEvent(stail, ev_vcon, 0));

    // end-of-fit checks (the value model has long finished by the time the classifier has)
    HIPCHK(hipEventSynchronize(ev_join));
    HIPCHK(hipGetLastError());
    for (int i = 0; i < n; ++i)
      if (!rb->valid[i]) return invalid_error(i);
    info = rb->info[1];
    if (info)
      return fail(GP_E_NOT_SPD, "Gram matrix not positive definite: pivot " + std::to_string(info - 1) +
                                    " (model row; increase noise_var)");
    m->fstar = rb->fstar;
    if (fused)
      HIPCHK(score_back(*m, SP, job->M, rows, job->o, m->n_reg_tiles, stail, pev, ev_front));
    if (cls && sc != stail) HIPCHK(hipStreamWaitEvent(stail, ev_it[last_enqueued % kStatusRing], 0));
    if (rehome_lin > 0) {
      HIPCHK(hipStreamWaitEvent(stail, ev_rehome, 0));
      CTile &tv = m->tiles[m->n_reg_tiles - 1];
      tv.lin = rehome_lin;
      tv.kend = (int)round_up(n, kKChunk);
      --m->ntiles;  // the dense column's own tile, the last one
    }
    if (stail != s) {
      HIPCHK(hipEventRecord(ev_done, stail));
      HIPCHK(hipStreamWaitEvent(s, ev_done, 0));
    }
    if (!job) HIPCHK(hipStreamSynchronize(s));  // gp_fit returns with its work done
    evg.ok = true;
    *out = m.release();
    g_err.clear();
    return GP_OK;
  }
}

}  // namespace

// =================================================================== C-ABI
extern "C" {

const char *gp_last_error(void) { return g_err.c_str(); }

int32_t gp_version(void) { return 100; }

size_t gp_fit_workspace_bytes(const gp_space *space, int32_t n, int32_t with_classifier) {
  Layout L;
  if (build_layout(space, nullptr, L) != GP_OK || n < 1 || n > kMaxN) return 0;
  Carver cv;
  plan_fit(cv, L, n, with_classifier != 0);
  return cv.off;
}

gp_status gp_fit(const gp_space *space, const void *const *X_cols, int32_t n, const double *y,
                 const uint8_t *feasible, const gp_hyper *reg, const gp_hyper *cls,
                 void *workspace, size_t ws_bytes, void *stream, gp_model **out) {
  try {
    return fit_impl(space, X_cols, n, y, feasible, reg, cls, workspace, ws_bytes,
                    static_cast<hipStream_t>(stream), nullptr, out);
  } catch (const std::exception &e) {
    return fail(GP_E_INVALID, std::string("internal error: ") + e.what());
  }
}

namespace {
// Fit region of a fused workspace (rounded so that the scoring region stays aligned),
// and the scoring region's bound; 0 if the space, n or M is rejected.
size_t fused_fit_bytes(const Layout &L, int32_t n, bool cls) {
  Carver cv;
  plan_fit(cv, L, n, cls);
  return (size_t)round_up((int64_t)cv.off, 256);
}
// The bound holds for any lengthscales: the code words per candidate are counted with
// every categorical in a word of its own (R_bound), as categoricals share a word only
// when their weights, i.e. their lengthscales, are equal.
size_t fused_score_bytes(const Layout &L, int32_t n, bool cls, int64_t M) {
  Carver cv;
  plan_score(cv, L.R_bound, (int)round_up(n, kKChunk), max_tiles(n, cls), n, n,
             round_up(std::max<int64_t>(M, 1), kRowTile));
  return cv.off;
}
}  // namespace

size_t gp_fit_score_workspace_bytes(const gp_space *space, int32_t n, int32_t with_classifier,
                                    int64_t M) {
  Layout L;
  if (build_layout(space, nullptr, L) != GP_OK || n < 1 || n > kMaxN || M < 0 || M > INT32_MAX)
    return 0;
  return fused_fit_bytes(L, n, with_classifier != 0) +
         fused_score_bytes(L, n, with_classifier != 0, M);
}

gp_status gp_fit_score(const gp_space *space, const void *const *X_cols, int32_t n,
                       const double *y, const uint8_t *feasible, const gp_hyper *reg,
                       const gp_hyper *cls, const void *const *C_cols, int64_t M,
                       const uint8_t *mask, float eps_f, float *mu, float *sigma, float *ei,
                       float *p_feas, float *acq, int64_t *argmax, void *workspace,
                       size_t ws_bytes, void *stream, gp_model **out) {
  try {
    if (!out) return fail(GP_E_INVALID, "out is NULL");
    *out = nullptr;
    if (M < 0 || M > INT32_MAX) return fail(GP_E_INVALID, "M must be in 0..2^31-1");
    if (n < 1 || n > kMaxN) return fail(GP_E_INVALID, "n must be in 1..4096");
    Layout L;
    gp_status st = build_layout(space, nullptr, L);
    if (st != GP_OK) return st;
    const size_t fit_bytes = fused_fit_bytes(L, n, cls != nullptr);
    if ((st = check_ws(workspace, ws_bytes,
                       fit_bytes + fused_score_bytes(L, n, cls != nullptr, M))) != GP_OK)
      return st;
    ScoreJob job{C_cols, M, ScoreOut{mask, eps_f, mu, sigma, ei, p_feas, acq, argmax},
                 static_cast<char *>(workspace) + fit_bytes, ws_bytes - fit_bytes};
    return fit_impl(space, X_cols, n, y, feasible, reg, cls, workspace, fit_bytes,
                    static_cast<hipStream_t>(stream), &job, out);
  } catch (const std::exception &e) {
    return fail(GP_E_INVALID, std::string("internal error: ") + e.what());
  }
}

gp_status gp_model_info(const gp_model *m, gp_model_info_t *info) {
  if (!m || !info) return fail(GP_E_INVALID, "NULL argument");
  info->n = m->n;
  info->n_feasible = m->n_f;
  info->d = m->lay.d;
  info->has_classifier = m->has_cls ? 1 : 0;
  info->cls_iterations = m->cls_iters;
  info->code_words = m->lay.R;
  info->fstar = m->fstar;
  info->signal_var = m->sv;
  info->noise_var = m->nv;
  info->cls_signal_var = m->csv;
  return GP_OK;
}

gp_status gp_model_export(const gp_model *m, int32_t field, double *dst, size_t count) {
  if (!m || !dst) return fail(GP_E_INVALID, "NULL argument");
  const size_t nf = (size_t)m->n_f, n = (size_t)m->n;
  const double *src = nullptr;
  size_t want = 0;
  switch (field) {
    case GP_FIELD_K: src = m->d_K; want = nf * nf; break;
    case GP_FIELD_L: src = m->d_L; want = nf * nf; break;
    case GP_FIELD_LINV: src = m->d_Linv; want = nf * nf; break;
    case GP_FIELD_KINV: src = m->d_Kinv; want = nf * nf; break;
    case GP_FIELD_ALPHA: src = m->d_alpha; want = nf; break;
    case GP_FIELD_FEASIBLE_INDEX: want = n; break;
    case GP_FIELD_CLS_F: src = m->d_cf; want = n; break;
    case GP_FIELD_CLS_GRAD: src = m->d_cgrad; want = n; break;
    case GP_FIELD_CLS_SQRTW: src = m->d_csw; want = n; break;
    case GP_FIELD_CLS_L: src = m->d_cL; want = n * n; break;
    default: return fail(GP_E_INVALID, "unknown field");
  }
  if (count != want) return fail(GP_E_INVALID, "count must be " + std::to_string(want));
  if (field == GP_FIELD_FEASIBLE_INDEX) {
    for (size_t i = 0; i < n; ++i) dst[i] = (double)m->order[i];
    return GP_OK;
  }
  if (!src) return fail(GP_E_INVALID, "the model has no classifier");
  if ((field == GP_FIELD_LINV || field == GP_FIELD_KINV) && !m->inv_ready) {
    // L^-1 = (L^-T)^T and K^-1 = L^-T L^-1, formed on first use (synchronous, as the copy)
    HIPCHK(launch_transpose(m->d_B64, m->d_Linv, (int32_t)nf, (int32_t)nf, nullptr));
    HIPCHK(launch_ata_lower(m->d_Linv, (int32_t)nf, m->d_Kinv, (int32_t)nf, nullptr));
    HIPCHK(hipStreamSynchronize(nullptr));
    m->inv_ready = true;
  }
  HIPCHK(hipMemcpy(dst, src, sizeof(double) * want, hipMemcpyDeviceToHost));
  if (field == GP_FIELD_CLS_L)
    for (size_t r = 0; r < n; ++r)
      for (size_t c = r + 1; c < n; ++c) dst[r * n + c] = 0.0;
  return GP_OK;
}

void gp_model_free(gp_model *m) { delete m; }

size_t gp_score_workspace_bytes(const gp_model *m, int64_t M) {
  if (!m || M < 0 || M > INT32_MAX) return 0;
  Carver cv;
  plan_score(cv, *m, round_up(std::max<int64_t>(M, 1), kRowTile));
  return cv.off;
}

gp_status gp_score(const gp_model *m, const void *const *C_cols, int64_t M, const uint8_t *mask,
                   float eps_f, float *mu, float *sigma, float *ei, float *p_feas, float *acq,
                   int64_t *argmax, void *workspace, size_t ws_bytes, void *stream) {
  try {
    if (!m) return fail(GP_E_INVALID, "model is NULL");
    const ScoreOut o{mask, eps_f, mu, sigma, ei, p_feas, acq, argmax};
    gp_status st = check_score_args(m->lay, C_cols, M, o);
    if (st != GP_OK || M == 0) return st;
    const int64_t rows = round_up(M, kRowTile);
    Carver meas;
    plan_score(meas, *m, rows);
    if ((st = check_ws(workspace, ws_bytes, meas.off)) != GP_OK) return st;
    Carver cv;
    cv.base = static_cast<char *>(workspace);
    cv.size = ws_bytes;
    const ScorePlan P = plan_score(cv, *m, rows);
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipEvent_t *ev = prof_begin();
    HIPCHK(score_front(*m, P, C_cols, M, rows, s, ev));
    HIPCHK(score_back(*m, P, M, rows, o, 0, s, ev));
    return GP_OK;
  } catch (const std::exception &e) {
    return fail(GP_E_INVALID, std::string("internal error: ") + e.what());
  }
}

// ------------------------------------------------------------------ scoring without allocation
// The scoring buffers of gp_score_noalloc live in one fixed device array per GPU (the
// library's only static device memory). Its address is taken once per device with that
// device current; host code uses only that address, never the array's name.
static __device__ __align__(256) unsigned char scratch[GP_NOALLOC_SCRATCH_BYTES];

namespace {
gp_status scratch_ptr(void **out) {
  static std::mutex mu;
  static std::vector<void *> ptrs;  // per device
  int dev = 0;
  HIPCHK(hipGetDevice(&dev));
  std::lock_guard<std::mutex> lk(mu);
  if ((int)ptrs.size() <= dev) ptrs.resize(dev + 1, nullptr);
  if (!ptrs[dev]) {
    void *p = nullptr;
    HIPCHK(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(GP_E_HIP, "hipGetSymbolAddress returned no address for the scratch array");
    ptrs[dev] = p;
  }
  *out = ptrs[dev];
  return GP_OK;
}
}  // namespace

size_t gp_score_noalloc_max_candidates(const gp_model *m) {
  if (!m) return 0;
  int64_t lo = 0, hi = INT32_MAX;  // largest M whose buffers fit the array
  while (lo < hi) {
    const int64_t mid = lo + (hi - lo + 1) / 2;
    Carver cv;
    plan_score(cv, *m, round_up(mid, kRowTile));
    if (cv.off <= (size_t)GP_NOALLOC_SCRATCH_BYTES) lo = mid;
    else hi = mid - 1;
  }
  return (size_t)lo;
}

gp_status gp_score_noalloc(const gp_model *m, const void *const *C_cols, int64_t M,
                           const uint8_t *mask, float eps_f, float *mu, float *sigma, float *ei,
                           float *p_feas, float *acq, int64_t *argmax, void *stream) {
  try {
    if (!m) return fail(GP_E_INVALID, "model is NULL");
    const ScoreOut o{mask, eps_f, mu, sigma, ei, p_feas, acq, argmax};
    gp_status st = check_score_args(m->lay, C_cols, M, o);
    if (st != GP_OK || M == 0) return st;
    const int64_t rows = round_up(M, kRowTile);
    Carver meas;
    plan_score(meas, *m, rows);
    if (meas.off > (size_t)GP_NOALLOC_SCRATCH_BYTES)
      return fail(GP_E_WORKSPACE, "gp_score_noalloc: " + std::to_string(M) + " candidates need " +
                                      std::to_string(meas.off) + " bytes of scratch, the fixed array holds " +
                                      std::to_string((size_t)GP_NOALLOC_SCRATCH_BYTES) +
                                      " (at most " + std::to_string(gp_score_noalloc_max_candidates(m)) +
                                      " candidates for this model)");
    void *base = nullptr;
    if ((st = scratch_ptr(&base)) != GP_OK) return st;
    Carver cv;
    cv.base = static_cast<char *>(base);
    cv.size = GP_NOALLOC_SCRATCH_BYTES;
    const ScorePlan P = plan_score(cv, *m, rows);
    if (!cv.ok) return fail(GP_E_WORKSPACE, "scratch array too small");
    hipStream_t s = static_cast<hipStream_t>(stream);
    // the same kernels as gp_score; every buffer that must start at zero (the count of
    // candidates for the fp64 recomputation) is cleared by the encoding kernel
    HIPCHK(score_front(*m, P, C_cols, M, rows, s, nullptr));
    HIPCHK(score_back(*m, P, M, rows, o, 0, s, nullptr));
    return GP_OK;
  } catch (const std::exception &e) {
    return fail(GP_E_INVALID, std::string("internal error: ") + e.what());
  }
}

// ------------------------------------------------------------------ local search
namespace {
// Space-order description of the neighbourhood, from the model's encode layout.
LSDesc ls_desc(const Layout &L) {
  LSDesc d{};
  d.d = L.d;
  for (size_t q = 0; q < L.penc.size(); ++q) {
    const ParamEnc &e = L.penc[q];
    const int p = e.col;
    d.penc_of[p] = (uint8_t)q;
    d.kind[p] = e.kind;
    d.log2[p] = (e.kind == GP_REAL && (e.flags & 1)) ? 1 : 0;
    switch (e.kind) {
      case GP_REAL:
        d.words[p] = 2;
        d.t_lo[p] = d.log2[p] ? std::log2(e.lo) : e.lo;
        d.t_hi[p] = d.log2[p] ? std::log2(e.hi) : e.hi;
        break;
      case GP_INT:
        d.words[p] = 1;
        d.lo[p] = (int32_t)e.lo;
        d.hi[p] = (int32_t)e.hi;
        break;
      case GP_ORD:
        d.words[p] = 1;
        d.lo[p] = 0;
        d.hi[p] = e.levels - 1;
        break;
      case GP_CAT:
        d.words[p] = 1;
        break;
      default:
        d.words[p] = e.levels;  // PERM: m
        break;
    }
  }
  for (int p = 0; p < L.d; ++p) {
    d.woff[p] = (uint16_t)d.W;
    for (int q = 0; q < d.words[p]; ++q) d.wparam[d.W + q] = (uint8_t)p;
    d.W += d.words[p];
  }
  int nnb = 0;
  for (int p = 0; p < L.d; ++p) {
    d.move0[p] = nnb;
    if (d.kind[p] == GP_CAT) {
      int lv = 0;
      for (const ParamEnc &e : L.penc)
        if (e.col == p) lv = e.levels;
      nnb += lv - 1;
    } else if (d.kind[p] == GP_PERM) {
      nnb += d.words[p] * (d.words[p] - 1) / 2;
    } else {
      nnb += 2;
    }
  }
  d.nnb = nnb;
  return d;
}

constexpr int kLsTopkParts = 256;
constexpr int kLsStepsPerCheck = 4;  // steps enqueued between host checks
// Start selection with a bound (from this many candidates on): kLsPruneTop candidates of
// largest bound are scored first, and only the candidates whose bound reaches the
// n_starts-th best of those are scored in full, when they are at most M / kLsPruneDiv.
constexpr int64_t kLsPruneMin = 65536;
constexpr int kLsPruneTop = kLsMaxStarts;
constexpr int64_t kLsPruneDiv = 4;

struct LSPlan {
  char *score_ws; size_t score_bytes;
  float *mu, *sigma, *ei, *acq;
  float *pv, *sv; int64_t *pi, *si;
  LSCols cur;
  uint8_t *mask;
  float *cur_acq; int32_t *active, *steps;
  // bounded start selection (M >= kLsPruneMin): candidate list, gathered configurations
  // and mask entries (cap rows), the counter, the kLsPruneTop first candidates
  int64_t cap;
  int64_t *list;
  LSCols G;
  uint8_t *mg;
  int32_t *count;
  float *tv, *tacq; int64_t *ti;
  float *kv; int64_t *ki;
};

LSPlan plan_ls(Carver &cv, const gp_model &m, const LSDesc &d, int64_t M, int k) {
  LSPlan P{};
  const int64_t N = (int64_t)k * d.nnb, rows = std::max<int64_t>(M, N);
  // the scoring workspace serves both the M candidates and the N neighbours
  Carver sa, sb;
  plan_score(sa, m, round_up(std::max<int64_t>(M, 1), kRowTile));
  plan_score(sb, m, round_up(std::max<int64_t>(N, 1), kRowTile));
  P.score_bytes = std::max(sa.off, sb.off);
  P.score_ws = cv.take<char>((int64_t)P.score_bytes);
  P.mu = cv.take<float>(rows);
  P.sigma = cv.take<float>(rows);
  P.ei = cv.take<float>(rows);
  P.acq = cv.take<float>(rows);
  const bool prune = M >= kLsPruneMin;
  const int kp = prune ? kLsPruneTop : k;  // widest top-k taken
  P.pv = cv.take<float>((int64_t)kLsTopkParts * kp);
  P.pi = cv.take<int64_t>((int64_t)kLsTopkParts * kp);
  P.sv = cv.take<float>(k);
  P.si = cv.take<int64_t>(k);
  for (int p = 0; p < d.d; ++p) {
    P.cur.col[p] = cv.take<uint32_t>((int64_t)k * d.words[p]);
  }
  P.mask = cv.take<uint8_t>(N);
  P.cur_acq = cv.take<float>(k);
  P.active = cv.take<int32_t>(k);
  P.steps = cv.take<int32_t>(k);
  if (prune) {
    P.cap = M / kLsPruneDiv;
    P.list = cv.take<int64_t>(P.cap);
    for (int p = 0; p < d.d; ++p) P.G.col[p] = cv.take<uint32_t>(P.cap * d.words[p]);
    P.mg = cv.take<uint8_t>(P.cap);
    P.count = cv.take<int32_t>(1);
    P.tv = cv.take<float>(kLsPruneTop);
    P.ti = cv.take<int64_t>(kLsPruneTop);
    P.tacq = cv.take<float>(kLsPruneTop);
    P.kv = cv.take<float>(k);
    P.ki = cv.take<int64_t>(k);
  }
  return P;
}

// pinned, per host thread (the calls are synchronous): two slots of kLsMaxStarts flags
int32_t *ls_active_host() {
  thread_local int32_t *buf = nullptr;
  thread_local uint64_t gen = 0;
  const uint64_t g = owned_gen();
  if (gen != g) {
    buf = nullptr;
    gen = g;
  }
  if (!buf) {
    void *p = nullptr;
    if (pinned_alloc(&p, sizeof(int32_t) * 2 * kLsMaxStarts, hipHostMallocDefault) != hipSuccess)
      return nullptr;
    buf = static_cast<int32_t *>(p);
  }
  return buf;
}
}  // namespace

size_t gp_local_search_workspace_bytes(const gp_model *m, int64_t M, int32_t n_starts) {
  if (!m || M < 1 || M > INT32_MAX || n_starts < 1 || n_starts > kLsMaxStarts) return 0;
  const int k = (int)std::min<int64_t>(n_starts, M);
  const LSDesc d = ls_desc(m->lay);
  Carver cv;
  plan_ls(cv, *m, d, M, k);
  return cv.off;
}

gp_status gp_local_search(const gp_model *m, const void *const *C_cols, int64_t M,
                          const uint8_t *mask, float eps_f, int32_t n_starts, int32_t max_steps,
                          void *const *out_cols, float *out_acq, int32_t *out_steps,
                          int64_t *out_start, void *workspace, size_t ws_bytes, void *stream) {
  try {
    if (!m) return fail(GP_E_INVALID, "model is NULL");
    if (M < 1 || M > INT32_MAX) return fail(GP_E_INVALID, "M must be in 1..2^31-1");
    if (n_starts < 1 || n_starts > kLsMaxStarts) return fail(GP_E_INVALID, "n_starts must be in 1..64");
    if (max_steps < 0) return fail(GP_E_INVALID, "max_steps must be >= 0");
    if (!out_cols || !out_acq || !out_steps || !out_start)
      return fail(GP_E_INVALID, "outputs are required");
    gp_status st = check_cols(C_cols, m->lay.d);
    if (st != GP_OK) return st;
    if ((st = check_cols(const_cast<const void *const *>(out_cols), m->lay.d)) != GP_OK) return st;
    const int k = (int)std::min<int64_t>(n_starts, M);
    const LSDesc d = ls_desc(m->lay);
    Carver meas;
    plan_ls(meas, *m, d, M, k);
    if ((st = check_ws(workspace, ws_bytes, meas.off)) != GP_OK) return st;
    Carver cv;
    cv.base = static_cast<char *>(workspace);
    cv.size = ws_bytes;
    const LSPlan P = plan_ls(cv, *m, d, M, k);
    hipStream_t s = static_cast<hipStream_t>(stream);
    int32_t *hact = ls_active_host();
    if (!hact) return fail(GP_E_HIP, "pinned host allocation failed");

    // score the candidates, pick the starts
    LSCols C{};
    for (int p = 0; p < d.d; ++p) C.col[p] = (uint32_t *)const_cast<void *>(C_cols[p]);
    bool picked = false;
    if (P.list && xkernel_splits(round_up(M, kRowTile), m->xa.n) == 1) {
      // Bounded selection: the cross-kernel's mean bounds every candidate's acquisition
      // value (launch_ls_bound); the kLsPruneTop candidates of largest bound are scored,
      // and the n_starts-th best of them, tau, is at most the n_starts-th best value of
      // all. A candidate whose bound is below tau cannot be among the n_starts best, so
      // only the others are scored, and their best (lower index first on ties) are those
      // of all. When more than M / kLsPruneDiv remain, everything is scored.
      auto score_rows = [&](const LSCols &G, const uint8_t *gm, int64_t cnt, float *acq_out) {
        const int64_t rows = round_up(cnt, kRowTile);
        Carver c2;
        c2.base = P.score_ws;
        c2.size = P.score_bytes;
        const ScorePlan S2 = plan_score(c2, *m, rows);
        std::vector<const void *> gc(d.d);
        for (int p = 0; p < d.d; ++p) gc[p] = G.col[p];
        const ScoreOut o2{gm, eps_f, P.mu, P.sigma, P.ei, nullptr, acq_out, nullptr};
        hipError_t e = c2.ok ? score_front(*m, S2, gc.data(), cnt, rows, s, nullptr)
                             : hipErrorInvalidValue;
        if (e == hipSuccess) e = score_back(*m, S2, cnt, rows, o2, 0, s, nullptr);
        return e;
      };
      const int64_t rowsM = round_up(M, kRowTile);
      Carver c1;
      c1.base = P.score_ws;
      c1.size = P.score_bytes;
      const ScorePlan S1 = plan_score(c1, *m, rowsM);
      if (!c1.ok) return fail(GP_E_INVALID, "internal error: local-search scoring buffers");
      HIPCHK(score_encode(*m, S1, C_cols, M, rowsM, s));
      HIPCHK(score_xkernel(*m, S1, rowsM, s, false));  // the means only
      HIPCHK(launch_ls_bound(S1.mu64, S1.sens, S1.valid, mask, M, m->fstar,
                             std::sqrt(m->sv) * (1.0 + 1e-6), P.acq, P.count, s));
      const int kt = (int)std::min<int64_t>(kLsPruneTop, M);
      HIPCHK(launch_ls_topk(P.acq, M, kt, P.pv, P.pi, kLsTopkParts, P.tv, P.ti, s));
      HIPCHK(launch_ls_gather_rows(d, C, P.ti, kt, P.G, mask, P.mg, s));
      HIPCHK(score_rows(P.G, mask ? P.mg : nullptr, kt, P.tacq));
      HIPCHK(launch_ls_topk(P.tacq, kt, k, P.pv, P.pi, kLsTopkParts, P.kv, P.ki, s, P.ti));
      HIPCHK(launch_ls_compact(P.acq, M, P.kv + (k - 1), P.list, P.count, P.cap, s));
      HIPCHK(hipMemcpyAsync(hact, P.count, sizeof(int32_t), hipMemcpyDeviceToHost, s));
      HIPCHK(hipStreamSynchronize(s));
      const int64_t cnt = hact[0];
      if (cnt >= k && cnt <= P.cap) {
        HIPCHK(launch_ls_gather_rows(d, C, P.list, cnt, P.G, mask, P.mg, s));
        HIPCHK(score_rows(P.G, mask ? P.mg : nullptr, cnt, P.acq));
        HIPCHK(launch_ls_topk(P.acq, cnt, k, P.pv, P.pi, kLsTopkParts, P.sv, P.si, s, P.list));
        picked = true;
      }
    }
    if (!picked) {
      if ((st = gp_score(m, C_cols, M, mask, eps_f, P.mu, P.sigma, P.ei, nullptr, P.acq, nullptr,
                         P.score_ws, P.score_bytes, stream)) != GP_OK)
        return st;
      HIPCHK(launch_ls_topk(P.acq, M, k, P.pv, P.pi, kLsTopkParts, P.sv, P.si, s));
    }
    HIPCHK(launch_ls_gather(d, C, M, P.si, P.sv, k, P.cur, P.cur_acq, P.active, P.steps, s));

    // climb: each step moves the active starts to their best neighbour of the step before
    // (from the second step of a batch on), encodes the new neighbours straight into the
    // scoring buffers and scores them; a batch ends with the moves of its last step
    const int64_t N = (int64_t)k * d.nnb;
    const int64_t rowsN = round_up(std::max<int64_t>(N, 1), kRowTile);
    Carver sc;
    sc.base = P.score_ws;
    sc.size = P.score_bytes;
    const ScorePlan SP = plan_score(sc, *m, rowsN);
    if (!sc.ok) return fail(GP_E_INVALID, "internal error: local-search scoring buffers");
    const LSEnc e{m->d_penc, m->d_table, SP.cand, SP.valid, SP.rcount, rowsN, m->lay.R, 0};
    const ScoreOut o{P.mask, eps_f, P.mu, P.sigma, P.ei, nullptr, P.acq, nullptr};
    struct EvPair {  // on an error exit: no enqueued work still uses the workspace
      hipEvent_t e[2] = {};
      hipStream_t s;
      bool ok = false;
      ~EvPair() {
        if (!ok) (void)hipStreamSynchronize(s);
        for (hipEvent_t x : e)
          if (x) (void)hipEventDestroy(x);
      }
    } evb;
    evb.s = s;
    for (auto &x : evb.e) HIPCHK(hipEventCreateWithFlags(&x, hipEventDisableTiming));
    int slot = 0, prev = -1;
    for (int done = 0; d.nnb > 0 && done < max_steps;) {
      const int batch = std::min(kLsStepsPerCheck, max_steps - done);
      for (int b = 0; b < batch; ++b) {
        HIPCHK(launch_ls_step(d, P.cur, k, P.active, b > 0 ? P.acq : nullptr, P.cur_acq, P.steps,
                              max_steps, true, e, P.mask, s));
        HIPCHK(score_xkernel(*m, SP, rowsN, s));
        HIPCHK(score_back(*m, SP, N, rowsN, o, 0, s, nullptr));
      }
      HIPCHK(launch_ls_step(d, P.cur, k, P.active, P.acq, P.cur_acq, P.steps, max_steps, false, e,
                            P.mask, s));
      done += batch;
      // The host reads a batch's active flags while the next batch runs (two readback
      // slots), so it waits only for work that is done or nearly; a batch enqueued after
      // every start has stopped changes nothing.
      HIPCHK(hipMemcpyAsync(hact + slot * kLsMaxStarts, P.active, sizeof(int32_t) * k,
                            hipMemcpyDeviceToHost, s));
      HIPCHK(hipEventRecord(evb.e[slot], s));
      if (prev >= 0) {
        HIPCHK(hipEventSynchronize(evb.e[prev]));
        bool any = false;
        for (int q = 0; q < k; ++q) any = any || hact[prev * kLsMaxStarts + q] != 0;
        if (!any) break;
      }
      prev = slot;
      slot ^= 1;
    }

    // outputs
    for (int p = 0; p < d.d; ++p)
      HIPCHK(hipMemcpyAsync(out_cols[p], P.cur.col[p], sizeof(uint32_t) * d.words[p] * k,
                            hipMemcpyDeviceToDevice, s));
    HIPCHK(hipMemcpyAsync(out_acq, P.cur_acq, sizeof(float) * k, hipMemcpyDeviceToDevice, s));
    HIPCHK(hipMemcpyAsync(out_steps, P.steps, sizeof(int32_t) * k, hipMemcpyDeviceToDevice, s));
    HIPCHK(hipMemcpyAsync(out_start, P.si, sizeof(int64_t) * k, hipMemcpyDeviceToDevice, s));
    HIPCHK(hipStreamSynchronize(s));
    evb.ok = true;
    g_err.clear();
    return GP_OK;
  } catch (const std::exception &e) {
    return fail(GP_E_INVALID, std::string("internal error: ") + e.what());
  }
}

// ------------------------------------------------------------------ hyperparameters
namespace {
struct HypPlan {
  ParamEnc *penc; double *table; TermDesc *tdesc; int32_t *order;
  uint32_t *codes; uint8_t *valid; double *yf, *T;
  double *A, *L, *X, *D; int32_t *info; double *alpha, *z, *val, *grad, *part;
  double *val0; int32_t *keep;
  LbfgsState st;
  int ld, B;
  int64_t sM, sD;
};

// Workspace of a call on n observations: batches of B settings, S0 sample values, K
// L-BFGS starts.
HypPlan plan_hyp(Carver &cv, const Layout &L, int n, int B, int S0, int K) {
  HypPlan P{};
  const int d = L.d, D = d + 2;
  P.B = B;
  P.ld = (int)round_up(n, kNB);
  P.sM = (int64_t)P.ld * P.ld;
  P.sD = (int64_t)(P.ld / kNB) * kNB * kNB;
  P.penc = cv.take<ParamEnc>(d);
  P.table = cv.take<double>((int64_t)L.table.size());
  P.tdesc = cv.take<TermDesc>(d);
  P.order = cv.take<int32_t>(n);
  P.codes = cv.take<uint32_t>((int64_t)n * L.R);
  P.valid = cv.take<uint8_t>(n);
  P.yf = cv.take<double>(n);
  P.T = cv.take<double>((int64_t)d * n * n);
  P.A = cv.take<double>(B * 2 * P.sM);  // per setting K, identity rows, then K^-1
  P.L = cv.take<double>(B * P.sM);
  P.X = cv.take<double>(B * P.sM);
  P.D = cv.take<double>(B * P.sD);
  P.info = cv.take<int32_t>(B);
  P.alpha = cv.take<double>((int64_t)B * n);
  P.z = cv.take<double>((int64_t)B * n);
  P.val = cv.take<double>(B);
  P.grad = cv.take<double>((int64_t)B * D);
  P.part = cv.take<double>(hyp_grad_part_elems(B, d));
  P.val0 = S0 > 0 ? cv.take<double>(S0) : nullptr;
  P.keep = K > 0 ? cv.take<int32_t>(K) : nullptr;
  if (K > 0) {
    LbfgsState &st = P.st;
    st.x = cv.take<double>((int64_t)K * D);
    st.xt = cv.take<double>((int64_t)K * D);
    st.g = cv.take<double>((int64_t)K * D);
    st.p = cv.take<double>((int64_t)K * D);
    st.S = cv.take<double>((int64_t)K * kLbfgsMem * D);
    st.Y = cv.take<double>((int64_t)K * kLbfgsMem * D);
    st.sy = cv.take<double>((int64_t)K * kLbfgsMem);
    st.F = cv.take<double>(K);
    st.t = cv.take<double>(K);
    st.slope = cv.take<double>(K);
    st.status = cv.take<int32_t>(K);
    st.phase = cv.take<int32_t>(K);
    st.it = cv.take<int32_t>(K);
    st.halv = cv.take<int32_t>(K);
    st.npairs = cv.take<int32_t>(K);
    st.head = cv.take<int32_t>(K);
    st.active = cv.take<int32_t>(K);
  }
  return P;
}

gp_status hyp_check_args(const gp_space *space, int32_t n, const gp_gamma_prior *prior,
                         double noise_floor, Layout &L) {
  if (!space) return fail(GP_E_INVALID, "space is NULL");
  if (n < 1 || n > kMaxN) return fail(GP_E_INVALID, "n must be in 1..4096");
  if (prior && !(prior->shape > 0.0 && prior->rate > 0.0 && std::isfinite(prior->shape) &&
                 std::isfinite(prior->rate)))
    return fail(GP_E_INVALID, "prior shape and rate must be finite and > 0");
  if (!(noise_floor >= 0.0) || !std::isfinite(noise_floor))
    return fail(GP_E_INVALID, "noise_floor must be finite and >= 0");
  if (space->d < 1 || space->d > kMaxD) return fail(GP_E_UNSUPPORTED, "space.d must be in 1..64");
  std::vector<double> ones((size_t)space->d, 1.0);
  return build_layout(space, ones.data(), L);
}

// Encodes the feasible observations (in index order), gathers their targets and builds
// the pair terms T. Synchronises (feasibility flags, validity).
gp_status hyp_prepare(const Layout &L, const void *const *X_cols, int32_t n, const double *y,
                      const uint8_t *feasible, const HypPlan &P, hipStream_t s, int *nf_out) {
  gp_status st = check_cols(X_cols, L.d);
  if (st != GP_OK) return st;
  std::vector<uint8_t> hf((size_t)n, 1);
  if (feasible) {
    HIPCHK(hipMemcpyAsync(hf.data(), feasible, n, hipMemcpyDeviceToHost, s));
    HIPCHK(hipStreamSynchronize(s));
  }
  std::vector<int32_t> order;
  for (int i = 0; i < n; ++i)
    if (hf[i]) order.push_back(i);
  const int nf = (int)order.size();
  if (nf == 0) return fail(GP_E_INVALID, "no feasible observation");
  HIPCHK(hipMemcpyAsync(P.penc, L.penc.data(), sizeof(ParamEnc) * L.penc.size(), hipMemcpyHostToDevice, s));
  if (!L.table.empty())
    HIPCHK(hipMemcpyAsync(P.table, L.table.data(), sizeof(double) * L.table.size(), hipMemcpyHostToDevice, s));
  HIPCHK(hipMemcpyAsync(P.tdesc, L.tdesc.data(), sizeof(TermDesc) * L.tdesc.size(), hipMemcpyHostToDevice, s));
  HIPCHK(hipMemcpyAsync(P.order, order.data(), sizeof(int32_t) * nf, hipMemcpyHostToDevice, s));
  HIPCHK(encode_into(L, X_cols, P.penc, P.table, nf, nf, P.order, P.codes, 1, L.R, P.valid, nullptr,
                     nullptr, s));
  std::vector<uint8_t> hv((size_t)nf);
  HIPCHK(hipMemcpyAsync(hv.data(), P.valid, nf, hipMemcpyDeviceToHost, s));
  HIPCHK(hipStreamSynchronize(s));
  for (int i = 0; i < nf; ++i)
    if (!hv[i])
      return fail(GP_E_INVALID, "observation " + std::to_string(order[i]) +
                                    " is not a valid configuration of the space");
  HIPCHK(launch_gather_f64(y, P.order, P.yf, nf, s));
  HIPCHK(launch_hyp_terms(P.codes, L.R, P.tdesc, L.d, nf, P.T, s));
  *nf_out = nf;
  return GP_OK;
}

HypArgs hyp_args(const Layout &L, const HypPlan &P, int nf, const gp_gamma_prior *prior,
                 double noise_floor) {
  HypArgs a{};
  a.T = P.T;
  a.y = P.yf;
  a.d = L.d;
  a.nf = nf;
  a.ld = P.ld;
  a.sM = P.sM;
  a.sA = 2 * P.sM;
  a.noise_floor = noise_floor;
  a.has_prior = prior ? 1 : 0;
  if (prior) {
    a.prior_shape = prior->shape;
    a.prior_rate = prior->rate;
    a.prior_c0 = prior->shape * std::log(prior->rate) - std::lgamma(prior->shape);
  }
  a.info = P.info;
  return a;
}

// value (and gradient) of the B settings a.theta[0..B) (stream-ordered, no sync)
hipError_t hyp_eval(const HypArgs &a, const HypPlan &P, int B, double *value, double *grad,
                    hipStream_t s) {
  hipError_t e;
  if ((e = launch_hyp_gram(a, B, P.A, s)) != hipSuccess) return e;
  CholBatch bt;
  bt.count = B;
  bt.sA = 2 * P.sM;
  bt.sL = P.sM;
  bt.sD = P.sD;
  bt.sX = P.sM;
  // [K; I] (both written by the Gram kernel) is factored: the identity rows' panels give
  // X = L^-1 (no triangular-inverse chain). L's blocks above the diagonal are never read
  // here: no clearing.
  if ((e = chol_factor_batched(P.A, P.ld, P.L, P.ld, P.D, a.nf, a.info, bt, s, false, P.X,
                               P.ld)) != hipSuccess)
    return e;
  if ((e = launch_hyp_value(a, B, P.L, P.X, value, P.alpha, P.z, s)) != hipSuccess) return e;
  if (!grad) return hipSuccess;
  if ((e = launch_ata_batched(P.X, P.ld, P.A, a.nf, a.info, bt, s)) != hipSuccess) return e;
  return launch_hyp_grad(a, B, P.A, P.alpha, P.part, grad, a.d + 2, s);
}
}  // namespace

size_t gp_hyper_workspace_bytes(const gp_space *space, int32_t n, int32_t n_settings,
                                int32_t n_keep) {
  Layout L;
  if (hyp_check_args(space, n, nullptr, 0.0, L) != GP_OK) return 0;
  if (n_settings < 1 || n_keep < 0 || n_keep > kHypBatch || n_keep > n_settings) return 0;
  const int B = std::max(std::min(n_settings, kHypBatch), n_keep);
  Carver cv;
  plan_hyp(cv, L, n, B, n_keep > 0 ? n_settings : 0, n_keep);
  return cv.off;
}

gp_status gp_log_posterior(const gp_space *space, const void *const *X_cols, int32_t n,
                           const double *y, const uint8_t *feasible, const double *theta,
                           int32_t count, const gp_gamma_prior *prior, double noise_floor,
                           double *value, double *grad, void *workspace, size_t ws_bytes,
                           void *stream) {
  try {
    Layout L;
    gp_status st = hyp_check_args(space, n, prior, noise_floor, L);
    if (st != GP_OK) return st;
    if (!y) return fail(GP_E_INVALID, "y is NULL");
    if (count < 1) return fail(GP_E_INVALID, "count must be >= 1");
    if (!theta || !value) return fail(GP_E_INVALID, "theta and value are required");
    const int B = std::min(count, kHypBatch), D = L.d + 2;
    Carver meas;
    plan_hyp(meas, L, n, B, 0, 0);
    if ((st = check_ws(workspace, ws_bytes, meas.off)) != GP_OK) return st;
    Carver cv;
    cv.base = static_cast<char *>(workspace);
    cv.size = ws_bytes;
    const HypPlan P = plan_hyp(cv, L, n, B, 0, 0);
    hipStream_t s = static_cast<hipStream_t>(stream);
    int nf = 0;
    if ((st = hyp_prepare(L, X_cols, n, y, feasible, P, s, &nf)) != GP_OK) return st;
    HypArgs a = hyp_args(L, P, nf, prior, noise_floor);
    a.theta_ld = D;
    for (int c0 = 0; c0 < count; c0 += B) {
      const int nb = std::min(B, count - c0);
      a.theta = theta + (int64_t)c0 * D;
      HIPCHK(hyp_eval(a, P, nb, value + c0, grad ? grad + (int64_t)c0 * D : nullptr, s));
    }
    HIPCHK(hipStreamSynchronize(s));
    g_err.clear();
    return GP_OK;
  } catch (const std::exception &e) {
    return fail(GP_E_INVALID, std::string("internal error: ") + e.what());
  }
}

gp_status gp_hyperfit(const gp_space *space, const void *const *X_cols, int32_t n,
                      const double *y, const uint8_t *feasible, const double *theta0,
                      int32_t n_samples, int32_t n_keep, const gp_gamma_prior *prior,
                      double noise_floor, int32_t max_iter, double gtol, double ftol,
                      double *theta_out, double *value_out, double *value0_out,
                      int32_t *keep_out, int32_t *iters_out, int32_t *status_out,
                      void *workspace, size_t ws_bytes, void *stream) {
  try {
    Layout L;
    gp_status st = hyp_check_args(space, n, prior, noise_floor, L);
    if (st != GP_OK) return st;
    if (!y) return fail(GP_E_INVALID, "y is NULL");
    if (n_samples < 1) return fail(GP_E_INVALID, "n_samples must be >= 1");
    if (n_keep < 1 || n_keep > kHypBatch || n_keep > n_samples)
      return fail(GP_E_INVALID, "n_keep must be in 1..min(64, n_samples)");
    if (max_iter < 0) return fail(GP_E_INVALID, "max_iter must be >= 0");
    if (!(gtol >= 0.0) || !(ftol >= 0.0)) return fail(GP_E_INVALID, "gtol and ftol must be >= 0");
    if (!theta0 || !theta_out || !value_out)
      return fail(GP_E_INVALID, "theta0, theta_out and value_out are required");
    const int D = L.d + 2, K = n_keep;
    const int B = std::max(std::min(n_samples, kHypBatch), K);
    Carver meas;
    plan_hyp(meas, L, n, B, n_samples, K);
    if ((st = check_ws(workspace, ws_bytes, meas.off)) != GP_OK) return st;
    Carver cv;
    cv.base = static_cast<char *>(workspace);
    cv.size = ws_bytes;
    const HypPlan P = plan_hyp(cv, L, n, B, n_samples, K);
    hipStream_t s = static_cast<hipStream_t>(stream);
    int32_t *hact = ls_active_host();
    if (!hact) return fail(GP_E_HIP, "pinned host allocation failed");
    int nf = 0;
    if ((st = hyp_prepare(L, X_cols, n, y, feasible, P, s, &nf)) != GP_OK) return st;
    HypArgs a = hyp_args(L, P, nf, prior, noise_floor);

    // objective of every sampled setting, then the n_keep best
    double *v0 = value0_out ? value0_out : P.val0;
    int32_t *keep = keep_out ? keep_out : P.keep;
    a.theta_ld = D;
    for (int c0 = 0; c0 < n_samples; c0 += B) {
      const int nb = std::min(B, n_samples - c0);
      a.theta = theta0 + (int64_t)c0 * D;
      HIPCHK(hyp_eval(a, P, nb, v0 + c0, nullptr, s));
    }
    HIPCHK(launch_hyp_select(v0, n_samples, K, theta0, D, keep, P.st.x, s));

    // L-BFGS from each kept setting: one batched evaluation of the trial points per
    // round; the host reads the running flags every few rounds
    constexpr int kRoundsPerCheck = 4;
    HIPCHK(launch_lbfgs_init(P.st, K, D, s));
    a.theta = P.st.xt;
    a.active = P.st.active;
    LbfgsParams prm{D, max_iter, gtol, ftol};
    const int64_t max_rounds = (int64_t)(max_iter + 1) * (kLbfgsMaxHalvings + 1) + 1;
    for (int64_t round = 0; round < max_rounds;) {
      for (int r = 0; r < kRoundsPerCheck && round < max_rounds; ++r, ++round) {
        HIPCHK(hyp_eval(a, P, K, P.val, P.grad, s));
        HIPCHK(launch_lbfgs_step(P.st, K, prm, P.val, P.grad, D, s));
      }
      HIPCHK(hipMemcpyAsync(hact, P.st.active, sizeof(int32_t) * K, hipMemcpyDeviceToHost, s));
      HIPCHK(hipStreamSynchronize(s));
      bool any = false;
      for (int q = 0; q < K; ++q) any = any || hact[q] != 0;
      if (!any) break;
    }
    HIPCHK(hipMemcpyAsync(theta_out, P.st.x, sizeof(double) * K * D, hipMemcpyDeviceToDevice, s));
    HIPCHK(launch_lbfgs_outputs(P.st, K, value_out, iters_out, status_out, s));
    HIPCHK(hipStreamSynchronize(s));
    g_err.clear();
    return GP_OK;
  } catch (const std::exception &e) {
    return fail(GP_E_INVALID, std::string("internal error: ") + e.what());
  }
}

// ------------------------------------------------------------------ Chain-of-Trees
struct gp_cot {
  bgp::CotDesc h;             // host copy of the descriptor
  bgp::CotDesc *d_desc = nullptr;
  uint64_t *d_keys = nullptr;
};

namespace {
struct CotPlan {
  CotDesc *desc; uint64_t *keys; unsigned long long *bad;
};
CotPlan plan_cot(Carver &cv, int64_t total_leaves) {
  CotPlan P{};
  P.desc = cv.take<CotDesc>(1);
  P.keys = cv.take<uint64_t>(std::max<int64_t>(total_leaves, 1));
  P.bad = cv.take<unsigned long long>(1);
  return P;
}

// Descriptor of the chain; checks the space, the trees and the key range.
gp_status cot_desc(const gp_space *space, int32_t n_trees, const int32_t *tree_size,
                   const int32_t *tree_params, const int64_t *n_leaves, CotDesc &D,
                   int64_t &total) {
  Layout L;
  gp_status st = build_layout(space, nullptr, L);
  if (st != GP_OK) return st;
  const int d = space->d;
  if (n_trees < 0 || n_trees > kCotMaxTrees) return fail(GP_E_INVALID, "n_trees must be in 0..64");
  if (n_trees > 0 && (!tree_size || !tree_params || !n_leaves))
    return fail(GP_E_INVALID, "tree_size, tree_params and n_leaves are required");
  std::memset(&D, 0, sizeof(D));
  D.d = d;
  D.n_trees = n_trees;
  for (int p = 0; p < d; ++p) {
    const int t = space->type[p];
    D.kind[p] = t;
    D.tree[p] = -1;
    if (t == GP_INT) {
      D.lo[p] = (int32_t)space->lo[p];
      D.dim[p] = (int32_t)(space->hi[p] - space->lo[p] + 1.0);
    } else if (t == GP_REAL) {
      D.rlo[p] = space->lo[p];
      D.rhi[p] = space->hi[p];
    } else {
      D.dim[p] = space->n_levels[p];  // ORD values, CAT levels, PERM m
    }
  }
  int np = 0;
  total = 0;
  for (int t = 0; t < n_trees; ++t) {
    const int k = tree_size[t];
    if (k < 1 || np + k > d) return fail(GP_E_INVALID, "tree sizes must be >= 1 and fit the space");
    if (n_leaves[t] < 1) return fail(GP_E_INVALID, "every tree needs at least one leaf");
    D.tstart[t] = np;
    D.tcount[t] = k;
    D.koff[t] = total;
    D.nleaves[t] = n_leaves[t];
    total += n_leaves[t];
    int bits = 0;
    unsigned __int128 range = 1;
    for (int l = k - 1; l >= 0; --l) {
      const int p = tree_params[np + l];
      if (p < 0 || p >= d) return fail(GP_E_INVALID, "tree parameter index out of range");
      if (D.tree[p] >= 0) return fail(GP_E_INVALID, "a parameter is in two trees");
      if (D.kind[p] != GP_INT && D.kind[p] != GP_ORD && D.kind[p] != GP_CAT)
        return fail(GP_E_UNSUPPORTED, "trees hold INT, ORD and CAT parameters only");
      int w = 0;
      while (w < 32 && ((int64_t)1 << w) < (int64_t)D.dim[p]) ++w;  // bits of dim - 1
      D.tree[p] = t;
      D.tparam[np + l] = p;
      D.shift[p] = bits;
      D.fmask[p] = w == 32 ? 0xffffffffu : (uint32_t)((1ull << w) - 1);
      bits += w;
      if (bits > 64) return fail(GP_E_UNSUPPORTED, "a tree's key needs more than 64 bits");
      range *= (unsigned __int128)D.dim[p];
    }
    if ((unsigned __int128)n_leaves[t] > range) return fail(GP_E_INVALID, "more leaves than configurations");
    np += k;
  }
  int words = n_trees;
  for (int p = 0; p < d; ++p)
    if (D.tree[p] < 0) words += D.kind[p] == GP_PERM ? D.dim[p] - 1 : 1;
  D.words = words;
  return GP_OK;
}
}  // namespace

size_t gp_cot_workspace_bytes(const gp_space *space, int32_t n_trees, const int32_t *tree_size,
                              const int32_t *tree_params, const int64_t *n_leaves) {
  CotDesc D;
  int64_t total = 0;
  if (cot_desc(space, n_trees, tree_size, tree_params, n_leaves, D, total) != GP_OK) return 0;
  Carver cv;
  plan_cot(cv, total);
  return cv.off;
}

gp_status gp_cot_create(const gp_space *space, int32_t n_trees, const int32_t *tree_size,
                        const int32_t *tree_params, const int64_t *n_leaves,
                        const int32_t *const *leaves, void *workspace, size_t ws_bytes,
                        void *stream, gp_cot **out) {
  try {
    if (!out) return fail(GP_E_INVALID, "out is NULL");
    *out = nullptr;
    std::unique_ptr<gp_cot> c(new gp_cot());
    int64_t total = 0;
    gp_status st = cot_desc(space, n_trees, tree_size, tree_params, n_leaves, c->h, total);
    if (st != GP_OK) return st;
    for (int t = 0; t < n_trees; ++t)
      if (!leaves || !leaves[t]) return fail(GP_E_INVALID, "leaves of tree " + std::to_string(t) + " are NULL");
    Carver meas;
    plan_cot(meas, total);
    if ((st = check_ws(workspace, ws_bytes, meas.off)) != GP_OK) return st;
    Carver cv;
    cv.base = static_cast<char *>(workspace);
    cv.size = ws_bytes;
    const CotPlan P = plan_cot(cv, total);
    hipStream_t s = static_cast<hipStream_t>(stream);
    c->d_desc = P.desc;
    c->d_keys = P.keys;
    HIPCHK(hipMemcpyAsync(P.desc, &c->h, sizeof(CotDesc), hipMemcpyHostToDevice, s));
    // keys of every tree; the first bad leaf (out of range or out of order) is reported
    for (int t = 0; t < n_trees; ++t) {
      unsigned long long bad = ~0ull;
      HIPCHK(hipMemcpyAsync(P.bad, &bad, sizeof(bad), hipMemcpyHostToDevice, s));
      HIPCHK(launch_cot_keys(P.desc, t, leaves[t], c->h.nleaves[t], P.keys + c->h.koff[t], P.bad, s));
      HIPCHK(hipMemcpyAsync(&bad, P.bad, sizeof(bad), hipMemcpyDeviceToHost, s));
      HIPCHK(hipStreamSynchronize(s));
      if (bad != ~0ull)
        return fail(GP_E_INVALID, "tree " + std::to_string(t) + ", leaf " + std::to_string(bad) +
                                      ": a value index out of range or leaves not in strictly "
                                      "increasing lexicographic order");
    }
    HIPCHK(hipStreamSynchronize(s));
    *out = c.release();
    g_err.clear();
    return GP_OK;
  } catch (const std::exception &e) {
    return fail(GP_E_INVALID, std::string("internal error: ") + e.what());
  }
}

gp_status gp_cot_sample(const gp_cot *c, int64_t M, uint64_t seed, uint64_t offset,
                        void *const *out_cols, void *stream) {
  if (!c) return fail(GP_E_INVALID, "chain is NULL");
  if (M < 0 || M > INT32_MAX) return fail(GP_E_INVALID, "M must be in 0..2^31-1");
  if (M == 0) return GP_OK;
  gp_status st = check_cols(const_cast<const void *const *>(out_cols), c->h.d);
  if (st != GP_OK) return st;
  CotCols oc{};
  for (int p = 0; p < c->h.d; ++p) oc.col[p] = out_cols[p];
  HIPCHK(launch_cot_sample(c->d_desc, c->d_keys, M, seed, offset, oc, static_cast<hipStream_t>(stream)));
  return GP_OK;
}

gp_status gp_cot_member(const gp_cot *c, const void *const *cols, int64_t M, uint8_t *mask,
                        void *stream) {
  if (!c) return fail(GP_E_INVALID, "chain is NULL");
  if (M < 0 || M > INT32_MAX) return fail(GP_E_INVALID, "M must be in 0..2^31-1");
  if (M == 0) return GP_OK;
  if (!mask) return fail(GP_E_INVALID, "mask is NULL");
  if (!cols) return fail(GP_E_INVALID, "column array is NULL");
  CotCols cc{};
  for (int p = 0; p < c->h.d; ++p) {
    if (c->h.tree[p] >= 0 && !cols[p])
      return fail(GP_E_INVALID, "column " + std::to_string(p) + " (in a tree) is NULL");
    cc.col[p] = const_cast<void *>(cols[p]);
  }
  HIPCHK(launch_cot_member(c->d_desc, c->d_keys, cc, M, mask, static_cast<hipStream_t>(stream)));
  return GP_OK;
}

void gp_cot_free(gp_cot *c) { delete c; }

// ------------------------------------------------------------------ random forest
struct gp_forest {
  bgp::ForestDesc h;
  bgp::ForestDesc *d_desc = nullptr;
  bgp::ForestNode *d_nodes = nullptr;
  int32_t *d_nnodes = nullptr;
};

namespace {
struct ForestPlan {
  ForestDesc *desc; ParamEnc *penc; double *table; uint32_t *codes; uint8_t *valid;
  double *X; int32_t *idx, *tmp, *aux, *nnodes; ForestNode *nodes;
};
ForestPlan plan_forest(Carver &cv, const Layout &L, int n, int F, int T) {
  ForestPlan P{};
  P.desc = cv.take<ForestDesc>(1);
  P.nodes = cv.take<ForestNode>((int64_t)T * 2 * n);
  P.nnodes = cv.take<int32_t>(T);
  P.penc = cv.take<ParamEnc>(L.d);
  P.table = cv.take<double>((int64_t)L.table.size());
  P.codes = cv.take<uint32_t>((int64_t)n * L.R);
  P.valid = cv.take<uint8_t>(n);
  P.X = cv.take<double>((int64_t)F * n);
  P.idx = cv.take<int32_t>((int64_t)T * n);
  P.tmp = cv.take<int32_t>((int64_t)T * n);
  P.aux = cv.take<int32_t>((int64_t)T * 2 * n * 3);
  return P;
}

gp_status forest_desc(const gp_space *space, int32_t n, int32_t n_trees, int32_t max_depth,
                      int32_t min_split, uint64_t seed, Layout &L, ForestDesc &D) {
  gp_status st = build_layout(space, nullptr, L);
  if (st != GP_OK) return st;
  if (n < 1 || n > kMaxN) return fail(GP_E_INVALID, "n must be in 1..4096");
  if (n_trees < 1 || n_trees > 4096) return fail(GP_E_INVALID, "n_trees must be in 1..4096");
  if (max_depth < 0) return fail(GP_E_INVALID, "max_depth must be >= 0");
  if (min_split < 1) return fail(GP_E_INVALID, "min_split must be >= 1");
  std::memset(&D, 0, sizeof(D));
  D.d = space->d;
  int F = 0;
  for (int p = 0; p < D.d; ++p) {
    D.kind[p] = space->type[p];
    D.m[p] = D.kind[p] == GP_PERM ? space->n_levels[p] : 1;
    D.fofs[p] = F;
    F += D.m[p];
  }
  if (F > kForestMaxF) return fail(GP_E_UNSUPPORTED, "more than 120 forest features");
  int mtry = 1;
  while ((mtry + 1) * (mtry + 1) <= F) ++mtry;
  D.F = F;
  D.n = n;
  D.n_trees = n_trees;
  D.max_depth = max_depth;
  D.min_split = min_split;
  D.mtry = mtry;
  D.cap = 2 * n;
  D.seed = seed;
  return GP_OK;
}
}  // namespace

size_t gp_forest_workspace_bytes(const gp_space *space, int32_t n, int32_t n_trees) {
  Layout L;
  ForestDesc D;
  if (forest_desc(space, n, n_trees, 0, 2, 0, L, D) != GP_OK) return 0;
  Carver cv;
  plan_forest(cv, L, n, D.F, n_trees);
  return cv.off;
}

gp_status gp_forest_fit(const gp_space *space, const void *const *X_cols, int32_t n,
                        const uint8_t *feasible, int32_t n_trees, int32_t max_depth,
                        int32_t min_split, uint64_t seed, void *workspace, size_t ws_bytes,
                        void *stream, gp_forest **out) {
  try {
    if (!out) return fail(GP_E_INVALID, "out is NULL");
    *out = nullptr;
    if (!feasible) return fail(GP_E_INVALID, "feasible is NULL");
    std::unique_ptr<gp_forest> f(new gp_forest());
    Layout L;
    gp_status st = forest_desc(space, n, n_trees, max_depth, min_split, seed, L, f->h);
    if (st != GP_OK) return st;
    if ((st = check_cols(X_cols, L.d)) != GP_OK) return st;
    Carver meas;
    plan_forest(meas, L, n, f->h.F, n_trees);
    if ((st = check_ws(workspace, ws_bytes, meas.off)) != GP_OK) return st;
    Carver cv;
    cv.base = static_cast<char *>(workspace);
    cv.size = ws_bytes;
    const ForestPlan P = plan_forest(cv, L, n, f->h.F, n_trees);
    hipStream_t s = static_cast<hipStream_t>(stream);
    // every observation must be a valid configuration of the space
    HIPCHK(hipMemcpyAsync(P.penc, L.penc.data(), sizeof(ParamEnc) * L.penc.size(), hipMemcpyHostToDevice, s));
    if (!L.table.empty())
      HIPCHK(hipMemcpyAsync(P.table, L.table.data(), sizeof(double) * L.table.size(), hipMemcpyHostToDevice, s));
    HIPCHK(encode_into(L, X_cols, P.penc, P.table, n, n, nullptr, P.codes, 1, L.R, P.valid, nullptr,
                       nullptr, s));
    std::vector<uint8_t> hv((size_t)n);
    HIPCHK(hipMemcpyAsync(hv.data(), P.valid, n, hipMemcpyDeviceToHost, s));
    HIPCHK(hipMemcpyAsync(P.desc, &f->h, sizeof(ForestDesc), hipMemcpyHostToDevice, s));
    HIPCHK(hipStreamSynchronize(s));
    for (int i = 0; i < n; ++i)
      if (!hv[i])
        return fail(GP_E_INVALID, "observation " + std::to_string(i) + " is not a valid configuration of the space");
    CotCols cc{};
    for (int p = 0; p < L.d; ++p) cc.col[p] = const_cast<void *>(X_cols[p]);
    HIPCHK(launch_forest_features(P.desc, cc, n, n, P.X, s));
    HIPCHK(launch_forest_train(P.desc, n_trees, P.X, feasible, P.idx, P.tmp, P.nodes, P.aux,
                               P.nnodes, s));
    HIPCHK(hipStreamSynchronize(s));
    f->d_desc = P.desc;
    f->d_nodes = P.nodes;
    f->d_nnodes = P.nnodes;
    *out = f.release();
    g_err.clear();
    return GP_OK;
  } catch (const std::exception &e) {
    return fail(GP_E_INVALID, std::string("internal error: ") + e.what());
  }
}

gp_status gp_forest_predict(const gp_forest *f, const void *const *C_cols, int64_t M,
                            const float *ei, const uint8_t *mask, float eps_f, float *p_feas,
                            float *acq, void *stream) {
  if (!f) return fail(GP_E_INVALID, "forest is NULL");
  if (M < 0 || M > INT32_MAX) return fail(GP_E_INVALID, "M must be in 0..2^31-1");
  if (M == 0) return GP_OK;
  if (!p_feas) return fail(GP_E_INVALID, "p_feas is NULL");
  if (acq && !ei) return fail(GP_E_INVALID, "acq needs ei");
  gp_status st = check_cols(C_cols, f->h.d);
  if (st != GP_OK) return st;
  CotCols cc{};
  for (int p = 0; p < f->h.d; ++p) cc.col[p] = const_cast<void *>(C_cols[p]);
  HIPCHK(launch_forest_predict(f->d_desc, f->h, f->d_nodes, cc, M, ei, mask, eps_f, p_feas, acq,
                               static_cast<hipStream_t>(stream)));
  return GP_OK;
}

gp_status gp_forest_tree(const gp_forest *f, int32_t tree, int32_t capacity, int32_t *n_nodes,
                         int32_t *feature, int32_t *left, double *value, void *stream) {
  if (!f) return fail(GP_E_INVALID, "forest is NULL");
  if (tree < 0 || tree >= f->h.n_trees) return fail(GP_E_INVALID, "tree out of range");
  if (!n_nodes || !feature || !left || !value) return fail(GP_E_INVALID, "NULL output");
  hipStream_t s = static_cast<hipStream_t>(stream);
  int32_t nn = 0;
  HIPCHK(hipMemcpyAsync(&nn, f->d_nnodes + tree, sizeof(int32_t), hipMemcpyDeviceToHost, s));
  HIPCHK(hipStreamSynchronize(s));
  *n_nodes = nn;
  if (nn > capacity) return fail(GP_E_INVALID, "capacity below the tree's node count");
  std::vector<ForestNode> h((size_t)nn);
  HIPCHK(hipMemcpyAsync(h.data(), f->d_nodes + (int64_t)tree * f->h.cap, sizeof(ForestNode) * nn,
                        hipMemcpyDeviceToHost, s));
  HIPCHK(hipStreamSynchronize(s));
  for (int k = 0; k < nn; ++k) {
    feature[k] = h[k].feature;
    left[k] = h[k].left;
    value[k] = h[k].val;
  }
  return GP_OK;
}

void gp_forest_free(gp_forest *f) { delete f; }

gp_status gp_score_refined_count(const gp_model *m, const void *workspace, int64_t M, void *stream,
                                 int64_t *count) {
  if (!m || !workspace || !count) return fail(GP_E_INVALID, "NULL argument");
  Carver cv;
  cv.base = static_cast<char *>(const_cast<void *>(workspace));
  const ScorePlan P = plan_score(cv, *m, round_up(std::max<int64_t>(M, 1), kRowTile));
  int32_t c = 0;
  hipStream_t s = static_cast<hipStream_t>(stream);
  HIPCHK(hipMemcpyAsync(&c, P.rcount, sizeof(int32_t), hipMemcpyDeviceToHost, s));
  HIPCHK(hipStreamSynchronize(s));
  *count = c;
  return GP_OK;
}

gp_status gp_debug_set_refine(gp_model *m, double var_frac, double sens) {
  if (!m) return fail(GP_E_INVALID, "NULL model");
  if (std::isnan(var_frac) || std::isnan(sens)) return fail(GP_E_INVALID, "NaN threshold");
  m->refine_var = var_frac;
  m->refine_sens = sens;
  return GP_OK;
}

// ------------------------------------------------------------------ inspection
size_t gp_debug_workspace_bytes(const gp_space *space, const gp_model *m, int64_t count) {
  if (count < 0 || count > INT32_MAX) return 0;
  Layout tmp;
  const Layout *L = nullptr;
  if (m) L = &m->lay;
  else if (build_layout(space, nullptr, tmp) == GP_OK) L = &tmp;
  else return 0;
  const int64_t rows = round_up(std::max<int64_t>(count, 1), kRowTile);
  Carver cv;
  cv.take<ParamEnc>(L->d);
  cv.take<double>((int64_t)L->table.size());
  cv.take<uint32_t>((int64_t)L->R_bound * rows);
  cv.take<uint8_t>(rows);
  if (m) {
    cv.take<uint16_t>(rows * 2 * m->lda);
    cv.take<double>(rows);
    cv.take<float>(rows);
    const int ns = xkernel_splits(rows, m->n);
    if (ns > 1) {
      cv.take<double>(ns * rows);
      cv.take<float>(ns * rows);
    }
  }
  return cv.off;
}

gp_status gp_debug_encode(const gp_space *space, const void *const *cols, int64_t count, float *out,
                          uint8_t *valid, void *workspace, size_t ws_bytes, void *stream) {
  try {
    Layout L;
    gp_status st = build_layout(space, nullptr, L);
    if (st != GP_OK) return st;
    if (count < 0 || count > INT32_MAX) return fail(GP_E_INVALID, "bad count");
    if (count == 0) return GP_OK;
    if (!out && L.n_num > 0) return fail(GP_E_INVALID, "out is NULL");
    if ((st = check_cols(cols, L.d)) != GP_OK) return st;
    const size_t need = gp_debug_workspace_bytes(space, nullptr, count);
    if ((st = check_ws(workspace, ws_bytes, need)) != GP_OK) return st;
    const int64_t rows = round_up(count, kRowTile);
    Carver cv;
    cv.base = static_cast<char *>(workspace);
    cv.size = ws_bytes;
    ParamEnc *penc = cv.take<ParamEnc>(L.d);
    double *table = cv.take<double>((int64_t)L.table.size());
    uint32_t *codes = cv.take<uint32_t>((int64_t)L.R_bound * rows);
    uint8_t *v = cv.take<uint8_t>(rows);
    hipStream_t s = static_cast<hipStream_t>(stream);
    if ((st = upload_layout(L, penc, table, nullptr, s)) != GP_OK) return st;
    HIPCHK(encode_into(L, cols, penc, table, count, rows, nullptr, codes, rows, 1, valid ? valid : v,
                       out, nullptr, s));
    HIPCHK(hipStreamSynchronize(s));  // the layout vectors are host staging for the copies
    return GP_OK;
  } catch (const std::exception &e) {
    return fail(GP_E_INVALID, std::string("internal error: ") + e.what());
  }
}

static gp_status debug_prep(const gp_model *m, const void *const *cols, int64_t count,
                            void *workspace, size_t ws_bytes, uint32_t **codes, int64_t *rows,
                            Carver &cv) {
  if (!m) return fail(GP_E_INVALID, "model is NULL");
  if (count < 0 || count > INT32_MAX) return fail(GP_E_INVALID, "bad count");
  gp_status st = check_cols(cols, m->lay.d);
  if (st != GP_OK) return st;
  if ((st = check_ws(workspace, ws_bytes, gp_debug_workspace_bytes(nullptr, m, count))) != GP_OK) return st;
  *rows = round_up(std::max<int64_t>(count, 1), kRowTile);
  cv.base = static_cast<char *>(workspace);
  cv.size = ws_bytes;
  cv.take<ParamEnc>(m->lay.d);
  cv.take<double>((int64_t)m->lay.table.size());
  *codes = cv.take<uint32_t>((int64_t)m->lay.R_bound * *rows);
  return GP_OK;
}

gp_status gp_debug_terms(const gp_model *m, const void *const *cols, int64_t count, float *terms,
                         void *workspace, size_t ws_bytes, void *stream) {
  Carver cv;
  uint32_t *codes;
  int64_t rows;
  gp_status st = debug_prep(m, cols, count, workspace, ws_bytes, &codes, &rows, cv);
  if (st != GP_OK) return st;
  if (count == 0) return GP_OK;
  if (!terms) return fail(GP_E_INVALID, "terms is NULL");
  uint8_t *v = cv.take<uint8_t>(rows);
  hipStream_t s = static_cast<hipStream_t>(stream);
  HIPCHK(encode_into(m->lay, cols, m->d_penc, m->d_table, count, rows, nullptr, codes, rows, 1, v,
                     nullptr, nullptr, s));
  HIPCHK(launch_terms(codes, rows, m->d_codes, m->lay.R, m->n, count, m->d_tdesc, m->lay.d, terms, s));
  return GP_OK;
}

gp_status gp_debug_xkernel(const gp_model *m, const void *const *cols, int64_t count, float *Kstar,
                           void *workspace, size_t ws_bytes, void *stream) {
  Carver cv;
  uint32_t *codes;
  int64_t rows;
  gp_status st = debug_prep(m, cols, count, workspace, ws_bytes, &codes, &rows, cv);
  if (st != GP_OK) return st;
  if (count == 0) return GP_OK;
  if (!Kstar) return fail(GP_E_INVALID, "Kstar is NULL");
  uint8_t *v = cv.take<uint8_t>(rows);
  uint16_t *K = cv.take<uint16_t>(rows * 2 * m->lda);
  double *mu64 = cv.take<double>(rows);
  float *sens = cv.take<float>(rows);
  XSplit xs{xkernel_splits(rows, m->n), nullptr, nullptr};
  if (xs.nsplit > 1) {
    xs.mu = cv.take<double>(xs.nsplit * rows);
    xs.sens = cv.take<float>(xs.nsplit * rows);
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  HIPCHK(encode_into(m->lay, cols, m->d_penc, m->d_table, count, rows, nullptr, codes, rows, 1, v,
                     nullptr, nullptr, s));
  XArgs xa = m->xa;
  xa.cand = codes;
  xa.ldc = rows;
  xa.Kstar = K;
  xa.mu = mu64;
  xa.sens = sens;
  xa.rows = rows;
  HIPCHK(launch_xkernel(xa, m->variant, xs, s));
  HIPCHK(launch_gather_rows_split(K, m->lda, std::ldexp(1.0f, -m->kexp), Kstar, m->n, count, m->n,
                                  s));
  return GP_OK;
}

gp_status gp_debug_pairs(const gp_model *m, const void *const *cols, int64_t count, float *r2,
                         int32_t *counts, uint64_t *word_params, int32_t *n_words,
                         void *workspace, size_t ws_bytes, void *stream) {
  Carver cv;
  uint32_t *codes;
  int64_t rows;
  gp_status st = debug_prep(m, cols, count, workspace, ws_bytes, &codes, &rows, cv);
  if (st != GP_OK) return st;
  const Layout &L = m->lay;
  const int W = L.n_bits + L.n_eq + L.n_dot;
  if (n_words) *n_words = W;
  if (word_params) {
    // the parameters behind each integer word (a Hamming permutation spans two BITS
    // words, a Spearman permutation is one entry for its pair of DOT words)
    for (int w = 0; w < W; ++w) word_params[w] = 0;
    for (const ParamEnc &e : L.penc) {
      const uint64_t bit = 1ull << e.col;
      const int perm = e.kind == GP_PERM ? (e.flags >> 8) : -1;
      if (e.word >= L.w_dot0) {
        word_params[L.n_bits + L.n_eq + (e.word - L.w_dot0) / 2] |= bit;
      } else if (e.word >= L.w_bits0) {
        word_params[e.word - L.w_bits0] |= bit;
        if (perm == GP_PERM_HAMMING) word_params[e.word - L.w_bits0 + 1] |= bit;
      }
    }
  }
  if (count == 0) return GP_OK;
  if (!r2 || (W > 0 && !counts)) return fail(GP_E_INVALID, "r2 and counts are required");
  uint8_t *v = cv.take<uint8_t>(rows);
  uint16_t *K = cv.take<uint16_t>(rows * 2 * m->lda);
  double *mu64 = cv.take<double>(rows);
  float *sens = cv.take<float>(rows);
  XSplit xs{xkernel_splits(rows, m->n), nullptr, nullptr};
  if (xs.nsplit > 1) {
    xs.mu = cv.take<double>(xs.nsplit * rows);
    xs.sens = cv.take<float>(xs.nsplit * rows);
  }
  if (!cv.ok) return fail(GP_E_WORKSPACE, "workspace too small");
  hipStream_t s = static_cast<hipStream_t>(stream);
  HIPCHK(encode_into(L, cols, m->d_penc, m->d_table, count, rows, nullptr, codes, rows, 1, v,
                     nullptr, nullptr, s));
  XArgs xa = m->xa;
  xa.cand = codes;
  xa.ldc = rows;
  xa.Kstar = K;
  xa.mu = mu64;
  xa.sens = sens;
  xa.rows = rows;
  xa.dbg_r2 = r2;
  // (with no integer words the kernel stores no counts: any device pointer will do)
  xa.dbg_cnt = W > 0 ? counts : reinterpret_cast<int32_t *>(r2);
  xa.dbg_count = count;
  HIPCHK(launch_xkernel(xa, m->variant, xs, s, true));
  return GP_OK;
}

// ------------------------------------------------------------------ profiling
gp_status gp_profile_start(void) {
  std::lock_guard<std::mutex> lk(g_prof.mu);
  g_prof.pool.reserve((size_t)kProfMaxCalls * kProfEvents);
  g_prof.calls.clear();
  g_prof.next = 0;
  g_prof.on = true;
  return GP_OK;
}

gp_status gp_profile_stop(double *stage_ms, int64_t *calls) {
  std::lock_guard<std::mutex> lk(g_prof.mu);
  g_prof.on = false;
  double tot[GP_STAGE_COUNT] = {};
  for (const auto &c : g_prof.calls) {
    hipEvent_t *ev = &g_prof.pool[c.first];
    HIPCHK(hipEventSynchronize(ev[GP_STAGE_COUNT]));
    for (int k = 0; k < GP_STAGE_COUNT; ++k) {
      float ms = 0.f;
      if (k == GP_STAGE_ENCODE && c.second) {
        HIPCHK(hipEventElapsedTime(&ms, ev[0], ev[kProfEncEnd]));
      } else if (k == GP_STAGE_CONTRACT && c.second) {
        float early = 0.f;
        HIPCHK(hipEventElapsedTime(&early, ev[kProfEarly], ev[kProfEarly + 1]));
        HIPCHK(hipEventElapsedTime(&ms, ev[kProfLate], ev[k + 1]));
        ms += early;
      } else if (k == GP_STAGE_EPILOGUE) {
        float val = 0.f;
        HIPCHK(hipEventElapsedTime(&val, ev[kProfValEpi], ev[kProfValEpi + 1]));
        HIPCHK(hipEventElapsedTime(&ms, ev[kProfClsEpi], ev[k + 1]));
        ms += val;
      } else if (k == GP_STAGE_REFINE) {
        float blk = 0.f;
        HIPCHK(hipEventElapsedTime(&blk, ev[kProfValEpi + 1], ev[kProfValEpi + 2]));
        HIPCHK(hipEventElapsedTime(&ms, ev[k], ev[k + 1]));
        ms += blk;
      } else {
        HIPCHK(hipEventElapsedTime(&ms, ev[k], ev[k + 1]));
      }
      tot[k] += ms;
    }
  }
  if (stage_ms)
    for (int k = 0; k < GP_STAGE_COUNT; ++k) stage_ms[k] = tot[k];
  if (calls) *calls = (int64_t)g_prof.calls.size();
  g_prof.calls.clear();
  g_prof.next = 0;
  return GP_OK;
}

gp_status gp_release(void) {
  hipError_t first = hipSuccess;
  auto note = [&](hipError_t e) {
    if (first == hipSuccess && e != hipSuccess) first = e;
  };
  {
    std::lock_guard<std::mutex> lk(g_prof.mu);
    g_prof.on = false;
    for (hipEvent_t e : g_prof.pool) note(hipEventDestroy(e));
    g_prof.pool.clear();
    g_prof.calls.clear();
    g_prof.next = 0;
  }
  std::vector<void *> pinned;
  std::vector<hipStream_t> streams;
  {
    std::lock_guard<std::mutex> lk(g_owned.mu);
    pinned.swap(g_owned.pinned);
    streams.swap(g_owned.streams);
    g_owned.side.clear();
    g_owned.split.clear();
    ++g_owned.gen;
  }
  for (hipStream_t q : streams) {
    note(hipStreamSynchronize(q));
    note(hipStreamDestroy(q));
  }
  for (void *p : pinned) note(hipHostFree(p));
  if (first != hipSuccess)
    return fail(GP_E_HIP, std::string("gp_release: ") + hipGetErrorString(first));
  return GP_OK;
}

}  // extern "C"
