// C ABI of the eviction path: host-side validation, workspace sizing and dispatch to the gfx950
// kernels.  Nothing here allocates device memory, keeps state between calls or launches anything
// before every argument has been checked.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdlib>
#include <cmath>
#include <cstdint>
#include <cstring>

#include "kernels.h"
#include "kvevict.h"

namespace {

constexpr int kMaxLen = 1 << 24;
constexpr int kMaxGrid = 65535;
constexpr int kMaxCompactBudget = 8192;
constexpr float kLog2eF = 1.4426950408889634f;  // log2(e): kernels take logits in base 2
constexpr int kMaxPool = 63;  // widest max-pool window of kv_mmr_select_ex
constexpr size_t kWsAlign = 256;

size_t align_up(size_t x) { return (x + kWsAlign - 1) & ~(kWsAlign - 1); }

int elem_bytes(int dtype) { return dtype == KV_BF16 ? 2 : 4; }

bool aligned16(const void* ptr) { return (reinterpret_cast<uintptr_t>(ptr) & 15u) == 0; }

// Checks shared by every entry point; fills the launch shape.
int check_problem(const kv_problem* pr, kv::Shape* s) {
  if (!pr) return KV_ERR_NULL;
  if (pr->dtype != KV_F32 && pr->dtype != KV_BF16) return KV_ERR_DTYPE;
  if (pr->n_prob < 1 || pr->n_prob > kMaxGrid) return KV_ERR_ARG;
  if (!pr->len_host || !pr->tok_off_host || !pr->len_dev || !pr->tok_off_dev) return KV_ERR_NULL;
  if (pr->h_kv < 1 || pr->h_q < pr->h_kv || pr->h_q % pr->h_kv != 0 || pr->h_kv > kMaxGrid)
    return KV_ERR_SHAPE;
  if (pr->d != 64 && pr->d != 128) return KV_ERR_SHAPE;
  if (pr->w < 2) return KV_ERR_SHAPE;
  const int64_t rows = (int64_t)(pr->h_q / pr->h_kv) * pr->w;
  if (rows > 128) return KV_ERR_SHAPE;
  if (pr->w != 32 && rows > 64) return KV_ERR_SHAPE;
  int max_len = 0;
  for (int p = 0; p < pr->n_prob; ++p) {
    const int L = pr->len_host[p];
    if (L < pr->w + 1 || L > kMaxLen) return KV_ERR_SHAPE;
    if (pr->tok_off_host[p] < 0) return KV_ERR_SHAPE;
    if (L > max_len) max_len = L;
  }
  s->dtype = pr->dtype == KV_BF16 ? kv::kDtBf16 : kv::kDtF32;
  s->n_prob = pr->n_prob;
  s->h_q = pr->h_q;
  s->h_kv = pr->h_kv;
  s->d = pr->d;
  s->w = pr->w;
  s->max_len = max_len;
  s->lens = pr->len_dev;
  s->tok_off = pr->tok_off_dev;
  if (s->max_chunks() > kMaxGrid) return KV_ERR_SHAPE;
  return KV_OK;
}

// The uniform budget (per_problem = false), or the row stride of per-problem budgets, which may
// exceed a short problem's candidates (its own B_p is checked by check_budgets).
int check_budget(const kv_problem* pr, int32_t budget, int32_t keep_tail, bool per_problem = false) {
  if (budget < 1) return KV_ERR_BUDGET;
  for (int p = 0; p < pr->n_prob; ++p) {
    const int L = pr->len_host[p];
    if (keep_tail < 0 || keep_tail > L - 1) return KV_ERR_ARG;
    if (!per_problem && budget > L - keep_tail) return KV_ERR_BUDGET;
  }
  return KV_OK;
}

// Per-problem budgets (both arrays or neither): every B_p in [1, budget] and <= L_p - keep_tail.
int check_budgets(const kv_problem* pr, int32_t budget, int32_t keep_tail, const int32_t* b_host,
                  const int32_t* b_dev) {
  if (!b_host && !b_dev) return KV_OK;
  if (!b_host || !b_dev) return KV_ERR_NULL;
  for (int p = 0; p < pr->n_prob; ++p) {
    const int32_t b = b_host[p];
    if (b < 1 || b > budget || b > pr->len_host[p] - keep_tail) return KV_ERR_BUDGET;
  }
  return KV_OK;
}

// Largest candidate count of the batch (budget of problem p: b_host[p], or `budget`).
int max_candidates(const kv_problem* pr, int32_t budget, int32_t cand_mult, int32_t keep_tail,
                   const int32_t* b_host = nullptr) {
  int m = 0;
  for (int p = 0; p < pr->n_prob; ++p) {
    const int n_cand = pr->len_host[p] - keep_tail;
    const int64_t b = b_host ? b_host[p] : budget;
    const int64_t c = cand_mult > 0 ? std::min<int64_t>((int64_t)cand_mult * b, n_cand) : n_cand;
    if (c > m) m = (int)c;
  }
  return m;
}

int launch_status(hipError_t e) { return e == hipSuccess ? KV_OK : KV_ERR_LAUNCH; }

// Polls a workgroup of the one-launch window path makes for its unit's other segments before it
// computes their partials itself: the default, or KVEVICT_SPIN_LIMIT (0 takes that path at once).
uint32_t spin_limit() {
  const char* e = std::getenv("KVEVICT_SPIN_LIMIT");
  if (e && *e) {
    char* end = nullptr;
    const unsigned long v = std::strtoul(e, &end, 10);
    if (end && *end == '\0') return (uint32_t)std::min<unsigned long>(v, 1ul << 30);
  }
  return kv::kDefaultSpinLimit;
}

// Segment plan of the streaming window kernels for this batch.
kv::StreamPlan stream_plan_of(const kv_problem* pr, const kv::Shape& s) {
  int64_t total = 0;
  for (int p = 0; p < pr->n_prob; ++p) total += (int64_t)pr->h_kv * pr->len_host[p];
  return kv::stream_plan(s, total);
}

// Workspace of the window entry points: the larger of the chunked and the streaming layouts.
size_t window_ws_bytes(const kv_problem* pr, const kv::Shape& s) {
  size_t b = kv::window_stats_ws_bytes(s);
  if (kv::stream_shape_ok(s, 1.f)) b = std::max(b, kv::stream_ws_bytes(s, stream_plan_of(pr, s)));
  return align_up(b);
}

// Token rows that per-token arrays of the batch span (mu, sigma and the scores per kv head):
// max_p tok_off[p] + L_p, which is sum_p L_p for packed offsets.  Arrays in the workspace are
// sized by it, so offsets with gaps cannot reach past them.
int64_t token_extent(const kv_problem* pr) {
  int64_t t = 0;
  for (int p = 0; p < pr->n_prob; ++p) t = std::max<int64_t>(t, pr->tok_off_host[p] + pr->len_host[p]);
  return t;
}

// Whether kv_window_base_scores forms the scores inside the window kernel's second pass (bf16
// streaming shapes with every unit one segment), or from mu / sigma in the workspace.
bool scores_in_window_pass(const kv_problem* pr, const kv::Shape& s, float scale) {
  return kv::stream_shape_ok(s, scale) && stream_plan_of(pr, s).max_segs == 1;
}

// Workspace of kv_window_base_scores: none for the fused path (with fused_ok, for a positive
// scale), else the window paths' part and rows of mu and sigma.
size_t base_scores_ws_bytes(const kv_problem* pr, const kv::Shape& s, bool fused_ok = true) {
  if (fused_ok && scores_in_window_pass(pr, s, 1.f)) return 0;
  const size_t keys = (size_t)token_extent(pr) * pr->h_kv;
  return window_ws_bytes(pr, s) + 2 * align_up(keys * sizeof(float));
}

// Candidate lists of kv_window_candidates: one list of `stride` 8-byte entries per (problem, kv
// head).
size_t cand_lists_bytes(const kv_problem* pr, int stride) {
  return align_up((size_t)pr->n_prob * pr->h_kv * stride * sizeof(uint64_t));
}

// Whether kv_window_candidates forms the candidate lists inside the window kernel: every unit one
// segment of a streaming shape, units of at most kCandMaxLen keys, cand_mult > 0 (the caller has
// checked the candidate count against the selection's limit).
bool cands_in_window_pass(const kv_problem* pr, const kv::Shape& s, float scale, int32_t cand_mult) {
  return scores_in_window_pass(pr, s, scale) && cand_mult > 0 && s.max_len <= kv::kCandMaxLen;
}

// Workspace of kv_window_candidates: the lists and the units' normalisers, then with the fused
// path the tile codes of its first pass, without it the scores and what kv_window_base_scores needs
// after them.
size_t cand_ws_bytes(const kv_problem* pr, const kv::Shape& s, int stride, bool fused) {
  const size_t head = cand_lists_bytes(pr, stride) + align_up((size_t)pr->n_prob * pr->h_kv * sizeof(float));
  if (fused)
    return head + align_up((size_t)pr->n_prob * pr->h_kv * kv::cand_code_stride(s) * sizeof(uint32_t));
  return head + align_up((size_t)token_extent(pr) * pr->h_kv * sizeof(float)) +
         base_scores_ws_bytes(pr, s, false);
}

// Selection, and with k_out / v_out the compaction of the selected rows, in one launch; base
// scores from mu / sigma, or given (score).
// Where the selection's base scores come from: mu / sigma (with lambda1), given scores, or the
// candidate lists of kv_window_candidates; with cut_out only the candidate cut runs (lists out).
struct ScoreSource {
  const float* mu = nullptr;
  const float* sigma = nullptr;
  const float* lambda1 = nullptr;
  const float* score = nullptr;
  const uint64_t* cand_in = nullptr;
  const float* cand_in_max = nullptr;
  uint64_t* cut_out = nullptr;
  float* cut_max = nullptr;
  int list_stride = 0;
};

int mmr_select_impl(const kv_problem* pr, const ScoreSource& src, const void* k, const void* v,
                    const float* lambda2, int32_t budget,
                    int32_t cand_mult, int32_t keep_tail, const kv_select_opts* opts,
                    int32_t* sel_idx, float* sel_score, int32_t* cand_idx, float* cand_corr,
                    void* k_out, void* v_out, void* stream) {
  kv::Shape s;
  int st = check_problem(pr, &s);
  if (st != KV_OK) return st;
  if (!src.score && !src.cand_in && (!src.mu || !src.sigma || !src.lambda1)) return KV_ERR_NULL;
  if (!k || (!src.cut_out && (!lambda2 || !sel_idx))) return KV_ERR_NULL;
  if (!aligned16(k)) return KV_ERR_ARG;
  if (k_out && (!aligned16(v) || !aligned16(k_out) || !aligned16(v_out))) return KV_ERR_ARG;
  // the kernels form cand_mult * B_p in 32-bit arithmetic (B_p <= budget)
  if (cand_mult < 0 || (int64_t)cand_mult * budget > INT32_MAX) return KV_ERR_ARG;
  const int32_t pool = opts ? opts->pool : 1;
  const float w_mu = opts ? opts->w_mu : 1.f;
  const int32_t* b_host = opts ? opts->budget_host : nullptr;
  const int32_t* b_dev = opts ? opts->budget_dev : nullptr;
  if (pool < 1 || pool > kMaxPool || pool % 2 == 0 || !std::isfinite(w_mu)) return KV_ERR_ARG;
  st = check_budget(pr, budget, keep_tail, b_host != nullptr || b_dev != nullptr);
  if (st != KV_OK) return st;
  st = check_budgets(pr, budget, keep_tail, b_host, b_dev);
  if (st != KV_OK) return st;
  if (k_out && budget > kMaxCompactBudget) return KV_ERR_BUDGET;
  const int max_cand = max_candidates(pr, budget, cand_mult, keep_tail, b_host);
  if (max_cand > kv::select_max_candidates(pr->d, elem_bytes(pr->dtype))) return KV_ERR_SHAPE;
  if ((src.cand_in || src.cut_out) && pool != 1) return KV_ERR_ARG;  // lists hold unpooled scores
  kv::SelectArgs a;
  a.mu = src.mu;
  a.sigma = src.sigma;
  a.score = src.score;
  a.cand_in = src.cand_in;
  a.cand_in_max = src.cand_in_max;
  a.cut_out = src.cut_out;
  a.cut_max = src.cut_max;
  a.list_stride = src.list_stride;
  a.k = k;
  a.lambda1 = src.lambda1;
  a.lambda2 = lambda2;
  a.pool = pool;
  a.w_mu = w_mu;
  a.budget = budget;
  a.budgets = b_dev;
  a.cand_mult = cand_mult;
  a.keep_tail = keep_tail;
  a.cand_stride = kv_candidate_stride(pr, budget, cand_mult, keep_tail);
  a.max_cand = max_cand;
  a.max_cand_all = max_candidates(pr, budget, 0, keep_tail);
  a.sel_idx = sel_idx;
  a.sel_score = sel_score;
  a.cand_idx = cand_idx;
  a.cand_corr = cand_corr;
  a.v = v;
  a.k_out = k_out;
  a.v_out = v_out;
  a.out_rows = budget + keep_tail;
  if ((cand_idx || cand_corr) && a.cand_stride < 1) return KV_ERR_ARG;
  return launch_status(kv::launch_mmr_select(s, a, static_cast<hipStream_t>(stream)));
}

// kv_window_candidates; with sel (the caller has checked that the window kernel cuts the
// candidates, every C_p <= kCandSelectMax, and the selection's arguments) the selection of each
// unit follows its cut in the same launch.
int window_candidates_impl(const kv_problem* pr, const void* q_win, const void* k, float scale,
                           const float* lambda1, int32_t sigma_rows, int32_t budget,
                           int32_t cand_mult, int32_t keep_tail, const kv_select_opts* opts,
                           float* row_max, float* row_sum, void* ws, size_t ws_bytes,
                           const kv::CandSelect* sel, void* stream) {
  kv::Shape s;
  int st = check_problem(pr, &s);
  if (st != KV_OK) return st;
  if (!q_win || !k || !lambda1 || !row_max || !row_sum) return KV_ERR_NULL;
  if (!aligned16(q_win) || !aligned16(k)) return KV_ERR_ARG;
  if (!std::isfinite(scale)) return KV_ERR_ARG;
  if (sigma_rows != KV_SIGMA_GROUP_MEAN && sigma_rows != KV_SIGMA_ALL_ROWS) return KV_ERR_ARG;
  if (cand_mult < 0 || (int64_t)cand_mult * budget > INT32_MAX) return KV_ERR_ARG;
  const int32_t pool = opts ? opts->pool : 1;
  const float w_mu = opts ? opts->w_mu : 1.f;
  const int32_t* b_host = opts ? opts->budget_host : nullptr;
  const int32_t* b_dev = opts ? opts->budget_dev : nullptr;
  if (pool != 1 || !std::isfinite(w_mu)) return KV_ERR_ARG;
  st = check_budget(pr, budget, keep_tail, b_host != nullptr || b_dev != nullptr);
  if (st != KV_OK) return st;
  st = check_budgets(pr, budget, keep_tail, b_host, b_dev);
  if (st != KV_OK) return st;
  const int stride = max_candidates(pr, budget, cand_mult, keep_tail, b_host);
  if (stride > kv::select_max_candidates(pr->d, elem_bytes(pr->dtype))) return KV_ERR_SHAPE;
  const bool fused = cands_in_window_pass(pr, s, scale, cand_mult);
  const size_t need = cand_ws_bytes(pr, s, stride, fused);
  if (ws_bytes < need || !ws || (reinterpret_cast<uintptr_t>(ws) & (kWsAlign - 1)))
    return KV_ERR_WORKSPACE;
  const bool all = sigma_rows == KV_SIGMA_ALL_ROWS;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  char* base = static_cast<char*>(ws);
  const size_t n_units = (size_t)pr->n_prob * pr->h_kv;
  uint64_t* lists = reinterpret_cast<uint64_t*>(base);
  float* cmax = reinterpret_cast<float*>(base + cand_lists_bytes(pr, stride));
  const size_t head = cand_lists_bytes(pr, stride) + align_up(n_units * sizeof(float));
  if (fused)
    return launch_status(kv::launch_stream_window_cands(
        s, stream_plan_of(pr, s), q_win, k, scale, lambda1, w_mu, budget, b_dev, cand_mult,
        keep_tail, row_max, row_sum, lists, cmax, stride, reinterpret_cast<uint32_t*>(base + head),
        all, sel, hs));
  if (sel) return KV_ERR_ARG;  // the selection follows the cut only in the window kernel
  // the scores into the workspace, then the candidate cut of the selection kernel
  float* score = reinterpret_cast<float*>(base + head);
  const size_t score_bytes = align_up((size_t)token_extent(pr) * pr->h_kv * sizeof(float));
  st = kv_window_base_scores(pr, q_win, k, scale, lambda1, w_mu, sigma_rows, row_max, row_sum,
                             score, base + head + score_bytes, ws_bytes - head - score_bytes,
                             stream);
  if (st != KV_OK) return st;
  ScoreSource src;
  src.score = score;
  src.cut_out = lists;
  src.cut_max = cmax;
  src.list_stride = stride;
  return mmr_select_impl(pr, src, k, nullptr, nullptr, budget, cand_mult, keep_tail, opts, nullptr,
                         nullptr, nullptr, nullptr, nullptr, nullptr, stream);
}

}  // namespace

extern "C" {

const char* kv_strerror(int status) {
  switch (status) {
    case KV_OK: return "success";
    case KV_ERR_NULL: return "a required pointer is NULL";
    case KV_ERR_SHAPE: return "unsupported head layout, window, length or candidate count";
    case KV_ERR_DTYPE: return "unsupported dtype";
    case KV_ERR_BUDGET: return "budget outside [1, L - keep_tail]";
    case KV_ERR_WORKSPACE: return "workspace too small or misaligned";
    case KV_ERR_LAUNCH: return "HIP launch failed";
    case KV_ERR_ARG: return "invalid argument";
    case KV_ERR_SCRATCH: return "batch needs more scratch than KV_NOALLOC_SCRATCH_BYTES";
    default: return "unknown status";
  }
}

int kv_version(void) { return 1; }

size_t kv_workspace_bytes(const kv_problem* pr, int32_t budget, int32_t cand_mult,
                          int32_t keep_tail) {
  kv::Shape s;
  if (check_problem(pr, &s) != KV_OK) return 0;
  (void)budget;
  (void)cand_mult;
  (void)keep_tail;
  return window_ws_bytes(pr, s);
}

int32_t kv_candidate_stride(const kv_problem* pr, int32_t budget, int32_t cand_mult,
                            int32_t keep_tail) {
  kv::Shape s;
  if (check_problem(pr, &s) != KV_OK || cand_mult < 0 || budget < 1) return 0;
  // `budget` may be the row stride of per-problem budgets: no bound by the candidates here
  if (check_budget(pr, budget, keep_tail, true) != KV_OK) return 0;
  if (cand_mult > 0) {
    const int64_t c = (int64_t)cand_mult * budget;
    return c > INT32_MAX ? 0 : (int32_t)c;
  }
  return max_candidates(pr, budget, 0, keep_tail);
}

int kv_window_scores(const kv_problem* pr, const void* q_win, const void* k, float scale,
                     float* row_max, float* row_sum, void* ws, size_t ws_bytes, void* stream) {
  kv::Shape s;
  int st = check_problem(pr, &s);
  if (st != KV_OK) return st;
  if (!q_win || !k || !row_max || !row_sum) return KV_ERR_NULL;
  if (!aligned16(q_win) || !aligned16(k)) return KV_ERR_ARG;
  if (!std::isfinite(scale)) return KV_ERR_ARG;
  if (ws_bytes < window_ws_bytes(pr, s) || !ws ||
      (reinterpret_cast<uintptr_t>(ws) & (kWsAlign - 1)))
    return KV_ERR_WORKSPACE;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  if (kv::stream_shape_ok(s, scale)) {
    const kv::StreamPlan plan = stream_plan_of(pr, s);
    if (plan.max_segs == 1)  // one segment per unit: pass 1 writes the row statistics itself
      return launch_status(kv::launch_stream_stats(s, plan, q_win, k, scale, nullptr, row_max,
                                                   row_sum, hs));
    st = launch_status(kv::launch_stream_stats(s, plan, q_win, k, scale, ws, nullptr, nullptr, hs));
    if (st != KV_OK) return st;
    return launch_status(kv::launch_combine_partials(s, ws, plan.seg_keys, plan.max_segs,
                                                     s.group() * 32, row_max, row_sum, hs));
  }
  return launch_status(kv::launch_window_stats(s, q_win, k, scale, ws, row_max, row_sum, hs));
}

int kv_mu_sigma(const kv_problem* pr, const void* q_win, const void* k, float scale,
                const float* row_max, const float* row_sum, float* mu, float* sigma, float* attn,
                void* stream) {
  return kv_mu_sigma_ex(pr, q_win, k, scale, row_max, row_sum, KV_SIGMA_GROUP_MEAN, mu, sigma,
                        attn, stream);
}

int kv_mu_sigma_ex(const kv_problem* pr, const void* q_win, const void* k, float scale,
                   const float* row_max, const float* row_sum, int32_t sigma_rows, float* mu,
                   float* sigma, float* attn, void* stream) {
  kv::Shape s;
  int st = check_problem(pr, &s);
  if (st != KV_OK) return st;
  if (!q_win || !k || !row_max || !row_sum || !mu || !sigma) return KV_ERR_NULL;
  if (!aligned16(q_win) || !aligned16(k)) return KV_ERR_ARG;
  if (!std::isfinite(scale)) return KV_ERR_ARG;
  if (sigma_rows != KV_SIGMA_GROUP_MEAN && sigma_rows != KV_SIGMA_ALL_ROWS) return KV_ERR_ARG;
  const bool all = sigma_rows == KV_SIGMA_ALL_ROWS;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  if (kv::stream_shape_ok(s, scale) && !attn)
    return launch_status(kv::launch_stream_mu_sigma(s, stream_plan_of(pr, s), q_win, k, scale,
                                                    nullptr, row_max, row_sum, nullptr, nullptr,
                                                    mu, sigma, all, hs));
  return launch_status(kv::launch_mu_sigma(s, q_win, k, scale, row_max, row_sum, mu, sigma, attn,
                                           all, hs));
}

int kv_window_mu_sigma(const kv_problem* pr, const void* q_win, const void* k, float scale,
                       float* row_max, float* row_sum, float* mu, float* sigma, void* ws,
                       size_t ws_bytes, void* stream) {
  return kv_window_mu_sigma_ex(pr, q_win, k, scale, KV_SIGMA_GROUP_MEAN, row_max, row_sum, mu,
                               sigma, ws, ws_bytes, stream);
}

int kv_window_mu_sigma_ex(const kv_problem* pr, const void* q_win, const void* k, float scale,
                          int32_t sigma_rows, float* row_max, float* row_sum, float* mu,
                          float* sigma, void* ws, size_t ws_bytes, void* stream) {
  kv::Shape s;
  int st = check_problem(pr, &s);
  if (st != KV_OK) return st;
  if (!q_win || !k || !row_max || !row_sum || !mu || !sigma) return KV_ERR_NULL;
  if (!aligned16(q_win) || !aligned16(k)) return KV_ERR_ARG;
  if (!std::isfinite(scale)) return KV_ERR_ARG;
  if (sigma_rows != KV_SIGMA_GROUP_MEAN && sigma_rows != KV_SIGMA_ALL_ROWS) return KV_ERR_ARG;
  const bool all = sigma_rows == KV_SIGMA_ALL_ROWS;
  if (ws_bytes < window_ws_bytes(pr, s) || !ws ||
      (reinterpret_cast<uintptr_t>(ws) & (kWsAlign - 1)))
    return KV_ERR_WORKSPACE;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  if (kv::stream_shape_ok(s, scale)) {
    const kv::StreamPlan plan = stream_plan_of(pr, s);
    if (plan.max_segs == 1)  // every unit one segment: both passes of a unit in one workgroup
      return launch_status(kv::launch_stream_window(s, plan, q_win, k, scale, row_max, row_sum, mu,
                                                    sigma, all, hs));
    // several segments per unit: one cooperative launch if the grid fits the chip at once
    bool launched = false;
    st = launch_status(kv::launch_stream_window_coop(s, plan, q_win, k, scale, ws, row_max, row_sum,
                                                     mu, sigma, all, spin_limit(), hs, &launched));
    if (st != KV_OK || launched) return st;
    // segment partials, then normalisers, row statistics and mu / sigma in one more pass
    st = launch_status(kv::launch_stream_stats(s, plan, q_win, k, scale, ws, nullptr, nullptr, hs));
    if (st != KV_OK) return st;
    return launch_status(kv::launch_stream_mu_sigma(s, plan, q_win, k, scale, ws, nullptr,
                                                    nullptr, row_max, row_sum, mu, sigma, all, hs));
  }
  // other shapes: chunked row statistics, then a second pass over K
  st = launch_status(kv::launch_window_stats(s, q_win, k, scale, ws, row_max, row_sum, hs));
  if (st != KV_OK) return st;
  return launch_status(kv::launch_mu_sigma(s, q_win, k, scale, row_max, row_sum, mu, sigma,
                                           nullptr, all, hs));
}

int kv_window_mu_sigma_noalloc(const kv_problem* pr, const void* q_win, const void* k, float scale,
                               int32_t sigma_rows, float* row_max, float* row_sum, float* mu,
                               float* sigma, void* stream) {
  static_assert(KV_NOALLOC_SCRATCH_BYTES == kv::kNoAllocScratchBytes, "scratch size");
  kv::Shape s;
  const int st = check_problem(pr, &s);
  if (st != KV_OK) return st;
  if (window_ws_bytes(pr, s) > kv::kNoAllocScratchBytes) return KV_ERR_SCRATCH;
  void* ws = nullptr;
  if (!q_win || !k || !row_max || !row_sum || !mu || !sigma) return KV_ERR_NULL;
  if (kv::noalloc_scratch(&ws) != hipSuccess) return KV_ERR_LAUNCH;
  return kv_window_mu_sigma_ex(pr, q_win, k, scale, sigma_rows, row_max, row_sum, mu, sigma, ws,
                               kv::kNoAllocScratchBytes, stream);
}

size_t kv_base_scores_workspace_bytes(const kv_problem* pr) {
  kv::Shape s;
  if (check_problem(pr, &s) != KV_OK) return 0;
  return base_scores_ws_bytes(pr, s);
}

int kv_window_base_scores(const kv_problem* pr, const void* q_win, const void* k, float scale,
                          const float* lambda1, float w_mu, int32_t sigma_rows, float* row_max,
                          float* row_sum, float* score, void* ws, size_t ws_bytes, void* stream) {
  kv::Shape s;
  int st = check_problem(pr, &s);
  if (st != KV_OK) return st;
  if (!q_win || !k || !lambda1 || !row_max || !row_sum || !score) return KV_ERR_NULL;
  if (!aligned16(q_win) || !aligned16(k) || !aligned16(score)) return KV_ERR_ARG;
  if (!std::isfinite(scale) || !std::isfinite(w_mu)) return KV_ERR_ARG;
  if (sigma_rows != KV_SIGMA_GROUP_MEAN && sigma_rows != KV_SIGMA_ALL_ROWS) return KV_ERR_ARG;
  const bool fused = scores_in_window_pass(pr, s, scale);
  const size_t need = fused ? 0 : base_scores_ws_bytes(pr, s, false);
  if (need > 0 && (ws_bytes < need || !ws || (reinterpret_cast<uintptr_t>(ws) & (kWsAlign - 1))))
    return KV_ERR_WORKSPACE;
  const bool all = sigma_rows == KV_SIGMA_ALL_ROWS;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  if (fused)
    return launch_status(kv::launch_stream_window_scores(s, stream_plan_of(pr, s), q_win, k, scale,
                                                         lambda1, w_mu, row_max, row_sum, score,
                                                         all, hs));
  const size_t win = window_ws_bytes(pr, s);
  if (kv::stream_shape_ok(s, scale)) {
    // several segments per unit: the one-launch path in base-score mode when the grid fits
    const kv::ScoreMode sm{score, lambda1, w_mu};
    bool launched = false;
    st = launch_status(kv::launch_stream_window_coop(s, stream_plan_of(pr, s), q_win, k, scale, ws,
                                                     row_max, row_sum, nullptr, nullptr, all,
                                                     spin_limit(), hs, &launched, &sm));
    if (st != KV_OK || launched) return st;
  }
  // mu / sigma into the workspace after the window paths' own part, then the scores from them
  const size_t keys = (size_t)token_extent(pr) * pr->h_kv;
  float* mu = reinterpret_cast<float*>(static_cast<char*>(ws) + win);
  float* sigma = reinterpret_cast<float*>(static_cast<char*>(ws) + win + align_up(keys * sizeof(float)));
  st = kv_window_mu_sigma_ex(pr, q_win, k, scale, sigma_rows, row_max, row_sum, mu, sigma, ws, win,
                             stream);
  if (st != KV_OK) return st;
  return launch_status(kv::launch_base_scores(s, mu, sigma, lambda1, w_mu, score, hs));
}

int kv_mmr_select(const kv_problem* pr, const float* mu, const float* sigma, const void* k,
                  const float* lambda1, const float* lambda2, int32_t budget, int32_t cand_mult,
                  int32_t keep_tail, int32_t* sel_idx, float* sel_score, int32_t* cand_idx,
                  float* cand_corr, void* ws, size_t ws_bytes, void* stream) {
  return kv_mmr_select_ex(pr, mu, sigma, k, lambda1, lambda2, budget, cand_mult, keep_tail, nullptr,
                          sel_idx, sel_score, cand_idx, cand_corr, ws, ws_bytes, stream);
}

int kv_mmr_select_ex(const kv_problem* pr, const float* mu, const float* sigma, const void* k,
                     const float* lambda1, const float* lambda2, int32_t budget, int32_t cand_mult,
                     int32_t keep_tail, const kv_select_opts* opts, int32_t* sel_idx,
                     float* sel_score, int32_t* cand_idx, float* cand_corr, void* ws,
                     size_t ws_bytes, void* stream) {
  (void)ws;
  (void)ws_bytes;
  ScoreSource src;
  src.mu = mu;
  src.sigma = sigma;
  src.lambda1 = lambda1;
  return mmr_select_impl(pr, src, k, nullptr, lambda2, budget, cand_mult, keep_tail, opts, sel_idx,
                         sel_score, cand_idx, cand_corr, nullptr, nullptr, stream);
}

int kv_mmr_select_compact(const kv_problem* pr, const float* mu, const float* sigma, const void* k,
                          const void* v, const float* lambda1, const float* lambda2,
                          int32_t budget, int32_t cand_mult, int32_t keep_tail, int32_t* sel_idx,
                          void* k_out, void* v_out, void* ws, size_t ws_bytes, void* stream) {
  (void)ws;
  (void)ws_bytes;
  if (!v || !k_out || !v_out) return KV_ERR_NULL;
  ScoreSource src;
  src.mu = mu;
  src.sigma = sigma;
  src.lambda1 = lambda1;
  return mmr_select_impl(pr, src, k, v, lambda2, budget, cand_mult, keep_tail, nullptr, sel_idx,
                         nullptr, nullptr, nullptr, k_out, v_out, stream);
}

int kv_mmr_select_scored(const kv_problem* pr, const float* score, const void* k, const void* v,
                         const float* lambda2, int32_t budget,
                         int32_t cand_mult, int32_t keep_tail, const kv_select_opts* opts,
                         int32_t* sel_idx, float* sel_score, int32_t* cand_idx, float* cand_corr,
                         void* k_out, void* v_out, void* stream) {
  if (!score) return KV_ERR_NULL;
  if (!aligned16(score)) return KV_ERR_ARG;
  if ((k_out != nullptr) != (v_out != nullptr)) return KV_ERR_NULL;
  if (k_out && !v) return KV_ERR_NULL;
  ScoreSource src;
  src.score = score;
  return mmr_select_impl(pr, src, k, v, lambda2, budget, cand_mult, keep_tail, opts, sel_idx,
                         sel_score, cand_idx, cand_corr, k_out, v_out, stream);
}

size_t kv_candidates_workspace_bytes(const kv_problem* pr, int32_t budget, int32_t cand_mult,
                                     int32_t keep_tail, const kv_select_opts* opts) {
  kv::Shape s;
  if (check_problem(pr, &s) != KV_OK) return 0;
  const int32_t* b_host = opts ? opts->budget_host : nullptr;
  if (cand_mult < 0 || budget < 1 || check_budget(pr, budget, keep_tail, b_host != nullptr) != KV_OK)
    return 0;
  if (opts && opts->pool != 1) return 0;
  const int stride = max_candidates(pr, budget, cand_mult, keep_tail, b_host);
  if (stride > kv::select_max_candidates(pr->d, elem_bytes(pr->dtype))) return 0;
  return cand_ws_bytes(pr, s, stride, cands_in_window_pass(pr, s, 1.f, cand_mult));
}

int kv_window_candidates(const kv_problem* pr, const void* q_win, const void* k, float scale,
                         const float* lambda1, int32_t sigma_rows, int32_t budget,
                         int32_t cand_mult, int32_t keep_tail, const kv_select_opts* opts,
                         float* row_max, float* row_sum, void* ws, size_t ws_bytes, void* stream) {
  return window_candidates_impl(pr, q_win, k, scale, lambda1, sigma_rows, budget, cand_mult,
                                keep_tail, opts, row_max, row_sum, ws, ws_bytes, nullptr, stream);
}

int kv_mmr_select_candidates(const kv_problem* pr, const void* ws, size_t ws_bytes, const void* k,
                             const void* v, const float* lambda2, int32_t budget,
                             int32_t cand_mult, int32_t keep_tail, const kv_select_opts* opts,
                             int32_t* sel_idx, float* sel_score, int32_t* cand_idx,
                             float* cand_corr, void* k_out, void* v_out, void* stream) {
  kv::Shape s;
  int st = check_problem(pr, &s);
  if (st != KV_OK) return st;
  if ((k_out != nullptr) != (v_out != nullptr)) return KV_ERR_NULL;
  if (k_out && !v) return KV_ERR_NULL;
  if (cand_mult < 0) return KV_ERR_ARG;
  const int32_t* b_host = opts ? opts->budget_host : nullptr;
  st = check_budget(pr, budget, keep_tail, b_host != nullptr);
  if (st != KV_OK) return st;
  const int stride = max_candidates(pr, budget, cand_mult, keep_tail, b_host);
  const size_t lists = cand_lists_bytes(pr, stride);
  if (ws_bytes < lists + align_up((size_t)pr->n_prob * pr->h_kv * sizeof(float)) || !ws ||
      (reinterpret_cast<uintptr_t>(ws) & (kWsAlign - 1)))
    return KV_ERR_WORKSPACE;
  ScoreSource src;
  src.cand_in = static_cast<const uint64_t*>(ws);
  src.cand_in_max = reinterpret_cast<const float*>(static_cast<const char*>(ws) + lists);
  src.list_stride = stride;
  return mmr_select_impl(pr, src, k, v, lambda2, budget, cand_mult, keep_tail, opts, sel_idx,
                         sel_score, cand_idx, cand_corr, k_out, v_out, stream);
}

int kv_evict_pass(const kv_problem* pr, const void* q_win, const void* k, const void* v,
                  float scale, const float* lambda1, const float* lambda2, int32_t sigma_rows,
                  int32_t budget, int32_t cand_mult, int32_t keep_tail, const kv_select_opts* opts,
                  float* row_max, float* row_sum, int32_t* sel_idx, float* sel_score, void* k_out,
                  void* v_out, void* ws, size_t ws_bytes, void* stream) {
  kv::Shape s;
  int st = check_problem(pr, &s);
  if (st != KV_OK) return st;
  // the selection's own checks first: nothing runs unless both calls would
  if (!lambda2 || !sel_idx) return KV_ERR_NULL;
  if ((k_out != nullptr) != (v_out != nullptr)) return KV_ERR_NULL;
  if (k_out && !v) return KV_ERR_NULL;
  if (k_out && (!aligned16(v) || !aligned16(k_out) || !aligned16(v_out))) return KV_ERR_ARG;
  if (k_out && budget > kMaxCompactBudget) return KV_ERR_BUDGET;
  if (cand_mult < 0 || (int64_t)cand_mult * budget > INT32_MAX) return KV_ERR_ARG;
  const int32_t* b_host = opts ? opts->budget_host : nullptr;
  const int32_t* b_dev = opts ? opts->budget_dev : nullptr;
  st = check_budget(pr, budget, keep_tail, b_host != nullptr || b_dev != nullptr);
  if (st != KV_OK) return st;
  const int stride = max_candidates(pr, budget, cand_mult, keep_tail, b_host);
  if (pr->dtype == KV_BF16 && cands_in_window_pass(pr, s, scale, cand_mult) &&
      stride <= kv::kCandSelectMax) {
    kv::CandSelect sel{lambda2, sel_idx, sel_score, v, k_out, v_out, budget + keep_tail};
    return window_candidates_impl(pr, q_win, k, scale, lambda1, sigma_rows, budget, cand_mult,
                                  keep_tail, opts, row_max, row_sum, ws, ws_bytes, &sel, stream);
  }
  st = kv_window_candidates(pr, q_win, k, scale, lambda1, sigma_rows, budget, cand_mult,
                            keep_tail, opts, row_max, row_sum, ws, ws_bytes, stream);
  if (st != KV_OK) return st;
  return kv_mmr_select_candidates(pr, ws, ws_bytes, k, v, lambda2, budget, cand_mult, keep_tail,
                                  opts, sel_idx, sel_score, nullptr, nullptr, k_out, v_out, stream);
}

int kv_compact_cache(const kv_problem* pr, const void* k, const void* v, const int32_t* sel_idx,
                     int32_t budget, int32_t keep_tail, void* k_out, void* v_out, void* stream) {
  return kv_compact_cache_ex(pr, k, v, sel_idx, budget, keep_tail, nullptr, nullptr, 0, k_out,
                             v_out, stream);
}

int kv_compact_cache_ex(const kv_problem* pr, const void* k, const void* v,
                        const int32_t* sel_idx, int32_t budget, int32_t keep_tail,
                        const int32_t* budget_host, const int32_t* budget_dev, int32_t out_rows,
                        void* k_out, void* v_out, void* stream) {
  kv::Shape s;
  int st = check_problem(pr, &s);
  if (st != KV_OK) return st;
  if (!k || !v || !sel_idx || !k_out || !v_out) return KV_ERR_NULL;
  if (!aligned16(k) || !aligned16(v) || !aligned16(k_out) || !aligned16(v_out)) return KV_ERR_ARG;
  st = check_budget(pr, budget, keep_tail, budget_host != nullptr || budget_dev != nullptr);
  if (st != KV_OK) return st;
  st = check_budgets(pr, budget, keep_tail, budget_host, budget_dev);
  if (st != KV_OK) return st;
  if (budget > kMaxCompactBudget) return KV_ERR_BUDGET;
  if (out_rows == 0) out_rows = budget + keep_tail;
  if (out_rows < budget + keep_tail) return KV_ERR_ARG;
  return launch_status(kv::launch_compact(s, k, v, sel_idx, budget, budget_dev, keep_tail,
                                          out_rows, k_out, v_out,
                                          static_cast<hipStream_t>(stream)));
}

namespace {

int check_cache_batch(const kv_cache_batch* cb) {
  if (!cb) return KV_ERR_NULL;
  if (cb->dtype != KV_F32 && cb->dtype != KV_BF16) return KV_ERR_DTYPE;
  if (cb->n_prob < 1 || cb->n_prob > kMaxGrid) return KV_ERR_ARG;
  if (!cb->len_host || !cb->len_dev) return KV_ERR_NULL;
  if (cb->h_kv < 1 || cb->h_kv > kMaxGrid || cb->h_q < cb->h_kv || cb->h_q % cb->h_kv != 0 ||
      cb->h_q / cb->h_kv > 8)
    return KV_ERR_SHAPE;
  if (cb->d != 64 && cb->d != 128) return KV_ERR_SHAPE;
  if (cb->row_stride < 1 || cb->row_stride > kMaxLen) return KV_ERR_SHAPE;
  for (int p = 0; p < cb->n_prob; ++p)
    if (cb->len_host[p] < 0 || cb->len_host[p] > cb->row_stride) return KV_ERR_SHAPE;
  return KV_OK;
}

kv::DecodePlan decode_plan_of(const kv_cache_batch* cb) {
  int max_len = 0;
  for (int p = 0; p < cb->n_prob; ++p) max_len = std::max(max_len, (int)cb->len_host[p]);
  return kv::decode_plan(cb->n_prob, cb->h_kv, max_len);
}

}  // namespace

size_t kv_decode_workspace_bytes(const kv_cache_batch* cb) {
  if (check_cache_batch(cb) != KV_OK) return 0;
  return align_up(kv::decode_ws_bytes(cb->n_prob, cb->h_q, cb->d, decode_plan_of(cb)));
}

int kv_decode_attention(const kv_cache_batch* cb, const void* q, void* k_cache, void* v_cache,
                        const void* k_new, const void* v_new, float scale, float* out, void* ws,
                        size_t ws_bytes, void* stream) {
  int st = check_cache_batch(cb);
  if (st != KV_OK) return st;
  if (!q || !k_cache || !v_cache || !out) return KV_ERR_NULL;
  if ((k_new == nullptr) != (v_new == nullptr)) return KV_ERR_NULL;
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) ||
      (k_new && (!aligned16(k_new) || !aligned16(v_new))))
    return KV_ERR_ARG;
  if (!std::isfinite(scale)) return KV_ERR_ARG;
  for (int p = 0; p < cb->n_prob; ++p) {
    const int len = cb->len_host[p];
    if (k_new ? len >= cb->row_stride : len < 1) return KV_ERR_SHAPE;
  }
  const kv::DecodePlan plan = decode_plan_of(cb);
  if (plan.n_split > kMaxGrid) return KV_ERR_SHAPE;
  const size_t need = align_up(kv::decode_ws_bytes(cb->n_prob, cb->h_q, cb->d, plan));
  if (need > 0 && (ws_bytes < need || !ws || (reinterpret_cast<uintptr_t>(ws) & (kWsAlign - 1))))
    return KV_ERR_WORKSPACE;
  kv::DecodeArgs a;
  a.q = q;
  a.k = k_cache;
  a.v = v_cache;
  a.k_new = k_new;
  a.v_new = v_new;
  a.lens = cb->len_dev;
  a.h_q = cb->h_q;
  a.h_kv = cb->h_kv;
  a.row_stride = cb->row_stride;
  a.c = scale * kLog2eF;
  a.split_rows = plan.split_rows;
  a.n_split = plan.n_split;
  a.out = out;
  a.part = static_cast<float*>(ws);
  return launch_status(kv::launch_decode(cb->dtype == KV_BF16 ? kv::kDtBf16 : kv::kDtF32, cb->d,
                                         cb->n_prob, a, static_cast<hipStream_t>(stream)));
}

int kv_pyramid_budgets(int32_t budget, int32_t n_layers, double beta, int32_t* budgets_host) {
  if (!budgets_host) return KV_ERR_NULL;
  if (budget < 1 || n_layers < 1 || !(beta >= 1.0) || !std::isfinite(beta)) return KV_ERR_ARG;
  if (n_layers == 1) {
    budgets_host[0] = budget;
    return KV_OK;
  }
  const int64_t b_min = std::max<int64_t>(1, (int64_t)std::floor((double)budget / beta));
  const int64_t b_max = 2 * (int64_t)budget - b_min, span = b_max - b_min, n1 = n_layers - 1;
  for (int64_t l = 0; l < n_layers; ++l) {
    // the linear budget of layer l rounded away from `budget`; layers l and n-1-l sum to 2 budget
    int64_t b;
    if (2 * l < n1) b = b_max - (l * span) / n1;
    else if (2 * l == n1) b = budget;
    else b = b_min + ((n1 - l) * span) / n1;
    budgets_host[l] = (int32_t)b;
  }
  return KV_OK;
}

int kv_depth_profile(int32_t family, const double* params_host, int32_t n_params,
                     int32_t n_layers, float* lambda_out_host) {
  if (!params_host || !lambda_out_host) return KV_ERR_NULL;
  if (n_layers < 1) return KV_ERR_ARG;
  switch (family) {
    case KV_PROFILE_GLOBAL:
      if (n_params != 1) return KV_ERR_ARG;
      break;
    case KV_PROFILE_SEGMENTS:
      if (n_params < 1 || n_params > n_layers) return KV_ERR_ARG;
      break;
    case KV_PROFILE_CURVE:
      if (n_params != 3) return KV_ERR_ARG;
      break;
    default:
      return KV_ERR_ARG;
  }
  for (int l = 0; l < n_layers; ++l) {
    double a;
    if (family == KV_PROFILE_GLOBAL) {
      a = params_host[0];
    } else if (family == KV_PROFILE_SEGMENTS) {
      a = params_host[((int64_t)n_params * l) / n_layers];
    } else {
      const double t = n_layers == 1 ? 0.0 : (double)l / (double)(n_layers - 1);
      a = params_host[0] + params_host[1] * t + params_host[2] * t * t;
    }
    lambda_out_host[l] = (float)std::sinh(a);
  }
  return KV_OK;
}

}  // extern "C"
