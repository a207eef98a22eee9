// Host-side launchers of the gfx950 kernels.  Arguments are validated by the C ABI layer before
// any of these is called; every launcher only enqueues work on `stream` and reports launch errors.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace kv {

constexpr int kDtF32 = 0;
constexpr int kDtBf16 = 1;

// Keys per work item of the window kernels (a multiple of 4 waves x 32 keys).
constexpr int kWindowChunk = 1024;

struct Shape {
  int dtype;  // 0 = fp32, 1 = bf16
  int n_prob, h_q, h_kv, d, w;
  int max_len;                 // max_p L_p
  const int32_t* lens;         // device [n_prob]
  const int64_t* tok_off;      // device [n_prob]
  int group() const { return h_q / h_kv; }
  int rows() const { return group() * w; }
  int row_blocks() const { return rows() <= 32 ? 1 : (rows() <= 64 ? 2 : 4); }
  int max_chunks() const { return (max_len + kWindowChunk - 1) / kWindowChunk; }
};

// Workspace bytes of the split-L row statistics.
size_t window_stats_ws_bytes(const Shape& s);

hipError_t launch_window_stats(const Shape& s, const void* q_win, const void* k, float scale,
                               void* ws, float* row_max, float* row_sum, hipStream_t stream);

hipError_t launch_mu_sigma(const Shape& s, const void* q_win, const void* k, float scale,
                           const float* row_max, const float* row_sum, float* mu, float* sigma,
                           float* attn, bool sigma_all, hipStream_t stream);

// Streaming two-pass row statistics + mu/sigma (bf16, w = 32, G in {1, 2, 4}, scale > 0): every
// unit is cut
// into segments of seg_keys keys (a multiple of 256), one workgroup each, sized so that a batch
// fills the chip about once; the segment partials (m, z) per window row live in the workspace,
// [n_units][max_segs][32 G] float2.
struct StreamPlan {
  int seg_keys;
  int max_segs;
};
bool stream_shape_ok(const Shape& s, float scale);
StreamPlan stream_plan(const Shape& s, int64_t total_keys);  // total_keys = sum_p h_kv L_p
size_t stream_ws_bytes(const Shape& s, const StreamPlan& plan);
size_t stream_counter_offset(const Shape& s, const StreamPlan& plan);  // counters after the partials
// Pass 1: segment partials into ws or, with ws == nullptr (only when plan.max_segs == 1), the
// row statistics into row_max / row_sum.
hipError_t launch_stream_stats(const Shape& s, const StreamPlan& plan, const void* q_win,
                               const void* k, float scale, void* ws, float* row_max,
                               float* row_sum, hipStream_t stream);
// Pass 2: normalisers from the partials in ws (then also row_max_out / row_sum_out), or, with
// ws == nullptr, from row_max_in / row_sum_in; mu / sigma out.
hipError_t launch_stream_mu_sigma(const Shape& s, const StreamPlan& plan, const void* q_win,
                                  const void* k, float scale, const void* ws,
                                  const float* row_max_in, const float* row_sum_in,
                                  float* row_max_out, float* row_sum_out, float* mu, float* sigma,
                                  bool sigma_all, hipStream_t stream);
// Both passes in one launch when every unit is one segment (plan.max_segs == 1): row_max /
// row_sum and mu / sigma out, no workspace.
hipError_t launch_stream_window(const Shape& s, const StreamPlan& plan, const void* q_win,
                                const void* k, float scale, float* row_max, float* row_sum,
                                float* mu, float* sigma, bool sigma_all, hipStream_t stream);
// Both passes in one launch, every unit one segment, in base-score mode: row_max / row_sum, and
// per key s = fma(lambda1[p], sigma, w_mu mu) into score instead of mu / sigma.
hipError_t launch_stream_window_scores(const Shape& s, const StreamPlan& plan, const void* q_win,
                                       const void* k, float scale, const float* lambda1,
                                       float w_mu, float* row_max, float* row_sum, float* score,
                                       bool sigma_all, hipStream_t stream);
// Window statistics and the candidate set in one launch, every unit one segment (candidate mode,
// stream_prune.hip): row_max / row_sum, and per unit the candidate list [n_units][cand_stride] of
// (order key of the score, position) entries packed as key << 32 | (0xFFFFFFFF - position): the
// unit's C_p best entries in ascending position order, then zeros; and cand_max [n_units], the
// largest base score over the candidate positions clamped at 1e-12.  The
// keys are read once in full; the second pass revisits only the tiles whose score bound reaches
// the unit's cut.  codes: scratch of n_units * cand_code_stride(s) words (the first pass's tile
// codes, then the evaluated keys' scores).  Units of at most kCandMaxLen keys.
// With sel, each unit's workgroup then runs the selection on its list (every C_p <= 256, bf16): the
// greedy of the selection kernel's Gram path, with sel_idx / sel_score ([n_prob][h_kv][budget],
// sel_score nullable) and, with k_out, the compaction (k_out / v_out [n_prob][h_kv][out_rows][D],
// both or neither, v required) as the selection kernel writes them from the same list.
constexpr int kCandMaxLen = 32768;
constexpr int kCandSelectMax = 256;  // candidates per unit of the selection in the window launch
struct CandSelect {
  const float* lambda2;
  int32_t* sel_idx;
  float* sel_score;
  const void* v;
  void* k_out;
  void* v_out;
  int out_rows;
};
int cand_code_stride(const Shape& s);
hipError_t launch_stream_window_cands(const Shape& s, const StreamPlan& plan, const void* q_win,
                                      const void* k, float scale, const float* lambda1, float w_mu,
                                      int budget, const int32_t* budgets, int cand_mult,
                                      int keep_tail, float* row_max, float* row_sum,
                                      uint64_t* cand_out, float* cand_max, int cand_stride,
                                      uint32_t* codes, bool sigma_all, const CandSelect* sel,
                                      hipStream_t stream);
// Base scores s = fma(lambda1[p], sigma, w_mu mu) of every key from mu / sigma rows (for batches
// that take the other window paths).
hipError_t launch_base_scores(const Shape& s, const float* mu, const float* sigma,
                              const float* lambda1, float w_mu, float* score, hipStream_t stream);
// Both passes in one launch when units span several segments: partials and per-unit arrival
// counters in ws; a workgroup polls at most spin_limit times for its unit's other segments before
// it computes their partials itself.  Sets *launched = false (and launches nothing) if the grid
// does not fit the chip at once; the caller then takes the two-launch path.
// With sm (base-score mode) the second pass stores scores instead of mu / sigma.
struct ScoreMode {
  float* score;
  const float* lambda1;
  float w_mu;
};
hipError_t launch_stream_window_coop(const Shape& s, const StreamPlan& plan, const void* q_win,
                                     const void* k, float scale, void* ws, float* row_max,
                                     float* row_sum, float* mu, float* sigma, bool sigma_all,
                                     uint32_t spin_limit, hipStream_t stream, bool* launched,
                                     const ScoreMode* sm = nullptr);
constexpr uint32_t kDefaultSpinLimit = 4096;  // polls (each a device-coherent load and a short sleep)
// row_max / row_sum from chunk partials [n_units][max_chunks][rows_pad] of chunk_keys keys each.
hipError_t launch_combine_partials(const Shape& s, const void* part, int chunk_keys,
                                   int max_chunks, int rows_pad, float* row_max, float* row_sum,
                                   hipStream_t stream);

struct SelectArgs {
  const float* mu;
  const float* sigma;
  // base scores given instead of mu / sigma (then lambda1 and w_mu are unused)
  const float* score = nullptr;
  // a candidate list given instead (cand_in, cand_in_max: as launch_stream_window_cands writes
  // them, list_stride entries per unit; no pooling), or, with cut_out, only the candidate cut:
  // each unit's C candidates in the same form and its normaliser into cut_max
  const uint64_t* cand_in = nullptr;
  const float* cand_in_max = nullptr;
  uint64_t* cut_out = nullptr;
  float* cut_max = nullptr;
  int list_stride = 0;
  const void* k;
  const float* lambda1;
  const float* lambda2;
  int pool;     // odd max-pool window over the candidate positions (1: none)
  float w_mu;   // weight of mu in the base score (1: the paper's score)
  int budget, cand_mult, keep_tail, cand_stride, max_cand;
  const int32_t* budgets;  // per-problem budgets (device, nullable): B_p <= budget, the row stride
  int max_cand_all;  // max_p (L_p - keep_tail): every position that competes for a candidate slot
  int32_t* sel_idx;
  float* sel_score;
  int32_t* cand_idx;
  float* cand_corr;
  // optional compaction after the selection (k_out == nullptr: none): K, V rows of the admitted
  // positions in position order, then the last keep_tail rows, into blocks of out_rows rows
  const void* v = nullptr;
  void* k_out = nullptr;
  void* v_out = nullptr;
  int out_rows = 0;
};

// Largest supported candidate count for a head dimension / element size.
int select_max_candidates(int d, int elem_bytes);

hipError_t launch_mmr_select(const Shape& s, const SelectArgs& a, hipStream_t stream);

hipError_t launch_compact(const Shape& s, const void* k, const void* v, const int32_t* sel_idx,
                          int budget, const int32_t* budgets, int keep_tail, int out_rows,
                          void* k_out, void* v_out, hipStream_t stream);

// The static scratch of the entry point that allocates nothing (noalloc.hip): its device address
// on the current device, looked up on the first call per device.
constexpr size_t kNoAllocScratchBytes = (size_t)16 << 20;
hipError_t noalloc_scratch(void** ptr);

// Decode attention over a compacted cache (decode.hip).
struct DecodeArgs {
  const void* q;      // [n_prob][h_q][d]
  void* k;            // [n_prob][h_kv][row_stride][d]; row len_p is written when k_new is set
  void* v;
  const void* k_new;  // [n_prob][h_kv][d] or null
  const void* v_new;
  const int32_t* lens;
  int h_q, h_kv, row_stride;
  float c;            // softmax scale * log2(e)
  int split_rows, n_split;
  float* out;         // [n_prob][h_q][d]
  float* part;        // [n_prob][h_q][n_split][d + 2] when n_split > 1
};
struct DecodePlan {
  int n_split, split_rows;
};
DecodePlan decode_plan(int n_prob, int h_kv, int max_len);
size_t decode_ws_bytes(int n_prob, int h_q, int d, const DecodePlan& plan);
hipError_t launch_decode(int dtype, int d, int n_prob, const DecodeArgs& a, hipStream_t stream);

}  // namespace kv
