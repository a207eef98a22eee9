/*
 * kvevict.h -- C ABI of the diversity-aware, layer-wise KV-cache eviction path on AMD Instinct
 * MI355X (gfx950).
 *
 * Method: "Beyond Mean Attention: Diversity-Aware, Layer-Wise Scoring for KV Cache Eviction".
 * After prefill, for every layer and kv head, the last W queries (the observation window) attend to
 * all L cached keys (section 3.1).  Each cached token i gets its mean attention mu_i (Eq. (1)) and
 * its sample dispersion sigma_i over the window queries (Eq. (3)).  B tokens are then admitted
 * greedily under s~_i + lambda2 corr(i, S), where s~ is the per-head normalised base score
 * s_i = mu_i + lambda1 sigma_i and corr(i, S) the clamped maximum cosine of key i to the admitted
 * keys (Eq. (2), (4), (5)); candidates are restricted to the top 4B base scores.  The per-layer
 * coefficients come from a depth profile (section 3.3, Eq. (6)).  Finally the kept rows of K and V
 * are compacted.
 *
 * Conventions shared by every entry point
 *   - A "problem" is one layer of one sequence.  A batch holds n_prob problems; problem p has
 *     context length L_p and its keys/values start at packed token offset tok_off[p].
 *   - Every tensor pointer is a caller-owned DEVICE pointer unless its name ends in _host.  The
 *     library never allocates or frees device memory; scratch comes from the caller's workspace
 *     (kv_window_mu_sigma_noalloc: from a static device array of the library instead).
 *   - Calls are asynchronous: after host-side validation they enqueue kernels on `stream` (a
 *     hipStream_t passed as void*, NULL = default stream) and return.  Device faults surface at the
 *     caller's next synchronisation.
 *   - On invalid arguments a call returns a negative KV_ERR_* code and launches nothing.  A launch
 *     failure returns KV_ERR_LAUNCH (work enqueued before the failing launch may still run).
 *   - Calls on one stream are ordered; calls that share output or workspace buffers must not run
 *     concurrently on different streams.
 *
 * Layouts (row-major; e = element size: 4 for KV_F32, 2 for KV_BF16 = raw bfloat16 bits)
 *   q_win   [n_prob][h_q][w][d]         window queries (positions L_p-w .. L_p-1); q-head h uses
 *                                       kv-head h / (h_q / h_kv)
 *   k, v    problem p at element offset tok_off[p]*h_kv*d, layout [h_kv][L_p][d] (keys after RoPE)
 *   row_max, row_sum  [n_prob][h_q][w]  fp32
 *   mu, sigma  problem p at tok_off[p]*h_kv, layout [h_kv][L_p], fp32
 *   attn    problem p at tok_off[p]*h_q*w, layout [h_q][w][L_p], fp32
 *   lambda1, lambda2  [n_prob] fp32
 *   sel_idx, sel_score [n_prob][h_kv][budget]
 *   cand_idx, cand_corr [n_prob][h_kv][cand_stride], cand_stride from kv_candidate_stride()
 *   k_out, v_out [n_prob][h_kv][budget + keep_tail][d], same dtype as k and v
 *
 * Supported shapes: d in {64, 128}; 2 <= w; h_q % h_kv == 0; G*w <= 128 with G = h_q / h_kv;
 * L_p >= w + 1 and L_p <= 2^24; 1 <= budget <= L_p - keep_tail (with per-problem budgets B_p,
 * each B_p <= L_p - keep_tail and `budget` only bounds them as the row stride); keep_tail in
 * [0, L_p - 1].
 */
#ifndef KVEVICT_H
#define KVEVICT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ---------------------------------------------------------------------------- */
#define KV_OK 0
#define KV_ERR_NULL (-1)      /* a required pointer is NULL                                     */
#define KV_ERR_SHAPE (-2)     /* head layout, window, length or candidate count not supported   */
#define KV_ERR_DTYPE (-3)     /* dtype is neither KV_F32 nor KV_BF16                            */
#define KV_ERR_BUDGET (-4)    /* budget < 1 or budget > L_p - keep_tail for some problem        */
#define KV_ERR_WORKSPACE (-5) /* workspace smaller than kv_workspace_bytes() asks for           */
#define KV_ERR_LAUNCH (-6)    /* a HIP launch or device query failed                            */
#define KV_ERR_ARG (-7)       /* any other invalid argument (n_prob, profile family, params)    */
#define KV_ERR_SCRATCH (-8)   /* the batch needs more than KV_NOALLOC_SCRATCH_BYTES of scratch  */

/* ---- element types --------------------------------------------------------------------------- */
#define KV_F32 0
#define KV_BF16 1

/* ---- depth-profile families (section 3.3) ----------------------------------------------------- */
#define KV_PROFILE_GLOBAL 0   /* a(l) = a0                                   (1 parameter)      */
#define KV_PROFILE_SEGMENTS 1 /* a(l) = a[floor(n_seg * l / n_layers)]       (n_seg parameters) */
#define KV_PROFILE_CURVE 2    /* a(l) = c0 + c1 t + c2 t^2, t = l/(n_layers-1) (3 parameters)   */

/* Shape of a batch of problems.  len_host/tok_off_host drive validation and grid sizing; the
 * kernels read len_dev/tok_off_dev, which must hold the same values. */
typedef struct kv_problem {
  int32_t dtype;  /* KV_F32 or KV_BF16 (q_win, k and v share it)                             */
  int32_t n_prob; /* number of problems, >= 1                                                */
  int32_t h_q;    /* query heads                                                             */
  int32_t h_kv;   /* key/value heads                                                         */
  int32_t d;      /* head dimension                                                          */
  int32_t w;      /* observation-window size |W|                                             */
  const int32_t* len_host;     /* [n_prob] context lengths (host)                              */
  const int64_t* tok_off_host; /* [n_prob] packed token offsets (host)                         */
  const int32_t* len_dev;      /* [n_prob] same lengths (device)                               */
  const int64_t* tok_off_dev;  /* [n_prob] same offsets (device)                               */
} kv_problem;

/* Human-readable text of a status code (static storage, never NULL). */
const char* kv_strerror(int status);

/* ABI version, currently 1. */
int kv_version(void);

/* Bytes of device workspace the calls below need for this batch (kv_window_scores and
 * kv_window_mu_sigma; kv_mmr_select, kv_mmr_select_ex and kv_mmr_select_compact take a workspace
 * argument but stage everything in on-chip memory, and kv_mu_sigma and kv_compact_cache need
 * none).  Returns 0 for invalid arguments.  The workspace must be 256-byte aligned; its contents
 * need no initialisation and are not preserved between calls. */
size_t kv_workspace_bytes(const kv_problem* pr, int32_t budget, int32_t cand_mult,
                          int32_t keep_tail);

/* Row stride of cand_idx / cand_corr: cand_mult * budget, or the largest candidate count
 * max_p(L_p - keep_tail) when cand_mult == 0.  Returns 0 for invalid arguments. */
int32_t kv_candidate_stride(const kv_problem* pr, int32_t budget, int32_t cand_mult,
                            int32_t keep_tail);

/* Observation-window logits and row-softmax statistics (section 3.1).
 * For every problem p, q-head h and window row r (absolute position L_p - w + r), over the keys
 * i <= L_p - w + r of kv-head h / G (causal mask), with l_i = scale * <q[p,h,r], k[p,g,i]>:
 *   row_max[p,h,r] = max_i l_i,   row_sum[p,h,r] = sum_i exp(l_i - row_max[p,h,r]).
 * scale is the softmax scale (1/sqrt(d) for scaled dot-product attention).  Logits are computed
 * from the stored inputs with fp32 accumulation and never leave the chip.  Needs workspace. */
int kv_window_scores(const kv_problem* pr, const void* q_win, const void* k, float scale,
                     float* row_max, float* row_sum, void* ws, size_t ws_bytes, void* stream);

/* Per-token mean and dispersion of the window attention (Eq. (1), Eq. (3)).
 * A[p,h,r,i] = exp(l - row_max) / row_sum (0 where masked), from the statistics of
 * kv_window_scores.  The G query heads that share a kv head are averaged,
 * a[r,i] = mean_h A[h,r,i]; then mu[i] = mean_r a[r,i] and
 * sigma[i] = sqrt(sum_r (a[r,i] - mu[i])^2 / (w - 1)), for every position i < L_p.
 * attn (nullable) receives A itself.  All fp32.  Needs no workspace. */
int kv_mu_sigma(const kv_problem* pr, const void* q_win, const void* k, float scale,
                const float* row_max, const float* row_sum, float* mu, float* sigma,
                float* attn, void* stream);

/* kv_window_scores followed by kv_mu_sigma (without attn): same results in one call.  The
 * normalisers go from the first pass to the second without a round trip through row_max /
 * row_sum: inside one workgroup when a batch is large enough for every (problem, kv head) to be
 * scored by one workgroup, else through the workspace (in one launch when the batch fits the chip
 * at once; a workgroup then polls the workspace for the other segments of its (problem, kv head)
 * and, if they are late, computes their partials itself; the environment variable
 * KVEVICT_SPIN_LIMIT sets the number of polls, 0 taking that path at once).  Needs workspace
 * (always validated); calls that overlap on one workspace race. */
int kv_window_mu_sigma(const kv_problem* pr, const void* q_win, const void* k, float scale,
                       float* row_max, float* row_sum, float* mu, float* sigma, void* ws,
                       size_t ws_bytes, void* stream);

/* kv_window_mu_sigma_ex for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): same arguments without the
 * workspace, same kernels, same results bit for bit.  The library's own static scratch of
 * KV_NOALLOC_SCRATCH_BYTES per GPU (held from the first call on that GPU until the process ends)
 * takes the workspace's place; nothing is allocated or freed, by the library or any routine it
 * calls.  A batch whose workspace (kv_workspace_bytes) exceeds it returns KV_ERR_SCRATCH and
 * launches nothing.  Every call on one GPU shares that GPU's scratch: calls that overlap on one GPU
 * (on different streams, or from different threads) race, and must be ordered by the caller. */
#define KV_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)
int kv_window_mu_sigma_noalloc(const kv_problem* pr, const void* q_win, const void* k, float scale,
                               int32_t sigma_rows, float* row_max, float* row_sum, float* mu,
                               float* sigma, void* stream);

/* Which window values the dispersion sigma of kv_mu_sigma_ex / kv_window_mu_sigma_ex runs over.
 * The paper defines Eq. (3) for one attention head and does not say how the G query heads that
 * share a kv head enter it:
 *   KV_SIGMA_GROUP_MEAN: the w rows of the group-mean attention a[r,i] = mean_h A[h,r,i], divisor
 *     w - 1 (the reading kv_mu_sigma and kv_window_mu_sigma use);
 *   KV_SIGMA_ALL_ROWS: all G w values A[h,r,i] of the group, divisor G w - 1.
 * mu is the same under both; for G = 1 so is sigma. */
#define KV_SIGMA_GROUP_MEAN 0
#define KV_SIGMA_ALL_ROWS 1

/* kv_mu_sigma with the dispersion taken over `sigma_rows` (KV_SIGMA_*; any other value returns
 * KV_ERR_ARG).  Every other argument, output and rule as in kv_mu_sigma. */
int kv_mu_sigma_ex(const kv_problem* pr, const void* q_win, const void* k, float scale,
                   const float* row_max, const float* row_sum, int32_t sigma_rows, float* mu,
                   float* sigma, float* attn, void* stream);

/* kv_window_mu_sigma with the dispersion taken over `sigma_rows` (KV_SIGMA_*; any other value
 * returns KV_ERR_ARG).  Every other argument, output and rule as in kv_window_mu_sigma. */
int kv_window_mu_sigma_ex(const kv_problem* pr, const void* q_win, const void* k, float scale,
                          int32_t sigma_rows, float* row_max, float* row_sum, float* mu,
                          float* sigma, void* ws, size_t ws_bytes, void* stream);

/* Window statistics and base scores in one call (section 3.1, Eq. (1), (3); section 3.2, Eq. (5)):
 * row_max / row_sum as from kv_window_mu_sigma_ex with the same sigma_rows, and for every key i of
 * every problem p and kv head
 *   score[i] = fmaf(lambda1[p], sigma[i], w_mu * mu[i])   (fp32, one rounding of the fma)
 * bit for bit what kv_window_mu_sigma_ex's mu and sigma give, without those two arrays.  score has
 * the layout of mu (problem p at tok_off[p]*h_kv, [h_kv][L_p], fp32, 16-byte aligned).
 * lambda1: [n_prob] fp32 device.  w_mu: finite (1 for the paper's score).
 * For bf16 batches (w = 32, d in {64, 128}, G in {1, 2, 4}, scale > 0) the scores are formed
 * inside the window kernel's second pass, which then writes one array instead of two; with every
 * (problem, kv head) scored by one workgroup no workspace is needed.  Otherwise, and when the
 * one-launch path cannot run, mu and sigma go through the workspace
 * (kv_base_scores_workspace_bytes).  Calls that overlap on one workspace race. */
int kv_window_base_scores(const kv_problem* pr, const void* q_win, const void* k, float scale,
                          const float* lambda1, float w_mu, int32_t sigma_rows, float* row_max,
                          float* row_sum, float* score, void* ws, size_t ws_bytes, void* stream);

/* Bytes of device workspace kv_window_base_scores needs for this batch with scale > 0 (0 if none;
 * 256-byte alignment).  Returns 0 for invalid arguments as well. */
size_t kv_base_scores_workspace_bytes(const kv_problem* pr);

/* Greedy diversity-aware selection (Eq. (2), (4), (5); section 3.2), per problem p and kv head g:
 *   candidates i in [0, n_cand), n_cand = L_p - keep_tail (the last keep_tail positions are always
 *   kept and never compete);
 *   s_i = mu_i + lambda1[p] * sigma_i (one fp32 rounding); s~_i = s_i / max(max_j s_j, 1e-12);
 *   the candidate set P is the C = min(cand_mult * budget, n_cand) largest s (cand_mult = 0: all
 *   n_cand), ties to the lower position;
 *   then `budget` times: admit argmax_{i in P \ S} s~_i + lambda2[p] * corr_i (ties to the lower
 *   position), where corr_i = max(0, max_{j in S} cos(k_i, k_j)) is a running maximum updated
 *   against each newly admitted key; a zero key has cosine 0.
 * Outputs: sel_idx[p,g,t] = position admitted at step t (admission order); sel_score (nullable) =
 * its score s~ + lambda2 corr; cand_idx (nullable) = P in ascending position order, padded with -1;
 * cand_corr (nullable) = each candidate's corr when it was admitted or, if never admitted, after the
 * last step (padding 0).  Decisions are taken in fp32.  Needs workspace.
 * Limit: C * d * e <= 131072 bytes (C <= 512 for bf16 keys of dimension 128). */
int kv_mmr_select(const kv_problem* pr, const float* mu, const float* sigma, const void* k,
                  const float* lambda1, const float* lambda2, int32_t budget, int32_t cand_mult,
                  int32_t keep_tail, int32_t* sel_idx, float* sel_score, int32_t* cand_idx,
                  float* cand_corr, void* ws, size_t ws_bytes, void* stream);

/* Scoring and budget options of kv_mmr_select_ex.  NULL options mean {pool = 1, w_mu = 1, no
 * per-problem budgets}, which is exactly kv_mmr_select.
 *   pool: odd window, 1 <= pool <= 63, of a max-pool over positions applied to the base score
 *     before normalisation and the top-C restriction (the pooling that the mean-attention baselines
 *     apply and that the paper keeps in its scoring, section 3.1):
 *     s'_i = max_{j in [i - pool/2, i + pool/2] and [0, n_cand)} s_j.  The normaliser
 *     max_j s'_j equals max_j s_j.
 *   w_mu: weight of mu in the base score, s_i = w_mu * mu_i + lambda1 * sigma_i, with w_mu * mu_i
 *     rounded to fp32 first (exact for w_mu = 1).  w_mu = 0 is the mean-free "dispersion and
 *     redundancy" rule of the term ablation (section 4.3, Table 3).
 *   budget_host / budget_dev: per-problem budgets B_p (n_prob int32 values, the same values in
 *     host and device memory; both NULL for the uniform `budget`).  The budgets of a depth schedule
 *     such as kv_pyramid_budgets (section 3.1: the runs use budgets that fall with depth at a fixed
 *     total).  Each B_p must satisfy 1 <= B_p <= budget and B_p <= L_p - keep_tail (else
 *     KV_ERR_BUDGET); `budget` stays the row stride of sel_idx / sel_score, and problem p runs B_p
 *     greedy steps, C_p = min(cand_mult * B_p, n_cand) candidates, and pads steps B_p .. budget-1
 *     with sel_idx = -1 and sel_score = 0.  One array without the other returns KV_ERR_NULL.
 * An even, non-positive or too large pool, or a non-finite w_mu, returns KV_ERR_ARG. */
typedef struct kv_select_opts {
  int32_t pool;
  float w_mu;
  const int32_t* budget_host;
  const int32_t* budget_dev;
} kv_select_opts;

/* kv_mmr_select with scoring options (opts nullable, see kv_select_opts); every other argument,
 * output and limit as in kv_mmr_select. */
int kv_mmr_select_ex(const kv_problem* pr, const float* mu, const float* sigma, const void* k,
                     const float* lambda1, const float* lambda2, int32_t budget, int32_t cand_mult,
                     int32_t keep_tail, const kv_select_opts* opts, int32_t* sel_idx,
                     float* sel_score, int32_t* cand_idx, float* cand_corr, void* ws,
                     size_t ws_bytes, void* stream);

/* Compacted cache (sections 1 and 3.1: each layer keeps `budget` entries plus the kept tail);
 * budget <= 8192.
 * For every problem and kv head, rows 0..budget-1 of k_out/v_out are the rows of k/v at the
 * selected positions in ascending order, rows budget..budget+keep_tail-1 the last keep_tail
 * positions.  Byte-exact copies.  A selected position outside [0, L_p) leaves its output row
 * unwritten.  Needs no workspace. */
int kv_compact_cache(const kv_problem* pr, const void* k, const void* v, const int32_t* sel_idx,
                     int32_t budget, int32_t keep_tail, void* k_out, void* v_out, void* stream);

/* kv_mmr_select (default scoring, no optional outputs) followed by kv_compact_cache, in one launch
 * (section 3.2, Eq. (2), (4), (5); sections 1 and 3.1): sel_idx [n_prob][h_kv][budget] as from
 * kv_mmr_select, k_out / v_out [n_prob][h_kv][budget + keep_tail][d] as from kv_compact_cache
 * with the same sel_idx; budget <= 8192.  k, v, k_out, v_out 16-byte aligned.  The workspace
 * (ws, ws_bytes) is that of kv_mmr_select.  Returns the codes of both calls. */
int kv_mmr_select_compact(const kv_problem* pr, const float* mu, const float* sigma, const void* k,
                          const void* v, const float* lambda1, const float* lambda2,
                          int32_t budget, int32_t cand_mult, int32_t keep_tail, int32_t* sel_idx,
                          void* k_out, void* v_out, void* ws, size_t ws_bytes, void* stream);

/* kv_mmr_select_ex, optionally followed by kv_compact_cache_ex's compaction in the same launch,
 * with the base scores given (section 3.2, Eq. (2), (4), (5)): score as from kv_window_base_scores
 * (16-byte aligned) takes the place of fmaf(lambda1[p], sigma, w_mu * mu), so that with the score
 * of the same mu, sigma, lambda1 and w_mu every output equals kv_mmr_select_ex's bit for bit.
 * opts (nullable) as in kv_mmr_select_ex, its w_mu unused.  With k_out and v_out (both or
 * neither; v then required) the compaction is kv_mmr_select_compact's: budget <= 8192, rows of
 * [n_prob][h_kv][budget + keep_tail][d], the first B_p rows of a block from the selection.
 * sel_score, cand_idx, cand_corr nullable as in kv_mmr_select.  Needs no workspace. */
int kv_mmr_select_scored(const kv_problem* pr, const float* score, const void* k, const void* v,
                         const float* lambda2, int32_t budget, int32_t cand_mult, int32_t keep_tail,
                         const kv_select_opts* opts, int32_t* sel_idx, float* sel_score,
                         int32_t* cand_idx, float* cand_corr, void* k_out, void* v_out,
                         void* stream);

/* Window statistics and the candidate set P of the selection in one call (section 3.1, Eq. (1),
 * (3); section 3.2, Eq. (4), (5)): row_max / row_sum as from kv_window_base_scores with the same
 * sigma_rows, and, in the workspace (ws, ws_bytes >= kv_candidates_workspace_bytes, 256-byte
 * aligned), for every problem p and kv head g the C_p = min(cand_mult * B_p, n_cand) candidates of
 * kv_mmr_select_ex (the largest base scores s_i = fmaf(lambda1[p], sigma_i, w_mu * mu_i) over
 * i < n_cand = L_p - keep_tail, ties to the lower position) with their scores, and the normaliser
 * max(max_i s_i, 1e-12), so that kv_mmr_select_candidates can run the greedy without the score
 * array.  The layout of the workspace is private to these two calls; it stays valid until the
 * next call that writes it.  budget, cand_mult, keep_tail and opts (pool must be 1, else
 * KV_ERR_ARG; w_mu and the per-problem budgets as in kv_mmr_select_ex) must be the values later
 * given to kv_mmr_select_candidates.  lambda1: [n_prob] fp32 device.
 * For bf16 batches that kv_window_base_scores scores inside the window kernel's second pass, with
 * cand_mult > 0 and L_p <= 32768, the keys are read once in full, the candidates
 * are cut inside that launch (a second pass revisits only the 32-key tiles whose score bound
 * reaches the cut) and no score is stored; otherwise the scores go through the workspace and the
 * selection kernel's first phases cut the candidates from them.  Calls that overlap on one
 * workspace race. */
int kv_window_candidates(const kv_problem* pr, const void* q_win, const void* k, float scale,
                         const float* lambda1, int32_t sigma_rows, int32_t budget,
                         int32_t cand_mult, int32_t keep_tail, const kv_select_opts* opts,
                         float* row_max, float* row_sum, void* ws, size_t ws_bytes, void* stream);

/* Bytes of device workspace kv_window_candidates needs for this batch and these selection
 * arguments with scale > 0 (256-byte alignment).  Returns 0 for invalid arguments. */
size_t kv_candidates_workspace_bytes(const kv_problem* pr, int32_t budget, int32_t cand_mult,
                                     int32_t keep_tail, const kv_select_opts* opts);

/* The greedy of kv_mmr_select_scored, and optionally its compaction, from the candidates that
 * kv_window_candidates left in the workspace (section 3.2, Eq. (2), (4)): with the same budget,
 * cand_mult, keep_tail and opts, every output equals kv_mmr_select_scored's given the score of
 * kv_window_base_scores, bit for bit (sel_idx, sel_score, cand_idx, cand_corr, k_out, v_out;
 * nullability, layouts and limits as there).  The workspace is only read. */
int kv_mmr_select_candidates(const kv_problem* pr, const void* ws, size_t ws_bytes, const void* k,
                             const void* v, const float* lambda2, int32_t budget,
                             int32_t cand_mult, int32_t keep_tail, const kv_select_opts* opts,
                             int32_t* sel_idx, float* sel_score, int32_t* cand_idx,
                             float* cand_corr, void* k_out, void* v_out, void* stream);

/* The whole eviction pass of a batch in one call (sections 3.1 and 3.2, Eq. (1)-(5)): exactly
 * kv_window_candidates followed by kv_mmr_select_candidates on the same workspace with the same
 * budget, cand_mult, keep_tail and opts (cand_idx / cand_corr not offered): row_max, row_sum,
 * sel_idx, sel_score (nullable) and, with k_out and v_out (both or neither; v then required), the
 * compacted cache, bit for bit as the two calls give them, and the workspace (ws, ws_bytes >=
 * kv_candidates_workspace_bytes) left holding the candidates.  Arguments, layouts, limits and
 * error codes as in the two calls; nothing is launched when either would refuse its arguments.
 * Where the window kernel cuts the candidates (bf16, L_p <= 32768, see kv_window_candidates) and
 * every C_p = min(cand_mult * B_p, n_cand) <= 256, each (problem, kv head) unit's workgroup runs
 * the greedy and the compaction right after its cut, in the same launch; otherwise the two calls
 * run in turn.  Calls that overlap on one workspace race. */
int kv_evict_pass(const kv_problem* pr, const void* q_win, const void* k, const void* v,
                  float scale, const float* lambda1, const float* lambda2, int32_t sigma_rows,
                  int32_t budget, int32_t cand_mult, int32_t keep_tail, const kv_select_opts* opts,
                  float* row_max, float* row_sum, int32_t* sel_idx, float* sel_score, void* k_out,
                  void* v_out, void* ws, size_t ws_bytes, void* stream);

/* kv_compact_cache with per-problem budgets and a chosen block size (budget_host / budget_dev as
 * in kv_select_opts; both NULL with out_rows = 0 is exactly kv_compact_cache).  The block of every
 * (problem, kv head) in k_out / v_out has out_rows rows (0: budget + keep_tail; otherwise at least
 * budget + keep_tail, else KV_ERR_ARG), so that rows for generated tokens can follow the kept ones
 * (kv_decode_attention appends there).  Rows 0..B_p-1 are the rows of the first B_p selected
 * positions in ascending order, rows B_p..B_p+keep_tail-1 the last keep_tail positions, and the
 * rows after them are not written. */
int kv_compact_cache_ex(const kv_problem* pr, const void* k, const void* v,
                        const int32_t* sel_idx, int32_t budget, int32_t keep_tail,
                        const int32_t* budget_host, const int32_t* budget_dev, int32_t out_rows,
                        void* k_out, void* v_out, void* stream);

/* A batch of caches for decoding: problem p (one layer of one sequence) holds, for every kv head
 * g, a block of row_stride rows of d elements starting at row (p * h_kv + g) * row_stride of the
 * K and V buffers, of which rows 0..len_p-1 are in use (the layout kv_compact_cache_ex writes, with
 * len_p = B_p + keep_tail).  len_host / len_dev: n_prob lengths in host and device memory. */
typedef struct kv_cache_batch {
  int32_t dtype; /* KV_F32 or KV_BF16: caches, queries and new rows */
  int32_t n_prob;
  int32_t h_q;
  int32_t h_kv;
  int32_t d;
  int32_t row_stride;
  const int32_t* len_host;
  const int32_t* len_dev;
} kv_cache_batch;

/* Bytes of device workspace kv_decode_attention needs for this batch (0 if none; 256-byte
 * alignment).  Returns 0 for invalid arguments as well. */
size_t kv_decode_workspace_bytes(const kv_cache_batch* cb);

/* Attention of one generated token per problem over its cache (section 4.3: after eviction the
 * model generates against the kept rows of every layer):
 *   out[p,h,:] = sum_r softmax_r(scale <q[p,h], k[p,g,r]>) v[p,g,r,:],  g = h / (h_q / h_kv),
 * over the rows r < len_p, plus the token's own row when k_new / v_new are given: then
 * k_new[p,g,:] / v_new[p,g,:] are also written into row len_p of every block (len_p < row_stride
 * required), so the next call passes len_p + 1.
 * q [n_prob, h_q, d] and k_new / v_new [n_prob, h_kv, d] in the cache dtype; out fp32
 * [n_prob, h_q, d].  Logits, softmax and the weighted sum in fp32.  k_new and v_new both or
 * neither (KV_ERR_NULL).  h_q / h_kv <= 8, d in {64, 128}, every len_p >= 1 (or >= 0 with a new
 * row) and <= row_stride, else KV_ERR_SHAPE.  Needs the workspace of kv_decode_workspace_bytes. */
int kv_decode_attention(const kv_cache_batch* cb, const void* q, void* k_cache, void* v_cache,
                        const void* k_new, const void* v_new, float scale, float* out, void* ws,
                        size_t ws_bytes, void* stream);

/* Per-layer budgets that fall with depth at the total of a uniform `budget` (section 3.1: the runs
 * use such an allocation; the paper prints no schedule), host-only.  With
 * B_min = max(1, floor(budget / beta)) and B_max = 2 budget - B_min, layer l gets the linear
 * value B_max - l (B_max - B_min) / (n_layers - 1) rounded away from `budget` (up above it, down
 * below it), so the layers sum to exactly n_layers * budget; one layer gets `budget`.
 * budgets_host receives n_layers values.  beta >= 1 (beta = 1: uniform).  KV_ERR_NULL for a NULL
 * output, KV_ERR_ARG for budget < 1, n_layers < 1 or beta < 1 or not finite. */
int kv_pyramid_budgets(int32_t budget, int32_t n_layers, double beta, int32_t* budgets_host);

/* Per-layer coefficients of a depth profile (section 3.3, Eq. (6)), host-only:
 * lambda_out_host[l] = (float) sinh(a(l)) for l = 0..n_layers-1, a(l) given by `family` and the
 * latent parameters `params_host` (n_params values).  Returns KV_ERR_ARG for an unknown family or
 * a wrong parameter count, KV_ERR_NULL for NULL pointers. */
int kv_depth_profile(int32_t family, const double* params_host, int32_t n_params,
                     int32_t n_layers, float* lambda_out_host);

#ifdef __cplusplus
}
#endif

#endif /* KVEVICT_H */
