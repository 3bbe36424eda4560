/*
 * prouter.h -- C ABI of the token-aware verifier hot path for MI355X (gfx950).
 *
 * The library turns each generated token's vocabulary logit row into
 * confidence features, summarises them per request and decides per request
 * whether the small model's answer ships or escalates (Pro-Router, Sec. 3.1:
 * per-token features, Eq. 3; the ship rule p >= tau stated with the gain,
 * Eq. 1; the quantile-summary verifier input, Sec. 4.2, Table "ablation").
 *
 * Conventions for every call:
 *  - Data pointers are DEVICE pointers unless a comment says otherwise. The
 *    caller owns all memory; the library never frees caller memory.
 *  - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *    Calls only enqueue work on it and return; nothing synchronises the
 *    stream except pr_validate_offsets, which says so.
 *  - Errors in host-visible arguments (NULL required pointer, bad sizes,
 *    misalignment, unknown enum) return PR_ERR_INVALID_ARG and launch
 *    nothing. Errors in device data (NaN logits, bad ids, bad temperature)
 *    cannot be seen without a sync: they set per-row flags and the call
 *    still returns PR_OK. A failed launch returns PR_ERR_HIP.
 *  - No C++ exception crosses this boundary.
 */
#ifndef PROUTER_H
#define PROUTER_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* The enumerations are int-sized in C. C++ gives them int as a fixed
 * underlying type, so that a caller's out-of-range value (which the calls
 * reject) is still a valid value of the type there. */
#ifdef __cplusplus
#define PR_ENUM_BASE : int
#else
#define PR_ENUM_BASE
#endif

typedef enum pr_status PR_ENUM_BASE {
  PR_OK = 0,
  PR_ERR_INVALID_ARG = 1,
  PR_ERR_UNSUPPORTED = 2,
  PR_ERR_HIP = 3,
  PR_ERR_NO_MEMORY = 4
} pr_status;

/* Storage type of the logits. bf16 is the upper 16 bits of an IEEE float32. */
typedef enum pr_dtype PR_ENUM_BASE { PR_F32 = 0, PR_BF16 = 1 } pr_dtype;

/* Per-row flags (bit set in pr_token_features_t.flags). */
#define PR_FLAG_NONFINITE 1u       /* a NaN or +inf logit, or every logit is -inf; all float
                                      outputs NaN, all integer outputs -1                     */
#define PR_FLAG_BAD_ID 2u          /* sampled id outside [0, V): logprob NaN, rank -1; the
                                      other outputs are still valid                           */
#define PR_FLAG_BAD_TP 4u          /* temperature not finite or below 2^-100, top-p NaN or
                                      <= 0, or |max logit| > 2^100 * T; outputs as for
                                      NONFINITE (which is still reported when it applies)     */
#define PR_FLAG_OUTSIDE_NUCLEUS 8u /* top-p on and the sampled token lies outside the
                                      nucleus: logprob = -inf, rank > cutoff                  */

/*
 * Per-token outputs, one array per feature, each [n_rows] (structure of
 * arrays). Definitions (u = z / T, order of tokens: larger raw logit first,
 * equal logits by lower index; N = the nucleus, all V tokens when top-p is off):
 *   max_logit  z_argmax / T
 *   lse        log sum_{v in N} exp(u_v)                  (nucleus normaliser)
 *   entropy    Shannon entropy in nats of softmax(u) renormalised on N
 *   logprob    log p_N(y), -inf if y is outside N          (Eq. 3, l_t)
 *   maxprob    max_v p_N(v)                                (Eq. 3, m_t)
 *   margin     (z_argmax - z_second) / T, over all tokens
 *   rank       1-based position of y in the order
 *   argmax     first token of the order
 *   cutoff     |N| (V when top-p is off)
 *   flags      PR_FLAG_* bits
 */
typedef struct pr_token_features_t {
  float* max_logit;
  float* lse;
  float* entropy;
  float* logprob;
  float* maxprob;
  float* margin;
  int32_t* rank;
  int32_t* argmax;
  int32_t* cutoff;
  uint32_t* flags;
} pr_token_features_t;

/*
 * Summary head. The summarised per-token tuple is
 *   A = (logprob, maxprob, -entropy, margin)        (feature index f = 0..3)
 * (the entropy is negated as the paper's h_t = -H_t so that every column
 * rises with confidence). Statistics (index s): 0 mean, 1 min, 2 the
 * nearest-rank q-quantile, i.e. the j-th smallest value with
 * j = max(1, ceil(q * n)), q * n rounded once in double.
 * score = link(b + sum over w[s*4+f] != 0 of w[s*4+f] * stat_s(A_f)),
 * link 0 = identity, 1 = logistic sigmoid. Zero weights are skipped.
 * Defaults (pr_agg_params_default): q = 0.1, w = 1 on mean(maxprob) only,
 * b = 0, identity -- the score is the request's mean max-probability.
 */
typedef struct pr_agg_params {
  double q;
  double w[12];
  double b;
  int32_t link;
} pr_agg_params;

/* Per-request outputs. mean/min/quant are [n_req][4] (row-major, feature
 * index fastest); count and score are [n_req]. Any member may be NULL when
 * that output is not wanted (score is needed by pr_route). An empty request
 * or a NaN value in a feature's segment gives NaN summaries (and score). */
typedef struct pr_request_agg_t {
  int32_t* count;
  float* mean;
  float* min;
  float* quant;
  float* score;
} pr_request_agg_t;

/* Human-readable name of a status code (static string, host). */
const char* pr_status_string(pr_status status);

/* Fills *params (host pointer) with the default summary head. */
void pr_agg_params_default(pr_agg_params* params);

/*
 * Bytes of device workspace pr_token_features needs for this shape (0 when
 * none). top_p_on: 1 if a top-p array will be passed.
 */
size_t pr_token_features_workspace(pr_dtype dtype, int64_t n_rows, int32_t vocab, int32_t top_p_on);

/*
 * Per-token features of n_rows logit rows (Sec. 3.1, Eq. 3, extended to the
 * feature set documented at pr_token_features_t; top-p as a nucleus prefix of
 * the token order).
 *   logits       [n_rows][row_stride] of dtype; row r starts at element
 *                r * row_stride. Requires vocab >= 2, row_stride >= vocab and
 *                the base aligned to the element size.
 *   sampled_ids  int32 [n_rows], the emitted token of each row.
 *   temperature  float [n_rows], per-row temperature (finite, >= 2^-100).
 *   top_p        float [n_rows] or NULL (off). P >= 1 switches a row's
 *                truncation off; 0 < P < 1 keeps the shortest prefix of the
 *                order whose mass reaches P of the total. With top_p, vocab
 *                must be below 2^24 (PR_ERR_UNSUPPORTED otherwise).
 *   out          host pointer to a struct of device output arrays, all
 *                required.
 *   workspace    device scratch of at least
 *                pr_token_features_workspace(...) bytes (may be NULL when that
 *                is 0). Its contents need no initialisation.
 * n_rows == 0 is valid and launches nothing.
 */
pr_status pr_token_features(const void* logits, pr_dtype dtype, int64_t n_rows, int32_t vocab,
                            int64_t row_stride, const int32_t* sampled_ids, const float* temperature,
                            const float* top_p, const pr_token_features_t* out, void* workspace,
                            size_t workspace_bytes, void* stream);

/*
 * pr_token_features for callers that cannot allocate device memory (code
 * under HIP graph capture, serving loops or harnesses that forbid
 * hipMalloc): the same arguments and outputs without the workspace. The
 * split-row scratch that small batches need (fewer than 256 rows) lives in a
 * static device array of PR_NOALLOC_SCRATCH_BYTES that each GPU holds until
 * the process ends; its address is looked up on the first call on a device.
 * Nothing is allocated and nothing needs clearing (every scratch entry is
 * written before it is read in the same call). Calls that overlap on one GPU
 * (other streams or host threads) share the array and race: serialise them.
 * Returns PR_ERR_UNSUPPORTED when a shape would need more scratch than the
 * array holds (no accepted shape does: the most is 12,272 bytes, 256 rows' or
 * workgroups' partial states), PR_ERR_HIP when the address lookup fails.
 */
#define PR_NOALLOC_SCRATCH_BYTES 16384
pr_status pr_token_features_noalloc(const void* logits, pr_dtype dtype, int64_t n_rows, int32_t vocab,
                                    int64_t row_stride, const int32_t* sampled_ids, const float* temperature,
                                    const float* top_p, const pr_token_features_t* out, void* stream);

/* Largest K of pr_feature_sequence's top-K entropy. */
#define PR_MAX_TOP_K 32

/*
 * The paper's verifier input sequence X (Sec. 3.1, Eq. 3 and the text after
 * it). Request i owns rows offsets[i] .. offsets[i+1]-1; row r is its token
 * t = r - offsets[i] + 1 of T_i = offsets[i+1] - offsets[i]. For every row:
 *   X[r][0] = l_t   = log p(y_t)               (logprob of pr_token_features)
 *   X[r][1] = m_t   = max_v p(v)               (maxprob)
 *   X[r][2] = h_t   = -H_t, H_t = -sum of p(v) log p(v) over the top_k most
 *                     probable tokens, p not renormalised over them
 *   X[r][3] = rho_t = t / T_i
 * p is the distribution after temperature and top-p, as in pr_token_features;
 * when the nucleus holds fewer than top_k tokens, H_t sums over the nucleus.
 * Tokens of probability 0 (logit -inf) add nothing.
 *   logits .. top_p  as for pr_token_features.
 *   offsets    int32 [n_req + 1], device: offsets[0] == 0, non-decreasing,
 *              offsets[n_req] == n_rows (a precondition, as for
 *              pr_request_aggregate; pr_validate_offsets checks it). A row
 *              outside the offsets gets rho = NaN.
 *   top_k      1 .. PR_MAX_TOP_K (the paper uses 20).
 *   X          float [n_rows][4], device, row-major.
 *   features   host pointer to a struct of device arrays that also receive
 *              the per-token features of pr_token_features (all members
 *              set), or NULL. Their flags give the reason of NaN entries: a
 *              row flagged PR_FLAG_NONFINITE or PR_FLAG_BAD_TP has NaN in
 *              l, m and h; PR_FLAG_BAD_ID makes l NaN only.
 * One workgroup reads each row once; no workspace. n_rows == 0 launches
 * nothing.
 */
pr_status pr_feature_sequence(const void* logits, pr_dtype dtype, int64_t n_rows, int32_t vocab,
                              int64_t row_stride, const int32_t* sampled_ids, const float* temperature,
                              const float* top_p, const int32_t* offsets, int32_t n_req, int32_t top_k,
                              float* X, const pr_token_features_t* features, void* stream);

/*
 * Fused sample-and-verify (the verifier reads the decoding distribution as a
 * side product of decoding, Sec. 3.1 and Sec. 4.1): one read of each row both
 * draws its token y_r from softmax(z_r / T_r) and computes the verifier's
 * outputs for that token.
 *   logits, dtype, n_rows, vocab, row_stride, temperature
 *              as for pr_token_features (no top-p).
 *   seed, offset
 *              the draw is a fixed function of (seed, offset, row index, the
 *              row's logits and temperature, and the workgroup size, which
 *              the number of rows selects: at least 2,048, 257..2,047, or up
 *              to 256): the same call gives the same tokens; a new offset
 *              (e.g. the decode step) gives fresh draws. Uniforms come from
 *              Threefry-2x32-13 (Salmon et al., SC 2011).
 *   sampled_ids
 *              int32 [n_rows], device, written: the drawn token, or -1 when
 *              the row's distribution is undefined (non-finite logits or a
 *              rejected temperature). A token of probability 0 is never
 *              drawn. Each token v is drawn with probability e_v / S up to
 *              float32 rounding of the masses (relative 1e-6).
 *   features   host pointer to a struct of device arrays (all members set),
 *              or NULL: the per-token features of pr_token_features for the
 *              drawn token, except rank, which is written as -1 ("not
 *              available", as for a bad id: counting the tokens above y
 *              needs z_y before the pass); a row with y = -1 is flagged
 *              PR_FLAG_BAD_ID besides its other flags.
 *   offsets, n_req, top_k, X
 *              X NULL: not computed. Otherwise the paper's verifier input
 *              sequence for the drawn tokens, with the arguments and layout
 *              of pr_feature_sequence.
 * One workgroup reads each row once; no workspace. n_rows == 0 launches
 * nothing.
 */
pr_status pr_sample_features(const void* logits, pr_dtype dtype, int64_t n_rows, int32_t vocab, int64_t row_stride,
                             const float* temperature, uint64_t seed, uint64_t offset, int32_t* sampled_ids,
                             const pr_token_features_t* features, const int32_t* offsets, int32_t n_req,
                             int32_t top_k, float* X, void* stream);

/* The verifier head (Sec. 3.1, the paragraph after Eq. 3; Sec. 4.2): its
 * number of float32 parameters, and the device workspace it needs. */
#define PR_HEAD_WEIGHTS 67329
size_t pr_verifier_head_workspace(int64_t n_rows);

/*
 * The paper's shipping confidence of each request from its input sequence X
 * (Sec. 3.1, after Eq. 3): a linear projection of each token's 4 features to
 * 64 with the sinusoidal positional encoding of its position t - 1 added,
 * two post-norm transformer encoder layers (4 heads of 16 dimensions,
 * softmax over every token of the same request, feed-forward width 128 with
 * ReLU, LayerNorm over the 64 features with eps 1e-5), the mean over the
 * request's tokens, a linear map to one logit and the logistic sigmoid.
 * Computed in float32. The paper publishes no weights; any weights of this
 * shape may be passed.
 *   X          float [n_rows][4], device (as written by pr_feature_sequence).
 *   offsets    int32 [n_req + 1], device; precondition as for
 *              pr_request_aggregate.
 *   max_len    at least the number of tokens of the longest request; a
 *              longer request scores NaN. 1 .. 2^20 (PR_ERR_UNSUPPORTED
 *              above).
 *   weights    float [PR_HEAD_WEIGHTS], device, 16-byte aligned, in this order (matrices
 *              row-major [out][in]): W_in [64][4], b_in [64]; per layer:
 *              W_qkv [192][64] (query rows, then key rows, then value rows;
 *              head k owns rows 16k .. 16k+15 of each), b_qkv [192],
 *              W_o [64][64], b_o [64], LayerNorm-1 gain [64] and shift [64],
 *              W_1 [128][64], b_1 [128], W_2 [64][128], b_2 [64],
 *              LayerNorm-2 gain [64] and shift [64]; then w_out [64], b_out [1].
 *   scores     float [n_req], device. An empty request scores NaN (it
 *              escalates under pr_route).
 *   workspace  device scratch of at least pr_verifier_head_workspace(n_rows)
 *              bytes, 16-byte aligned; no initialisation needed.
 */
pr_status pr_verifier_head(const float* X, int64_t n_rows, const int32_t* offsets, int32_t n_req, int32_t max_len,
                           const float* weights, float* scores, void* workspace, size_t workspace_bytes,
                           void* stream);

/*
 * Ragged per-request summaries and score (Sec. 3.1, the stacked feature
 * sequence X; Sec. 4.2, Table "ablation", quantile-summary input).
 *   feats     host pointer to the per-token arrays; logprob, maxprob, entropy
 *             and margin are read.
 *   offsets   int32 [n_req + 1], device. Request i owns rows
 *             offsets[i] .. offsets[i+1]-1. Precondition (not checked here,
 *             see pr_validate_offsets): offsets[0] >= 0, non-decreasing.
 *   params    host pointer, or NULL for the defaults.
 *   out       host pointer to a struct of device output arrays.
 */
pr_status pr_request_aggregate(const pr_token_features_t* feats, const int32_t* offsets, int32_t n_req,
                               const pr_agg_params* params, const pr_request_agg_t* out, void* stream);

/*
 * Ship-or-escalate (Sec. 3.1: ship iff p >= tau). ship[i] = 1 iff
 * scores[i] >= threshold; a NaN score escalates (0). n_ship, if not NULL,
 * receives the number of shipped requests (device int32).
 */
pr_status pr_route(const float* scores, int32_t n_req, float threshold, uint8_t* ship, int32_t* n_ship,
                   void* stream);

/*
 * Threshold calibration for a ship fraction (Sec. 3.1: tau is fixed in
 * advance by calibration on a validation pool; Sec. 4.1: the coverage rule,
 * a fraction q of the pool ships). scores: device float32 [n], the pool's
 * shipping confidences; NaN scores are not part of the pool (they always
 * escalate). tau[0] (device float32) = the k-th largest of the n_valid
 * non-NaN scores, k = max(1, ceil(ship_fraction * n_valid)) with the product
 * rounded once in double; n_ship[0] (device int32, may be NULL) =
 * #{scores >= tau}, at least k (more when scores tie at tau). -0 counts as
 * +0. ship_fraction == 0 or no valid score: tau = +inf, n_ship = 0.
 * ship_fraction must lie in [0, 1] (NaN rejected); n >= 0; scores may be
 * NULL only when n == 0. Exact: tau is one of the scores. workspace: device
 * memory of at least pr_calibrate_workspace(n) bytes, 4-byte aligned, owned
 * by the caller and not shared with a concurrent call (NULL when that size
 * is 0: pools of up to 16,384 scores need none); otherwise
 * PR_ERR_INVALID_ARG.
 */
pr_status pr_calibrate_threshold(const float* scores, int32_t n, double ship_fraction, float* tau, int32_t* n_ship,
                                 void* workspace, size_t workspace_bytes, void* stream);

/* Workspace bytes pr_calibrate_threshold needs for a pool of n scores (0 for n <= 16,384). */
size_t pr_calibrate_workspace(int32_t n);

/*
 * Synchronous debug check of an offsets array (device pointer): returns
 * PR_OK iff offsets[0] == 0, offsets are non-decreasing and
 * offsets[n_req] == n_rows. Synchronises `stream`.
 */
pr_status pr_validate_offsets(const int32_t* offsets, int32_t n_req, int64_t n_rows, void* stream);

/* ------------------------------------------------------------------------
 * Streaming decode-step variant. Per-request state stays on the device
 * between steps; a request's verdict is taken when it finishes, as the
 * paper's verifier decides when the engine reports a request finished
 * (Sec. 4.1, implementation details).
 * ------------------------------------------------------------------------ */
typedef struct pr_stream pr_stream;

/*
 * Allocates the device state for max_slots concurrent requests of at most
 * max_len tokens each, on the current device (the only allocating call of
 * the streaming API). params may be NULL (defaults). *state is a host handle.
 * max_len == 0 selects bounded memory: no per-token history is kept and the
 * tail quantile is the P-square estimate of the params' q (Jain and
 * Chlamtac, CACM 1985), 224 bytes per slot, any number of tokens per
 * request. Its estimate is exact up to 5 tokens; an infinite value of a
 * column (a margin of +inf, a log-prob of -inf) makes that column's
 * quantile NaN for the request (the mean and minimum keep it).
 */
pr_status pr_stream_create(int32_t max_slots, int32_t max_len, const pr_agg_params* params, pr_stream** state);

/*
 * One decode step: features of n_active rows (same layout and rules as
 * pr_token_features), and for each row r the slot slot_ids[r] (device
 * int32 [n_active]) gains one token: count, running sums and minima of A,
 * and the token's A is appended to the slot's history (needed for the exact
 * quantile). A slot may appear at most once per step (duplicates race).
 * Tokens past max_len are counted in sums and minima but not kept, and the
 * slot's quantile becomes NaN. In bounded-memory mode (max_len == 0) the
 * token instead updates the slot's P-square markers. out may be NULL (features not returned).
 * top_p (device float [n_active]) or NULL: with it, the features and the
 * tuple A that joins the slot are those of the renormalised nucleus, as in
 * pr_token_features (vocab below 2^24, PR_ERR_UNSUPPORTED otherwise).
 */
pr_status pr_stream_step(pr_stream* state, const void* logits, pr_dtype dtype, int32_t n_active,
                         int32_t vocab, int64_t row_stride, const int32_t* slot_ids,
                         const int32_t* sampled_ids, const float* temperature, const float* top_p,
                         const pr_token_features_t* out, void* stream);

/*
 * Finishes n requests: for each slots[i] (device int32 [n]) computes the
 * summaries and score as pr_request_aggregate would over the slot's tokens,
 * writes them to out[i] (members may be NULL; the struct pointer is a host
 * pointer), sets ship[i] (device uint8 [n], may be NULL) by
 * score >= threshold, then clears the slot for reuse.
 */
pr_status pr_stream_finish(pr_stream* state, const int32_t* slots, int32_t n, float threshold,
                           const pr_request_agg_t* out, uint8_t* ship, void* stream);

/* Clears n slots (device int32 [n]) without producing a verdict. */
pr_status pr_stream_reset_slots(pr_stream* state, const int32_t* slots, int32_t n, void* stream);

/* Frees the state (synchronises the device first). NULL is ignored. */
void pr_stream_destroy(pr_stream* state);

#ifdef __cplusplus
}
#endif

#endif /* PROUTER_H */
