/*
 * ss.h -- C ABI of the MI355X fused LLM sampler (libss.so).
 *
 * Operations (SonicSampler, arXiv 2607.20475):
 *   ss_sample          singular-mode sampling: prologue (Appendix C.1), top-k /
 *                      top-p / min-p truncation in Alg. 11 order (Appendix C.2),
 *                      greedy or stochastic selection (Section 3.5, Appendix C.3)
 *   ss_sample_full     the same with top-p / min-p over the whole row for
 *                      requests without a top-k cut (Appendix C.2)
 *   ss_sample_gumbel   the same with the Gumbel-max draw over the kept set and
 *                      caller-drawn noise (Appendix C.3; the Stage-2 selection)
 *   ss_verify          multistep speculative verification (Section 3.1,
 *                      Appendix C.4): accept when u*q(d) <= p(d), else resample
 *                      from normalize(max(0, p - q)); bonus token on full acceptance
 *   ss_verify_sparse   the same against sparse draft distributions: the
 *                      (id, probability) lists a singular-mode draft step
 *                      emits over its candidate set (Section 3.2)
 *   ss_verify_tree     one path through a draft tree, its positions mapped to
 *                      the target rows of the tree (Appendix C.4)
 *   ss_topk            exact top-k (value, index) per row (Section 3.4)
 *   ss_process_logits  materialised processed logits and final probabilities
 *   ss_logprobs        top-k log-probabilities under the full-row distribution
 *                      (indicator bit 0x400, Section 3.5)
 *
 * Conventions (all functions):
 *   - Every array argument is a DEVICE pointer owned by the caller, except
 *     `const ss_params*`, which is a host struct whose members are device
 *     pointers.  The library never allocates, frees or synchronises; every
 *     launch goes to `stream` (a hipStream_t, NULL = default stream).
 *   - Row-major layouts with an explicit row stride `ld` (elements).
 *   - Per-request parameter arrays have B entries.  A NULL parameter array
 *     disables the indicator bits that need it (e.g. temperature == NULL
 *     clears SS_TEMP for every request), so a call never reads it.
 *   - Host-side validation happens before any launch; on error nothing is
 *     launched and a negative ss_status is returned.  Data-dependent
 *     conditions never stop the call: they are reported per row in `flags`.
 *   - Launch shapes depend only on (B, V, L, k_max, dtype): every call can be
 *     captured in a HIP graph.  Per-call values (seed, position, params) are
 *     read from device memory.
 *   - The workspace needs no initialisation: every call writes what it reads
 *     (its contents between calls are unspecified), so one workspace of the
 *     largest size may serve calls of any operation and shape.  Calls that
 *     share one workspace must not overlap in time.
 *   - Processed logits are float32 (one correctly rounded operation per
 *     prologue step).  Each kept token's weight exp((y - M)/tau) has its
 *     exponent formed in double and the exponential taken in float32 (about
 *     1 ulp, relative error below 2e-7; exponents below about -87 give float32
 *     subnormals and below about -104 zero, i.e. weights under 1e-38 of the
 *     row maximum's).  Weights are summed exactly as 2^-50 fixed-point
 *     integers; probabilities, cuts and draws are then taken in double.
 */
#ifndef SS_H_
#define SS_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t ss_status;
#define SS_OK 0
#define SS_ERR_INVALID_ARG (-1)
#define SS_ERR_UNSUPPORTED (-2)
#define SS_ERR_WORKSPACE (-3)
#define SS_ERR_HIP (-4)

/* Logit element types. */
#define SS_F32 0
#define SS_BF16 1

/* Per-request indicator bits: the paper's bit-level encoding table (Section 3.5). */
#define SS_GRAMMAR 0x001u  /* grammar bit-mask                                   */
#define SS_REP 0x002u      /* multiplicative repetition penalty                  */
#define SS_FREQ 0x004u     /* frequency penalty                                  */
#define SS_PRES 0x008u     /* presence penalty                                   */
#define SS_BIAS 0x010u     /* logit bias                                         */
#define SS_TEMP 0x020u     /* temperature scaling (tau <= 0 means greedy)        */
#define SS_GREEDY 0x040u   /* greedy selection                                   */
#define SS_TOPK 0x080u     /* top-k filtering                                    */
#define SS_TOPP 0x100u     /* top-p filtering                                    */
#define SS_MINP 0x200u     /* min-p filtering                                    */
#define SS_LOGPROBS 0x400u /* top-k log-probabilities (ss_logprobs)              */

/* Per-row result flags (int32 flags[rows]). */
#define SS_FLAG_EMPTY 1      /* every token masked: token -1                       */
#define SS_FLAG_FALLBACK 2   /* exact slow path used (skewed or tied row)          */
#define SS_FLAG_OUT_TRUNC 4  /* kept set longer than k_out                         */
#define SS_FLAG_KCAP 8       /* candidate set bounded by k_max (no or large top-k) */

/* Operations, for ss_workspace_bytes. */
#define SS_OP_TOPK 0
#define SS_OP_SAMPLE 1
#define SS_OP_VERIFY 2
#define SS_OP_PROCESS 3
#define SS_OP_LOGPROBS 4

/* Limits. */
#define SS_MAX_K 4096      /* k_max upper bound                                    */
#define SS_MAX_L 16        /* draft length upper bound                             */
#define SS_MAX_V (1 << 20) /* vocabulary upper bound                               */

/*
 * Per-request parameters (host struct of device pointers), read at call time.
 *
 * mode          uint32[B]  indicator bits above.
 * temperature   float[B]   tau (Appendix C.1); tau <= 0 with SS_TEMP means greedy.
 * top_k         int32[B]   k (Appendix C.2); k <= 0 means no top-k cut.
 * top_p         float[B]   p; p >= 1 means no cut.
 * min_p         float[B]   theta; theta <= 0 means no cut.
 * rep_penalty   float[B]   alpha (> 0, finite).
 * freq_penalty  float[B]   beta (finite).
 * pres_penalty  float[B]   gamma (finite).
 * hist_offsets  int32[B+1], hist_ids int32[nnz]: CSR of decoded token ids per request
 *               (multiplicity = occurrence count; ids outside [0,V) ignored).
 * bias_offsets  int32[B+1], bias_ids int32[nnz], bias_vals float[nnz]: CSR of sparse
 *               logit-bias entries; duplicate ids are summed in list order.
 * bitmask       uint32[rows, bitmask_ld], bitmask_ld >= ceil(V/32): allow bits,
 *               bit (i & 31) of word (i >> 5), 1 = allowed.  rows = B for
 *               ss_sample / ss_process_logits, B*(L+1) for ss_verify.
 * seed          uint64[B]  Philox4x32-10 key.
 * position      int64[B]   Philox counter position of this step.
 */
typedef struct ss_params {
  int32_t B;
  int32_t V;
  const uint32_t *mode;
  const float *temperature;
  const int32_t *top_k;
  const float *top_p;
  const float *min_p;
  const float *rep_penalty;
  const float *freq_penalty;
  const float *pres_penalty;
  const int32_t *hist_offsets;
  const int32_t *hist_ids;
  const int32_t *bias_offsets;
  const int32_t *bias_ids;
  const float *bias_vals;
  const uint32_t *bitmask;
  int64_t bitmask_ld;
  const uint64_t *seed;
  const int64_t *position;
} ss_params;

/* Workspace bytes for one call of `op` (host only, pure).  L is used by
 * SS_OP_VERIFY only; dtype is SS_F32 or SS_BF16.  Returns 0 for invalid sizes. */
size_t ss_workspace_bytes(int op, int B, int V, int L, int k_max, int dtype);

/* Zero-fills a workspace with a kernel on `stream` (no memset node).  Not
 * required before use; kept for callers that want deterministic contents. */
ss_status ss_workspace_init(void *ws, size_t ws_bytes, void *stream);

/*
 * Exact top-k per row on raw values (no prologue; Section 3.4 ordering:
 * value descending, lower index first on ties; NaN ranks as -inf and is never
 * returned; -0 returns as +0).
 *   x        [B, ld] logits of `dtype`, ld >= V.
 *   k        int32[B] per-row k (NULL: k_max for every row); clamped to [0, k_max].
 *   out_val  float[B, k_max], out_idx int32[B, k_max]: the first min(k, valid)
 *            entries, padded with (-inf, -1).
 *   flags    int32[B] or NULL.
 */
ss_status ss_topk(const void *x, int dtype, int B, int V, int64_t ld, const int32_t *k, int k_max,
                  float *out_val, int32_t *out_idx, int32_t *flags, void *ws, size_t ws_bytes,
                  void *stream);

/*
 * Singular-mode sampling (one token per request).
 *   logits      [B, ld] of `dtype`.
 *   k_max       candidate bound, 1..SS_MAX_K: the top-k cut is min(k, k_max);
 *               rows with no top-k use k_max (flag SS_FLAG_KCAP).
 *   out_token   int32[B]: sampled id; -1 if every token is masked.
 *   out_logprob float[B] or NULL: ln P(token) under the final truncated
 *               distribution (0 for greedy rows).
 *   out_idx, out_prob  int32[B, k_out], float[B, k_out] or NULL: the kept set in
 *               canonical order with its probabilities, padded (-1, 0).
 *   flags       int32[B] or NULL.
 */
ss_status ss_sample(const void *logits, int dtype, int64_t ld, const ss_params *p, int k_max,
                    int32_t *out_token, float *out_logprob, int32_t *out_idx, float *out_prob,
                    int k_out, int32_t *flags, void *ws, size_t ws_bytes, void *stream);

/*
 * Singular-mode sampling with full-row truncation (Appendix C.2 defines top-p
 * and min-p over the whole vocabulary; ss_sample bounds requests without a
 * top-k cut to their k_max leading tokens, the bounded regime of Section
 * 3.3).  For a stochastic request whose top-k bit is off (or k <= 0), top-p
 * takes its boundary against the normaliser of every valid token of the row
 * (computed in the same pass over the logits) and min-p is as ever; that
 * result is returned when the kept set holds fewer than k_max tokens.  A
 * longer kept set gives ss_sample's bounded result with SS_FLAG_KCAP.  Other
 * requests, arguments and outputs are as for ss_sample (workspace
 * ss_workspace_bytes(SS_OP_SAMPLE, ...)).
 */
ss_status ss_sample_full(const void *logits, int dtype, int64_t ld, const ss_params *p, int k_max,
                         int32_t *out_token, float *out_logprob, int32_t *out_idx, float *out_prob, int k_out,
                         int32_t *flags, void *ws, size_t ws_bytes, void *stream);

/*
 * Singular-mode sampling with the Gumbel-max draw (Appendix C.3: the argmax
 * of the perturbed logits is distributed as the categorical; the Stage-2
 * selection takes pre-drawn noise).  Everything is as for ss_sample except the
 * draw: a stochastic request's token is the kept id i with the largest
 *     (y_i - M) / tau - g_i        (in double; 0 - g_i for y_i = M),
 * the lower id on equal scores, where g = ln z, z ~ Exp(1), is drawn by the
 * caller (so results are reproducible and calls capture in graphs without an
 * RNG state).  Greedy requests ignore the noise; out_logprob is ln P(token)
 * under the truncated distribution, as for ss_sample.
 *   noise     float[B, ld_noise] (ld_noise >= V), g per token; read at the
 *             kept ids only.  NaN noise is outside the contract.
 */
ss_status ss_sample_gumbel(const void *logits, int dtype, int64_t ld, const ss_params *p, int k_max,
                           const float *noise, int64_t ld_noise, int32_t *out_token, float *out_logprob,
                           int32_t *out_idx, float *out_prob, int k_out, int32_t *flags, void *ws,
                           size_t ws_bytes, void *stream);

/*
 * Multistep speculative verification.
 *   target_logits  [B, L+1, V] rows of `dtype`, row stride ld_row (row (b, l) at
 *                  (b*(L+1) + l) * ld_row); row l is the target for draft position l+1.
 *                  Its penalty history is the request history plus drafts d_1..d_l.
 *   draft_probs    float[B, L, ld_q] draft probabilities q (used as given).
 *   draft_tokens   int32[B, L]; an id outside [0, V) ends the draft (that position
 *                  then samples the target).
 *   out_tokens     int32[B, L+1]: accepted drafts, then one correction or bonus
 *                  token, then -1.
 *   out_num_accepted int32[B] in [0, L].
 *   flags          int32[B] or NULL (OR over the request's rows).
 */
ss_status ss_verify(const void *target_logits, int dtype, int64_t ld_row, const float *draft_probs,
                    int64_t ld_q, const int32_t *draft_tokens, int L, const ss_params *p, int k_max,
                    int32_t *out_tokens, int32_t *out_num_accepted, int32_t *flags, void *ws,
                    size_t ws_bytes, void *stream);

/*
 * Multistep speculative verification against sparse draft distributions
 * (Section 3.1 with the draft probabilities a singular-mode draft step emits
 * over its candidate set, Section 3.2): position l of request b lists kq
 * (id, probability) entries, e.g. the out_idx / out_prob rows of ss_sample.
 * q_l(j) is the sum of the entries naming j; unlisted ids have q = 0, and ids
 * outside [0, V) (the padding -1 among them) are ignored.  Everything else,
 * results included, is as for ss_verify.
 *   draft_idx   int32[B, L, kq], draft_q float[B, L, kq] (used as given).
 *   kq          1..SS_MAX_K entries per draft position.
 *   ws          ss_workspace_bytes(SS_OP_VERIFY, B, V, L, k_max, dtype) bytes.
 */
ss_status ss_verify_sparse(const void *target_logits, int dtype, int64_t ld_row, const int32_t *draft_idx,
                           const float *draft_q, int kq, const int32_t *draft_tokens, int L,
                           const ss_params *p, int k_max, int32_t *out_tokens, int32_t *out_num_accepted,
                           int32_t *flags, void *ws, size_t ws_bytes, void *stream);

/*
 * Verification of one path through a draft tree (the draft-to-target mapping
 * of Appendix C.4, as tree speculation needs): the target evaluated Lt rows
 * per request for the tree's nodes, and path position l (0-based, l = L being
 * the bonus / correction position after L acceptances) is verified against
 * target row row_map[b, l].  A map entry outside [0, Lt) gives a target row
 * with every token masked (SS_FLAG_EMPTY: the path ends there with no
 * correction token).  Draft lists are sparse, as for ss_verify_sparse.  The
 * penalty history, the grammar rows (bitmask rows B*(L+1), one per path
 * position), the uniforms and the outputs follow the path, as for ss_verify.
 *   target_logits  [B, Lt, V] rows of `dtype`, row stride ld_row (request b's
 *                  row t at (b*Lt + t) * ld_row).
 *   Lt             target rows per request, >= 1.
 *   row_map        int32[B, L+1].
 *   ws             ss_workspace_bytes(SS_OP_VERIFY, B, V, L, k_max, dtype) bytes.
 */
ss_status ss_verify_tree(const void *target_logits, int dtype, int64_t ld_row, int Lt, const int32_t *row_map,
                         const int32_t *draft_idx, const float *draft_q, int kq, const int32_t *draft_tokens,
                         int L, const ss_params *p, int k_max, int32_t *out_tokens, int32_t *out_num_accepted,
                         int32_t *flags, void *ws, size_t ws_bytes, void *stream);

/*
 * Materialised pipeline (unfused reference path).
 *   out_logits float[B, V] (row stride V): processed logits y before temperature
 *              (-inf where masked).  May be NULL.
 *   out_probs  float[B, V] (row stride V): final truncated distribution (zero
 *              outside the kept set; one-hot at the argmax for greedy rows).  May be NULL.
 */
ss_status ss_process_logits(const void *logits, int dtype, int64_t ld, const ss_params *p, int k_max,
                            float *out_logits, float *out_probs, int32_t *flags, void *ws,
                            size_t ws_bytes, void *stream);

/*
 * Top-k log-probabilities (indicator bit SS_LOGPROBS = 0x400 of the
 * bit-level encoding table, Section 3.5; the log-probability output of
 * Alg. 11).  For every request whose mode has the bit: the n_lp leading
 * tokens of the canonical order of its processed logits y (the Appendix C.1
 * prologue: grammar mask, penalties, bias; value descending, lower index
 * first) and their log-probabilities under the untruncated distribution
 * softmax(y / tau) over all valid tokens of the row:
 *     lp_i = (y_i - M) / tau - ln sum_j exp((y_j - M) / tau),   M = max_j y_j,
 * tau being the request's temperature when SS_TEMP is set, tau > 0 and the
 * request is not greedy, else 1.  Top-k, top-p and min-p do not apply.
 *   logits    [B, ld] of `dtype`.
 *   n_lp      1..SS_MAX_K entries per request.
 *   out_idx   int32[B, n_lp], out_lp float[B, n_lp]: padded with (-1, -inf)
 *             beyond the valid tokens and for requests without the bit.
 *   flags     int32[B] or NULL.
 *   ws        ss_workspace_bytes(SS_OP_LOGPROBS, B, V, 0, n_lp, dtype) bytes.
 * The normaliser's terms are float32 exponentials summed in double
 * (relative error below about 2e-7).
 */
ss_status ss_logprobs(const void *logits, int dtype, int64_t ld, const ss_params *p, int n_lp,
                      int32_t *out_idx, float *out_lp, int32_t *flags, void *ws, size_t ws_bytes,
                      void *stream);

/*
 * ss_sample with no workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, serving loops and harnesses
 * that forbid allocation).  The workspace is an SS_NOALLOC_BYTES array in the
 * library's device memory, one copy per GPU, held until the process ends;
 * this call allocates and frees nothing.  Arguments and results are those of
 * ss_sample.  SS_ERR_WORKSPACE when ss_workspace_bytes(SS_OP_SAMPLE, B, V, 0,
 * k_max, dtype) exceeds SS_NOALLOC_BYTES (B = 64, V = 2^17, k_max = 1024
 * fits).  Every call on one GPU uses that GPU's single array: calls that
 * overlap in time on one GPU (other streams, other threads) race.
 */
#define SS_NOALLOC_BYTES (48u << 20)
ss_status ss_sample_noalloc(const void *logits, int dtype, int64_t ld, const ss_params *p, int k_max,
                            int32_t *out_token, float *out_logprob, int32_t *out_idx, float *out_prob,
                            int k_out, int32_t *flags, void *stream);

const char *ss_status_string(ss_status s);

#ifdef __cplusplus
}
#endif
#endif /* SS_H_ */
