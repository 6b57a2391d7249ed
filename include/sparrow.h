/*
 * sparrow.h - C ABI of the MI355X (gfx950) sparse-decode attention library.
 *
 * One decode step of one attention layer over a paged KV cache, as used by
 * sparse rollout in Sparrow (arXiv 2606.08446):
 *
 *   1. sparrow_page_meta_update   per-page key min/max metadata (the page
 *                                 landmark scored in Sec. 3.3 / Appendix C),
 *                                 or sparrow_append_kv: write the decoded token's
 *                                 K/V and update its page's metadata in O(1),
 *   2. sparrow_page_score_topk    page scores against the current query, the
 *                                 per-sequence page budget from the dynamic
 *                                 sparsity schedule (Sec. 3.2 Method box) and
 *                                 the block top-k page selection (Sec. 2,
 *                                 Appendix D: block top-k attention),
 *   3. sparrow_sparse_decode_attn softmax attention over the selected pages only
 *                                 (the "sparse, no scoring" term of the sparse
 *                                 cost model, Eq. sparse-cost),
 *   4. sparrow_dense_decode_attn  the dense paged decode it is measured against
 *                                 (Eq. dense-cost).
 *   sparrow_append_score_topk fuses the append into step 2, and
 *   sparrow_decode_step runs the append and steps 2 and 3 in one call.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Every array argument is a DEVICE pointer owned by the caller.  The library
 *    allocates nothing, keeps no state between calls and never synchronises:
 *    each call only validates its host-visible arguments and enqueues kernels
 *    on `stream` (a hipStream_t passed as void*; NULL = the null stream).
 *  - Return value: SPARROW_OK (0) or a negative status (see below).  Nothing is
 *    enqueued when a negative status is returned.  Device contents are checked
 *    only where an index could leave a buffer: a block-table entry outside
 *    [0, num_phys_pages) marks an absent page - no kernel reads or writes that
 *    physical page; scoring sees zero metadata for it (score 0), attention
 *    leaves its tokens out, and an append to it writes nothing - and page
 *    indices, lengths and budgets are clamped to what the shape allows (a
 *    negative length is an empty sequence; one beyond max_pages_per_seq *
 *    page_size tokens counts as that many, and its token is not appended).
 *  - bf16 tensors are IEEE bfloat16 bit patterns.  NaN inputs are not supported.
 *  - Alignment: q, k_cache, v_cache, meta, out and workspace start on a 16-byte
 *    boundary and the int32 arrays on a 4-byte boundary (any hipMalloc or PyTorch
 *    allocation is); a misaligned pointer is rejected with SPARROW_EINVAL.
 *  - Layouts (row-major, no padding):
 *      q            bf16  [batch][num_q_heads][head_dim]
 *      k_cache      bf16  [num_phys_pages][num_kv_heads][page_size][head_dim]
 *      v_cache      bf16  [num_phys_pages][num_kv_heads][page_size][head_dim]
 *      meta         bf16  [num_phys_pages][num_kv_heads][2][head_dim]
 *                         (row 0: channel-wise min, row 1: channel-wise max), or with
 *                         SPARROW_LANDMARK_MEAN fp32 [num_phys_pages][num_kv_heads][head_dim]
 *                         (channel-wise sum of the page's valid keys) - 512 B per
 *                         (page, head) either way
 *      block_table  int32 [batch][max_pages_per_seq]  logical -> physical page
 *      seq_lens     int32 [batch]  tokens of each sequence, including the token
 *                                  being decoded (0 allowed)
 *      idx          int32 [batch][num_kv_heads][k_max]  selected logical pages
 *      out          fp32 or bf16 [batch][num_q_heads][head_dim]
 *    Sequence b uses logical pages 0 .. ceil(seq_lens[b] / page_size) - 1; the
 *    rest of its block-table row may be read (the array must be whole) but its
 *    values never matter.  Query head j reads KV head
 *    j / G with G = num_q_heads / num_kv_heads (grouped-query attention).
 *  - Supported shapes: head_dim == 128; page_size in {16, 32, 64, 128};
 *    landmark in {SPARROW_LANDMARK_MINMAX, SPARROW_LANDMARK_MEAN};
 *    num_q_heads a multiple of num_kv_heads with G <= 16;
 *    1 <= max_pages_per_seq <= SPARROW_MAX_PAGES_PER_SEQ;
 *    batch * num_kv_heads <= 65535; batch <= SPARROW_MAX_BATCH for the
 *    scoring and attention entry points.
 */
#ifndef SPARROW_H
#define SPARROW_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SPARROW_OK 0
#define SPARROW_EINVAL (-1)       /* null pointer, negative or inconsistent size      */
#define SPARROW_EUNSUPPORTED (-2) /* head_dim, page size, group size or dtype not supported */
#define SPARROW_EWORKSPACE (-3)   /* workspace missing or smaller than required       */
#define SPARROW_EHIP (-4)         /* a kernel launch failed                           */

#define SPARROW_MAX_PAGES_PER_SEQ 15360
#define SPARROW_MAX_BATCH 8192

#define SPARROW_OUT_F32 0
#define SPARROW_OUT_BF16 1

#define SPARROW_LANDMARK_MINMAX 0 /* per page: channel-wise min and max of the keys (bf16)  */
#define SPARROW_LANDMARK_MEAN 1   /* per page: channel-wise sum of the keys (fp32); scored
                                     as the mean key                                       */

#define SPARROW_LOGITS_F32 0
#define SPARROW_LOGITS_BF16 1

#define SPARROW_OP_SCORE_TOPK 0
#define SPARROW_OP_SPARSE_ATTN 1
#define SPARROW_OP_DENSE_ATTN 2
#define SPARROW_OP_DECODE_STEP 3

/* Shape of one layer's decode batch (host struct, read during the call only).
   `landmark` selects the page metadata (SPARROW_LANDMARK_*; 0 = min/max), used by the
   metadata, append and scoring entry points and ignored by attention. */
typedef struct sparrow_shape {
    int32_t batch;
    int32_t num_q_heads;
    int32_t num_kv_heads;
    int32_t head_dim;
    int32_t page_size;
    int32_t max_pages_per_seq;
    int64_t num_phys_pages;
    int32_t landmark;
} sparrow_shape_t;

/*
 * Dynamic sparsity schedule (Sec. 3.2 Method box: the budget grows with the
 * current length so that the tail acceptance rate stays constant; lengths are
 * grouped into bins of 2K tokens in the paper).  Host struct whose two tables
 * are DEVICE arrays of n_bins int32.  For a sequence of L >= 1 tokens and
 * n = ceil(L / page_size) pages:
 *     bin = min((L - 1) / bin_tokens, n_bins - 1)
 *     k   = clamp(max(min_pages[bin], ceil(n * frac_num[bin] / frac_den)), 1, n)
 * and k = 0 for L = 0.  A fixed budget is min_pages = {P}, frac_num = {0}; a
 * fixed fraction is min_pages = {0}, frac_num = {num}, frac_den = den.  When
 * k == n every page is kept (Appendix F: attention is dense while the context
 * fits the budget).  Requires bin_tokens >= 1, n_bins >= 1, frac_den >= 1 and
 * non-negative table entries.
 *
 * sink_pages s and local_pages l (0 = pure top-k) force the logical pages
 * [0, s) (attention sinks) and [n - l, n) (the most recent pages) into the
 * selection ahead of every scored page, lower index first; the rest of the budget
 * k goes by score.  Both >= 0.
 */
typedef struct sparrow_schedule {
    int32_t bin_tokens;
    int32_t n_bins;
    const int32_t *min_pages;
    const int32_t *frac_num;
    int32_t frac_den;
    int32_t sink_pages;
    int32_t local_pages;
} sparrow_schedule_t;

/*
 * Per-page key metadata (Sec. 3.3 and Appendix C: landmark scores; the
 * landmark is the channel-wise min and max of the page's keys).
 *
 * For every sequence b and every logical page p that overlaps the token range
 * [first_pos[b], seq_lens[b]), and for every KV head h and channel i:
 *     meta[phys][h][0][i] = min over the valid tokens t of the page of K[t][i]
 *     meta[phys][h][1][i] = max over the same tokens
 * (SPARROW_LANDMARK_MEAN: meta[phys][h][i] = the fp32 sum of K[t][i] over the same
 * tokens, added in token order)
 * where phys = block_table[b][p] and the valid tokens of page p are
 * p*page_size .. min((p+1)*page_size, seq_lens[b]) - 1.  Values are copied
 * exactly (bf16 in, bf16 out); -0 orders below +0.  first_pos == NULL rebuilds
 * every page of every sequence.  A decode step that has just written token
 * L-1 passes first_pos[b] = L-1.  Entries of first_pos below 0 are treated as
 * 0; entries >= seq_lens[b] update nothing.
 *
 * Arguments: shape (host), k_cache (device, layout above), block_table,
 * seq_lens, first_pos (device [batch] or NULL), meta (device, written), stream.
 * Errors: SPARROW_EINVAL for a null shape/k_cache/block_table/seq_lens/meta or
 * a bad size; SPARROW_EUNSUPPORTED for head_dim/page_size; SPARROW_EHIP.
 */
int sparrow_page_meta_update(const sparrow_shape_t *shape, const void *k_cache,
                             const int32_t *block_table, const int32_t *seq_lens,
                             const int32_t *first_pos, void *meta, void *stream);

/*
 * Appending the token being decoded (the per-token landmark upkeep of Sec. 3.3:
 * the page metadata follows every generated key).
 *
 * seq_lens[b] counts the new token, which goes to position L - 1 = seq_lens[b] - 1:
 * logical page (L - 1) / page_size, slot (L - 1) % page_size.  For every KV head h:
 *     k_cache[phys][h][slot][:] = k_new[b][h][:],  v_cache[phys][h][slot][:] = v_new[b][h][:]
 * with phys = block_table[b][(L - 1) / page_size], and the page's metadata becomes the
 * channel-wise min/max of its old metadata and the new key (the key itself when the
 * slot is 0); with SPARROW_LANDMARK_MEAN its key sum plus the new key.  This equals
 * the metadata rebuilt from the page's L - page*page_size valid tokens
 * (sparrow_page_meta_update) provided the old metadata described the tokens before
 * L - 1.  Sequences with seq_lens[b] < 1 or seq_lens[b] > max_pages_per_seq *
 * page_size are left untouched.  Sequences must use distinct physical pages.
 *
 * Arguments: shape (host); k_new, v_new (device bf16 [batch][num_kv_heads][head_dim]);
 * k_cache, v_cache, meta (device, updated in place); block_table, seq_lens (device);
 * stream.
 * Errors: SPARROW_EINVAL (null or misaligned pointer, bad size), SPARROW_EUNSUPPORTED,
 * SPARROW_EHIP.
 */
int sparrow_append_kv(const sparrow_shape_t *shape, const void *k_new, const void *v_new,
                      void *k_cache, void *v_cache, const int32_t *block_table,
                      const int32_t *seq_lens, void *meta, void *stream);

/*
 * Page scoring and block top-k selection (Sec. 3.3: landmark scores and top-k
 * page picking; Sec. 3.2: the budget from the sparsity schedule).
 *
 * For every sequence b and KV head h, each logical page p < n_b is scored
 *     S_h(p) = sum over the G query heads j of head h of
 *              sum_i max(q[b][j][i] * mn_i(p), q[b][j][i] * mx_i(p))
 * (an upper bound of q_j . k_t over the tokens of the page), with fp32
 * arithmetic; with SPARROW_LANDMARK_MEAN, S_h(p) = sum_j q_j . (sum(p) / n_valid(p)),
 * the query group against the page's mean key.  k_b is the schedule's budget (see
 * sparrow_schedule_t), capped at k_max.  The k_b pages of largest S_h are kept, ties going to the lower
 * page index (-0 equals +0), and written in ascending page order to
 * out_idx[b][h][0 .. k_b); the rest of the row up to k_max is set to -1.
 * out_k[b] = k_b.  When k_b == n_b no page is scored and every page is kept.
 *
 * Arguments: shape (host); q, meta, block_table, seq_lens (device);
 * schedule (host struct with device tables); 1 <= k_max <= SPARROW_MAX_PAGES_PER_SEQ
 * (the row length of out_idx; callers pass at least the largest budget); out_k (device [batch]);
 * out_idx (device [batch][num_kv_heads][k_max]); workspace of at least
 * sparrow_workspace_size(shape, k_max, SPARROW_OP_SCORE_TOPK) bytes (device,
 * contents need not be initialised); stream.
 * Errors: SPARROW_EINVAL (null pointers, k_max out of range, bad schedule sizes or negative
 * forced-page counts), SPARROW_EUNSUPPORTED, SPARROW_EWORKSPACE, SPARROW_EHIP.
 */
int sparrow_page_score_topk(const sparrow_shape_t *shape, const void *q, const void *meta,
                            const int32_t *block_table, const int32_t *seq_lens,
                            const sparrow_schedule_t *schedule, int32_t k_max, int32_t *out_k,
                            int32_t *out_idx, void *workspace, size_t ws_bytes, void *stream);

/*
 * sparrow_append_kv followed by sparrow_page_score_topk, in one pass: the scoring
 * kernel's workgroup that owns a sequence's last page writes the new K/V rows and that
 * page's metadata and scores the page from the updated metadata, so no separate
 * metadata pass runs.  Results (caches, meta, out_k, out_idx) are identical to the two
 * calls in sequence.  Arguments are those of the two calls; the workspace is that of
 * SPARROW_OP_SCORE_TOPK.
 * Errors: as sparrow_page_score_topk, plus SPARROW_EINVAL for a null or misaligned
 * k_new, v_new, k_cache or v_cache.
 */
int sparrow_append_score_topk(const sparrow_shape_t *shape, const void *q, const void *k_new,
                              const void *v_new, void *k_cache, void *v_cache, void *meta,
                              const int32_t *block_table, const int32_t *seq_lens,
                              const sparrow_schedule_t *schedule, int32_t k_max, int32_t *out_k,
                              int32_t *out_idx, void *workspace, size_t ws_bytes, void *stream);

/*
 * Sparse decode attention over the selected pages (block-sparse attention,
 * Sec. 2; the attention term of Eq. sparse-cost).
 *
 * For every sequence b and query head j (KV head h = j / G) the token set T is
 * the valid tokens of the pages idx[b][h][0 .. min(k[b], k_max)); entries
 * outside [0, n_b) are skipped.  Then
 *     z_t = scale * (q[b][j] . K[t]),  w_t = exp(z_t - max z) / sum exp(z - max z)
 *     out[b][j] = sum_t w_t V[t]
 * computed with bf16 operands and fp32 accumulation (the softmax weights are
 * rounded to bf16 before they multiply V).  An empty token set gives a zero
 * row.  out_dtype is SPARROW_OUT_F32 or SPARROW_OUT_BF16.
 * The order of the fp32 sums depends only on the shape, k_max, the page lists
 * and the device (its count of resident waves), so repeated calls on one GPU
 * give identical results.  A call with at most 256
 * (sequence, KV head) units, at most 8 query heads per KV head,
 * k_max * page_size <= 1024 and max_pages_per_seq <= 4096 runs one workgroup
 * per unit and leaves the workspace untouched; larger calls split the lists
 * over all resident waves and merge partials kept in the workspace.  With every page listed and k_max
 * equal to max_pages_per_seq the result equals sparrow_dense_decode_attn's bit
 * for bit (the dense call's list bound is max_pages_per_seq).
 *
 * Arguments: shape (host); q, k_cache, v_cache, block_table, seq_lens, k
 * (device [batch]), idx (device [batch][num_kv_heads][k_max]);
 * 1 <= k_max <= SPARROW_MAX_PAGES_PER_SEQ;
 * scale (typically 1/sqrt(head_dim)); out (device, written); out_dtype;
 * workspace of at least sparrow_workspace_size(shape, k_max,
 * SPARROW_OP_SPARSE_ATTN) bytes; stream.
 * Errors: SPARROW_EINVAL, SPARROW_EUNSUPPORTED, SPARROW_EWORKSPACE, SPARROW_EHIP.
 */
int sparrow_sparse_decode_attn(const sparrow_shape_t *shape, const void *q, const void *k_cache,
                               const void *v_cache, const int32_t *block_table,
                               const int32_t *seq_lens, const int32_t *k, const int32_t *idx,
                               int32_t k_max, float scale, void *out, int32_t out_dtype,
                               void *workspace, size_t ws_bytes, void *stream);

/*
 * sparrow_sparse_decode_attn for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation): the same
 * computation and results, with the workspace taken from a buffer of
 * SPARROW_NOALLOC_SCRATCH_BYTES that the library holds on each GPU it runs on (from the
 * first call on that GPU until the process ends).  The call allocates nothing.
 *
 * Every call on one GPU uses that GPU's buffer: calls that can overlap on one GPU (on
 * different streams, or from several host threads without ordering) race and must not be
 * issued; calls in one stream are ordered and safe.  The buffer needs no initialisation.
 * Shapes whose workspace (sparrow_workspace_size with SPARROW_OP_SPARSE_ATTN) exceeds
 * SPARROW_NOALLOC_SCRATCH_BYTES are refused with SPARROW_EWORKSPACE; the Qwen3-shaped decode
 * batches here need 5-13 MiB.
 *
 * Arguments and the other errors are those of sparrow_sparse_decode_attn without the
 * workspace; SPARROW_EHIP also when the buffer's address cannot be obtained.
 */
#define SPARROW_NOALLOC_SCRATCH_BYTES 33554432 /* 32 MiB */
int sparrow_sparse_decode_attn_noalloc(const sparrow_shape_t *shape, const void *q,
                                       const void *k_cache, const void *v_cache,
                                       const int32_t *block_table, const int32_t *seq_lens,
                                       const int32_t *k, const int32_t *idx, int32_t k_max,
                                       float scale, void *out, int32_t out_dtype, void *stream);

/*
 * One decode step of one layer in one call (the whole sparse step of Sec. 3.3:
 * append, landmark scores, the schedule's budget of Sec. 3.2, block top-k and
 * attention over the selected pages): sparrow_append_score_topk - or
 * sparrow_page_score_topk when k_new and v_new are both NULL - followed by
 * sparrow_sparse_decode_attn on the selection it made (k = out_k, idx =
 * out_idx).  Results (caches, meta, out_k, out_idx, out) equal those of the two
 * calls in sequence bit for bit.  When the attention call would run one
 * workgroup per unit (see sparrow_sparse_decode_attn), the budget, the top-k
 * and the attention run in one kernel after the scoring kernel, with the
 * selection kept on chip: two launches instead of three.
 *
 * Arguments: those of the two calls (k_new and v_new both NULL or both set);
 * workspace of at least sparrow_workspace_size(shape, k_max,
 * SPARROW_OP_DECODE_STEP) bytes.
 * Errors: those of the two calls.
 */
int sparrow_decode_step(const sparrow_shape_t *shape, const void *q, const void *k_new,
                        const void *v_new, void *k_cache, void *v_cache, void *meta,
                        const int32_t *block_table, const int32_t *seq_lens,
                        const sparrow_schedule_t *schedule, int32_t k_max, float scale,
                        int32_t *out_k, int32_t *out_idx, void *out, int32_t out_dtype,
                        void *workspace, size_t ws_bytes, void *stream);

/*
 * Dense paged decode attention (the dense rollout baseline, Eq. dense-cost):
 * the same as sparrow_sparse_decode_attn with T = every valid token of the
 * sequence, and max_pages_per_seq in place of k_max when choosing between one
 * workgroup per unit and the streaming split.
 *
 * Arguments as above, without k/idx/k_max; workspace of at least
 * sparrow_workspace_size(shape, 0, SPARROW_OP_DENSE_ATTN) bytes.
 * Errors: SPARROW_EINVAL, SPARROW_EUNSUPPORTED, SPARROW_EWORKSPACE, SPARROW_EHIP.
 */
int sparrow_dense_decode_attn(const sparrow_shape_t *shape, const void *q, const void *k_cache,
                              const void *v_cache, const int32_t *block_table,
                              const int32_t *seq_lens, float scale, void *out, int32_t out_dtype,
                              void *workspace, size_t ws_bytes, void *stream);

/*
 * Per-token acceptance rate between the dense policy and the sparse rollout
 * (Sec. 3.1, Eq. 1: the expectation under the draft of min(p/q, 1), which equals
 * the sum over the vocabulary of min(p(x), q(x))).
 *
 * For every token t < num_tokens, with a = target_logits[t][:] (dense policy) and
 * b = draft_logits[t][:] (sparse rollout), rows of `vocab` entries:
 *     p = softmax(inv_temperature * a),  q = softmax(inv_temperature * b),
 *     alpha[t] = sum_x min(p(x), q(x))
 * computed in fp32 (two passes: log-sum-exp of both rows, then the sum).  Agrees
 * with an fp64 evaluation to about 1e-5.  A logit of -inf (a masked vocabulary entry)
 * has probability 0; each row needs at least one finite logit, and -inf entries need
 * inv_temperature > 0.  NaN and +inf logits are not supported.  logits_dtype is SPARROW_LOGITS_F32 or
 * SPARROW_LOGITS_BF16; rows are contiguous ([num_tokens][vocab], row-major).
 *
 * Arguments: num_tokens >= 0; vocab >= 1; target_logits, draft_logits (device,
 * element-aligned); inv_temperature finite; alpha (device fp32 [num_tokens],
 * written); stream.
 * Errors: SPARROW_EINVAL (null/misaligned pointer, bad size, non-finite
 * temperature), SPARROW_EUNSUPPORTED (dtype), SPARROW_EHIP.
 */
int sparrow_acceptance_rate(int64_t num_tokens, int32_t vocab, int32_t logits_dtype,
                            const void *target_logits, const void *draft_logits,
                            float inv_temperature, float *alpha, void *stream);

/*
 * The approximation of the paper's measurement (Sec. 3.1, footnote: the inference
 * engine returns the top-20 tokens and their log-probabilities per position):
 *     alpha[t] = sum_{i < k} min(exp(lp_target[t][i]), exp(lp_draft[t][i]))
 * over the k listed tokens, whose normalised log-probabilities under the two
 * distributions are given (fp32 [num_tokens][k], device).  A lower bound of the
 * exact rate.
 * Errors: SPARROW_EINVAL (null/misaligned pointer, num_tokens < 0, k < 1), SPARROW_EHIP.
 */
int sparrow_acceptance_rate_topk(int64_t num_tokens, int32_t k, const float *lp_target,
                                 const float *lp_draft, float *alpha, void *stream);

/*
 * Lower-tail statistic of the acceptance rate per length bin (Sec. 3.1 Method:
 * the 5-percentile of the per-token rate; Sec. 3.2: tokens grouped by position
 * in 2K-token bins).
 *
 * Token t (alpha[t], positions[t]) belongs to bin min(positions[t] / bin_tokens,
 * n_bins - 1); tokens with a negative position are ignored.  For each bin b:
 * count[b] = its number of tokens N, mean[b] = the fp64 mean of their alpha, and
 * quantile[b] = the `percentile`-percentile with linear interpolation between
 * order statistics: with the values sorted x_0 <= ... <= x_{N-1},
 * h = (N - 1) * percentile / 100, lo = floor(h),
 * quantile = x_lo + (h - lo) * (x_{lo+1} - x_lo)   (x_lo when lo = N - 1),
 * in fp64.  Empty bins get count 0 and NaN mean and quantile.
 *
 * Arguments: num_tokens >= 0; alpha (device fp32), positions (device int32), both
 * may be NULL when num_tokens is 0;
 * bin_tokens >= 1; 1 <= n_bins <= 65535; 0 <= percentile <= 100; quantile,
 * mean (device fp64 [n_bins]) and count (device int64 [n_bins]), written; stream.
 * Errors: SPARROW_EINVAL, SPARROW_EHIP.
 */
int sparrow_tail_stats(int64_t num_tokens, const float *alpha, const int32_t *positions,
                       int32_t bin_tokens, int32_t n_bins, double percentile, double *quantile,
                       double *mean, int64_t *count, void *stream);

/*
 * Read-only streaming reference (a measurement helper, not a step of the method): reads
 * `bytes` bytes at src once, with the 16-byte non-temporal vector loads and the
 * consecutive-lanes layout of the decode-step kernels, from a grid that keeps every
 * compute unit busy, and adds every 32-bit word of the buffer into *checksum (modulo
 * 2^32, on top of its current value: the caller sets it, usually to 0).  Timing a call
 * gives the rate a pure read stream sustains on the device, the practical ceiling of the
 * read-dominated decode kernels beside the HBM peak.
 *
 * Arguments: src (device, 16-byte aligned, may be NULL when bytes is 0); bytes >= 0, a
 * multiple of 16; checksum (device uint32, 4-byte aligned); stream.
 * Errors: SPARROW_EINVAL (null or misaligned pointer, bad size), SPARROW_EHIP.
 */
int sparrow_stream_read(const void *src, int64_t bytes, uint32_t *checksum, void *stream);

/*
 * Host-side page budgets of the dynamic sparsity schedule (Sec. 3.2 Method box; the
 * formula of sparrow_schedule_t, evaluated by the same code the scoring kernels use), to
 * size k_max before a call of sparrow_page_score_topk or sparrow_append_score_topk.
 *
 * For every b < num_seqs: budgets[b] = k_b of a sequence of seq_lens[b] tokens (0 when
 * seq_lens[b] <= 0), not capped by any k_max.  Returns max(1, max_b k_b), the smallest
 * k_max that caps no budget, or a negative status.
 *
 * Arguments: seq_lens (HOST int32 [num_seqs], may be NULL when num_seqs is 0); num_seqs
 * >= 0; page_size >= 1; bin_tokens >= 1; n_bins >= 1; min_pages, frac_num (HOST int32
 * [n_bins], non-negative); frac_den >= 1; budgets (HOST int32 [num_seqs], written) or
 * NULL.  Every pointer is a host pointer; nothing runs on the GPU.
 * Errors: SPARROW_EINVAL (bad size, null table, negative table entry, or a length above
 * page_size * SPARROW_MAX_PAGES_PER_SEQ).
 */
int32_t sparrow_budget_bound(const int32_t *seq_lens, int64_t num_seqs, int32_t page_size,
                             int32_t bin_tokens, int32_t n_bins, const int32_t *min_pages,
                             const int32_t *frac_num, int32_t frac_den, int32_t *budgets);

/*
 * Workspace bytes needed by one call of `op` (SPARROW_OP_*: SCORE_TOPK for the
 * two scoring calls, SPARSE_ATTN, DENSE_ATTN, DECODE_STEP) with this shape
 * and k_max (ignored for SPARROW_OP_DENSE_ATTN).  Returns 0 for an invalid or
 * unsupported shape.  The workspace holds scratch results of one call only;
 * calls that run concurrently need separate workspaces.
 */
size_t sparrow_workspace_size(const sparrow_shape_t *shape, int32_t k_max, int32_t op);

/* Static, human-readable name of a status code. */
const char *sparrow_status_string(int32_t status);

#ifdef __cplusplus
}
#endif

#endif /* SPARROW_H */
