// C ABI of libsparrow: argument validation, workspace sizing and kernel launches.
// Declarations and the contract of every entry point are in include/sparrow.h.
#include <cmath>

#include "common.h"

using namespace sparrow;

namespace {

int check_shape(const sparrow_shape_t *s)
{
    if (!s)
        return SPARROW_EINVAL;
    if (s->batch < 0 || s->num_q_heads < 1 || s->num_kv_heads < 1 || s->max_pages_per_seq < 1 ||
        s->num_phys_pages < 1)
        return SPARROW_EINVAL;
    if (s->num_q_heads % s->num_kv_heads != 0)
        return SPARROW_EINVAL;
    if (s->num_q_heads / s->num_kv_heads > 16)
        return SPARROW_EUNSUPPORTED;
    if (s->head_dim != kHeadDim)
        return SPARROW_EUNSUPPORTED;
    if (s->page_size != 16 && s->page_size != 32 && s->page_size != 64 && s->page_size != 128)
        return SPARROW_EUNSUPPORTED;
    if (s->max_pages_per_seq > SPARROW_MAX_PAGES_PER_SEQ)
        return SPARROW_EUNSUPPORTED;
    if (s->landmark != SPARROW_LANDMARK_MINMAX && s->landmark != SPARROW_LANDMARK_MEAN)
        return SPARROW_EUNSUPPORTED;
    if ((int64_t)s->batch * s->num_q_heads > 0x7fffffff / kHeadDim)
        return SPARROW_EINVAL;
    return SPARROW_OK;
}

// The kernels move bf16/fp32 data in 16-byte vectors and indices as int32.
bool al16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool al4(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

int status_of(hipError_t e) { return e == hipSuccess ? SPARROW_OK : SPARROW_EHIP; }

size_t round256(size_t n) { return (n + 255) / 256 * 256; }

// sparrow_decode_step's workspace: the scores, then the attention's workspace.
size_t decode_step_workspace(const sparrow_shape_t &s)
{
    return round256(score_topk_workspace(s)) + plan_attention(s).workspace_bytes;
}

}  // namespace

extern "C" {

int sparrow_page_meta_update(const sparrow_shape_t *shape, const void *k_cache,
                             const int32_t *block_table, const int32_t *seq_lens,
                             const int32_t *first_pos, void *meta, void *stream)
{
    const int rc = check_shape(shape);
    if (rc != SPARROW_OK)
        return rc;
    if (!k_cache || !block_table || !seq_lens || !meta)
        return SPARROW_EINVAL;
    if (!al16(k_cache) || !al16(meta) || !al4(block_table) || !al4(seq_lens) || !al4(first_pos))
        return SPARROW_EINVAL;
    if (shape->batch == 0)
        return SPARROW_OK;
    if (first_pos == nullptr && shape->batch > 65535)
        return SPARROW_EINVAL;
    return status_of(launch_meta_update(*shape, k_cache, block_table, seq_lens, first_pos, meta,
                                        static_cast<hipStream_t>(stream)));
}

int sparrow_append_kv(const sparrow_shape_t *shape, const void *k_new, const void *v_new,
                      void *k_cache, void *v_cache, const int32_t *block_table,
                      const int32_t *seq_lens, void *meta, void *stream)
{
    const int rc = check_shape(shape);
    if (rc != SPARROW_OK)
        return rc;
    if (!k_new || !v_new || !k_cache || !v_cache || !block_table || !seq_lens || !meta)
        return SPARROW_EINVAL;
    if (!al16(k_new) || !al16(v_new) || !al16(k_cache) || !al16(v_cache) || !al16(meta) ||
        !al4(block_table) || !al4(seq_lens))
        return SPARROW_EINVAL;
    if (shape->batch == 0)
        return SPARROW_OK;
    return status_of(launch_append_kv(*shape, k_new, v_new, k_cache, v_cache, block_table,
                                      seq_lens, meta, static_cast<hipStream_t>(stream)));
}

// Shared by sparrow_page_score_topk and sparrow_append_score_topk.
static int score_topk_call(const sparrow_shape_t *shape, const void *q, void *meta,
                           const int32_t *block_table, const int32_t *seq_lens,
                           const sparrow_schedule_t *schedule, int32_t k_max, int32_t *out_k,
                           int32_t *out_idx, void *workspace, size_t ws_bytes,
                           const AppendArgs &app, void *stream)
{
    const int rc = check_shape(shape);
    if (rc != SPARROW_OK)
        return rc;
    if (!q || !meta || !block_table || !seq_lens || !schedule || !out_k || !out_idx)
        return SPARROW_EINVAL;
    if (!al16(q) || !al16(meta) || !al4(block_table) || !al4(seq_lens) || !al4(out_k) ||
        !al4(out_idx) || !al16(workspace))
        return SPARROW_EINVAL;
    if (k_max < 1 || k_max > SPARROW_MAX_PAGES_PER_SEQ || schedule->bin_tokens < 1 || schedule->n_bins < 1 || schedule->frac_den < 1 ||
        !schedule->min_pages || !schedule->frac_num || schedule->sink_pages < 0 ||
        schedule->local_pages < 0)
        return SPARROW_EINVAL;
    if (shape->batch == 0)
        return SPARROW_OK;
    if ((int64_t)shape->batch * shape->num_kv_heads > 65535)
        return SPARROW_EINVAL;
    if (shape->batch > kMaxBatch)
        return SPARROW_EUNSUPPORTED;
    if (!workspace || ws_bytes < score_topk_workspace(*shape))
        return SPARROW_EWORKSPACE;
    Sched sched{schedule->bin_tokens, schedule->n_bins,     schedule->frac_den,
                schedule->min_pages,  schedule->frac_num, schedule->sink_pages,
                schedule->local_pages};
    return status_of(launch_score_topk(*shape, q, meta, block_table, seq_lens, sched, k_max,
                                       out_k, out_idx, workspace, app,
                                       static_cast<hipStream_t>(stream)));
}

int sparrow_page_score_topk(const sparrow_shape_t *shape, const void *q, const void *meta,
                            const int32_t *block_table, const int32_t *seq_lens,
                            const sparrow_schedule_t *schedule, int32_t k_max, int32_t *out_k,
                            int32_t *out_idx, void *workspace, size_t ws_bytes, void *stream)
{
    const AppendArgs none{nullptr, nullptr, nullptr, nullptr};
    // Without an append the kernel only reads the metadata.
    return score_topk_call(shape, q, const_cast<void *>(meta), block_table, seq_lens, schedule,
                           k_max, out_k, out_idx, workspace, ws_bytes, none, stream);
}

int sparrow_append_score_topk(const sparrow_shape_t *shape, const void *q, const void *k_new,
                              const void *v_new, void *k_cache, void *v_cache, void *meta,
                              const int32_t *block_table, const int32_t *seq_lens,
                              const sparrow_schedule_t *schedule, int32_t k_max, int32_t *out_k,
                              int32_t *out_idx, void *workspace, size_t ws_bytes, void *stream)
{
    const int rc = check_shape(shape);
    if (rc != SPARROW_OK)
        return rc;
    if (!k_new || !v_new || !k_cache || !v_cache)
        return SPARROW_EINVAL;
    if (!al16(k_new) || !al16(v_new) || !al16(k_cache) || !al16(v_cache))
        return SPARROW_EINVAL;
    const AppendArgs app{k_new, v_new, k_cache, v_cache};
    return score_topk_call(shape, q, meta, block_table, seq_lens, schedule, k_max, out_k, out_idx,
                           workspace, ws_bytes, app, stream);
}

int sparrow_sparse_decode_attn(const sparrow_shape_t *shape, const void *q, const void *k_cache,
                               const void *v_cache, const int32_t *block_table,
                               const int32_t *seq_lens, const int32_t *k, const int32_t *idx,
                               int32_t k_max, float scale, void *out, int32_t out_dtype,
                               void *workspace, size_t ws_bytes, void *stream)
{
    const int rc = check_shape(shape);
    if (rc != SPARROW_OK)
        return rc;
    if (!q || !k_cache || !v_cache || !block_table || !seq_lens || !k || !idx || !out)
        return SPARROW_EINVAL;
    if (!al16(q) || !al16(k_cache) || !al16(v_cache) || !al4(block_table) || !al4(seq_lens) ||
        !al4(k) || !al4(idx) || !al16(out) || !al16(workspace))
        return SPARROW_EINVAL;
    if (k_max < 1 || k_max > SPARROW_MAX_PAGES_PER_SEQ)
        return SPARROW_EINVAL;
    if (out_dtype != SPARROW_OUT_F32 && out_dtype != SPARROW_OUT_BF16)
        return SPARROW_EUNSUPPORTED;
    if (shape->batch == 0)
        return SPARROW_OK;
    if (shape->batch > kMaxBatch)
        return SPARROW_EUNSUPPORTED;
    const AttnPlan plan = plan_attention(*shape);
    if (!workspace || ws_bytes < plan.workspace_bytes)
        return SPARROW_EWORKSPACE;
    return status_of(launch_attention(*shape, plan, q, k_cache, v_cache, block_table, seq_lens, k,
                                      idx, k_max, scale, out, out_dtype, workspace,
                                      static_cast<hipStream_t>(stream)));
}

int sparrow_sparse_decode_attn_noalloc(const sparrow_shape_t *shape, const void *q,
                                       const void *k_cache, const void *v_cache,
                                       const int32_t *block_table, const int32_t *seq_lens,
                                       const int32_t *k, const int32_t *idx, int32_t k_max,
                                       float scale, void *out, int32_t out_dtype, void *stream)
{
    const int rc = check_shape(shape);
    if (rc != SPARROW_OK)
        return rc;
    if (!q || !k_cache || !v_cache || !block_table || !seq_lens || !k || !idx || !out)
        return SPARROW_EINVAL;
    if (!al16(q) || !al16(k_cache) || !al16(v_cache) || !al4(block_table) || !al4(seq_lens) ||
        !al4(k) || !al4(idx) || !al16(out))
        return SPARROW_EINVAL;
    if (k_max < 1 || k_max > SPARROW_MAX_PAGES_PER_SEQ)
        return SPARROW_EINVAL;
    if (out_dtype != SPARROW_OUT_F32 && out_dtype != SPARROW_OUT_BF16)
        return SPARROW_EUNSUPPORTED;
    if (shape->batch == 0)
        return SPARROW_OK;
    if (shape->batch > kMaxBatch)
        return SPARROW_EUNSUPPORTED;
    const AttnPlan plan = plan_attention(*shape);
    if (plan.workspace_bytes > kScratchBytes)
        return SPARROW_EWORKSPACE;
    void *ws = attention_scratch();
    if (ws == nullptr)
        return SPARROW_EHIP;
    return status_of(launch_attention(*shape, plan, q, k_cache, v_cache, block_table, seq_lens, k,
                                      idx, k_max, scale, out, out_dtype, ws,
                                      static_cast<hipStream_t>(stream)));
}

int sparrow_dense_decode_attn(const sparrow_shape_t *shape, const void *q, const void *k_cache,
                              const void *v_cache, const int32_t *block_table,
                              const int32_t *seq_lens, float scale, void *out, int32_t out_dtype,
                              void *workspace, size_t ws_bytes, void *stream)
{
    const int rc = check_shape(shape);
    if (rc != SPARROW_OK)
        return rc;
    if (!q || !k_cache || !v_cache || !block_table || !seq_lens || !out)
        return SPARROW_EINVAL;
    if (!al16(q) || !al16(k_cache) || !al16(v_cache) || !al4(block_table) || !al4(seq_lens) ||
        !al16(out) || !al16(workspace))
        return SPARROW_EINVAL;
    if (out_dtype != SPARROW_OUT_F32 && out_dtype != SPARROW_OUT_BF16)
        return SPARROW_EUNSUPPORTED;
    if (shape->batch == 0)
        return SPARROW_OK;
    if (shape->batch > kMaxBatch)
        return SPARROW_EUNSUPPORTED;
    const AttnPlan plan = plan_attention(*shape);
    if (!workspace || ws_bytes < plan.workspace_bytes)
        return SPARROW_EWORKSPACE;
    return status_of(launch_attention(*shape, plan, q, k_cache, v_cache, block_table, seq_lens,
                                      nullptr, nullptr, 0, scale, out, out_dtype, workspace,
                                      static_cast<hipStream_t>(stream)));
}

int sparrow_decode_step(const sparrow_shape_t *shape, const void *q, const void *k_new,
                        const void *v_new, void *k_cache, void *v_cache, void *meta,
                        const int32_t *block_table, const int32_t *seq_lens,
                        const sparrow_schedule_t *schedule, int32_t k_max, float scale,
                        int32_t *out_k, int32_t *out_idx, void *out, int32_t out_dtype,
                        void *workspace, size_t ws_bytes, void *stream)
{
    const int rc = check_shape(shape);
    if (rc != SPARROW_OK)
        return rc;
    if (!q || !k_cache || !v_cache || !meta || !block_table || !seq_lens || !schedule || !out_k ||
        !out_idx || !out || (k_new == nullptr) != (v_new == nullptr))
        return SPARROW_EINVAL;
    if (!al16(q) || !al16(k_new) || !al16(v_new) || !al16(k_cache) || !al16(v_cache) ||
        !al16(meta) || !al4(block_table) || !al4(seq_lens) || !al4(out_k) || !al4(out_idx) ||
        !al16(out) || !al16(workspace))
        return SPARROW_EINVAL;
    if (k_max < 1 || k_max > SPARROW_MAX_PAGES_PER_SEQ || schedule->bin_tokens < 1 ||
        schedule->n_bins < 1 || schedule->frac_den < 1 || !schedule->min_pages ||
        !schedule->frac_num || schedule->sink_pages < 0 || schedule->local_pages < 0)
        return SPARROW_EINVAL;
    if (out_dtype != SPARROW_OUT_F32 && out_dtype != SPARROW_OUT_BF16)
        return SPARROW_EUNSUPPORTED;
    if (shape->batch == 0)
        return SPARROW_OK;
    if ((int64_t)shape->batch * shape->num_kv_heads > 65535)
        return SPARROW_EINVAL;
    if (shape->batch > kMaxBatch)
        return SPARROW_EUNSUPPORTED;
    if (!workspace || ws_bytes < decode_step_workspace(*shape))
        return SPARROW_EWORKSPACE;
    const Sched sched{schedule->bin_tokens, schedule->n_bins,     schedule->frac_den,
                      schedule->min_pages,  schedule->frac_num, schedule->sink_pages,
                      schedule->local_pages};
    const AppendArgs app{k_new, v_new, k_new ? k_cache : nullptr, k_new ? v_cache : nullptr};
    const hipStream_t st = static_cast<hipStream_t>(stream);
    float *scores = static_cast<float *>(workspace);
    void *attn_ws = static_cast<char *>(workspace) + round256(score_topk_workspace(*shape));
    hipError_t e = launch_page_score(*shape, q, meta, block_table, seq_lens, sched, k_max, scores,
                                     app, st);
    if (e != hipSuccess)
        return SPARROW_EHIP;
    if (attention_unit_path(*shape, k_max))
        return status_of(launch_select_attention(*shape, q, k_cache, v_cache, block_table,
                                                 seq_lens, sched, k_max, scores, out_k, out_idx,
                                                 scale, out, out_dtype, st));
    e = launch_topk(*shape, seq_lens, sched, k_max, scores, out_k, out_idx, st);
    if (e != hipSuccess)
        return SPARROW_EHIP;
    return status_of(launch_attention(*shape, plan_attention(*shape), q, k_cache, v_cache,
                                      block_table, seq_lens, out_k, out_idx, k_max, scale, out,
                                      out_dtype, attn_ws, st));
}

int sparrow_acceptance_rate(int64_t num_tokens, int32_t vocab, int32_t logits_dtype,
                            const void *target_logits, const void *draft_logits,
                            float inv_temperature, float *alpha, void *stream)
{
    if (num_tokens < 0 || vocab < 1 || !target_logits || !draft_logits || !alpha)
        return SPARROW_EINVAL;
    if (logits_dtype != SPARROW_LOGITS_F32 && logits_dtype != SPARROW_LOGITS_BF16)
        return SPARROW_EUNSUPPORTED;
    const uintptr_t esz = logits_dtype == SPARROW_LOGITS_BF16 ? 2 : 4;
    if ((reinterpret_cast<uintptr_t>(target_logits) % esz) != 0 ||
        (reinterpret_cast<uintptr_t>(draft_logits) % esz) != 0 || !al4(alpha))
        return SPARROW_EINVAL;
    // both rows of a token must share their alignment for the vector loads
    if ((reinterpret_cast<uintptr_t>(target_logits) & 15u) !=
        (reinterpret_cast<uintptr_t>(draft_logits) & 15u))
        return SPARROW_EINVAL;
    if (!std::isfinite(inv_temperature) || num_tokens > 0x7fffffff)
        return SPARROW_EINVAL;
    if (num_tokens == 0)
        return SPARROW_OK;
    return status_of(launch_acceptance(num_tokens, vocab, logits_dtype, target_logits,
                                       draft_logits, inv_temperature, alpha,
                                       static_cast<hipStream_t>(stream)));
}

int sparrow_acceptance_rate_topk(int64_t num_tokens, int32_t k, const float *lp_target,
                                 const float *lp_draft, float *alpha, void *stream)
{
    if (num_tokens < 0 || k < 1 || !lp_target || !lp_draft || !alpha)
        return SPARROW_EINVAL;
    if (!al4(lp_target) || !al4(lp_draft) || !al4(alpha))
        return SPARROW_EINVAL;
    if (num_tokens == 0)
        return SPARROW_OK;
    return status_of(launch_acceptance_topk(num_tokens, k, lp_target, lp_draft, alpha,
                                            static_cast<hipStream_t>(stream)));
}

int sparrow_tail_stats(int64_t num_tokens, const float *alpha, const int32_t *positions,
                       int32_t bin_tokens, int32_t n_bins, double percentile, double *quantile,
                       double *mean, int64_t *count, void *stream)
{
    if (num_tokens < 0 || bin_tokens < 1 || n_bins < 1 || n_bins > 65535)
        return SPARROW_EINVAL;
    if (!(percentile >= 0.0 && percentile <= 100.0))
        return SPARROW_EINVAL;
    if (!quantile || !mean || !count || (num_tokens > 0 && (!alpha || !positions)))
        return SPARROW_EINVAL;
    if (!al4(alpha) || !al4(positions) || (reinterpret_cast<uintptr_t>(quantile) & 7u) ||
        (reinterpret_cast<uintptr_t>(mean) & 7u) || (reinterpret_cast<uintptr_t>(count) & 7u))
        return SPARROW_EINVAL;
    return status_of(launch_tail_stats(num_tokens, alpha, positions, bin_tokens, n_bins,
                                       percentile, quantile, mean, count,
                                       static_cast<hipStream_t>(stream)));
}

int sparrow_stream_read(const void *src, int64_t bytes, uint32_t *checksum, void *stream)
{
    if (bytes < 0 || (bytes & 15) != 0 || !checksum || (bytes > 0 && !src))
        return SPARROW_EINVAL;
    if (!al16(src) || !al4(checksum))
        return SPARROW_EINVAL;
    if (bytes == 0)
        return SPARROW_OK;
    return status_of(launch_stream_read(src, bytes, checksum, static_cast<hipStream_t>(stream)));
}

int32_t sparrow_budget_bound(const int32_t *seq_lens, int64_t num_seqs, int32_t page_size,
                             int32_t bin_tokens, int32_t n_bins, const int32_t *min_pages,
                             const int32_t *frac_num, int32_t frac_den, int32_t *budgets)
{
    if (num_seqs < 0 || page_size < 1 || bin_tokens < 1 || n_bins < 1 || frac_den < 1)
        return SPARROW_EINVAL;
    if (!min_pages || !frac_num || (num_seqs > 0 && !seq_lens))
        return SPARROW_EINVAL;
    for (int32_t i = 0; i < n_bins; ++i)
        if (min_pages[i] < 0 || frac_num[i] < 0)
            return SPARROW_EINVAL;
    const int64_t max_len = (int64_t)page_size * SPARROW_MAX_PAGES_PER_SEQ;
    int32_t best = 1;
    for (int64_t b = 0; b < num_seqs; ++b) {
        const int32_t L = seq_lens[b];
        if (L > max_len)
            return SPARROW_EINVAL;
        int32_t k = 0;
        if (L > 0) {
            const int bin = budget_bin(L, bin_tokens, n_bins);
            k = budget_from(L, page_size, min_pages[bin], frac_num[bin], frac_den, 0x7fffffff);
        }
        if (budgets)
            budgets[b] = k;
        if (k > best)
            best = k;
    }
    return best;
}

size_t sparrow_workspace_size(const sparrow_shape_t *shape, int32_t k_max, int32_t op)
{
    if (check_shape(shape) != SPARROW_OK)
        return 0;
    switch (op) {
    case SPARROW_OP_SCORE_TOPK: return shape->batch > kMaxBatch ? 0 : score_topk_workspace(*shape);
    case SPARROW_OP_SPARSE_ATTN:
        return k_max < 1 || k_max > SPARROW_MAX_PAGES_PER_SEQ || shape->batch > kMaxBatch
                   ? 0
                   : plan_attention(*shape).workspace_bytes;
    case SPARROW_OP_DENSE_ATTN:
        return shape->batch > kMaxBatch ? 0 : plan_attention(*shape).workspace_bytes;
    case SPARROW_OP_DECODE_STEP:
        return k_max < 1 || k_max > SPARROW_MAX_PAGES_PER_SEQ || shape->batch > kMaxBatch
                   ? 0
                   : decode_step_workspace(*shape);
    default: return 0;
    }
}

const char *sparrow_status_string(int32_t status)
{
    switch (status) {
    case SPARROW_OK: return "ok";
    case SPARROW_EINVAL: return "invalid argument (null pointer or bad size)";
    case SPARROW_EUNSUPPORTED: return "unsupported head_dim, page size, group size or dtype";
    case SPARROW_EWORKSPACE: return "workspace missing or too small";
    case SPARROW_EHIP: return "kernel launch failed";
    default: return "unknown status";
    }
}

}  // extern "C"
