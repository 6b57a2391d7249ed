/*
 * CPU oracle for the sparse-decode attention step of Sparrow (arXiv 2606.08446).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, obviously correct
 * reference that the HIP library is checked against.  Only the test suite,
 * the smoke check and the benchmark's CPU-baseline leg load it.  It shares no
 * code, header, table or helper with the GPU library, and the GPU library never
 * calls it.
 *
 * What it computes (one decode step, one layer):
 *   - per-page key metadata: channel-wise min and max of the keys of each page
 *     (the page "landmark" that block top-k selection scores against the
 *     query; the paper names landmark scoring and top-k page selection in
 *     Sec. 3.3 and Appendix C, and the selector is read as the min/max page
 *     bound of the Quest line of work it cites in Sec. 1),
 *   - the page score: for query head j and page p,
 *         s_j(p) = sum_i max(q_{j,i} * mn_i(p), q_{j,i} * mx_i(p)),
 *     summed over the G query heads that share one KV head,
 *   - the page budget from the dynamic sparsity schedule (Sec. 3.2, Method
 *     box: the budget grows with the current length; lengths are grouped in
 *     2K-token bins),
 *   - the top-k pages (largest score first, ties to the lower page index),
 *   - softmax attention of every query head over the tokens of the selected
 *     pages (block-sparse attention, Sec. 2), and over all tokens (dense).
 *
 * Precision: attention is computed in fp64 throughout.  Page scores are
 * computed twice: in fp32 (the precision the GPU takes the top-k decision
 * in, accumulated channel by channel and then head by head) and in fp64 (used
 * only to adjudicate near-ties).  The top-k decision is taken on the fp32
 * scores.  Keys, values, queries and metadata arrive as bf16 bit patterns.
 *
 * Data layouts (all row-major):
 *   q           bf16 [B][Hq][D]
 *   k/v cache   bf16 [P_phys][Hkv][ps][D]
 *   meta        bf16 [P_phys][Hkv][2][D]   (row 0 = min, row 1 = max)
 *   block_table int32 [B][max_pages]       logical page -> physical page
 *   seq_lens    int32 [B]                  tokens in the sequence
 * Query head j reads KV head j / G with G = Hq / Hkv.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

static double bf16_value(uint16_t bits)
{
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

static float bf16_value_f(uint16_t bits)
{
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

static int64_t pages_of(int64_t len, int64_t ps)
{
    return len <= 0 ? 0 : (len + ps - 1) / ps;
}

/* ------------------------------------------------------------------------ */
/* Budget from the dynamic sparsity schedule (Sec. 3.2 Method box; 2K-token  */
/* length bins; Appendix F: a budget that covers the whole context means     */
/* dense attention).                                                         */
/*                                                                           */
/* For a sequence of L tokens (n = ceil(L / ps) pages) the bin is            */
/* min(floor((L - 1) / bin_tokens), n_bins - 1) and the budget is            */
/*   k = clamp(max(min_pages[bin], ceil(n * frac_num[bin] / frac_den)), 1, n) */
/* An empty sequence gets k = 0.                                             */
/* ------------------------------------------------------------------------ */
int32_t oracle_budget(int32_t L, int32_t ps, int32_t bin_tokens, int32_t n_bins,
                      const int32_t *min_pages, const int32_t *frac_num, int32_t frac_den)
{
    if (L <= 0)
        return 0;
    int64_t n = pages_of(L, ps);
    int64_t bin = (int64_t)(L - 1) / bin_tokens;
    if (bin > n_bins - 1)
        bin = n_bins - 1;
    int64_t frac_pages = (n * (int64_t)frac_num[bin] + frac_den - 1) / frac_den;
    int64_t k = frac_pages;
    if (k < min_pages[bin])
        k = min_pages[bin];
    if (k < 1)
        k = 1;
    if (k > n)
        k = n;
    return (int32_t)k;
}

void oracle_budgets(int32_t B, const int32_t *seq_lens, int32_t ps, int32_t bin_tokens,
                    int32_t n_bins, const int32_t *min_pages, const int32_t *frac_num,
                    int32_t frac_den, int32_t *out_k)
{
    for (int32_t b = 0; b < B; ++b)
        out_k[b] = oracle_budget(seq_lens[b], ps, bin_tokens, n_bins, min_pages, frac_num,
                                 frac_den);
}

/* ------------------------------------------------------------------------ */
/* Page metadata: per channel, the min and the max of the keys of the valid  */
/* tokens of the page.  Ties between -0 and +0 are resolved by the total     */
/* order -0 < +0, so the result is one input bit pattern, exactly.           */
/* Pages that overlap [first_pos[b], L_b) are recomputed from all of their   */
/* valid tokens; first_pos == NULL recomputes every page.                    */
/* ------------------------------------------------------------------------ */
static int total_less(uint16_t a_bits, uint16_t b_bits)
{
    float a = bf16_value_f(a_bits), b = bf16_value_f(b_bits);
    if (a < b)
        return 1;
    if (a == b && (a_bits & 0x8000u) && !(b_bits & 0x8000u))
        return 1;
    return 0;
}

void oracle_page_meta(int32_t B, int32_t Hkv, int32_t D, int32_t ps, int32_t max_pages,
                      const uint16_t *k_cache, const int32_t *block_table,
                      const int32_t *seq_lens, const int32_t *first_pos, uint16_t *meta)
{
    for (int32_t b = 0; b < B; ++b) {
        int64_t L = seq_lens[b];
        int64_t n = pages_of(L, ps);
        int64_t p_first = 0;
        if (first_pos) {
            int64_t f = first_pos[b];
            if (f < 0)
                f = 0;
            if (f >= L)
                continue;
            p_first = f / ps;
        }
        for (int64_t p = p_first; p < n; ++p) {
            int64_t phys = block_table[(int64_t)b * max_pages + p];
            int64_t t_end = L - p * ps < ps ? L - p * ps : ps;
            for (int32_t h = 0; h < Hkv; ++h) {
                const uint16_t *page = k_cache + ((phys * Hkv + h) * ps) * D;
                uint16_t *mrow = meta + ((phys * Hkv + h) * 2) * D;
                for (int32_t i = 0; i < D; ++i) {
                    uint16_t mn = page[i], mx = page[i];
                    for (int64_t t = 1; t < t_end; ++t) {
                        uint16_t v = page[t * D + i];
                        if (total_less(v, mn))
                            mn = v;
                        if (total_less(mx, v))
                            mx = v;
                    }
                    mrow[i] = mn;
                    mrow[D + i] = mx;
                }
            }
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Appending the token being decoded (the step that precedes scoring in a    */
/* decode step; Sec. 3.3 counts the landmark upkeep per generated token).    */
/* L_b counts the new token, so it sits at position L_b - 1: logical page    */
/* (L_b - 1) / ps, slot (L_b - 1) % ps.  Its key and value rows of every KV  */
/* head are copied into the caches, then the metadata of that page is        */
/* recomputed from all of its valid tokens (the definition above).           */
/* Sequences with L_b < 1, or with L_b beyond what the block table can       */
/* address, are left untouched.  New rows: k_new, v_new bf16 [B][Hkv][D].    */
/* ------------------------------------------------------------------------ */
void oracle_append_kv(int32_t B, int32_t Hkv, int32_t D, int32_t ps, int32_t max_pages,
                      const uint16_t *k_new, const uint16_t *v_new, uint16_t *k_cache,
                      uint16_t *v_cache, const int32_t *block_table, const int32_t *seq_lens,
                      uint16_t *meta)
{
    for (int32_t b = 0; b < B; ++b) {
        int64_t L = seq_lens[b];
        if (L < 1 || L > (int64_t)ps * max_pages)
            continue;
        int64_t pos = L - 1;
        int64_t phys = block_table[(int64_t)b * max_pages + pos / ps];
        int64_t slot = pos % ps;
        for (int32_t h = 0; h < Hkv; ++h) {
            int64_t row = ((phys * Hkv + h) * ps + slot) * D;
            const uint16_t *kn = k_new + ((int64_t)b * Hkv + h) * D;
            const uint16_t *vn = v_new + ((int64_t)b * Hkv + h) * D;
            for (int32_t i = 0; i < D; ++i) {
                k_cache[row + i] = kn[i];
                v_cache[row + i] = vn[i];
            }
        }
        int32_t first = (int32_t)pos;
        oracle_page_meta(1, Hkv, D, ps, max_pages, k_cache, block_table + (int64_t)b * max_pages,
                         seq_lens + b, &first, meta);
    }
}

/* ------------------------------------------------------------------------ */
/* Page scores.  s_j(p) = sum_i max(q_{j,i} mn_i, q_{j,i} mx_i) is an upper  */
/* bound of q_j . k_t over the tokens t of page p; the KV-head score is the  */
/* sum of s_j over its G query heads.  scores32 is accumulated in fp32,      */
/* channel order then head order; scores64 in fp64.  Output layout           */
/* [B][Hkv][max_pages]; entries at p >= n_b are left untouched.              */
/* ------------------------------------------------------------------------ */
void oracle_page_scores(int32_t B, int32_t Hq, int32_t Hkv, int32_t D, int32_t ps,
                        int32_t max_pages, const uint16_t *q, const uint16_t *meta,
                        const int32_t *block_table, const int32_t *seq_lens,
                        float *scores32, double *scores64)
{
    int32_t G = Hq / Hkv;
#pragma omp parallel for schedule(dynamic) collapse(2)
    for (int32_t b = 0; b < B; ++b) {
        for (int32_t h = 0; h < Hkv; ++h) {
            int64_t n = pages_of(seq_lens[b], ps);
            for (int64_t p = 0; p < n; ++p) {
                int64_t phys = block_table[(int64_t)b * max_pages + p];
                const uint16_t *mn = meta + ((phys * Hkv + h) * 2) * D;
                const uint16_t *mx = mn + D;
                float head_sum32 = 0.0f;
                double head_sum64 = 0.0;
                for (int32_t g = 0; g < G; ++g) {
                    const uint16_t *qj = q + ((int64_t)b * Hq + (int64_t)h * G + g) * D;
                    float s32 = 0.0f;
                    double s64 = 0.0;
                    for (int32_t i = 0; i < D; ++i) {
                        float qi = bf16_value_f(qj[i]);
                        float lo = qi * bf16_value_f(mn[i]); /* exact: bf16 x bf16 */
                        float hi = qi * bf16_value_f(mx[i]);
                        s32 += lo > hi ? lo : hi;
                        if (scores64) { /* the adjudication copy, only when asked for */
                            double lo64 = (double)qi * bf16_value(mn[i]);
                            double hi64 = (double)qi * bf16_value(mx[i]);
                            s64 += lo64 > hi64 ? lo64 : hi64;
                        }
                    }
                    head_sum32 += s32;
                    head_sum64 += s64;
                }
                int64_t o = ((int64_t)b * Hkv + h) * max_pages + p;
                if (scores32)
                    scores32[o] = head_sum32;
                if (scores64)
                    scores64[o] = head_sum64;
            }
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Top-k: order pages by (score descending, page index ascending), keep the  */
/* first k and return them in ascending page order.  -0 and +0 compare       */
/* equal.  NaN scores are not supported.                                     */
/* ------------------------------------------------------------------------ */
typedef struct {
    float s;
    int32_t p;
} scored_page;

static int by_score_then_index(const void *x, const void *y)
{
    const scored_page *a = (const scored_page *)x, *b = (const scored_page *)y;
    if (a->s > b->s)
        return -1;
    if (a->s < b->s)
        return 1;
    return (a->p > b->p) - (a->p < b->p);
}

static int by_index(const void *x, const void *y)
{
    int32_t a = *(const int32_t *)x, b = *(const int32_t *)y;
    return (a > b) - (a < b);
}

void oracle_topk(const float *scores, int32_t n, int32_t k, int32_t *out)
{
    if (k > n)
        k = n;
    if (k <= 0)
        return;
    scored_page *all = (scored_page *)malloc(sizeof(scored_page) * (size_t)n);
    for (int32_t p = 0; p < n; ++p) {
        all[p].s = scores[p];
        all[p].p = p;
    }
    qsort(all, (size_t)n, sizeof(scored_page), by_score_then_index);
    for (int32_t i = 0; i < k; ++i)
        out[i] = all[i].p;
    qsort(out, (size_t)k, sizeof(int32_t), by_index);
    free(all);
}

/* Top-k for every (sequence, KV head): idx[B][Hkv][k_max], padded with -1.  */
void oracle_select(int32_t B, int32_t Hkv, int32_t ps, int32_t max_pages,
                   const int32_t *seq_lens, const int32_t *k_of_seq, const float *scores32,
                   int32_t k_max, int32_t *idx)
{
#pragma omp parallel for schedule(dynamic) collapse(2)
    for (int32_t b = 0; b < B; ++b) {
        for (int32_t h = 0; h < Hkv; ++h) {
            int32_t *row = idx + ((int64_t)b * Hkv + h) * k_max;
            for (int32_t i = 0; i < k_max; ++i)
                row[i] = -1;
            int64_t n = pages_of(seq_lens[b], ps);
            int32_t k = k_of_seq[b] < k_max ? k_of_seq[b] : k_max;
            oracle_topk(scores32 + ((int64_t)b * Hkv + h) * max_pages, (int32_t)n, k, row);
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Attention of every query head over a token set, in fp64:                  */
/*   z_t = scale * (q . k_t),  w_t = exp(z_t - max z) / sum exp(z - max z),  */
/*   o = sum_t w_t v_t                                                       */
/* (two passes over materialised logits).  The token set is every valid      */
/* token of the listed pages; the list is idx[b][h][0 .. k_of_seq[b]) for    */
/* sparse attention, and all pages 0 .. n_b - 1 when idx == NULL (dense).    */
/* A sequence with no tokens produces a zero output.  out is [B][Hq][D].     */
/* ------------------------------------------------------------------------ */
void oracle_attention(int32_t B, int32_t Hq, int32_t Hkv, int32_t D, int32_t ps,
                      int32_t max_pages, const uint16_t *q, const uint16_t *k_cache,
                      const uint16_t *v_cache, const int32_t *block_table,
                      const int32_t *seq_lens, const int32_t *k_of_seq, const int32_t *idx,
                      int32_t k_max, double scale, double *out)
{
    int32_t G = Hq / Hkv;
#pragma omp parallel for schedule(dynamic) collapse(2)
    for (int32_t b = 0; b < B; ++b) {
        for (int32_t j = 0; j < Hq; ++j) {
            int32_t h = j / G;
            int64_t L = seq_lens[b];
            int64_t n = pages_of(L, ps);
            double *o = out + ((int64_t)b * Hq + j) * D;
            for (int32_t i = 0; i < D; ++i)
                o[i] = 0.0;
            int64_t n_list = n;
            const int32_t *list = NULL;
            if (idx) {
                n_list = k_of_seq[b] < k_max ? k_of_seq[b] : k_max;
                list = idx + ((int64_t)b * Hkv + h) * k_max;
            }
            if (L <= 0 || n_list <= 0)
                continue;
            const uint16_t *qj = q + ((int64_t)b * Hq + j) * D;
            double *z = (double *)malloc(sizeof(double) * (size_t)(n_list * ps));
            int64_t *tok_page = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n_list * ps));
            int64_t *tok_slot = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n_list * ps));
            int64_t n_tok = 0;
            for (int64_t e = 0; e < n_list; ++e) {
                int64_t p = list ? list[e] : e;
                int64_t phys = block_table[(int64_t)b * max_pages + p];
                int64_t t_end = L - p * ps < ps ? L - p * ps : ps;
                for (int64_t t = 0; t < t_end; ++t) {
                    const uint16_t *kt = k_cache + ((phys * Hkv + h) * ps + t) * D;
                    double dot = 0.0;
                    for (int32_t i = 0; i < D; ++i)
                        dot += bf16_value(qj[i]) * bf16_value(kt[i]);
                    z[n_tok] = scale * dot;
                    tok_page[n_tok] = phys;
                    tok_slot[n_tok] = t;
                    ++n_tok;
                }
            }
            double m = z[0];
            for (int64_t t = 1; t < n_tok; ++t)
                if (z[t] > m)
                    m = z[t];
            double denom = 0.0;
            for (int64_t t = 0; t < n_tok; ++t)
                denom += exp(z[t] - m);
            for (int64_t t = 0; t < n_tok; ++t) {
                double w = exp(z[t] - m) / denom;
                const uint16_t *vt = v_cache + ((tok_page[t] * Hkv + h) * ps + tok_slot[t]) * D;
                for (int32_t i = 0; i < D; ++i)
                    o[i] += w * bf16_value(vt[i]);
            }
            free(z);
            free(tok_page);
            free(tok_slot);
        }
    }
}

/* Sum of the softmax weights of one query head (used by the weight-sum pin). */
double oracle_weight_sum(int32_t D, int64_t n_tok, const uint16_t *qj, const uint16_t *keys,
                         double scale)
{
    double *z = (double *)malloc(sizeof(double) * (size_t)n_tok);
    double m = -INFINITY;
    for (int64_t t = 0; t < n_tok; ++t) {
        double dot = 0.0;
        for (int32_t i = 0; i < D; ++i)
            dot += bf16_value(qj[i]) * bf16_value(keys[t * D + i]);
        z[t] = scale * dot;
        if (z[t] > m)
            m = z[t];
    }
    double denom = 0.0;
    for (int64_t t = 0; t < n_tok; ++t)
        denom += exp(z[t] - m);
    double total = 0.0;
    for (int64_t t = 0; t < n_tok; ++t)
        total += exp(z[t] - m) / denom;
    free(z);
    return total;
}

/* Threads of the parallel loops (the OpenMP default is every host core). */
void oracle_set_num_threads(int32_t n)
{
#ifdef _OPENMP
    extern void omp_set_num_threads(int);
    omp_set_num_threads(n < 1 ? 1 : n);
#else
    (void)n;
#endif
}

int32_t oracle_num_threads(void)
{
#ifdef _OPENMP
    extern int omp_get_max_threads(void);
    return omp_get_max_threads();
#else
    return 1;
#endif
}
