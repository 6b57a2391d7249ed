/*
 * CPU oracle for the selector variants of Sparrow's sparse decode (arXiv 2606.08446):
 * the mean-key page landmark (one D-vector per page, the landmark the cost model of
 * Sec. 3.3 counts in its scoring term) and top-k selection with forced sink and local
 * pages.
 *
 * TEST INFRASTRUCTURE ONLY.  Plain reference code the HIP library is checked against;
 * only the test suite loads it.  It shares no code with the GPU library.
 *
 * Mean landmark.  The metadata of a (page, KV head) is the fp32 sum over the page's
 * valid tokens of their keys, accumulated token by token in position order (one D-vector,
 * [P_phys][Hkv][D] fp32).  The landmark is sum / n_valid (the mean key) and the page
 * score of KV head h is the sum over its G query heads j of q_j . mean:
 *     S_h(p) = sum_j sum_i q_{j,i} * (sum_i(p) / n_valid(p)).
 * scores32 computes mean_i in fp32 (one division per channel), the dot product channel by
 * channel and then the heads in order; scores64 the same in fp64 from the same fp32 sums.
 *
 * Forced pages.  With sink pages s and local pages l, the logical pages [0, s) and
 * [n - l, n) are always taken first (lower index first), the rest of the budget by score
 * (largest first, ties to the lower index); the kept pages are returned ascending.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

static float bf16f(uint16_t bits)
{
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

static int64_t n_pages(int64_t len, int64_t ps)
{
    return len <= 0 ? 0 : (len + ps - 1) / ps;
}

/* Key sums of the pages that overlap [first_pos[b], L_b) (every page when first_pos is
   NULL); sums is [P][Hkv][D] fp32. */
void oracle_page_key_sums(int32_t B, int32_t Hkv, int32_t D, int32_t ps, int32_t max_pages,
                          const uint16_t *k_cache, const int32_t *block_table,
                          const int32_t *seq_lens, const int32_t *first_pos, float *sums)
{
    for (int32_t b = 0; b < B; ++b) {
        int64_t L = seq_lens[b];
        int64_t n = n_pages(L, ps);
        int64_t p0 = 0;
        if (first_pos) {
            int64_t f = first_pos[b] < 0 ? 0 : first_pos[b];
            if (f >= L)
                continue;
            p0 = f / ps;
        }
        for (int64_t p = p0; p < n; ++p) {
            int64_t phys = block_table[(int64_t)b * max_pages + p];
            int64_t valid = L - p * ps < ps ? L - p * ps : ps;
            for (int32_t h = 0; h < Hkv; ++h) {
                const uint16_t *page = k_cache + ((phys * Hkv + h) * ps) * D;
                float *out = sums + (phys * Hkv + h) * D;
                for (int32_t i = 0; i < D; ++i) {
                    float s = 0.0f;
                    for (int64_t t = 0; t < valid; ++t)
                        s += bf16f(page[t * D + i]);
                    out[i] = s;
                }
            }
        }
    }
}

void oracle_page_scores_mean(int32_t B, int32_t Hq, int32_t Hkv, int32_t D, int32_t ps,
                             int32_t max_pages, const uint16_t *q, const float *sums,
                             const int32_t *block_table, const int32_t *seq_lens,
                             float *scores32, double *scores64)
{
    int32_t G = Hq / Hkv;
    for (int32_t b = 0; b < B; ++b) {
        int64_t L = seq_lens[b];
        int64_t n = n_pages(L, ps);
        for (int32_t h = 0; h < Hkv; ++h) {
            for (int64_t p = 0; p < n; ++p) {
                int64_t phys = block_table[(int64_t)b * max_pages + p];
                int64_t valid = L - p * ps < ps ? L - p * ps : ps;
                const float *sm = sums + (phys * Hkv + h) * D;
                float tot32 = 0.0f;
                double tot64 = 0.0;
                for (int32_t g = 0; g < G; ++g) {
                    const uint16_t *qj = q + ((int64_t)b * Hq + (int64_t)h * G + g) * D;
                    float s32 = 0.0f;
                    double s64 = 0.0;
                    for (int32_t i = 0; i < D; ++i) {
                        s32 += bf16f(qj[i]) * (sm[i] / (float)valid);
                        if (scores64) /* the adjudication copy, only when asked for */
                            s64 += (double)bf16f(qj[i]) * ((double)sm[i] / (double)valid);
                    }
                    tot32 += s32;
                    tot64 += s64;
                }
                int64_t o = ((int64_t)b * Hkv + h) * max_pages + p;
                if (scores32)
                    scores32[o] = tot32;
                if (scores64)
                    scores64[o] = tot64;
            }
        }
    }
}

struct ranked {
    int32_t forced; /* 0 = forced, 1 = by score */
    float s;
    int32_t p;
};

static int by_rank(const void *x, const void *y)
{
    const struct ranked *a = x, *b = y;
    if (a->forced != b->forced)
        return a->forced - b->forced;
    if (a->forced == 0 || a->s == b->s) /* forced pages, or equal scores (-0 == +0) */
        return (a->p > b->p) - (a->p < b->p);
    return a->s > b->s ? -1 : 1;
}

static int ascending(const void *x, const void *y)
{
    int32_t a = *(const int32_t *)x, b = *(const int32_t *)y;
    return (a > b) - (a < b);
}

/* idx[B][Hkv][k_max]: the min(k_b, k_max) kept pages of each (sequence, head), ascending,
   padded with -1; pages [0, sink) and [n - local, n) are forced. */
void oracle_select_forced(int32_t B, int32_t Hkv, int32_t ps, int32_t max_pages,
                          const int32_t *seq_lens, const int32_t *k_of_seq,
                          const float *scores32, int32_t sink, int32_t local, int32_t k_max,
                          int32_t *idx)
{
    struct ranked *r = (struct ranked *)malloc((size_t)(max_pages > 0 ? max_pages : 1) *
                                               sizeof(struct ranked));
    for (int32_t b = 0; b < B; ++b) {
        int64_t n = n_pages(seq_lens[b], ps);
        int32_t k = k_of_seq[b] < k_max ? k_of_seq[b] : k_max;
        if (k > n)
            k = (int32_t)n;
        for (int32_t h = 0; h < Hkv; ++h) {
            int32_t *row = idx + ((int64_t)b * Hkv + h) * k_max;
            for (int32_t i = 0; i < k_max; ++i)
                row[i] = -1;
            const float *s = scores32 + ((int64_t)b * Hkv + h) * max_pages;
            for (int64_t p = 0; p < n; ++p) {
                r[p].forced = (p < sink || p >= n - local) ? 0 : 1;
                r[p].s = s[p];
                r[p].p = (int32_t)p;
            }
            qsort(r, (size_t)n, sizeof *r, by_rank);
            for (int32_t i = 0; i < k; ++i)
                row[i] = r[i].p;
            qsort(row, (size_t)k, sizeof(int32_t), ascending);
        }
    }
    free(r);
}
