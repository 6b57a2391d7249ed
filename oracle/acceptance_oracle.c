/*
 * CPU oracle for the per-token acceptance rate of Sparrow (arXiv 2606.08446,
 * Sec. 3.1, Eq. 1) and its lower-tail statistic per length bin (Sec. 3.1-3.2).
 *
 * TEST INFRASTRUCTURE ONLY.  Plain, slow reference code that the HIP library is
 * checked against; only the test suite and the benchmark's CPU-baseline leg load
 * it.  It shares no code with the GPU library.
 *
 * Acceptance rate of one generated token: p is the target distribution (the
 * dense policy) and q the draft distribution (the sparse rollout) over the
 * vocabulary, each the softmax of a logit row at inverse temperature tau:
 *     p(x) = exp(tau z_x) / sum_y exp(tau z_y).
 * Eq. 1 writes alpha as the expectation over x ~ q of min(p(x)/q(x), 1), which
 * equals the sum over the vocabulary of min(p(x), q(x)) (= 1 - total variation
 * distance); that sum is what is computed here, in fp64: each row's
 * log-sum-exp, then sum_x min(exp(tau p_x - P), exp(tau q_x - Q)).
 *
 * The paper's own measurement (Sec. 3.1, footnote on the inference engine)
 * only had the top-20 tokens of each position with their log-probabilities;
 * oracle_acceptance_topk is that approximation: the same sum over the listed
 * tokens only, from normalised log-probabilities.
 *
 * Tail statistic (Sec. 3.1 Method: the 5-percentile of the per-token
 * acceptance rate; Sec. 3.2: tokens grouped by position in 2K-token bins):
 * per bin, the count, the mean and the pct-percentile of alpha, the percentile
 * taken with linear interpolation between order statistics.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

static double logit_value(const void *row, int32_t dtype, int64_t i)
{
    if (dtype == 1) {
        uint32_t u = (uint32_t)((const uint16_t *)row)[i] << 16;
        float f;
        memcpy(&f, &u, sizeof f);
        return (double)f;
    }
    return (double)((const float *)row)[i];
}

/* log sum_x exp(tau z_x) of one row, in fp64 */
static double row_lse(const void *row, int32_t dtype, int32_t V, double tau)
{
    double m = -INFINITY;
    for (int32_t x = 0; x < V; ++x) {
        double v = tau * logit_value(row, dtype, x);
        if (v > m)
            m = v;
    }
    double s = 0.0;
    for (int32_t x = 0; x < V; ++x)
        s += exp(tau * logit_value(row, dtype, x) - m);
    return m + log(s);
}

/* alpha[t] for T tokens; logit rows of V entries, row t at offset t * V; dtype 0 = fp32,
   1 = bf16 bit patterns. */
void oracle_acceptance(int64_t T, int32_t V, int32_t dtype, const void *target,
                       const void *draft, double tau, double *alpha)
{
    const size_t esz = dtype == 1 ? 2 : 4;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t t = 0; t < T; ++t) {
        const void *pr = (const char *)target + (size_t)t * V * esz;
        const void *qr = (const char *)draft + (size_t)t * V * esz;
        double P = row_lse(pr, dtype, V, tau);
        double Q = row_lse(qr, dtype, V, tau);
        double a = 0.0;
        for (int32_t x = 0; x < V; ++x) {
            double p = exp(tau * logit_value(pr, dtype, x) - P);
            double q = exp(tau * logit_value(qr, dtype, x) - Q);
            a += p < q ? p : q;
        }
        alpha[t] = a;
    }
}

/* The top-K approximation: lp_target/lp_draft [T][K] are the normalised log-probabilities
   of the same K tokens under the two distributions. */
void oracle_acceptance_topk(int64_t T, int32_t K, const float *lp_target, const float *lp_draft,
                            double *alpha)
{
    for (int64_t t = 0; t < T; ++t) {
        double a = 0.0;
        for (int32_t i = 0; i < K; ++i) {
            double p = exp((double)lp_target[t * K + i]);
            double q = exp((double)lp_draft[t * K + i]);
            a += p < q ? p : q;
        }
        alpha[t] = a;
    }
}

static int cmp_float(const void *a, const void *b)
{
    float x = *(const float *)a, y = *(const float *)b;
    return (x > y) - (x < y);
}

/* Per bin b < n_bins: count[b], mean[b] and quantile[b] (the pct-percentile, 0 <= pct <=
   100) of the alpha values of the tokens in the bin.  Token t is in bin
   min(pos[t] / bin_tokens, n_bins - 1); tokens with pos[t] < 0 are ignored.  With the
   bin's values sorted, x_0 <= ... <= x_{N-1}: h = (N - 1) * pct / 100, lo = floor(h),
   quantile = x_lo + (h - lo) * (x_{lo+1} - x_lo) (x_lo itself when lo = N - 1).  Empty
   bins get count 0 and NaN mean and quantile. */
void oracle_tail_stats(int64_t T, const float *alpha, const int32_t *pos, int32_t bin_tokens,
                       int32_t n_bins, double pct, double *quantile, double *mean,
                       int64_t *count)
{
    float *vals = (float *)malloc((size_t)(T > 0 ? T : 1) * sizeof(float));
    for (int32_t b = 0; b < n_bins; ++b) {
        int64_t N = 0;
        double sum = 0.0;
        for (int64_t t = 0; t < T; ++t) {
            if (pos[t] < 0)
                continue;
            int64_t bin = pos[t] / bin_tokens;
            if (bin > n_bins - 1)
                bin = n_bins - 1;
            if (bin != b)
                continue;
            vals[N++] = alpha[t];
            sum += (double)alpha[t];
        }
        count[b] = N;
        if (N == 0) {
            quantile[b] = NAN;
            mean[b] = NAN;
            continue;
        }
        qsort(vals, (size_t)N, sizeof(float), cmp_float);
        double h = (double)(N - 1) * pct / 100.0;
        int64_t lo = (int64_t)floor(h);
        if (lo > N - 1)
            lo = N - 1;
        double x_lo = (double)vals[lo];
        double x_hi = lo + 1 < N ? (double)vals[lo + 1] : x_lo;
        quantile[b] = x_lo + (h - (double)lo) * (x_hi - x_lo);
        mean[b] = sum / (double)N;
    }
    free(vals);
}
