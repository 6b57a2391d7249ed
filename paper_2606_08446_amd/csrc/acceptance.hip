// Per-token acceptance rate between the dense policy and the sparse rollout (Sec. 3.1,
// Eq. 1 of arXiv 2606.08446) and its lower-tail statistic per length bin (Sec. 3.1-3.2).
//
// k_acceptance: alpha_t = sum_x min(p(x), q(x)) with p, q the softmax of the target and draft
// logit rows at inverse temperature tau.  One 1024-thread workgroup per token (one per CU)
// makes two passes over its two rows: an online log-sum-exp of both (plain loads), then
// sum_x exp(min(tau a_x - P, tau b_x - Q)) - one exp per vocabulary entry, since
// min(e^u, e^v) = e^min(u, v).  The first vectors of the rows stay on chip between the
// passes, 128 KiB of them in LDS and 12 (fp32) or 10 (bf16) per thread and row in registers
// (43 % of an fp32 row pair of Qwen3's vocabulary, three quarters of a bf16 one); the
// rest is read again, with non-temporal loads and from the end of the rows back, so the
// part read last in the first pass is read first again while the L2 may still hold it.
// Rows are read as 16-byte vectors; a row that does not start 16-byte aligned is handled
// with scalar head and tail elements.  Accumulation is fp32 per thread, tree reductions
// across the workgroup.
//
// k_acceptance_topk: the approximation from the top-K listed tokens' normalised
// log-probabilities, sum_i min(exp(lp_i), exp(lq_i)); one thread per token.
//
// k_tail_stats: one workgroup per position bin.  Count and fp64 sum of the bin's values,
// then the order statistics x_lo and x_lo+1 (lo = floor((N - 1) pct / 100)) by a radix
// select over order-preserving uint32 keys (8-bit digits, one scan of the tokens per
// digit), and the percentile x_lo + (h - lo)(x_lo+1 - x_lo) in fp64 with the multiply and
// the add rounded separately.
#include "common.h"

namespace sparrow {
namespace {

constexpr int kAccThreads = 1024;
constexpr int kAccWaves = kAccThreads / 64;
constexpr int kAccLdsVecs = 4;  // 16-byte vectors of each row a thread keeps in LDS
constexpr int kTailThreads = 1024;
constexpr int kTailWaves = kTailThreads / 64;

template <typename T> struct Logit;
template <> struct Logit<float> {
    static constexpr int kVec = 4;  // elements per 16-byte vector
    static constexpr int kKeep = 12;  // vectors of each row a thread keeps in registers
    static constexpr int kBatch = 1;  // vectors of each row per load batch of either pass
    __device__ static float at(const float *row, int64_t i) { return row[i]; }
    __device__ static void unpack(u32x4_t v, float (&x)[kVec])
    {
#pragma unroll
        for (int e = 0; e < 4; ++e)
            x[e] = __uint_as_float(v[e]);
    }
};
template <> struct Logit<uint16_t> {
    static constexpr int kVec = 8;
    static constexpr int kKeep = 10;  // (measured: the fastest pairs that compile without
    static constexpr int kBatch = 2;  // spills)
    __device__ static float at(const uint16_t *row, int64_t i)
    {
        return __uint_as_float((uint32_t)row[i] << 16);
    }
    __device__ static void unpack(u32x4_t v, float (&x)[kVec])
    {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            x[2 * e] = bf16_lo(v[e]);
            x[2 * e + 1] = bf16_hi(v[e]);
        }
    }
};

// 2^x and log2 x on the VALU's transcendental unit (v_exp_f32 / v_log_f32).  The rate is
// computed in the base-2 domain with the scale ts = |tau| log2(e) folded into each
// exponent's FMA: 2^(ts x - m) is one v_fma_f32 and one v_exp_f32 per element, and the
// running maximum is taken on the unscaled values (ts >= 0 preserves their order; a
// negative tau is handled by negating the logits as they are read).
__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float log2_hw(float x) { return __builtin_amdgcn_logf(x); }

// Running (max, sum of 2^(ts x - max)) of base-2-scaled logits (max on the scaled scale).
struct Lse {
    float m, s;
};

__device__ __forceinline__ Lse lse_merge(Lse a, Lse b)
{
    const float m = fmaxf(a.m, b.m);
    if (m == -INFINITY)
        return {m, 0.f};
    return {m, a.s * exp2_hw(a.m - m) + b.s * exp2_hw(b.m - m)};
}

// Adds the unscaled values x (scale ts >= 0) to the running log-sum-exp.
template <int N>
__device__ __forceinline__ void lse_add(Lse &r, const float (&x)[N], float ts)
{
    float mx = x[0];
#pragma unroll
    for (int e = 1; e < N; ++e)
        mx = fmaxf(mx, x[e]);
    mx *= ts;
    if (mx > r.m) {
        r.s = r.m == -INFINITY ? 0.f : r.s * exp2_hw(r.m - mx);
        r.m = mx;
    }
    // While every entry seen is -inf (masked vocabulary entries), the chunk adds nothing:
    // 2^(x - 0) = 0 for x = -inf, where x - r.m would be -inf - (-inf) = NaN.
    const float m = r.m == -INFINITY ? 0.f : r.m;
    float s = 0.f;
#pragma unroll
    for (int e = 0; e < N; ++e)
        s += exp2_hw(fmaf(ts, x[e], -m));
    r.s += s;
}

template <typename T>
__device__ __forceinline__ void row_split(const T *row, int V, int &head, int &nvec)
{
    constexpr int W = Logit<T>::kVec;
    const uintptr_t mis = reinterpret_cast<uintptr_t>(row) & 15u;
    head = mis == 0 ? 0 : (int)((16u - mis) / sizeof(T));
    if (head > V)
        head = V;
    nvec = (V - head) / W;
}

// Workgroup-wide reduction of a pair of Lse (target, draft) through LDS.
__device__ void block_lse2(Lse &a, Lse &b, Lse (*s_red)[2])
{
#pragma unroll
    for (int x = 1; x < 64; x <<= 1) {
        a = lse_merge(a, {__shfl_xor(a.m, x, 64), __shfl_xor(a.s, x, 64)});
        b = lse_merge(b, {__shfl_xor(b.m, x, 64), __shfl_xor(b.s, x, 64)});
    }
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
        s_red[wave][0] = a;
        s_red[wave][1] = b;
    }
    __syncthreads();
    a = s_red[0][0];
    b = s_red[0][1];
    for (int w = 1; w < kAccWaves; ++w) {
        a = lse_merge(a, s_red[w][0]);
        b = lse_merge(b, s_red[w][1]);
    }
}

// Logit as read, negated when the inverse temperature is negative (so that the scale ts
// applied to it is >= 0).
template <bool kNeg>
__device__ __forceinline__ float oriented(float x)
{
    return kNeg ? -x : x;
}

template <typename T, bool kNeg>
__device__ __forceinline__ void lse_add_vec(Lse &a, Lse &b, u32x4_t va, u32x4_t vb, float ts)
{
    constexpr int W = Logit<T>::kVec;
    float xa[W], xb[W];
    Logit<T>::unpack(va, xa);
    Logit<T>::unpack(vb, xb);
#pragma unroll
    for (int e = 0; e < W; ++e) {
        xa[e] = oriented<kNeg>(xa[e]);
        xb[e] = oriented<kNeg>(xb[e]);
    }
    lse_add(a, xa, ts);
    lse_add(b, xb, ts);
}

// sum over the vector's entries of 2^min(ts a - P, ts b - Q)
template <typename T, bool kNeg>
__device__ __forceinline__ float min_sum_vec(u32x4_t va, u32x4_t vb, float ts, float P, float Q)
{
    constexpr int W = Logit<T>::kVec;
    float xa[W], xb[W];
    Logit<T>::unpack(va, xa);
    Logit<T>::unpack(vb, xb);
    float acc = 0.f;
#pragma unroll
    for (int e = 0; e < W; ++e)
        acc += exp2_hw(fminf(fmaf(ts, oriented<kNeg>(xa[e]), -P),
                             fmaf(ts, oriented<kNeg>(xb[e]), -Q)));
    return acc;
}

// The row pair's 16-byte vectors v = tid + j * kAccThreads: j < kAccLdsVecs stay in LDS
// between the passes (s_keep, the thread's own slots), the next Logit<T>::kKeep in this
// thread's registers, the rest are read again in the second pass.
template <typename T, bool kNeg>
__global__ __launch_bounds__(kAccThreads) void k_acceptance(const T *__restrict__ target,
                                                            const T *__restrict__ draft, int V,
                                                            float ts, float *__restrict__ alpha)
{
    extern __shared__ u32x4_t s_keep[];  // [2][kAccLdsVecs][kAccThreads]
    __shared__ Lse s_red[kAccWaves][2];
    __shared__ float s_sum[kAccWaves];
    constexpr int R = Logit<T>::kKeep, L = kAccLdsVecs, NB = Logit<T>::kBatch;
    const int64_t t = blockIdx.x;
    const T *pr = target + t * V;
    const T *qr = draft + t * V;
    const int tid = threadIdx.x;
    int head, nvec;
    row_split(pr, V, head, nvec);
    const int tail0 = head + nvec * Logit<T>::kVec;
    const u32x4_t *pv = reinterpret_cast<const u32x4_t *>(pr + head);
    const u32x4_t *qv = reinterpret_cast<const u32x4_t *>(qr + head);
    const int onchip = (R + L) * kAccThreads;  // vectors of each row held on chip

    // ---- pass 1: log-sum-exp of both rows (plain loads), keeping the first vectors: those
    // for LDS first (their registers are free again before the kept ones are loaded)
    Lse a{-INFINITY, 0.f}, b{-INFINITY, 0.f};
    for (int i = tid; i < head; i += kAccThreads) {
        const float xa[1] = {oriented<kNeg>(Logit<T>::at(pr, i))};
        const float xb[1] = {oriented<kNeg>(Logit<T>::at(qr, i))};
        lse_add(a, xa, ts);
        lse_add(b, xb, ts);
    }
    for (int i = tail0 + tid; i < V; i += kAccThreads) {
        const float xa[1] = {oriented<kNeg>(Logit<T>::at(pr, i))};
        const float xb[1] = {oriented<kNeg>(Logit<T>::at(qr, i))};
        lse_add(a, xa, ts);
        lse_add(b, xb, ts);
    }
    {
        u32x4_t la[L], lb[L];
#pragma unroll
        for (int j = 0; j < L; ++j) {
            const int v = tid + j * kAccThreads;
            la[j] = lb[j] = (u32x4_t){0u, 0u, 0u, 0u};
            if (v < nvec) {
                la[j] = pv[v];
                lb[j] = qv[v];
            }
        }
#pragma unroll
        for (int j = 0; j < L; ++j) {
            if (tid + j * kAccThreads < nvec) {
                lse_add_vec<T, kNeg>(a, b, la[j], lb[j], ts);
                s_keep[j * kAccThreads + tid] = la[j];
                s_keep[(L + j) * kAccThreads + tid] = lb[j];
            }
        }
    }
    __builtin_amdgcn_sched_barrier(0);  // the kept vectors' loads stay behind this point
    u32x4_t ka[R], kb[R];
#pragma unroll
    for (int j = 0; j < R; ++j) {
        const int v = tid + (L + j) * kAccThreads;
        ka[j] = kb[j] = (u32x4_t){0u, 0u, 0u, 0u};
        if (v < nvec) {
            ka[j] = pv[v];
            kb[j] = qv[v];
        }
    }
#pragma unroll
    for (int j = 0; j < R; ++j)
        if (tid + (L + j) * kAccThreads < nvec)
            lse_add_vec<T, kNeg>(a, b, ka[j], kb[j], ts);
    int v = onchip + tid;
    for (; v + (NB - 1) * kAccThreads < nvec; v += NB * kAccThreads) {
        u32x4_t ra[NB], rb[NB];
#pragma unroll
        for (int u = 0; u < NB; ++u) {
            ra[u] = pv[v + u * kAccThreads];
            rb[u] = qv[v + u * kAccThreads];
        }
#pragma unroll
        for (int u = 0; u < NB; ++u)
            lse_add_vec<T, kNeg>(a, b, ra[u], rb[u], ts);
    }
    for (; v < nvec; v += kAccThreads)
        lse_add_vec<T, kNeg>(a, b, pv[v], qv[v], ts);
    block_lse2(a, b, s_red);
    const float P = a.m + log2_hw(a.s);  // base-2 log-sum-exp of the scaled rows
    const float Q = b.m + log2_hw(b.s);

    // ---- pass 2: sum of 2^min(ts a - P, ts b - Q) = exp(min(tau a - lse_a, tau b - lse_b)):
    // the vectors read again first, from the end of the rows back (non-temporal loads), then
    // those in LDS and in registers
    float acc = 0.f;
    for (int i = tid; i < head; i += kAccThreads)
        acc += exp2_hw(fminf(fmaf(ts, oriented<kNeg>(Logit<T>::at(pr, i)), -P),
                             fmaf(ts, oriented<kNeg>(Logit<T>::at(qr, i)), -Q)));
    for (int i = tail0 + tid; i < V; i += kAccThreads)
        acc += exp2_hw(fminf(fmaf(ts, oriented<kNeg>(Logit<T>::at(pr, i)), -P),
                             fmaf(ts, oriented<kNeg>(Logit<T>::at(qr, i)), -Q)));
    const int nre = nvec - onchip;  // vectors read again (none if <= 0)
    int w = tid;
    for (; w + (NB - 1) * kAccThreads < nre; w += NB * kAccThreads) {
        u32x4_t ra[NB], rb[NB];
#pragma unroll
        for (int u = 0; u < NB; ++u) {
            ra[u] = ld16_nt(pv + (nvec - 1 - (w + u * kAccThreads)));
            rb[u] = ld16_nt(qv + (nvec - 1 - (w + u * kAccThreads)));
        }
#pragma unroll
        for (int u = 0; u < NB; ++u)
            acc += min_sum_vec<T, kNeg>(ra[u], rb[u], ts, P, Q);
    }
    for (; w < nre; w += kAccThreads)
        acc += min_sum_vec<T, kNeg>(ld16_nt(pv + (nvec - 1 - w)), ld16_nt(qv + (nvec - 1 - w)),
                                    ts, P, Q);
#pragma unroll
    for (int j = 0; j < R; ++j) {
        // (opaque to the compiler, so that it unpacks the kept vectors again here instead of
        // holding the first pass's unpacked bf16 elements, twice the registers, until now)
        if constexpr (sizeof(T) == 2)
            asm volatile("" : "+v"(ka[j]), "+v"(kb[j]));
        if (tid + (L + j) * kAccThreads < nvec)
            acc += min_sum_vec<T, kNeg>(ka[j], kb[j], ts, P, Q);
    }
#pragma unroll
    for (int j = 0; j < L; ++j)
        if (tid + j * kAccThreads < nvec)
            acc += min_sum_vec<T, kNeg>(s_keep[j * kAccThreads + tid],
                                        s_keep[(L + j) * kAccThreads + tid], ts, P, Q);
#pragma unroll
    for (int x = 1; x < 64; x <<= 1)
        acc += __shfl_xor(acc, x, 64);
    if ((tid & 63) == 0)
        s_sum[tid >> 6] = acc;
    __syncthreads();
    if (tid == 0) {
        float total = 0.f;
        for (int w2 = 0; w2 < kAccWaves; ++w2)
            total += s_sum[w2];
        alpha[t] = total;
    }
}

__global__ __launch_bounds__(256) void k_acceptance_topk(const float *__restrict__ lp_target,
                                                         const float *__restrict__ lp_draft,
                                                         int64_t T, int K,
                                                         float *__restrict__ alpha)
{
    for (int64_t t = blockIdx.x * 256ll + threadIdx.x; t < T; t += (int64_t)gridDim.x * 256) {
        float acc = 0.f;
        for (int i = 0; i < K; ++i)
            acc += __expf(fminf(lp_target[t * K + i], lp_draft[t * K + i]));
        alpha[t] = acc;
    }
}

// fp32 -> uint32 whose unsigned order is the order of the values (-0 == +0).
__device__ __forceinline__ uint32_t float_key(float s)
{
    uint32_t u = __float_as_uint(s);
    if (u == 0x80000000u)
        u = 0u;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float key_float(uint32_t k)
{
    return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

__device__ __forceinline__ int bin_of(int32_t pos, int bin_tokens, int n_bins)
{
    if (pos < 0)
        return -1;
    const int b = pos / bin_tokens;
    return b > n_bins - 1 ? n_bins - 1 : b;
}

// Exclusive-count radix select: the key of rank k (0-based) among the bin's keys.
__device__ uint32_t select_rank(const float *alpha, const int32_t *pos, int64_t T, int bin,
                                int bin_tokens, int n_bins, int64_t k, uint32_t *hist,
                                int64_t *s_sel)
{
    uint32_t prefix = 0, mask = 0;
    for (int shift = 24; shift >= 0; shift -= 8) {
        for (int i = threadIdx.x; i < 256; i += kTailThreads)
            hist[i] = 0;
        __syncthreads();
        for (int64_t t = threadIdx.x; t < T; t += kTailThreads) {
            if (bin_of(pos[t], bin_tokens, n_bins) != bin)
                continue;
            const uint32_t key = float_key(alpha[t]);
            if ((key & mask) == prefix)
                atomicAdd(&hist[(key >> shift) & 255u], 1u);
        }
        __syncthreads();
        if (threadIdx.x == 0) {  // 256 bins: a serial walk is short
            int64_t below = 0;
            int d = 0;
            for (; d < 255; ++d) {
                if (below + hist[d] > k)
                    break;
                below += hist[d];
            }
            s_sel[0] = d;
            s_sel[1] = k - below;
        }
        __syncthreads();
        prefix |= (uint32_t)s_sel[0] << shift;
        mask |= 255u << shift;
        k = s_sel[1];
        __syncthreads();
    }
    return prefix;
}

__global__ __launch_bounds__(kTailThreads) void k_tail_stats(
    const float *__restrict__ alpha, const int32_t *__restrict__ pos, int64_t T, int bin_tokens,
    int n_bins, double pct, double *__restrict__ quantile, double *__restrict__ mean,
    int64_t *__restrict__ count)
{
    __shared__ uint32_t hist[256];
    __shared__ int64_t s_sel[2];
    __shared__ double s_sum[kTailWaves];
    __shared__ unsigned long long s_cnt[kTailWaves];
    __shared__ uint32_t s_min;
    const int bin = blockIdx.x;
    double sum = 0.0;
    unsigned long long n = 0;
    for (int64_t t = threadIdx.x; t < T; t += kTailThreads) {
        if (bin_of(pos[t], bin_tokens, n_bins) == bin) {
            sum += (double)alpha[t];
            ++n;
        }
    }
#pragma unroll
    for (int x = 1; x < 64; x <<= 1) {
        sum += __shfl_xor(sum, x, 64);
        n += __shfl_xor(n, x, 64);
    }
    if ((threadIdx.x & 63) == 0) {
        s_sum[threadIdx.x >> 6] = sum;
        s_cnt[threadIdx.x >> 6] = n;
    }
    __syncthreads();
    double total = 0.0;
    int64_t N = 0;
    for (int w = 0; w < kTailWaves; ++w) {
        total += s_sum[w];
        N += (int64_t)s_cnt[w];
    }
    if (N == 0) {
        if (threadIdx.x == 0) {
            count[bin] = 0;
            mean[bin] = __builtin_nan("");
            quantile[bin] = __builtin_nan("");
        }
        return;
    }
    const double h = (double)(N - 1) * pct / 100.0;
    int64_t lo = (int64_t)floor(h);
    if (lo > N - 1)
        lo = N - 1;
    const uint32_t klo = select_rank(alpha, pos, T, bin, bin_tokens, n_bins, lo, hist, s_sel);
    double x_hi;
    const double x_lo = (double)key_float(klo);
    if (lo + 1 >= N) {
        x_hi = x_lo;
    } else {
        // rank lo + 1: x_lo again if enough keys equal it, else the smallest key above it
        if (threadIdx.x == 0)
            s_min = 0xffffffffu;
        __syncthreads();
        unsigned int le = 0;  // keys <= x_lo seen by this thread
        uint32_t above = 0xffffffffu;
        for (int64_t t = threadIdx.x; t < T; t += kTailThreads) {
            if (bin_of(pos[t], bin_tokens, n_bins) != bin)
                continue;
            const uint32_t key = float_key(alpha[t]);
            if (key <= klo)
                ++le;
            else if (key < above)
                above = key;
        }
#pragma unroll
        for (int x = 1; x < 64; x <<= 1) {
            le += __shfl_xor(le, x, 64);
            above = min(above, (uint32_t)__shfl_xor((int)above, x, 64));
        }
        if ((threadIdx.x & 63) == 0) {
            s_cnt[threadIdx.x >> 6] = le;
            atomicMin(&s_min, above);
        }
        __syncthreads();
        int64_t n_le = 0;
        for (int w = 0; w < kTailWaves; ++w)
            n_le += (int64_t)s_cnt[w];
        x_hi = n_le > lo + 1 ? x_lo : (double)key_float(s_min);
    }
    if (threadIdx.x == 0) {
        // the definition's separate multiply and add (device code otherwise contracts to fma)
#pragma clang fp contract(off)
        count[bin] = N;
        mean[bin] = total / (double)N;
        quantile[bin] = x_lo + (h - (double)lo) * (x_hi - x_lo);
    }
}

}  // namespace

hipError_t launch_acceptance(int64_t T, int V, int dtype, const void *target, const void *draft,
                             float tau, float *alpha, hipStream_t stream)
{
    // The vectors kept in LDS between the passes (128 KiB: one workgroup per CU).
    constexpr size_t kKeep = 2 * (size_t)kAccLdsVecs * kAccThreads * sizeof(u32x4_t);
    const bool neg = tau < 0.f;
    const float ts = (neg ? -tau : tau) * 1.44269504088896340736f;  // |tau| log2(e)
    const dim3 grid((unsigned)T), block(kAccThreads);
    if (dtype == SPARROW_LOGITS_BF16) {
        auto k = neg ? k_acceptance<uint16_t, true> : k_acceptance<uint16_t, false>;
        hipLaunchKernelGGL(k, grid, block, kKeep, stream,
                           static_cast<const uint16_t *>(target),
                           static_cast<const uint16_t *>(draft), V, ts, alpha);
    } else {
        auto k = neg ? k_acceptance<float, true> : k_acceptance<float, false>;
        hipLaunchKernelGGL(k, grid, block, kKeep, stream, static_cast<const float *>(target),
                           static_cast<const float *>(draft), V, ts, alpha);
    }
    return hipGetLastError();
}

hipError_t launch_acceptance_topk(int64_t T, int K, const float *lp_target, const float *lp_draft,
                                  float *alpha, hipStream_t stream)
{
    int64_t blocks = (T + 255) / 256;
    if (blocks > 65535)
        blocks = 65535;
    hipLaunchKernelGGL(k_acceptance_topk, dim3((unsigned)blocks), dim3(256), 0, stream, lp_target,
                       lp_draft, T, K, alpha);
    return hipGetLastError();
}

hipError_t launch_tail_stats(int64_t T, const float *alpha, const int32_t *pos, int bin_tokens,
                             int n_bins, double pct, double *quantile, double *mean,
                             int64_t *count, hipStream_t stream)
{
    hipLaunchKernelGGL(k_tail_stats, dim3(n_bins), dim3(kTailThreads), 0, stream, alpha, pos, T,
                       bin_tokens, n_bins, pct, quantile, mean, count);
    return hipGetLastError();
}

}  // namespace sparrow
