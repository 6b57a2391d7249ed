// Page scoring and block top-k selection (Sec. 3.3 and Sec. 3.2 of arXiv 2606.08446).
//
// k_page_score: the score of page p for KV head h is
//     S(p) = sum_{g<G} sum_i max(q_{g,i} mn_i, q_{g,i} mx_i).
// Because mn_i <= mx_i, max(q mn, q mx) = q+ mx + q- mn with q+ = max(q, 0) and
// q- = min(q, 0), so S(p) = sum_i (Q-_i mn_i + Q+_i mx_i) with Q+-_i = sum_g q+-_{g,i}:
// one 256-long dot product of the page's metadata row [mn | mx] with a weight vector w
// that depends only on the query group.  Pages of a sequence form the rows of a
// (pages x 256) bf16 matrix, so the scores are a matrix-vector product, run on MFMA
// 16x16x32 bf16 tiles: 16 pages x 32 channels per instruction, w split exactly into
// three bf16 parts (hi + mid + lo == w) placed in the first three columns of B.  The
// three partial sums are added in fp32.  Every page goes through the same instruction
// sequence, so pages with identical metadata get bit-identical scores (exact ties stay
// ties).  Each workgroup scores 256 pages of one (sequence, KV head) and writes fp32
// scores to the workspace; sequences whose budget covers every page are skipped.
//
// k_topk: one workgroup per (sequence, KV head) selects the k largest scores with ties
// to the lower page index.  Scores become order-preserving uint32 keys in LDS; a radix
// select over 8-bit digits (starting below the bits all keys share) finds the k-th key
// T and how many keys equal to T to keep; one block scan of (count > T, count == T)
// then places every kept page at its rank in ascending page order.
#include "common.h"

namespace sparrow {
namespace {

constexpr int kScoreThreads = 256;
constexpr int kScorePagesPerWave = 64;
constexpr int kScorePagesPerGroup = kScoreThreads / 64 * kScorePagesPerWave;  // 256
constexpr int kTopkThreads = 512;
constexpr int kTopkWaves = kTopkThreads / 64;

__global__ __launch_bounds__(kScoreThreads) void k_page_score(
    const uint16_t *__restrict__ q, const uint16_t *__restrict__ meta,
    const int32_t *__restrict__ block_table, const int32_t *__restrict__ seq_lens, Sched sched,
    int k_max, int num_q_heads, int num_kv_heads, int ps, int max_pages, float *__restrict__ scores)
{
    __shared__ __attribute__((aligned(16))) uint16_t w_parts[3][2 * kHeadDim];

    const int unit = blockIdx.y;
    const int b = unit / num_kv_heads;
    const int h = unit - b * num_kv_heads;
    const int L = clamp_len(seq_lens[b], ps, max_pages);
    const int n = (L + ps - 1) / ps;
    const int page0 = blockIdx.x * kScorePagesPerGroup;
    if (page0 >= n)
        return;
    if (budget_pages(L, ps, sched, k_max) >= n)
        return;  // every page is kept: nothing to score
    const int G = num_q_heads / num_kv_heads;
    const int tid = threadIdx.x;

    // Weight vector: element e < 128 multiplies mn_e, element e >= 128 multiplies mx_{e-128}.
    {
        const int e = tid;
        const int i = e & (kHeadDim - 1);
        const uint16_t *qh = q + ((int64_t)b * num_q_heads + (int64_t)h * G) * kHeadDim + i;
        float acc = 0.f;
        for (int g = 0; g < G; ++g) {
            const float v = __uint_as_float((uint32_t)qh[g * kHeadDim] << 16);
            acc += e < kHeadDim ? fminf(v, 0.f) : fmaxf(v, 0.f);
        }
        // acc == hi + mid + lo exactly: each remainder is exact (Sterbenz) and the three
        // 8-bit significands cover the 24 bits of acc.
        const uint32_t hi = to_bf16_bits(acc);
        const float r1 = acc - __uint_as_float(hi << 16);
        const uint32_t mid = to_bf16_bits(r1);
        const float r2 = r1 - __uint_as_float(mid << 16);
        const uint32_t lo = to_bf16_bits(r2);
        w_parts[0][e] = (uint16_t)hi;
        w_parts[1][e] = (uint16_t)mid;
        w_parts[2][e] = (uint16_t)lo;
    }
    __syncthreads();

    const int wave = tid >> 6;
    const int lane = tid & 63;
    const int lr = lane & 15;  // A: page row; B and D: column
    const int lg = lane >> 4;  // k sub-block of the operands; row block of D

    // B operand (k = channel e, n = part): lane holds w_parts[lr][32c + 8lg .. +8) for lr < 3.
    bf16x8_t wf[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) {
        u32x4_t v = {0u, 0u, 0u, 0u};
        if (lr < 3)
            v = *reinterpret_cast<const u32x4_t *>(&w_parts[lr][32 * c + 8 * lg]);
        wf[c] = __builtin_bit_cast(bf16x8_t, v);
    }

    const int64_t row_stride = (int64_t)num_kv_heads * 2 * kHeadDim;  // elements per phys page
    float *out = scores + (int64_t)unit * max_pages;
    for (int gi = 0; gi < kScorePagesPerWave / 16; ++gi) {
        const int base = page0 + wave * kScorePagesPerWave + gi * 16;
        if (base >= n)
            break;
        const int p = base + lr;
        u32x4_t a[8];
        if (p < n) {
            const int64_t phys = block_table[(int64_t)b * max_pages + p];
            const uint16_t *row = meta + phys * row_stride + (int64_t)h * 2 * kHeadDim + 8 * lg;
#pragma unroll
            for (int c = 0; c < 8; ++c)
                a[c] = ld16(row + 32 * c);
        } else {
#pragma unroll
            for (int c = 0; c < 8; ++c)
                a[c] = (u32x4_t){0u, 0u, 0u, 0u};
        }
        f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < 8; ++c)
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a[c]),
                                                          wf[c], acc, 0, 0, 0);
        // acc[i] = partial score of page base + 4lg + i against weight part lr.
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float d1 = __shfl_down(acc[i], 1, 16);
            const float d2 = __shfl_down(acc[i], 2, 16);
            const int pp = base + 4 * lg + i;
            if (lr == 0 && pp < n)
                out[pp] = acc[i] + (d1 + d2);
        }
    }
}

// fp32 score -> uint32 whose unsigned order is the order of the scores (-0 == +0).
__device__ __forceinline__ uint32_t score_key(float s)
{
    uint32_t u = __float_as_uint(s);
    if (u == 0x80000000u)
        u = 0u;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ uint32_t wave_inclusive_scan(uint32_t x, int lane)
{
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const uint32_t t = __shfl_up(x, d, 64);
        if (lane >= d)
            x += t;
    }
    return x;
}

__global__ __launch_bounds__(kTopkThreads) void k_topk(
    const float *__restrict__ scores, const int32_t *__restrict__ seq_lens, Sched sched,
    int k_max, int num_kv_heads, int ps, int max_pages, int32_t *__restrict__ out_k,
    int32_t *__restrict__ out_idx)
{
    extern __shared__ uint32_t keys[];  // [max_pages]
    __shared__ uint32_t hist[256];
    __shared__ uint32_t red_a[kTopkWaves], red_b[kTopkWaves], red_c[kTopkWaves];
    __shared__ uint32_t s_digit, s_rem;

    const int unit = blockIdx.x;
    const int b = unit / num_kv_heads;
    const int h = unit - b * num_kv_heads;
    const int L = clamp_len(seq_lens[b], ps, max_pages);
    const int n = (L + ps - 1) / ps;
    const int k = budget_pages(L, ps, sched, k_max);
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    int32_t *row = out_idx + (int64_t)unit * k_max;
    if (h == 0 && tid == 0)
        out_k[b] = k;
    if (k >= n) {  // every page kept (also n == 0)
        for (int i = tid; i < k_max; i += kTopkThreads)
            row[i] = i < n ? i : -1;
        return;
    }

    // Keys into LDS; block min and max.
    const float *src = scores + (int64_t)unit * max_pages;
    uint32_t kmin = 0xffffffffu, kmax = 0u;
    for (int i = tid; i < n; i += kTopkThreads) {
        const uint32_t key = score_key(src[i]);
        keys[i] = key;
        kmin = min(kmin, key);
        kmax = max(kmax, key);
    }
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) {
        kmin = min(kmin, (uint32_t)__shfl_xor(kmin, d, 64));
        kmax = max(kmax, (uint32_t)__shfl_xor(kmax, d, 64));
    }
    if (lane == 0) {
        red_a[wave] = kmin;
        red_b[wave] = kmax;
    }
    __syncthreads();
    kmin = red_a[0];
    kmax = red_b[0];
#pragma unroll
    for (int w = 1; w < kTopkWaves; ++w) {
        kmin = min(kmin, red_a[w]);
        kmax = max(kmax, red_b[w]);
    }

    // Radix select of the k-th largest key T, MSB digit first.  Bits above the highest
    // bit where kmin and kmax differ are shared by every key.
    uint32_t prefix = kmax;
    uint32_t rem = (uint32_t)k;  // keys still to take among those matching the prefix
    int shift = -8;
    if (kmin != kmax)
        shift = ((31 - __builtin_clz(kmin ^ kmax)) >> 3) << 3;
    for (; shift >= 0; shift -= 8) {
        const uint32_t hi_mask = shift >= 24 ? 0u : (0xffffffffu << (shift + 8));
        const uint32_t want = prefix & hi_mask;
        for (int i = tid; i < 256; i += kTopkThreads)
            hist[i] = 0u;
        __syncthreads();
        for (int i = tid; i < n; i += kTopkThreads) {
            const uint32_t key = keys[i];
            if ((key & hi_mask) == want)
                atomicAdd(&hist[(key >> shift) & 255u], 1u);
        }
        __syncthreads();
        if (wave == 0) {
            // lane l owns digits 255-4l .. 252-4l; counts accumulate from the top digit down
            const uint32_t c0 = hist[255 - 4 * lane], c1 = hist[254 - 4 * lane];
            const uint32_t c2 = hist[253 - 4 * lane], c3 = hist[252 - 4 * lane];
            const uint32_t tot = c0 + c1 + c2 + c3;
            const uint32_t incl = wave_inclusive_scan(tot, lane);
            uint32_t acc = incl - tot;  // keys with a larger digit
            if (acc < rem && rem <= incl) {
                int d;
                if (rem <= acc + c0) {
                    d = 255 - 4 * lane;
                } else if (rem <= acc + c0 + c1) {
                    acc += c0;
                    d = 254 - 4 * lane;
                } else if (rem <= acc + c0 + c1 + c2) {
                    acc += c0 + c1;
                    d = 253 - 4 * lane;
                } else {
                    acc += c0 + c1 + c2;
                    d = 252 - 4 * lane;
                }
                s_digit = (uint32_t)d;
                s_rem = rem - acc;
            }
        }
        __syncthreads();
        prefix = want | (s_digit << shift);
        rem = s_rem;
    }
    const uint32_t T = prefix;  // k-th largest key; keep every key > T and `rem` keys == T

    // Ranks: a kept page's position is (#keys > T before it) + min(#keys == T before it, rem).
    const int seg = (n + kTopkThreads - 1) / kTopkThreads;
    const int s0 = min(n, tid * seg);
    const int s1 = min(n, s0 + seg);
    uint32_t gt = 0u, eq = 0u;
    for (int i = s0; i < s1; ++i) {
        const uint32_t key = keys[i];
        gt += key > T;
        eq += key == T;
    }
    const uint32_t packed = (gt << 16) | eq;  // n <= 15360 < 2^16
    uint32_t incl = wave_inclusive_scan(packed, lane);
    if (lane == 63)
        red_c[wave] = incl;
    __syncthreads();
    uint32_t before = incl - packed;
    for (int w = 0; w < wave; ++w)
        before += red_c[w];
    uint32_t gt_b = before >> 16, eq_b = before & 0xffffu;
    for (int i = s0; i < s1; ++i) {
        const uint32_t key = keys[i];
        if (key > T) {
            const uint32_t pos = gt_b + min(eq_b, rem);
            if (pos < (uint32_t)k)
                row[pos] = i;
            ++gt_b;
        } else if (key == T) {
            if (eq_b < rem && gt_b + eq_b < (uint32_t)k)
                row[gt_b + eq_b] = i;
            ++eq_b;
        }
    }
    for (int i = k + tid; i < k_max; i += kTopkThreads)
        row[i] = -1;
}

}  // namespace

size_t score_topk_workspace(const sparrow_shape_t &s)
{
    return (size_t)s.batch * s.num_kv_heads * s.max_pages_per_seq * sizeof(float);
}

hipError_t launch_score_topk(const sparrow_shape_t &s, const void *q, const void *meta,
                             const int32_t *block_table, const int32_t *seq_lens,
                             const Sched &sched, int32_t k_max, int32_t *out_k,
                             int32_t *out_idx, void *workspace, hipStream_t stream)
{
    float *scores = static_cast<float *>(workspace);
    const int units = s.batch * s.num_kv_heads;
    const dim3 sgrid((s.max_pages_per_seq + kScorePagesPerGroup - 1) / kScorePagesPerGroup, units);
    hipLaunchKernelGGL(k_page_score, sgrid, dim3(kScoreThreads), 0, stream,
                       static_cast<const uint16_t *>(q), static_cast<const uint16_t *>(meta),
                       block_table, seq_lens, sched, k_max, s.num_q_heads, s.num_kv_heads,
                       s.page_size, s.max_pages_per_seq, scores);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    const size_t lds = (size_t)s.max_pages_per_seq * sizeof(uint32_t);
    hipLaunchKernelGGL(k_topk, dim3(units), dim3(kTopkThreads), lds, stream, scores, seq_lens,
                       sched, k_max, s.num_kv_heads, s.page_size, s.max_pages_per_seq, out_k,
                       out_idx);
    return hipGetLastError();
}

}  // namespace sparrow
