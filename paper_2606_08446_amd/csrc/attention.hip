// GQA decode attention over a paged KV cache, sparse (selected pages) or dense (all pages):
// the attention term of the cost models of Sec. 3.3 (Eq. dense-cost, Eq. sparse-cost) of
// arXiv 2606.08446, with the block-sparse token set of Sec. 2.
//
// Work split: one workgroup (4 waves) per (sequence, KV head, split), a split being up to
// `pages_per_split` consecutive entries of the page list (the top-k list, or 0..n-1).  The
// waves of a workgroup take the split's pages round-robin and run an online softmax over
// 16-token chunks; their states are merged in LDS and written as one partial (m, l, o).
// k_combine merges the partials of a (sequence, query head) with log-sum-exp weights.
//
// Per 16-token chunk, one wave computes all G <= 16 query heads of its KV head on MFMA:
//   QK:  D[t][g] = sum_d K[t][d] q[g][d]  - 4 x mfma_f32_16x16x32_bf16
//        A = K (row = token, lane row lane%16, 8 channels per lane, read straight from HBM),
//        B = q (column = head).  D lands as lane (g = lane%16, r = lane/16) holding the
//        logits of tokens 4r..4r+3 of head g.
//   PV:  O^T[d][g] += sum_t V[t][d] p[t][g]  - 8 x mfma_f32_16x16x16_bf16
//        B = the softmax numerators p, already in the layout the QK result left them in
//        (lane (g, r): tokens 4r..4r+3), rounded to bf16.  A = V^T: lane (m, r) loads the
//        16 bytes V[4r+j][8m .. 8m+8) of each of its 4 tokens and tile `c` takes element c
//        of each, so output row m of tile c is channel 8m + c.  No LDS transpose is needed.
//   O accumulators: lane (g, r) holds head g, channels 32r .. 32r+31 (8 tiles x 4 rows).
// The softmax runs in the log2 domain (scale * log2(e) folded into one multiply).
#include "common.h"

namespace sparrow {
namespace {

constexpr int kAttnThreads = 256;
constexpr int kAttnWaves = kAttnThreads / 64;
constexpr int kMaxPagesPerSplit = 64;
constexpr int kTokensPerSplit = 512;
constexpr int kOStride = kHeadDim + 4;  // LDS row stride of the wave merge (bank spread)

struct Chunk {
    u32x4_t k[4];  // A operand of the 4 QK instructions
    u32x4_t v[4];  // V rows 4r+j, channels 8m..8m+7
};

__device__ __forceinline__ void load_chunk(Chunk &c, const uint16_t *__restrict__ kbase,
                                           const uint16_t *__restrict__ vbase, int lr, int lg)
{
    const uint16_t *kp = kbase + lr * kHeadDim + 8 * lg;
#pragma unroll
    for (int i = 0; i < 4; ++i)
        c.k[i] = ld16_nt(kp + 32 * i);
    const uint16_t *vp = vbase + (4 * lg) * kHeadDim + 8 * lr;
#pragma unroll
    for (int j = 0; j < 4; ++j)
        c.v[j] = ld16_nt(vp + j * kHeadDim);
}

// Element `c` (0..7) of two 8 x bf16 vectors, packed as (x[c], y[c]).
__device__ __forceinline__ uint32_t pair_of(u32x4_t x, u32x4_t y, int c)
{
    const uint32_t a = x[c >> 1], b = y[c >> 1];
    return (c & 1) ? __builtin_amdgcn_perm(b, a, 0x07060302u)
                   : __builtin_amdgcn_perm(b, a, 0x05040100u);
}

template <bool kSparse>
__global__ __launch_bounds__(kAttnThreads) void k_attn_split(
    const uint16_t *__restrict__ q, const uint16_t *__restrict__ k_cache,
    const uint16_t *__restrict__ v_cache, const int32_t *__restrict__ block_table,
    const int32_t *__restrict__ seq_lens, const int32_t *__restrict__ ksel,
    const int32_t *__restrict__ idx, int k_max, int num_q_heads, int num_kv_heads, int ps,
    int max_pages, int pages_per_split, int max_splits, float scale_log2,
    float *__restrict__ o_part, float *__restrict__ ml_part)
{
    __shared__ int32_t s_phys[kMaxPagesPerSplit];
    __shared__ int32_t s_tok0[kMaxPagesPerSplit];
    __shared__ float s_m[kAttnWaves][16];
    __shared__ float s_l[kAttnWaves][16];
    __shared__ float s_o[kAttnWaves][16][kOStride];

    const int unit = blockIdx.y;
    const int split = blockIdx.x;
    const int b = unit / num_kv_heads;
    const int h = unit - b * num_kv_heads;
    const int G = num_q_heads / num_kv_heads;
    const int L = clamp_len(seq_lens[b], ps, max_pages);
    const int n = (L + ps - 1) / ps;
    int count = n;
    if (kSparse) {
        count = ksel[b];
        count = count < 0 ? 0 : (count > k_max ? k_max : count);
    }
    const int j0 = split * pages_per_split;
    if (j0 >= count)
        return;
    const int npg = min(pages_per_split, count - j0);
    const int tid = threadIdx.x;
    if (tid < npg) {
        const int lp = kSparse ? idx[(int64_t)unit * k_max + j0 + tid] : j0 + tid;
        int ph = -1;
        if (lp >= 0 && lp < n)
            ph = block_table[(int64_t)b * max_pages + lp];
        s_phys[tid] = ph;
        s_tok0[tid] = lp * ps;
    }

    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63;
    const int lr = lane & 15;
    const int lg = lane >> 4;

    // B operand of QK: lane (g = lr, r = lg) holds q[g][32i + 8r .. +8) for instruction i.
    bf16x8_t qf[4];
    {
        const uint16_t *qrow = q + ((int64_t)b * num_q_heads + (int64_t)h * G + lr) * kHeadDim;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            u32x4_t v = {0u, 0u, 0u, 0u};
            if (lr < G)
                v = ld16(qrow + 32 * i + 8 * lg);
            qf[i] = __builtin_bit_cast(bf16x8_t, v);
        }
    }
    __syncthreads();

    const int cpp = ps >> 4;  // 16-token chunks per page
    const int my_pages = npg > wave ? (npg - wave + kAttnWaves - 1) / kAttnWaves : 0;
    const int n_it = my_pages * cpp;
    const int64_t head_elems = (int64_t)ps * kHeadDim;

    // Chunk `it` of this wave: page slot wave + 4 * (it / cpp), sub-chunk it % cpp.
    auto chunk_info = [&](int it, int64_t &off, int &tok0) -> bool {
        const int slot = wave + kAttnWaves * (it / cpp);
        const int sub = it - (it / cpp) * cpp;
        const int ph = __builtin_amdgcn_readfirstlane(s_phys[slot]);
        tok0 = __builtin_amdgcn_readfirstlane(s_tok0[slot]) + 16 * sub;
        off = ((int64_t)ph * num_kv_heads + h) * head_elems + (int64_t)(16 * sub) * kHeadDim;
        return ph >= 0 && tok0 < L;
    };
    auto next_live = [&](int it, int64_t &off, int &tok0) -> int {
        while (it < n_it && !chunk_info(it, off, tok0))
            ++it;
        return it;
    };

    float m_run = -INFINITY;
    float l_run = 0.f;
    f32x4_t O[8];
#pragma unroll
    for (int c = 0; c < 8; ++c)
        O[c] = (f32x4_t){0.f, 0.f, 0.f, 0.f};

    int64_t off_next = 0;
    int tok_next = 0;
    int it = next_live(0, off_next, tok_next);
    Chunk nxt;
    if (it < n_it)
        load_chunk(nxt, k_cache + off_next, v_cache + off_next, lr, lg);
    while (it < n_it) {
        Chunk cur = nxt;
        const int tok0 = tok_next;
        it = next_live(it + 1, off_next, tok_next);
        if (it < n_it)
            load_chunk(nxt, k_cache + off_next, v_cache + off_next, lr, lg);

        // ---- logits of 16 tokens x 16 (padded) heads
        f32x4_t s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int i = 0; i < 4; ++i)
            s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, cur.k[i]),
                                                        qf[i], s, 0, 0, 0);
        const int valid = L - tok0;  // >= 1
        float z[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
            z[i] = (4 * lg + i < valid) ? s[i] * scale_log2 : -INFINITY;
        float cm = fmaxf(fmaxf(z[0], z[1]), fmaxf(z[2], z[3]));
        cm = fmaxf(cm, __shfl_xor(cm, 16, 64));
        cm = fmaxf(cm, __shfl_xor(cm, 32, 64));
        const float m_new = fmaxf(m_run, cm);
        const float alpha = exp2f(m_run - m_new);
        const uint32_t p01 = pack_bf16(exp2f(z[0] - m_new), exp2f(z[1] - m_new));
        const uint32_t p23 = pack_bf16(exp2f(z[2] - m_new), exp2f(z[3] - m_new));
        l_run = l_run * alpha + ((bf16_lo(p01) + bf16_hi(p01)) + (bf16_lo(p23) + bf16_hi(p23)));
        m_run = m_new;
        if (__ballot(alpha != 1.f)) {
#pragma unroll
            for (int c = 0; c < 8; ++c)
                O[c] *= alpha;
        }
        if (valid < 16) {  // tokens past the length: zero V (cache slots may hold anything)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (4 * lg + j >= valid)
                    cur.v[j] = (u32x4_t){0u, 0u, 0u, 0u};
        }
        // ---- O^T += V^T P
        const s16x4_t pb = __builtin_bit_cast(s16x4_t, (u32x2_t){p01, p23});
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            const u32x2_t a = {pair_of(cur.v[0], cur.v[1], c), pair_of(cur.v[2], cur.v[3], c)};
            O[c] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4_t, a), pb,
                                                             O[c], 0, 0, 0);
        }
    }

    // ---- merge the waves of the workgroup
    l_run += __shfl_xor(l_run, 16, 64);
    l_run += __shfl_xor(l_run, 32, 64);
    if (lg == 0) {
        s_m[wave][lr] = m_run;
        s_l[wave][lr] = l_run;
    }
#pragma unroll
    for (int c = 0; c < 8; ++c)
#pragma unroll
        for (int i = 0; i < 4; ++i)
            s_o[wave][lr][32 * lg + 8 * i + c] = O[c][i];
    __syncthreads();

    const int64_t pbase = (int64_t)unit * max_splits + split;
    for (int e = tid; e < G * kHeadDim; e += kAttnThreads) {
        const int g = e >> 7;
        const int d = e & (kHeadDim - 1);
        float M = s_m[0][g];
#pragma unroll
        for (int w = 1; w < kAttnWaves; ++w)
            M = fmaxf(M, s_m[w][g]);
        float acc = 0.f, lsum = 0.f;
        if (M != -INFINITY) {
#pragma unroll
            for (int w = 0; w < kAttnWaves; ++w) {
                const float f = exp2f(s_m[w][g] - M);
                acc += f * s_o[w][g][d];
                lsum += f * s_l[w][g];
            }
        }
        o_part[(pbase * G + g) * kHeadDim + d] = acc;
        if (d == 0) {
            ml_part[(pbase * G + g) * 2 + 0] = M;
            ml_part[(pbase * G + g) * 2 + 1] = lsum;
        }
    }
}

__global__ __launch_bounds__(kHeadDim) void k_combine(
    const float *__restrict__ o_part, const float *__restrict__ ml_part,
    const int32_t *__restrict__ seq_lens, const int32_t *__restrict__ ksel, int k_max,
    int sparse, int num_q_heads, int num_kv_heads, int ps, int max_pages, int pages_per_split,
    int max_splits, void *__restrict__ out, int out_bf16)
{
    const int bj = blockIdx.x;
    const int b = bj / num_q_heads;
    const int j = bj - b * num_q_heads;
    const int G = num_q_heads / num_kv_heads;
    const int h = j / G;
    const int g = j - h * G;
    const int unit = b * num_kv_heads + h;
    const int d = threadIdx.x;
    const int L = clamp_len(seq_lens[b], ps, max_pages);
    int count = (L + ps - 1) / ps;
    if (sparse) {
        count = ksel[b];
        count = count < 0 ? 0 : (count > k_max ? k_max : count);
    }
    const int n_splits = (count + pages_per_split - 1) / pages_per_split;
    const float *ml = ml_part + ((int64_t)unit * max_splits * G + g) * 2;
    const float *op = o_part + ((int64_t)unit * max_splits * G + g) * kHeadDim + d;
    float M = -INFINITY;
    for (int s = 0; s < n_splits; ++s)
        M = fmaxf(M, ml[(int64_t)s * G * 2]);
    float result = 0.f;
    if (M != -INFINITY) {
        float acc = 0.f, lsum = 0.f;
        for (int s = 0; s < n_splits; ++s) {
            const float f = exp2f(ml[(int64_t)s * G * 2] - M);
            acc += f * op[(int64_t)s * G * kHeadDim];
            lsum += f * ml[(int64_t)s * G * 2 + 1];
        }
        result = acc / lsum;
    }
    const int64_t o = (int64_t)bj * kHeadDim + d;
    if (out_bf16)
        static_cast<uint16_t *>(out)[o] = (uint16_t)to_bf16_bits(result);
    else
        static_cast<float *>(out)[o] = result;
}

}  // namespace

AttnPlan plan_attention(const sparrow_shape_t &s, int32_t max_count)
{
    AttnPlan p;
    const int64_t units = (int64_t)s.batch * s.num_kv_heads;
    int pps = kTokensPerSplit / s.page_size;
    if (pps > kMaxPagesPerSplit)
        pps = kMaxPagesPerSplit;
    const int min_pps = kAttnWaves;
    if (max_count < 1)
        max_count = 1;
    // Small batches: shorter splits so that the grid still covers the chip.
    while (pps > min_pps && units * ((max_count + pps - 1) / pps) < 2048)
        pps >>= 1;
    if (pps < min_pps)
        pps = min_pps;
    p.pages_per_split = pps;
    p.max_splits = (max_count + pps - 1) / pps;
    const int G = s.num_q_heads / s.num_kv_heads;
    const size_t per_split = (size_t)G * (kHeadDim + 2) * sizeof(float);
    p.workspace_bytes = (size_t)units * p.max_splits * per_split;
    return p;
}

hipError_t launch_attention(const sparrow_shape_t &s, const AttnPlan &plan, const void *q,
                            const void *k_cache, const void *v_cache, const int32_t *block_table,
                            const int32_t *seq_lens, const int32_t *k, const int32_t *idx,
                            int32_t k_max, float scale, void *out, int out_dtype,
                            void *workspace, hipStream_t stream)
{
    const int units = s.batch * s.num_kv_heads;
    const int G = s.num_q_heads / s.num_kv_heads;
    float *o_part = static_cast<float *>(workspace);
    float *ml_part = o_part + (size_t)units * plan.max_splits * G * kHeadDim;
    const float scale_log2 = scale * 1.4426950408889634f;
    const bool sparse = idx != nullptr;
    const dim3 grid(plan.max_splits, units);
    if (sparse)
        hipLaunchKernelGGL(k_attn_split<true>, grid, dim3(kAttnThreads), 0, stream,
                           static_cast<const uint16_t *>(q), static_cast<const uint16_t *>(k_cache),
                           static_cast<const uint16_t *>(v_cache), block_table, seq_lens, k, idx,
                           k_max, s.num_q_heads, s.num_kv_heads, s.page_size,
                           s.max_pages_per_seq, plan.pages_per_split, plan.max_splits, scale_log2,
                           o_part, ml_part);
    else
        hipLaunchKernelGGL(k_attn_split<false>, grid, dim3(kAttnThreads), 0, stream,
                           static_cast<const uint16_t *>(q), static_cast<const uint16_t *>(k_cache),
                           static_cast<const uint16_t *>(v_cache), block_table, seq_lens, nullptr,
                           nullptr, 0, s.num_q_heads, s.num_kv_heads, s.page_size,
                           s.max_pages_per_seq, plan.pages_per_split, plan.max_splits, scale_log2,
                           o_part, ml_part);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(k_combine, dim3(s.batch * s.num_q_heads), dim3(kHeadDim), 0, stream,
                       o_part, ml_part, seq_lens, k, k_max, sparse ? 1 : 0, s.num_q_heads,
                       s.num_kv_heads, s.page_size, s.max_pages_per_seq, plan.pages_per_split,
                       plan.max_splits, out, out_dtype == SPARROW_OUT_BF16 ? 1 : 0);
    return hipGetLastError();
}

}  // namespace sparrow
