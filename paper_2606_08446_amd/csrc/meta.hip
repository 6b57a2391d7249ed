// Per-page key metadata: channel-wise min and max of each page's keys (the page landmark
// that block top-k selection scores, Sec. 3.3 / Appendix C of arXiv 2606.08446).
//
// One workgroup per (sequence, logical page) when rebuilding, or per sequence when
// updating the pages touched by freshly written tokens.  A thread owns one (KV head,
// 8-channel slice): it streams the slice of every valid token of the page (16 bytes per
// token, the 16 threads of a head covering one contiguous 256-byte key row), keeps
// min/max in registers and writes two 16-byte rows.  Min/max run on an integer image of
// the bf16 bit pattern whose order is the total order of the values (-0 below +0), so
// the result is one of the input patterns, bit for bit.
//
// With the mean landmark the thread instead sums its 8 channels over the page's tokens in
// token order (fp32 adds of exactly converted bf16 keys) and writes 8 fp32 sums.
#include "common.h"

namespace sparrow {
namespace {

constexpr int kMetaThreads = 128;

__device__ __forceinline__ void fold(u32x4_t v, int32_t (&mn)[8], int32_t (&mx)[8])
{
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        const int32_t lo = order16(v[w] & 0xffffu);
        const int32_t hi = order16(v[w] >> 16);
        mn[2 * w] = min(mn[2 * w], lo);
        mx[2 * w] = max(mx[2 * w], lo);
        mn[2 * w + 1] = min(mn[2 * w + 1], hi);
        mx[2 * w + 1] = max(mx[2 * w + 1], hi);
    }
}

// Min/max of one (page, head, 8-channel slice) over `valid` tokens of a page of PS tokens.
template <int PS>
__device__ __forceinline__ void slice_minmax(const uint16_t *__restrict__ src, int valid,
                                             uint16_t *__restrict__ dst)
{
    int32_t mn[8], mx[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        mn[e] = 0x7fffffff;
        mx[e] = -0x7fffffff - 1;
    }
    // 16 tokens at a time: all loads of a batch are independent and issue together.
    for (int t0 = 0; t0 < PS; t0 += 16) {
        if (t0 >= valid)
            break;
        u32x4_t v[16];
        v[0] = ld16_nt(src + (size_t)t0 * kHeadDim);
#pragma unroll
        for (int t = 1; t < 16; ++t)
            v[t] = (t0 + t < valid) ? ld16_nt(src + (size_t)(t0 + t) * kHeadDim) : v[0];
        // token t0 is valid; re-folding it for slots past the length changes nothing.
#pragma unroll
        for (int t = 0; t < 16; ++t)
            fold(v[t], mn, mx);
    }
    u32x4_t lo, hi;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        lo[w] = unorder16(mn[2 * w]) | (unorder16(mn[2 * w + 1]) << 16);
        hi[w] = unorder16(mx[2 * w]) | (unorder16(mx[2 * w + 1]) << 16);
    }
    st16(dst, lo);
    st16(dst + kHeadDim, hi);
}

// Key sums of one (page, head, 8-channel slice) over `valid` tokens, in token order.
template <int PS>
__device__ __forceinline__ void slice_sum(const uint16_t *__restrict__ src, int valid,
                                          float *__restrict__ dst)
{
    float acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e)
        acc[e] = 0.f;
    for (int t0 = 0; t0 < PS; t0 += 16) {
        if (t0 >= valid)
            break;
        const int nt = valid - t0 < 16 ? valid - t0 : 16;
        u32x4_t v[16];
#pragma unroll
        for (int t = 0; t < 16; ++t)
            v[t] = (t < nt) ? ld16_nt(src + (size_t)(t0 + t) * kHeadDim) : (u32x4_t){0u, 0u, 0u, 0u};
#pragma unroll
        for (int t = 0; t < 16; ++t) {
            if (t < nt) {
#pragma unroll
                for (int w = 0; w < 4; ++w) {
                    acc[2 * w] += bf16_lo(v[t][w]);
                    acc[2 * w + 1] += bf16_hi(v[t][w]);
                }
            }
        }
    }
    st16(dst, __builtin_bit_cast(u32x4_t, (f32x4_t){acc[0], acc[1], acc[2], acc[3]}));
    st16(dst + 4, __builtin_bit_cast(u32x4_t, (f32x4_t){acc[4], acc[5], acc[6], acc[7]}));
}

template <int PS, bool kMean>
__global__ __launch_bounds__(kMetaThreads) void k_meta_update(
    const uint16_t *__restrict__ k_cache, const int32_t *__restrict__ block_table,
    const int32_t *__restrict__ seq_lens, const int32_t *__restrict__ first_pos,
    void *__restrict__ meta, int num_kv_heads, int max_pages, int64_t num_phys, int rebuild)
{
    const int b = rebuild ? blockIdx.y : blockIdx.x;
    const int L = clamp_len(seq_lens[b], PS, max_pages);
    const int n = (L + PS - 1) / PS;
    int p_begin, p_end;
    if (rebuild) {
        p_begin = blockIdx.x;
        p_end = p_begin + 1 < n ? p_begin + 1 : n;
    } else {
        int f = first_pos[b];
        f = f < 0 ? 0 : f;
        if (f >= L)
            return;
        p_begin = f / PS;
        p_end = n;
    }
    const int slices = num_kv_heads * (kHeadDim / 8);
    for (int p = p_begin; p < p_end; ++p) {
        const int64_t phys = block_table[(int64_t)b * max_pages + p];
        if (phys < 0 || phys >= num_phys)
            continue;  // an entry outside the cache: an absent page, nothing to build
        const int valid = L - p * PS < PS ? L - p * PS : PS;
        for (int u = threadIdx.x; u < slices; u += kMetaThreads) {
            const int h = u >> 4;
            const int c = u & 15;
            const uint16_t *src = k_cache + ((phys * num_kv_heads + h) * PS) * kHeadDim + c * 8;
            if (kMean) {
                float *dst = static_cast<float *>(meta) + (phys * num_kv_heads + h) * kHeadDim + c * 8;
                slice_sum<PS>(src, valid, dst);
            } else {
                uint16_t *dst = static_cast<uint16_t *>(meta) +
                                ((phys * num_kv_heads + h) * 2) * kHeadDim + c * 8;
                slice_minmax<PS>(src, valid, dst);
            }
        }
    }
}

template <int PS>
hipError_t launch_ps(const sparrow_shape_t &s, const void *k_cache, const int32_t *bt,
                     const int32_t *lens, const int32_t *first_pos, void *meta, hipStream_t st)
{
    const int rebuild = first_pos == nullptr;
    const dim3 grid = rebuild ? dim3(s.max_pages_per_seq, s.batch) : dim3(s.batch);
    if (s.landmark == SPARROW_LANDMARK_MEAN)
        hipLaunchKernelGGL((k_meta_update<PS, true>), grid, dim3(kMetaThreads), 0, st,
                           static_cast<const uint16_t *>(k_cache), bt, lens, first_pos, meta,
                           s.num_kv_heads, s.max_pages_per_seq, s.num_phys_pages, rebuild);
    else
        hipLaunchKernelGGL((k_meta_update<PS, false>), grid, dim3(kMetaThreads), 0, st,
                           static_cast<const uint16_t *>(k_cache), bt, lens, first_pos, meta,
                           s.num_kv_heads, s.max_pages_per_seq, s.num_phys_pages, rebuild);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_meta_update(const sparrow_shape_t &s, const void *k_cache,
                              const int32_t *block_table, const int32_t *seq_lens,
                              const int32_t *first_pos, void *meta, hipStream_t stream)
{
    switch (s.page_size) {
    case 16: return launch_ps<16>(s, k_cache, block_table, seq_lens, first_pos, meta, stream);
    case 32: return launch_ps<32>(s, k_cache, block_table, seq_lens, first_pos, meta, stream);
    case 64: return launch_ps<64>(s, k_cache, block_table, seq_lens, first_pos, meta, stream);
    default: return launch_ps<128>(s, k_cache, block_table, seq_lens, first_pos, meta, stream);
    }
}

}  // namespace sparrow
