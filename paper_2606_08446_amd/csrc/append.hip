// Appending the token being decoded to the paged KV cache, with the O(1) metadata update
// of its page (the per-token landmark upkeep of Sec. 3.3 of arXiv 2606.08446).
//
// The new token sits at position L - 1 (L counts it): page (L - 1) / ps, slot (L - 1) % ps.
// A half-wave owns one KV head: lane i handles elements 8i .. 8i+7 of the page's metadata
// row [mn | mx], i.e. channels 8i mod 128 of the new key.  Lanes 0-15 also write the key
// row (256 B) and lanes 16-31 the value row.  The page's metadata becomes
// min/max(old, key) - or the key itself on the page's first slot - which equals the
// rebuild from all of the page's tokens whenever the old metadata described them.
// With the mean landmark lane i owns the fp32 sums of channels 4i .. 4i+3 and adds the
// key's channels to them (the key itself on the page's first slot) - the same fp32 adds,
// in the same token order, as the rebuild.
#include "common.h"

namespace sparrow {
namespace {

constexpr int kAppendThreads = 256;
constexpr int kAppendHeads = kAppendThreads / 32;  // KV heads per workgroup

template <bool kMean>
__global__ __launch_bounds__(kAppendThreads) void k_append_kv(
    const uint16_t *__restrict__ k_new, const uint16_t *__restrict__ v_new,
    uint16_t *__restrict__ k_cache, uint16_t *__restrict__ v_cache,
    const int32_t *__restrict__ block_table, const int32_t *__restrict__ seq_lens,
    void *__restrict__ meta, int num_kv_heads, int ps, int max_pages, int64_t num_phys)
{
    const int b = blockIdx.x;
    const int h = blockIdx.y * kAppendHeads + (threadIdx.x >> 5);
    if (h >= num_kv_heads)
        return;
    const int L = seq_lens[b];
    if (L < 1 || L > ps * max_pages)
        return;  // nothing to append, or a position the block table cannot address
    const int pos = L - 1;
    const int lp = pos / ps;
    const int tok = pos - lp * ps;
    const int e0 = 8 * (threadIdx.x & 31);  // element of [mn | mx]
    const int i0 = e0 & (kHeadDim - 1);     // channel
    const int64_t phys = block_table[(int64_t)b * max_pages + lp];
    if (phys < 0 || phys >= num_phys)
        return;  // the page is outside the cache: nothing is written
    const int64_t nrow = ((int64_t)b * num_kv_heads + h) * kHeadDim + i0;
    const u32x4_t kn = ld16(k_new + nrow);
    const int64_t crow = ((phys * num_kv_heads + h) * ps + tok) * kHeadDim + i0;
    if (e0 < kHeadDim)
        st16(k_cache + crow, kn);
    else
        st16(v_cache + crow, ld16(v_new + nrow));
    if (kMean) {
        const int c0 = 4 * (threadIdx.x & 31);
        float *srow = static_cast<float *>(meta) + (phys * num_kv_heads + h) * kHeadDim + c0;
        const u32x2_t k4 = *reinterpret_cast<const u32x2_t *>(k_new + nrow - i0 + c0);
        st16(srow, sums_with_key(tok == 0, ld16(srow), k4));
    } else {
        uint16_t *mrow = static_cast<uint16_t *>(meta) + (phys * num_kv_heads + h) * 2 * kHeadDim + e0;
        st16(mrow, meta_with_key(tok == 0 ? kn : ld16(mrow), kn, e0 >= kHeadDim, tok == 0));
    }
}

}  // namespace

hipError_t launch_append_kv(const sparrow_shape_t &s, const void *k_new, const void *v_new,
                            void *k_cache, void *v_cache, const int32_t *block_table,
                            const int32_t *seq_lens, void *meta, hipStream_t stream)
{
    const dim3 grid(s.batch, (s.num_kv_heads + kAppendHeads - 1) / kAppendHeads);
    if (s.landmark == SPARROW_LANDMARK_MEAN)
        hipLaunchKernelGGL(k_append_kv<true>, grid, dim3(kAppendThreads), 0, stream,
                           static_cast<const uint16_t *>(k_new),
                           static_cast<const uint16_t *>(v_new), static_cast<uint16_t *>(k_cache),
                           static_cast<uint16_t *>(v_cache), block_table, seq_lens, meta,
                           s.num_kv_heads, s.page_size, s.max_pages_per_seq, s.num_phys_pages);
    else
        hipLaunchKernelGGL(k_append_kv<false>, grid, dim3(kAppendThreads), 0, stream,
                           static_cast<const uint16_t *>(k_new),
                           static_cast<const uint16_t *>(v_new), static_cast<uint16_t *>(k_cache),
                           static_cast<uint16_t *>(v_cache), block_table, seq_lens, meta,
                           s.num_kv_heads, s.page_size, s.max_pages_per_seq, s.num_phys_pages);
    return hipGetLastError();
}

}  // namespace sparrow
