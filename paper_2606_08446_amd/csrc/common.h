// Internal helpers shared by the gfx950 kernels of libsparrow (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "sparrow.h"

namespace sparrow {

constexpr int kHeadDim = 128;
constexpr int kMaxBatch = SPARROW_MAX_BATCH;  // sequences per call (page offsets live in LDS)

// MFMA operand / accumulator types (wave64, 16x16 tiles).
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));  // 16x16x32 bf16 operand
typedef short s16x4_t __attribute__((ext_vector_type(4)));     // 16x16x16 bf16 operand
typedef float f32x4_t __attribute__((ext_vector_type(4)));     // 16x16 fp32 accumulator
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Budget schedule as the kernels see it (tables are device pointers).
struct Sched {
    int32_t bin_tokens;
    int32_t n_bins;
    int32_t frac_den;
    const int32_t *min_pages;
    const int32_t *frac_num;
    int32_t sink_pages;   // logical pages [0, sink) always kept
    int32_t local_pages;  // logical pages [n - local, n) always kept
};

__device__ __forceinline__ u32x4_t ld16(const void *p)
{
    return *reinterpret_cast<const u32x4_t *>(p);
}

// Streaming load (non-temporal hint) for data that is read exactly once.
__device__ __forceinline__ u32x4_t ld16_nt(const void *p)
{
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(p));
}

__device__ __forceinline__ void st16(void *p, u32x4_t v)
{
    *reinterpret_cast<u32x4_t *>(p) = v;
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Two fp32 values -> packed bf16 pair (round to nearest even), lo in bits 0..15.
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi)
{
    bf16x2_t v = __builtin_convertvector((float __attribute__((ext_vector_type(2)))){lo, hi},
                                         bf16x2_t);
    return __builtin_bit_cast(uint32_t, v);
}

// One fp32 value -> bf16 bits (round to nearest even).
__device__ __forceinline__ uint32_t to_bf16_bits(float x) { return pack_bf16(x, 0.f) & 0xffffu; }

// bf16 bit pattern -> signed integer with the same order as the values (-0 < +0).
__device__ __forceinline__ int32_t order16(uint32_t bits)
{
    const int32_t s = (int32_t)(int16_t)(uint16_t)bits;
    return s ^ ((s >> 15) & 0x7fff);
}

// Inverse of order16 (the map is an involution on 16-bit patterns).
__device__ __forceinline__ uint32_t unorder16(int32_t key)
{
    return (uint32_t)(key ^ ((key >> 15) & 0x7fff)) & 0xffffu;
}

// Metadata of a page after one more key: 8 bf16 elements of the [mn | mx] row.  `old` is
// the current slice (min row if !is_max, else max row), `key` the new key's 8 channels;
// a fresh page (its first token) takes the key itself.  Exact: the result is an input
// pattern under the total order -0 < +0.
__device__ __forceinline__ u32x4_t meta_with_key(u32x4_t old, u32x4_t key, bool is_max,
                                                 bool fresh)
{
    if (fresh)
        return key;
    u32x4_t r;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        uint32_t out = 0;
#pragma unroll
        for (int hw = 0; hw < 2; ++hw) {
            const int32_t a = order16(old[w] >> (16 * hw));
            const int32_t k = order16(key[w] >> (16 * hw));
            const int32_t m = is_max ? max(a, k) : min(a, k);
            out |= unorder16(m) << (16 * hw);
        }
        r[w] = out;
    }
    return r;
}

// Mean landmark: fp32 key sums of 4 channels after one more key (4 bf16 in `k4`); a fresh
// page (its first token) takes the key itself (the rebuild's 0 + k).
__device__ __forceinline__ u32x4_t sums_with_key(bool fresh, u32x4_t old, u32x2_t k4)
{
    const float k[4] = {bf16_lo(k4[0]), bf16_hi(k4[0]), bf16_lo(k4[1]), bf16_hi(k4[1])};
    u32x4_t r;
#pragma unroll
    for (int e = 0; e < 4; ++e)
        r[e] = __float_as_uint(fresh ? 0.f + k[e] : __uint_as_float(old[e]) + k[e]);
    return r;
}

// Sequence length clamped to what the block table can address.
__device__ __forceinline__ int clamp_len(int L, int ps, int max_pages)
{
    const int cap = ps * max_pages;
    return L < 0 ? 0 : (L > cap ? cap : L);
}

// Schedule bin of a sequence of L >= 1 tokens (the position of its last token).  Shared by
// the kernels and the host-side bound (sparrow_budget_bound), so both use one definition.
__host__ __device__ __forceinline__ int budget_bin(int L, int bin_tokens, int n_bins)
{
    const int bin = (L - 1) / bin_tokens;
    return bin > n_bins - 1 ? n_bins - 1 : bin;
}

__device__ __forceinline__ int budget_bin(int L, const Sched &s)
{
    return budget_bin(L, s.bin_tokens, s.n_bins);
}

// Page budget of a sequence of L >= 1 tokens from its bin's table entries, capped at k_max:
// clamp(max(min_pages, ceil(n * frac_num / frac_den)), 1, n) with n = ceil(L / ps).
__host__ __device__ __forceinline__ int budget_from(int L, int ps, int32_t min_pages,
                                                    int32_t frac_num, int32_t frac_den,
                                                    int k_max)
{
    const int64_t n = ((int64_t)L + ps - 1) / ps;
    int64_t k = (n * (int64_t)frac_num + frac_den - 1) / frac_den;
    if (k < min_pages)
        k = min_pages;
    if (k < 1)
        k = 1;
    if (k > n)
        k = n;
    if (k > k_max)
        k = k_max;
    return (int)k;
}

// Page budget of a sequence of L tokens from the schedule, capped at k_max.
__device__ __forceinline__ int budget_pages(int L, int ps, const Sched &s, int k_max)
{
    if (L <= 0)
        return 0;
    const int bin = budget_bin(L, s);
    return budget_from(L, ps, s.min_pages[bin], s.frac_num[bin], s.frac_den, k_max);
}

// ---------------------------------------------------------------------------------------------
// Launchers (host side, one per kernel family).  All return hipSuccess or the launch error.
// ---------------------------------------------------------------------------------------------
hipError_t launch_meta_update(const sparrow_shape_t &s, const void *k_cache,
                              const int32_t *block_table, const int32_t *seq_lens,
                              const int32_t *first_pos, void *meta, hipStream_t stream);

hipError_t launch_append_kv(const sparrow_shape_t &s, const void *k_new, const void *v_new,
                            void *k_cache, void *v_cache, const int32_t *block_table,
                            const int32_t *seq_lens, void *meta, hipStream_t stream);

// Token append folded into scoring (k_new == nullptr: no append).
struct AppendArgs {
    const void *k_new;
    const void *v_new;
    void *k_cache;
    void *v_cache;
};

size_t score_topk_workspace(const sparrow_shape_t &s);
// Scores of every page into `scores` [batch][num_kv_heads][max_pages] (with the append when
// app.k_new != nullptr); sequences whose budget keeps every page are skipped.
hipError_t launch_page_score(const sparrow_shape_t &s, const void *q, void *meta,
                             const int32_t *block_table, const int32_t *seq_lens,
                             const Sched &sched, int32_t k_max, float *scores,
                             const AppendArgs &app, hipStream_t stream);
// Budgets and top-k page lists from the scores.
hipError_t launch_topk(const sparrow_shape_t &s, const int32_t *seq_lens, const Sched &sched,
                       int32_t k_max, const float *scores, int32_t *out_k, int32_t *out_idx,
                       hipStream_t stream);
// Both of the above.
hipError_t launch_score_topk(const sparrow_shape_t &s, const void *q, void *meta,
                             const int32_t *block_table, const int32_t *seq_lens,
                             const Sched &sched, int32_t k_max, int32_t *out_k,
                             int32_t *out_idx, void *workspace, const AppendArgs &app,
                             hipStream_t stream);

hipError_t launch_acceptance(int64_t T, int V, int dtype, const void *target, const void *draft,
                             float tau, float *alpha, hipStream_t stream);
hipError_t launch_acceptance_topk(int64_t T, int K, const float *lp_target, const float *lp_draft,
                                  float *alpha, hipStream_t stream);
hipError_t launch_tail_stats(int64_t T, const float *alpha, const int32_t *pos, int bin_tokens,
                             int n_bins, double pct, double *quantile, double *mean,
                             int64_t *count, hipStream_t stream);

hipError_t launch_stream_read(const void *src, int64_t bytes, uint32_t *checksum,
                              hipStream_t stream);

struct AttnPlan {
    size_t plan_bytes;       // page offsets and unit wave ranges at the start of the workspace
    size_t segments;         // partial-result slots (waves + units)
    size_t workspace_bytes;
    size_t lds_bytes;        // dynamic LDS of the streaming kernel
};

AttnPlan plan_attention(const sparrow_shape_t &s);

// The library's own attention workspace on the current device (kScratchBytes), or nullptr
// when its address cannot be obtained.
constexpr size_t kScratchBytes = (size_t)SPARROW_NOALLOC_SCRATCH_BYTES;
void *attention_scratch();
hipError_t launch_attention(const sparrow_shape_t &s, const AttnPlan &plan, const void *q,
                            const void *k_cache, const void *v_cache, const int32_t *block_table,
                            const int32_t *seq_lens, const int32_t *k, const int32_t *idx,
                            int32_t k_max, float scale, void *out, int out_dtype,
                            void *workspace, hipStream_t stream);
// Whether attention with this list bound (k_max, or max_pages_per_seq for dense) runs one
// workgroup per (sequence, KV head) unit.
bool attention_unit_path(const sparrow_shape_t &s, int64_t list_bound);
// Budgets, top-k and sparse attention of a problem on the unit path, from the scoring
// kernel's scores, in one launch (writes out_k, out_idx and out).
hipError_t launch_select_attention(const sparrow_shape_t &s, const void *q, const void *k_cache,
                                   const void *v_cache, const int32_t *block_table,
                                   const int32_t *seq_lens, const Sched &sched, int32_t k_max,
                                   const float *scores, int32_t *out_k, int32_t *out_idx,
                                   float scale, void *out, int out_dtype, hipStream_t stream);

}  // namespace sparrow
