// Page scoring and block top-k selection (Sec. 3.3 and Sec. 3.2 of arXiv 2606.08446).
//
// k_page_score: the score of page p for KV head h is
//     S(p) = sum_{g<G} sum_i max(q_{g,i} mn_i, q_{g,i} mx_i).
// Because mn_i <= mx_i, max(q mn, q mx) = q+ mx + q- mn with q+ = max(q, 0) and
// q- = min(q, 0), so S(p) = sum_i (Q-_i mn_i + Q+_i mx_i) with Q+-_i = sum_g q+-_{g,i}:
// one 256-long dot product of the page's metadata row [mn | mx] with a weight vector that
// depends only on the query group.  This is a matrix-vector product (pages x 256 against
// one vector): HBM-bound with about one flop per byte, so it runs on VALU FMAs in fp32,
// with the loads laid out for fully coalesced 1 KiB reads (see the kernel).  Scores are
// written as fp32 to the workspace; sequences whose budget covers every page are skipped.
// A page whose block-table entry lies outside the cache is absent: score 0, nothing read.
//
// k_topk: one workgroup per (sequence, KV head) - 512 threads, or 256 from 1024 units on -
// selects the k largest scores with ties to the lower page index.  Scores become
// order-preserving uint32 keys in LDS; a radix select over 8-bit digits (from the highest
// bit where the keys differ, stopping as soon as the selection is decided) finds the
// threshold T and how many keys equal to T to keep; one block scan of (count > T,
// count == T) then places every kept page at its rank in ascending page order.  That
// select-and-rank core is block_topk (topk.h), shared with the attention kernel that selects
// and attends in one workgroup for small problems.
#include "common.h"
#include "topk.h"
#include "wave.h"

namespace sparrow {
namespace {

constexpr int kScoreThreads = 256;
constexpr int kScoreWaves = kScoreThreads / 64;
constexpr int kScorePages = 32;  // pages per workgroup
constexpr int kScorePagesSmall = 8;  // pages per workgroup when the grid would be small
constexpr int kScoreSmallGrid = 256;  // below this many 32-page workgroups: 8-page ones
constexpr int kScoreBatch = 8;   // pages per load batch of a wave
constexpr int kScoreHeads = 8;   // KV heads per workgroup (at most)
constexpr int kTopkManyUnits = 1024;  // from this many units on: 256-thread workgroups
constexpr int kTopkBatch = 8;   // score loads in flight per thread

// Sum of 8 per-lane values over the 32 lanes of a half-wave: afterwards lane i holds the
// total of value (i & 7).  Butterfly: each xor step halves the number of values a lane
// keeps.  Every value is summed by the same tree of commutative pairwise additions, so
// identical inputs give identical sums wherever they sit in the batch.
__device__ __forceinline__ float butterfly8(const float (&v)[8], int li)
{
    const bool b0 = li & 1, b1 = li & 2, b2 = li & 4;
    float v1[4], v2[2];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const float keep = b0 ? v[2 * j + 1] : v[2 * j];
        const float send = b0 ? v[2 * j] : v[2 * j + 1];
        v1[j] = keep + __shfl_xor(send, 1, 64);
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const float keep = b1 ? v1[2 * j + 1] : v1[2 * j];
        const float send = b1 ? v1[2 * j] : v1[2 * j + 1];
        v2[j] = keep + __shfl_xor(send, 2, 64);
    }
    const float keep = b2 ? v2[1] : v2[0];
    const float send = b2 ? v2[0] : v2[1];
    float r = keep + __shfl_xor(send, 4, 64);
    r += __shfl_xor(r, 8, 64);
    r += __shfl_xor(r, 16, 64);
    return r;
}

// One lane's share of a page's dot product: its 8 metadata elements against its 8 weights,
// in a fixed FMA order.
__device__ __forceinline__ float lane_dot(const float (&w)[8], u32x4_t v)
{
    float acc = 0.f;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        acc = fmaf(w[2 * t], bf16_lo(v[t]), acc);
        acc = fmaf(w[2 * t + 1], bf16_hi(v[t]), acc);
    }
    return acc;
}

// Mean landmark: 4 fp32 key sums against the lane's 4 weights, in a fixed FMA order.
__device__ __forceinline__ float lane_dot4(const float (&w)[8], u32x4_t v)
{
    float acc = 0.f;
#pragma unroll
    for (int t = 0; t < 4; ++t)
        acc = fmaf(w[t], __uint_as_float(v[t]), acc);
    return acc;
}

// Valid tokens of logical page p of a sequence of L tokens.
__device__ __forceinline__ int page_tokens(int p, int L, int ps)
{
    const int left = L - p * ps;
    return left < ps ? left : ps;
}

// One workgroup scores kPages (32, or 8 for small grids) consecutive logical pages of one
// sequence for up to kScoreHeads KV heads.  A wave owns a pair of KV heads: each load instruction reads the
// two heads' metadata rows of one page, 1 KiB contiguous (lanes 0-31 the first head,
// 32-63 the second; lane i takes elements 8i..8i+7 of the 256-long row [mn | mx]).  A lane
// multiplies its 8 bf16 elements by its 8 fp32 weights (Q- for the mn half, Q+ for the mx
// half, built from the group's queries) in a fixed FMA chain; butterfly8 then completes
// the dot products of a batch of 8 pages.  Batches are double-buffered in registers.
//
// With kAppend (sparrow_append_score_topk) the token being decoded is appended first: the
// wave that scores a sequence's last page writes the new key/value rows of its two heads
// and the page's updated metadata (lane slices of [mn | mx] are exactly the slices
// meta_with_key works on), and scores that page from the updated slice it holds.
template <bool kAppend, bool kMean, int kPages>
__global__ __launch_bounds__(kScoreThreads) void k_page_score(
    const uint16_t *__restrict__ q, const uint16_t *__restrict__ meta,
    const int32_t *__restrict__ block_table, const int32_t *__restrict__ seq_lens, Sched sched,
    int k_max, int num_q_heads, int num_kv_heads, int ps, int max_pages, int64_t num_phys,
    float *__restrict__ scores, AppendArgs app)
{
    __shared__ int32_t s_phys[kPages];
    __shared__ int32_t s_tab[2][kScoreThreads];  // the schedule's tables, when they fit

    const int b = blockIdx.y;
    const int h0 = blockIdx.z * kScoreHeads;
    const int nh = min(kScoreHeads, num_kv_heads - h0);
    const int page0 = blockIdx.x * kPages;
    const int G = num_q_heads / num_kv_heads;
    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63;
    const int half = lane >> 5;
    const int li = lane & 31;
    const int e0 = 8 * li;  // first element of this lane in the [mn | mx] row

    // Wave -> (head pair, page subset).
    const int npairs = (nh + 1) >> 1;
    const int wpp = kScoreWaves / npairs;  // waves sharing one head pair
    const int pair = wave % npairs;
    const int sub = wave / npairs;
    const int head = 2 * pair + half;      // within the workgroup's heads
    const bool active = sub < wpp;
    const bool lane_on = active && head < nh;

    // The length, this block's block-table entries and the schedule's tables are requested
    // together (the last two before the length is known); the queries go out right behind
    // the first batch of metadata, so a workgroup past the end of its sequence leaves after
    // one round trip.
    const int L_raw = seq_lens[b];
    int32_t pp = -1;
    if (tid < kPages && page0 + tid < max_pages)
        pp = block_table[(int64_t)b * max_pages + page0 + tid];
    const bool tab_lds = sched.n_bins <= kScoreThreads;
    int32_t t_min = 0, t_frac = 0;
    if (tab_lds && tid < sched.n_bins) {
        t_min = sched.min_pages[tid];
        t_frac = sched.frac_num[tid];
    }
    // (stored before the length arrives, so the compiler keeps these loads beside it; slots
    // past the sequence's last page are never read)
    if (tid < kPages)  // -1: an entry outside the cache, an absent page (score 0)
        s_phys[tid] = pp >= 0 && pp < num_phys ? pp : -1;
    if (tab_lds && tid < sched.n_bins) {
        s_tab[0][tid] = t_min;
        s_tab[1][tid] = t_frac;
    }
    const int L = clamp_len(L_raw, ps, max_pages);
    const int n = (L + ps - 1) / ps;
    if (page0 >= n)
        return;
    const int npg = min(kPages, n - page0);
    __syncthreads();
    const int i0 = e0 & (kHeadDim - 1);

    // Append of the token being decoded (position L - 1, on the last page n - 1).
    int last_slot = -1;  // slot of the appended page in this workgroup, for this lane
    u32x4_t upd = {0u, 0u, 0u, 0u};
    if (kAppend && L_raw >= 1 && L_raw <= ps * max_pages) {
        const int slot = n - 1 - page0;
        if (slot < npg && active && sub == slot % wpp && head < nh) {
            const int hh = h0 + head;
            const int tok = L - 1 - (n - 1) * ps;  // slot of the token within its page
            const int64_t phys = s_phys[slot];
            if (phys >= 0) {  // else the page is outside the cache: no append
                const int64_t nrow = ((int64_t)b * num_kv_heads + hh) * kHeadDim + i0;
                const u32x4_t kn = ld16(static_cast<const uint16_t *>(app.k_new) + nrow);
                const int64_t crow = ((phys * num_kv_heads + hh) * ps + tok) * kHeadDim + i0;
                if (e0 < kHeadDim)
                    st16(static_cast<uint16_t *>(app.k_cache) + crow, kn);
                else
                    st16(static_cast<uint16_t *>(app.v_cache) + crow,
                         ld16(static_cast<const uint16_t *>(app.v_new) + nrow));
                // The metadata row of this page is read and written only here.
                uint16_t *mrow = const_cast<uint16_t *>(meta) +
                                 (phys * num_kv_heads + hh) * 2 * kHeadDim + e0;
                if (kMean) {
                    const u32x2_t k4 = *reinterpret_cast<const u32x2_t *>(
                        static_cast<const uint16_t *>(app.k_new) + nrow - i0 + 4 * li);
                    upd = sums_with_key(tok == 0, tok == 0 ? upd : ld16(mrow), k4);
                } else {
                    upd = meta_with_key(tok == 0 ? kn : ld16(mrow), kn, e0 >= kHeadDim,
                                        tok == 0);
                }
                st16(mrow, upd);
                last_slot = slot;
            }
        }
    }

    // Only now is the budget needed to decide whether this sequence is scored at all.
    int budget;
    if (tab_lds) {
        const int bin = L > 0 ? budget_bin(L, sched) : 0;
        budget = L > 0 ? budget_from(L, ps, s_tab[0][bin], s_tab[1][bin], sched.frac_den, k_max)
                       : 0;
    } else {
        budget = budget_pages(L, ps, sched, k_max);
    }
    if (budget >= n || !active)
        return;  // every page is kept: nothing to score (or an idle wave)

    const int64_t page_elems = (int64_t)num_kv_heads * 2 * kHeadDim;
    const uint16_t *mbase = meta + (int64_t)(h0 + head) * 2 * kHeadDim + e0;
    float *out = scores + ((int64_t)b * num_kv_heads + h0 + head) * max_pages + page0;
    const int my_pages = (npg - sub + wpp - 1) / wpp;  // slots sub, sub + wpp, ...

    auto load_batch = [&](int j0, u32x4_t (&v)[kScoreBatch]) {
#pragma unroll
        for (int j = 0; j < kScoreBatch; ++j) {
            const int slot = sub + wpp * (j0 + j);
            v[j] = (u32x4_t){0u, 0u, 0u, 0u};
            if (j0 + j < my_pages && head < nh) {
                const int ph = __builtin_amdgcn_readfirstlane(s_phys[slot]);
                // (an absent page reads page 0; its score is replaced by 0 when stored)
                v[j] = ld16_nt(mbase + (int64_t)(ph < 0 ? 0 : ph) * page_elems);
            }
        }
    };

    u32x4_t nxt[kScoreBatch];
    load_batch(0, nxt);
    // Weights: 8 consecutive elements of Q- (mn half) or Q+ (mx half) of this lane's head;
    // with the mean landmark, channels 4 li .. 4 li + 3 of the group's summed queries (the
    // lane's 16 bytes of the row are 4 fp32 key sums).  Up to 8 query rows are requested
    // together, then added in head order.
    float w[8];
#pragma unroll
    for (int j = 0; j < 8; ++j)
        w[j] = 0.f;
    const uint16_t *qh = q + ((int64_t)b * num_q_heads + (int64_t)(h0 + head) * G) * kHeadDim +
                         (kMean ? 4 * li : i0);
    auto add_rows = [&](int g0) {
        u32x4_t v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            v[u] = (u32x4_t){0u, 0u, 0u, 0u};
            if (lane_on && g0 + u < G) {
                if (kMean) {
                    const u32x2_t x =
                        *reinterpret_cast<const u32x2_t *>(qh + (g0 + u) * kHeadDim);
                    v[u][0] = x[0];
                    v[u][1] = x[1];
                } else {
                    v[u] = ld16(qh + (g0 + u) * kHeadDim);
                }
            }
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            if (!(lane_on && g0 + u < G))
                continue;
            if (kMean) {
                w[0] += bf16_lo(v[u][0]);
                w[1] += bf16_hi(v[u][0]);
                w[2] += bf16_lo(v[u][1]);
                w[3] += bf16_hi(v[u][1]);
            } else {
                const bool neg = e0 < kHeadDim;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const float x0 = bf16_lo(v[u][j]), x1 = bf16_hi(v[u][j]);
                    w[2 * j] += neg ? fminf(x0, 0.f) : fmaxf(x0, 0.f);
                    w[2 * j + 1] += neg ? fminf(x1, 0.f) : fmaxf(x1, 0.f);
                }
            }
        }
    };
    add_rows(0);  // straight-line code: these loads go right behind the batch
    for (int g0 = 8; g0 < G; g0 += 8)
        add_rows(g0);
    for (int j0 = 0; j0 < my_pages; j0 += kScoreBatch) {
        u32x4_t cur[kScoreBatch];
#pragma unroll
        for (int j = 0; j < kScoreBatch; ++j)
            cur[j] = nxt[j];
        if (j0 + kScoreBatch < my_pages)
            load_batch(j0 + kScoreBatch, nxt);
        float part[kScoreBatch];
#pragma unroll
        for (int j = 0; j < kScoreBatch; ++j)
            part[j] = kMean ? lane_dot4(w, cur[j]) : lane_dot(w, cur[j]);
        const float total = butterfly8(part, li);
        const int j = j0 + (li & 7);
        const int slot = sub + wpp * j;
        // (the appended page was read here before its update landed: its score is
        // written below instead)
        if (li < kScoreBatch && j < my_pages && head < nh &&
            !(kAppend && slot == last_slot))
            out[slot] = s_phys[slot] < 0 ? 0.f
                        : kMean           ? total / (float)page_tokens(page0 + slot, L, ps)
                                          : total;
    }
    if (kAppend && last_slot >= 0) {
        // Score of the appended page from the updated slice: the same per-lane FMA chain,
        // and a 32-lane xor reduction (1, 2, 4, 8, 16) - the same tree of additions that
        // butterfly8 applies to every page, so the score is bit-identical to scoring the
        // updated metadata from memory.
        float total = kMean ? lane_dot4(w, upd) : lane_dot(w, upd);
#pragma unroll
        for (int x = 1; x < 32; x <<= 1)
            total += __shfl_xor(total, x, 64);
        if (li == 0)
            out[last_slot] =
                kMean ? total / (float)page_tokens(page0 + last_slot, L, ps) : total;
    }
}

template <int kTopkThreads>
__global__ __launch_bounds__(kTopkThreads) void k_topk(
    const float *__restrict__ scores, const int32_t *__restrict__ seq_lens, Sched sched,
    int k_max, int num_kv_heads, int ps, int max_pages, int32_t *__restrict__ out_k,
    int32_t *__restrict__ out_idx)
{
    extern __shared__ uint32_t keys[];  // [max_pages]
    __shared__ TopkLds t;

    const int unit = blockIdx.x;
    const int b = unit / num_kv_heads;
    const int h = unit - b * num_kv_heads;
    const int L = clamp_len(seq_lens[b], ps, max_pages);
    const int n = (L + ps - 1) / ps;
    const int tid = threadIdx.x;
    int32_t *row = out_idx + (int64_t)unit * k_max;

    // The first batch of scores is requested before the schedule lookup is resolved.
    const float *src = scores + (int64_t)unit * max_pages;
    float v[kTopkBatch];
#pragma unroll
    for (int j = 0; j < kTopkBatch; ++j) {
        const int i = tid + kTopkThreads * j;
        v[j] = i < n ? src[i] : 0.f;
    }
    const int k = budget_pages(L, ps, sched, k_max);
    if (h == 0 && tid == 0)
        out_k[b] = k;
    if (k >= n) {  // every page kept (also n == 0)
        for (int i = tid; i < k_max; i += kTopkThreads)
            row[i] = i < n ? i : -1;
        return;
    }

    // Keys into LDS; this thread's min and max of them.
    uint32_t kmin = 0xffffffffu, kmax = 0u;
    for (int base = 0; base < n; base += kTopkThreads * kTopkBatch) {
        if (base > 0) {
#pragma unroll
            for (int j = 0; j < kTopkBatch; ++j) {
                const int i = base + tid + kTopkThreads * j;
                v[j] = i < n ? src[i] : 0.f;
            }
        }
#pragma unroll
        for (int j = 0; j < kTopkBatch; ++j) {
            const int i = base + tid + kTopkThreads * j;
            if (i < n) {
                // forced pages (sinks, most recent pages) outrank every score
                const bool forced = i < sched.sink_pages || i >= n - sched.local_pages;
                const uint32_t key = forced ? 0xffffffffu : score_key(v[j]);
                keys[i] = key;
                kmin = min(kmin, key);
                kmax = max(kmax, key);
            }
        }
    }
    block_topk<kTopkThreads>(keys, n, k, kmin, kmax, t,
                             [&](uint32_t pos, int i) { row[pos] = i; });
    for (int i = k + tid; i < k_max; i += kTopkThreads)
        row[i] = -1;
}

}  // namespace

size_t score_topk_workspace(const sparrow_shape_t &s)
{
    return (size_t)s.batch * s.num_kv_heads * s.max_pages_per_seq * sizeof(float);
}

hipError_t launch_page_score(const sparrow_shape_t &s, const void *q, void *meta,
                             const int32_t *block_table, const int32_t *seq_lens,
                             const Sched &sched, int32_t k_max, float *scores,
                             const AppendArgs &app, hipStream_t stream)
{
    const int zs = (s.num_kv_heads + kScoreHeads - 1) / kScoreHeads;
    // A grid of fewer 32-page workgroups than compute units (a small batch: the step is
    // latency-bound) takes 8-page workgroups instead, so that a wave scores one batch and
    // the kernel lasts two round trips, not five (one 4096-token sequence, 8 KV heads:
    // 15.7 -> 12.9 us for the selection, bit-identical scores).
    const bool small = (int64_t)((s.max_pages_per_seq + kScorePages - 1) / kScorePages) *
                           s.batch * zs < kScoreSmallGrid;
    const int pages = small ? kScorePagesSmall : kScorePages;
    const dim3 sgrid((s.max_pages_per_seq + pages - 1) / pages, s.batch, zs);
    const bool mean = s.landmark == SPARROW_LANDMARK_MEAN;
    const bool append = app.k_new != nullptr;
    constexpr int P8 = kScorePagesSmall, P32 = kScorePages;
    auto kernel =
        small ? (append ? (mean ? k_page_score<true, true, P8> : k_page_score<true, false, P8>)
                        : (mean ? k_page_score<false, true, P8> : k_page_score<false, false, P8>))
              : (append ? (mean ? k_page_score<true, true, P32> : k_page_score<true, false, P32>)
                        : (mean ? k_page_score<false, true, P32>
                                : k_page_score<false, false, P32>));
    hipLaunchKernelGGL(kernel, sgrid, dim3(kScoreThreads), 0, stream,
                       static_cast<const uint16_t *>(q), static_cast<const uint16_t *>(meta),
                       block_table, seq_lens, sched, k_max, s.num_q_heads, s.num_kv_heads,
                       s.page_size, s.max_pages_per_seq, s.num_phys_pages, scores, app);
    return hipGetLastError();
}

hipError_t launch_topk(const sparrow_shape_t &s, const int32_t *seq_lens, const Sched &sched,
                       int32_t k_max, const float *scores, int32_t *out_k, int32_t *out_idx,
                       hipStream_t stream)
{
    const int units = s.batch * s.num_kv_heads;
    // Many units: smaller workgroups, so more of them share a CU (the per-unit work is
    // latency-bound); few units: larger ones, so each finishes sooner.
    const bool many = units >= kTopkManyUnits;
    hipLaunchKernelGGL(many ? k_topk<256> : k_topk<512>, dim3(units), dim3(many ? 256 : 512),
                       (size_t)s.max_pages_per_seq * sizeof(uint32_t), stream, scores, seq_lens,
                       sched, k_max, s.num_kv_heads, s.page_size, s.max_pages_per_seq, out_k,
                       out_idx);
    return hipGetLastError();
}

hipError_t launch_score_topk(const sparrow_shape_t &s, const void *q, void *meta,
                             const int32_t *block_table, const int32_t *seq_lens,
                             const Sched &sched, int32_t k_max, int32_t *out_k,
                             int32_t *out_idx, void *workspace, const AppendArgs &app,
                             hipStream_t stream)
{
    float *scores = static_cast<float *>(workspace);
    const hipError_t e = launch_page_score(s, q, meta, block_table, seq_lens, sched, k_max,
                                           scores, app, stream);
    if (e != hipSuccess)
        return e;
    return launch_topk(s, seq_lens, sched, k_max, scores, out_k, out_idx, stream);
}

}  // namespace sparrow
