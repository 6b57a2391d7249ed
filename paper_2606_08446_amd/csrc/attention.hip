// GQA decode attention over a paged KV cache, sparse (selected pages) or dense (all pages):
// the attention term of the cost models of Sec. 3.3 (Eq. dense-cost, Eq. sparse-cost) of
// arXiv 2606.08446, with the block-sparse token set of Sec. 2.
//
// Work split (streaming waves).  All (sequence, KV head, listed page) positions are laid
// end to end - sequence by sequence, head by head, in list order - and every resident
// wave takes one equal, contiguous range of them (fewer waves for a small problem: at
// most one per position and kUnitSegments per unit on average).  A wave streams its
// range chunk by chunk with the next 16-token chunk's K/V loads always in flight, and the
// page list is prefetched in batches of 64 pages one batch ahead, across (sequence, head)
// boundaries.
// Its online-softmax state is flushed whenever its range leaves a (sequence, KV head):
// a unit whose pages all fall in one wave is normalised and written to `out` directly;
// otherwise the wave writes a partial (m, l, o) to segment slot `wave + unit` (unique
// along the partition) and k_attn_merge combines the partials of that unit.
// Small problems (a few units with short lists) take k_attn_unit instead: one workgroup per
// unit, its waves' states merged in LDS, one launch.
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
#include <atomic>

#include "common.h"
#include "topk.h"
#include "wave.h"

namespace sparrow {
namespace {

constexpr int kAttnThreads = 256;
constexpr int kAttnWaves = kAttnThreads / 64;
constexpr int kBatch = 64;        // pages per prefetched page-list batch
constexpr int kMaxWaves = 4096;   // upper bound of streaming waves (sizes the workspace)
constexpr int kUnitSegments = 64;  // streaming waves per (sequence, KV head) unit, on average

struct AttnArgs {
    const uint16_t *q;
    const uint16_t *k_cache;
    const uint16_t *v_cache;
    const int32_t *block_table;
    const int32_t *seq_lens;
    const int32_t *ksel;
    const int32_t *idx;
    int32_t *plan_off;    // [batch + 1] page offsets of the sequences (written by workgroup 0)
    int32_t *unit_waves;  // [batch * num_kv_heads][2] first and last wave of each unit
    float *o_part;
    float *ml_part;
    void *out;
    int k_max, batch, num_q_heads, num_kv_heads, ps, max_pages, out_bf16, total_waves;
    int64_t num_phys;  // physical pages in the caches
    float scale_log2;
};

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

__device__ __forceinline__ void store_out(void *out, int out_bf16, int64_t i, float v)
{
    if (out_bf16)
        static_cast<uint16_t *>(out)[i] = (uint16_t)to_bf16_bits(v);
    else
        static_cast<float *>(out)[i] = v;
}

// Pages in the attention list of sequence b.
template <bool kSparse>
__device__ __forceinline__ int list_pages(const AttnArgs &a, int b)
{
    const int L = clamp_len(a.seq_lens[b], a.ps, a.max_pages);
    const int n = (L + a.ps - 1) / a.ps;
    if (!kSparse)
        return n;
    const int c = a.ksel[b];
    return c < 0 ? 0 : (c > a.k_max ? a.k_max : c);
}

// Block-wide exclusive prefix of list_pages over the batch into s_off[0 .. batch].
template <bool kSparse>
__device__ void seq_prefix(const AttnArgs &a, int32_t *s_off, int32_t *s_tmp)
{
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int B = a.batch;
    const int per = (B + kAttnThreads - 1) / kAttnThreads;
    const int b0 = min(B, tid * per);
    const int b1 = min(B, b0 + per);
    int local = 0;
    for (int b = b0; b < b1; ++b)
        local += list_pages<kSparse>(a, b);
    const int incl = (int)wave_scan_add((uint32_t)local);  // totals < 2^31 (max batch x pages)
    if (lane == 63)
        s_tmp[wave] = incl;
    __syncthreads();
    int run = incl - local;
    for (int w = 0; w < wave; ++w)
        run += s_tmp[w];
    for (int b = b0; b < b1; ++b) {
        s_off[b] = run;
        run += list_pages<kSparse>(a, b);
    }
    if (tid == kAttnThreads - 1)
        s_off[B] = run;  // this thread's range ends at B (or is empty): run is the total
    __syncthreads();
}

// Position cursor over the (sequence, head, page) list.
struct Cursor {
    int b, h, j, cnt;  // sequence, KV head, page position within the unit, unit length
    int64_t pos;       // global position
};

// One page-list batch of at most kBatch pages of one unit; lane i describes page j0 + i.
struct Batch {
    int b, h, j0, n, L;
    bool ends_unit;
    int lp;    // logical page (-1: none)
    int phys;  // physical page, as the block table gives it (checked when used)
    int tok0;  // first token of the page
};

// A page-list batch is fetched in two phases so that no wait on its loads drains the K/V
// loads in flight (a wave's loads complete in order): fetch_batch_begin issues the index
// loads and advances the cursor; fetch_batch_end, called one chunk later, when the
// indices have arrived, issues the block-table loads, which are consumed a batch later.
template <bool kSparse>
__device__ __forceinline__ void fetch_batch_begin(const AttnArgs &a, const int32_t *s_off,
                                                  Cursor &c, int64_t pos_end, Batch &t, int lane)
{
    const int Hkv = a.num_kv_heads;
    t.b = c.b;
    t.h = c.h;
    t.j0 = c.j;
    const int64_t left = pos_end - c.pos;
    int n = c.cnt - c.j;
    if (n > kBatch)
        n = kBatch;
    if (n > left)
        n = (int)left;
    t.n = n;
    t.ends_unit = c.j + n == c.cnt;
    t.L = clamp_len(a.seq_lens[c.b], a.ps, a.max_pages);
    t.lp = -1;
    if (lane < n)
        t.lp = kSparse ? a.idx[((int64_t)c.b * Hkv + c.h) * a.k_max + c.j + lane] : c.j + lane;
    c.pos += n;
    c.j += n;
    if (c.j == c.cnt && c.pos < pos_end) {  // next unit with pages
        c.j = 0;
        if (++c.h == Hkv) {
            c.h = 0;
            do {
                ++c.b;
            } while (s_off[c.b + 1] == s_off[c.b]);
        }
        c.cnt = s_off[c.b + 1] - s_off[c.b];
    }
}

__device__ __forceinline__ void fetch_batch_end(const AttnArgs &a, Batch &t)
{
    const int np = (t.L + a.ps - 1) / a.ps;
    t.phys = -1;
    t.tok0 = 0;
    if (t.lp >= 0 && t.lp < np) {  // entries outside the sequence: no page
        t.phys = a.block_table[(int64_t)t.b * a.max_pages + t.lp];
        t.tok0 = t.lp * a.ps;
    }
}

// One live 16-token chunk into a wave's online-softmax state: logits on MFMA, the running
// maximum and sum in the log2 domain, O^T += V^T P.  `valid` (>= 1) tokens of the chunk
// lie inside the sequence; the rest get weight 0 and their V rows are zeroed.
__device__ __forceinline__ void attend_chunk(Chunk &ch, int valid, const bf16x8_t (&qf)[4],
                                             float scale_log2, int lg, float &m_run,
                                             float &l_run, f32x4_t (&O)[8])
{
    // ---- logits of 16 tokens x 16 (padded) heads
    f32x4_t s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < 4; ++i)
        s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, ch.k[i]), qf[i],
                                                    s, 0, 0, 0);
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
                ch.v[j] = (u32x4_t){0u, 0u, 0u, 0u};
    }
    // ---- O^T += V^T P
    const s16x4_t pb = __builtin_bit_cast(s16x4_t, (u32x2_t){p01, p23});
#pragma unroll
    for (int c = 0; c < 8; ++c) {
        const u32x2_t av = {pair_of(ch.v[0], ch.v[1], c), pair_of(ch.v[2], ch.v[3], c)};
        O[c] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4_t, av), pb,
                                                         O[c], 0, 0, 0);
    }
}

__device__ __forceinline__ void load_q(const AttnArgs &a, int b, int h, int lr, int lg,
                                       bf16x8_t (&qf)[4])
{
    const int G = a.num_q_heads / a.num_kv_heads;
    const uint16_t *qrow = a.q + ((int64_t)b * a.num_q_heads + (int64_t)h * G + lr) * kHeadDim;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        u32x4_t v = {0u, 0u, 0u, 0u};
        if (lr < G)
            v = ld16(qrow + 32 * i + 8 * lg);
        qf[i] = __builtin_bit_cast(bf16x8_t, v);
    }
}

template <bool kSparse>
__global__ __launch_bounds__(kAttnThreads) void k_attn_stream(AttnArgs a)
{
    extern __shared__ int32_t s_off[];  // [batch + 1]
    __shared__ int32_t s_tmp[kAttnWaves];

    seq_prefix<kSparse>(a, s_off, s_tmp);
    const int B = a.batch;
    const int Hkv = a.num_kv_heads;
    const int G = a.num_q_heads / Hkv;
    if (blockIdx.x == 0)
        for (int b = threadIdx.x; b <= B; b += kAttnThreads)
            a.plan_off[b] = s_off[b];

    const int64_t P = (int64_t)s_off[B] * Hkv;
    // One wave per listed page at most, and at most kUnitSegments waves per unit on average:
    // a unit split over hundreds of one-page waves leaves the merge a long serial chain of
    // partials (one 4096-token sequence, dense: 33 -> 21 us per step with the cap).
    int64_t W = P < a.total_waves ? P : a.total_waves;
    if (W > (int64_t)B * Hkv * kUnitSegments)
        W = (int64_t)B * Hkv * kUnitSegments;
    const int w = blockIdx.x * kAttnWaves + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (w >= W)
        return;
    const int64_t pos_begin = (int64_t)w * P / W;
    const int64_t pos_end = (int64_t)(w + 1) * P / W;
    const int lane = threadIdx.x & 63;
    const int lr = lane & 15;
    const int lg = lane >> 4;
    const int ps = a.ps;
    const int cpp = ps >> 4;  // 16-token chunks per page
    const int64_t head_elems = (int64_t)ps * kHeadDim;

    // Locate the first position: the last sequence whose offset is <= pos_begin is the one
    // holding it (empty sequences before it share its offset).  The offsets do not decrease,
    // so a wave narrows [lo, lo + span) 64-fold per round: lane l tests entry lo + l step,
    // and the number of lanes that pass gives the last entry <= pos_begin (s_off[lo] always
    // is).
    Cursor cur;
    {
        int lo = 0, span = B;
        while (span > 1) {
            const int step = (span + 63) >> 6;
            const bool ok = lane * step < span && (int64_t)s_off[lo + lane * step] * Hkv <= pos_begin;
            const int t = __popcll(__ballot(ok)) - 1;
            lo += t * step;
            span = min(step, span - t * step);
        }
        cur.b = lo;
        cur.cnt = s_off[lo + 1] - s_off[lo];
        const int64_t rel = pos_begin - (int64_t)s_off[lo] * Hkv;
        cur.h = (int)(rel / cur.cnt);
        cur.j = (int)(rel - (int64_t)cur.h * cur.cnt);
        cur.pos = pos_begin;
    }

    Batch bc, bn;
    fetch_batch_begin<kSparse>(a, s_off, cur, pos_end, bc, lane);
    fetch_batch_end(a, bc);
    bool have_next = cur.pos < pos_end;
    bool bn_pending = have_next;  // bn's block-table loads not issued yet
    if (have_next)
        fetch_batch_begin<kSparse>(a, s_off, cur, pos_end, bn, lane);

    bf16x8_t qf[4], qn[4];
    load_q(a, bc.b, bc.h, lr, lg, qf);
    bool from_start = bc.j0 == 0;

    float m_run = -INFINITY;
    float l_run = 0.f;
    f32x4_t O[8];
#pragma unroll
    for (int c = 0; c < 8; ++c)
        O[c] = (f32x4_t){0.f, 0.f, 0.f, 0.f};

    // chunk `ci` of batch t: page ci / cpp, sub-chunk ci % cpp
    auto issue = [&](const Batch &t, int ci, Chunk &ch, int &tok) -> bool {
        const int pi = ci / cpp;
        const int sub = ci - pi * cpp;
        const int ph = __builtin_amdgcn_readlane(t.phys, pi);
        tok = __builtin_amdgcn_readlane(t.tok0, pi) + 16 * sub;
        // a block-table entry outside the cache is an absent page
        const bool live = ph >= 0 && ph < a.num_phys && tok < t.L;
        if (live) {
            const int64_t off =
                ((int64_t)ph * Hkv + t.h) * head_elems + (int64_t)(16 * sub) * kHeadDim;
            load_chunk(ch, a.k_cache + off, a.v_cache + off, lr, lg);
        }
        return live;
    };

    // A unit's finished state: written as the output when the unit lies in this wave alone,
    // else as a partial (segment `wave + unit`) for the merge.
    auto write_unit = [&](const f32x4_t (&Os)[8], float m, float l, int b, int h,
                          bool first, bool last) {
        const int unit = b * Hkv + h;
        if (lane == 0) {
            if (first)
                a.unit_waves[2 * unit] = w;
            if (last)
                a.unit_waves[2 * unit + 1] = w;
        }
        if (lr >= G)
            return;
        if (first && last) {
            const float inv = l > 0.f ? 1.f / l : 0.f;
            const int64_t orow = ((int64_t)b * a.num_q_heads + (int64_t)h * G + lr) * kHeadDim;
#pragma unroll
            for (int c = 0; c < 8; ++c)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    store_out(a.out, a.out_bf16, orow + 32 * lg + 8 * i + c, Os[c][i] * inv);
        } else {
            const int64_t seg = (int64_t)w + unit;
            float *op = a.o_part + (seg * G + lr) * kHeadDim + 32 * lg;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                st16(op + 8 * i, __builtin_bit_cast(
                                     u32x4_t, (f32x4_t){Os[0][i], Os[1][i], Os[2][i], Os[3][i]}));
                st16(op + 8 * i + 4, __builtin_bit_cast(u32x4_t, (f32x4_t){Os[4][i], Os[5][i],
                                                                          Os[6][i], Os[7][i]}));
            }
            if (lg == 0) {
                a.ml_part[(seg * G + lr) * 2 + 0] = m;
                a.ml_part[(seg * G + lr) * 2 + 1] = l;
            }
        }
    };
    // Up to two finished units are held in registers until the range ends: on this GPU a
    // store counts in the wave's in-order memory counter, so a store issued mid-range would
    // make the next waits on K/V loads wait for its acknowledgement as well (waves with three
    // unit ends ran ~8 us longer at a 2 % budget).  A third one before the end is written.
    struct Held {
        f32x4_t O[8];
        float m, l;
        int b, h;
        bool from_start, ends_unit;
    };
    Held held0, held1;
    int n_held = 0;

    Chunk nxt;
    int tok_next = 0;
    bool live_next = issue(bc, 0, nxt, tok_next);
    int ci = 0;
    for (;;) {
        Chunk ch = nxt;
        const bool live = live_next;
        const int tok0 = tok_next;
        const int L = bc.L;
        const bool last_in_batch = ci + 1 == bc.n * cpp;
        if (!last_in_batch) {
            live_next = issue(bc, ci + 1, nxt, tok_next);
            if (bn_pending) {
                fetch_batch_end(a, bn);
                bn_pending = false;
            }
        } else if (have_next) {
            if (bn_pending) {  // a one-chunk batch: bn is needed now
                fetch_batch_end(a, bn);
                bn_pending = false;
            }
            live_next = issue(bn, 0, nxt, tok_next);
            if (bc.ends_unit)
                load_q(a, bn.b, bn.h, lr, lg, qn);
        }

        if (live)
            attend_chunk(ch, L - tok0, qf, a.scale_log2, lg, m_run, l_run, O);

        if (!last_in_batch) {
            ++ci;
            continue;
        }
        if (bc.ends_unit || !have_next) {
            // ---- the unit's state: written at the end of the range (the output itself, or a
            // partial for the merge), or held until then
            float l_tot = l_run + __shfl_xor(l_run, 16, 64);
            l_tot += __shfl_xor(l_tot, 32, 64);
            if (!have_next) {
                write_unit(O, m_run, l_tot, bc.b, bc.h, from_start, bc.ends_unit);
                if (n_held > 0)
                    write_unit(held0.O, held0.m, held0.l, held0.b, held0.h, held0.from_start,
                               held0.ends_unit);
                if (n_held > 1)
                    write_unit(held1.O, held1.m, held1.l, held1.b, held1.h, held1.from_start,
                               held1.ends_unit);
                break;
            }
            if (n_held == 0) {
                held0 = Held{{O[0], O[1], O[2], O[3], O[4], O[5], O[6], O[7]}, m_run, l_tot, bc.b,
                             bc.h, from_start, bc.ends_unit};
                n_held = 1;
            } else if (n_held == 1) {
                held1 = Held{{O[0], O[1], O[2], O[3], O[4], O[5], O[6], O[7]}, m_run, l_tot, bc.b,
                             bc.h, from_start, bc.ends_unit};
                n_held = 2;
            } else {
                write_unit(O, m_run, l_tot, bc.b, bc.h, from_start, bc.ends_unit);
            }
            m_run = -INFINITY;
            l_run = 0.f;
#pragma unroll
            for (int c = 0; c < 8; ++c)
                O[c] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int i = 0; i < 4; ++i)
                qf[i] = qn[i];
            from_start = bn.j0 == 0;
        }
        bc = bn;
        ci = 0;
        have_next = cur.pos < pos_end;
        bn_pending = have_next;
        if (have_next)
            fetch_batch_begin<kSparse>(a, s_off, cur, pos_end, bn, lane);
    }
}

// Small problems (few units, short lists): one workgroup per (sequence, KV head) unit.  The
// unit's list is split evenly over the workgroup's waves and the waves' (m, l, o) states are
// merged in LDS in wave order, so the output is written with no partials in HBM and no merge
// launch.  At this size the step is a chain of dependent launches and memory round trips,
// so the kernel requests the query rows, the length, the budget, the whole page list and the
// block-table row (staged in LDS) together.  Each wave then streams its pages with the next
// chunk's loads in flight; a unit's K/V reads are bound by what one compute unit can fetch
// (about 64 GB/s measured), which is why the path is kept to short lists.
constexpr int kUnitThreads = 512;
constexpr int kUnitWaves = kUnitThreads / 64;
constexpr int kUnitMaxUnits = 256;     // at most one workgroup per compute unit
constexpr int kUnitMaxTokens = 1024;   // list bound x page size, per unit
constexpr int kUnitMaxGroup = 8;       // query heads per KV head (sizes the LDS)
constexpr int kUnitRow = kHeadDim + 4;  // LDS row stride of a wave's o (floats)
constexpr int kUnitBtLds = 4096;       // widest block-table row (staged in LDS)
// A list holds at most 64 pages (the smallest page is 16 tokens), one per lane.
static_assert(kUnitMaxTokens / 16 <= 64, "a unit's list must fit one wave's lanes");

// The attention of one unit over the `cnt` pages of its list, by the workgroup's waves, with
// the output written: wave w streams list positions [w cnt / 8, (w + 1) cnt / 8), and the
// waves' (m, l, o) states are merged in LDS in wave order.  entry_of(p) gives the logical
// page at list position p (every lane calls it; positions past the list are ignored).  The
// block-table row is in s_bt; s_o, s_m, s_l are the merge's LDS.
template <typename EntryOf>
__device__ __forceinline__ void unit_attend(const AttnArgs &a, int b, int h, int L, int cnt,
                                            const bf16x8_t (&qf)[4], const int32_t *s_bt,
                                            float *s_o, float *s_m, float *s_l, EntryOf entry_of)
{
    const int Hkv = a.num_kv_heads;
    const int G = a.num_q_heads / Hkv;  // <= kUnitMaxGroup (checked by the launcher)
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const int lr = lane & 15;
    const int lg = lane >> 4;
    const int ps = a.ps;
    const int cpp = ps >> 4;  // 16-token chunks per page
    const int64_t head_elems = (int64_t)ps * kHeadDim;
    const int np = (L + ps - 1) / ps;
    const int p0 = (int)((int64_t)wv * cnt / kUnitWaves);
    const int nw = (int)((int64_t)(wv + 1) * cnt / kUnitWaves) - p0;  // <= 8 pages
    // lane i < nw describes list position p0 + i
    const int e = entry_of(p0 + lane);
    int phys = -1, tok_first = 0;
    if (lane < nw && e >= 0 && e < np) {  // entries outside the sequence: no page
        phys = s_bt[e];
        tok_first = e * ps;
    }

    float m_run = -INFINITY;
    float l_run = 0.f;
    f32x4_t O[8];
#pragma unroll
    for (int c = 0; c < 8; ++c)
        O[c] = (f32x4_t){0.f, 0.f, 0.f, 0.f};

    // chunk `ci` of the wave's share: page ci / cpp, sub-chunk ci % cpp; a block-table entry
    // outside the cache is an absent page
    auto issue = [&](int ci, Chunk &ch, int &tok) -> bool {
        const int pi = ci / cpp;
        const int sub = ci - pi * cpp;
        const int ph = __builtin_amdgcn_readlane(phys, pi);
        tok = __builtin_amdgcn_readlane(tok_first, pi) + 16 * sub;
        const bool live = ph >= 0 && ph < a.num_phys && tok < L;
        if (live) {
            const int64_t off =
                ((int64_t)ph * Hkv + h) * head_elems + (int64_t)(16 * sub) * kHeadDim;
            load_chunk(ch, a.k_cache + off, a.v_cache + off, lr, lg);
        }
        return live;
    };
    // the wave's chunks in order, the next one's loads in flight
    const int nch = nw * cpp;
    Chunk nxt;
    int tok_next = 0;
    bool live_next = nch > 0 && issue(0, nxt, tok_next);
    for (int ci = 0; ci < nch; ++ci) {
        Chunk ch = nxt;
        const bool lv = live_next;
        const int t0 = tok_next;
        if (ci + 1 < nch)
            live_next = issue(ci + 1, nxt, tok_next);
        if (lv)
            attend_chunk(ch, L - t0, qf, a.scale_log2, lg, m_run, l_run, O);
    }

    // ---- the waves' states into LDS (lane (g, r) holds head g, channels 32r .. 32r+31)
    float l_tot = l_run + __shfl_xor(l_run, 16, 64);
    l_tot += __shfl_xor(l_tot, 32, 64);
    if (lr < G) {
        float *op = s_o + (wv * kUnitMaxGroup + lr) * kUnitRow + 32 * lg;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            *reinterpret_cast<f32x4_t *>(op + 8 * i) = (f32x4_t){O[0][i], O[1][i], O[2][i], O[3][i]};
            *reinterpret_cast<f32x4_t *>(op + 8 * i + 4) =
                (f32x4_t){O[4][i], O[5][i], O[6][i], O[7][i]};
        }
        if (lg == 0) {
            s_m[wv * kUnitMaxGroup + lr] = m_run;
            s_l[wv * kUnitMaxGroup + lr] = l_tot;
        }
    }
    __syncthreads();

    // ---- merge in wave order: o = sum_w 2^(m_w - M) o_w / sum_w 2^(m_w - M) l_w
    for (int x = threadIdx.x; x < G * kHeadDim; x += kUnitThreads) {
        const int g = x / kHeadDim;
        const int d = x - g * kHeadDim;
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < kUnitWaves; ++w)
            M = fmaxf(M, s_m[w * kUnitMaxGroup + g]);
        float lsum = 0.f, acc = 0.f;
        if (M != -INFINITY) {
#pragma unroll
            for (int w = 0; w < kUnitWaves; ++w) {
                const float m = s_m[w * kUnitMaxGroup + g];
                const float f = m == -INFINITY ? 0.f : exp2f(m - M);  // no pages: weight 0
                lsum += f * s_l[w * kUnitMaxGroup + g];
                acc += f * s_o[(w * kUnitMaxGroup + g) * kUnitRow + d];
            }
        }
        const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
        store_out(a.out, a.out_bf16, ((int64_t)b * a.num_q_heads + (int64_t)h * G + g) * kHeadDim + d,
                  acc * inv);
    }
}

// The block-table row of sequence b into LDS (max_pages <= kUnitBtLds): every load is issued
// before the first store waits on one.
__device__ __forceinline__ void stage_block_table(const AttnArgs &a, int b, int32_t *s_bt)
{
    int32_t v[kUnitBtLds / kUnitThreads];
#pragma unroll
    for (int i = 0; i < kUnitBtLds / kUnitThreads; ++i) {
        const int t = threadIdx.x + i * kUnitThreads;
        v[i] = t < a.max_pages ? a.block_table[(int64_t)b * a.max_pages + t] : 0;
    }
#pragma unroll
    for (int i = 0; i < kUnitBtLds / kUnitThreads; ++i) {
        const int t = threadIdx.x + i * kUnitThreads;
        if (t < a.max_pages)
            s_bt[t] = v[i];
    }
}

template <bool kSparse>
__global__ __launch_bounds__(kUnitThreads) void k_attn_unit(AttnArgs a)
{
    __shared__ float s_o[kUnitWaves * kUnitMaxGroup * kUnitRow];
    __shared__ float s_m[kUnitWaves * kUnitMaxGroup];
    __shared__ float s_l[kUnitWaves * kUnitMaxGroup];
    __shared__ int32_t s_bt[kUnitBtLds];
    __shared__ int32_t s_hdr[2];  // length, budget
    const int Hkv = a.num_kv_heads;
    const int unit = blockIdx.x;
    const int b = unit / Hkv;
    const int h = unit - b * Hkv;
    const int lane = threadIdx.x & 63;

    // ---- one round trip for everything the K/V loads depend on: the query rows, the
    // length and the budget, the unit's page list (lane i holds entry i; k_max <= 64 on this
    // path) and the block-table row, staged in LDS (max_pages <= kUnitBtLds on this path).
    // The length and the budget are read with relaxed atomic loads so that they are vector
    // loads: scalar loads would share their wait counter with the kernel-argument loads and
    // add a round trip of their own.
    bf16x8_t qf[4];
    load_q(a, b, h, lane & 15, lane >> 4, qf);
    int entry = -1;
    if (kSparse && lane < a.k_max)
        entry = a.idx[((int64_t)b * Hkv + h) * a.k_max + lane];
    int32_t hdr = 0;
    if (threadIdx.x < 2) {
        const int32_t *hp = kSparse && threadIdx.x == 1 ? a.ksel + b : a.seq_lens + b;
        hdr = __hip_atomic_load(hp, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    stage_block_table(a, b, s_bt);
    if (threadIdx.x < 2)
        s_hdr[threadIdx.x] = hdr;
    __syncthreads();

    const int L = clamp_len(s_hdr[0], a.ps, a.max_pages);
    const int np = (L + a.ps - 1) / a.ps;
    const int c = s_hdr[1];
    const int cnt = kSparse ? (c < 0 ? 0 : (c > a.k_max ? a.k_max : c)) : np;
    unit_attend(a, b, h, L, cnt, qf, s_bt, s_o, s_m, s_l,
                [&](int p) { return kSparse ? __shfl(entry, p, 64) : p; });
}

// Small problems, after the scoring kernel (sparrow_decode_step): the budget, the top-k and
// the attention of one unit in one workgroup.  The selection stays in LDS - it is written to
// out_k / out_idx as well, as k_topk writes them - so the step needs no top-k launch and no
// page-list round trip.  The selection is k_topk's (block_topk on the same keys) and the
// attention k_attn_unit's (unit_attend on the same list), so the results equal those of the
// separate calls bit for bit.
constexpr int kUnitMaxList = kUnitMaxTokens / 16;  // pages in a unit's list, at most

struct SelectArgs {
    const float *scores;  // [batch][num_kv_heads][max_pages], from the scoring kernel
    Sched sched;
    int32_t *out_k;
    int32_t *out_idx;
};

__global__ __launch_bounds__(kUnitThreads) void k_select_attn_unit(AttnArgs a, SelectArgs sel)
{
    // s_o holds the top-k keys first (n <= kUnitBtLds of them), then the waves' o
    __shared__ float s_o[kUnitWaves * kUnitMaxGroup * kUnitRow];
    __shared__ float s_m[kUnitWaves * kUnitMaxGroup];
    __shared__ float s_l[kUnitWaves * kUnitMaxGroup];
    __shared__ int32_t s_bt[kUnitBtLds];
    __shared__ int32_t s_tab[2][kUnitThreads];  // the schedule's tables, when they fit
    __shared__ int32_t s_sel[kUnitMaxList];
    __shared__ int32_t s_len;
    __shared__ TopkLds t;
    static_assert(kUnitWaves * kUnitMaxGroup * kUnitRow >= kUnitBtLds, "the keys fit s_o");
    constexpr int kPer = kUnitBtLds / kUnitThreads;  // scores per thread
    const int Hkv = a.num_kv_heads;
    const int unit = blockIdx.x;
    const int b = unit / Hkv;
    const int h = unit - b * Hkv;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const Sched &sc = sel.sched;

    // ---- one round trip: the query rows, the length (a vector load, as in k_attn_unit), the
    // schedule's tables, the unit's scores up to the block table's width (entries past the
    // sequence are never used) and the block-table row
    bf16x8_t qf[4];
    load_q(a, b, h, lane & 15, lane >> 4, qf);
    int32_t len = 0;
    if (tid == 0)
        len = __hip_atomic_load(a.seq_lens + b, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const bool tab_lds = sc.n_bins <= kUnitThreads;
    int32_t t_min = 0, t_frac = 0;
    if (tab_lds && tid < sc.n_bins) {
        t_min = sc.min_pages[tid];
        t_frac = sc.frac_num[tid];
    }
    const float *src = sel.scores + (int64_t)unit * a.max_pages;
    float v[kPer];
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
        const int i = tid + kUnitThreads * j;
        v[j] = i < a.max_pages ? src[i] : 0.f;
    }
    stage_block_table(a, b, s_bt);
    if (tab_lds && tid < sc.n_bins) {
        s_tab[0][tid] = t_min;
        s_tab[1][tid] = t_frac;
    }
    if (tid == 0)
        s_len = len;
    __syncthreads();

    // ---- budget (capped at k_max <= kUnitMaxList) and selection into s_sel
    const int L = clamp_len(s_len, a.ps, a.max_pages);
    const int n = (L + a.ps - 1) / a.ps;
    int k;
    if (tab_lds) {
        const int bin = L > 0 ? budget_bin(L, sc) : 0;
        k = L > 0 ? budget_from(L, a.ps, s_tab[0][bin], s_tab[1][bin], sc.frac_den, a.k_max) : 0;
    } else {
        k = budget_pages(L, a.ps, sc, a.k_max);
    }
    if (h == 0 && tid == 0)
        sel.out_k[b] = k;
    if (k >= n) {  // every page kept (k == n <= kUnitMaxList; also n == 0)
        if (tid < n)
            s_sel[tid] = tid;
    } else {
        uint32_t *keys = reinterpret_cast<uint32_t *>(s_o);
        uint32_t kmin = 0xffffffffu, kmax = 0u;
#pragma unroll
        for (int j = 0; j < kPer; ++j) {
            const int i = tid + kUnitThreads * j;
            if (i < n) {
                // forced pages (sinks, most recent pages) outrank every score
                const bool forced = i < sc.sink_pages || i >= n - sc.local_pages;
                const uint32_t key = forced ? 0xffffffffu : score_key(v[j]);
                keys[i] = key;
                kmin = min(kmin, key);
                kmax = max(kmax, key);
            }
        }
        block_topk<kUnitThreads>(keys, n, k, kmin, kmax, t,
                                 [&](uint32_t pos, int i) { s_sel[pos] = i; });
    }
    __syncthreads();  // s_sel complete; the keys are dead, s_o is free for the merge

    int32_t *row = sel.out_idx + (int64_t)unit * a.k_max;
    for (int i = tid; i < a.k_max; i += kUnitThreads)
        row[i] = i < k ? s_sel[i] : -1;
    unit_attend(a, b, h, L, k, qf, s_bt, s_o, s_m, s_l,
                [&](int p) { return s_sel[p < kUnitMaxList ? p : kUnitMaxList - 1]; });
}

// Merges the partials of a query-head row whose (sequence, KV head) unit spans several waves,
// and writes zero rows for sequences without pages.  A half-wave (32 lanes, 4 channels per
// lane) per query-head row, 8 rows per 256-thread workgroup, no LDS.  Segments are taken
// kMergeChunk at a time: every lane issues the loads of its channels for the whole chunk at
// once while lane t loads the (m, l) pair of segment t; the weights 2^(m - M) against the
// running maximum M are formed with half-wave DPP reductions and lane reads.
constexpr int kMergeChunk = 16;
constexpr int kMergeThreads = 256;
constexpr int kMergeRows = kMergeThreads / 32;

__device__ __forceinline__ void store_out4(void *out, int out_bf16, int64_t i, f32x4_t v)
{
    if (out_bf16)
        *reinterpret_cast<u32x2_t *>(static_cast<uint16_t *>(out) + i) =
            (u32x2_t){pack_bf16(v[0], v[1]), pack_bf16(v[2], v[3])};
    else
        st16(static_cast<float *>(out) + i, __builtin_bit_cast(u32x4_t, v));
}

__global__ __launch_bounds__(kMergeThreads) void k_attn_merge(AttnArgs a)
{
    const int Hq = a.num_q_heads;
    const int Hkv = a.num_kv_heads;
    const int G = Hq / Hkv;
    const int row = blockIdx.x * kMergeRows + (threadIdx.x >> 5);
    if (row >= a.batch * Hq)
        return;
    const int t = threadIdx.x & 31;  // lane within the half-wave
    const int b = row / Hq;
    const int j = row - b * Hq;
    const int h = j / G;
    const int g = j - h * G;
    const int unit = b * Hkv + h;
    const int64_t orow = (int64_t)row * kHeadDim + 4 * t;
    const int32_t o0 = a.plan_off[b], o1 = a.plan_off[b + 1];
    const int wf = a.unit_waves[2 * unit];      // wave holding the unit's first page
    const int wl = a.unit_waves[2 * unit + 1];  // wave holding its last page
    if (o1 == o0) {
        store_out4(a.out, a.out_bf16, orow, (f32x4_t){0.f, 0.f, 0.f, 0.f});
        return;
    }
    if (wf == wl)
        return;  // one wave held the whole unit and wrote its output
    const int nseg = wl - wf + 1;
    const int64_t seg0 = (int64_t)wf + unit;  // segment of wave wf for this unit
    f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
    float M = -INFINITY, lsum = 0.f;
    for (int c0 = 0; c0 < nseg; c0 += kMergeChunk) {
        const int n = nseg - c0 < kMergeChunk ? nseg - c0 : kMergeChunk;
        f32x4_t o[kMergeChunk];
#pragma unroll
        for (int i = 0; i < kMergeChunk; ++i) {
            o[i] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
            if (i < n)
                o[i] = __builtin_bit_cast(
                    f32x4_t, ld16(a.o_part + ((seg0 + c0 + i) * G + g) * kHeadDim + 4 * t));
        }
        float m = -INFINITY, l = 0.f;
        if (t < n) {
            const int64_t sg = (seg0 + c0 + t) * G + g;
            m = a.ml_part[sg * 2];
            l = a.ml_part[sg * 2 + 1];
        }
        const float cm = half_wave_max(m);
        const float Mn = fmaxf(M, cm);
        const float r = M == -INFINITY ? 0.f : exp2f(M - Mn);
        const float f = m == -INFINITY ? 0.f : exp2f(m - Mn);  // no valid pages: weight 0
        const float fl = half_wave_sum(f * l);
        lsum = lsum * r + fl;
        M = Mn;
        acc *= r;
        const bool upper = threadIdx.x & 32;  // this half-wave's weights sit in lanes 32..
#pragma unroll
        for (int i = 0; i < kMergeChunk; ++i) {
            const float f_lo = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(f), i));
            const float f_hi = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(f), 32 + i));
            acc += (upper ? f_hi : f_lo) * o[i];
        }
    }
    const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
    store_out4(a.out, a.out_bf16, orow, acc * inv);
}

// Streaming waves on the current device: compute units x resident workgroups x 4, capped.
// (A per-process cache of device attributes, safe to fill from several host threads at
// once - they all store the same value; no per-call state.)
int device_waves()
{
    static std::atomic<int> cached[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64)
        return kMaxWaves;
    int w = cached[dev].load(std::memory_order_relaxed);
    if (w == 0) {
        int cus = 0, per_cu = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            cus < 1)
            cus = 256;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_attn_stream<true>,
                                                         kAttnThreads, 4096) != hipSuccess ||
            per_cu < 1)
            per_cu = 1;
        w = cus * per_cu * kAttnWaves;
        w = w < kMaxWaves ? w : kMaxWaves;
        cached[dev].store(w, std::memory_order_relaxed);
    }
    return w;
}

// Attention workspace that lives in the library, for callers that cannot allocate
// (sparrow_sparse_decode_attn_noalloc).  Each GPU the library runs on holds one copy of the
// array until the process ends; host code reaches it only through the address that
// hipGetSymbolAddress returns on that device (the array's name is a host-side stand-in).
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

}  // namespace

void *attention_scratch()
{
    static std::atomic<void *> addr[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64)
        return nullptr;
    void *p = addr[dev].load(std::memory_order_acquire);
    if (p == nullptr) {
        // once per device, with that device current (concurrent first calls all store the
        // same address)
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess)
            return nullptr;
        addr[dev].store(p, std::memory_order_release);
    }
    return p;
}

AttnPlan plan_attention(const sparrow_shape_t &s)
{
    AttnPlan p;
    const int64_t units = (int64_t)s.batch * s.num_kv_heads;
    const int G = s.num_q_heads / s.num_kv_heads;
    p.plan_bytes = ((size_t)(s.batch + 1) * sizeof(int32_t) + 255) / 256 * 256 +
                   ((size_t)units * 2 * sizeof(int32_t) + 255) / 256 * 256;
    p.segments = (size_t)kMaxWaves + (size_t)units;
    p.workspace_bytes = p.plan_bytes + p.segments * (size_t)G * (kHeadDim + 2) * sizeof(float);
    p.lds_bytes = (size_t)(s.batch + 1) * sizeof(int32_t);
    return p;
}

namespace {

AttnArgs make_args(const sparrow_shape_t &s, const AttnPlan &plan, const void *q,
                   const void *k_cache, const void *v_cache, const int32_t *block_table,
                   const int32_t *seq_lens, const int32_t *k, const int32_t *idx, int32_t k_max,
                   float scale, void *out, int out_dtype, void *workspace)
{
    const int G = s.num_q_heads / s.num_kv_heads;
    AttnArgs a;
    a.q = static_cast<const uint16_t *>(q);
    a.k_cache = static_cast<const uint16_t *>(k_cache);
    a.v_cache = static_cast<const uint16_t *>(v_cache);
    a.block_table = block_table;
    a.seq_lens = seq_lens;
    a.ksel = k;
    a.idx = idx;
    a.plan_off = static_cast<int32_t *>(workspace);
    a.unit_waves = a.plan_off == nullptr
                       ? nullptr
                       : a.plan_off + ((size_t)(s.batch + 1) + 63) / 64 * 64;
    a.o_part = workspace == nullptr
                   ? nullptr
                   : reinterpret_cast<float *>(static_cast<char *>(workspace) + plan.plan_bytes);
    a.ml_part = a.o_part == nullptr ? nullptr : a.o_part + plan.segments * G * kHeadDim;
    a.out = out;
    a.k_max = k_max;
    a.batch = s.batch;
    a.num_q_heads = s.num_q_heads;
    a.num_kv_heads = s.num_kv_heads;
    a.ps = s.page_size;
    a.max_pages = s.max_pages_per_seq;
    a.num_phys = s.num_phys_pages;
    a.out_bf16 = out_dtype == SPARROW_OUT_BF16 ? 1 : 0;
    a.total_waves = device_waves();
    a.scale_log2 = scale * 1.4426950408889634f;
    return a;
}

}  // namespace

// A small problem: one workgroup per unit, merged in LDS (no partials, no merge launch).  The
// list bound is k_max for a sparse call and the block table's width for a dense one, so a
// full-budget sparse call with k_max = that width takes the same path as the dense call.
bool attention_unit_path(const sparrow_shape_t &s, int64_t list_bound)
{
    const int G = s.num_q_heads / s.num_kv_heads;
    return (int64_t)s.batch * s.num_kv_heads <= kUnitMaxUnits && G <= kUnitMaxGroup &&
           list_bound * s.page_size <= kUnitMaxTokens && s.max_pages_per_seq <= kUnitBtLds;
}

hipError_t launch_attention(const sparrow_shape_t &s, const AttnPlan &plan, const void *q,
                            const void *k_cache, const void *v_cache, const int32_t *block_table,
                            const int32_t *seq_lens, const int32_t *k, const int32_t *idx,
                            int32_t k_max, float scale, void *out, int out_dtype,
                            void *workspace, hipStream_t stream)
{
    const AttnArgs a = make_args(s, plan, q, k_cache, v_cache, block_table, seq_lens, k, idx,
                                 k_max, scale, out, out_dtype, workspace);
    const int64_t units = (int64_t)s.batch * s.num_kv_heads;
    if (attention_unit_path(s, idx != nullptr ? k_max : s.max_pages_per_seq)) {
        if (idx != nullptr)
            hipLaunchKernelGGL(k_attn_unit<true>, dim3((unsigned)units), dim3(kUnitThreads), 0,
                               stream, a);
        else
            hipLaunchKernelGGL(k_attn_unit<false>, dim3((unsigned)units), dim3(kUnitThreads), 0,
                               stream, a);
        return hipGetLastError();
    }
    const dim3 grid(a.total_waves / kAttnWaves);
    if (idx != nullptr)
        hipLaunchKernelGGL(k_attn_stream<true>, grid, dim3(kAttnThreads), plan.lds_bytes, stream,
                           a);
    else
        hipLaunchKernelGGL(k_attn_stream<false>, grid, dim3(kAttnThreads), plan.lds_bytes, stream,
                           a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    const int rows = s.batch * s.num_q_heads;
    hipLaunchKernelGGL(k_attn_merge, dim3((rows + kMergeRows - 1) / kMergeRows),
                       dim3(kMergeThreads), 0, stream, a);
    return hipGetLastError();
}

hipError_t launch_select_attention(const sparrow_shape_t &s, const void *q, const void *k_cache,
                                   const void *v_cache, const int32_t *block_table,
                                   const int32_t *seq_lens, const Sched &sched, int32_t k_max,
                                   const float *scores, int32_t *out_k, int32_t *out_idx,
                                   float scale, void *out, int out_dtype, hipStream_t stream)
{
    AttnPlan none{};
    const AttnArgs a = make_args(s, none, q, k_cache, v_cache, block_table, seq_lens, out_k,
                                 out_idx, k_max, scale, out, out_dtype, nullptr);
    const SelectArgs sel{scores, sched, out_k, out_idx};
    const int64_t units = (int64_t)s.batch * s.num_kv_heads;
    hipLaunchKernelGGL(k_select_attn_unit, dim3((unsigned)units), dim3(kUnitThreads), 0, stream,
                       a, sel);
    return hipGetLastError();
}

}  // namespace sparrow
