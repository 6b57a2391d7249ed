// Block top-k over order-preserving keys in LDS (internal to libsparrow, not part of the
// ABI): the selection step of Sec. 2 / Sec. 3.3 of arXiv 2606.08446 - the k pages of
// largest score, ties to the lower page index, emitted in ascending page order.  Shared by
// k_topk (one workgroup per unit after the scoring kernel) and by the attention kernel that
// selects and attends in one workgroup for small problems.
#pragma once

#include "common.h"
#include "wave.h"

namespace sparrow {

// fp32 score -> uint32 whose unsigned order is the order of the scores (-0 == +0).
__device__ __forceinline__ uint32_t score_key(float s)
{
    uint32_t u = __float_as_uint(s);
    if (u == 0x80000000u)
        u = 0u;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// LDS of one block top-k (at most 16 waves).
struct TopkLds {
    uint32_t hist[2][256];
    uint32_t red_a[16], red_b[16], red_c[16];
    uint32_t digit, rem, done;
};

// Selects the k largest of keys[0 .. n) (0 < k < n <= 65535), ties to the lower index, and
// calls emit(pos, i) for every kept index i with its rank pos in ascending index order
// (0 .. k-1).  The caller has written the keys to LDS and passes this thread's minimum and
// maximum of the keys it wrote (identities 0xffffffff / 0 if none); every thread of the
// block calls this, which synchronises the block.
//
// A radix select over 8-bit digits, from the highest bit where the keys differ down (the
// bits above it are common to all keys), finds the threshold T and how many keys equal to
// T to keep; it stops as soon as the chosen digit's bin holds exactly the keys still to
// take.  One block scan of the packed pair (count > T, count == T) then gives every kept
// index its rank: pos = (#keys > T before it) + min(#keys == T before it, quota).
template <int kThreads, typename Emit>
__device__ __forceinline__ void block_topk(const uint32_t *keys, int n, int k, uint32_t kmin,
                                           uint32_t kmax, TopkLds &t, Emit emit)
{
    constexpr int kWaves = kThreads / 64;
    static_assert(kWaves <= 16, "TopkLds holds 16 waves");
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;

    for (int x = tid; x < 256; x += kThreads)
        t.hist[0][x] = 0u;
    kmin = wave_min(kmin);
    kmax = wave_max(kmax);
    if (lane == 0) {
        t.red_a[wave] = kmin;
        t.red_b[wave] = kmax;
    }
    __syncthreads();
    kmin = t.red_a[0];
    kmax = t.red_b[0];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) {
        kmin = min(kmin, t.red_a[w]);
        kmax = max(kmax, t.red_b[w]);
    }

    // After each digit the candidates are the keys whose bits >= lo equal `prefix`; `rem`
    // of them are still to be taken.  When the chosen bin holds exactly `rem` keys every
    // candidate is taken and the selection is "bits >= lo at least prefix", with no tie
    // left to break.
    uint32_t prefix = kmax;
    uint32_t rem = (uint32_t)k;
    bool exact = true;  // false: stopped early, keep keys >= prefix (bits below lo zero)
    int lo = 0;
    if (kmin != kmax) {
        int hi = 31 - __builtin_clz(kmin ^ kmax);
        int cur = 0;
        while (hi >= 0) {
            lo = hi >= 7 ? hi - 7 : 0;
            const uint32_t width_mask = (1u << (hi - lo + 1)) - 1u;
            const uint32_t above = hi >= 31 ? 0u : (0xffffffffu << (hi + 1));
            const uint32_t want = prefix & above;
            for (int base = 0; base < n; base += kThreads * 4) {
                uint32_t kv[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int i = base + tid + kThreads * j;
                    kv[j] = i < n ? keys[i] : 0u;
                }
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (base + tid + kThreads * j < n && (kv[j] & above) == want)
                        atomicAdd(&t.hist[cur][(kv[j] >> lo) & width_mask], 1u);
            }
            for (int x = tid; x < 256; x += kThreads)
                t.hist[cur ^ 1][x] = 0u;  // ready for the next digit
            __syncthreads();
            if (wave == 0) {
                // lane l owns digits 255-4l .. 252-4l; counts accumulate from the top down
                const uint32_t c0 = t.hist[cur][255 - 4 * lane], c1 = t.hist[cur][254 - 4 * lane];
                const uint32_t c2 = t.hist[cur][253 - 4 * lane], c3 = t.hist[cur][252 - 4 * lane];
                const uint32_t tot = c0 + c1 + c2 + c3;
                const uint32_t incl = wave_scan_add(tot);
                uint32_t acc = incl - tot;  // keys with a larger digit
                if (acc < rem && rem <= incl) {
                    int d;
                    uint32_t cnt;
                    if (rem <= acc + c0) {
                        d = 255 - 4 * lane;
                        cnt = c0;
                    } else if (rem <= acc + c0 + c1) {
                        acc += c0;
                        d = 254 - 4 * lane;
                        cnt = c1;
                    } else if (rem <= acc + c0 + c1 + c2) {
                        acc += c0 + c1;
                        d = 253 - 4 * lane;
                        cnt = c2;
                    } else {
                        acc += c0 + c1 + c2;
                        d = 252 - 4 * lane;
                        cnt = c3;
                    }
                    t.digit = (uint32_t)d;
                    t.rem = rem - acc;
                    t.done = cnt == rem - acc;
                }
            }
            __syncthreads();
            prefix = want | (t.digit << lo);
            rem = t.rem;
            if (t.done) {
                exact = false;
                break;
            }
            hi = lo - 1;
            cur ^= 1;
        }
    }
    // Selection rule as "key > T" plus the first `rem` keys equal to T in index order.
    uint32_t T = prefix;
    if (!exact) {
        T = prefix - 1u;  // keys >= prefix (prefix > 0 here, as fewer than n keys are kept)
        rem = 0u;
    }

    // Ranks from one block scan of (count > T, count == T) over contiguous segments.
    const int seg = (n + kThreads - 1) / kThreads;
    const int s0 = min(n, tid * seg);
    const int s1 = min(n, s0 + seg);
    uint32_t gt = 0u, eq = 0u;
    for (int i = s0; i < s1; ++i) {
        const uint32_t key = keys[i];
        gt += key > T;
        eq += key == T;
    }
    const uint32_t packed = (gt << 16) | eq;  // n < 2^16
    uint32_t incl = wave_scan_add(packed);
    if (lane == 63)
        t.red_c[wave] = incl;
    __syncthreads();
    uint32_t before = incl - packed;
    for (int w = 0; w < wave; ++w)
        before += t.red_c[w];
    uint32_t gt_b = before >> 16, eq_b = before & 0xffffu;
    for (int i = s0; i < s1; ++i) {
        const uint32_t key = keys[i];
        if (key > T) {
            const uint32_t pos = gt_b + min(eq_b, rem);
            if (pos < (uint32_t)k)
                emit(pos, i);
            ++gt_b;
        } else if (key == T) {
            if (eq_b < rem && gt_b + eq_b < (uint32_t)k)
                emit(gt_b + eq_b, i);
            ++eq_b;
        }
    }
}

}  // namespace sparrow
