// Wave-wide (64-lane) scans on DPP row operations, for the latency-bound parts of the
// kernels (internal to libsparrow, not part of the ABI).
//
// A cross-lane shuffle (__shfl_up, __shfl_xor) compiles to ds_bpermute, a round trip
// through the LDS unit; a 6-step scan built from them is 6 dependent LDS latencies.  The
// DPP forms below move data between lanes inside the VALU: a Hillis-Steele scan inside
// each 16-lane row (row_shr:1, 2, 4, 8), then the row totals carried across rows with
// row_bcast:15 (row 0 -> 1 and row 2 -> 3) and row_bcast:31 (rows 0-1 -> 2 and 3), the
// GFX9 cross-row forms that gfx950 keeps.  A lane whose DPP source lies outside its row,
// or whose row is masked off, receives the operation's identity instead.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sparrow {

// DPP controls (GFX9 encoding).
constexpr int kDppRowShr1 = 0x111;
constexpr int kDppRowShr2 = 0x112;
constexpr int kDppRowShr4 = 0x114;
constexpr int kDppRowShr8 = 0x118;
constexpr int kDppRowBcast15 = 0x142;
constexpr int kDppRowBcast31 = 0x143;

// x moved by one DPP control; lanes without a source (or in a masked row) get `identity`.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ uint32_t dpp_move(uint32_t x, uint32_t identity)
{
    return (uint32_t)__builtin_amdgcn_update_dpp((int)identity, (int)x, kCtrl, kRowMask, 0xf,
                                                 false);
}

// Inclusive scan with the associative, commutative `op`: lane i gets op(x_0, ..., x_i).
template <typename Op>
__device__ __forceinline__ uint32_t wave_scan(uint32_t x, uint32_t identity, Op op)
{
    x = op(x, dpp_move<kDppRowShr1, 0xf>(x, identity));
    x = op(x, dpp_move<kDppRowShr2, 0xf>(x, identity));
    x = op(x, dpp_move<kDppRowShr4, 0xf>(x, identity));
    x = op(x, dpp_move<kDppRowShr8, 0xf>(x, identity));
    x = op(x, dpp_move<kDppRowBcast15, 0xa>(x, identity));
    x = op(x, dpp_move<kDppRowBcast31, 0xc>(x, identity));
    return x;
}

__device__ __forceinline__ uint32_t wave_scan_add(uint32_t x)
{
    return wave_scan(x, 0u, [](uint32_t a, uint32_t b) { return a + b; });
}

// Minimum / maximum over the wave (every lane gets it).
__device__ __forceinline__ uint32_t wave_min(uint32_t x)
{
    x = wave_scan(x, 0xffffffffu, [](uint32_t a, uint32_t b) { return a < b ? a : b; });
    return (uint32_t)__builtin_amdgcn_readlane((int)x, 63);
}

__device__ __forceinline__ uint32_t wave_max(uint32_t x)
{
    x = wave_scan(x, 0u, [](uint32_t a, uint32_t b) { return a > b ? a : b; });
    return (uint32_t)__builtin_amdgcn_readlane((int)x, 63);
}

// Reduction over each 32-lane half of the wave with the associative, commutative `op` on
// fp32: the row scan, then row_bcast:15 adds row 0 into row 1 and row 2 into row 3, so
// lanes 31 and 63 hold the two halves' results.  Every lane gets its own half's.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ float dpp_move_f(float x, float identity)
{
    return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(identity), __float_as_int(x),
                                                      kCtrl, kRowMask, 0xf, false));
}

template <typename Op>
__device__ __forceinline__ float half_wave_reduce(float x, float identity, Op op)
{
    x = op(x, dpp_move_f<kDppRowShr1, 0xf>(x, identity));
    x = op(x, dpp_move_f<kDppRowShr2, 0xf>(x, identity));
    x = op(x, dpp_move_f<kDppRowShr4, 0xf>(x, identity));
    x = op(x, dpp_move_f<kDppRowShr8, 0xf>(x, identity));
    x = op(x, dpp_move_f<kDppRowBcast15, 0xa>(x, identity));
    const float lo = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 31));
    const float hi = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 63));
    return (threadIdx.x & 32) ? hi : lo;
}

__device__ __forceinline__ float half_wave_max(float x)
{
    return half_wave_reduce(x, -INFINITY, [](float a, float b) { return fmaxf(a, b); });
}

__device__ __forceinline__ float half_wave_sum(float x)
{
    return half_wave_reduce(x, 0.f, [](float a, float b) { return a + b; });
}

}  // namespace sparrow
