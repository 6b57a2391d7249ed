// Read-only HBM streaming reference (a measurement helper beside the method's kernels).
//
// k_stream_read reads a buffer once with the access the method's streaming kernels use -
// 16-byte vector loads with the non-temporal hint, consecutive lanes on consecutive
// vectors - from a persistent grid of two 256-thread workgroups per compute unit.  A
// workgroup takes contiguous 32 KiB tiles (tile t, t + grid, ...), eight loads in flight
// per thread, each load instruction of a wave reading 1 KiB; this layout sustained the
// highest rate among the grid-stride and tiled layouts with 2-16 workgroups per CU that
// were measured for it.  Every 32-bit word is added into a per-thread sum (so no load can
// be dropped); the workgroup totals go to one counter with an atomic add.  The achieved
// bytes per second are the rate a pure read stream sustains on the device, the practical
// ceiling that the read-dominated kernels of the decode step can be compared with, beside
// the HBM peak.
#include "common.h"

namespace sparrow {
namespace {

constexpr int kProbeThreads = 256;
constexpr int kProbeInFlight = 8;
constexpr int kProbeTile = kProbeThreads * kProbeInFlight;  // 16-byte vectors per tile
constexpr int kProbeBlocksPerCu = 2;

__global__ __launch_bounds__(kProbeThreads) void k_stream_read(const u32x4_t *__restrict__ src,
                                                               int64_t nvec,
                                                               uint32_t *__restrict__ checksum)
{
    __shared__ uint32_t s_sum[kProbeThreads / 64];
    const int64_t tiles = nvec / kProbeTile;
    uint32_t acc = 0;
    for (int64_t t = blockIdx.x; t < tiles; t += gridDim.x) {
        const u32x4_t *p = src + t * kProbeTile + threadIdx.x;
        u32x4_t x[kProbeInFlight];
#pragma unroll
        for (int j = 0; j < kProbeInFlight; ++j)
            x[j] = __builtin_nontemporal_load(p + j * kProbeThreads);
#pragma unroll
        for (int j = 0; j < kProbeInFlight; ++j)
            acc += x[j][0] + x[j][1] + x[j][2] + x[j][3];
    }
    // the vectors after the last whole tile
    for (int64_t v = tiles * kProbeTile + (int64_t)blockIdx.x * kProbeThreads + threadIdx.x;
         v < nvec; v += (int64_t)gridDim.x * kProbeThreads) {
        const u32x4_t x = __builtin_nontemporal_load(src + v);
        acc += x[0] + x[1] + x[2] + x[3];
    }
#pragma unroll
    for (int off = 1; off < 64; off <<= 1)
        acc += __shfl_xor(acc, off, 64);
    if ((threadIdx.x & 63) == 0)
        s_sum[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t total = 0;
        for (int w = 0; w < kProbeThreads / 64; ++w)
            total += s_sum[w];
        atomicAdd(checksum, total);
    }
}

}  // namespace

hipError_t launch_stream_read(const void *src, int64_t bytes, uint32_t *checksum,
                              hipStream_t stream)
{
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus < 1)
        cus = 256;
    const int64_t nvec = bytes / 16;
    int64_t blocks = (int64_t)cus * kProbeBlocksPerCu;
    const int64_t need = (nvec + kProbeTile - 1) / kProbeTile;
    if (blocks > need)
        blocks = need > 0 ? need : 1;
    hipLaunchKernelGGL(k_stream_read, dim3((unsigned)blocks), dim3(kProbeThreads), 0, stream,
                       static_cast<const u32x4_t *>(src), nvec, checksum);
    return hipGetLastError();
}

}  // namespace sparrow
