// Diagnostic: the rate at which this GPU streams the decode kernels' page
// pattern, without their arithmetic.  The kernel reads every tile of a pool
// once, tiles of a KV page's size at scattered places, with the non-temporal
// 16-byte loads the attention kernel issues, and XORs every word into one
// result (so nothing is skipped and the result can be checked exactly).  Its
// bandwidth is the ceiling against which the attention kernel's can be read.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/bellman.h"
#include "internal.h"

namespace bellman {
namespace {

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

constexpr int kProbeBlock = 256;
constexpr int kProbeDepth = 4;          // tiles in flight per wave while it folds the previous four
constexpr uint64_t kProbeMul1 = 0x9E3779B97F4A7C15ull;   // odd multipliers: bijections mod 2^k
constexpr uint64_t kProbeMul2 = 0xD6E8FEB86659FD93ull;

// The tile read at position t: a bijection of [0, n), n = 2^k, that spreads
// both a wave's consecutive positions and the positions that all waves read
// at the same time over the whole pool (multiplications by odd constants and
// xor-shifts by h = k / 2 are each invertible mod 2^k), as a batch's random
// pages are spread.
__device__ __forceinline__ uint64_t probe_tile(uint64_t t, uint64_t mask, int h) {
    uint64_t x = (t * kProbeMul1) & mask;
    if (h > 0) x ^= x >> h;
    x = (x * kProbeMul2) & mask;
    if (h > 0) x ^= x >> h;
    return x;
}

// Wave w of W takes positions [n w / W, n (w + 1) / W) of the visiting order.
template <int TB>
__global__ void __launch_bounds__(kProbeBlock) gather_probe_kernel(const char* pool, int64_t n, int h, int waves,
                                                                   uint32_t* sink) {
    constexpr int NL = TB / (kWaveSize * 16);   // 16-byte loads per lane per tile
    const int lane = threadIdx.x & (kWaveSize - 1);
    const int w = __builtin_amdgcn_readfirstlane(blockIdx.x * (kProbeBlock / kWaveSize) + (threadIdx.x >> 6));
    if (w >= waves) return;
    const int64_t lo = n * w / waves, hi = n * (w + 1) / waves;
    const uint64_t mask = (uint64_t)n - 1;
    u32x4 acc = {0u, 0u, 0u, 0u};
    u32x4 buf[2][kProbeDepth][NL];
    auto issue = [&](u32x4 (&b)[kProbeDepth][NL], int64_t t0) {
#pragma unroll
        for (int d = 0; d < kProbeDepth; ++d) {
            const int64_t t = t0 + d < hi ? t0 + d : hi - 1;   // past the range: re-read, not folded
            const char* tile = pool + (int64_t)probe_tile((uint64_t)t, mask, h) * TB;
#pragma unroll
            for (int i = 0; i < NL; ++i)
                b[d][i] = __builtin_nontemporal_load((const u32x4*)(tile + (size_t)(i * kWaveSize + lane) * 16));
        }
    };
    auto fold = [&](const u32x4 (&b)[kProbeDepth][NL], int64_t t0) {
#pragma unroll
        for (int d = 0; d < kProbeDepth; ++d)
            if (t0 + d < hi)
#pragma unroll
                for (int i = 0; i < NL; ++i) acc ^= b[d][i];
    };
    if (lo < hi) {
        issue(buf[0], lo);
        int64_t t = lo;
        for (;;) {
            issue(buf[1], t + kProbeDepth);
            fold(buf[0], t);
            t += kProbeDepth;
            if (t >= hi) break;
            issue(buf[0], t + kProbeDepth);
            fold(buf[1], t);
            t += kProbeDepth;
            if (t >= hi) break;
        }
    }
    uint32_t x = acc.x ^ acc.y ^ acc.z ^ acc.w;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) x ^= (uint32_t)__shfl_xor((int)x, off, kWaveSize);
    if (lane == 0) atomicXor(sink, x);
}

}  // namespace

int launch_gather_probe(const void* pool, int64_t n, int tile_bytes, int waves, uint32_t* sink, hipStream_t s) {
    const dim3 grid((waves + kProbeBlock / kWaveSize - 1) / (kProbeBlock / kWaveSize)), blk(kProbeBlock);
    const char* p = (const char*)pool;
    int k = 0;
    while ((int64_t(1) << k) < n) ++k;
    const int h = k / 2;
    switch (tile_bytes) {
        case 2048: hipLaunchKernelGGL(gather_probe_kernel<2048>, grid, blk, 0, s, p, n, h, waves, sink); break;
        case 4096: hipLaunchKernelGGL(gather_probe_kernel<4096>, grid, blk, 0, s, p, n, h, waves, sink); break;
        case 8192: hipLaunchKernelGGL(gather_probe_kernel<8192>, grid, blk, 0, s, p, n, h, waves, sink); break;
        default: return -1;
    }
    return 0;
}

int gather_probe_blocks_per_cu(int tile_bytes) {
    int nb = 0;
    hipError_t e = hipErrorInvalidValue;
    switch (tile_bytes) {
        case 2048: e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, gather_probe_kernel<2048>, kProbeBlock, 0); break;
        case 4096: e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, gather_probe_kernel<4096>, kProbeBlock, 0); break;
        case 8192: e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, gather_probe_kernel<8192>, kProbeBlock, 0); break;
        default: break;
    }
    return (e == hipSuccess && nb > 0) ? nb : 1;
}

}  // namespace bellman
