// Footprint-bitmap helpers shared by the compaction kernels (compaction
// count, which runs inside the data-gradient preparation launch, and the
// scatter).
#pragma once

#include "common.hpp"
#include "kernels.hpp"

namespace cbw {

constexpr int kCompactThreads = 256;   // threads (= pixels) per compaction block

// Any bit set in the bit range [lo, hi) of a packed bitmap.
__device__ __forceinline__ bool any_bits(const uint32_t* __restrict__ bits, int64_t lo, int64_t hi)
{
    if (lo >= hi) return false;
    int64_t w0 = lo >> 5, w1 = (hi - 1) >> 5;
    uint32_t acc = 0;
    for (int64_t w = w0; w <= w1; ++w) {
        uint32_t v = bits[w];
        if (w == w0) v &= 0xffffffffu << (lo & 31);
        if (w == w1) {
            const int top = (int)((hi - 1) & 31);
            v &= (top == 31) ? 0xffffffffu : ((2u << top) - 1u);
        }
        acc |= v;
    }
    return acc != 0;
}

// Liveness of (pixel, channel group g): any footprint bit set among the
// group's channels.  With C a multiple of 256 the group's 8 words are one
// 32-byte aligned run, read as two vectors.
__device__ __forceinline__ bool pixel_live(const CompactParams& p, int px, int g)
{
    if (px >= p.npix) return false;
    const int64_t base = (int64_t)px * p.C;
    const int lo = g * p.G;
    if (p.G == 256 && (p.C & 255) == 0) {
        const uint4* w = reinterpret_cast<const uint4*>(p.mask + ((base + lo) >> 5));
        const uint4 a = w[0], b = w[1];
        return ((a.x | a.y | a.z | a.w) | (b.x | b.y | b.z | b.w)) != 0;
    }
    const int hi = min(p.C, lo + p.G);
    return any_bits(p.mask, base + lo, base + hi);
}

// Number of set flags among the block's 256 threads (one pixel each).
__device__ __forceinline__ int block_count(bool flag, int* red)
{
    const uint64_t b = __ballot(flag);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0) red[wave] = __popcll(b);
    __syncthreads();
    return red[0] + red[1] + red[2] + red[3];
}

// Counts the live pixels of compaction block `blk` of group `g` into
// blk_counts[g][blk] (called by a whole 256-thread block).
__device__ __forceinline__ void compact_count_block(const CompactParams& p, int blk, int g)
{
    __shared__ int red[4];
    const bool live = pixel_live(p, blk * kCompactThreads + threadIdx.x, g);
    const int tot = block_count(live, red);
    if (threadIdx.x == 0) p.blk_counts[(int64_t)g * p.nblk + blk] = tot;
}

}  // namespace cbw
