// Footprint-bitmap helpers of the compaction: the counts, which run inside
// the data-gradient preparation launch, and the per-pixel liveness test the
// data-gradient GEMM repeats when it lists its own tile's pixels.
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

// Liveness of (pixel px, channel group g of width G): any footprint bit set
// among the group's channels.  With C a multiple of G and G = 256, 128 or 64
// the group's 8, 4 or 2 words are one aligned run, read as vectors.
__device__ __forceinline__ bool pixel_live_bits(const uint32_t* __restrict__ mask, int64_t npix, int C, int G, int px,
                                                int g)
{
    if (px >= npix) return false;
    const int64_t base = (int64_t)px * C;
    const int lo = g * G;
    if (G == 256 && (C & 255) == 0) {
        const uint4* w = reinterpret_cast<const uint4*>(mask + ((base + lo) >> 5));
        const uint4 a = w[0], b = w[1];
        return ((a.x | a.y | a.z | a.w) | (b.x | b.y | b.z | b.w)) != 0;
    }
    if (G == 128 && (C & 127) == 0) {
        const uint4 a = *reinterpret_cast<const uint4*>(mask + ((base + lo) >> 5));
        return (a.x | a.y | a.z | a.w) != 0;
    }
    if (G == 64 && (C & 63) == 0) {
        const uint2 a = *reinterpret_cast<const uint2*>(mask + ((base + lo) >> 5));
        return (a.x | a.y) != 0;
    }
    const int hi = min(C, lo + G);
    return any_bits(mask, base + lo, base + hi);
}

__device__ __forceinline__ bool pixel_live(const CompactParams& p, int px, int g)
{
    return pixel_live_bits(p.mask, p.npix, p.C, p.G, px, g);
}

// Counts the live pixels of compaction block `blk` of group `g` into
// blk_counts[g][blk] and clears the dX rows of the group's dead pixels in
// the block (the data-gradient GEMM never visits them).  Called by a whole
// kCompactThreads-thread block.
__device__ __forceinline__ void compact_count_block(const CompactParams& p, int blk, int g)
{
    constexpr int T = kCompactThreads, NWV = kCompactThreads / 64;
    __shared__ int wc[NWV], wd[NWV];
    __shared__ int dead_s[T];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int px = blk * T + tid;
    const bool live = pixel_live(p, px, g);   // false past the last pixel
    const bool dead = px < p.npix && !live;
    const uint64_t lb = __ballot(live), db = __ballot(dead);
    if (lane == 0) {
        wc[wave] = __popcll(lb);
        wd[wave] = __popcll(db);
    }
    __syncthreads();
    int wb = 0, ndead = 0, nlive = 0;
#pragma unroll
    for (int w = 0; w < NWV; ++w) {
        if (w < wave) wb += wd[w];
        ndead += wd[w];
        nlive += wc[w];
    }
    if (tid == 0) {
        p.blk_counts[(int64_t)g * p.nblk + blk] = nlive;
        if (nlive < min(T, p.npix - blk * T)) p.dead_flags[g] = 1;   // every writer stores 1
    }
    if (ndead == 0) return;   // uniform
    // dead pixels listed, then their rows cleared by the whole block:
    // consecutive threads write consecutive 16-byte pieces of one row, so a
    // wave covers whole rows
    const uint64_t below = lane == 0 ? 0ull : ((~0ull) >> (64 - lane));
    if (dead) dead_s[wb + __popcll(db & below)] = px;
    __syncthreads();
    const int lo = g * p.G, hi = min(p.C, lo + p.G);
    const int nvec = (hi - lo) * p.elem_bytes / 16;
    for (int q = tid; q < ndead * nvec; q += T) {
        const int d = q / nvec, v = q - d * nvec;
        uint4* row = reinterpret_cast<uint4*>(static_cast<char*>(p.dx) + ((int64_t)dead_s[d] * p.C + lo) * p.elem_bytes);
        row[v] = make_uint4(0, 0, 0, 0);
    }
}

}  // namespace cbw
