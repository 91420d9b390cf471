// Device bodies shared by the stand-alone integer launches and the combined
// preparation launch of both gradients: the non-zero test of 16-byte
// vectors, and the dY block occupancy (with the X-window liveness).
#pragma once

#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"
#include "footprint.hpp"

namespace cbw {

// Bit per element: relu ? (value > 0) : (value != 0), over 16-byte vectors.
template <typename T>
__device__ __forceinline__ uint32_t vec_bits(const uint4& v, bool relu)
{
    constexpr int E = Elem<T>::E;
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    uint32_t b = 0;
#pragma unroll
    for (int i = 0; i < E; ++i) {
        uint32_t u;
        if (sizeof(T) == 2) u = (w[i >> 1] >> ((i & 1) * 16)) & 0xffffu;
        else u = w[i];
        bool on;
        if (sizeof(T) == 2) {
            const uint32_t mag = u & 0x7fffu;
            on = relu ? ((u & 0x8000u) == 0 && mag != 0 && mag <= 0x7f80u) : (mag != 0);
        } else {
            const uint32_t mag = u & 0x7fffffffu;
            on = relu ? ((u >> 31) == 0 && mag != 0 && mag <= 0x7f800000u) : (mag != 0);
        }
        b |= (on ? 1u : 0u) << i;
    }
    return b;
}

// Workgroup `block` of the occupancy pass (256 threads):
// occ[chunk][kt] = 1 iff dY has a non-zero in pixels of the chunk and
// channels of k-tile kt (from the packed footprint when given: one (pixel,
// k-tile) pair per thread and round, eight rounds' loads issued together,
// the tile's words read as one or two vectors when K is a multiple of the
// tile width).  A workgroup covers p.cpw consecutive chunks, about four
// pairs per thread, so narrow layers do not launch one nearly idle workgroup
// per 64-pixel chunk.
__device__ __forceinline__ void occupancy_block(const OccParams& p, int block)
{
    __shared__ int flags[1024];                  // [chunk of the group][k tile]
    const int chunk0 = block * p.cpw;
    const int nloc = min(p.cpw, p.nchunks - chunk0);
    const int px0 = chunk0 * p.chunk;
    const int npx = min(nloc * p.chunk, p.npq - px0);   // pixels of the group
    for (int i = threadIdx.x; i < nloc * p.ktiles; i += blockDim.x) flags[i] = 0;
    __syncthreads();
    if (p.bits) {
        // whole 8-, 16- or 32-byte aligned word runs per (pixel, k tile) when
        // K is a multiple of the tile width (64, 128 or 256 channels)
        const int vw = (p.K % p.BNk) == 0 ? (p.BNk == 256 ? 8 : p.BNk == 128 ? 4 : p.BNk == 64 ? 2 : 0) : 0;
        const int pairs = npx * p.ktiles;
        const int64_t bits_bytes = ((int64_t)p.npq * p.K + 31) / 32 * 4;
        const int lane = threadIdx.x & 63;
        // eight (pixel, k tile) pairs per thread and round; consecutive
        // threads read consecutive runs.  The runs go through a buffer
        // descriptor, so every load is issued unconditionally (a pair past
        // the group gets offset kOOB and reads zeros) and the eight of a
        // round are in flight together.  A lane marks its pair's flag only
        // when the lane before it does not mark the same one, so a wave
        // whose pairs share a chunk writes that flag once.
        auto rounds = [&](auto vw_tag) {
            constexpr int VW = decltype(vw_tag)::value;
            const __amdgpu_buffer_rsrc_t rs = make_rsrc(p.bits, (uint32_t)bits_bytes);
            for (int i0 = threadIdx.x; i0 < pairs; i0 += 8 * blockDim.x) {
                int idx[8];
                uint32_t off[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    const int i = i0 + u * blockDim.x;
                    const int j = (int)fdiv((uint32_t)i, p.div_ktiles), kt = i - j * p.ktiles;   // pixel of the group, k tile
                    idx[u] = (int)fdiv((uint32_t)j, p.div_chunk) * p.ktiles + kt;
                    off[u] = i < pairs ? (uint32_t)(((int64_t)(px0 + j) * p.K + kt * p.BNk) >> 3) : kOOB;
                }
                uint32_t w[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    if constexpr (VW == 2) {
                        const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(rs, off[u], 0, 0);
                        w[u] = v.x | v.y;
                    } else if constexpr (VW == 4) {
                        const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(rs, off[u], 0, 0);
                        w[u] = v.x | v.y | v.z | v.w;
                    } else {
                        const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(rs, off[u], 0, 0);
                        const u32x4 v2 = __builtin_amdgcn_raw_buffer_load_b128(rs, off[u] + 16u, 0, 0);
                        w[u] = (v.x | v.y | v.z | v.w) | (v2.x | v2.y | v2.z | v2.w);
                    }
                }
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    const int key = w[u] != 0u ? idx[u] : -1;
                    const int prev = __shfl_up(key, 1, 64);
                    if (key >= 0 && (lane == 0 || prev != key)) flags[idx[u]] = 1;   // every writer stores 1
                }
            }
        };
        if (vw == 2 && bits_bytes < (int64_t)kOOB) rounds(std::integral_constant<int, 2>{});
        else if (vw == 4 && bits_bytes < (int64_t)kOOB) rounds(std::integral_constant<int, 4>{});
        else if (vw == 8 && bits_bytes < (int64_t)kOOB) rounds(std::integral_constant<int, 8>{});
        else {
            for (int i = threadIdx.x; i < pairs; i += blockDim.x) {
                const int j = (int)fdiv((uint32_t)i, p.div_ktiles), kt = i - j * p.ktiles;
                const int64_t base = (int64_t)(px0 + j) * p.K;
                const int lo = kt * p.BNk, hi = min(p.K, lo + p.BNk);
                if (any_bits(p.bits, base + lo, base + hi))
                    flags[(int)fdiv((uint32_t)j, p.div_chunk) * p.ktiles + kt] = 1;   // every writer stores 1
            }
        }
    } else {
        const int E = p.dtype == 1 ? 8 : 4;
        const int vpp = p.K / E;  // vectors per pixel
        const int nv = npx * vpp;
        const uint4* v4 = reinterpret_cast<const uint4*>(static_cast<const char*>(p.dy) +
                                                         (int64_t)px0 * p.K * (p.dtype == 1 ? 2 : 4));
        for (int i = threadIdx.x; i < nv; i += blockDim.x) {
            const uint4 v = v4[i];
            const uint32_t b = p.dtype == 1 ? vec_bits<uint16_t>(v, false) : vec_bits<float>(v, false);
            const int j = i / vpp;
            if (b) flags[(int)fdiv((uint32_t)j, p.div_chunk) * p.ktiles + ((i - j * vpp) * E) / p.BNk] = 1;
        }
    }
    __syncthreads();
    bool dead = false;
    for (int i = threadIdx.x; i < nloc * p.ktiles; i += blockDim.x) {
        p.occ[(int64_t)chunk0 * p.ktiles + i] = (uint8_t)(flags[i] != 0);
        dead |= flags[i] == 0;
    }
    // the call's dead-block flag (every writer stores the same number)
    if (__syncthreads_or(dead) && p.any_dead && threadIdx.x == 0) *p.any_dead = (int)p.gen;

    // X-window liveness for every (tap group, channel tile) of the weight
    // gradient's tiling: 1 iff some pixel of the chunk has, at one of the
    // group's taps, an X pixel inside the image with a non-zero among the
    // tile's channels (from the packed X footprint).
    if (p.xlive) {
        __shared__ int xflags[1024];             // [chunk of the group][combo]
        const int ncombo = p.tgroups * p.ctiles;
        for (int i = threadIdx.x; i < nloc * ncombo; i += blockDim.x) xflags[i] = 0;
        __syncthreads();
        const int pairs = ncombo * npx;
        for (int i = threadIdx.x; i < pairs; i += blockDim.x) {
            const int combo = i / npx, j = i - combo * npx;
            const int tg = combo / p.ctiles, ct = combo - tg * p.ctiles;
            const uint32_t pix = (uint32_t)(px0 + j);
            const uint32_t nq = fdiv(pix, p.div_q);
            const int qq = (int)pix - (int)nq * p.Q;
            const uint32_t nn = fdiv(nq, p.div_p);
            const int pp = (int)nq - (int)nn * p.P;
            const int lo = ct * p.ctw, hi = min(p.C, lo + p.ctw);
            // whole 256-channel tiles on 128-bit boundaries: two vector loads
            const bool vec = hi - lo == 256 && (p.C & 127) == 0;
            bool any = false;
            for (int tl = 0; tl < p.tpg && !any; ++tl) {
                const int tap = tg * p.tpg + tl;
                if (tap >= p.RS) break;
                const int r = tap / p.S, s = tap - r * p.S;
                const int h = pp * p.stride_h - p.pad_h + r, w = qq * p.stride_w - p.pad_w + s;
                if (h < 0 || h >= p.H || w < 0 || w >= p.W) continue;
                const int64_t base = (((int64_t)nn * p.H + h) * p.W + w) * p.C;
                if (vec) {
                    const uint4* v = reinterpret_cast<const uint4*>(p.xbits + ((base + lo) >> 5));
                    const uint4 a = v[0], b = v[1];
                    any = ((a.x | a.y | a.z | a.w) | (b.x | b.y | b.z | b.w)) != 0;
                } else {
                    any = any_bits(p.xbits, base + lo, base + hi);
                }
            }
            if (any) xflags[(int)fdiv((uint32_t)j, p.div_chunk) * ncombo + combo] = 1;   // every writer stores 1
        }
        __syncthreads();
        bool xdead = false;
        for (int i = threadIdx.x; i < nloc * ncombo; i += blockDim.x) {
            p.xlive[(int64_t)chunk0 * ncombo + i] = (uint8_t)(xflags[i] != 0);
            xdead |= xflags[i] == 0;
        }
        if (__syncthreads_or(xdead) && p.any_dead && threadIdx.x == 0) *p.any_dead = (int)p.gen;
    }
}

}  // namespace cbw
