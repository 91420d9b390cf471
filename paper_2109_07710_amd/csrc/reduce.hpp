// Split-K reduction of the weight gradient (device body, shared by its own
// launch, the combined reduction launch and the tail workgroups of the
// data-gradient GEMM launch).
#pragma once

#include "common.hpp"
#include "kernels.hpp"

namespace cbw {

// Workgroup `block` (256 threads) of the reduction.
// dW = sum over splits of the partials in a fixed order.  part is
// [nsplit][K][RS][C]; dW is written in KRSC or KCRS.  A block covers 256/G
// float4 outputs with G threads each: thread g sums the consecutive splits
// [g*nsplit/G, (g+1)*nsplit/G) in order, then the G group sums are added in
// group order.  G grows (up to 16) until the launch has enough threads to
// fill the machine, so that few outputs with many splits do not run one
// long serial sum per thread.  The order depends only on (nsplit, G), so
// results are reproducible.
template <int G>
__device__ __forceinline__ void splitk_reduce_core(const float* __restrict__ part, float* __restrict__ dw, int nsplit,
                                                   int K, int RS, int C, int krsc, int block, int t,
                                                   float4 (*red)[256 / G])
{
    constexpr int OPB = 256 / G;   // float4 outputs per block
    const int64_t total = (int64_t)K * RS * C;
    const int ol = t % OPB, g = t / OPB;
    const int64_t i4 = (int64_t)block * OPB + ol;
    const float4* p4 = reinterpret_cast<const float4*>(part);
    const int z0 = (int)((int64_t)g * nsplit / G), z1 = (int)((int64_t)(g + 1) * nsplit / G);
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    if (i4 * 4 < total) {
        // the loads of up to sixteen splits are issued before any is added
        // (one round trip for the usual 4 to 16 splits per thread: the sum
        // is a chain of load latencies otherwise), then added in order
        constexpr int NL = 16;
        for (int zb = z0; zb < z1; zb += NL) {
            float4 v[NL];
#pragma unroll
            for (int u = 0; u < NL; ++u)
                v[u] = zb + u < z1 ? p4[(int64_t)(zb + u) * (total / 4) + i4] : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
            for (int u = 0; u < NL; ++u) {
                if (zb + u >= z1) break;
                if (zb + u == z0) s = v[u];
                else { s.x += v[u].x; s.y += v[u].y; s.z += v[u].z; s.w += v[u].w; }
            }
        }
    }
    if (G > 1) {
        red[g][ol] = s;
        __syncthreads();
        if (g != 0) return;
        for (int gg = 1; gg < G; ++gg) {
            const float4 v = red[gg][ol];
            // groups with no splits (nsplit < G) hold zeros and add nothing
            if ((int64_t)(gg + 1) * nsplit / G > (int64_t)gg * nsplit / G) {
                s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
            }
        }
    }
    if (i4 * 4 >= total) return;
    if (krsc) {
        reinterpret_cast<float4*>(dw)[i4] = s;
    } else {
        const int64_t i = i4 * 4;
        const int c = (int)(i % C);
        const int64_t kt = i / C;
        const int tap = (int)(kt % RS);
        const int k = (int)(kt / RS);
        const float vals[4] = {s.x, s.y, s.z, s.w};
        for (int j = 0; j < 4; ++j) dw[((int64_t)k * C + c + j) * RS + tap] = vals[j];
    }
}

template <int G>
__device__ __forceinline__ void splitk_reduce_block(const float* __restrict__ part, float* __restrict__ dw,
                                                    int nsplit, int K, int RS, int C, int krsc, int block)
{
    __shared__ float4 red[G > 1 ? G : 1][256 / G];
    splitk_reduce_core<G>(part, dw, nsplit, K, RS, C, krsc, block, threadIdx.x, red);
}

// Blocks 4 q .. 4 q + 3 of the reduction run by one 1024-thread workgroup
// (the tail items of the data-gradient GEMM launch), with the same
// summation order as four 256-thread workgroups: each quarter of the
// threads takes one block, with its own share of `scratch` (at least 16 KB
// of LDS) for the group sums.  Every thread reaches the one barrier.
__device__ __forceinline__ void splitk_reduce_quad(const ReduceParams& rp, int q, void* scratch)
{
    const int sub = threadIdx.x >> 8, t = threadIdx.x & 255;
    float4* base = static_cast<float4*>(scratch) + sub * 256;
    switch (rp.G) {
#define CBW_REDUCE_QUAD_CASE(GG) \
    case GG: \
        splitk_reduce_core<GG>(rp.part, rp.dw, rp.nsplit, rp.K, rp.RS, rp.C, rp.krsc, 4 * q + sub, t, \
                               reinterpret_cast<float4 (*)[256 / GG]>(base)); \
        break;
        CBW_REDUCE_QUAD_CASE(1) CBW_REDUCE_QUAD_CASE(2) CBW_REDUCE_QUAD_CASE(4) CBW_REDUCE_QUAD_CASE(8)
    default:
        splitk_reduce_core<16>(rp.part, rp.dw, rp.nsplit, rp.K, rp.RS, rp.C, rp.krsc, 4 * q + sub, t,
                               reinterpret_cast<float4 (*)[16]>(base));
        break;
#undef CBW_REDUCE_QUAD_CASE
    }
}

// Threads per output of the reduction for nsplit partials of n4 float4
// outputs: the smallest power of two that gives about 2^19 threads (every CU
// full), at most 16 and at most nsplit.
inline int splitk_reduce_group(int nsplit, int64_t n4)
{
    int G = 1;
    while (G < 16 && 2 * G <= nsplit && n4 * G < (1 << 19)) G *= 2;
    return G;
}

}  // namespace cbw
