// Integer kernels around the GEMMs: footprint bitmaps, dY block occupancy
// and the split-K reduction of dW.  (The compaction counts run in the
// data-gradient preparation launch, the live lists inside the GEMM.)
#include "common.hpp"
#include "kernels.hpp"
#include "footprint.hpp"

namespace cbw {

namespace {

constexpr int CNT = kCompactThreads;     // threads (= pixels) per compaction block
constexpr int BLK_PX = CNT;

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

template <typename T>
__device__ __forceinline__ uint32_t elem_bit(const T* p, int64_t i, bool relu)
{
    uint4 v = make_uint4(0, 0, 0, 0);
    if (sizeof(T) == 2) v.x = reinterpret_cast<const uint16_t*>(p)[i];
    else v.x = reinterpret_cast<const uint32_t*>(p)[i];
    return vec_bits<T>(v, relu) & 1u;
}

// One thread per 16-byte vector; the E bits of L = 32/E neighbouring lanes
// are OR-ed into one word written by the first of them.
template <typename T>
__global__ void mask_pack_kernel(const T* __restrict__ x, uint32_t* __restrict__ bits, int64_t count,
                                 int64_t nvec, bool relu)
{
    constexpr int E = Elem<T>::E;
    constexpr int L = 32 / E;
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    uint32_t b = 0;
    if (v < nvec) {
        const int64_t e0 = v * E;
        if (e0 + E <= count) {
            b = vec_bits<T>(*reinterpret_cast<const uint4*>(x + e0), relu);
        } else {
            for (int i = 0; i < E && e0 + i < count; ++i) b |= elem_bit<T>(x, e0 + i, relu) << i;
        }
    }
    const int lane = threadIdx.x & 63;
    b <<= (lane % L) * E;
#pragma unroll
    for (int off = 1; off < L; off <<= 1) b |= __shfl_xor(b, off);
    if (lane % L == 0 && v < nvec) bits[v / L] = b;
}


// occ[chunk][kt] = 1 iff dY has a non-zero in pixels of the chunk and
// channels of k-tile kt (from the packed footprint when given: one (pixel,
// k-tile) pair per thread, the tile's words read as vectors when the k-tile
// is 256 wide and K a multiple of 256).  A workgroup covers p.cpw
// consecutive chunks, enough pairs for its 256 threads, so narrow layers do
// not launch one nearly idle workgroup per 64-pixel chunk.
__global__ __launch_bounds__(256) void occupancy_kernel(OccParams p)
{
    __shared__ int flags[1024];                  // [chunk of the group][k tile]
    const int chunk0 = blockIdx.x * p.cpw;
    const int nloc = min(p.cpw, p.nchunks - chunk0);
    const int px0 = chunk0 * p.chunk;
    const int npx = min(nloc * p.chunk, p.npq - px0);   // pixels of the group
    for (int i = threadIdx.x; i < nloc * p.ktiles; i += blockDim.x) flags[i] = 0;
    __syncthreads();
    if (p.bits) {
        const bool vec = p.BNk == 256 && (p.K & 255) == 0;
        const int pairs = npx * p.ktiles;
        for (int i = threadIdx.x; i < pairs; i += blockDim.x) {
            const int j = i / p.ktiles, kt = i - j * p.ktiles;   // pixel of the group, k tile
            const int64_t base = (int64_t)(px0 + j) * p.K;
            const int lo = kt * p.BNk, hi = min(p.K, lo + p.BNk);
            bool any;
            if (vec) {
                const uint4* w = reinterpret_cast<const uint4*>(p.bits + ((base + lo) >> 5));
                const uint4 a = w[0], b = w[1];
                any = ((a.x | a.y | a.z | a.w) | (b.x | b.y | b.z | b.w)) != 0;
            } else {
                any = any_bits(p.bits, base + lo, base + hi);
            }
            if (any) flags[(j / p.chunk) * p.ktiles + kt] = 1;   // every writer stores 1
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
            if (b) flags[(j / p.chunk) * p.ktiles + ((i - j * vpp) * E) / p.BNk] = 1;
        }
    }
    __syncthreads();
    for (int i = threadIdx.x; i < nloc * p.ktiles; i += blockDim.x)
        p.occ[(int64_t)chunk0 * p.ktiles + i] = (uint8_t)(flags[i] != 0);

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
            if (any) xflags[(j / p.chunk) * ncombo + combo] = 1;   // every writer stores 1
        }
        __syncthreads();
        for (int i = threadIdx.x; i < nloc * ncombo; i += blockDim.x)
            p.xlive[(int64_t)chunk0 * ncombo + i] = (uint8_t)(xflags[i] != 0);
    }
}

// dW = sum over splits of the partials in a fixed order.  part is
// [nsplit][K][RS][C]; dW is written in KRSC or KCRS.  A block covers 256/G
// float4 outputs with G threads each: thread g sums the consecutive splits
// [g*nsplit/G, (g+1)*nsplit/G) in order, then the G group sums are added in
// group order.  G grows (up to 16) until the launch has enough threads to
// fill the machine, so that few outputs with many splits do not run one
// long serial sum per thread.  The order depends only on (nsplit, G), so
// results are reproducible.
template <int G>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ part, float* __restrict__ dw,
                                                           int nsplit, int K, int RS, int C, int krsc)
{
    constexpr int OPB = 256 / G;   // float4 outputs per block
    __shared__ float4 red[G > 1 ? G : 1][OPB];
    const int64_t total = (int64_t)K * RS * C;
    const int ol = threadIdx.x % OPB, g = threadIdx.x / OPB;
    const int64_t i4 = (int64_t)blockIdx.x * OPB + ol;
    const float4* p4 = reinterpret_cast<const float4*>(part);
    const int z0 = (int)((int64_t)g * nsplit / G), z1 = (int)((int64_t)(g + 1) * nsplit / G);
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    if (i4 * 4 < total) {
        // the loads of four splits are issued before they are added, in order
        for (int zb = z0; zb < z1; zb += 4) {
            float4 v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u)
                v[u] = zb + u < z1 ? p4[(int64_t)(zb + u) * (total / 4) + i4] : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
            for (int u = 0; u < 4; ++u) {
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

}  // namespace

int compact_block_pixels() { return BLK_PX; }

hipError_t launch_relu_mask_pack(int dtype, int64_t count, const void* x, uint32_t* bits, int relu,
                                 hipStream_t stream)
{
    const int E = dtype == 1 ? 8 : 4;
    const int L = 32 / E;
    int64_t nvec = (count + E - 1) / E;
    nvec = (nvec + L - 1) / L * L;  // whole words
    const int64_t blocks = (nvec + 255) / 256;
    if (blocks == 0) return hipSuccess;
    if (dtype == 1)
        mask_pack_kernel<uint16_t><<<(unsigned)blocks, 256, 0, stream>>>((const uint16_t*)x, bits, count, nvec,
                                                                         relu != 0);
    else
        mask_pack_kernel<float><<<(unsigned)blocks, 256, 0, stream>>>((const float*)x, bits, count, nvec,
                                                                      relu != 0);
    return hipGetLastError();
}

hipError_t launch_occupancy(const OccParams& p, hipStream_t stream)
{
    if (p.cpw < 1 || p.cpw * p.ktiles > 1024 || (p.xlive && p.cpw * p.tgroups * p.ctiles > 1024))
        return hipErrorInvalidValue;
    occupancy_kernel<<<(p.nchunks + p.cpw - 1) / p.cpw, 256, 0, stream>>>(p);
    return hipGetLastError();
}

hipError_t launch_splitk_reduce(const float* part, float* dw, int nsplit, int K, int RS, int C, int krsc,
                                hipStream_t stream)
{
    const int64_t n4 = (int64_t)K * RS * C / 4;
    // G threads per output (each summing a consecutive 1/G of the splits),
    // G the smallest power of two that gives about 2^19 threads (every CU
    // full), at most 16 and at most nsplit
    int G = 1;
    while (G < 16 && 2 * G <= nsplit && n4 * G < (1 << 19)) G *= 2;
    const unsigned blocks = (unsigned)((n4 * G + 255) / 256);
    switch (G) {
    case 1: splitk_reduce_kernel<1><<<blocks, 256, 0, stream>>>(part, dw, nsplit, K, RS, C, krsc); break;
    case 2: splitk_reduce_kernel<2><<<blocks, 256, 0, stream>>>(part, dw, nsplit, K, RS, C, krsc); break;
    case 4: splitk_reduce_kernel<4><<<blocks, 256, 0, stream>>>(part, dw, nsplit, K, RS, C, krsc); break;
    case 8: splitk_reduce_kernel<8><<<blocks, 256, 0, stream>>>(part, dw, nsplit, K, RS, C, krsc); break;
    default: splitk_reduce_kernel<16><<<blocks, 256, 0, stream>>>(part, dw, nsplit, K, RS, C, krsc); break;
    }
    return hipGetLastError();
}

}  // namespace cbw
