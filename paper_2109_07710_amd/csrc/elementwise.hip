// Data gradient with per-element input and output sparsity on the vector
// ALUs: the software form of the paper's non-zero indexing (Sec. III-B input
// and output sparsity; Sec. IV-B, each lane walks only the non-zero offsets
// of its gradient column and skips outputs the ReLU killed).
//
//   dX[pix, c] = mask[pix, c] ? sum_{tap} sum_{k : dY[src(pix, tap), k] != 0}
//                                    dY[src, k] * W[k][tap][c]  : +0.0
//
// One wave per output pixel; lane l owns channels [l*CPL, l*CPL + CPL) with
// CPL = C / 64.  A pixel whose footprint row is entirely dead is written as
// +0.0 and costs nothing else (output sparsity at pixel granularity; single
// dead channels are zeroed by the select, as in the matrix-core path).  For
// every filter tap the wave ballots the non-zeros of the source dY row (512 k
// per pass) into a wave-local list in LDS and then walks only that list: per
// entry one 64-lane load of the filter row W[k][r][s][:] (KRSC, contiguous
// over c) and CPL multiply-adds per lane, the loads of 8 or 16 entries issued
// before their multiply-adds.  The entries of successive taps accumulate in
// the list (tagged with their tap) until it could overflow, so at low density
// the filter loads of all taps of a pixel share a few round trips; the next
// tap's dY row is loaded while the current one is listed.  Every pixel records the number of
// (tap, k) products it executed (0 for a dead pixel) in the workspace.
//
// The order of summation is fixed by the data (the list's order), so results
// are reproducible.  No barrier is used: the LDS
// list of a wave is written and read by that wave only.
#include <hip/hip_runtime.h>

#include "common.hpp"
#include "kernels.hpp"

namespace cbw {

namespace {

constexpr int EW_WAVES = 4;      // waves (pixels) per workgroup
constexpr int EW_PASS = 512;     // k per list pass (8 per lane)
constexpr int EW_CAP = 1024;     // list capacity per wave (at least one pass)

template <int CPL>
struct Vec;
template <> struct Vec<1> { typedef uint16_t T; };
template <> struct Vec<2> { typedef uint32_t T; };
template <> struct Vec<4> { typedef uint2 T; };
template <> struct Vec<8> { typedef uint4 T; };

template <int CPL>
__device__ __forceinline__ void unpack(const typename Vec<CPL>::T& v, float (&f)[CPL])
{
    if constexpr (CPL == 1) {
        f[0] = __uint_as_float((uint32_t)v << 16);
    } else if constexpr (CPL == 2) {
        f[0] = __uint_as_float(v << 16);
        f[1] = __uint_as_float(v & 0xffff0000u);
    } else if constexpr (CPL == 4) {
        f[0] = __uint_as_float(v.x << 16); f[1] = __uint_as_float(v.x & 0xffff0000u);
        f[2] = __uint_as_float(v.y << 16); f[3] = __uint_as_float(v.y & 0xffff0000u);
    } else {
        f[0] = __uint_as_float(v.x << 16); f[1] = __uint_as_float(v.x & 0xffff0000u);
        f[2] = __uint_as_float(v.y << 16); f[3] = __uint_as_float(v.y & 0xffff0000u);
        f[4] = __uint_as_float(v.z << 16); f[5] = __uint_as_float(v.z & 0xffff0000u);
        f[6] = __uint_as_float(v.w << 16); f[7] = __uint_as_float(v.w & 0xffff0000u);
    }
}

template <int CPL>
__device__ __forceinline__ typename Vec<CPL>::T load_w(__amdgpu_buffer_rsrc_t rs, uint32_t off)
{
    if constexpr (CPL == 1) return (uint16_t)__builtin_amdgcn_raw_buffer_load_b16(rs, off, 0, 0);
    if constexpr (CPL == 2) return __builtin_amdgcn_raw_buffer_load_b32(rs, off, 0, 0);
    if constexpr (CPL == 4) {
        const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(rs, off, 0, 0);
        return make_uint2(v.x, v.y);
    }
    if constexpr (CPL == 8) {
        const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0);
        return make_uint4(v.x, v.y, v.z, v.w);
    }
}

// Store CPL bf16 values (packed in pairs, the first in the low half).
template <int CPL>
__device__ __forceinline__ void store_bf16(__amdgpu_buffer_rsrc_t rs, uint32_t off, const uint32_t (&v)[(CPL + 1) / 2])
{
    if constexpr (CPL == 1) __builtin_amdgcn_raw_buffer_store_b16((uint16_t)(v[0] & 0xffffu), rs, off, 0, 0);
    if constexpr (CPL == 2) __builtin_amdgcn_raw_buffer_store_b32(v[0], rs, off, 0, 0);
    if constexpr (CPL == 4) __builtin_amdgcn_raw_buffer_store_b64(u32x2{v[0], v[1]}, rs, off, 0, 0);
    if constexpr (CPL == 8) __builtin_amdgcn_raw_buffer_store_b128(u32x4{v[0], v[1], v[2], v[3]}, rs, off, 0, 0);
}

template <int CPL>
__global__ __launch_bounds__(EW_WAVES * 64) void elementwise_data_kernel(EwParams p)
{
    // wave-local list of non-zero dY entries: (k << 16) | bf16 bits, and the tap
    __shared__ uint32_t list_s[EW_WAVES][EW_CAP];
    __shared__ uint8_t tap_s[EW_WAVES][EW_CAP];
    __shared__ uint32_t src_s[EW_WAVES][256];        // byte offset of dY[src(tap)][0], kOOB if the tap misses
    constexpr int U = CPL == 8 ? 8 : 16;              // entries whose filter loads are issued together
    const int lane = threadIdx.x & 63;
    const int wv = threadIdx.x >> 6;
    const int pix = xcd_remap(blockIdx.x, gridDim.x) * EW_WAVES + wv;
    if (pix >= p.npix) return;                      // whole wave; no barrier follows
    uint32_t* list = list_s[wv];
    uint8_t* ltap = tap_s[wv];

    const uint32_t nh = fdiv((uint32_t)pix, p.div_w);
    const int w = pix - (int)nh * p.W;
    const uint32_t n = fdiv(nh, p.div_h);
    const int h = (int)nh - (int)n * p.H;

    const __amdgpu_buffer_rsrc_t rs_dx = make_rsrc(p.dx, p.dx_bytes);
    const __amdgpu_buffer_rsrc_t rs_w = make_rsrc(p.w, p.w_bytes);
    const __amdgpu_buffer_rsrc_t rs_dy = make_rsrc(p.dy, p.dy_bytes);
    const int c0 = lane * CPL;                       // first channel of this lane
    const uint32_t dx_off = (uint32_t)(pix * p.C + c0) * 2u;

    // Output sparsity: the footprint bits of this lane's channels, and
    // whether any channel of the pixel is live.
    const int64_t bit0 = (int64_t)pix * p.C + c0;
    const uint32_t keep = (p.mask[bit0 >> 5] >> (bit0 & 31)) & ((1u << CPL) - 1u);
    constexpr int NO = (CPL + 1) / 2;
    if (__ballot(keep != 0) == 0) {
        const uint32_t zero[NO] = {};
        store_bf16<CPL>(rs_dx, dx_off, zero);
        if (lane == 0) p.counts[pix] = 0;
        return;
    }

    // The source row of every filter tap, computed once per pixel by the
    // lanes in parallel: an off-grid or out-of-image tap gets kOOB, reads
    // zeros and lists nothing.
    const int RS = p.R * p.S;
    uint32_t* srcoff = src_s[wv];
    for (int t = lane; t < RS; t += 64) {
        const int r = t / p.S, s = t - r * p.S;
        const int hh = h + p.pad_h - r, ww = w + p.pad_w - s;
        uint32_t o = kOOB;
        if (hh >= 0 && ww >= 0 && hh % p.stride_h == 0 && ww % p.stride_w == 0) {
            const int pp = hh / p.stride_h, qq = ww / p.stride_w;
            if (pp < p.P && qq < p.Q) o = (uint32_t)((((int)n * p.P + pp) * p.Q + qq) * p.K) * 2u;
        }
        srcoff[t] = o;
    }
    __builtin_amdgcn_wave_barrier();
    // Steps are (tap, k pass) pairs; the dY row segment of the next step is
    // loaded while the current one is listed.
    auto row_offset = [&](int tap, int kb) -> uint32_t {
        const uint32_t base = __builtin_amdgcn_readfirstlane(srcoff[tap]);
        const int kl = kb + 8 * lane;
        return (base == kOOB || kl >= p.K) ? kOOB : base + (uint32_t)kl * 2u;
    };

    float acc[CPL];
#pragma unroll
    for (int i = 0; i < CPL; ++i) acc[i] = 0.f;
    int executed = 0;
    const uint32_t k_stride = (uint32_t)(RS * p.C) * 2u;            // bytes between W[k] and W[k+1]
    // walk the list, U entries per round with their filter loads issued together
    auto walk = [&](int cnt) {
        for (int e0 = 0; e0 < cnt; e0 += U) {
            typename Vec<CPL>::T wv_[U];
            float val[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int e = e0 + u;
                const uint32_t kv = __builtin_amdgcn_readfirstlane(e < cnt ? list[e] : 0u);
                const uint32_t tap = __builtin_amdgcn_readfirstlane(e < cnt ? (uint32_t)ltap[e] : 0u);
                val[u] = e < cnt ? __uint_as_float(kv << 16) : 0.f;
                const uint32_t off = e < cnt ? (kv >> 16) * k_stride + (tap * (uint32_t)p.C + (uint32_t)c0) * 2u : kOOB;
                wv_[u] = load_w<CPL>(rs_w, off);
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                float f[CPL];
                unpack<CPL>(wv_[u], f);
#pragma unroll
                for (int i = 0; i < CPL; ++i) acc[i] = __builtin_fmaf(val[u], f[i], acc[i]);
            }
        }
        __builtin_amdgcn_wave_barrier();
    };
    // Entries of successive taps accumulate in the list, which is walked when
    // the next row segment might not fit and once at the end, so that the
    // filter loads of several taps share their round trips.
    int cnt = 0;
    u32x4 yv = __builtin_amdgcn_raw_buffer_load_b128(rs_dy, row_offset(0, 0), 0, 0);
    int tap = 0, kb = 0;
    while (tap < RS) {
        int ntap = tap, nkb = kb + EW_PASS;   // the next step
        if (nkb >= p.K) {
            nkb = 0;
            ++ntap;
        }
        const uint32_t half[4] = {yv.x, yv.y, yv.z, yv.w};
        if (ntap < RS) yv = __builtin_amdgcn_raw_buffer_load_b128(rs_dy, row_offset(ntap, nkb), 0, 0);
        if (cnt + EW_PASS > EW_CAP) {
            walk(cnt);
            cnt = 0;
        }
        // the non-zeros of this row segment: lane l holds k = kb + 8l .. 8l+7
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const uint32_t bits = (half[i >> 1] >> (16 * (i & 1))) & 0xffffu;
            const bool nz = (bits & 0x7fffu) != 0;       // +0.0 and -0.0 are zeros
            const uint64_t m = __ballot(nz);
            const int below = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
            if (nz) {
                list[cnt + below] = ((uint32_t)(kb + 8 * lane + i) << 16) | bits;
                ltap[cnt + below] = (uint8_t)tap;
            }
            const int added = __popcll(m);
            cnt += added;
            executed += added;
        }
        __builtin_amdgcn_wave_barrier();
        tap = ntap;
        kb = nkb;
    }
    walk(cnt);
    if (lane == 0) p.counts[pix] = executed;

    // select (never acc * bit, which would give -0.0) and round to bf16
    float sel[2 * NO];
#pragma unroll
    for (int i = 0; i < 2 * NO; ++i) sel[i] = (i < CPL && ((keep >> i) & 1u)) ? acc[i < CPL ? i : 0] : 0.f;
    uint32_t out[NO];
#pragma unroll
    for (int i = 0; i < NO; ++i) out[i] = pack_bf16x2(sel[2 * i], sel[2 * i + 1]);
    store_bf16<CPL>(rs_dx, dx_off, out);
}

}  // namespace

hipError_t launch_elementwise_data(const EwParams& p, hipStream_t stream)
{
    const int nb = (p.npix + EW_WAVES - 1) / EW_WAVES;
    const dim3 grid(nb), block(EW_WAVES * 64);
    switch (p.C / 64) {
    case 1: elementwise_data_kernel<1><<<grid, block, 0, stream>>>(p); break;
    case 2: elementwise_data_kernel<2><<<grid, block, 0, stream>>>(p); break;
    case 4: elementwise_data_kernel<4><<<grid, block, 0, stream>>>(p); break;
    case 8: elementwise_data_kernel<8><<<grid, block, 0, stream>>>(p); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace cbw
