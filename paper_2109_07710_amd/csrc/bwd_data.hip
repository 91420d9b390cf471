// Data gradient as an implicit GEMM on the gfx950 matrix cores.
//
//   dX[pix, c] = sum_{tap=(r,s)} sum_k  Wt[tap][c][k] * dY[src(pix, tap)][k]
//
// (Sec. IV-B: the backward pass is the forward convolution with M and C
// interchanged.)  GEMM view: M = channels c (A = transformed filters, k
// contiguous), N = pixels (B = dY rows, k contiguous in NHWC), reduction =
// (tap, k).  The output tile is therefore D[c][pix]; every lane ends up with
// four consecutive channels of one pixel, which it stores as one vector.
//
// Modes
//   dense   : every pixel is a row; plain store.
//   select  : every pixel is a row; the epilogue keeps an output only where
//             its footprint bit is set and writes the +0.0 pattern elsewhere
//             (never acc * bit, which would give -0.0 for a negative acc).
//   gather  : the rows of channel group g are the compacted ascending list of
//             pixels live in that group (output-bitmap-driven address
//             generation, Sec. IV-B); the epilogue applies the per-element
//             select.  Rows dead for the whole group were zero-filled by the
//             compaction kernel and are never touched here.
#include "common.hpp"
#include "kernels.hpp"

namespace cbw {

namespace {

constexpr int BM = 128;         // channels per tile (= compaction group width)
constexpr int BN = 128;         // pixels per tile
constexpr int NT = 256;         // threads: 4 waves in a 2 x 2 arrangement
constexpr int CH = 8;           // 16-byte chunks of reduction per row per step
constexpr int LDSROW = CH + 1;  // padded row length in chunks (144 bytes)

template <typename T, int MODE>
__global__ __launch_bounds__(NT, 2) void bwd_data_kernel(DataParams p)
{
    constexpr int E = Elem<T>::E;
    constexpr int BK = CH * E;  // reduction elements per step

    __shared__ uint4 As[BM * LDSROW];
    __shared__ uint4 Bs[BN * LDSROW];
    __shared__ int pix_s[BN];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;

    const int t = xcd_remap(blockIdx.x, gridDim.x);
    const int ptile = t / p.ctiles;
    const int ctile = t - ptile * p.ctiles;
    const int c0 = ctile * BM;
    const int row0 = ptile * BN;

    int nrows = p.npix;
    if (MODE == MODE_GATHER) nrows = p.counts[ctile];
    if (row0 >= nrows) return;  // uniform across the workgroup

    if (tid < BN) {
        const int r = row0 + tid;
        int pix = -1;
        if (r < nrows) pix = (MODE == MODE_GATHER) ? p.lists[(int64_t)ctile * p.npix + r] : r;
        pix_s[tid] = pix;
    }
    __syncthreads();

    // Each thread loads rows (tid / CH) + 32 j, j = 0..3, chunk tid % CH, of
    // both operands.  Pixel coordinates of its four B rows:
    const int lrow = tid / CH, lch = tid % CH;
    int bn_[4], bh_[4], bw_[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int pix = pix_s[lrow + 32 * j];
        if (pix >= 0) {
            const uint32_t nh = fdiv((uint32_t)pix, p.div_w);
            bw_[j] = pix - (int)nh * p.W;
            const uint32_t n = fdiv(nh, p.div_h);
            bh_[j] = (int)nh - (int)n * p.H;
            bn_[j] = (int)n;
        } else {
            bn_[j] = -1; bh_[j] = 0; bw_[j] = 0;
        }
    }

    floatx4 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

    const int kchunks = (p.K + BK - 1) / BK;
    const int nsteps = p.R * p.S * kchunks;
    const T* __restrict__ wt = reinterpret_cast<const T*>(p.wt);
    const T* __restrict__ dy = reinterpret_cast<const T*>(p.dy);

    uint4 ra[4], rb[4];
    int src[4];  // element offset of the B rows' dY pixel for the current tap, -1 = none
    int cur_tap = -1;

    auto set_tap = [&](int tap) {
        const int r = tap / p.S, s = tap - (tap / p.S) * p.S;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            src[j] = -1;
            if (bn_[j] < 0) continue;
            int hh = bh_[j] + p.pad_h - r, ww = bw_[j] + p.pad_w - s;
            if (hh < 0 || ww < 0) continue;
            int pp, qq;
            if (p.stride_h == 1) { pp = hh; } else { if (hh % p.stride_h) continue; pp = hh / p.stride_h; }
            if (p.stride_w == 1) { qq = ww; } else { if (ww % p.stride_w) continue; qq = ww / p.stride_w; }
            if (pp >= p.P || qq >= p.Q) continue;
            src[j] = ((bn_[j] * p.P + pp) * p.Q + qq) * p.K;
        }
    };

    auto load = [&](int step) {
        const int tap = step / kchunks;
        const int k0 = (step - tap * kchunks) * BK + lch * E;
        if (tap != cur_tap) { set_tap(tap); cur_tap = tap; }
        const bool kin = k0 < p.K;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int c = c0 + lrow + 32 * j;
            ra[j] = make_uint4(0, 0, 0, 0);
            if (kin && c < p.C)
                ra[j] = *reinterpret_cast<const uint4*>(wt + ((int64_t)(tap * p.C + c) * p.K + k0));
            rb[j] = make_uint4(0, 0, 0, 0);
            if (kin && src[j] >= 0)
                rb[j] = *reinterpret_cast<const uint4*>(dy + ((int64_t)src[j] + k0));
        }
    };

    load(0);
    for (int step = 0; step < nsteps; ++step) {
        __syncthreads();
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            As[(lrow + 32 * j) * LDSROW + lch] = ra[j];
            Bs[(lrow + 32 * j) * LDSROW + lch] = rb[j];
        }
        __syncthreads();
        if (step + 1 < nsteps) load(step + 1);
#pragma unroll
        for (int kc = 0; kc < CH / 4; ++kc) {
            const int ch = kc * 4 + (lane >> 4);
            uint4 fa[4], fb[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) fa[i] = As[(wm * 64 + i * 16 + (lane & 15)) * LDSROW + ch];
#pragma unroll
            for (int j = 0; j < 4; ++j) fb[j] = Bs[(wn * 64 + j * 16 + (lane & 15)) * LDSROW + ch];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = mfma_chunk(acc[i][j], fa[i], fb[j], T{});
        }
    }

    // Epilogue: lane holds channels c0 + wm*64 + i*16 + 4*(lane/16) + v of
    // pixel row wn*64 + j*16 + lane%16.
    T* __restrict__ dx = reinterpret_cast<T*>(p.dx);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int pix = pix_s[wn * 64 + j * 16 + (lane & 15)];
        if (pix < 0) continue;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int c = c0 + wm * 64 + i * 16 + 4 * (lane >> 4);
            if (c >= p.C) continue;
            const int64_t o = (int64_t)pix * p.C + c;
            floatx4 v = acc[i][j];
            uint32_t keep = 0xfu;
            if (MODE != MODE_DENSE) keep = (p.mask[o >> 5] >> (o & 31)) & 0xfu;
            if constexpr (sizeof(T) == 2) {
                uint32_t h0 = (keep & 1u) ? f32_to_bf16_rne(v.x) : 0u;
                uint32_t h1 = (keep & 2u) ? f32_to_bf16_rne(v.y) : 0u;
                uint32_t h2 = (keep & 4u) ? f32_to_bf16_rne(v.z) : 0u;
                uint32_t h3 = (keep & 8u) ? f32_to_bf16_rne(v.w) : 0u;
                *reinterpret_cast<uint2*>(dx + o) = make_uint2(h0 | (h1 << 16), h2 | (h3 << 16));
            } else {
                uint4 u;
                u.x = (keep & 1u) ? __float_as_uint(v.x) : 0u;
                u.y = (keep & 2u) ? __float_as_uint(v.y) : 0u;
                u.z = (keep & 4u) ? __float_as_uint(v.z) : 0u;
                u.w = (keep & 8u) ? __float_as_uint(v.w) : 0u;
                *reinterpret_cast<uint4*>(dx + o) = u;
            }
        }
    }
}

// Wt[tap][c][k] = W[k][tap][c] (KRSC) or W[k][c][tap] (KCRS).  Also stamps the
// workspace header with the call's mode.
template <typename T>
__global__ void transform_filters_kernel(const T* __restrict__ w, T* __restrict__ wt, int K, int C, int RS,
                                         int krsc, int* header, int mode)
{
    const int64_t total = (int64_t)K * C * RS;
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i == 0 && header) header[0] = mode;
    if (i >= total) return;
    const int k = (int)(i % K);
    const int64_t tc = i / K;
    const int c = (int)(tc % C);
    const int tap = (int)(tc / C);
    const int64_t srci = krsc ? ((int64_t)k * RS + tap) * C + c : ((int64_t)k * C + c) * RS + tap;
    wt[i] = w[srci];
}

}  // namespace

int data_tile_channels() { return BM; }
int data_tile_pixels() { return BN; }

hipError_t launch_transform_filters(int dtype, const void* w, void* wt, int K, int C, int RS, int krsc,
                                    int* header, int mode, hipStream_t stream)
{
    const int64_t total = (int64_t)K * C * RS;
    const int blocks = (int)((total + 255) / 256);
    if (dtype == 1)
        transform_filters_kernel<uint16_t><<<blocks, 256, 0, stream>>>(
            (const uint16_t*)w, (uint16_t*)wt, K, C, RS, krsc, header, mode);
    else
        transform_filters_kernel<float><<<blocks, 256, 0, stream>>>(
            (const float*)w, (float*)wt, K, C, RS, krsc, header, mode);
    return hipGetLastError();
}

hipError_t launch_bwd_data(int dtype, int mode, const DataParams& p, hipStream_t stream)
{
    const int ptiles = (p.npix + BN - 1) / BN;
    const int nb = ptiles * p.ctiles;
    if (nb <= 0) return hipSuccess;
#define CBW_LAUNCH(T, M) bwd_data_kernel<T, M><<<nb, NT, 0, stream>>>(p)
    if (dtype == 1) {
        if (mode == MODE_DENSE) CBW_LAUNCH(uint16_t, MODE_DENSE);
        else if (mode == MODE_SELECT) CBW_LAUNCH(uint16_t, MODE_SELECT);
        else CBW_LAUNCH(uint16_t, MODE_GATHER);
    } else {
        if (mode == MODE_DENSE) CBW_LAUNCH(float, MODE_DENSE);
        else if (mode == MODE_SELECT) CBW_LAUNCH(float, MODE_SELECT);
        else CBW_LAUNCH(float, MODE_GATHER);
    }
#undef CBW_LAUNCH
    return hipGetLastError();
}

}  // namespace cbw
