// Pointwise data gradient for 1 x 1, stride-1, unpadded layers (bf16, NHWC)
// with C, K in {64, 128, 256} and C * K <= 16384: the 1 x 1 reductions and
// expansions of ResNet bottlenecks.
//
// Output sparsity (Sec. III-B) with a single filter tap:
//
//   dX[pix, c] = x_mask ? sum_k W[k, c] * dY[pix, k] : 0
//
// These layers move C + K values per pixel for 2 C K flops, far below the
// MFMA/HBM balance point: the tiled GEMM's staging, barriers and one-step
// tiles leave them at a third of the bandwidth.  Here every wave streams
// its own run of 16-pixel blocks with no LDS traffic and no barrier after
// the start: the filters sit in registers for the whole kernel (staged once
// per workgroup through LDS), dY fragments and footprint words are read
// straight from global memory into a ring of registers, two blocks ahead
// (one when K = 256), and each block's outputs are masked, rounded and
// stored as soon as its MFMAs end, through a per-wave LDS stage that turns
// the fragments' 8-byte pieces of 16 rows into whole 1 KB runs.
//
// GEMM view per block: M = c (A = filters, registers), N = 16 pixels (B =
// dY rows, 8 consecutive k per lane), reduction = k.  Masked calls skip the
// MFMAs of a block whose footprint is empty (every output +0.0) and count
// the pixels of the blocks computed.

#include "common.hpp"
#include "kernels.hpp"

namespace cbw {
namespace {

constexpr int PW_NT = 256;   // 4 waves

template <int C, int K, bool MASKED>
__global__ __launch_bounds__(PW_NT, 2) void bwd_data_pw_kernel(DataPwParams p)
{
    constexpr int CB = C / 16;    // 16-channel blocks (A fragments per k step, accumulators)
    constexpr int KC = K / 32;    // 32-k steps (B fragments per block)
    constexpr int MW = C / 32;    // footprint words per pixel
    static_assert(CB * KC * 4 <= 128, "filters in at most 128 registers");
    // blocks in flight: three, or two when a block's dY fragments take 32
    // registers (K = 256), which keeps the kernel within 256 registers
    constexpr int RD = KC >= 8 ? 2 : 3;
    __shared__ uint4 Ws[C * K / 8];   // filters [c][k], 16-byte vectors of 8 k
    // footprint nibble (4 channels) -> the two output words' masks, 16 bits
    // per channel
    __shared__ uint2 mtab[16];
    // each wave's block of outputs on its way out: 16 pixel rows of C bf16,
    // padded by 16 bytes (the fragment writes of 16 rows then spread over
    // the banks), read back as 16-byte row pieces for whole-line stores
    constexpr int SROW = 2 * C + 16;
    __shared__ __attribute__((aligned(16))) char Os[PW_NT / 64][16 * SROW];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, col = lane & 15;

    // this wave's blocks [b_begin, b_end) of 16 pixels
    const int gw = blockIdx.x * (PW_NT / 64) + wave;
    const int b_begin = min(p.nblk, gw * p.bpw);
    const int b_end = min(p.nblk, b_begin + p.bpw);

    const __amdgpu_buffer_rsrc_t rs_dy = make_rsrc(p.dy, p.dy_bytes);
    const __amdgpu_buffer_rsrc_t rs_dx = make_rsrc(p.dx, p.dx_bytes);
    const __amdgpu_buffer_rsrc_t rs_m = make_rsrc(p.mask, p.mask_bytes);

    // operands of block b: the lane's dY vectors (pixel 16 b + col) and, when
    // masked, that pixel's footprint words (past the last pixel: zeros)
    struct Blk {
        uint4 y[KC];
        uint32_t m[MASKED ? MW : 1];
    };
    auto fetch = [&](int b, Blk& o) {
        const uint32_t pix = (uint32_t)(16 * b + col);
#pragma unroll
        for (int kc = 0; kc < KC; ++kc) o.y[kc] = buf_load16(rs_dy, (pix * K + 32 * kc + 8 * g) * 2u);
        if constexpr (MASKED) {
            const uint32_t mb = pix * (uint32_t)(C / 8);
            if constexpr (MW >= 4) {
#pragma unroll
                for (int w = 0; w < MW; w += 4) {
                    const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(rs_m, mb + 4u * w, 0, 0);
                    o.m[w] = v.x; o.m[w + 1] = v.y; o.m[w + 2] = v.z; o.m[w + 3] = v.w;
                }
            } else {
                const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(rs_m, mb, 0, 0);
                o.m[0] = v.x; o.m[1] = v.y;
            }
        }
    };

    // a ring of RD blocks of registers; the copies of the first RD - 1
    // blocks go out before the filters are staged, so their latency
    // overlaps the staging's
    Blk bk[RD];
#pragma unroll
    for (int j = 0; j + 1 < RD; ++j)
        if (b_begin + j < b_end) fetch(b_begin + j, bk[j]);

    // the filters, once per workgroup: 16-byte copies into LDS, then each
    // wave's A fragments (lane: channel 16 cb + col, k = 32 kc + 8 g .. + 7)
    {
        const uint4* src = static_cast<const uint4*>(p.wt);
#pragma unroll
        for (int i = tid; i < C * K / 8; i += PW_NT) Ws[i] = src[i];
        if (tid < 16) {
            auto half = [](int b) { return b ? 0xffffu : 0u; };
            mtab[tid] = make_uint2(half(tid & 1) | (half(tid & 2) << 16), half(tid & 4) | (half(tid & 8) << 16));
        }
    }
    __syncthreads();
    uint4 afr[CB][KC];
#pragma unroll
    for (int cb = 0; cb < CB; ++cb)
#pragma unroll
        for (int kc = 0; kc < KC; ++kc) afr[cb][kc] = Ws[((16 * cb + col) * K + 32 * kc + 8 * g) / 8];

    int computed = 0;
    // the block's outputs in groups of at most 8 channel blocks (128
    // channels), which bounds the accumulators to 32 registers
    constexpr int GB = CB < 8 ? CB : 8;
    auto process = [&](int b, const Blk& o) {
        const int pix = 16 * b + col;
        bool live = true;
        if (MASKED && p.skip) {
            uint32_t any = 0;
#pragma unroll
            for (int w = 0; w < MW; ++w) any |= o.m[w];
            live = __ballot(any != 0u) != 0ull;
        }
        if (live) computed += min(16, p.npix - 16 * b);
        (void)pix;
        // lane: channels 16 cb + 4 g .. + 3 of pixel row col, 8 bytes each
        char* const os = Os[wave];
        const int wbase = col * SROW + 8 * g;
#pragma unroll
        for (int c0 = 0; c0 < CB; c0 += GB) {
            floatx4 acc[GB];
#pragma unroll
            for (int i = 0; i < GB; ++i) acc[i] = floatx4{0.f, 0.f, 0.f, 0.f};
            if (live) {
#pragma unroll
                for (int kc = 0; kc < KC; ++kc)
#pragma unroll
                    for (int i = 0; i < GB; ++i) acc[i] = mfma_chunk(acc[i], afr[c0 + i][kc], o.y[kc], uint16_t{});
            }
#pragma unroll
            for (int i = 0; i < GB; ++i) {
                const int cb = c0 + i;
                const floatx4 v = acc[i];
                uint32_t lo = pack_bf16x2(v.x, v.y), hi = pack_bf16x2(v.z, v.w);
                if constexpr (MASKED) {
                    // the footprint bits of the lane's 4 channels, widened
                    // through the table
                    const uint32_t nib = (o.m[(16 * cb) / 32] >> ((16 * cb + 4 * g) & 31)) & 15u;
                    const uint2 km = mtab[nib];
                    lo &= km.x;
                    hi &= km.y;
                }
                *reinterpret_cast<uint2*>(os + wbase + 32 * cb) = make_uint2(lo, hi);
            }
        }
        // the block's rows are consecutive in dX: 16 * 2C bytes, 1 KB per
        // store instruction, lane l at byte 1024 u + 16 l (past the last
        // pixel: offsets at or beyond the tensor's end, dropped)
        __builtin_amdgcn_wave_barrier();
        const uint32_t gbase = (uint32_t)(16 * b) * (uint32_t)(2 * C);
#pragma unroll
        for (int u = 0; u < C / 32; ++u) {
            const int byte = 1024 * u + 16 * lane;
            const int row = byte / (2 * C), off = byte - row * (2 * C);
            const uint4 v = *reinterpret_cast<const uint4*>(os + row * SROW + off);
            __builtin_amdgcn_raw_buffer_store_b128(u32x4{v.x, v.y, v.z, v.w}, rs_dx, gbase + (uint32_t)byte, 0, 0);
        }
        __builtin_amdgcn_wave_barrier();
    };

    // block b + RD - 1 is fetched before block b is processed, into the
    // registers block b - 1 has released
    for (int b = b_begin; b < b_end; b += RD) {
#pragma unroll
        for (int j = 0; j < RD; ++j) {
            if (b + j < b_end) {
                if (b + j + RD - 1 < b_end) fetch(b + j + RD - 1, bk[(j + RD - 1) % RD]);
                process(b + j, bk[j]);
            }
        }
    }

    // the workgroup's computed pixels: the sum over its waves
    __shared__ int wave_counts[PW_NT / 64];
    if (lane == 0) wave_counts[wave] = computed;
    __syncthreads();
    if (tid == 0) {
        int total = 0;
#pragma unroll
        for (int w = 0; w < PW_NT / 64; ++w) total += wave_counts[w];
        p.counts[blockIdx.x] = total;
    }
}

template <int C, int K>
hipError_t launch_ck(const DataPwParams& p, int grid, hipStream_t stream, const ProfEvents& ev)
{
    hipError_t e_launch;
    if (p.mask)
        e_launch = launch_timed(bwd_data_pw_kernel<C, K, true>, dim3(grid), dim3(PW_NT), stream, ev, p);
    else
        e_launch = launch_timed(bwd_data_pw_kernel<C, K, false>, dim3(grid), dim3(PW_NT), stream, ev, p);
    return e_launch;
}

}  // namespace

int data_pw_waves_per_group() { return PW_NT / 64; }

hipError_t launch_bwd_data_pw(const DataPwParams& p, int grid, hipStream_t stream, const ProfEvents& ev)
{
    // every block belongs to exactly one wave of the grid
    const int nblk = (p.npix + 15) / 16;
    if (p.npix <= 0 || p.nblk != nblk || p.bpw <= 0 || (int64_t)grid * (PW_NT / 64) * p.bpw < nblk ||
        (int64_t)(grid - 1) * (PW_NT / 64) * p.bpw >= nblk)
        return hipErrorInvalidValue;
    // every access stays inside the tensors' descriptors
    if ((int64_t)p.npix * p.K * 2 > (int64_t)p.dy_bytes || (int64_t)p.npix * p.C * 2 > (int64_t)p.dx_bytes ||
        (p.mask && ((int64_t)p.npix * p.C + 31) / 32 * 4 > (int64_t)p.mask_bytes))
        return hipErrorInvalidValue;
    const int ck = p.C * 1000 + p.K;
    switch (ck) {
    case 64064: return launch_ck<64, 64>(p, grid, stream, ev);
    case 64128: return launch_ck<64, 128>(p, grid, stream, ev);
    case 64256: return launch_ck<64, 256>(p, grid, stream, ev);
    case 128064: return launch_ck<128, 64>(p, grid, stream, ev);
    case 128128: return launch_ck<128, 128>(p, grid, stream, ev);
    case 256064: return launch_ck<256, 64>(p, grid, stream, ev);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace cbw
