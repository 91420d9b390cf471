// Row-window data gradient for 3 x 3, stride-1 layers with 64 input and 64
// output channels (bf16, NHWC), the narrow layers at the largest images
// (VGG-16 conv1_2, the 3 x 3 layers of ResNet bottlenecks at 56 x 56).
//
// Output sparsity (Sec. III-B) and the backward-pass phase of Sec. IV-B:
//
//   dX[n, h, w, c] = x_mask ? sum_{r, s, k} W[k, r, s, c] * dY[n, h + ph - r, w + pw - s, k] : 0
//
// The tiled GEMM walks one (tap, 64-channel) step at a time for these
// layers: each step copies a 512-pixel dY tile for 64 multiply-adds per
// element, so copies, address arithmetic and the per-step barrier dominate.
// Here a workgroup owns a strip of consecutive output rows (one segment of
// up to 224 columns) and walks it one output row per step.  The three dY
// rows an output row needs sit in LDS in a ring of five, each copied once
// with its halo columns; consecutive output rows of an image share two of
// them, so a step copies one new dY row (two steps ahead) and reads all nine
// taps from the ring: the tap shift s is an offset of the LDS row at which
// the fragments are read.  The filters (9 x 64 x 64) stay in registers for
// the whole kernel, one channel half per wave.
//
// GEMM view per step: M = c (A = filters, registers), N = output columns w
// (B = shifted dY rows, LDS), reduction = (r, s, k).  Masked calls stage the
// row's footprint words next to its dY copies, zero the dead outputs in the
// epilogue and skip the matrix work of a row whose footprint is empty (all
// outputs +0.0; counted as not computed).
#include <hip/hip_ext.h>

#include "common.hpp"
#include "kernels.hpp"

namespace cbw {
namespace {

constexpr int DR_NT = 512;                 // 8 waves: 2 channel halves x 4 column groups
constexpr int DR_WT = 224;                 // output columns per segment
constexpr int DR_ROWS = 240;               // LDS rows (dY columns) per plane: DR_WT + 2 halo, whole copy groups
constexpr int DR_PLANE = DR_ROWS * 64;     // one plane: 32 output channels k of every column
constexpr int DR_SLOT = 2 * DR_PLANE;      // one dY row segment (both k halves)
constexpr int DR_SLOTS = 5;                // ring: the 3 rows in use and the next two steps' new rows
constexpr int DR_MSLOT = 2048;             // footprint of one output row segment: 8 bytes per pixel
constexpr int DR_MSLOTS = 3;               // this step's and the next two
constexpr int DR_MW = DR_WT * 8 / 256;     // word copies (256 bytes each) per footprint row
constexpr int DR_NU = 2 * DR_ROWS / 16;    // copy instructions per dY row (16 LDS rows of 64 bytes each)
constexpr int DR_UPW = (DR_NU + 7) / 8;    // per wave
static_assert(DR_ROWS % 16 == 0 && DR_ROWS >= DR_WT + 2 && DR_PLANE < 65536, "row-window shape");
static_assert(DR_WT * 8 <= DR_MSLOT && DR_WT * 8 % 256 == 0 && DR_MW <= 8, "footprint slot");

// Planes of 64-byte rows: a 16-byte chunk j of row i sits at physical chunk
// (j + i / 4) mod 4.  A fragment read takes 16 lanes per cycle, sixteen
// consecutive rows at one logical chunk: rows i and i + 4m land in the same
// quarter of the banks (64 bytes = 16 banks per row) and the four of them
// at four different chunks, so the cycle covers all 64 banks.
__device__ __forceinline__ int dr_chunk(int row, int j) { return (j + (row >> 2)) & 3; }

// Ring slot of dY row p (p >= -16): (p + 20) mod 5 by a multiply and shift.
__device__ __forceinline__ int dr_slot(int p)
{
    static_assert(DR_SLOTS == 5, "the slot formula divides by 5");
    const uint32_t x = (uint32_t)(p + 20);
    return (int)(x - ((x * 52429u) >> 18) * 5u);
}

// NBW: 16-column blocks per wave at most; MASKED: x_mask applied.
template <int NBW, bool MASKED>
__global__ __launch_bounds__(DR_NT) void bwd_data_rows_kernel(DataRowsParams p)
{
    static_assert(NBW >= 1 && NBW <= 4, "column blocks per wave");
    __shared__ __attribute__((aligned(1024))) char Ys[DR_SLOTS * DR_SLOT];
    __shared__ __attribute__((aligned(1024))) char Ms[MASKED ? DR_MSLOTS * DR_MSLOT : 16];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int cw = wave & 1, wg = wave >> 1;          // channel half, column group
    const int g = lane >> 4, col = lane & 15;          // k group of a fragment, column of a block

    const int t = xcd_remap(blockIdx.x, gridDim.x);
    const int seg = t % p.nseg, strip = t / p.nseg;
    const int w0 = seg * DR_WT;
    const int wn = min(DR_WT, p.W - w0);               // valid columns of the segment
    const int row_begin = strip * p.rows_per_strip;
    const int row_end = min(row_begin + p.rows_per_strip, p.nrows);

    // this wave's column blocks [b0, b0 + cnt) of the segment's nwb
    const int nwb = (wn + 15) >> 4;
    const int nb_base = nwb >> 2, nb_rem = nwb & 3;
    const int cnt = nb_base + (wg < nb_rem ? 1 : 0);
    const int b0 = wg * nb_base + min(wg, nb_rem);

    // Filters, per wave: channels 32 cw .. + 31 (two 16-channel blocks), all
    // nine taps and both 32-channel halves of k, as MFMA A fragments (lane:
    // channel col of the block, k = 32 kc + 8 g .. + 7).  wt is [tap][c][k].
    uint4 afr[9][2][2];
    {
        const __amdgpu_buffer_rsrc_t rw = make_rsrc(p.wt, p.wt_bytes);
#pragma unroll
        for (int tap = 0; tap < 9; ++tap)
#pragma unroll
            for (int cb = 0; cb < 2; ++cb)
#pragma unroll
                for (int kc = 0; kc < 2; ++kc) {
                    const int c = 32 * cw + 16 * cb + col;
                    afr[tap][cb][kc] = buf_load16(rw, (uint32_t)(((tap * 64 + c) * 64 + kc * 32 + 8 * g) * 2));
                }
    }

    // B fragment offsets in a ring slot: output column block j, tap column
    // s; LDS row i = 16 (b0 + j) + col + 2 - s holds dY column
    // w0 + pw - 2 + i.  The k half adds DR_PLANE (an instruction offset).
    int boff[3][NBW];
#pragma unroll
    for (int s = 0; s < 3; ++s)
#pragma unroll
        for (int j = 0; j < NBW; ++j) {
            const int i = 16 * (b0 + j) + col + 2 - s;
            boff[s][j] = i * 64 + 16 * dr_chunk(i, g);
        }

    // Copies of a dY row segment: instruction u writes LDS bytes
    // [1024 u, 1024 u + 1024) of the slot, i.e. plane u / 15, rows
    // 16 (u % 15) + l / 4 at physical chunk l % 4 for lane l.
    const u32x4_t rs_dy = make_rsrc_words(p.dy, p.dy_bytes);
    uint32_t ylane[DR_UPW];
#pragma unroll
    for (int m = 0; m < DR_UPW; ++m) {
        const int u = wave + 8 * m;
        const int kc = u / (DR_ROWS / 16), tg = u - kc * (DR_ROWS / 16);
        const int i = 16 * tg + (lane >> 2), pc = lane & 3;
        const int j = (pc - (i >> 2)) & 3;             // logical chunk stored at physical chunk pc
        const int q = w0 + p.pad_w - 2 + i;
        ylane[m] = (u < DR_NU && q >= 0 && q < p.Q) ? (uint32_t)((q * 64 + kc * 32 + j * 8) * 2) : kOOB;
    }
    auto copy_y = [&](int n, int pp) -> int {          // dY row (n, pp) into its ring slot
        if (pp < 0 || pp >= p.P) return 0;             // rows outside the image are never read
        const uint32_t base = (uint32_t)(n * p.P + pp) * (uint32_t)(p.Q * 128);
        const uint32_t lds = lds_addr(Ys) + (uint32_t)(dr_slot(pp) * DR_SLOT);
        int issued = 0;
#pragma unroll
        for (int m = 0; m < DR_UPW; ++m) {
            const int u = wave + 8 * m;
            if (u < DR_NU) {
                buf_load16_lds(rs_dy, ylane[m] == kOOB ? kOOB : base + ylane[m], lds + 1024u * u);
                ++issued;
            }
        }
        return issued;
    };
    const u32x4_t rs_m = make_rsrc_words(p.mask, p.mask_bytes);
    auto copy_m = [&](int row) -> int {                // footprint of output row `row`: 4 bytes per lane
        if (!MASKED || wave >= DR_MW) return 0;        // (waves 0 .. DR_MW - 1, one word copy each)
        const uint32_t byte = 256u * wave + 4u * lane;
        const uint32_t off = byte < (uint32_t)(wn * 8) ? (uint32_t)(row * p.W + w0) * 8u + byte : kOOB;
        buf_load4_lds(rs_m, off, lds_addr(Ms) + (uint32_t)((row % DR_MSLOTS) * DR_MSLOT) + 256u * wave);
        return 1;
    };
    auto image = [&](int row) { return (int)fdiv((uint32_t)row, p.div_h); };
    auto follows = [&](int a, int b) { return b == a + 1 && image(a) == image(b); };
    auto all_rows = [&](int row) {                     // the three dY rows of output row `row`
        const int n = image(row), h = row - n * p.H;
#pragma unroll
        for (int r = 0; r < 3; ++r) copy_y(n, h + p.pad_h - r);
    };
    auto new_row = [&](int row) -> int {               // the dY row the window gains at `row`
        const int n = image(row), h = row - n * p.H;
        return copy_y(n, h + p.pad_h);
    };

    floatx4 acc[2][NBW];
#pragma unroll
    for (int j = 0; j < NBW; ++j) acc[0][j] = acc[1][j] = floatx4{0.f, 0.f, 0.f, 0.f};
    uint2 outv[2][NBW];                                // the previous row's outputs, stored one step later
    int computed = 0;                                  // pixels of the rows whose matrix work ran

    auto compute = [&](int row) {
        const int n = image(row), h = row - n * p.H;
#pragma unroll
        for (int r = 0; r < 3; ++r) {
            const int pp = h + p.pad_h - r;
            if (pp >= 0 && pp < p.P) {                 // uniform
                const char* yb = Ys + dr_slot(pp) * DR_SLOT;
#pragma unroll
                for (int s = 0; s < 3; ++s)
#pragma unroll
                    for (int kc = 0; kc < 2; ++kc)
#pragma unroll
                        for (int j = 0; j < NBW; ++j) {
                            if (j < cnt) {             // uniform; indices stay compile-time constants
                                const uint4 fb = *reinterpret_cast<const uint4*>(yb + boff[s][j] + kc * DR_PLANE);
                                acc[0][j] = mfma_chunk(acc[0][j], afr[3 * r + s][0][kc], fb, uint16_t{});
                                acc[1][j] = mfma_chunk(acc[1][j], afr[3 * r + s][1][kc], fb, uint16_t{});
                            }
                        }
            }
        }
    };

    // One output row: footprint words, the matrix work unless the row is
    // dead, then the outputs rounded, masked and held for the next step.
    auto step = [&](int row) {
        uint32_t mw[NBW];
        bool live = true;
        if (MASKED) {
            const char* mrow = Ms + (row % DR_MSLOTS) * DR_MSLOT;
#pragma unroll
            for (int j = 0; j < NBW; ++j) {
                const int px = 16 * (b0 + j) + col;
                mw[j] = (j < cnt && px < wn) ? *reinterpret_cast<const uint32_t*>(mrow + px * 8 + cw * 4) : 0u;
            }
            if (p.skip) {
                // the whole segment's footprint, read by every wave alike
                const uint4* mv = reinterpret_cast<const uint4*>(mrow);
                uint32_t any = 0;
#pragma unroll
                for (int v = 0; v < DR_MSLOT / 16 / 64; ++v) {
                    const int idx = lane + 64 * v;   // pixels 2 idx and 2 idx + 1
                    if (2 * idx < wn) {
                        const uint4 x = mv[idx];
                        any |= x.x | x.y;
                        if (2 * idx + 1 < wn) any |= x.z | x.w;
                    }
                }
                live = __ballot(any != 0u) != 0ull;
            }
        }
        if (live) {
            compute(row);
            computed += wn;
        }
#pragma unroll
        for (int j = 0; j < NBW; ++j) {
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) {
                const floatx4 v = acc[cb][j];
                uint32_t lo = pack_bf16x2(v.x, v.y), hi = pack_bf16x2(v.z, v.w);
                if (MASKED) {
                    const uint32_t keep = mw[j] >> (16 * cb + 4 * g);
                    lo &= ((0u - (keep & 1u)) & 0xffffu) | ((0u - ((keep >> 1) & 1u)) & 0xffff0000u);
                    hi &= ((0u - ((keep >> 2) & 1u)) & 0xffffu) | ((0u - ((keep >> 3) & 1u)) & 0xffff0000u);
                }
                outv[cb][j] = make_uint2(lo, hi);
                acc[cb][j] = floatx4{0.f, 0.f, 0.f, 0.f};
            }
        }
    };
    const __amdgpu_buffer_rsrc_t rs_dx = make_rsrc(p.dx, p.dx_bytes);
    auto store = [&](int row) {                        // outputs of `row`: 4 channels of one pixel per lane
#pragma unroll
        for (int j = 0; j < NBW; ++j) {
            if (j < cnt) {
                const int w = 16 * (b0 + j) + col;
                const uint32_t base = (uint32_t)(((row * p.W + w0 + w) * 64 + 32 * cw + 4 * g) * 2);
#pragma unroll
                for (int cb = 0; cb < 2; ++cb) {
                    const uint32_t off = w < wn ? base + 32u * cb : kOOB;
                    __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, outv[cb][j]), rs_dx, off, 0, 0);
                }
            }
        }
    };

    // Pipeline over the strip's rows: at step i the copies of step i + 2 are
    // issued (its new dY row when rows i .. i + 2 are consecutive rows of one
    // image, and its footprint) and the outputs of step i - 1 are stored
    // before them; the wait at the end of step i leaves only the copies just
    // issued in flight (stores issued before them have completed by then, as
    // have the older copies, which land in issue order).  A row that starts a
    // new image has its three dY rows loaded after the step before it.
    int ra = row_begin;
    if (ra < row_end) {
        all_rows(ra);
        copy_m(ra);
        if (ra + 1 < row_end) {
            if (follows(ra, ra + 1)) new_row(ra + 1);
            copy_m(ra + 1);
        }
    }
    wait_vmem();
    __syncthreads();
    for (; ra < row_end; ++ra) {
        const int rb = ra + 1, rc = ra + 2;
        if (ra > row_begin) store(ra - 1);
        int issued = 0;
        if (rc < row_end) {
            if (follows(ra, rb) && follows(rb, rc)) issued += new_row(rc);
            issued += copy_m(rc);
        }
        step(ra);
        wait_vmem_upto(issued);
        __syncthreads();
        if (rb < row_end && !follows(ra, rb)) {
            all_rows(rb);
            if (rc < row_end && follows(rb, rc)) new_row(rc);
            wait_vmem();
            __syncthreads();
        }
    }
    if (row_end > row_begin) store(row_end - 1);
    if (tid == 0) p.row_counts[blockIdx.x] = computed;
}

template <int NBW>
hipError_t launch_nbw(const DataRowsParams& p, int grid, hipStream_t stream, const ProfEvents& ev)
{
    if (p.mask)
        hipExtLaunchKernelGGL(bwd_data_rows_kernel<NBW, true>, dim3(grid), dim3(DR_NT), 0, stream, ev.start, ev.stop,
                              0, p);
    else
        hipExtLaunchKernelGGL(bwd_data_rows_kernel<NBW, false>, dim3(grid), dim3(DR_NT), 0, stream, ev.start,
                              ev.stop, 0, p);
    return hipGetLastError();
}

}  // namespace

int data_rows_segment() { return DR_WT; }

hipError_t launch_bwd_data_rows(const DataRowsParams& p, int grid, int nbw, hipStream_t stream, const ProfEvents& ev)
{
    // the grid must cover every (segment, strip) pair exactly as planned
    const int nstrips = (p.nrows + p.rows_per_strip - 1) / p.rows_per_strip;
    if (p.nseg != (p.W + DR_WT - 1) / DR_WT || grid != nstrips * p.nseg || p.nrows != p.N * p.H)
        return hipErrorInvalidValue;
    if (nbw < (((p.W < DR_WT ? p.W : DR_WT) + 15) / 16 + 3) / 4) return hipErrorInvalidValue;
    switch (nbw) {
    case 1: return launch_nbw<1>(p, grid, stream, ev);
    case 2: return launch_nbw<2>(p, grid, stream, ev);
    case 3: return launch_nbw<3>(p, grid, stream, ev);
    case 4: return launch_nbw<4>(p, grid, stream, ev);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace cbw
