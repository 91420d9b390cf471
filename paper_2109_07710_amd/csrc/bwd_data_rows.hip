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
// row's footprint words next to its dY copies, zero the dead outputs when
// they are stored, and a wave skips the matrix work of a row when every one
// of its outputs there (its channel half of its columns) is dead: those
// outputs are +0.0 and are counted as not computed.

#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"
#include "tiles.hpp"

namespace cbw {
namespace {

constexpr int DR_NT = 512;                 // 8 waves: 2 channel halves x 4 column groups
constexpr int DR_WT = kDataRowsSegment;    // output columns per segment (at most)
static_assert(DR_WT * 8 <= 256 * 8, "footprint copies: one per wave at most");

// 128-byte rows (one dY column, all 64 k): the 16-byte chunk j of row i sits
// at physical chunk j ^ (i mod 8).  A fragment read covers sixteen
// consecutive rows at one logical chunk, starting at any row (the tap shift
// s moves the start by 0, 1 or 2).  Measured with the bank-conflict counter
// on single-wave reads of this shape: chunk ^ (i mod 8) is conflict-free for
// every start; the tiled GEMM's chunk ^ ((i / 2) mod 8) is conflict-free
// only for starts that are multiples of 16 (4 conflict cycles per read
// otherwise), and rows of 64 bytes in two k planes conflict for every start.
__device__ __forceinline__ int dr_swz(int row) { return row & 7; }

// Ring slot of dY row p (p >= -16): (p + 20) mod 5 by a multiply and shift.
// Wait until at most n (0 .. 63) of this wave's vector memory operations
// are outstanding (s_waitcnt takes the count as an immediate).
__device__ __forceinline__ void wait_vmem_le(int n)
{
    switch (n) {
#define CBW_VMCNT_CASE(k) \
    case k: __builtin_amdgcn_s_waitcnt(0x0f70 | ((k) & 15) | ((((k) >> 4) & 3) << 14)); break;
#define CBW_VMCNT_8(k) CBW_VMCNT_CASE(k) CBW_VMCNT_CASE(k + 1) CBW_VMCNT_CASE(k + 2) CBW_VMCNT_CASE(k + 3) \
    CBW_VMCNT_CASE(k + 4) CBW_VMCNT_CASE(k + 5) CBW_VMCNT_CASE(k + 6) CBW_VMCNT_CASE(k + 7)
        CBW_VMCNT_8(0) CBW_VMCNT_8(8) CBW_VMCNT_8(16) CBW_VMCNT_8(24)
        CBW_VMCNT_8(32) CBW_VMCNT_8(40) CBW_VMCNT_8(48) CBW_VMCNT_8(56)
#undef CBW_VMCNT_8
#undef CBW_VMCNT_CASE
    default: __builtin_amdgcn_s_waitcnt(0x0f70); break;   // vmcnt(0)
    }
}

// NBW: 16-column blocks per wave at most; MASKED: x_mask applied.
template <int NBW, bool MASKED>
__global__ __launch_bounds__(DR_NT) void bwd_data_rows_kernel(DataRowsParams p)
{
    static_assert(NBW >= 1 && NBW <= 4, "column blocks per wave");
    // The ring of dY rows (p.nslot slots of p.slot_bytes) and, masked, the
    // ring of footprint rows (p.depth + 2 slots of p.mslot_bytes) after it:
    // this step's, the previous one's (stored now) and the next depth.
    __shared__ __attribute__((aligned(1024))) char Ys[kDataRowsLds];
    char* const Ms = Ys + p.mask_off;
    // footprint nibble (4 channels) -> the masks of the lane's two output
    // words, 16 bits per channel
    __shared__ uint2 mtab[16];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int cw = wave & 1, wg = wave >> 1;          // channel half, column group
    const int g = lane >> 4, col = lane & 15;          // k group of a fragment, column of a block

    const int t = xcd_remap(blockIdx.x, gridDim.x);
    const int seg = t % p.nseg, strip = t / p.nseg;
    const int w0 = seg * DR_WT;
    const int wn = min(DR_WT, p.W - w0);               // valid columns of the segment
    const int nu = p.slot_bytes >> 10;                 // copy instructions per dY row
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
    // The 72 KB of filters go into LDS once per workgroup (the start of the
    // dY ring, not yet in use; 1 KB copies spread over the waves), and each
    // wave reads its fragments from there: the eight waves would otherwise
    // read 36 KB each from L2, four times the same bytes per workgroup, and
    // that burst at the start of every workgroup measured 6 to 10 us.
    uint4 afr[9][2][2];
    if (MASKED && tid < 16) {
        auto half = [](int b) { return b ? 0xffffu : 0u; };
        mtab[tid] = make_uint2(half(tid & 1) | (half(tid & 2) << 16), half(tid & 4) | (half(tid & 8) << 16));
    }
    {
        static_assert(9 * 64 * 64 * 2 <= kDataRowsLds, "the filters fit the ring's LDS");
        const u32x4_t rw = make_rsrc_words(p.wt, p.wt_bytes);
        for (int u = wave; u < 9 * 64 * 64 * 2 / 1024; u += DR_NT / 64)
            buf_load16_lds(rw, (uint32_t)(1024 * u + 16 * lane), lds_addr(Ys) + 1024u * u);
        wait_vmem();
        __syncthreads();
#pragma unroll
        for (int tap = 0; tap < 9; ++tap)
#pragma unroll
            for (int cb = 0; cb < 2; ++cb)
#pragma unroll
                for (int kc = 0; kc < 2; ++kc) {
                    const int c = 32 * cw + 16 * cb + col;
                    afr[tap][cb][kc] = *reinterpret_cast<const uint4*>(Ys + ((tap * 64 + c) * 64 + kc * 32 + 8 * g) * 2);
                }
        __syncthreads();   // every wave holds its fragments before the ring overwrites them
    }

    // B fragment offsets in a ring slot: output column block b0, tap column
    // s, k half kc; LDS row i = 16 b0 + col + 2 - s holds dY column
    // w0 + pw - 2 + i.  Block b0 + j adds 16 rows (2048 bytes, an
    // instruction offset: the swizzle repeats every 16 rows).
    int boff[3][2];
#pragma unroll
    for (int s = 0; s < 3; ++s)
#pragma unroll
        for (int kc = 0; kc < 2; ++kc) {
            const int i = 16 * b0 + col + 2 - s;
            boff[s][kc] = i * 128 + 16 * ((4 * kc + g) ^ dr_swz(i));
        }

    // Copies of a dY row segment: instruction u writes LDS bytes
    // [1024 u, 1024 u + 1024) of the slot, i.e. rows 8 u + l / 8 at physical
    // chunk l % 8 for lane l.
    // Ring slots: dY row p in slot (p + 16) mod nslot, the footprint of
    // output row `row` in slot row mod (depth + 2).  The pipeline below
    // advances both by one per step instead of dividing.
    auto dr_slot = [&](int pp) { const uint32_t x = (uint32_t)(pp + 16); return (int)(x - fdiv(x, p.div_nslot) * p.nslot); };
    auto mslot = [&](int row) { return (int)((uint32_t)row - fdiv((uint32_t)row, p.div_nmslot) * (p.depth + 2)); };
    auto wrap = [](int x, int n) { return x >= n ? x - n : (x < 0 ? x + n : x); };   // |x| < 2n
    const u32x4_t rs_dy = make_rsrc_words(p.dy, p.dy_bytes);
    // Copy instruction m of this wave fills LDS rows 8 (wave + 8 m) + l / 8
    // of a slot; the wave issues ny of them per dY row.  Loop-invariant
    // per-instruction conditions are kept as counts and recomputed offsets,
    // not as predicates: the compiler would hold each predicate as a
    // 64-bit lane mask for the whole kernel and spill them.
    const int ny = nu > wave ? (nu - wave + 7) / 8 : 0;
    // dY row (n, pp) into ring slot `slot`; a row outside the image (the
    // padding above and below) is written as zeros, so that the matrix loop
    // reads every tap's row without a branch
    auto copy_y = [&](int n, int pp, int slot) -> int {
        const bool in = pp >= 0 && pp < p.P;
        const uint32_t base = (uint32_t)(n * p.P + pp) * (uint32_t)(p.Q * 128);
        const uint32_t lds = lds_addr(Ys) + (uint32_t)(slot * p.slot_bytes);
        for (int m = 0; m < ny; ++m) {
            const int u = wave + 8 * m;
            const int i = 8 * u + (lane >> 3);
            const int j = (lane & 7) ^ dr_swz(i);      // logical chunk stored at physical chunk lane % 8
            const int q = w0 + p.pad_w - 2 + i;
            const bool ok = in && q >= 0 && q < p.Q;
            buf_load16_lds(rs_dy, ok ? base + (uint32_t)((q * 64 + j * 8) * 2) : kOOB, lds + 1024u * u);
        }
        return ny;
    };
    const u32x4_t rs_m = make_rsrc_words(p.mask, p.mask_bytes);
    // footprint of output row `row` (8 bytes per pixel, wn pixels): 16 bytes
    // per lane when the row is a whole number of 16-byte pieces (wn even),
    // else 4 bytes per lane; one copy per wave of the first waves, over the
    // row's 16-pixel blocks (128 nwb bytes, what the readers reach).  mlane
    // is the lane's byte in the row, or kOOB past the row's end (src + kOOB
    // stays past the buffer's end: src < 2^31), which writes zeros, so the
    // pixels of the last block past the segment read as dead.
    const bool m16 = (wn & 1) == 0;
    const int nm_copy = MASKED && wave * (m16 ? 1024 : 256) < 128 * nwb ? 1 : 0;
    const uint32_t mbyte = m16 ? 1024u * wave + 16u * lane : 256u * wave + 4u * lane;
    const uint32_t mlane = mbyte < (uint32_t)(wn * 8) ? mbyte : kOOB;
    auto copy_m = [&](int row, int slot) -> int {
        if (!MASKED) return 0;
        const uint32_t src = (uint32_t)(row * p.W + w0) * 8u;
        const uint32_t dst = lds_addr(Ms) + (uint32_t)(slot * p.mslot_bytes);
        for (int k = 0; k < nm_copy; ++k) {
            if (m16) buf_load16_lds(rs_m, src + mlane, dst + 1024u * wave);
            else buf_load4_lds(rs_m, src + mlane, dst + 256u * wave);
        }
        return nm_copy;
    };
    auto image = [&](int row) { return (int)fdiv((uint32_t)row, p.div_h); };

    floatx4 acc[2][NBW];
#pragma unroll
    for (int j = 0; j < NBW; ++j) acc[0][j] = acc[1][j] = floatx4{0.f, 0.f, 0.f, 0.f};
    uint2 outv[2][NBW];                                // the previous row's outputs, stored one step later
    int computed = 0;                                  // pixels of the rows whose matrix work ran

    // The wave's NB column blocks (NB = cnt, a compile-time constant in each
    // copy of the pipeline below, so the block loops carry no branches and
    // the fragment reads of a (tap, k half) are issued ahead of its MFMAs).
    auto compute = [&](int h, int sl0, auto nb_tag) {   // output row h of its image; slot of dY row h + ph
        constexpr int NB = decltype(nb_tag)::value;
        (void)h;
        const char* yb[3];
#pragma unroll
        for (int r = 0; r < 3; ++r) yb[r] = Ys + wrap(sl0 - r, p.nslot) * p.slot_bytes;
        // straight-line code over the 9 taps and both k halves: the fragment
        // reads of later taps can be issued ahead of earlier MFMAs
#pragma unroll
        for (int r = 0; r < 3; ++r)
#pragma unroll
            for (int s = 0; s < 3; ++s)
#pragma unroll
                for (int kc = 0; kc < 2; ++kc) {
                    uint4 fb[NB > 0 ? NB : 1];
#pragma unroll
                    for (int j = 0; j < NB; ++j)
                        fb[j] = *reinterpret_cast<const uint4*>(yb[r] + boff[s][kc] + 2048 * j);
#pragma unroll
                    for (int j = 0; j < NB; ++j) {
                        acc[0][j] = mfma_chunk(acc[0][j], afr[3 * r + s][0][kc], fb[j], uint16_t{});
                        acc[1][j] = mfma_chunk(acc[1][j], afr[3 * r + s][1][kc], fb[j], uint16_t{});
                    }
                }
    };

    // The wave's footprint words of row slot `ms`: channels 32 cw .. + 31 of
    // pixel 16 (b0 + j) + col (0 past the segment).
    const int mw_off = (16 * b0 + col) * 8 + cw * 4;   // the lane's word of block b0; block b0 + j: + 128 j
    auto mask_words = [&](int ms, uint32_t* mw, auto nb_tag) {
        constexpr int NB = decltype(nb_tag)::value;
        const char* mrow = Ms + ms * p.mslot_bytes + mw_off;
#pragma unroll
        for (int j = 0; j < NB; ++j) mw[j] = *reinterpret_cast<const uint32_t*>(mrow + 128 * j);
    };
    // pixels of this wave's columns (each pixel belongs to two waves, one
    // per channel half)
    const int wave_px = max(0, min(16 * (b0 + cnt), wn) - 16 * b0);

    // One output row: the matrix work unless every output of this wave is
    // dead (its channel half of its columns; mw: the row's footprint words),
    // then the sums rounded and held for the next step, which applies the
    // footprint and stores them.
    auto step = [&](int h, int sl0, const uint32_t* mw, auto nb_tag) {
        constexpr int NB = decltype(nb_tag)::value;
        bool live = true;
        if (MASKED && p.skip) {
            uint32_t any = 0;
#pragma unroll
            for (int j = 0; j < NB; ++j) any |= mw[j];
            live = __ballot(any != 0u) != 0ull;
        }
        if (live) {
            compute(h, sl0, nb_tag);
            computed += wave_px;
        }
#pragma unroll
        for (int j = 0; j < NB; ++j) {
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) {
                const floatx4 v = acc[cb][j];
                outv[cb][j] = make_uint2(pack_bf16x2(v.x, v.y), pack_bf16x2(v.z, v.w));
                acc[cb][j] = floatx4{0.f, 0.f, 0.f, 0.f};
            }
        }
    };
    const __amdgpu_buffer_rsrc_t rs_dx = make_rsrc(p.dx, p.dx_bytes);
    // outputs of `row` (footprint slot ms): a lane holds 4 channels of one
    // pixel in each of its two 16-channel blocks; a dead output is stored
    // as +0.0 (the bit pattern 0).  Lanes l and l + 16 (k groups 0 and 1,
    // and 2 and 3) then swap a block each, so that every lane holds 8
    // consecutive channels (16 bytes) and a store instruction writes
    // 64-byte pieces of 16 pixel rows rather than 32-byte ones (the
    // memory's write granule is 64 bytes): group g gets channels
    // 16 (g % 2) + 8 (g / 2) .. + 7 of the wave's half.
    const int choff = 16 * (g & 1) + 8 * (g >> 1);
    auto store = [&](int row, const uint32_t* mw, auto nb_tag) {
        constexpr int NB = decltype(nb_tag)::value;
#pragma unroll
        for (int j = 0; j < NB; ++j) {
            const int w = 16 * (b0 + j) + col;
            uint2 v[2];
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) {
                v[cb] = outv[cb][j];
                if (MASKED) {
                    const uint2 km = mtab[(mw[j] >> (16 * cb + 4 * g)) & 15u];
                    v[cb].x &= km.x;
                    v[cb].y &= km.y;
                }
            }
            // odd lane rows of block 0 <-> even lane rows of block 1
            const auto sx = __builtin_amdgcn_permlane16_swap(v[0].x, v[1].x, false, false);
            const auto sy = __builtin_amdgcn_permlane16_swap(v[0].y, v[1].y, false, false);
            const uint32_t base = (uint32_t)(((row * p.W + w0 + w) * 64 + 32 * cw + choff) * 2);
            __builtin_amdgcn_raw_buffer_store_b128(u32x4{sx[0], sy[0], sx[1], sy[1]}, rs_dx, w < wn ? base : kOOB, 0,
                                                   0);
        }
    };

    // Pipeline over the strip's rows, D = p.depth steps ahead: at step i the
    // copies of step i + D are issued (its new dY row when it lies in the
    // same image as row i, and its footprint) after the outputs of step i - 1
    // are stored; the wait at the end of step i leaves only the copies of
    // steps i + 2 .. i + D in flight (stores issued before them have
    // completed by then, as have the older copies, which land in issue
    // order).  A window starts at the strip's first row and at every first
    // row of an image: its three dY rows and the new rows of the next D - 1
    // steps are loaded after the step before it, and waited for.  Every
    // wave runs the same steps and barriers, in the copy of this loop for
    // its own block count.
    auto pipeline = [&](auto nb_tag) {
        const int D = p.depth, nm = p.depth + 2;
        // state of step row ra: image n, row h, ring slot sl0 of dY row
        // h + ph, footprint slot ms; allowed = copies issued at the last
        // D - 1 steps, hist = the issue counts of the last steps, a byte each
        int n = 0, h = 0, sl0 = 0, ms = 0, allowed = 0;
        uint64_t hist = 0;
        auto open_window = [&](int rs) {
            n = image(rs);
            h = rs - n * p.H;
            sl0 = dr_slot(h + p.pad_h);
#pragma unroll
            for (int r = 0; r < 3; ++r) copy_y(n, h + p.pad_h - r, wrap(sl0 - r, p.nslot));
            for (int d = 1; d < D && rs + d < row_end && h + d < p.H; ++d)
                copy_y(n, h + p.pad_h + d, wrap(sl0 + d, p.nslot));
            hist = 0;
            allowed = 0;
        };
        int ra = row_begin;
        if (ra < row_end) {
            open_window(ra);
            ms = mslot(ra);
            for (int d = 0; d < D && ra + d < row_end; ++d) copy_m(ra + d, wrap(ms + d, nm));
        }
        wait_vmem();
        __syncthreads();
        // footprint words of the row stored at this step (read at the step
        // before, for its skip test) and of the row computed now: each row's
        // words are read from LDS once, first thing in its step, so their
        // latency passes under the stores and copies issued behind them
        constexpr int NB = decltype(nb_tag)::value;
        uint32_t mwp[NB > 0 ? NB : 1] = {};
        for (; ra < row_end; ++ra) {
            uint32_t mwc[NB > 0 ? NB : 1] = {};
            if (MASKED) mask_words(ms, mwc, nb_tag);
            if (ra > row_begin) store(ra - 1, mwp, nb_tag);
            int issued = 0;
            if (ra + D < row_end) {
                if (h + D < p.H) issued += copy_y(n, h + p.pad_h + D, wrap(sl0 + D, p.nslot));
                issued += copy_m(ra + D, wrap(ms + D, nm));
            }
            hist = (hist << 8) | (uint64_t)issued;
            allowed += issued - (int)((hist >> (8 * (D - 1))) & 0xffu);
            step(h, sl0, mwc, nb_tag);
#pragma unroll
            for (int j = 0; j < (NB > 0 ? NB : 1); ++j) mwp[j] = mwc[j];
            wait_vmem_le(allowed);
            __syncthreads();
            // advance to row ra + 1
            ms = wrap(ms + 1, nm);
            if (h + 1 < p.H) {
                ++h;
                sl0 = wrap(sl0 + 1, p.nslot);
            } else if (ra + 1 < row_end) {
                open_window(ra + 1);   // the next image
                wait_vmem();
                __syncthreads();
            }
        }
        if (row_end > row_begin) store(row_end - 1, mwp, nb_tag);
    };
    // cnt <= NBW (checked by the host for the first segment, which is the widest)
    if (cnt >= NBW) pipeline(std::integral_constant<int, NBW>{});
    else if (NBW >= 2 && cnt == NBW - 1) pipeline(std::integral_constant<int, (NBW >= 2 ? NBW - 1 : 0)>{});
    else if (NBW >= 3 && cnt == NBW - 2) pipeline(std::integral_constant<int, (NBW >= 3 ? NBW - 2 : 0)>{});
    else if (NBW >= 4 && cnt == NBW - 3) pipeline(std::integral_constant<int, (NBW >= 4 ? NBW - 3 : 0)>{});
    else pipeline(std::integral_constant<int, 0>{});
    // the workgroup's count: the sum over its waves
    __shared__ int wave_counts[DR_NT / 64];
    if (lane == 0) wave_counts[wave] = computed;
    __syncthreads();
    if (tid == 0) {
        int total = 0;
#pragma unroll
        for (int w = 0; w < DR_NT / 64; ++w) total += wave_counts[w];
        p.row_counts[blockIdx.x] = total;
    }
}

template <int NBW>
hipError_t launch_nbw(const DataRowsParams& p, int grid, hipStream_t stream, const ProfEvents& ev)
{
    hipError_t e_launch;
    if (p.mask)
        e_launch = launch_timed(bwd_data_rows_kernel<NBW, true>, dim3(grid), dim3(DR_NT), stream, ev, p);
    else
        e_launch = launch_timed(bwd_data_rows_kernel<NBW, false>, dim3(grid), dim3(DR_NT), stream, ev, p);
    return e_launch;
}

}  // namespace

int data_rows_segment() { return DR_WT; }

hipError_t launch_bwd_data_rows(const DataRowsParams& p, int grid, int nbw, hipStream_t stream, const ProfEvents& ev)
{
    // the grid must cover every (segment, strip) pair exactly as planned
    const int nstrips = (p.nrows + p.rows_per_strip - 1) / p.rows_per_strip;
    if (p.nseg != (p.W + DR_WT - 1) / DR_WT || grid != nstrips * p.nseg || p.nrows != p.N * p.H)
        return hipErrorInvalidValue;
    // the rings as the planner laid them out
    const int wseg = p.W < DR_WT ? p.W : DR_WT;
    if (p.depth < 1 || p.depth > 8 || p.nslot != p.depth + 3 || p.slot_bytes != ((wseg + 15) / 16 * 16 + 2 + 7) / 8 * 1024 ||
        p.mslot_bytes != (wseg * 8 + 1023) / 1024 * 1024 || p.mask_off != p.nslot * p.slot_bytes ||
        p.mask_off + (p.depth + 2) * p.mslot_bytes > kDataRowsLds || p.div_nslot.d != (uint32_t)p.nslot ||
        p.div_nmslot.d != (uint32_t)(p.depth + 2))
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
