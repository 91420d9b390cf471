// Launch interfaces between the host dispatcher (api.cpp) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.hpp"

namespace cbw {

// Data-gradient GEMM modes; MODE_FWD runs the same GEMM as the forward
// convolution (flipped filters, padding R-1-pad, stride 1) with a ReLU
// epilogue that also emits the output's footprint bits.
enum { MODE_DENSE = 0, MODE_SELECT = 1, MODE_GATHER = 2, MODE_FWD = 3 };
// Workspace header stamps of a data-gradient call served by the row-window
// kernel (bwd_data_rows.hip) or the pointwise kernel (bwd_data_pw.hip)
// instead of the tiled GEMM.
constexpr int MODE_ROWS = 4;
constexpr int MODE_PW = 5;

// Optional timing events attached to the dispatch of a GEMM kernel (both
// may be null): they record the kernel's own begin and end.
struct ProfEvents {
    hipEvent_t start = nullptr, stop = nullptr;
};

// A kernel launch with the optional timing events recorded on the stream
// right before and after it (plain event records: events attached to the
// launch itself were measured to slow the kernel they bracket by about 12%).
// Returns the first error.
template <typename Kern, typename Params>
hipError_t launch_timed(Kern kernel, dim3 grid, dim3 block, hipStream_t stream, const ProfEvents& ev,
                        const Params& p)
{
    hipError_t e = hipSuccess;
    if (ev.start && (e = hipEventRecord(ev.start, stream)) != hipSuccess) return e;
    hipLaunchKernelGGL(kernel, grid, block, 0, stream, p);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (ev.stop) e = hipEventRecord(ev.stop, stream);
    return e;
}

struct ReduceParams {
    const float* part;       // [nsplit][K][RS][C] weight-gradient partials
    float* dw;
    int nsplit, K, RS, C, krsc;
    int G;                   // threads per output (splitk_reduce_group)
    int blocks;              // 256-thread workgroups of the weight-gradient part
};

struct DataParams {
    const void* dy;          // [N*P*Q][K]
    const void* wt;          // [R*S][C][K]
    void* dx;                // [N*H*W][C]
    const uint32_t* mask;    // packed footprint of X (select / gather)
    // gather mode: the compaction counts written by the preparation launch,
    // and the outputs the GEMM writes for the reduction kernel and readers
    const int32_t* blk_counts;   // [groups][nblk] live pixels per 256-pixel block
    int nblk;
    int32_t* lists;          // [groups][npix] live pixels, ascending (written by the tiles of
                             // groups with dead pixels; a fully live group's list is 0, 1, 2, ...)
    int32_t* counts;         // [groups] live-pixel counts (written by workgroup 0)
    int32_t* dead_flags;     // [groups] 1 when the group has a dead pixel (raised by the
                             // preparation launch, lowered by the reduction launch)
    int N, H, W, C, K, R, S, P, Q;
    int stride_h, stride_w, pad_h, pad_w;
    int npix;                // N*H*W
    int ctiles;              // channel tiles = compaction groups
    int ptiles;              // pixel tiles (dense / select modes)
    int brows;               // pixel rows per tile (dense / select modes; gather derives its own)
    int split;               // reduction split (dense / select modes; gather derives its own)
    int nslots, smax;        // resident workgroups; largest split
    float* partial;          // [item][BN][BM] fp32 partial tiles when split
    uint32_t dy_bytes, wt_bytes, dx_bytes;
    uint32_t* out_mask;      // MODE_FWD: footprint bits of the output (nullable)
    int tile;                // kDataTiles entry the plan chose
    FastDiv div_w, div_h;    // pixel -> (n, h, w)
    // The weight gradient's split-K reduction run by the GEMM launch's
    // tail workgroups (the call that computes both gradients; blocks = 0
    // otherwise): workgroups from gemm_grid on each take four of its
    // 256-thread blocks, after every GEMM workgroup has been dispatched.
    ReduceParams dw_red;
    int gemm_grid;
};

// Row-window data gradient (3 x 3, stride 1, C = K = 64, bf16, NHWC): a
// workgroup per (column segment, strip of rows_per_strip output rows).
struct DataRowsParams {
    const void* dy;          // [N*P*Q][64]
    const void* wt;          // [9][64][64]: filters by tap, input channel c, then k
    void* dx;                // [N*H*W][64]
    const uint32_t* mask;    // packed footprint of X, or null (dense)
    int32_t* row_counts;     // [grid] pixels computed per workgroup, counted once per channel half
    int N, H, W, P, Q, pad_h, pad_w;
    int nseg, rows_per_strip, nrows;   // nrows = N*H
    int skip;                // masked: rows whose footprint is empty skip the matrix work
    uint32_t dy_bytes, dx_bytes, mask_bytes, wt_bytes;
    FastDiv div_h;           // output row -> image
    // rings in LDS: depth steps of prefetch, nslot = depth + 3 dY rows of
    // slot_bytes, then (from mask_off) depth + 2 footprint rows of mslot_bytes
    int depth, nslot, slot_bytes, mslot_bytes, mask_off;
    FastDiv div_nslot, div_nmslot;
};
int data_rows_segment();
hipError_t launch_bwd_data_rows(const DataRowsParams& p, int grid, int nbw, hipStream_t stream, const ProfEvents& ev);

// Pointwise data gradient (1 x 1, stride 1, no padding, bf16, NHWC, C and K
// in {64, 128, 256}, C * K <= 16384): wave w of the grid owns the 16-pixel
// blocks [w * bpw, (w + 1) * bpw).
struct DataPwParams {
    const void* dy;          // [npix][K]
    const void* wt;          // [C][K]
    void* dx;                // [npix][C]
    const uint32_t* mask;    // packed footprint of X, or null (dense)
    int32_t* counts;         // [grid] pixels of the blocks computed per workgroup
    int npix, C, K, nblk, bpw;
    int skip;                // masked: blocks whose footprint is empty skip the matrix work
    uint32_t dy_bytes, dx_bytes, mask_bytes;
};
int data_pw_waves_per_group();
hipError_t launch_bwd_data_pw(const DataPwParams& p, int grid, hipStream_t stream, const ProfEvents& ev);

struct CompactParams {
    const uint32_t* mask;    // packed footprint, NHWC bit order
    int32_t* blk_counts;     // [groups][nblk] live pixels per 256-pixel block
    int32_t* dead_flags;     // [groups] set to 1 by a block with a dead pixel
    void* dx;                // zero-filled at (pixel, group) rows dead for the whole group
    int npix, C, G, groups, nblk, elem_bytes;
};

struct WeightParams {
    const void* x;           // [N*H*W][C]
    const void* dy;          // [N*P*Q][K]
    float* out;              // [nsplit][K][R*S][C] partials, or dW (KRSC) when nsplit == 1
    const uint8_t* occ;      // [nchunks][ktiles] block occupancy, or null (no skipping)
    const uint8_t* xlive;    // [nchunks][tgroups*ctiles] X-window liveness, or null (no X-block skipping)
    int32_t* skip_slots;     // [grid] skipped-block count per workgroup
    int32_t* work_slots;     // [grid] executed blocks per work item (item order)
    int* header;
    int N, H, W, C, K, R, S, P, Q;
    int stride_h, stride_w, pad_h, pad_w;
    int npq;                 // N*P*Q
    int nchunks;             // ceil(npq / chunk)
    int chunks_per_split;
    int ctiles, ktiles, nsplit;
    int bk;                  // output channels per tile (64, 128, 256)
    int tpg, tgroups;        // filter taps per 256-column channel tile, and tap groups
    int cg;                  // channel columns per packed tap (C when packed, else 256)
    int rows;                // row-window kernel: chunks are output rows, tgroups are 128-column segments
    int mode_flags;
    uint32_t x_bytes, dy_bytes;
    FastDiv div_q, div_p;    // pixel -> (n, p, q)
    // this call's number: header[kDeadWord] == gen when the occupancy pass
    // found a dead block (bf16 kernels; see OccParams)
    uint32_t gen;
};
constexpr int kDeadWord = 4;   // weight workspace header word of the dead-block flag

struct OccParams {
    const void* dy;          // values [npq][K] (used when bits == null)
    const uint32_t* bits;    // packed dY footprint, or null
    uint8_t* occ;            // [nchunks][ktiles]
    int npq, K, chunk, BNk, ktiles, nchunks, dtype;
    int cpw;                 // chunks per workgroup (cpw * ktiles, and cpw * combos, at most 1024)
    // X-window liveness (only when xlive is set): xlive[chunk][tg*ctiles+ct]
    // = 1 iff a pixel of the chunk has, at one of tap group tg's taps, an X
    // pixel inside the image with a non-zero among channel tile ct's channels.
    const uint32_t* xbits;   // packed X footprint (a superset of X's non-zeros)
    uint8_t* xlive;
    int N, H, W, C, P, Q, S, RS, stride_h, stride_w, pad_h, pad_w;
    int tpg, tgroups, ctiles, ctw;   // taps per group, groups, channel tiles, channels per tile
    FastDiv div_q, div_p;
    FastDiv div_chunk, div_ktiles;   // pixel -> chunk, pair -> pixel
    // The call's dead-block flag: a workgroup that finds a dead block (or a
    // dead X window) stores gen, this call's number, into *any_dead, which
    // the GEMM compares with the same number (nullable).
    int* any_dead;
    uint32_t gen;
};

// Per-element data gradient on the vector ALUs (bf16, NHWC, KRSC filters).
struct EwParams {
    const void* dy;          // [N*P*Q][K]
    const void* w;           // [K][R][S][C]
    const uint32_t* mask;    // footprint of X, bit per element of [N*H*W][C]
    void* dx;                // [N*H*W][C]
    int32_t* counts;         // [N*H*W] (tap, k) products executed per pixel
    int N, H, W, C, K, R, S, P, Q;
    int stride_h, stride_w, pad_h, pad_w;
    int npix;
    uint32_t dy_bytes, w_bytes, dx_bytes;
    FastDiv div_w, div_h;
};
hipError_t launch_elementwise_data(const EwParams& p, hipStream_t stream);

int data_tile_channels(int tile);
int data_tile_pixels(int tile);
int weight_tile_channels();
int weight_tile_k();
int weight_chunk(int dtype);
int compact_block_pixels();

// Filter transform (and, when cp is given, the compaction counts and the
// dead-row zero fill; when op is given, the weight gradient's dY block
// occupancy) in one launch.
hipError_t launch_data_prep(int dtype, const void* w, void* wt, int K, int C, int RS, int krsc, int* header,
                            int mode, const CompactParams* cp, hipStream_t stream, const OccParams* op = nullptr);
// with_reduce = false leaves a split reduction to launch_bwd_reduce.
hipError_t launch_bwd_data(int dtype, int mode, const DataParams& p, hipStream_t stream, const ProfEvents& ev,
                           bool with_reduce = true);
// The weight gradient's split-K reduction (rp.blocks workgroups, none when
// dW was written directly) and, when dx_reduce, the data gradient's split
// tiles, in one launch.
hipError_t launch_bwd_reduce(int dtype, int dx_mode, const DataParams& dp, bool dx_reduce, const ReduceParams& rp,
                             hipStream_t stream);
// Forward preparation: Wf[tap'][k][c] = W[k][tap][c] with tap' the flipped tap
// (R-1-r, S-1-s), the workspace header stamped, and `zero_words` words of
// `zero` cleared (footprint words filled by atomic OR), in one launch.
hipError_t launch_fwd_prep(int dtype, const void* w, void* wt, int K, int C, int R, int S, int krsc, int* header,
                           uint32_t* zero, int64_t zero_words, hipStream_t stream);
// Boundary layout conversion (NCHW callers): dst[b][c][r] = src[b][r][c] for
// `batch` matrices of rows x cols elements, and footprint bits in NCHW
// element order reordered to NHWC element order.
hipError_t launch_transpose(int dtype, const void* src, void* dst, int batch, int rows, int cols, hipStream_t s);
hipError_t launch_bits_nchw_to_nhwc(const uint32_t* src, uint32_t* dst, int N, int C, int HW, hipStream_t s);
hipError_t launch_relu_mask_pack(int dtype, int64_t count, const void* x, uint32_t* bits, int relu,
                                 hipStream_t stream);
hipError_t launch_occupancy(const OccParams& p, hipStream_t stream);
hipError_t launch_bwd_weight(int dtype, const WeightParams& p, hipStream_t stream, const ProfEvents& ev);
hipError_t launch_splitk_reduce(const float* part, float* dw, int nsplit, int K, int RS, int C, int krsc,
                                hipStream_t stream);

}  // namespace cbw
