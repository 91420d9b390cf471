// Host-only planning: descriptor validation, tile counts, split-K choice and
// workspace layout.  No HIP dependency, so it is testable without a GPU.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "../../include/convbwd.h"
#include "tiles.hpp"

namespace cbw {

// Tile constants shared with the kernels (asserted equal at dispatch time).
constexpr int kWeightTileC = CBW_DW_BM; // channels c per weight-gradient tile
constexpr int kWeightTileK = CBW_DW_BN; // output channels k per weight-gradient tile
constexpr int kCompactBlock = 256;      // pixels per compaction block
constexpr int kRowSegment = 128;        // output columns per segment of the row-window weight gradient
// Resident weight-gradient workgroups the split-K factor aims to fill exactly.
constexpr int kWeightSlots = CBW_NUM_CUS * CBW_DW_OCC;

inline int weight_chunk_px(int dtype) { return 8 * (dtype == CBW_BF16 ? 8 : 4); }

struct Region {
    size_t off = 0, bytes = 0;
};

// Data-gradient tile for C output channels: the widest whose channel padding
// stays within C/8, else the least padded (ties to the wider).
int data_tile_index(int C);

struct DataPlan {
    int tile = 0, bm = 0, bn = 0;   // kDataTiles entry and its shape
    int64_t npix = 0;
    int groups = 0, nblk = 0;
    int ptiles = 0, nsteps = 0;
    int brows = 0;          // dense / select: pixel rows per tile (data_rows_pick)
    int split = 1;          // dense / select: host-chosen reduction split
    // Row-window kernel (data_rows_eligible): a workgroup per (column
    // segment, strip of rows_per_strip output rows), nbw 16-column blocks
    // per wave at most; it replaces the tiled GEMM and its compaction.
    bool rows = false;
    int rows_grid = 0, rows_per_strip = 0, rows_nseg = 0, rows_nbw = 0;
    int rows_depth = 0, rows_slot = 0, rows_mslot = 0;   // prefetch depth, ring slot bytes
    // Pointwise kernel (data_pw_eligible): pw_grid workgroups of
    // kDataPwWaves waves, each wave pw_bpw 16-pixel blocks; it too replaces
    // the tiled GEMM and its compaction (per-workgroup counts in row_counts).
    bool pw = false;
    int pw_grid = 0, pw_bpw = 0;
    Region header, wt, blk_counts, counts, dead_flags, lists, partial, row_counts;
    // NCHW callers: NHWC copies of dY and dX and the NHWC-order footprint,
    // after every other region (the other offsets do not depend on layout)
    Region t_dy, t_dx, t_mask;
    size_t total = 0;
};

constexpr int kDataSlots = CBW_NUM_CUS * CBW_DX_OCC;  // resident data-gradient workgroups

// Layers the row-window data gradient serves: bf16, 3 x 3 filters, stride
// 1, 64 input and 64 output channels (any padding, any layout: NCHW calls
// run it on their NHWC copies).
bool data_rows_eligible(const cbw_conv_desc* d);
// Layers the pointwise data gradient serves: bf16, 1 x 1 filters, stride 1,
// no padding, C and K in {64, 128, 256} with C * K <= 16384.
bool data_pw_eligible(const cbw_conv_desc* d);
constexpr int kDataMaxSplit = 16;

// Same rule as the kernels' data_split (see common.hpp).
inline int host_data_split(int T, int nsteps)
{
    if (T <= 0 || 2 * T > kDataSlots) return 1;
    int sp = kDataSlots / T;
    if (sp > kDataMaxSplit) sp = kDataMaxSplit;
    if (sp > nsteps) sp = nsteps;
    return sp < 1 ? 1 : sp;
}

// Weight-gradient tiling (bf16): output channels per tile (64, 128 or 256,
// from K) and, when C <= 128, up to floor(256/C) filter taps packed side by
// side in one 256-column channel tile, C columns each, so narrow layers fill
// the tile; the R*S taps go into as few groups as that allows, spread
// evenly over them.
int weight_tile_k_for(const cbw_conv_desc* d);
int weight_taps_per_group(const cbw_conv_desc* d);

struct WeightPlan {
    bool rows = false;      // row-window kernel (narrow stride-1 layers): chunks are output rows
    int chunk = 0;          // pixels per occupancy chunk (64, or Q for the row-window kernel)
    int64_t npq = 0;
    int bk = 0, tpg = 1, tgroups = 0;   // output-channel tile width, taps per group, tap groups
    int cg = 0;                         // channel columns per packed tap (C, or 256 without packing)
    int nchunks = 0, ctiles = 0, ktiles = 0, nsplit = 0, chunks_per_split = 0, grid = 0;
    int nparts = 0;         // partials the reduction sums
    bool direct = false;  // partial of the single split is dW itself
    Region header, occ, xlive, xbits, skip_slots, work_slots, partials;
    // NCHW callers: NHWC copies of X and dY and the NHWC-order dY footprint
    // (a caller's X footprint is reordered into xbits), after every other region
    Region t_x, t_dy, t_dymask;
    size_t total = 0;
};

// Accepts NHWC and NCHW activations (NCHW is served through the boundary
// transposes of the three backward operations); require_nhwc() is for the
// operations that run on NHWC only.
int validate_desc(const cbw_conv_desc* d);
int require_nhwc(const cbw_conv_desc* d);
// no_split: the reduction is never split (no partial-tile region; the
// kernels get a split bound of 1), for callers with a bounded scratch.
// allow_rows = false plans the tiled GEMM even for layers the row-window
// kernel serves (the forward convolution, the tiling inspection).
int plan_data(const cbw_conv_desc* d, bool masked, DataPlan* out, bool no_split = false, bool allow_rows = true);
// allow_rows: narrow stride-1 layers (C and K multiples of 64, at most 128,
// filters of at most 3 x 3, bf16) get the row-window kernel; callers that
// need the chunked kernel (X-block skipping) pass false.
int plan_weight(const cbw_conv_desc* d, WeightPlan* out, bool allow_rows = true);
bool weight_rows_eligible(const cbw_conv_desc* d);
// Workspace bytes of the weight gradient: enough for either kernel.
int weight_ws_bytes(const cbw_conv_desc* d, size_t* bytes);
// The forward convolution as a data-gradient GEMM: for stride 1, Y = conv(X, W)
// is the backward-data operation with the roles of C and K, of (H, W) and
// (P, Q) interchanged, the filter taps flipped and padding R-1-pad.  Writes that
// descriptor (validated) or returns CBW_ERR_UNSUPPORTED for stride > 1 or
// pad > R-1 (S-1).
int fwd_as_data_desc(const cbw_conv_desc* d, cbw_conv_desc* out);
inline int elem_bytes(int dtype) { return dtype == CBW_BF16 ? 2 : 4; }

}  // namespace cbw
