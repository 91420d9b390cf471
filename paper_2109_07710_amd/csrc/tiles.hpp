// Tile shapes shared by the kernels and the host planner (the dispatcher
// refuses to run if kernels and planner disagree).  The weight-gradient and
// occupancy macros can be overridden at build time for tuning sweeps.
#pragma once

#ifndef CBW_DX_OCC
#define CBW_DX_OCC 1    // resident workgroups per CU
#endif
#ifndef CBW_DW_BM
#define CBW_DW_BM 256   // weight gradient: channels c per tile
#endif
#ifndef CBW_DW_BN
#define CBW_DW_BN 256   // weight gradient: output channels k per tile
#endif
#ifndef CBW_DW_WM
#define CBW_DW_WM 2
#endif
#ifndef CBW_DW_WN
#define CBW_DW_WN 4
#endif
#ifndef CBW_DW_OCC
#define CBW_DW_OCC 1
#endif
#define CBW_NUM_CUS 256

// Data-gradient tiles: output channels x pixels, and the waves along each.
// Every tile runs 16 waves (four per SIMD; wave blocks of 32 x 112, 32 x 112
// and 32 x 64): more waves hide more of the copy and LDS latency than the
// larger wave blocks of 8 waves save.  The planner picks one per layer from
// the output channel count, so narrow layers do not pad their channels to
// 256; the channel width is also the compaction group width.
struct DataTile {
    int bm, bn, wm, wn;
};
constexpr int kDataTileCount = 3;
// Compaction groups (channel tiles) the gather mode handles; wider layers
// run the masked data gradient without compaction (footprint select only).
constexpr int kGatherMaxGroups = 16;
constexpr DataTile kDataTiles[kDataTileCount] = {{256, 224, 8, 2}, {128, 448, 4, 4}, {64, 512, 2, 8}};

// Row-window data gradient (3 x 3, stride 1, 64 channels in and out): output
// columns per segment at most, and the LDS its two rings share (dY rows of
// 128 bytes per column plus halo, footprint rows of 8 bytes per pixel).
constexpr int kDataPwWaves = 4;          // waves per pointwise workgroup
constexpr int kDataPwMaxWaves = 2048;    // resident pointwise waves (two workgroups per CU)
constexpr int kDataRowsSegment = 224;
constexpr int kDataRowsLds = 159744;

// Pixel rows a data-gradient tile actually covers: its capacity BN, or 16 or
// 32 rows less.  With `slots` resident workgroups the busiest CU runs
// ceil(tiles / slots) tiles one after another, so the rows that make
// ceil(tiles / slots) * rows smallest finish first (ties go to the larger
// tile).  Example: 32 images of 56 x 56 (100352 pixels) on 256 CUs take 448
// tiles of 224 rows (two rounds of 14 pixel blocks) or 483 tiles of 208 rows (two
// rounds of 13).  When so few tiles exist that the reduction is split
// (2 * tiles <= slots) the full tile is kept.  tiles[d] is the tile count at
// BN - 16 d rows; a choice with more than `cap` tiles is not taken (the
// gather mode's grid holds the dense tiling's tile count, and the full tile
// never exceeds it).  constexpr, so host planner and kernels share this one
// rule.
#ifndef CBW_DX_ROW_CHOICES
#define CBW_DX_ROW_CHOICES 3
#endif
constexpr int kDataRowChoices = CBW_DX_ROW_CHOICES;
constexpr int data_rows_pick(const int* tiles, int bn, int slots, int cap = 0x7fffffff)
{
    if (2 * tiles[0] <= slots) return bn;
    int best = bn;
    long long best_cost = (long long)((tiles[0] + slots - 1) / slots) * bn;
    for (int d = 1; d < kDataRowChoices; ++d) {
        if (tiles[d] > cap) continue;
        const int rows = bn - 16 * d;
        const long long cost = (long long)((tiles[d] + slots - 1) / slots) * rows;
        if (cost < best_cost) {
            best = rows;
            best_cost = cost;
        }
    }
    return best;
}
