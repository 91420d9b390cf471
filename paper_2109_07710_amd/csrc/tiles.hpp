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
constexpr DataTile kDataTiles[kDataTileCount] = {{256, 224, 8, 2}, {128, 448, 4, 4}, {64, 512, 2, 8}};
