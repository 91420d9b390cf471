// Tile shapes shared by the kernels and the host planner.  Each can be
// overridden at build time (-DCBW_DX_BM=... etc.) for tuning sweeps; the
// dispatcher refuses to run if kernels and planner disagree.
#pragma once

#ifndef CBW_DX_BM
#define CBW_DX_BM 256   // data gradient: channels per tile = compaction group width
#endif
#ifndef CBW_DX_BN
#define CBW_DX_BN 224   // data gradient: pixels per tile
#endif
#ifndef CBW_DX_WM
#define CBW_DX_WM 4     // waves along channels
#endif
#ifndef CBW_DX_WN
#define CBW_DX_WN 2     // waves along pixels
#endif
#ifndef CBW_DX_OCC
#define CBW_DX_OCC 1    // resident workgroups per CU
#endif
#ifndef CBW_DX_PIPE
#define CBW_DX_PIPE 0   // data gradient: fragments of the next chunk group read during the MFMAs
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
