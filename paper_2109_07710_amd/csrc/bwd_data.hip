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
//             generation, Sec. IV-B), which each tile derives for itself from
//             the footprint and the preparation launch's counts; the epilogue
//             applies the per-element select.  Rows dead for the whole group
//             were zero-filled by the preparation launch and are never
//             touched here.
//
// Main loop: both operand tiles are copied by the load unit straight from
// global memory into a double-buffered LDS ring (no staging registers, one
// barrier per reduction step).  LDS rows are 128 bytes (8 chunks of 16
// bytes) with an XOR chunk swizzle so that the MFMA fragment reads of 16
// consecutive rows spread over all banks.
#include <algorithm>
#include <type_traits>


#include "common.hpp"
#include "kernels.hpp"
#include "footprint.hpp"
#include "tiles.hpp"
#include "occupancy.hpp"
#include "reduce.hpp"


namespace cbw {

namespace {

constexpr int CH = 8;     // 16-byte chunks of reduction per row per step

// Compile-time shape of data-gradient tile TI (kDataTiles[TI]).
template <int TI>
struct Tile {
    static constexpr int BM = kDataTiles[TI].bm;       // channels per tile (= compaction group width)
    static constexpr int BN = kDataTiles[TI].bn;       // pixels per tile
    static constexpr int WM = kDataTiles[TI].wm;       // waves along channels
    static constexpr int WN = kDataTiles[TI].wn;       // waves along pixels
    static constexpr int NW = WM * WN;                 // waves: 8 or 16
    static constexpr int NT = NW * 64;
    static constexpr int TM = BM / WM, TN = BN / WN;   // wave tile
    static constexpr int FM = TM / 16, FN = TN / 16;   // 16x16 MFMA tiles per wave
    static constexpr int IA = (BM / 8 + NW - 1) / NW;  // 1 KB copy instructions per wave per step, A
    static constexpr int IB = (BN / 8 + NW - 1) / NW;  // same for B
    static_assert(NW == 16, "four waves per SIMD");
    static_assert(BM % 8 == 0 && BN % 8 == 0, "tiles are copied in groups of 8 rows");
    static_assert(TM % 16 == 0 && TN % 16 == 0, "wave tile must be a multiple of 16");
};

__device__ __forceinline__ int swz8(int row) { return (row >> 1) & 7; }

// Wave coordinates (wm along channels, wn along pixels) of wave w.  The
// waves w, w + 4, w + 8 and w + 12 of a workgroup share one SIMD (measured:
// which SIMD varies between workgroups, the grouping does not), and the
// coordinates are spread so that those four waves sit in different pixel
// columns where WN allows: when a tile's pixel blocks do not divide evenly
// among the WN columns, the columns with one block more fall on different
// SIMDs and every SIMD gets the same matrix work.
template <int WN>
__device__ __forceinline__ void wave_coords(int w, int& wm, int& wn)
{
    static_assert(WN == 2 || WN == 4 || WN == 8, "16-wave tiles only");
    const int s = w & 3, q = w >> 2;
    if (WN == 2) {
        wm = s + 4 * (q >> 1);
        wn = q & 1;
    } else if (WN == 4) {
        wm = s;
        wn = q;
    } else {
        wm = s >> 1;
        wn = 2 * q + (s & 1);
    }
}

// Rows per tile in gather mode, from the live counts of every channel group
// (the host makes the same choice for the other modes from the pixel count),
// among the choices that give at most `cap` tiles.
template <int BN>
__device__ __forceinline__ int gather_rows(const int32_t* counts, int groups, int slots, int cap)
{
    int tiles[kDataRowChoices];
#pragma unroll
    for (int c = 0; c < kDataRowChoices; ++c) {
        const int rows = BN - 16 * c;
        int t = 0;
        for (int g = 0; g < groups; ++g) t += (counts[g] + rows - 1) / rows;
        tiles[c] = t;
    }
    return data_rows_pick(tiles, BN, slots, cap);
}

// Channel group and pixel tile of gather-mode tile `tile`.  Tiles are taken
// round by round: round r holds the r-th pixel tile of every group that has
// more than r tiles, groups in order.  The groups of one pixel range thus sit
// next to each other in the order, as in the dense mode (tile = ptile *
// groups + group), and the XCD that runs them reads their shared dY rows
// into one L2 instead of every group's XCD reading them again.  Rounds in
// which every group still has a tile are resolved in closed form.
__device__ __forceinline__ void gather_tile(const int32_t* counts, int groups, int rows, int tile, int& g,
                                            int& ptile)
{
    int tmin = 0x7fffffff, tmax = 0;
    for (int k = 0; k < groups; ++k) {
        const int t = (counts[k] + rows - 1) / rows;
        tmin = min(tmin, t);
        tmax = max(tmax, t);
    }
    if (tile < tmin * groups) {
        ptile = tile / groups;
        g = tile - ptile * groups;
        return;
    }
    int before = tmin * groups;
    for (int r = tmin; r < tmax; ++r) {
        for (int k = 0; k < groups; ++k) {
            if ((counts[k] + rows - 1) / rows <= r) continue;
            if (before == tile) {
                g = k;
                ptile = r;
                return;
            }
            ++before;
        }
    }
    // not reached for tile < the total tile count; past it, a tile beyond
    // every group's rows (no pixel is read or written)
    g = 0;
    ptile = tmax;
}

// Sum over the 64 lanes of a wave (every lane gets the total).
__device__ __forceinline__ int wave_sum(int v)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    return v;
}

// Gather mode: lists the live pixels of ranks [row0, row_end) of group g
// (live pixels in ascending pixel order, Sec. IV-B's output-bitmap-driven
// address generation) into pix_s[0, row_end - row0), straight from the
// footprint, so no list has to be built by an earlier launch.  An exclusive
// scan of the preparation launch's 256-pixel block counts over the threads
// locates the block holding rank row0; from there the workgroup tests NT
// pixels at a time: wave ballots and popcounts rank each live pixel, and
// those inside the range are stored.  scr: 64 ints of LDS.  Called by the
// whole workgroup; every loop bound is uniform.
template <int NT>
__device__ void gather_list(const DataParams& p, int G, int g, int row0, int row_end, int* pix_s, int* scr)
{
    constexpr int NWV = NT / 64;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // (a) the block holding rank row0: each thread sums a contiguous run of
    // block counts (loads of up to 8 in flight), then an exclusive scan
    const int32_t* bc = p.blk_counts + (int64_t)g * p.nblk;
    const int per = (p.nblk + NT - 1) / NT;
    const int b0 = min(p.nblk, tid * per), b1 = min(p.nblk, b0 + per);
    int cnt = 0;
    for (int b = b0; b < b1; b += 8) {
        int v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = b + u < b1 ? bc[b + u] : 0;
#pragma unroll
        for (int u = 0; u < 8; ++u) cnt += v[u];
    }
    int incl = cnt;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int v = __shfl_up(incl, off, 64);
        if (lane >= off) incl += v;
    }
    if (lane == 63) scr[wave] = incl;
    __syncthreads();
    int run = incl - cnt;
    for (int w = 0; w < wave; ++w) run += scr[w];
    if (run <= row0 && row0 < run + cnt) {
        // this thread's run holds rank row0 (exactly one thread's does)
        for (int b = b0; b < b1; ++b) {
            const int c = bc[b];
            if (row0 < run + c) {
                scr[16] = b * kCompactThreads;
                scr[17] = run;
                break;
            }
            run += c;
        }
    }
    __syncthreads();
    // (b) rank the pixels from that block on until rank row_end is passed
    int px0 = scr[16], base = scr[17], buf = 0;
    const uint64_t below = lane == 0 ? 0ull : ((~0ull) >> (64 - lane));
    while (base < row_end && px0 < p.npix) {
        const int px = px0 + tid;
        const bool live = pixel_live_bits(p.mask, p.npix, p.C, G, px, g);
        const uint64_t bal = __ballot(live);
        if (lane == 0) scr[32 + buf * NWV + wave] = __popcll(bal);
        __syncthreads();
        int wb = 0, tot = 0;
#pragma unroll
        for (int w = 0; w < NWV; ++w) {
            const int v = scr[32 + buf * NWV + w];
            if (w < wave) wb += v;
            tot += v;
        }
        const int rank = base + wb + __popcll(bal & below);
        if (live && rank >= row0 && rank < row_end) pix_s[rank - row0] = px;
        base += tot;
        px0 += NT;
        buf ^= 1;   // the next round's counts go to the other half (no barrier needed before writing them)
    }
}

template <typename T, int MODE, bool UNIT, int TI>
__global__ __launch_bounds__(Tile<TI>::NT) void bwd_data_kernel(DataParams p)
{
    using TL = Tile<TI>;
    constexpr int BM = TL::BM, BN = TL::BN, WN = TL::WN, NW = TL::NW;
    constexpr int TM = TL::TM, FM = TL::FM, FN = TL::FN, IA = TL::IA, IB = TL::IB;
    constexpr int NT = TL::NT;
    constexpr int E = Elem<T>::E;
    constexpr int BK = CH * E;     // reduction elements per step
    constexpr uint32_t ESZ = sizeof(T);

    // the operand buffers, one array: after the main loop the bf16
    // epilogue stages the output tile in it
    __shared__ uint4 AB[2 * BM * CH + 2 * BN * CH];
    static_assert(sizeof(AB) >= 16384, "the tail reduction's group sums fit the operand buffers");
    if constexpr (NT == 1024) {
        // tail workgroups: four blocks of the weight gradient's split-K
        // reduction each (dispatched after every GEMM workgroup, they fill
        // the CUs the GEMM's last round leaves idle)
        if ((int)blockIdx.x >= p.gemm_grid) {
            splitk_reduce_quad(p.dw_red, (int)blockIdx.x - p.gemm_grid, AB);
            return;
        }
    }
    uint4 (*const As)[BM * CH] = reinterpret_cast<uint4 (*)[BM * CH]>(AB);
    uint4 (*const Bs)[BN * CH] = reinterpret_cast<uint4 (*)[BN * CH]>(AB + 2 * BM * CH);
    __shared__ int pix_s[BN];
    constexpr bool SEL = MODE == MODE_SELECT || MODE == MODE_GATHER;   // footprint select in the epilogue
    // footprint words, BM/32 per pixel row.  bf16: copied straight into LDS
    // with step 0's copies (rows unpadded: the staged epilogue reads 16
    // consecutive words per store instruction; room for every copy lane, past
    // the tile's words too).  fp32: fetched into registers and staged after
    // the main loop, rows padded by a word so that the epilogue's 16 lanes
    // reading one word column hit 16 different banks.
    constexpr int MSTR = sizeof(T) == 2 ? BM / 32 : BM / 32 + 1;
    constexpr int MSLOTS = SEL ? (sizeof(T) == 2 ? (BN * (BM / 32) + NT - 1) / NT * NT : BN * MSTR) : 1;
    __shared__ uint32_t msk_s[MSLOTS];
    // footprint nibble (4 channels) -> masks of two bf16 pairs, for the
    // staged epilogue
    __shared__ uint2 mtab[16];
    if (SEL && sizeof(T) == 2 && threadIdx.x < 16) {
        const uint32_t t = threadIdx.x;
        auto half = [](uint32_t b) { return b ? 0xffffu : 0u; };
        mtab[t] = make_uint2(half(t & 1) | (half(t & 2) << 16), half(t & 4) | (half(t & 8) << 16));
    }

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    int wm, wn;
    wave_coords<WN>(wave, wm, wn);

    // Work items are (tile, reduction split).  When the tiles are few
    // against the resident workgroups, each tile's reduction (taps x channel
    // chunks) is split S ways and the partial tiles are summed afterwards
    // (splitk_data_reduce_kernel); every workgroup derives the same S.
    //
    // Gather mode speculates: it first takes the dense mode's tiles, which
    // are exactly its own when every pixel of every group is live (the usual
    // case for element-wise footprints), and issues their first copies at
    // once; when the preparation launch flagged a dead pixel, the copies are
    // dropped and the tiles are rebuilt over the live lists.
    const int kchunks = (p.K + (CH * Elem<T>::E) - 1) / (CH * Elem<T>::E);
    const int nsteps = p.R * p.S * kchunks;
    constexpr int GG = MODE == MODE_GATHER ? kGatherMaxGroups : 1;
    __shared__ int gsum_s[GG * NW];
    __shared__ int gtot_s[GG];
    __shared__ int gscr_s[MODE == MODE_GATHER ? 64 : 1];

    const u32x4_t rs_wt = make_rsrc_words(p.wt, p.wt_bytes);
    const u32x4_t rs_dy = make_rsrc_words(p.dy, p.dy_bytes);
    const int wave_u = __builtin_amdgcn_readfirstlane(wave);
    const bool kfull = (p.K % BK) == 0;
    // Staging: every wave copies whole groups of 8 LDS rows (1 KB) straight
    // from global memory into LDS.  Row group g = wave + NW*j; lane l serves
    // row 8g + l/8 at physical chunk l%8, i.e. logical chunk (l%8) ^ swz(row).
    const int lrow8 = lane >> 3, pch = lane & 7;

    // The work item of this workgroup and everything derived from it.
    int nsplit = 1, brows = 0, item = 0, z = 0, ctile = 0, ptile = 0, c0 = 0, row0 = 0;
    int fnw = 0, wrow0 = 0, nrows = 0, st_begin = 0, nloc = 0;
    bool active = false, listed = false;
    uint32_t a_off[IA];   // A: byte offset without the step part, kOOB when no such channel
    int a_lc[IA];
    auto map_item = [&](bool dense_rule) {
        int ntiles;
        if (dense_rule) {
            brows = p.brows;
            ntiles = p.ptiles * p.ctiles;
            nsplit = p.split;
        } else {
            // values read from LDS are per-lane to the compiler: made scalar
            // here, or everything derived from them (the step range, the tap
            // walk of the main loop) would be carried in vector registers
            brows = __builtin_amdgcn_readfirstlane(gather_rows<BN>(gtot_s, p.ctiles, p.nslots, p.ptiles * p.ctiles));
            ntiles = 0;
            for (int g = 0; g < p.ctiles; ++g) ntiles += (gtot_s[g] + brows - 1) / brows;
            ntiles = __builtin_amdgcn_readfirstlane(ntiles);
            nsplit = data_split(ntiles, nsteps, p.nslots, p.smax);
        }
        // The grid may hold more workgroups than items (gather mode sizes it
        // for the most tiles any row choice gives); the surplus has no item,
        // and the XCD remap runs over the items alone so that every XCD gets
        // its share.
        const int nitems = ntiles * nsplit;
        active = (int)blockIdx.x < nitems;   // uniform across the workgroup
        if (!active) return;
        item = xcd_remap(blockIdx.x, nitems);
        const int tile = item / nsplit;
        z = item - tile * nsplit;
        if (dense_rule) {
            ptile = tile / p.ctiles;
            ctile = tile - ptile * p.ctiles;
        } else {
            gather_tile(gtot_s, p.ctiles, brows, tile, ctile, ptile);
            ctile = __builtin_amdgcn_readfirstlane(ctile);
            ptile = __builtin_amdgcn_readfirstlane(ptile);
        }
        c0 = ctile * BM;
        row0 = ptile * brows;
        // The tile's brows / 16 pixel blocks are shared out among the WN
        // pixel columns of waves as evenly as possible: this wave's column
        // covers fnw blocks (FN or FN - 1) from row wrow0.
        const int nblk16 = brows >> 4;
        const int fn_base = nblk16 / WN, fn_rem = nblk16 - fn_base * WN;
        fnw = __builtin_amdgcn_readfirstlane(fn_base + (wn < fn_rem ? 1 : 0));
        wrow0 = 16 * (wn * fn_base + (wn < fn_rem ? wn : fn_rem));
        nrows = dense_rule ? p.npix : __builtin_amdgcn_readfirstlane(gtot_s[ctile]);
        listed = !dense_rule && nrows < p.npix;
        st_begin = (int)((int64_t)z * nsteps / nsplit);
        nloc = (int)((int64_t)(z + 1) * nsteps / nsplit) - st_begin;
#pragma unroll
        for (int j = 0; j < IA; ++j) {
            const int row = 8 * (wave + NW * j) + lrow8;
            const int lc = pch ^ swz8(row);
            const int c = c0 + row;
            a_lc[j] = lc;
            a_off[j] = (row < BM && c < p.C) ? (uint32_t)(c * p.K + lc * E) * ESZ : kOOB;
        }
    };

    // Queue the copies of step (tap, k0) into LDS buffer `buf`.  The A part
    // (filters) does not depend on the pixel list, so step 0's is issued
    // before the list is read.
    auto load_a = [&](int buf, int tap, int k0) {
        const uint32_t a_step = (uint32_t)((tap * p.C) * p.K + k0) * ESZ;
#pragma unroll
        for (int j = 0; j < IA; ++j) {
            const int g = wave + NW * j;
            if (IA * NW * 8 == BM || g * 8 < BM) {
                const bool kin = kfull || (k0 + a_lc[j] * E < p.K);
                buf_load16_lds(rs_wt, kin ? a_off[j] + a_step : kOOB,
                               lds_addr(&As[buf][(wave_u + NW * j) * 8 * CH]));
            }
        }
    };

    int bn_[IB], bh_[IB], bw_[IB], bbase[IB], b_lc[IB];
    uint32_t b_off[IB];   // B byte offset for the current tap, kOOB when the tap misses
    int ld_tap = 0, ld_kc = 0;  // next step to load

    auto set_tap = [&](int tap) {
        const int r = tap / p.S, s = tap - r * p.S;
        if (UNIT) {
            const int delta = ((p.pad_h - r) * p.Q + (p.pad_w - s)) * p.K;
#pragma unroll
            for (int j = 0; j < IB; ++j) {
                const int hh = bh_[j] + p.pad_h - r, ww = bw_[j] + p.pad_w - s;
                const bool ok = bn_[j] >= 0 && hh >= 0 && hh < p.P && ww >= 0 && ww < p.Q;
                b_off[j] = ok ? (uint32_t)(bbase[j] + delta) * ESZ : kOOB;
            }
        } else {
#pragma unroll
            for (int j = 0; j < IB; ++j) {
                b_off[j] = kOOB;
                const int hh = bh_[j] + p.pad_h - r, ww = bw_[j] + p.pad_w - s;
                if (bn_[j] < 0 || hh < 0 || ww < 0) continue;
                if (hh % p.stride_h || ww % p.stride_w) continue;
                const int pp = hh / p.stride_h, qq = ww / p.stride_w;
                if (pp >= p.P || qq >= p.Q) continue;
                b_off[j] = (uint32_t)(((bn_[j] * p.P + pp) * p.Q + qq) * p.K + b_lc[j] * E) * ESZ;
            }
        }
    };

    auto load_b = [&](int buf, int k0) {
        const uint32_t b_step = (uint32_t)k0 * ESZ;
#pragma unroll
        for (int j = 0; j < IB; ++j) {
            const int g = wave_u + NW * j;
            if (g * 8 < brows) {
                const bool kin = kfull || (k0 + b_lc[j] * E < p.K);
                buf_load16_lds(rs_dy, kin ? b_off[j] + b_step : kOOB,
                               lds_addr(&Bs[buf][(wave_u + NW * j) * 8 * CH]));
            }
        }
    };
    auto load = [&](int buf) {
        if (ld_kc == 0) set_tap(ld_tap);
        const int k0 = ld_kc * BK;
        load_a(buf, ld_tap, k0);
        load_b(buf, k0);
        if (++ld_kc == kchunks) { ld_kc = 0; ++ld_tap; }
    };

    floatx4 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

    // NB: the wave's pixel blocks (fnw, a compile-time FN or FN - 1)
    auto compute = [&](int buf, auto nb_tag) {
        constexpr int NB = decltype(nb_tag)::value;
#pragma unroll
        for (int kc = 0; kc < CH / 4; ++kc) {
            const int chl = kc * 4 + (lane >> 4);
            uint4 fa[FM], fb[NB];
#pragma unroll
            for (int i = 0; i < FM; ++i) {
                const int row = wm * TM + i * 16 + (lane & 15);
                fa[i] = As[buf][row * CH + (chl ^ swz8(row))];
            }
#pragma unroll
            for (int j = 0; j < NB; ++j) {
                const int row = wrow0 + j * 16 + (lane & 15);
                fb[j] = Bs[buf][row * CH + (chl ^ swz8(row))];
            }
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < NB; ++j) acc[i][j] = mfma_chunk(acc[i][j], fa[i], fb[j], T{});

        }
    };

    // Footprint words of the tile (pixel row x 32-channel word, valid when
    // every pixel's group of BM channels starts on a word).  Only the
    // epilogue needs them: they are fetched together with step 0's copies
    // (their latency hides under the copies').  bf16: direct-to-LDS copies
    // of one word per lane, complete once step 0's copies are (the waits
    // count every copy); fp32: held in registers through the main loop and
    // staged in LDS after it.  (Fetching them next to step 1's copies
    // instead measured 1.5 us slower per launch.)
    bool mask_lds = false;
    constexpr int MW = SEL ? BN * (BM / 32) : 0;                  // footprint words per tile
    constexpr int MI = MW > 0 ? (MW + NT - 1) / NT : 1;          // per thread
    constexpr bool MDMA = sizeof(T) == 2;
    uint32_t mwords[MDMA ? 1 : MI];
    auto fetch_mask = [&]() {
        if constexpr (MDMA) {
            const u32x4_t rs_m = make_rsrc_words(p.mask, (uint32_t)(((int64_t)p.npix * p.C + 31) / 32 * 4));
#pragma unroll
            for (int u = 0; u < MI; ++u) {
                const int i = tid + u * NT;   // the copy lanes past the tile's words fill msk_s's slack
                uint32_t off = kOOB;
                if (i < MW) {
                    const int pr = i / (BM / 32), wi = i - pr * (BM / 32);
                    const int pix = pix_s[pr];
                    if (pix >= 0 && c0 + 32 * wi < p.C) off = (uint32_t)(((int64_t)pix * p.C + c0) / 32 + wi) * 4u;
                }
                buf_load4_lds(rs_m, off, lds_addr(msk_s) + 4u * (uint32_t)(u * NT + wave_u * 64));
            }
        } else {
#pragma unroll
            for (int u = 0; u < MI; ++u) {
                const int i = tid + u * NT;
                uint32_t word = 0;
                if (i < MW) {
                    const int pr = i / (BM / 32), wi = i - pr * (BM / 32);
                    const int pix = pix_s[pr];
                    if (pix >= 0 && c0 + 32 * wi < p.C) word = p.mask[((int64_t)pix * p.C + c0) / 32 + wi];
                }
                mwords[u] = word;
            }
        }
    };

    // Step 0 of the work item: the filter copies, the tile's pixel rows
    // (consecutive pixels, or in gather mode the group's live pixels of ranks
    // row0 .. row0 + brows - 1), the dY copies and the footprint words.
    auto start_item = [&]() {
        ld_tap = st_begin / kchunks;
        ld_kc = st_begin % kchunks;
        load_a(0, ld_tap, ld_kc * BK);
        for (int i = tid; i < BN; i += NT) {
            const int r = row0 + i;
            pix_s[i] = (!listed && i < brows && r < nrows) ? r : -1;
        }
        if (listed) gather_list<NT>(p, BM, ctile, row0, min(row0 + brows, nrows), pix_s, gscr_s);
        __syncthreads();
        if (listed) {
            // the rows' pixels, for the split reduction and the list readers
            const int n = min(brows, nrows - row0);
            for (int i = tid; i < n; i += NT) p.lists[(int64_t)ctile * p.npix + row0 + i] = pix_s[i];
        }
#pragma unroll
        for (int j = 0; j < IB; ++j) {
            const int row = 8 * (wave + NW * j) + lrow8;
            const int lc = pch ^ swz8(row);
            b_lc[j] = lc;
            const int pix = row < BN ? pix_s[row] : -1;
            bn_[j] = -1; bh_[j] = 0; bw_[j] = 0;
            if (pix >= 0) {
                const uint32_t nh = fdiv((uint32_t)pix, p.div_w);
                bw_[j] = pix - (int)nh * p.W;
                const uint32_t n = fdiv(nh, p.div_h);
                bh_[j] = (int)nh - (int)n * p.H;
                bn_[j] = (int)n;
            }
            // unit stride: element offset of dY at (n, h, w) before the tap shift
            bbase[j] = ((bn_[j] * p.P + bh_[j]) * p.Q + bw_[j]) * p.K + lc * E;
        }
        set_tap(ld_tap);
        load_b(0, ld_kc * BK);
        if (++ld_kc == kchunks) { ld_kc = 0; ++ld_tap; }
        mask_lds = SEL && (p.C % 32) == 0 && nsplit == 1;
        if (mask_lds) fetch_mask();
    };

    // Gather mode: whether some group has a dead pixel, a flag per group that
    // the preparation launch raised (the reduction launch lowers it again).
    // The flags are read by one vector load per lane (lane g: group g's
    // flag), issued behind step 0's copies and complete with them, so the
    // usual case (every pixel live) pays nothing: a scalar read loop ahead of
    // the copies waited for each load before the first copy went out (1.8 us
    // per launch).
    map_item(true);
    if (active) start_item();
    uint32_t dflag = 0;
    if (MODE == MODE_GATHER) {
        const __amdgpu_buffer_rsrc_t rs_f = make_rsrc(p.dead_flags, (uint32_t)p.ctiles * 4u);
        dflag = __builtin_amdgcn_raw_buffer_load_b32(rs_f, lane < p.ctiles ? 4u * lane : kOOB, 0, 0);
    }
    wait_vmem();
    __syncthreads();
    const bool anydead = MODE == MODE_GATHER && __ballot(dflag != 0u) != 0ull;
    if (MODE == MODE_GATHER && anydead) {
        // speculation failed (the copies have landed): every group's live
        // total from the block counts (workgroup 0 also stores them for the
        // reduction kernel and the readers), then the tiles over the live lists
        for (int g = 0; g < p.ctiles; ++g) {
            const int32_t* bc = p.blk_counts + (int64_t)g * p.nblk;
            int v = 0;
            for (int i0 = 0; i0 < p.nblk; i0 += 8 * NT) {
                int c[8];   // eight loads in flight
#pragma unroll
                for (int u = 0; u < 8; ++u) c[u] = i0 + u * NT + tid < p.nblk ? bc[i0 + u * NT + tid] : 0;
#pragma unroll
                for (int u = 0; u < 8; ++u) v += c[u];
            }
            v = wave_sum(v);
            if (lane == 0) gsum_s[g * NW + wave] = v;
        }
        __syncthreads();
        if (tid < p.ctiles) {
            int tot = 0;
#pragma unroll
            for (int w = 0; w < NW; ++w) tot += gsum_s[tid * NW + w];
            gtot_s[tid] = tot;
            if (blockIdx.x == 0) p.counts[tid] = tot;
        }
        __syncthreads();
        map_item(false);
        if (active) start_item();
        wait_vmem();
        __syncthreads();
    } else if (MODE == MODE_GATHER && blockIdx.x == 0 && tid < p.ctiles) {
        p.counts[tid] = p.npix;   // every pixel live
    }
    if (!active) return;   // uniform across the workgroup
    auto main_loop = [&](auto nb_tag) {
        for (int step = 0; step < nloc; ++step) {
            const int buf = step & 1;
            if (step + 1 < nloc) load(buf ^ 1);
            compute(buf, nb_tag);
            wait_vmem();
            __syncthreads();
        }
    };
    static_assert(FN >= 2, "a wave column holds at least two pixel blocks");
    if (fnw == FN) main_loop(std::integral_constant<int, FN>{});
    else main_loop(std::integral_constant<int, FN - 1>{});

    if constexpr (!MDMA) {
        if (mask_lds) {
            // msk_s is not an operand buffer: no barrier is needed before writing it
#pragma unroll
            for (int u = 0; u < MI; ++u) {
                const int i = tid + u * NT;
                if (i < MW) {
                    const int pr = i / (BM / 32), wi = i - pr * (BM / 32);
                    msk_s[pr * MSTR + wi] = mwords[u];
                }
            }
            __syncthreads();
        }
    }

    // Epilogue: lane holds channels c0 + wm*TM + i*16 + 4*(lane/16) + v of
    // pixel row wrow0 + j*16 + lane%16, j < fnw.
    if (nsplit > 1) {
        // partial tile [item][row][channel] in fp32, reduced afterwards
        float* __restrict__ part = p.partial + (int64_t)item * BN * BM;
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            if (j >= fnw) break;   // uniform: the wave's column has fnw blocks
            const int pr = wrow0 + j * 16 + (lane & 15);
#pragma unroll
            for (int i = 0; i < FM; ++i) {
                const int cl = wm * TM + i * 16 + 4 * (lane >> 4);
                *reinterpret_cast<floatx4*>(part + (int64_t)pr * BM + cl) = acc[i][j];
            }
        }
        return;
    }
    // Stores go through a buffer descriptor: a lane whose pixel or channel
    // lies outside the tensor gets offset kOOB and the store is dropped,
    // so the epilogue has no branches.  Footprint words are read from LDS
    // in one batch first (a 16-channel block never straddles a word, so a
    // lane needs TM/32 words per pixel row).
    const __amdgpu_buffer_rsrc_t rs_dx = make_rsrc(p.dx, p.dx_bytes);
    constexpr int MWJ = TM / 32 > 0 ? TM / 32 : 1;
    uint32_t ew[FN][MWJ];
    if (sizeof(T) == 4 && mask_lds) {   // the bf16 staged epilogue reads the words itself
        static_assert(TM % 32 == 0, "wave tile must cover whole footprint words");
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            if (j >= fnw) break;   // uniform: the wave's column has fnw blocks
            const int pr = wrow0 + j * 16 + (lane & 15);
#pragma unroll
            for (int w = 0; w < MWJ; ++w) ew[j][w] = msk_s[pr * MSTR + (wm * TM) / 32 + w];
        }
    }
    // Forward: ReLU, rounding to the output type, and the footprint of the
    // stored output (bit = stored value > 0, i.e. non-zero after the ReLU)
    // in the same pass.  With the output channel count a multiple of 32 the
    // 4-bit pieces of the four lanes that cover one 32-channel word (lanes
    // l, l+16, l+32, l+48) are merged by two lane exchanges and stored as a
    // whole word; otherwise each piece is OR-ed into its word atomically
    // (those words were cleared by the preparation kernel).  Non-positive
    // and NaN sums give +0.0.
    auto fwd_epilogue = [&]() {
        static_assert(FM % 2 == 0 && TM % 32 == 0, "two 16-channel blocks per footprint word");
        const bool emit = p.out_mask != nullptr;
        const bool whole_words = (p.C % 32) == 0;
        const int q = lane >> 4;
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            if (j >= fnw) break;   // uniform: the wave's column has fnw blocks
            const int pr = wrow0 + j * 16 + (lane & 15);
            const int pix = pix_s[pr];
            const int clane = wm * TM + 4 * q;
            const uint32_t base = (uint32_t)(pix * p.C + c0 + clane) * ESZ;
            uint32_t nib[FM];
#pragma unroll
            for (int i = 0; i < FM; ++i) {
                const bool ok = pix >= 0 && c0 + clane + i * 16 < p.C;
                const uint32_t off = ok ? base + (uint32_t)(i * 16) * ESZ : kOOB;
                const floatx4 v = acc[i][j];
                const float y0 = v.x > 0.f ? v.x : 0.f, y1 = v.y > 0.f ? v.y : 0.f;
                const float y2 = v.z > 0.f ? v.z : 0.f, y3 = v.w > 0.f ? v.w : 0.f;
                uint32_t bits;
                if constexpr (sizeof(T) == 2) {
                    const uint32_t h01 = pack_bf16x2(y0, y1), h23 = pack_bf16x2(y2, y3);
                    __builtin_amdgcn_raw_buffer_store_b64(u32x2{h01, h23}, rs_dx, off, 0, 0);
                    bits = (uint32_t)((h01 & 0xffffu) != 0) | ((uint32_t)((h01 >> 16) != 0) << 1) |
                           ((uint32_t)((h23 & 0xffffu) != 0) << 2) | ((uint32_t)((h23 >> 16) != 0) << 3);
                } else {
                    const u32x4 d = {__float_as_uint(y0), __float_as_uint(y1), __float_as_uint(y2), __float_as_uint(y3)};
                    __builtin_amdgcn_raw_buffer_store_b128(d, rs_dx, off, 0, 0);
                    bits = (uint32_t)(y0 > 0.f) | ((uint32_t)(y1 > 0.f) << 1) | ((uint32_t)(y2 > 0.f) << 2) |
                           ((uint32_t)(y3 > 0.f) << 3);
                }
                nib[i] = ok ? bits : 0u;
            }
            if (!emit) continue;
            if (whole_words) {
#pragma unroll
                for (int w = 0; w < FM / 2; ++w) {
                    uint32_t x = (nib[2 * w] << (4 * q)) | (nib[2 * w + 1] << (16 + 4 * q));
                    x |= __shfl_xor(x, 16);
                    x |= __shfl_xor(x, 32);
                    const int cw = c0 + wm * TM + 32 * w;
                    if (q == 0 && pix >= 0 && cw < p.C) p.out_mask[((int64_t)pix * p.C + cw) >> 5] = x;
                }
            } else {
#pragma unroll
                for (int i = 0; i < FM; ++i) {
                    if (nib[i] == 0) continue;
                    const int64_t o = (int64_t)pix * p.C + c0 + clane + i * 16;
                    atomicOr(&p.out_mask[o >> 5], nib[i] << (o & 31));
                }
            }
        }
    };

    // One straight-line body per footprint source (words staged in LDS, or
    // read per element when C is not a multiple of 32); the choice is
    // uniform across the workgroup.
    auto epilogue = [&](auto lds_tag) {
        constexpr bool LDSW = decltype(lds_tag)::value;
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            if (j >= fnw) break;   // uniform: the wave's column has fnw blocks
            const int pr = wrow0 + j * 16 + (lane & 15);
            const int pix = pix_s[pr];
            const int clane = wm * TM + 4 * (lane >> 4);   // first channel of the lane's block, i = 0
            const uint32_t base = (uint32_t)(pix * p.C + c0 + clane) * ESZ;
#pragma unroll
            for (int i = 0; i < FM; ++i) {
                const int cl = clane + i * 16;
                const bool ok = pix >= 0 && c0 + cl < p.C;
                const uint32_t off = ok ? base + (uint32_t)(i * 16) * ESZ : kOOB;
                uint32_t keep = 0xfu;
                if (SEL) {
                    if constexpr (LDSW) {
                        keep = (ew[j][(i * 16) / 32] >> (cl & 31)) & 0xfu;
                    } else {
                        const int64_t o = ok ? (int64_t)pix * p.C + c0 + cl : 0;
                        keep = (p.mask[o >> 5] >> (o & 31)) & 0xfu;
                    }
                }
                const floatx4 v = acc[i][j];
                if constexpr (sizeof(T) == 2) {
                    const uint32_t m01 = ((0u - (keep & 1u)) & 0xffffu) | ((0u - ((keep >> 1) & 1u)) & 0xffff0000u);
                    const uint32_t m23 = ((0u - ((keep >> 2) & 1u)) & 0xffffu) | ((0u - ((keep >> 3) & 1u)) & 0xffff0000u);
                    const u32x2 d = {pack_bf16x2(v.x, v.y) & m01, pack_bf16x2(v.z, v.w) & m23};
                    __builtin_amdgcn_raw_buffer_store_b64(d, rs_dx, off, 0, 0);
                } else {
                    const u32x4 d = {__float_as_uint(v.x) & (0u - (keep & 1u)),
                                     __float_as_uint(v.y) & (0u - ((keep >> 1) & 1u)),
                                     __float_as_uint(v.z) & (0u - ((keep >> 2) & 1u)),
                                     __float_as_uint(v.w) & (0u - ((keep >> 3) & 1u))};
                    __builtin_amdgcn_raw_buffer_store_b128(d, rs_dx, off, 0, 0);
                }
            }
        }
    };
    // bf16 with the footprint words staged (or none needed): the tile's
    // rounded outputs go into LDS by fragment (pixel row pr of SROW bytes,
    // 8 bytes per lane and channel block), then out by whole 16-byte row
    // pieces, 1 KB per store instruction, with the footprint applied to
    // each piece (one byte of a staged word, widened through mtab): every
    // tile row is BM consecutive channels of one pixel, so each
    // instruction writes whole 128-byte lines (the fragments' own stores
    // would write 32-byte pieces of 16 rows each).
    auto staged_epilogue = [&]() {
        constexpr int SROW = 2 * BM + 16;   // padded: the 16 rows of a fragment write spread over the banks
        static_assert(BN * SROW <= (int)sizeof(AB), "the output tile fits the operand buffers");
        char* const stage = reinterpret_cast<char*>(AB);
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            if (j >= fnw) break;   // uniform: the wave's column has fnw blocks
            const int pr = wrow0 + j * 16 + (lane & 15);
            const int clane = wm * TM + 4 * (lane >> 4);
#pragma unroll
            for (int i = 0; i < FM; ++i) {
                const int cl = clane + i * 16;
                const floatx4 v = acc[i][j];
                *reinterpret_cast<uint2*>(stage + pr * SROW + 2 * cl) =
                    make_uint2(pack_bf16x2(v.x, v.y), pack_bf16x2(v.z, v.w));
            }
        }
        __syncthreads();
        // lane l of a store instruction: row l / (BM / 8), 16-byte piece l % (BM / 8)
        constexpr int PPR = BM / 8, RPI = 64 / PPR;
        const int prow = lane / PPR, piece = lane - prow * PPR;
        const bool cin = c0 + 8 * piece < p.C;
        for (int r0 = wave_u * RPI; r0 < BN; r0 += NW * RPI) {
            const int row = r0 + prow;
            const int pix = pix_s[row];
            const uint32_t off = (pix >= 0 && cin) ? (uint32_t)(pix * p.C + c0 + 8 * piece) * ESZ : kOOB;
            uint4 v = *reinterpret_cast<const uint4*>(stage + row * SROW + 16 * piece);
            if (SEL) {
                const uint32_t byte = (msk_s[row * MSTR + piece / 4] >> (8 * (piece & 3))) & 0xffu;
                const uint2 k0 = mtab[byte & 15u], k1 = mtab[byte >> 4];
                v.x &= k0.x; v.y &= k0.y; v.z &= k1.x; v.w &= k1.y;
            }
            __builtin_amdgcn_raw_buffer_store_b128(u32x4{v.x, v.y, v.z, v.w}, rs_dx, off, 0, 0);
        }
    };
    if constexpr (MODE == MODE_FWD) {
        fwd_epilogue();
        return;
    } else if constexpr (sizeof(T) == 2) {
        if (MODE == MODE_DENSE || mask_lds) staged_epilogue();
        else epilogue(std::false_type{});
    } else {
        if (MODE == MODE_DENSE || mask_lds) epilogue(std::true_type{});
        else epilogue(std::false_type{});
    }
}

// Wt[tap][c][k] = W[k][tap][c] (KRSC) or W[k][c][tap] (KCRS).  Threads run
// along k (coalesced stores); a KRSC thread reads one 16-byte vector of E
// channels, a KCRS thread the R*S taps of one (k, c).  Returns after its part.
template <typename T>
__device__ __forceinline__ void transform_filters(const T* __restrict__ w, T* __restrict__ wt, int K, int C, int RS,
                                                  int krsc, int64_t t)
{
    constexpr int E = Elem<T>::E;
    if (krsc) {
        const int CV = C / E;
        if (t >= (int64_t)K * RS * CV) return;
        const int k = (int)(t % K);
        const int64_t rest = t / K;
        const int cv = (int)(rest % CV);
        const int tap = (int)(rest / CV);
        const uint4 v = *reinterpret_cast<const uint4*>(w + ((int64_t)k * RS + tap) * C + cv * E);
        const T* e = reinterpret_cast<const T*>(&v);
#pragma unroll
        for (int i = 0; i < E; ++i) wt[((int64_t)tap * C + cv * E + i) * K + k] = e[i];
    } else {
        if (t >= (int64_t)K * C) return;
        const int k = (int)(t % K);
        const int c = (int)(t / K);
        for (int tap = 0; tap < RS; ++tap) wt[((int64_t)tap * C + c) * K + k] = w[((int64_t)k * C + c) * RS + tap];
    }
}

// One launch for the preparation of the data gradient (and, in the call
// that computes both gradients, of the weight gradient): blocks [0, ntb)
// transform the filters (block 0 also stamps the workspace header), the next
// ncb blocks (gather mode) count the live pixels of one compaction block each
// and clear the dX rows of its dead pixels, and the rest compute the dY
// block occupancy of the weight gradient.
template <typename T>
__global__ __launch_bounds__(256) void data_prep_kernel(const T* __restrict__ w, T* __restrict__ wt, int K, int C,
                                                        int RS, int krsc, int* header, int mode, int ntb,
                                                        CompactParams cp, int ncb, OccParams op)
{
    if ((int)blockIdx.x < ntb) {
        if (blockIdx.x == 0 && threadIdx.x == 0) header[0] = mode;
        transform_filters<T>(w, wt, K, C, RS, krsc, (int64_t)blockIdx.x * 256 + threadIdx.x);
        return;
    }
    const int b = blockIdx.x - ntb;
    if (b < ncb) {
        compact_count_block(cp, b % cp.nblk, b / cp.nblk);
        return;
    }
    occupancy_block(op, b - ncb);
}

// Forward preparation (launch_fwd_prep).  Blocks [0, ntb) build the GEMM
// operand Wf[tap'][k][c] = W[k][tap][c] with tap' = (R-1-r)*S + (S-1-s): a
// KRSC thread moves one 16-byte vector of E channels of (k, tap) (coalesced
// on both sides), a KCRS thread the R*S taps of one (k, c).  The remaining
// blocks clear zero_words footprint words.
template <typename T>
__global__ __launch_bounds__(256) void fwd_prep_kernel(const T* __restrict__ w, T* __restrict__ wt, int K, int C,
                                                       int R, int S, int krsc, int* header, uint32_t* zero,
                                                       int64_t zero_words, int ntb)
{
    constexpr int E = Elem<T>::E;
    const int RS = R * S;
    if ((int)blockIdx.x < ntb) {
        if (blockIdx.x == 0 && threadIdx.x == 0) header[0] = MODE_FWD;
        const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
        if (krsc) {
            const int CV = C / E;
            if (t >= (int64_t)K * RS * CV) return;
            const int cv = (int)(t % CV);
            const int64_t rest = t / CV;
            const int tap = (int)(rest % RS);
            const int k = (int)(rest / RS);
            const int r = tap / S, s = tap - r * S;
            const int tf = (R - 1 - r) * S + (S - 1 - s);
            *reinterpret_cast<uint4*>(wt + ((int64_t)tf * K + k) * C + cv * E) =
                *reinterpret_cast<const uint4*>(w + ((int64_t)k * RS + tap) * C + cv * E);
        } else {
            if (t >= (int64_t)K * C) return;
            const int c = (int)(t % C);
            const int k = (int)(t / C);
            for (int tap = 0; tap < RS; ++tap) {
                const int r = tap / S, s = tap - r * S;
                const int tf = (R - 1 - r) * S + (S - 1 - s);
                wt[((int64_t)tf * K + k) * C + c] = w[((int64_t)k * C + c) * RS + tap];
            }
        }
        return;
    }
    const int64_t stride = (int64_t)(gridDim.x - ntb) * 256;
    for (int64_t i = (int64_t)(blockIdx.x - ntb) * 256 + threadIdx.x; i < zero_words; i += stride) zero[i] = 0u;
}

// Sums the nsplit partial tiles of every live tile in split order and writes
// dX like the GEMM epilogue would (footprint select, rounding).  Runs with a
// fixed grid; exits at once when the GEMM did not split.
constexpr int kMaxDataSplit = 16;   // the planner's kDataMaxSplit (checked at dispatch)

template <typename T, int MODE, int TI>
__device__ __forceinline__ void data_reduce_block(const DataParams& p, int block, int nblocks)
{
    constexpr int BM = Tile<TI>::BM, BN = Tile<TI>::BN;
    constexpr int E = Elem<T>::E;
    const int kchunks = (p.K + CH * E - 1) / (CH * E);
    const int nsteps = p.R * p.S * kchunks;
    // the GEMM has read the dead-pixel flags: lower them for the next call
    if (MODE == MODE_GATHER && block == 0 && (int)threadIdx.x < p.ctiles) p.dead_flags[threadIdx.x] = 0;
    int ntiles, nsplit;
    bool dense_map = MODE != MODE_GATHER;   // gather mode with every pixel live tiles like the dense mode
    if (MODE == MODE_GATHER) {
        ntiles = 0;
        bool all = true;
        for (int g = 0; g < p.ctiles; ++g) {
            ntiles += (p.counts[g] + BN - 1) / BN;
            all &= p.counts[g] == p.npix;
        }
        nsplit = data_split(ntiles, nsteps, p.nslots, p.smax);
        dense_map = all;
    } else {
        ntiles = p.ptiles * p.ctiles;
        nsplit = p.split;
    }
    // A split reduction only happens with full BN-row tiles (data_rows_pick
    // keeps BN whenever 2 * tiles <= slots), so tiles are counted at BN here.
    if (nsplit <= 1) return;
    const int64_t nvec = (int64_t)ntiles * BN * (BM / 4);
    T* __restrict__ dx = reinterpret_cast<T*>(p.dx);
    for (int64_t v = (int64_t)block * 256 + threadIdx.x; v < nvec; v += (int64_t)nblocks * 256) {
        const int tile = (int)(v / (BN * (BM / 4)));
        const int rem = (int)(v - (int64_t)tile * BN * (BM / 4));
        const int pr = rem / (BM / 4), cl = (rem - pr * (BM / 4)) * 4;
        int ctile, ptile;
        if (!dense_map) {
            gather_tile(p.counts, p.ctiles, BN, tile, ctile, ptile);
        } else {
            ptile = tile / p.ctiles;
            ctile = tile - ptile * p.ctiles;
        }
        const int r = ptile * BN + pr;
        const int nrows = dense_map ? p.npix : p.counts[ctile];
        const int c = ctile * BM + cl;
        if (r >= nrows || c >= p.C) continue;
        // (a fully live group's list is 0, 1, 2, ... and is not stored)
        const int pix = nrows < p.npix ? p.lists[(int64_t)ctile * p.npix + r] : r;
        const int64_t o = (int64_t)pix * p.C + c;
        // the footprint word goes out with the partials, not after their sum
        // (a second round trip per vector otherwise)
        uint32_t mword = 0u;
        if constexpr (MODE == MODE_SELECT || MODE == MODE_GATHER) mword = p.mask[o >> 5];
        // every split's partial is loaded before any is added (latency, not
        // bandwidth, bounds a serial chain of loads); the sum runs in split order
        const float* __restrict__ base = p.partial + ((int64_t)tile * nsplit * BN + pr) * BM + cl;
        floatx4 pv[kMaxDataSplit];
#pragma unroll
        for (int zz = 0; zz < kMaxDataSplit; ++zz)
            if (zz < nsplit) pv[zz] = *reinterpret_cast<const floatx4*>(base + (int64_t)zz * BN * BM);
        floatx4 s = pv[0];
#pragma unroll
        for (int zz = 1; zz < kMaxDataSplit; ++zz)
            if (zz < nsplit) s += pv[zz];
        if constexpr (MODE == MODE_FWD) {
            // ReLU, rounding and footprint bits as in the GEMM's forward epilogue
            // (the footprint words were cleared by the preparation kernel)
            const float y0 = s.x > 0.f ? s.x : 0.f, y1 = s.y > 0.f ? s.y : 0.f;
            const float y2 = s.z > 0.f ? s.z : 0.f, y3 = s.w > 0.f ? s.w : 0.f;
            uint32_t bits;
            if constexpr (sizeof(T) == 2) {
                const uint32_t h01 = pack_bf16x2(y0, y1), h23 = pack_bf16x2(y2, y3);
                *reinterpret_cast<uint2*>(dx + o) = make_uint2(h01, h23);
                bits = (uint32_t)((h01 & 0xffffu) != 0) | ((uint32_t)((h01 >> 16) != 0) << 1) |
                       ((uint32_t)((h23 & 0xffffu) != 0) << 2) | ((uint32_t)((h23 >> 16) != 0) << 3);
            } else {
                *reinterpret_cast<uint4*>(dx + o) =
                    make_uint4(__float_as_uint(y0), __float_as_uint(y1), __float_as_uint(y2), __float_as_uint(y3));
                bits = (uint32_t)(y0 > 0.f) | ((uint32_t)(y1 > 0.f) << 1) | ((uint32_t)(y2 > 0.f) << 2) |
                       ((uint32_t)(y3 > 0.f) << 3);
            }
            if (p.out_mask != nullptr && bits != 0) atomicOr(&p.out_mask[o >> 5], bits << (o & 31));
            continue;
        }
        uint32_t keep = 0xfu;
        if (MODE != MODE_DENSE) keep = (mword >> (o & 31)) & 0xfu;
        if constexpr (sizeof(T) == 2) {
            uint32_t h0 = (keep & 1u) ? f32_to_bf16_rne(s.x) : 0u;
            uint32_t h1 = (keep & 2u) ? f32_to_bf16_rne(s.y) : 0u;
            uint32_t h2 = (keep & 4u) ? f32_to_bf16_rne(s.z) : 0u;
            uint32_t h3 = (keep & 8u) ? f32_to_bf16_rne(s.w) : 0u;
            *reinterpret_cast<uint2*>(dx + o) = make_uint2(h0 | (h1 << 16), h2 | (h3 << 16));
        } else {
            uint4 u;
            u.x = (keep & 1u) ? __float_as_uint(s.x) : 0u;
            u.y = (keep & 2u) ? __float_as_uint(s.y) : 0u;
            u.z = (keep & 4u) ? __float_as_uint(s.z) : 0u;
            u.w = (keep & 8u) ? __float_as_uint(s.w) : 0u;
            *reinterpret_cast<uint4*>(dx + o) = u;
        }
    }
}

template <typename T, int MODE, int TI>
__global__ __launch_bounds__(256) void splitk_data_reduce_kernel(DataParams p)
{
    data_reduce_block<T, MODE, TI>(p, blockIdx.x, gridDim.x);
}

// Workgroups of the data gradient's split reduction: one output vector per
// thread when the dense tiling is split (the host knows that split), and at
// least one per resident GEMM workgroup, which covers gather mode's split
// (decided on the device, over at most half that many tiles) with a few
// vectors per thread.  Each vector's loads are one chain of latency, so the
// grid follows the work rather than a fixed size.
int data_reduce_blocks(const DataParams& p)
{
    int64_t nvec = 0;
    if (p.split > 1) {
        const int bm = p.tile == 0 ? Tile<0>::BM : p.tile == 1 ? Tile<1>::BM : Tile<2>::BM;
        const int bn = p.tile == 0 ? Tile<0>::BN : p.tile == 1 ? Tile<1>::BN : Tile<2>::BN;
        nvec = (int64_t)p.ptiles * p.ctiles * bn * (bm / 4);
    }
    return (int)std::max<int64_t>(p.nslots, (nvec + 255) / 256);
}

// The split reductions of both gradients in one launch (the call that
// computes both): blocks [0, dw_blocks) sum the weight gradient's split-K
// partials (G threads per output), the next dx_blocks blocks the data
// gradient's split tiles (when its reduction was split; they exit at once
// otherwise).
template <typename T>
__global__ __launch_bounds__(256) void bwd_reduce_kernel(DataParams dp, int dx_mode, int dx_blocks, ReduceParams rp)
{
    const int b = blockIdx.x;
    if (b < rp.blocks) {
        switch (rp.G) {
        case 1: splitk_reduce_block<1>(rp.part, rp.dw, rp.nsplit, rp.K, rp.RS, rp.C, rp.krsc, b); break;
        case 2: splitk_reduce_block<2>(rp.part, rp.dw, rp.nsplit, rp.K, rp.RS, rp.C, rp.krsc, b); break;
        case 4: splitk_reduce_block<4>(rp.part, rp.dw, rp.nsplit, rp.K, rp.RS, rp.C, rp.krsc, b); break;
        case 8: splitk_reduce_block<8>(rp.part, rp.dw, rp.nsplit, rp.K, rp.RS, rp.C, rp.krsc, b); break;
        default: splitk_reduce_block<16>(rp.part, rp.dw, rp.nsplit, rp.K, rp.RS, rp.C, rp.krsc, b); break;
        }
        return;
    }
    const int db = b - rp.blocks;
    if (dx_mode == MODE_GATHER) {
        if (dp.tile == 0) data_reduce_block<T, MODE_GATHER, 0>(dp, db, dx_blocks);
        else if (dp.tile == 1) data_reduce_block<T, MODE_GATHER, 1>(dp, db, dx_blocks);
        else data_reduce_block<T, MODE_GATHER, 2>(dp, db, dx_blocks);
    } else if (dx_mode == MODE_SELECT) {
        if (dp.tile == 0) data_reduce_block<T, MODE_SELECT, 0>(dp, db, dx_blocks);
        else if (dp.tile == 1) data_reduce_block<T, MODE_SELECT, 1>(dp, db, dx_blocks);
        else data_reduce_block<T, MODE_SELECT, 2>(dp, db, dx_blocks);
    } else {
        if (dp.tile == 0) data_reduce_block<T, MODE_DENSE, 0>(dp, db, dx_blocks);
        else if (dp.tile == 1) data_reduce_block<T, MODE_DENSE, 1>(dp, db, dx_blocks);
        else data_reduce_block<T, MODE_DENSE, 2>(dp, db, dx_blocks);
    }
}

}  // namespace

int data_tile_channels(int tile)
{
    return tile == 0 ? Tile<0>::BM : tile == 1 ? Tile<1>::BM : Tile<2>::BM;
}
int data_tile_pixels(int tile)
{
    return tile == 0 ? Tile<0>::BN : tile == 1 ? Tile<1>::BN : Tile<2>::BN;
}

hipError_t launch_data_prep(int dtype, const void* w, void* wt, int K, int C, int RS, int krsc, int* header,
                            int mode, const CompactParams* cp, hipStream_t stream, const OccParams* op)
{
    const int E = dtype == 1 ? 8 : 4;
    const int64_t nthreads = krsc ? (int64_t)K * RS * (C / E) : (int64_t)K * C;
    const int ntb = (int)((nthreads + 255) / 256);
    CompactParams c{};
    int ncb = 0;
    if (cp) {
        c = *cp;
        ncb = c.nblk * c.groups;
    }
    OccParams o{};
    int nob = 0;
    if (op) {
        o = *op;
        if (o.cpw < 1 || o.cpw * o.ktiles > 1024 || (o.xlive && o.cpw * o.tgroups * o.ctiles > 1024))
            return hipErrorInvalidValue;
        nob = (o.nchunks + o.cpw - 1) / o.cpw;
    }
    if (dtype == 1)
        data_prep_kernel<uint16_t><<<ntb + ncb + nob, 256, 0, stream>>>((const uint16_t*)w, (uint16_t*)wt, K, C, RS,
                                                                        krsc, header, mode, ntb, c, ncb, o);
    else
        data_prep_kernel<float><<<ntb + ncb + nob, 256, 0, stream>>>((const float*)w, (float*)wt, K, C, RS, krsc,
                                                                     header, mode, ntb, c, ncb, o);
    return hipGetLastError();
}

hipError_t launch_bwd_reduce(int dtype, int dx_mode, const DataParams& dp, bool dx_reduce, const ReduceParams& rp,
                             hipStream_t stream)
{
    const int dx_blocks = dx_reduce ? data_reduce_blocks(dp) : 0;
    const int nb = rp.blocks + dx_blocks;
    if (nb == 0) return hipSuccess;
    if (dx_reduce && (dp.tile < 0 || dp.tile >= kDataTileCount || dp.smax > kMaxDataSplit)) return hipErrorInvalidValue;
    if (dtype == 1) bwd_reduce_kernel<uint16_t><<<nb, 256, 0, stream>>>(dp, dx_mode, dx_blocks, rp);
    else bwd_reduce_kernel<float><<<nb, 256, 0, stream>>>(dp, dx_mode, dx_blocks, rp);
    return hipGetLastError();
}

hipError_t launch_fwd_prep(int dtype, const void* w, void* wt, int K, int C, int R, int S, int krsc, int* header,
                           uint32_t* zero, int64_t zero_words, hipStream_t stream)
{
    const int E = dtype == 1 ? 8 : 4;
    const int64_t nthreads = krsc ? (int64_t)K * R * S * (C / E) : (int64_t)K * C;
    const int ntb = (int)((nthreads + 255) / 256);
    const int64_t zb = (zero_words + 255) / 256;
    const int nzb = zero_words > 0 ? (int)(zb < 1024 ? zb : 1024) : 0;
    if (dtype == 1)
        fwd_prep_kernel<uint16_t><<<ntb + nzb, 256, 0, stream>>>((const uint16_t*)w, (uint16_t*)wt, K, C, R, S, krsc,
                                                                 header, zero, zero_words, ntb);
    else
        fwd_prep_kernel<float><<<ntb + nzb, 256, 0, stream>>>((const float*)w, (float*)wt, K, C, R, S, krsc, header,
                                                              zero, zero_words, ntb);
    return hipGetLastError();
}

namespace {

// GEMM (and, when the reduction may be split, the partial-tile reduction) of
// one element type, mode and tile shape.
template <typename T, int MODE, int TI>
hipError_t launch_shape(const DataParams& p, int nb, hipStream_t stream, const ProfEvents& ev, bool with_reduce)
{
    hipError_t e_launch;
    if (p.stride_h == 1 && p.stride_w == 1)
        e_launch = launch_timed(bwd_data_kernel<T, MODE, true, TI>, dim3(nb), dim3(Tile<TI>::NT), stream, ev, p);
    else
        e_launch = launch_timed(bwd_data_kernel<T, MODE, false, TI>, dim3(nb), dim3(Tile<TI>::NT), stream, ev, p);
    hipError_t e = e_launch;
    if (e != hipSuccess) return e;
    // in gather mode the split is only known on the device
    if (with_reduce && (MODE == MODE_GATHER || p.split > 1)) {
        splitk_data_reduce_kernel<T, MODE, TI><<<data_reduce_blocks(p), 256, 0, stream>>>(p);
        e = hipGetLastError();
    }
    return e;
}

template <typename T, int MODE>
hipError_t launch_mode(const DataParams& p, int nb, hipStream_t stream, const ProfEvents& ev, bool wr)
{
    if (p.tile == 0) return launch_shape<T, MODE, 0>(p, nb, stream, ev, wr);
    if (p.tile == 1) return launch_shape<T, MODE, 1>(p, nb, stream, ev, wr);
    return launch_shape<T, MODE, 2>(p, nb, stream, ev, wr);
}

template <typename T>
hipError_t launch_type(int mode, const DataParams& p, int nb, hipStream_t stream, const ProfEvents& ev, bool wr)
{
    if (mode == MODE_DENSE) return launch_mode<T, MODE_DENSE>(p, nb, stream, ev, wr);
    if (mode == MODE_SELECT) return launch_mode<T, MODE_SELECT>(p, nb, stream, ev, wr);
    if (mode == MODE_FWD) return launch_mode<T, MODE_FWD>(p, nb, stream, ev, wr);
    return launch_mode<T, MODE_GATHER>(p, nb, stream, ev, wr);
}

}  // namespace

hipError_t launch_bwd_data(int dtype, int mode, const DataParams& p, hipStream_t stream, const ProfEvents& ev,
                           bool with_reduce)
{
    // enough workgroups for every tile of the dense tiling unsplit, or for
    // nslots split items.  Gather mode fits too: with at most as many live
    // pixels per group its tiles at the dense row count are no more, its row
    // choice is capped at the dense tile count, and a split tiling has at
    // most nslots items.
    const int nb = max(p.ptiles * p.ctiles, p.nslots);
    if (nb <= 0) return hipSuccess;
    if (p.tile < 0 || p.tile >= kDataTileCount || p.smax > kMaxDataSplit) return hipErrorInvalidValue;
    // the weight gradient's reduction in tail workgroups, four 256-thread
    // blocks each
    DataParams q = p;
    q.gemm_grid = nb;
    int tail = 0;
    if (q.dw_red.blocks > 0) {
        const ReduceParams& r = q.dw_red;
        if (!r.part || !r.dw || r.nsplit < 1 || (r.G != 1 && r.G != 2 && r.G != 4 && r.G != 8 && r.G != 16) ||
            (int64_t)r.blocks * (256 / r.G) * 4 < (int64_t)r.K * r.RS * r.C)
            return hipErrorInvalidValue;
        tail = (r.blocks + 3) / 4;
    }
    return dtype == 1 ? launch_type<uint16_t>(mode, q, nb + tail, stream, ev, with_reduce)
                      : launch_type<float>(mode, q, nb + tail, stream, ev, with_reduce);
}

}  // namespace cbw
