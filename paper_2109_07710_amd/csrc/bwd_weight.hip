// Weight gradient as a split-K implicit GEMM on the gfx950 matrix cores.
//
//   dW[k, tap, c] = sum_{pix=(n,p,q)}  X[n, p*sh-ph+r, q*sw-pw+s, c] * dY[pix, k]
//
// (weight-gradient phase, Sec. IV-B).  GEMM view: M = channels c of one tap
// (A = shifted X), N = output channels k (B = dY), reduction = pixels.  Both
// operands are pixel-major in NHWC, so the reduction index is the strided
// one.  Each staging thread loads an E x E block (E pixels x E channels, one
// 16-byte vector per pixel, coalesced along channels), transposes it in
// registers and writes E vectors of E consecutive pixels into LDS, where the
// MFMA fragments then read reduction-contiguous 16-byte chunks.  Half of the
// workgroup stages X blocks, the other half dY blocks.
//
// Input sparsity (Sec. III-B): a (pixel chunk, k tile) block in which dY is
// entirely zero contributes exactly zero, so the workgroup skips its loads
// and MFMAs when the occupancy map says so.
//
// Split-K: the pixel chunks are divided among nsplit workgroups per output
// tile; each writes a float32 partial tile, reduced afterwards in a fixed
// order (deterministic).
#include <hip/hip_ext.h>

#include "common.hpp"
#include "kernels.hpp"
#include "tiles.hpp"


namespace cbw {

namespace {

constexpr int BM = CBW_DW_BM;   // channels c per tile
constexpr int BN = CBW_DW_BN;   // output channels k per tile
constexpr int WM = CBW_DW_WM, WN = CBW_DW_WN;
constexpr int NT = 64 * WM * WN;
constexpr int HT = NT / 2;      // staging threads per operand
constexpr int TM = BM / WM, TN = BN / WN;
constexpr int FM = TM / 16, FN = TN / 16;
constexpr int CH = 8;           // 16-byte chunks per LDS row (128 bytes)
constexpr int OCC_WIN = 1024;   // occupancy bytes cached per workgroup

// X-operand liveness of chunks [ch_begin, ch_begin + nwin) for a tile over
// filter taps [tap0, tap0 + ntaps) and channel tile ct: chunk i is live when
// one of its dY pixels has, at one of those taps, an X pixel inside the image
// whose channel tile holds a non-zero (xocc).  A chunk that is not live
// multiplies an all-zero X operand, so skipping it changes no sum.  Every
// writer stores 1, so concurrent stores to one byte agree.  Called by the
// whole workgroup.
__device__ void x_liveness(const WeightParams& p, int ch_begin, int nwin, int chunk_px, int tap0, int ntaps,
                           int ct, uint8_t* xlive)
{
    constexpr int U = 4;   // pixels per thread per round, their loads issued together
    const int tap_end = min(tap0 + ntaps, p.R * p.S);
    for (int i = threadIdx.x; i < nwin; i += blockDim.x) xlive[i] = 0;
    __syncthreads();
    const int total = nwin * chunk_px;
    for (int base = threadIdx.x; base < total; base += blockDim.x * U) {
        int ci[U], nn[U], pp[U], qq[U];
        bool ok[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int idx = base + u * (int)blockDim.x;
            ci[u] = idx / chunk_px;
            const int pix = (ch_begin + ci[u]) * chunk_px + (idx - ci[u] * chunk_px);
            ok[u] = idx < total && pix < p.npq;
            const uint32_t px = ok[u] ? (uint32_t)pix : 0u;
            const uint32_t nq = fdiv(px, p.div_q);
            qq[u] = (int)px - (int)nq * p.Q;
            const uint32_t n = fdiv(nq, p.div_p);
            pp[u] = (int)nq - (int)n * p.P;
            nn[u] = (int)n;
        }
        uint32_t any = 0;   // bit u: pixel u sees a non-zero X
        for (int tap = tap0; tap < tap_end; ++tap) {
            const int r = tap / p.S, s = tap - r * p.S;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int h = pp[u] * p.stride_h - p.pad_h + r, w = qq[u] * p.stride_w - p.pad_w + s;
                const bool in = ok[u] && h >= 0 && h < p.H && w >= 0 && w < p.W;
                const int64_t a = in ? ((int64_t)(nn[u] * p.H + h) * p.W + w) * p.ctiles + ct : 0;
                const uint8_t v = in ? p.xocc[a] : (uint8_t)0;
                any |= (uint32_t)(v != 0) << u;
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
            if ((any >> u) & 1u) xlive[ci[u]] = 1;
    }
    __syncthreads();
}
static_assert(BM == BN, "both operands share the staging layout");

// Chunk swizzle: bijective on 16 consecutive rows (fragment reads) and
// two-to-one on rows 8c + j, c = 0..15 (transposed block writes).
__device__ __forceinline__ int swz(int row) { return ((row >> 1) ^ (row >> 3)) & 7; }

template <typename T>
__device__ __forceinline__ void transpose_block(const uint4 (&v)[Elem<T>::E], uint4 (&u)[Elem<T>::E]);

// 8 x 8 bf16: v[e] holds channels 0..7 of pixel e; u[j] gets pixels 0..7 of
// channel j.
template <>
__device__ __forceinline__ void transpose_block<uint16_t>(const uint4 (&v)[8], uint4 (&u)[8])
{
    uint32_t d[8][4], o[8][4];
#pragma unroll
    for (int e = 0; e < 8; ++e) { d[e][0] = v[e].x; d[e][1] = v[e].y; d[e][2] = v[e].z; d[e][3] = v[e].w; }
#pragma unroll
    for (int m = 0; m < 4; ++m)           // channel pair (2m, 2m+1)
#pragma unroll
        for (int mp = 0; mp < 4; ++mp) {  // pixel pair (2mp, 2mp+1)
            const uint32_t a = d[2 * mp][m], b = d[2 * mp + 1][m];
            o[2 * m][mp] = (a & 0xffffu) | (b << 16);
            o[2 * m + 1][mp] = (a >> 16) | (b & 0xffff0000u);
        }
#pragma unroll
    for (int j = 0; j < 8; ++j) u[j] = make_uint4(o[j][0], o[j][1], o[j][2], o[j][3]);
}

// 4 x 4 fp32: a renaming.
template <>
__device__ __forceinline__ void transpose_block<float>(const uint4 (&v)[4], uint4 (&u)[4])
{
    u[0] = make_uint4(v[0].x, v[1].x, v[2].x, v[3].x);
    u[1] = make_uint4(v[0].y, v[1].y, v[2].y, v[3].y);
    u[2] = make_uint4(v[0].z, v[1].z, v[2].z, v[3].z);
    u[3] = make_uint4(v[0].w, v[1].w, v[2].w, v[3].w);
}

template <typename T>
__global__ __launch_bounds__(NT) void bwd_weight_kernel(WeightParams p)
{
    constexpr int E = Elem<T>::E;
    constexpr int BK = CH * E;                  // pixels per chunk
    constexpr int CB = BM / E;                  // channel blocks
    constexpr int NBLK = CB * (BK / E);         // E x E blocks per operand tile
    constexpr int BPT = NBLK / HT;              // blocks per staging thread
    static_assert(NBLK % HT == 0, "blocks must divide evenly");

    __shared__ uint4 As[2][BM * CH];
    __shared__ uint4 Bs[2][BN * CH];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;
    const bool stage_b = tid >= HT;             // wave-uniform role
    const int st = stage_b ? tid - HT : tid;

    const int RS = p.R * p.S;
    const int tiles = RS * p.ctiles * p.ktiles;
    const int t = xcd_remap(blockIdx.x, gridDim.x);
    const int z = t / tiles;
    int rem = t - z * tiles;
    const int kt = rem % p.ktiles;
    rem /= p.ktiles;
    const int ct = rem % p.ctiles;
    const int tap = rem / p.ctiles;
    const int r = tap / p.S, s = tap - r * p.S;
    const int c0 = ct * BM, k0 = kt * BN;

    if (blockIdx.x == 0 && tid == 0) p.header[0] = p.mode_flags;

    const int ch_begin = z * p.chunks_per_split;
    const int ch_end = min(p.nchunks, ch_begin + p.chunks_per_split);

    floatx4 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

    const T* __restrict__ x = reinterpret_cast<const T*>(p.x);
    const T* __restrict__ dy = reinterpret_cast<const T*>(p.dy);

    uint4 rg[BPT][E];
    int skipped = 0;

    const __amdgpu_buffer_rsrc_t rs_x = make_rsrc(p.x, p.x_bytes);
    const __amdgpu_buffer_rsrc_t rs_dy = make_rsrc(p.dy, p.dy_bytes);
    constexpr uint32_t ESZ = sizeof(T);

    // Staging thread st owns blocks st + bi*HT: channel block cb, pixel block pb.
    auto load = [&](int chunk) {
        const int px_base = chunk * BK;
#pragma unroll
        for (int bi = 0; bi < BPT; ++bi) {
            const int blk = st + bi * HT;
            const int cb = blk % CB, pb = blk / CB;
            const int pix0 = px_base + pb * E;
            if (stage_b) {
                const int kB = k0 + cb * E;
#pragma unroll
                for (int e = 0; e < E; ++e) {
                    const int pix = pix0 + e;
                    const bool ok = pix < p.npq && kB < p.K;
                    rg[bi][e] = buf_load16(rs_dy, ok ? (uint32_t)(pix * p.K + kB) * ESZ : kOOB);
                }
            } else {
                const int cA = c0 + cb * E;
                // decode the block's first pixel once, then step along q
                const uint32_t nq = fdiv((uint32_t)pix0, p.div_q);
                int q = pix0 - (int)nq * p.Q;
                const uint32_t nn = fdiv(nq, p.div_p);
                int pp = (int)nq - (int)nn * p.P;
                int n = (int)nn;
#pragma unroll
                for (int e = 0; e < E; ++e) {
                    const int h = pp * p.stride_h - p.pad_h + r;
                    const int w = q * p.stride_w - p.pad_w + s;
                    const bool ok = n < p.N && cA < p.C && h >= 0 && h < p.H && w >= 0 && w < p.W;
                    rg[bi][e] = buf_load16(rs_x, ok ? (uint32_t)(((n * p.H + h) * p.W + w) * p.C + cA) * ESZ : kOOB);
                    if (++q == p.Q) {
                        q = 0;
                        if (++pp == p.P) { pp = 0; ++n; }
                    }
                }
            }
        }
    };

    auto store = [&](int buf) {
        uint4* dst = stage_b ? Bs[buf] : As[buf];
#pragma unroll
        for (int bi = 0; bi < BPT; ++bi) {
            const int blk = st + bi * HT;
            const int cb = blk % CB, pb = blk / CB;
            uint4 u[E];
            transpose_block<T>(rg[bi], u);
#pragma unroll
            for (int j = 0; j < E; ++j) {
                const int row = cb * E + j;
                dst[row * CH + (pb ^ swz(row))] = u[j];
            }
        }
    };

    auto compute = [&](int buf) {
#pragma unroll
        for (int kc = 0; kc < CH / 4; ++kc) {
            const int chl = kc * 4 + (lane >> 4);
            uint4 fa[FM], fb[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i) {
                const int row = wm * TM + i * 16 + (lane & 15);
                fa[i] = As[buf][row * CH + (chl ^ swz(row))];
            }
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                const int row = wn * TN + j * 16 + (lane & 15);
                fb[j] = Bs[buf][row * CH + (chl ^ swz(row))];
            }
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j) acc[i][j] = mfma_chunk(acc[i][j], fa[i], fb[j], T{});
        }
    };

    // The occupancy bytes of this workgroup's chunk range are read once into
    // LDS (up to OCC_WIN of them); the loop then tests them without a global
    // read on its critical path.
    __shared__ uint8_t occ_s[OCC_WIN];
    __shared__ uint8_t xlive_s[OCC_WIN];
    if (p.occ) {
        for (int i = tid; i < OCC_WIN && ch_begin + i < ch_end; i += NT)
            occ_s[i] = p.occ[(int64_t)(ch_begin + i) * p.ktiles + kt];
    }
    __syncthreads();
    // Blocks whose X operand is entirely zero are skipped as well when the X
    // occupancy is given (chunks past the cached window count as X-live).
    const int nwin = min(OCC_WIN, max(ch_end - ch_begin, 0));
    if (p.xocc) x_liveness(p, ch_begin, nwin, BK, tap, 1, ct, xlive_s);
    auto live = [&](int chunk) {
        if (p.occ == nullptr) return true;
        const int i = chunk - ch_begin;
        int v = i < OCC_WIN ? occ_s[i] : p.occ[(int64_t)chunk * p.ktiles + kt];
        if (p.xocc && i < OCC_WIN) v &= xlive_s[i];
        return __builtin_amdgcn_readfirstlane(v) != 0;  // the same byte for the whole workgroup
    };
    auto next_live = [&](int chunk) {
        while (chunk < ch_end && !live(chunk)) { ++chunk; ++skipped; }
        return chunk;
    };

    int chunk = next_live(ch_begin);
    int buf = 0;
    if (chunk < ch_end) {
        load(chunk);
        store(0);
    }
    __syncthreads();
    while (chunk < ch_end) {
        const int next = next_live(chunk + 1);
        if (next < ch_end) load(next);
        compute(buf);
        if (next < ch_end) store(buf ^ 1);
        __syncthreads();
        buf ^= 1;
        chunk = next;
    }

    if (tid == 0) p.skip_slots[blockIdx.x] = skipped;

    // Epilogue: lane holds channels c0 + wm*TM + i*16 + 4*(lane/16) + v of
    // output channel k0 + wn*TN + j*16 + lane%16; written to [z][k][tap][c].
    // Buffer stores over this split's [K][RS][C] region: lanes past K or C
    // get offset kOOB and their stores are dropped (no branches).
    const uint32_t split_bytes = (uint32_t)p.K * RS * p.C * 4u;
    const __amdgpu_buffer_rsrc_t rs_out = make_rsrc(p.out + (int64_t)z * p.K * RS * p.C, split_bytes);
#pragma unroll
    for (int j = 0; j < FN; ++j) {
        const int k = k0 + wn * TN + j * 16 + (lane & 15);
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            const int c = c0 + wm * TM + i * 16 + 4 * (lane >> 4);
            const uint32_t off = (k < p.K && c < p.C) ? (uint32_t)((k * RS + tap) * p.C + c) * 4u : kOOB;
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, acc[i][j]), rs_out, off, 0, 0);
        }
    }
}

// bf16 kernel with natural-layout staging.  Both operand tiles are copied
// by the load unit straight into LDS in their NHWC order, one 512-byte row
// (256 channels) per pixel: A_s[pixel][c], B_s[pixel][k].  The MFMA fragments
// need 8 consecutive pixels of one channel per lane; ds_read_b64_tr_b16
// delivers exactly that from the natural layout: within each group of 16
// lanes, the lane at position q + 4m addresses the four channels
// cbase+4q..cbase+4q+3 of pixel k0+m, and the lane at position j receives
// channel cbase+j of pixels k0..k0+3.  Two such reads (pixels k0..k0+3 and
// k0+4..k0+7) form one 16x16x32 operand fragment.  No register transposes,
// no staging registers, no LDS store instructions.
//
// LDS rows are 32 chunks of 16 bytes; chunk c of pixel row r is stored at
// c ^ trswz(r), which makes each 32-lane half of a transpose read hit 16
// different chunk positions.
__device__ __forceinline__ int trswz(int row) { return 2 * ((row & 3) | (((row >> 3) & 1) << 2)); }

typedef short v4i16 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint2 ds_read_tr16(const void* lds)
{
    const v4i16 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4i16*)lds);
    return __builtin_bit_cast(uint2, v);
}

constexpr int TR_NT = 1024;            // 16 waves (four per SIMD): more waves hide more copy and LDS latency
constexpr int TR_BK = 64;              // pixels per step
constexpr int TR_ROW = BM / 8;         // 16-byte chunks per LDS row (one pixel)
constexpr int TR_IA = TR_BK * BM * 2 / 1024 / (TR_NT / 64);  // 1 KB copies per wave per step, per operand
static_assert(BM == 256 && BN == 256, "the natural-layout kernel assumes 256-wide rows");

// Tiling of the natural-layout kernel for BKT output channels per tile
// (256, 128 or 64): the 16 waves split the 256 channel columns WM ways and the
// BKT output channels WN ways, so every wave holds 64 output channels and
// 256/WM channel columns.  The channel columns are tpg filter taps of C
// channels each when taps are packed (C <= 128; columns past tpg*C are
// empty), else 256 channels of one tap.  dY rows keep the 512-byte LDS layout; chunks past BKT are
// copied as out-of-range zeros and never read.
template <int BKT>
struct WTile {
    static constexpr int WN = BKT / 64, WM = (TR_NT / 64) / WN;
    static constexpr int TM = BM / WM, TN = BKT / WN;
    static constexpr int FM = TM / 16, FN = TN / 16;
    static_assert(WM * WN * 64 == TR_NT && TN == 64, "64 output channels per wave");
};

template <int BKT>
__global__ __launch_bounds__(TR_NT) void bwd_weight_tr_kernel(WeightParams p)
{
    constexpr uint32_t ESZ = 2;
    constexpr int NW = TR_NT / 64;
    constexpr int WN = WTile<BKT>::WN;
    constexpr int TM = WTile<BKT>::TM, TN = WTile<BKT>::TN, FM = WTile<BKT>::FM, FN = WTile<BKT>::FN;
    __shared__ uint4 As[2][TR_BK * TR_ROW];
    __shared__ uint4 Bs[2][TR_BK * TR_ROW];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;
    const int wave_u = __builtin_amdgcn_readfirstlane(wave);

    const int RS = p.R * p.S;
    const int tiles = p.tgroups * p.ctiles * p.ktiles;
    const int t = xcd_remap(blockIdx.x, gridDim.x);
    const int z = t / tiles;
    int rem = t - z * tiles;
    const int kt = rem % p.ktiles;
    rem /= p.ktiles;
    const int ct = rem % p.ctiles;
    const int tg = rem / p.ctiles;          // tap group: taps tg*tpg .. tg*tpg + tpg - 1
    const int cg = p.cg;                    // channel columns per packed tap (a multiple of 8)
    const int c0 = ct * BM, k0 = kt * BKT;

    if (blockIdx.x == 0 && tid == 0) p.header[0] = p.mode_flags;

    const int ch_begin = z * p.chunks_per_split;
    const int ch_end = min(p.nchunks, ch_begin + p.chunks_per_split);

    const u32x4_t rs_x = make_rsrc_words(p.x, p.x_bytes);
    const u32x4_t rs_dy = make_rsrc_words(p.dy, p.dy_bytes);

    // Copy assignment: instruction j of a wave fills LDS rows 2g, 2g+1 with
    // g = wave + NW*j; lane l serves row 2g + l/32 at physical chunk l%32,
    // i.e. logical chunk (l%32) ^ trswz(row): columns 8*lc .. 8*lc+7, which
    // are channels of one tap (cg is a multiple of 8).
    int rowj[TR_IA];
    uint32_t xch[TR_IA], dych[TR_IA];   // channel byte offset, kOOB for columns past C, R*S or BKT
    int xr[TR_IA], xs[TR_IA];           // filter tap of the lane's X columns
    int xn[TR_IA], xp[TR_IA], xq[TR_IA];   // pixel coordinates of the row at the next chunk to load
    int dpix[TR_IA];
#pragma unroll
    for (int j = 0; j < TR_IA; ++j) {
        const int row = 2 * (wave + NW * j) + (lane >> 5);
        const int lc = (lane & 31) ^ trswz(row);
        rowj[j] = row;
        const int tl = (8 * lc) / cg, cc = (8 * lc) - tl * cg;
        const int tap = tg * p.tpg + tl;
        xr[j] = tap / p.S;
        xs[j] = tap - xr[j] * p.S;
        xch[j] = (tl < p.tpg && tap < RS && c0 + cc < p.C) ? (uint32_t)(c0 + cc) * ESZ : kOOB;
        dych[j] = (8 * lc < BKT && k0 + 8 * lc < p.K) ? (uint32_t)(k0 + 8 * lc) * ESZ : kOOB;
    }
    auto set_chunk = [&](int chunk) {
#pragma unroll
        for (int j = 0; j < TR_IA; ++j) {
            const int pix = chunk * TR_BK + rowj[j];
            dpix[j] = pix;
            const uint32_t nq = fdiv((uint32_t)pix, p.div_q);
            xq[j] = pix - (int)nq * p.Q;
            const uint32_t nn = fdiv(nq, p.div_p);
            xp[j] = (int)nq - (int)nn * p.P;
            xn[j] = (int)nn;
        }
    };

    auto load = [&](int buf) {
#pragma unroll
        for (int j = 0; j < TR_IA; ++j) {
            const int h = xp[j] * p.stride_h - p.pad_h + xr[j];
            const int w = xq[j] * p.stride_w - p.pad_w + xs[j];
            const bool ok = xn[j] < p.N && h >= 0 && h < p.H && w >= 0 && w < p.W && xch[j] != kOOB;
            const uint32_t xo = ok ? (uint32_t)(((xn[j] * p.H + h) * p.W + w) * p.C) * ESZ + xch[j] : kOOB;
            buf_load16_lds(rs_x, xo, lds_addr(&As[buf][(wave_u + NW * j) * 2 * TR_ROW]));
            const uint32_t yo = dpix[j] < p.npq ? (uint32_t)(dpix[j] * p.K) * ESZ + dych[j] : kOOB;
            buf_load16_lds(rs_dy, yo, lds_addr(&Bs[buf][(wave_u + NW * j) * 2 * TR_ROW]));
        }
    };

    // Per-lane transpose-read addresses (bytes within a buffer): for fragment
    // base column cb and k-step kc, lane (kg = lane/16, q = lane%4,
    // m = (lane%16)/4) reads row kc*32 + 8*kg + m (+4), columns cb+4q..+3.
    const int kg = lane >> 4, q4 = lane & 3, m4 = (lane >> 2) & 3;
    auto tr_addr = [&](int row, int cb) {
        const int col = cb + 4 * q4;
        return row * (TR_ROW * 16) + (((col >> 3) ^ trswz(row)) << 4) + ((col & 7) << 1);
    };

    floatx4 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

    auto compute = [&](int buf) {
        const char* Ab = reinterpret_cast<const char*>(As[buf]);
        const char* Bb = reinterpret_cast<const char*>(Bs[buf]);
#pragma unroll
        for (int kc = 0; kc < TR_BK / 32; ++kc) {
            const int r0 = kc * 32 + 8 * kg + m4;
            uint4 fa[FM], fb[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i) {
                const int cb = wm * TM + i * 16;
                const uint2 lo = ds_read_tr16(Ab + tr_addr(r0, cb));
                const uint2 hi = ds_read_tr16(Ab + tr_addr(r0 + 4, cb));
                fa[i] = make_uint4(lo.x, lo.y, hi.x, hi.y);
            }
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                const int cb = wn * TN + j * 16;
                const uint2 lo = ds_read_tr16(Bb + tr_addr(r0, cb));
                const uint2 hi = ds_read_tr16(Bb + tr_addr(r0 + 4, cb));
                fb[j] = make_uint4(lo.x, lo.y, hi.x, hi.y);
            }
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j) acc[i][j] = mfma_chunk(acc[i][j], fa[i], fb[j], uint16_t{});
        }
    };

    // The occupancy bytes of this workgroup's chunk range are read once into
    // LDS (up to OCC_WIN of them); the loop then tests them without a global
    // read on its critical path.
    __shared__ uint8_t occ_s[OCC_WIN];
    __shared__ uint8_t xlive_s[OCC_WIN];
    if (p.occ) {
        for (int i = tid; i < OCC_WIN && ch_begin + i < ch_end; i += TR_NT)
            occ_s[i] = p.occ[(int64_t)(ch_begin + i) * p.ktiles + kt];
    }
    __syncthreads();
    // Blocks whose X operand is entirely zero are skipped as well when the X
    // occupancy is given (chunks past the cached window count as X-live).
    const int nwin = min(OCC_WIN, max(ch_end - ch_begin, 0));
    if (p.xocc) x_liveness(p, ch_begin, nwin, TR_BK, tg * p.tpg, p.tpg, ct, xlive_s);
    auto live = [&](int chunk) {
        if (p.occ == nullptr) return true;
        const int i = chunk - ch_begin;
        int v = i < OCC_WIN ? occ_s[i] : p.occ[(int64_t)chunk * p.ktiles + kt];
        if (p.xocc && i < OCC_WIN) v &= xlive_s[i];
        return __builtin_amdgcn_readfirstlane(v) != 0;  // the same byte for the whole workgroup
    };
    int skipped = 0;
    auto next_live = [&](int chunk) {
        while (chunk < ch_end && !live(chunk)) { ++chunk; ++skipped; }
        return chunk;
    };

    int chunk = next_live(ch_begin);
    int buf = 0;
    if (chunk < ch_end) {
        set_chunk(chunk);
        load(0);
    }
    wait_vmem();
    __syncthreads();
    while (chunk < ch_end) {
        const int next = next_live(chunk + 1);
        if (next < ch_end) {
            set_chunk(next);
            load(buf ^ 1);
        }
        compute(buf);
        wait_vmem();
        __syncthreads();
        buf ^= 1;
        chunk = next;
    }

    if (tid == 0) p.skip_slots[blockIdx.x] = skipped;

    // Buffer stores over this split's [K][RS][C] region: lanes past K, C or
    // the last tap get offset kOOB and their stores are dropped (no branches).
    // A lane's 4 columns are channels of one tap (cg is a multiple of 16).
    const uint32_t split_bytes = (uint32_t)p.K * RS * p.C * 4u;
    const __amdgpu_buffer_rsrc_t rs_out = make_rsrc(p.out + (int64_t)z * p.K * RS * p.C, split_bytes);
#pragma unroll
    for (int j = 0; j < FN; ++j) {
        const int k = k0 + wn * TN + j * 16 + (lane & 15);
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            const int col = wm * TM + i * 16 + 4 * (lane >> 4);
            const int tl = col / cg, cc = col - tl * cg;
            const int tap = tg * p.tpg + tl, c = c0 + cc;
            const bool ok = k < p.K && c < p.C && tl < p.tpg && tap < RS;
            const uint32_t off = ok ? (uint32_t)((k * RS + tap) * p.C + c) * 4u : kOOB;
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, acc[i][j]), rs_out, off, 0, 0);
        }
    }
}

}  // namespace

int weight_tile_channels() { return BM; }
int weight_tile_k() { return BN; }
int weight_chunk(int dtype) { return CH * (dtype == 1 ? 8 : 4); }

hipError_t launch_bwd_weight(int dtype, const WeightParams& p, hipStream_t stream, const ProfEvents& ev)
{
    const int nb = p.tgroups * p.ctiles * p.ktiles * p.nsplit;
    const dim3 grid(nb), block(dtype == 1 ? TR_NT : NT);
    if (dtype == 1) {
        if (p.bk == 64) hipExtLaunchKernelGGL(bwd_weight_tr_kernel<64>, grid, block, 0, stream, ev.start, ev.stop, 0, p);
        else if (p.bk == 128) hipExtLaunchKernelGGL(bwd_weight_tr_kernel<128>, grid, block, 0, stream, ev.start, ev.stop, 0, p);
        else hipExtLaunchKernelGGL(bwd_weight_tr_kernel<256>, grid, block, 0, stream, ev.start, ev.stop, 0, p);
    }
    else hipExtLaunchKernelGGL(bwd_weight_kernel<float>, grid, block, 0, stream, ev.start, ev.stop, 0, p);
    return hipGetLastError();
}

}  // namespace cbw
