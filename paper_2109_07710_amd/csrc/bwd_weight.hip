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

// The chunk range [begin, end) of split z of a weight-gradient tile, with the
// liveness of its first OCC_WIN chunks cached in live_s.
//
// Without skipping the splits are equal ranges of chunks.  With skipping a
// chunk is live when its dY block holds a non-zero (occ) and, when X blocks
// are skipped too, its tap-shifted X window does (xlive).  Work
// redistribution (Sec. IV-F): the tile's live chunks are ranked in chunk
// order and split z takes the ranks [z*share, (z+1)*share), share =
// ceil(live / nsplit), so no workgroup executes more than share blocks,
// however the dead blocks cluster.  The ranges still partition all chunks
// (a dead chunk goes with the live one after it), so skip counts stay exact;
// and when every chunk is live they are the unskipped ranges, which keeps
// the two results bitwise equal.
//
// One coalesced pass over the tile's liveness (eight loads in flight per
// thread) decides the all-live case; tiles of up to TILE_LIVE_CAP chunks also
// stage their liveness in LDS in it.  Otherwise each thread then counts a
// contiguous segment of it, from LDS when staged, else from global memory (a
// bit mask for segments of up to 32 chunks).  The ranks come from a wave-level shuffle
// scan and one exchange of wave totals.  Called by the whole workgroup before
// any operand copy; scratch is SPLIT_SCRATCH_BYTES of LDS, free until the
// function returns.
constexpr int TILE_LIVE_CAP = 16384;
constexpr int SPLIT_SCRATCH_BYTES = 256 + TILE_LIVE_CAP;

//
// Returns true when the range needs no liveness tests: no skipping, or every
// chunk of the tile live.  The main loop then runs exactly as without
// skipping, with no per-step liveness probe.
__device__ bool split_range(const WeightParams& p, int kt, int combo, int z, int& begin, int& end,
                            uint8_t* live_s, uint8_t* scratch)
{
    const int nch = p.nchunks, T = blockDim.x, tid = threadIdx.x;
    if (p.occ == nullptr) {
        begin = min(nch, z * p.chunks_per_split);
        end = min(nch, begin + p.chunks_per_split);
        return true;
    }
    const int ncombo = p.tgroups * p.ctiles;
    auto live = [&](int c) -> int {
        int v = p.occ[(int64_t)c * p.ktiles + kt];
        if (p.xlive) v &= p.xlive[(int64_t)c * ncombo + combo];
        return v != 0;
    };
    // Fast test first: every byte of the occupancy map (and of the X-window
    // liveness) is 1, read 16 bytes at a time with eight loads in flight --
    // the usual case for element-wise footprints, decided with a few loads
    // per thread even for tiles of tens of thousands of chunks.
    auto all_ones = [&](const uint8_t* m, int64_t n) -> bool {
        const uint4* v = reinterpret_cast<const uint4*>(m);
        const int64_t nv = n / 16;
        bool ok = true;
        for (int64_t i0 = tid; i0 < nv; i0 += 8 * T) {
            uint4 a[8];
#pragma unroll
            for (int u = 0; u < 8; ++u)
                a[u] = i0 + u * T < nv ? v[i0 + u * T] : make_uint4(0x01010101u, 0x01010101u, 0x01010101u, 0x01010101u);
#pragma unroll
            for (int u = 0; u < 8; ++u) ok &= (a[u].x & a[u].y & a[u].z & a[u].w) == 0x01010101u;
        }
        for (int64_t i = nv * 16 + tid; i < n; i += T) ok &= m[i] == 1;
        return ok;
    };
    bool every = all_ones(p.occ, (int64_t)nch * p.ktiles);
    if (p.xlive) every &= all_ones(p.xlive, (int64_t)nch * ncombo);
    if (__syncthreads_and(every)) {
        begin = min(nch, z * p.chunks_per_split);
        end = min(nch, begin + p.chunks_per_split);
        return true;
    }
    int* wsum = reinterpret_cast<int*>(scratch);         // [0, 16): wave totals
    int* pos = wsum + 32;                                // [32, 34): chunk of ranks r0, r1
    uint8_t* tl = scratch + 256;                         // tile liveness when staged
    const bool staged = nch <= TILE_LIVE_CAP;
    const int per = (nch + T - 1) / T;
    const int s0 = min(nch, tid * per), s1 = min(nch, s0 + per);
    int cnt = 0;
    uint32_t bits = 0;   // bit i: chunk s0 + i is live (segments of up to 32 chunks)
    // one coalesced pass over the tile's liveness, eight loads in flight per
    // thread, decides the all-live case (and stages the liveness when it fits)
    bool all = true;
    for (int cb = tid; cb < nch; cb += 8 * T) {
        int v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = cb + u * T < nch ? live(cb + u * T) : 1;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            if (staged && cb + u * T < nch) tl[cb + u * T] = (uint8_t)v[u];
            all &= v[u] != 0;
        }
    }
    // every chunk live (the usual case for element-wise footprints): the
    // ranges are the unskipped ones and nothing needs ranking
    if (__syncthreads_and(all)) {
        begin = min(nch, z * p.chunks_per_split);
        end = min(nch, begin + p.chunks_per_split);
        return true;
    }
    for (int c = s0; c < s1; ++c) {
        const int v = staged ? (int)tl[c] : live(c);
        cnt += v;
        bits |= (uint32_t)v << ((c - s0) & 31);
    }
    // otherwise an inclusive scan of the counts over the threads: within
    // each wave by shuffles, then across the waves' totals
    const int lane = tid & 63, wave = tid >> 6, nw = T >> 6;
    int incl = cnt;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int v = __shfl_up(incl, off, 64);
        if (lane >= off) incl += v;
    }
    if (lane == 63) wsum[wave] = incl;
    if (tid == 0) {
        pos[0] = nch;
        pos[1] = nch;
    }
    __syncthreads();
    int total = 0;
    for (int w = 0; w < nw; ++w) {
        const int v = wsum[w];
        if (w < wave) incl += v;
        total += v;
    }
    const int excl = incl - cnt;
    const int share = (total + p.nsplit - 1) / p.nsplit;
    const int r0 = min(z * share, total), r1 = min(r0 + share, total);
    // chunk index of ranks r0 and r1 (nch past the last live chunk), found by
    // the thread whose segment holds the rank
    for (int q = 0; q < 2; ++q) {
        const int r = q == 0 ? r0 : r1;
        if (r < total && excl <= r && r < incl) {
            int k = excl;
            for (int c = s0; c < s1; ++c) {
                if (!(per <= 32 ? (int)((bits >> (c - s0)) & 1u) : live(c))) continue;
                if (k == r) {
                    pos[q] = c;
                    break;
                }
                ++k;
            }
        }
    }
    __syncthreads();
    // the bounds are the same for the whole workgroup: keep them scalar so the
    // chunk loop and its addressing stay on the scalar unit
    begin = __builtin_amdgcn_readfirstlane(z == 0 ? 0 : pos[0]);
    end = __builtin_amdgcn_readfirstlane(z == p.nsplit - 1 ? nch : pos[1]);
    const int n = min(OCC_WIN, max(end - begin, 0));
    for (int i = tid; i < n; i += T) {
        const int c = begin + i;
        live_s[i] = staged ? tl[c] : (uint8_t)live(c);
    }
    __syncthreads();
    return false;
}
// The first live chunk in [chunk, end) (end when there is none), counting the
// dead chunks passed in skipped.  Each lane tests one of 64 consecutive
// chunks and the wave's ballot names the first live one, so a long run of
// dead chunks (a balanced range can open with one) costs one probe per 64
// chunks instead of one per chunk.  Liveness of the first OCC_WIN chunks of
// the range comes from live_s, later ones from the global bytes.  Called in
// uniform control flow; every result is the same for the whole workgroup.
__device__ __forceinline__ int next_live_chunk(const WeightParams& p, const uint8_t* live_s, int begin, int end,
                                               int kt, int combo, int chunk, int& skipped)
{
    if (p.occ == nullptr) return chunk;
    const int lane = threadIdx.x & 63, ncombo = p.tgroups * p.ctiles;
    if (chunk < end && chunk - begin < OCC_WIN &&
        __builtin_amdgcn_readfirstlane((int)live_s[chunk - begin]) != 0)
        return chunk;   // the common case: the next chunk is live
    for (; chunk < end; chunk += 64) {
        const int c = chunk + lane;
        int v = 0;
        if (c < end) {
            const int i = c - begin;
            if (i < OCC_WIN) {
                v = live_s[i];
            } else {
                v = p.occ[(int64_t)c * p.ktiles + kt];
                if (p.xlive) v &= p.xlive[(int64_t)c * ncombo + combo];
            }
        }
        const uint64_t m = __ballot(v != 0);
        if (m != 0) {
            const int f = __builtin_ctzll(m);
            skipped += f;
            return chunk + f;
        }
        skipped += min(64, end - chunk);
    }
    return end;
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

    if (blockIdx.x == 0 && tid == 0) {
        p.header[0] = p.mode_flags;
        p.header[1] = 0;   // the readers' plan: 64-pixel chunks
    }

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

    // This split's chunk range (balanced over the tile's live chunks when
    // skipping), with the liveness of its first OCC_WIN chunks read once into
    // LDS so the loop tests them without a global read on its critical path.
    // The ranking scratch borrows the second operand buffer, not yet in use.
    __shared__ uint8_t live_s[OCC_WIN];
    const int combo = tap * p.ctiles + ct;
    int ch_begin, ch_end;
    static_assert(sizeof(As[1]) >= SPLIT_SCRATCH_BYTES, "ranking scratch fits the second operand buffer");
    const bool all_live = split_range(p, kt, combo, z, ch_begin, ch_end, live_s, reinterpret_cast<uint8_t*>(As[1]));
    auto next_live = [&](int chunk) {
        return all_live ? chunk : next_live_chunk(p, live_s, ch_begin, ch_end, kt, combo, chunk, skipped);
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

    if (tid == 0) {
        p.skip_slots[blockIdx.x] = skipped;
        p.work_slots[t] = ch_end - ch_begin - skipped;
    }

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
#ifndef CBW_DW_TR64_NT
#define CBW_DW_TR64_NT 1024
#endif
constexpr int TR_BK = 64;              // pixels per step
constexpr int TR_ROW = BM / 8;         // 16-byte chunks per LDS row (one pixel)
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
    static constexpr int NT = BKT == 64 ? CBW_DW_TR64_NT : TR_NT;   // threads per workgroup
    static constexpr int WN = BKT / 64, WM = (NT / 64) / WN;
    static constexpr int TM = BM / WM, TN = BKT / WN;
    static constexpr int FM = TM / 16, FN = TN / 16;
    static constexpr int IA = TR_BK * BM * 2 / 1024 / (NT / 64);  // 1 KB copies per wave per step, per operand
    static_assert(WM * WN * 64 == NT && TN == 64, "64 output channels per wave");
};

template <int BKT>
__global__ __launch_bounds__(WTile<BKT>::NT) void bwd_weight_tr_kernel(WeightParams p)
{
    constexpr uint32_t ESZ = 2;
    constexpr int NW = WTile<BKT>::NT / 64;
    constexpr int TR_IA = WTile<BKT>::IA;
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
    // Columns of this tile that hold data: the group's taps (fewer in a last,
    // short group) or the channels left in a last channel tile.  A wave whose
    // columns all lie past them has only zero operands, so it skips its
    // fragment reads and matrix instructions (it still copies and waits).
    const int used_cols = p.tpg > 1 ? min(p.tpg, RS - tg * p.tpg) * cg : min(BM, p.C - c0);

    if (blockIdx.x == 0 && tid == 0) {
        p.header[0] = p.mode_flags;
        p.header[1] = 0;   // the readers' plan: 64-pixel chunks
    }

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

    const bool wave_busy = __builtin_amdgcn_readfirstlane(wm * TM) < used_cols;
    auto compute = [&](int buf) {
        if (!wave_busy) return;
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

    // This split's chunk range (balanced over the tile's live chunks when
    // skipping), with the liveness of its first OCC_WIN chunks read once into
    // LDS so the loop tests them without a global read on its critical path.
    // The ranking scratch borrows the second operand buffer, not yet in use.
    //
    // The unskipped range's step-0 copies go out first and the call's
    // dead-block flag is read behind them: when the occupancy pass found no
    // dead block (the usual case for element-wise footprints) that range is
    // this split's range and the copies stand; otherwise the range is ranked
    // over the live chunks once the copies have landed, and step 0 copied
    // again.
    __shared__ uint8_t live_s[OCC_WIN];
    const int combo = tg * p.ctiles + ct;
    int ch_begin = min(p.nchunks, z * p.chunks_per_split);
    int ch_end = min(p.nchunks, ch_begin + p.chunks_per_split);
    static_assert(sizeof(As[1]) >= SPLIT_SCRATCH_BYTES, "ranking scratch fits the second operand buffer");
    int chunk = ch_begin;
    if (chunk < ch_end) {
        set_chunk(chunk);
        load(0);
    }
    uint32_t dflag = 0;
    if (p.occ) dflag = __builtin_amdgcn_raw_buffer_load_b32(make_rsrc(p.header, 64), 4 * kDeadWord, 0, 0);
    wait_vmem();
    __syncthreads();
    bool all_live = true;
    int skipped = 0;
    if (p.occ && __builtin_amdgcn_readfirstlane(dflag) == p.gen) {
        all_live = split_range(p, kt, combo, z, ch_begin, ch_end, live_s, reinterpret_cast<uint8_t*>(As[1]));
        chunk = all_live ? ch_begin : next_live_chunk(p, live_s, ch_begin, ch_end, kt, combo, ch_begin, skipped);
        if (chunk < ch_end) {
            set_chunk(chunk);
            load(0);
        }
        wait_vmem();
        __syncthreads();
    }
    auto next_live = [&](int c) {
        return all_live ? c : next_live_chunk(p, live_s, ch_begin, ch_end, kt, combo, c, skipped);
    };
    int buf = 0;
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

    if (tid == 0) {
        p.skip_slots[blockIdx.x] = skipped;
        p.work_slots[t] = ch_end - ch_begin - skipped;
    }

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

// Row-window weight gradient for narrow stride-1 layers (64 or 128 input and
// output channels, filters of at most 3 x 3).  A workgroup owns a 64-wide
// output-channel tile, a 64-wide channel tile and a segment of up to 128
// output columns q, and accumulates all R*S taps of dW over a range of
// output rows (n, p) -- one row per step:
//
//   dW[k, r, s, c] += sum_q  X[n, p - ph + r, q - pw + s, c] * dY[n, p, q, k]
//
// The X rows a step needs are the R input rows p - ph .. p - ph + R - 1, each
// read into LDS once with its halo columns (zeros outside the image) and
// shared by the S taps of its filter row: the tap shift s is an offset of
// the row index at which the matrix fragments are read.  Consecutive output
// rows of one image share R - 1 of those input rows, so X rows sit in a ring
// of four and a step copies one new input row and one dY row segment while
// the previous step computes.  Per output pixel that is 2 x 128 bytes of
// copies for 2 * 64 * R*S * 64 multiply-adds (the chunked kernel copies the
// X row once per tap).
//
// GEMM view per step: M = (tap, c) columns (A = shifted X rows), N = k
// (B = dY), reduction = q in 32-column chunks; both operands sit in LDS in
// their natural [column][channel] order and the fragments are read with
// ds_read_b64_tr_b16 (as in the chunked kernel).  Input sparsity: the
// "chunks" of the skip machinery are whole output rows (occupancy per row
// and k tile), ranked into balanced splits exactly as above.
constexpr int RW_NT = 512;               // 8 waves: 2 along k (32 each) x 4 column quarters
constexpr int RW_QT = 128;               // output columns per segment (multiple of 32)
constexpr int RW_XROWS = 136;            // X row slots: RW_QT + S - 1 halo columns, in groups of 8
constexpr int RW_SLOTS = 5;              // X ring: R rows in use plus the next two steps' new rows
constexpr int RW_YBUF = 3;               // dY segments: this step and the next two
constexpr int RW_NB = 9;                 // column blocks (16 columns) per wave at most: 36 / 4
static_assert(RW_QT % 32 == 0 && RW_XROWS >= RW_QT + 2 && RW_XROWS % 8 == 0, "row-window shape");

// LDS chunk swizzle of the 128-byte rows (8 chunks).  The LDS serves 256
// bytes (64 banks) per cycle, a row of even index the lower half of the
// banks and one of odd index the upper half, and a transpose read takes 32
// lanes per cycle: rows b .. b+3 and b+8 .. b+11, 32 bytes (one chunk pair)
// each.  The pair is moved by bits 1 and 3 of the row, which differ among
// the four rows of either parity for every b (tap shifts included), so the
// eight chunk pairs of a cycle never share a bank.  (Moving the pair by the
// row's two low bits, as first tried, left the rows 8 apart on the same
// banks: bank-conflict cycles were half of the LDS's active cycles.)
__device__ __forceinline__ int trswz8(int row) { return 2 * (((row >> 1) & 1) | (((row >> 3) & 1) << 1)); }

// Ring slot of input row h (h >= -16): (h + 20) mod 5 by a multiply and shift
// (x / 5 = (x * 52429) >> 18 for 0 <= x < 2^16).
__device__ __forceinline__ int ring_slot(int h)
{
    static_assert(RW_SLOTS == 5, "the slot formula divides by 5");
    const uint32_t x = (uint32_t)(h + 20);
    return (int)(x - ((x * 52429u) >> 18) * 5u);
}

// NB: column blocks per wave, R*S (every wave holds R*S of the 4 R*S blocks).
template <int NB>
__global__ __launch_bounds__(RW_NT) void bwd_weight_rows_kernel(WeightParams p)
{
    static_assert(NB >= 1 && NB <= RW_NB, "at most 3 x 3 taps");
    constexpr uint32_t ESZ = 2;
    constexpr int NW = RW_NT / 64;
    __shared__ uint4 Ys[RW_YBUF][RW_QT * 8];         // dY segments of output rows, [q][k]
    __shared__ uint4 Xs[RW_SLOTS][RW_XROWS * 8];     // input rows with halo, [w][c]
    __shared__ uint8_t live_s[OCC_WIN];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wave_u = __builtin_amdgcn_readfirstlane(wave);
    const int wk = wave_u & 1, wq = wave_u >> 1;     // k half, column quarter
    const int RS = p.R * p.S;

    // work item: split z of tile (q segment, channel tile, k tile)
    const int tiles = p.tgroups * p.ctiles * p.ktiles;   // tgroups = q segments here
    const int t = xcd_remap(blockIdx.x, gridDim.x);
    const int z = t / tiles;
    int rem = t - z * tiles;
    const int kt = rem % p.ktiles;
    rem /= p.ktiles;
    const int ct = rem % p.ctiles;
    const int qt = rem / p.ctiles;
    const int k0 = kt * 64, c0 = ct * 64, q0 = qt * RW_QT;
    const int qn = min(RW_QT, p.Q - q0);             // valid columns of the segment
    const int nqc = (qn + 31) >> 5;                  // 32-column reduction chunks
    const int xn = qn + p.S - 1;                     // X columns the segment reads
    if (blockIdx.x == 0 && tid == 0) {
        p.header[0] = p.mode_flags;
        p.header[1] = 1;   // the readers' plan: row-window chunks
    }

    const u32x4_t rs_x = make_rsrc_words(p.x, p.x_bytes);
    const u32x4_t rs_dy = make_rsrc_words(p.dy, p.dy_bytes);

    // this wave's column blocks: [cb0, cb0 + nbw) of the R*S*4 blocks
    // (block b = tap b / 4, channels 16 (b % 4) .. + 15 of the tile)
    const int ncb = RS * 4;
    const int nbq = (ncb + 3) >> 2;
    const int cb0 = wq * nbq;
    constexpr int nbw = NB;
    (void)nbq;

    floatx4 acc[NB][2];
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[j][0] = acc[j][1] = floatx4{0.f, 0.f, 0.f, 0.f};

    // copies: lane l of a wave serves row 8g + l/8 at physical chunk l%8,
    // i.e. logical chunk (l%8) ^ trswz8(row)
    const int lrow8 = lane >> 3, pch = lane & 7;
    // Each copy helper returns how many copy instructions this wave issued
    // (the waits below count them).  A lane's byte offset is a scalar row
    // base plus a per-lane part computed once here (kOOB where the column
    // lies outside the segment or the image).
    constexpr int YG = (RW_QT / 8 + NW - 1) / NW, XG = (RW_XROWS / 8 + NW - 1) / NW;
    uint32_t ylane[YG], xlane[XG];
#pragma unroll
    for (int u = 0; u < YG; ++u) {
        const int i = 8 * (wave_u + NW * u) + lrow8;
        const int lc = pch ^ trswz8(i);
        ylane[u] = i < qn ? (uint32_t)(((q0 + i) * p.K + k0 + lc * 8) * ESZ) : kOOB;
    }
#pragma unroll
    for (int u = 0; u < XG; ++u) {
        const int i = 8 * (wave_u + NW * u) + lrow8;
        const int lc = pch ^ trswz8(i);
        const int w = q0 - p.pad_w + i;
        xlane[u] = (i < xn && w >= 0 && w < p.W) ? (uint32_t)((w * p.C + c0 + lc * 8) * ESZ) : kOOB;
    }
    auto copy_y = [&](int buf, int row) -> int {   // dY segment of output row `row` = n*P + p
        const uint32_t base = (uint32_t)row * (uint32_t)(p.Q * p.K * ESZ);
        int issued = 0;
#pragma unroll
        for (int u = 0; u < YG; ++u) {
            const int g = wave_u + NW * u;
            if (g < RW_QT / 8) {
                buf_load16_lds(rs_dy, ylane[u] == kOOB ? kOOB : base + ylane[u], lds_addr(&Ys[buf][g * 64]));
                ++issued;
            }
        }
        return issued;
    };
    auto copy_x = [&](int n, int h) -> int {   // input row h of image n into its ring slot
        const int slot = ring_slot(h);
        const bool hin = h >= 0 && h < p.H;
        const uint32_t base = hin ? (uint32_t)(n * p.H + h) * (uint32_t)(p.W * p.C * ESZ) : 0u;
        int issued = 0;
#pragma unroll
        for (int u = 0; u < XG; ++u) {
            const int g = wave_u + NW * u;
            if (g < RW_XROWS / 8) {
                buf_load16_lds(rs_x, (!hin || xlane[u] == kOOB) ? kOOB : base + xlane[u],
                               lds_addr(&Xs[slot][g * 64]));
                ++issued;
            }
        }
        return issued;
    };

    // fragment addresses (bytes in a buffer of 128-byte rows), as tr_addr
    const int kg = lane >> 4, q4 = lane & 3, m4 = (lane >> 2) & 3;
    auto tr8 = [&](int row, int cb) {
        const int col = cb + 4 * q4;
        return row * 128 + (((col >> 3) ^ trswz8(row)) << 4) + ((col & 7) << 1);
    };
    // per column block of this wave: filter row, column shift and channel base
    int b_r[NB], b_s[NB], b_c[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j) {
        const int b = cb0 + j, tap = b >> 2;
        b_r[j] = tap / p.S;
        b_s[j] = tap - b_r[j] * p.S;
        b_c[j] = (b & 3) * 16;
    }

    // Fragment addresses.  Within a buffer the address of a fragment read is
    // a per-lane part fixed for the whole kernel (row 8 kg + m, plus the
    // column shift s, and the swizzled column) plus 4096 bytes per 32-row
    // chunk (the swizzle does not depend on bits 5 and up), which the
    // unrolled chunk loop folds into the instructions' offset fields; only
    // the ring slot of each X block changes from step to step.  So the inner
    // loop issues reads and matrix instructions with no address arithmetic.
    int xl[NB][2], yl[2][2];
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
        for (int h = 0; h < 2; ++h) xl[j][h] = tr8(8 * kg + m4 + 4 * h + b_s[j], b_c[j]);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int h = 0; h < 2; ++h) yl[i][h] = tr8(8 * kg + m4 + 4 * h, wk * 32 + i * 16);
    const char* X0 = reinterpret_cast<const char*>(Xs);
    auto compute = [&](int ybuf, int pp) {
        const char* Yb = reinterpret_cast<const char*>(Ys[ybuf]);
        const char* Xb[NB];
#pragma unroll
        for (int j = 0; j < NB; ++j) {
            const int h = pp - p.pad_h + b_r[j];
            Xb[j] = X0 + ring_slot(h) * (int)sizeof(Xs[0]) + xl[j][0];
        }
        // per 32-column chunk: the chunk's eleven fragment pairs are read,
        // then its 18 matrix instructions; the other wave on the SIMD
        // overlaps its reads with them
#pragma unroll
        for (int kc = 0; kc < RW_QT / 32; ++kc) {
            if (kc < nqc) {   // uniform
                uint4 fb[2], fa[NB];
#pragma unroll
                for (int i = 0; i < 2; ++i) {
                    const uint2 lo = ds_read_tr16(Yb + yl[i][0] + kc * 4096);
                    const uint2 hi = ds_read_tr16(Yb + yl[i][1] + kc * 4096);
                    fb[i] = make_uint4(lo.x, lo.y, hi.x, hi.y);
                }
#pragma unroll
                for (int j = 0; j < NB; ++j) {
                    if (j < nbw) {   // uniform; every index stays a compile-time constant
                        const uint2 lo = ds_read_tr16(Xb[j] + kc * 4096);
                        const uint2 hi = ds_read_tr16(Xb[j] + (xl[j][1] - xl[j][0]) + kc * 4096);
                        fa[j] = make_uint4(lo.x, lo.y, hi.x, hi.y);
                    }
                }
#pragma unroll
                for (int j = 0; j < NB; ++j) {
                    if (j < nbw) {
                        acc[j][0] = mfma_chunk(acc[j][0], fa[j], fb[0], uint16_t{});
                        acc[j][1] = mfma_chunk(acc[j][1], fa[j], fb[1], uint16_t{});
                    }
                }
            }
        }
    };

    // this split's row range, balanced over the live rows when skipping:
    // the unskipped range first, its step-0 copies issued at once with the
    // call's dead-block flag read behind them; only when the occupancy pass
    // found a dead row is the range ranked (in the X ring, once the copies
    // have landed) and step 0 copied again
    const int combo = qt * p.ctiles + ct;
    int ch_begin = min(p.nchunks, z * p.chunks_per_split);
    int ch_end = min(p.nchunks, ch_begin + p.chunks_per_split);
    static_assert(sizeof(Xs) >= SPLIT_SCRATCH_BYTES, "ranking scratch fits the X ring");
    bool all_live = true;
    int skipped = 0;
    auto next_live = [&](int row) {
        return all_live ? row : next_live_chunk(p, live_s, ch_begin, ch_end, kt, combo, row, skipped);
    };

    // Pipeline over the live output rows ra (this step), rb and rc (the next
    // two): the copies of step i + 2 are issued at step i (its dY
    // segment, and its one new input row when steps i .. i + 2 are
    // consecutive rows of one image), so every copy has two steps' matrix
    // work to land; the wait at the end of step i leaves exactly the copies
    // just issued in flight.  A step that does not follow its predecessor
    // (next image, or dead rows skipped) has its R input rows loaded after
    // the step before it, with the next step's new row if that one follows.
    auto follows = [&](int a, int b) {   // output row b comes right after a in the same image
        return b == a + 1 && fdiv((uint32_t)b, p.div_p) == fdiv((uint32_t)a, p.div_p);
    };
    auto new_row = [&](int c) {          // the input row a following output row adds to the window
        const int n = (int)fdiv((uint32_t)c, p.div_p), pp = c - n * p.P;
        return copy_x(n, pp - p.pad_h + p.R - 1);
    };
    auto all_rows = [&](int c) {
        const int n = (int)fdiv((uint32_t)c, p.div_p), pp = c - n * p.P;
        for (int r = 0; r < p.R; ++r) copy_x(n, pp - p.pad_h + r);
    };
    int ra, rb, rc;
    auto first_steps = [&]() {           // rows of steps 0 .. 2 and the copies of steps 0 and 1
        ra = next_live(ch_begin);
        rb = ra < ch_end ? next_live(ra + 1) : ch_end;
        rc = rb < ch_end ? next_live(rb + 1) : ch_end;
        if (ra < ch_end) {
            copy_y(0, ra);
            all_rows(ra);
            if (rb < ch_end) {
                copy_y(1, rb);
                if (follows(ra, rb)) new_row(rb);
            }
        }
    };
    first_steps();
    uint32_t dflag = 0;
    if (p.occ) dflag = __builtin_amdgcn_raw_buffer_load_b32(make_rsrc(p.header, 64), 4 * kDeadWord, 0, 0);
    wait_vmem();
    __syncthreads();
    if (p.occ && __builtin_amdgcn_readfirstlane(dflag) == p.gen) {
        all_live = split_range(p, kt, combo, z, ch_begin, ch_end, live_s, reinterpret_cast<uint8_t*>(Xs));
        __syncthreads();   // the ranking scratch is free before the ring is copied again
        first_steps();
        wait_vmem();
        __syncthreads();
    }
    int ybuf = 0;
    while (ra < ch_end) {
        int issued = 0;   // this wave's copies for step i + 2
        if (rc < ch_end) {
            issued += copy_y(ybuf == 0 ? 2 : ybuf - 1, rc);
            if (follows(ra, rb) && follows(rb, rc)) issued += new_row(rc);
        }
        compute(ybuf, ra - (int)fdiv((uint32_t)ra, p.div_p) * p.P);
        wait_vmem_upto(issued);
        __syncthreads();
        if (rb < ch_end && !follows(ra, rb)) {
            // step i + 1 starts a new window
            all_rows(rb);
            if (rc < ch_end && follows(rb, rc)) new_row(rc);
            wait_vmem();
            __syncthreads();
        }
        ybuf = ybuf == 2 ? 0 : ybuf + 1;
        ra = rb;
        rb = rc;
        rc = rc < ch_end ? next_live(rc + 1) : ch_end;
    }

    if (tid == 0) {
        p.skip_slots[blockIdx.x] = skipped;
        p.work_slots[t] = ch_end - ch_begin - skipped;
    }

    // Partial [qt * nsplit + z][K][RS][C]: lane holds columns 4 (lane/16) .. +3
    // of column block j (4 channels of one tap) for output channel
    // k0 + 32 wk + 16 i + lane%16.
    const uint32_t part_bytes = (uint32_t)p.K * RS * p.C * 4u;
    const __amdgpu_buffer_rsrc_t rs_out =
        make_rsrc(p.out + (int64_t)(qt * p.nsplit + z) * p.K * RS * p.C, part_bytes);
#pragma unroll
    for (int j = 0; j < NB; ++j) {
        if (j < nbw) {   // uniform
            const int b = cb0 + j, tap = b >> 2;
            const int c = c0 + (b & 3) * 16 + 4 * (lane >> 4);
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int k = k0 + wk * 32 + i * 16 + (lane & 15);
                const uint32_t off = (uint32_t)((k * RS + tap) * p.C + c) * 4u;
                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, acc[j][i]), rs_out, off, 0, 0);
            }
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
    hipError_t e_launch = hipSuccess;
    if (p.rows) {
        if (dtype != 1 || p.R > 3 || p.S > 3 || p.bk != 64 || p.cg != 64) return hipErrorInvalidValue;
        switch (p.R * p.S) {
        case 1: e_launch = launch_timed(bwd_weight_rows_kernel<1>, dim3(nb), dim3(RW_NT), stream, ev, p); break;
        case 2: e_launch = launch_timed(bwd_weight_rows_kernel<2>, dim3(nb), dim3(RW_NT), stream, ev, p); break;
        case 3: e_launch = launch_timed(bwd_weight_rows_kernel<3>, dim3(nb), dim3(RW_NT), stream, ev, p); break;
        case 4: e_launch = launch_timed(bwd_weight_rows_kernel<4>, dim3(nb), dim3(RW_NT), stream, ev, p); break;
        case 6: e_launch = launch_timed(bwd_weight_rows_kernel<6>, dim3(nb), dim3(RW_NT), stream, ev, p); break;
        case 9: e_launch = launch_timed(bwd_weight_rows_kernel<9>, dim3(nb), dim3(RW_NT), stream, ev, p); break;
        default: return hipErrorInvalidValue;
        }
        return e_launch;
    }
    const dim3 grid(nb), block(dtype != 1 ? NT : p.bk == 64 ? WTile<64>::NT : WTile<256>::NT);
    if (dtype == 1) {
        if (p.bk == 64) e_launch = launch_timed(bwd_weight_tr_kernel<64>, grid, block, stream, ev, p);
        else if (p.bk == 128) e_launch = launch_timed(bwd_weight_tr_kernel<128>, grid, block, stream, ev, p);
        else e_launch = launch_timed(bwd_weight_tr_kernel<256>, grid, block, stream, ev, p);
    }
    else e_launch = launch_timed(bwd_weight_kernel<float>, grid, block, stream, ev, p);
    return e_launch;
}

}  // namespace cbw
