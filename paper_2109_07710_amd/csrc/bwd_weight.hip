// Weight gradient as a split-K implicit GEMM on the gfx950 matrix cores.
//
//   dW[k, tap, c] = sum_{pix=(n,p,q)}  X[n, p*sh-ph+r, q*sw-pw+s, c] * dY[pix, k]
//
// (weight-gradient phase, Sec. IV-B).  GEMM view: M = channels c of one tap
// (A = shifted X), N = output channels k (B = dY), reduction = pixels.  Both
// operands are pixel-major in NHWC, so the reduction index is the strided
// one.  Each thread loads an E x E block (E pixels x E channels, one
// 16-byte vector per pixel, coalesced along channels), transposes it in
// registers and writes E vectors of E consecutive pixels into LDS, where the
// MFMA fragments then read reduction-contiguous 16-byte chunks.
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

namespace cbw {

namespace {

constexpr int BM = 128;   // channels c per tile
constexpr int BN = 128;   // output channels k per tile
constexpr int NT = 256;
constexpr int CHR = 16;   // 16-byte chunks per LDS row (256 bytes)

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
    for (int m = 0; m < 4; ++m)        // channel pair (2m, 2m+1)
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
__global__ __launch_bounds__(NT, 2) void bwd_weight_kernel(WeightParams p)
{
    constexpr int E = Elem<T>::E;
    constexpr int BK = CHR * E;                 // pixels per chunk
    constexpr int CB = BM / E;                  // channel blocks per tile row set
    constexpr int NBLK = (BM / E) * (BK / E);   // E x E blocks per operand tile
    constexpr int BPT = NBLK / NT;              // blocks per thread per operand

    __shared__ uint4 As[BM * CHR];
    __shared__ uint4 Bs[BN * CHR];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;

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

    floatx4 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

    const T* __restrict__ x = reinterpret_cast<const T*>(p.x);
    const T* __restrict__ dy = reinterpret_cast<const T*>(p.dy);

    uint4 ra[BPT][E], rb[BPT][E];
    int skipped = 0;

    auto load = [&](int chunk) {
        const int px_base = chunk * BK;
#pragma unroll
        for (int bi = 0; bi < BPT; ++bi) {
            const int blk = tid + bi * NT;
            const int cb = blk % CB, pb = blk / CB;
            const int cA = c0 + cb * E;   // A: channel block of X
            const int kB = k0 + cb * E;   // B: channel block of dY
#pragma unroll
            for (int e = 0; e < E; ++e) {
                const int pix = px_base + pb * E + e;
                ra[bi][e] = make_uint4(0, 0, 0, 0);
                rb[bi][e] = make_uint4(0, 0, 0, 0);
                if (pix < p.npq) {
                    if (kB < p.K) rb[bi][e] = *reinterpret_cast<const uint4*>(dy + ((int64_t)pix * p.K + kB));
                    if (cA < p.C) {
                        const uint32_t nq = fdiv((uint32_t)pix, p.div_q);
                        const int q = pix - (int)nq * p.Q;
                        const uint32_t n = fdiv(nq, p.div_p);
                        const int pp = (int)nq - (int)n * p.P;
                        const int h = pp * p.stride_h - p.pad_h + r;
                        const int w = q * p.stride_w - p.pad_w + s;
                        if (h >= 0 && h < p.H && w >= 0 && w < p.W)
                            ra[bi][e] = *reinterpret_cast<const uint4*>(
                                x + ((((int64_t)n * p.H + h) * p.W + w) * p.C + cA));
                    }
                }
            }
        }
    };

    auto store = [&]() {
#pragma unroll
        for (int bi = 0; bi < BPT; ++bi) {
            const int blk = tid + bi * NT;
            const int cb = blk % CB, pb = blk / CB;
            uint4 ua[E], ub[E];
            transpose_block<T>(ra[bi], ua);
            transpose_block<T>(rb[bi], ub);
#pragma unroll
            for (int j = 0; j < E; ++j) {
                const int row = cb * E + j;
                As[row * CHR + (pb ^ swz16(row))] = ua[j];
                Bs[row * CHR + (pb ^ swz16(row))] = ub[j];
            }
        }
    };

    auto live = [&](int chunk) { return p.occ == nullptr || p.occ[(int64_t)chunk * p.ktiles + kt] != 0; };

    // advance to the first chunk that is not skipped
    int chunk = ch_begin;
    while (chunk < ch_end && !live(chunk)) { ++chunk; ++skipped; }
    if (chunk < ch_end) load(chunk);
    while (chunk < ch_end) {
        __syncthreads();
        store();
        __syncthreads();
        int next = chunk + 1;
        while (next < ch_end && !live(next)) { ++next; ++skipped; }
        if (next < ch_end) load(next);
#pragma unroll
        for (int kc = 0; kc < CHR / 4; ++kc) {
            const int chl = kc * 4 + (lane >> 4);
            uint4 fa[4], fb[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int row = wm * 64 + i * 16 + (lane & 15);
                fa[i] = As[row * CHR + (chl ^ swz16(row))];
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int row = wn * 64 + j * 16 + (lane & 15);
                fb[j] = Bs[row * CHR + (chl ^ swz16(row))];
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = mfma_chunk(acc[i][j], fa[i], fb[j], T{});
        }
        chunk = next;
    }

    if (tid == 0) p.skip_slots[blockIdx.x] = skipped;

    // Epilogue: lane holds channels c0 + wm*64 + i*16 + 4*(lane/16) + v of
    // output channel k0 + wn*64 + j*16 + lane%16; written to [z][k][tap][c].
    float* __restrict__ out = p.out + (int64_t)z * p.K * RS * p.C;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int k = k0 + wn * 64 + j * 16 + (lane & 15);
        if (k >= p.K) continue;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int c = c0 + wm * 64 + i * 16 + 4 * (lane >> 4);
            if (c >= p.C) continue;
            *reinterpret_cast<floatx4*>(out + (((int64_t)k * RS + tap) * p.C + c)) = acc[i][j];
        }
    }
}

}  // namespace

int weight_tile_channels() { return BM; }
int weight_tile_k() { return BN; }
int weight_chunk(int dtype) { return CHR * (dtype == 1 ? 8 : 4); }

hipError_t launch_bwd_weight(int dtype, const WeightParams& p, hipStream_t stream)
{
    const int nb = p.R * p.S * p.ctiles * p.ktiles * p.nsplit;
    if (dtype == 1) bwd_weight_kernel<uint16_t><<<nb, NT, 0, stream>>>(p);
    else bwd_weight_kernel<float><<<nb, NT, 0, stream>>>(p);
    return hipGetLastError();
}

}  // namespace cbw
