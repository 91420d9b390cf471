// Boundary layout conversion for callers whose activations are NCHW.  The
// kernels of the path run on channel-innermost data (NHWC: the channel-first
// storage indexed through the channels, Sec. IV-B), so an NCHW call is served
// by transposing its inputs into workspace, running the NHWC path there and
// transposing dX back.  These passes are HBM-bound copies; they are timed
// apart from the path itself.
#include <hip/hip_runtime.h>

#include "kernels.hpp"

namespace cbw {
namespace {

// dst[n][c][r] = src[n][r][c] for a batch of rows x cols matrices.  A tile of
// TR x TC elements goes through LDS; global accesses are 16-byte vectors
// along a row whenever that row length is a multiple of the vector, else
// single elements.  Out-of-range elements of a ragged tile are neither read
// nor written.  Tiles are 64 x 64 (a 128 x 128 bf16 tile with 256-byte
// segments was measured no faster: about 25 us per 51 MB tensor either way,
// against 15 us for a plain copy of it).
template <typename T, int TR, int TC, int NTH>
__global__ __launch_bounds__(NTH) void transpose_kernel(const T* __restrict__ src, T* __restrict__ dst, int rows,
                                                        int cols)
{
    constexpr int V = 16 / sizeof(T);   // elements per vector
    using U = typename std::conditional<sizeof(T) == 2, uint16_t, uint32_t>::type;
    __shared__ U tile[TR][TC + 2];      // [source row][source column]
    const int c0 = blockIdx.x * TC, r0 = blockIdx.y * TR;
    const int64_t base = (int64_t)blockIdx.z * rows * cols;
    const U* s = reinterpret_cast<const U*>(src) + base;
    U* d = reinterpret_cast<U*>(dst) + base;
    const bool vin = cols % V == 0, vout = rows % V == 0;

    constexpr int VIN = TC / V;         // vectors per source tile row
    for (int idx = threadIdx.x; idx < TR * VIN; idx += NTH) {
        const int r = idx / VIN, cv = (idx % VIN) * V;
        const int gr = r0 + r, gc = c0 + cv;
        if (gr >= rows) continue;
        if (vin) {
            if (gc < cols) {
                const uint4 v = *reinterpret_cast<const uint4*>(s + (int64_t)gr * cols + gc);
                const U* e = reinterpret_cast<const U*>(&v);
#pragma unroll
                for (int j = 0; j < V; ++j) tile[r][cv + j] = e[j];
            }
        } else {
#pragma unroll
            for (int j = 0; j < V; ++j)
                if (gc + j < cols) tile[r][cv + j] = s[(int64_t)gr * cols + gc + j];
        }
    }
    __syncthreads();
    constexpr int VOUT = TR / V;        // vectors per output tile row
    for (int idx = threadIdx.x; idx < TC * VOUT; idx += NTH) {
        const int c = idx / VOUT, rv = (idx % VOUT) * V;   // output row c (a source column), columns rv..rv+V-1
        const int gc = c0 + c, gr = r0 + rv;
        if (gc >= cols) continue;
        if (vout) {
            if (gr < rows) {
                uint4 v;
                U* e = reinterpret_cast<U*>(&v);
#pragma unroll
                for (int j = 0; j < V; ++j) e[j] = tile[rv + j][c];
                *reinterpret_cast<uint4*>(d + (int64_t)gc * rows + gr) = v;
            }
        } else {
#pragma unroll
            for (int j = 0; j < V; ++j)
                if (gr + j < rows) d[(int64_t)gc * rows + gr + j] = tile[rv + j][c];
        }
    }
}

// Footprint bits in NCHW element order -> NHWC element order (bit i of word
// i/32 is element i of the tensor in that layout).
//
// C a multiple of 32: a workgroup takes 32 pixels of one image and up to 256
// channels, a wave 64 of those channels, one channel per lane.  Each lane
// loads the 32 bits of its channel row over the 32 pixels (two words funnel-
// shifted when the row does not start on a word boundary); a ballot of bit q
// across the wave is then pixel q's 64 channel bits, two output words, and
// lanes 2q and 2q+1 store them.  The four waves cover the 256 channels of
// the same pixels, so the 32-byte rows of C = 256 are written whole.
__global__ __launch_bounds__(256) void bits_nchw_to_nhwc_ballot_kernel(const uint32_t* __restrict__ src,
                                                                       uint32_t* __restrict__ dst, int C, int HW,
                                                                       int csuper, int64_t nwords)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int n = blockIdx.y / csuper, cs = blockIdx.y % csuper;
    const int cbase = cs * 256 + wave * 64;     // first channel of this wave
    if (cbase >= C) return;                     // whole wave past C: uniform exit
    const int p0 = blockIdx.x * 32;
    const int c = cbase + lane;
    uint32_t w = 0;
    if (c < C) {
        const int64_t s = ((int64_t)n * C + c) * HW + p0;     // bit of (n, c, p0)
        const int64_t wi = s >> 5;
        const int sh = (int)(s & 31);
        const uint32_t lo = src[wi];
        const uint32_t hi = (sh != 0 && wi + 1 < nwords) ? src[wi + 1] : 0u;
        w = sh ? (lo >> sh) | (hi << (32 - sh)) : lo;
    }
    uint32_t out = 0;
#pragma unroll
    for (int q = 0; q < 32; ++q) {
        const uint64_t m = __ballot((w >> q) & 1u);
        if ((lane >> 1) == q) out = (lane & 1) ? (uint32_t)(m >> 32) : (uint32_t)m;
    }
    const int p = p0 + (lane >> 1);
    const int cw = (cbase >> 5) + (lane & 1);
    if (p < HW && cw < C / 32) dst[((int64_t)n * HW + p) * (C / 32) + cw] = out;
}

// Any C (a multiple of the 16-byte vector): one thread per output word, each
// bit located on its own.  Bits past the last element stay 0.
__global__ __launch_bounds__(256) void bits_nchw_to_nhwc_kernel(const uint32_t* __restrict__ src,
                                                                uint32_t* __restrict__ dst, int N, int C, int HW)
{
    const int64_t total = (int64_t)N * C * HW;
    const int64_t nwords = (total + 31) / 32;
    const int64_t wi = (int64_t)blockIdx.y * gridDim.x * 256 + (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (wi >= nwords) return;
    uint32_t word = 0;
    for (int j = 0; j < 32; ++j) {
        const int64_t i = wi * 32 + j;    // NHWC element index
        if (i >= total) break;
        const int64_t np = i / C;
        const int c = (int)(i - np * C);
        const int64_t n = np / HW;
        const int p = (int)(np - n * HW);
        const int64_t s = (n * C + c) * HW + p;
        word |= ((src[s >> 5] >> (s & 31)) & 1u) << j;
    }
    dst[wi] = word;
}

}  // namespace

hipError_t launch_transpose(int dtype, const void* src, void* dst, int batch, int rows, int cols, hipStream_t s)
{
    if (batch <= 0 || rows <= 0 || cols <= 0) return hipSuccess;
    const dim3 grid((cols + 63) / 64, (rows + 63) / 64, batch);
    if (dtype == 1)
        transpose_kernel<uint16_t, 64, 64, 256><<<grid, 256, 0, s>>>(static_cast<const uint16_t*>(src),
                                                                     static_cast<uint16_t*>(dst), rows, cols);
    else
        transpose_kernel<float, 64, 64, 256><<<grid, 256, 0, s>>>(static_cast<const float*>(src),
                                                                  static_cast<float*>(dst), rows, cols);
    return hipGetLastError();
}

hipError_t launch_bits_nchw_to_nhwc(const uint32_t* src, uint32_t* dst, int N, int C, int HW, hipStream_t s)
{
    if (N <= 0 || C <= 0 || HW <= 0) return hipSuccess;
    const int64_t nwords = ((int64_t)N * C * HW + 31) / 32;
    const int csuper = (C + 255) / 256;
    if (C % 32 == 0 && (int64_t)N * csuper <= 65535) {
        const dim3 grid((HW + 31) / 32, N * csuper);
        bits_nchw_to_nhwc_ballot_kernel<<<grid, 256, 0, s>>>(src, dst, C, HW, csuper, nwords);
    } else {
        const int64_t blocks = (nwords + 255) / 256;
        const int gx = (int)(blocks < 65535 ? blocks : 65535);
        const int gy = (int)((blocks + gx - 1) / gx);
        bits_nchw_to_nhwc_kernel<<<dim3(gx, gy), 256, 0, s>>>(src, dst, N, C, HW);
    }
    return hipGetLastError();
}

}  // namespace cbw
