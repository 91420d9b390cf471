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

constexpr int TT = 64;    // tile edge, elements
constexpr int TNT = 256;  // threads per tile

// dst[n][c][r] = src[n][r][c] for a batch of rows x cols matrices.  A tile of
// 64 x 64 elements goes through LDS; global accesses are 16-byte vectors
// along a row whenever that row length is a multiple of the vector, else
// single elements.  Out-of-range elements of a ragged tile are neither read
// nor written.
template <typename T>
__global__ __launch_bounds__(TNT) void transpose_kernel(const T* __restrict__ src, T* __restrict__ dst, int rows,
                                                        int cols)
{
    constexpr int V = 16 / sizeof(T);   // elements per vector
    constexpr int VR = TT / V;          // vectors per tile row
    using U = typename std::conditional<sizeof(T) == 2, uint16_t, uint32_t>::type;
    __shared__ U tile[TT][TT + 2];      // [source row][source column]
    const int c0 = blockIdx.x * TT, r0 = blockIdx.y * TT;
    const int64_t base = (int64_t)blockIdx.z * rows * cols;
    const U* s = reinterpret_cast<const U*>(src) + base;
    U* d = reinterpret_cast<U*>(dst) + base;
    const bool vin = cols % V == 0, vout = rows % V == 0;

    for (int idx = threadIdx.x; idx < TT * VR; idx += TNT) {
        const int r = idx / VR, cv = (idx % VR) * V;
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
    for (int idx = threadIdx.x; idx < TT * VR; idx += TNT) {
        const int c = idx / VR, rv = (idx % VR) * V;   // output row c (a source column), columns rv..rv+V-1
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
// i/32 is element i of the tensor in that layout).  With C a multiple of 32
// (per_pixel) an output word is 32 channels of one pixel: thread = pixel
// (consecutive lanes read consecutive bits of each channel row).  Otherwise
// each output bit is located on its own, one thread per output word.  Bits
// past the last element stay 0.
__global__ __launch_bounds__(256) void bits_nchw_to_nhwc_kernel(const uint32_t* __restrict__ src,
                                                                uint32_t* __restrict__ dst, int N, int C, int HW,
                                                                int per_pixel)
{
    const int64_t total = (int64_t)N * C * HW;
    if (per_pixel) {   // C % 32 == 0; grid (pixel blocks, N * C/32)
        const int cw = C / 32;
        const int p = blockIdx.x * 256 + threadIdx.x;
        const int n = blockIdx.y / cw, w = blockIdx.y % cw;
        if (p >= HW) return;
        uint32_t word = 0;
        const int64_t s0 = ((int64_t)n * C + 32 * w) * HW + p;
#pragma unroll 8
        for (int j = 0; j < 32; ++j) {
            const int64_t s = s0 + (int64_t)j * HW;
            word |= ((src[s >> 5] >> (s & 31)) & 1u) << j;
        }
        dst[((int64_t)n * HW + p) * cw + w] = word;
        return;
    }
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
    const dim3 grid((cols + TT - 1) / TT, (rows + TT - 1) / TT, batch);
    if (dtype == 1)
        transpose_kernel<uint16_t><<<grid, TNT, 0, s>>>(static_cast<const uint16_t*>(src),
                                                        static_cast<uint16_t*>(dst), rows, cols);
    else
        transpose_kernel<float><<<grid, TNT, 0, s>>>(static_cast<const float*>(src), static_cast<float*>(dst),
                                                     rows, cols);
    return hipGetLastError();
}

hipError_t launch_bits_nchw_to_nhwc(const uint32_t* src, uint32_t* dst, int N, int C, int HW, hipStream_t s)
{
    if (N <= 0 || C <= 0 || HW <= 0) return hipSuccess;
    if (C % 32 == 0 && (int64_t)N * (C / 32) <= 65535) {
        const dim3 grid((HW + 255) / 256, N * (C / 32));
        bits_nchw_to_nhwc_kernel<<<grid, 256, 0, s>>>(src, dst, N, C, HW, 1);
    } else {
        const int64_t nwords = ((int64_t)N * C * HW + 31) / 32;
        const int64_t blocks = (nwords + 255) / 256;
        const int gx = (int)(blocks < 65535 ? blocks : 65535);
        const int gy = (int)((blocks + gx - 1) / gx);
        bits_nchw_to_nhwc_kernel<<<dim3(gx, gy), 256, 0, s>>>(src, dst, N, C, HW, 0);
    }
    return hipGetLastError();
}

}  // namespace cbw
