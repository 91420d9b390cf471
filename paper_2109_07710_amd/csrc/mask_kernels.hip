// Integer kernels around the GEMMs: footprint bitmaps, dY block occupancy
// and the split-K reduction of dW.  (The compaction counts run in the
// data-gradient preparation launch, the live lists inside the GEMM.)
#include "common.hpp"
#include "kernels.hpp"
#include "footprint.hpp"
#include "occupancy.hpp"
#include "reduce.hpp"

namespace cbw {

namespace {

constexpr int CNT = kCompactThreads;     // threads (= pixels) per compaction block
constexpr int BLK_PX = CNT;

template <typename T>
__device__ __forceinline__ uint32_t elem_bit(const T* p, int64_t i, bool relu)
{
    uint4 v = make_uint4(0, 0, 0, 0);
    if (sizeof(T) == 2) v.x = reinterpret_cast<const uint16_t*>(p)[i];
    else v.x = reinterpret_cast<const uint32_t*>(p)[i];
    return vec_bits<T>(v, relu) & 1u;
}

// One thread per 16-byte vector; the E bits of L = 32/E neighbouring lanes
// are OR-ed into one word written by the first of them.
template <typename T>
__global__ void mask_pack_kernel(const T* __restrict__ x, uint32_t* __restrict__ bits, int64_t count,
                                 int64_t nvec, bool relu)
{
    constexpr int E = Elem<T>::E;
    constexpr int L = 32 / E;
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    uint32_t b = 0;
    if (v < nvec) {
        const int64_t e0 = v * E;
        if (e0 + E <= count) {
            b = vec_bits<T>(*reinterpret_cast<const uint4*>(x + e0), relu);
        } else {
            for (int i = 0; i < E && e0 + i < count; ++i) b |= elem_bit<T>(x, e0 + i, relu) << i;
        }
    }
    const int lane = threadIdx.x & 63;
    b <<= (lane % L) * E;
#pragma unroll
    for (int off = 1; off < L; off <<= 1) b |= __shfl_xor(b, off);
    if (lane % L == 0 && v < nvec) bits[v / L] = b;
}


__global__ __launch_bounds__(256) void occupancy_kernel(OccParams p) { occupancy_block(p, blockIdx.x); }

template <int G>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ part, float* __restrict__ dw,
                                                           int nsplit, int K, int RS, int C, int krsc)
{
    splitk_reduce_block<G>(part, dw, nsplit, K, RS, C, krsc, blockIdx.x);
}

}  // namespace

int compact_block_pixels() { return BLK_PX; }

hipError_t launch_relu_mask_pack(int dtype, int64_t count, const void* x, uint32_t* bits, int relu,
                                 hipStream_t stream)
{
    const int E = dtype == 1 ? 8 : 4;
    const int L = 32 / E;
    int64_t nvec = (count + E - 1) / E;
    nvec = (nvec + L - 1) / L * L;  // whole words
    const int64_t blocks = (nvec + 255) / 256;
    if (blocks == 0) return hipSuccess;
    if (dtype == 1)
        mask_pack_kernel<uint16_t><<<(unsigned)blocks, 256, 0, stream>>>((const uint16_t*)x, bits, count, nvec,
                                                                         relu != 0);
    else
        mask_pack_kernel<float><<<(unsigned)blocks, 256, 0, stream>>>((const float*)x, bits, count, nvec,
                                                                      relu != 0);
    return hipGetLastError();
}

hipError_t launch_occupancy(const OccParams& p, hipStream_t stream)
{
    if (p.cpw < 1 || p.cpw * p.ktiles > 1024 || (p.xlive && p.cpw * p.tgroups * p.ctiles > 1024))
        return hipErrorInvalidValue;
    occupancy_kernel<<<(p.nchunks + p.cpw - 1) / p.cpw, 256, 0, stream>>>(p);
    return hipGetLastError();
}

hipError_t launch_splitk_reduce(const float* part, float* dw, int nsplit, int K, int RS, int C, int krsc,
                                hipStream_t stream)
{
    const int64_t n4 = (int64_t)K * RS * C / 4;
    // G threads per output, each summing a consecutive 1/G of the splits
    const int G = splitk_reduce_group(nsplit, n4);
    const unsigned blocks = (unsigned)((n4 * G + 255) / 256);
    switch (G) {
    case 1: splitk_reduce_kernel<1><<<blocks, 256, 0, stream>>>(part, dw, nsplit, K, RS, C, krsc); break;
    case 2: splitk_reduce_kernel<2><<<blocks, 256, 0, stream>>>(part, dw, nsplit, K, RS, C, krsc); break;
    case 4: splitk_reduce_kernel<4><<<blocks, 256, 0, stream>>>(part, dw, nsplit, K, RS, C, krsc); break;
    case 8: splitk_reduce_kernel<8><<<blocks, 256, 0, stream>>>(part, dw, nsplit, K, RS, C, krsc); break;
    default: splitk_reduce_kernel<16><<<blocks, 256, 0, stream>>>(part, dw, nsplit, K, RS, C, krsc); break;
    }
    return hipGetLastError();
}

}  // namespace cbw
