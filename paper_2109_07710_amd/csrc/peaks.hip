// Measured machine ceilings for the roofline of the convolution kernels:
// a matrix-core loop (bf16 MFMA with fp32 accumulation, no memory traffic)
// and two HBM streams (read only, and read + write).  Built into its own
// library (libcbwpeaks.so); the benchmark times each launch with events and
// reports the rates next to the published peaks.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/cbw_peaks.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;   // four waves, one per SIMD of a CU
constexpr int kAcc16 = 8;       // independent 16x16x32 accumulators per wave
constexpr int kAcc32 = 4;       // independent 32x32x16 accumulators per wave

// Every wave runs `iters` rounds of independent matrix instructions on
// register operands.  The operands come from memory (so nothing folds) and
// the sums are stored only when they equal a value the inputs cannot
// produce, so the loop is kept but stores nothing.
template <int SHAPE>
__global__ __launch_bounds__(kThreads) void mfma_peak_kernel(const uint4* __restrict__ seed, int iters,
                                                             float* __restrict__ sink)
{
    const int lane = threadIdx.x & 63;
    const bf16x8 a = __builtin_bit_cast(bf16x8, seed[lane]);
    const bf16x8 b = __builtin_bit_cast(bf16x8, seed[64 + lane]);
    float total = 0.f;
    if constexpr (SHAPE == CBW_PEAK_MFMA_16X16X32) {
        // Eight accumulators, the instructions issued from inline assembly:
        // with the builtin the register allocator moved the loop-carried
        // accumulators between registers every iteration (about one move per
        // matrix instruction), which is not what a peak loop should measure.
        // Each accumulator is reused eight instructions later.
        floatx4 c0 = {0.f, 0.f, 0.f, 0.f}, c1 = c0, c2 = c0, c3 = c0, c4 = c0, c5 = c0, c6 = c0, c7 = c0;
        static_assert(kAcc16 == 8, "eight accumulators");
#define CBW_MFMA16(c) asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+v"(c) : "v"(a), "v"(b))
        for (int i = 0; i < iters; ++i) {
            CBW_MFMA16(c0); CBW_MFMA16(c1); CBW_MFMA16(c2); CBW_MFMA16(c3);
            CBW_MFMA16(c4); CBW_MFMA16(c5); CBW_MFMA16(c6); CBW_MFMA16(c7);
        }
#undef CBW_MFMA16
        const floatx4 s = ((c0 + c1) + (c2 + c3)) + ((c4 + c5) + (c6 + c7));
        total = s.x + s.y + s.z + s.w;
    } else {
        floatx16 acc[kAcc32];
#pragma unroll
        for (int j = 0; j < kAcc32; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[j][v] = 0.f;
        for (int i = 0; i < iters; ++i) {
#pragma unroll
            for (int j = 0; j < kAcc32; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
        }
#pragma unroll
        for (int j = 0; j < kAcc32; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) total += acc[j][v];
    }
    if (total == -1.0e30f) sink[blockIdx.x * kThreads + threadIdx.x] = total;
}

constexpr int kStreamBlocks = 256 * 8;   // eight workgroups per CU
constexpr int kUnroll = 4;               // 16-byte loads in flight per thread

// Read-only stream: every 16-byte vector of src is loaded once; the XOR of
// all words is stored only when it equals a marker (never, in practice).
__global__ __launch_bounds__(kThreads) void hbm_read_kernel(const u32x4* __restrict__ src, int64_t nvec,
                                                            uint32_t* __restrict__ sink)
{
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    uint32_t x = 0;
    for (; i + (kUnroll - 1) * stride < nvec; i += kUnroll * stride) {
        u32x4 v[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) v[u] = __builtin_nontemporal_load(src + i + u * stride);
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) x ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
    for (; i < nvec; i += stride) {
        const u32x4 v = src[i];
        x ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    if (x == 0x9e3779b9u) sink[blockIdx.x * kThreads + threadIdx.x] = x;
}

// Copy stream: dst = src in 16-byte vectors.
__global__ __launch_bounds__(kThreads) void hbm_copy_kernel(const u32x4* __restrict__ src, u32x4* __restrict__ dst,
                                                            int64_t nvec)
{
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    for (; i + (kUnroll - 1) * stride < nvec; i += kUnroll * stride) {
        u32x4 v[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) v[u] = __builtin_nontemporal_load(src + i + u * stride);
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) __builtin_nontemporal_store(v[u], dst + i + u * stride);
    }
    for (; i < nvec; i += stride) dst[i] = src[i];
}

int status(hipError_t e)
{
    if (e == hipSuccess) return 0;
    (void)hipGetLastError();
    return -4;
}

}  // namespace

extern "C" {

size_t cbw_peak_seed_bytes(void) { return 128 * 16; }

size_t cbw_peak_sink_words(int blocks) { return (size_t)(blocks > kStreamBlocks ? blocks : kStreamBlocks) * kThreads; }

double cbw_peak_mfma_flops(int shape, int blocks, int iters)
{
    const double per = shape == CBW_PEAK_MFMA_16X16X32 ? 2.0 * 16 * 16 * 32 * kAcc16 : 2.0 * 32 * 32 * 16 * kAcc32;
    return per * iters * (double)blocks * (kThreads / 64);
}

int cbw_peak_mfma(int shape, int blocks, int iters, const void* seed, float* sink, void* stream)
{
    if ((shape != CBW_PEAK_MFMA_16X16X32 && shape != CBW_PEAK_MFMA_32X32X16) || blocks <= 0 || iters <= 0 ||
        !seed || !sink)
        return -1;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const uint4* sd = static_cast<const uint4*>(seed);
    if (shape == CBW_PEAK_MFMA_16X16X32)
        mfma_peak_kernel<CBW_PEAK_MFMA_16X16X32><<<blocks, kThreads, 0, s>>>(sd, iters, sink);
    else
        mfma_peak_kernel<CBW_PEAK_MFMA_32X32X16><<<blocks, kThreads, 0, s>>>(sd, iters, sink);
    return status(hipGetLastError());
}

int cbw_peak_hbm_read(const void* src, size_t bytes, uint32_t* sink, void* stream)
{
    if (!src || !sink || bytes == 0 || (bytes & 15) || ((uintptr_t)src & 15)) return -1;
    hbm_read_kernel<<<kStreamBlocks, kThreads, 0, static_cast<hipStream_t>(stream)>>>(
        static_cast<const u32x4*>(src), (int64_t)(bytes / 16), sink);
    return status(hipGetLastError());
}

int cbw_peak_hbm_copy(const void* src, void* dst, size_t bytes, void* stream)
{
    if (!src || !dst || bytes == 0 || (bytes & 15) || ((uintptr_t)src & 15) || ((uintptr_t)dst & 15)) return -1;
    hbm_copy_kernel<<<kStreamBlocks, kThreads, 0, static_cast<hipStream_t>(stream)>>>(
        static_cast<const u32x4*>(src), static_cast<u32x4*>(dst), (int64_t)(bytes / 16));
    return status(hipGetLastError());
}

}  // extern "C"
