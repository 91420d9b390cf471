// Shared device helpers for the gfx950 kernels: element traits, bf16
// rounding, fast integer division, MFMA wrappers and the LDS swizzle.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cbw {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Element traits.  bf16 is stored as its 16-bit pattern.  A "vector" is 16
// bytes: E elements.  One MFMA "chunk step" consumes one 16-byte fragment of
// A and of B per lane and reduces 4*E elements of the reduction dimension
// (the four 16-lane groups each hold E consecutive reduction indices).
template <typename T> struct Elem;
template <> struct Elem<uint16_t> { static constexpr int E = 8; };
template <> struct Elem<float> { static constexpr int E = 4; };

__device__ __forceinline__ floatx4 mfma_chunk(floatx4 acc, const uint4& a, const uint4& b, uint16_t)
{
    // 16x16x32 bf16 -> fp32.  Lane l supplies row (l % 16) of A and column
    // (l % 16) of B, with the same 8 reduction indices for both; the result
    // holds rows 4*(l/16)+v, v = 0..3, of column l % 16.
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                    __builtin_bit_cast(bf16x8, b), acc, 0, 0, 0);
}

__device__ __forceinline__ floatx4 mfma_chunk(floatx4 acc, const uint4& a, const uint4& b, float)
{
    // Four 16x16x4 fp32 MFMAs.  In MFMA j a lane supplies element j of its
    // fragment for both A and B, so the four reduction indices a lane group
    // covers are the same on both sides; the sum over all of them is the
    // full product whatever index each lane is assigned.
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
    return acc;
}

// fp32 -> bf16 bit pattern, round to nearest, ties to even; NaN stays NaN.
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f)
{
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}

// Two floats to packed bf16 (a in the low half) with round-to-nearest-even:
// one v_cvt_pk_bf16_f32 on gfx950, identical to f32_to_bf16_rne for every
// fp32 input (NaN and subnormal inputs included).
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b)
{
    const floatx2 v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

// Unsigned division by a runtime constant d (1 <= d < 2^31) for numerators
// below 2^31: q = (mulhi(n, m) + n) >> s with s = ceil(log2 d) and
// m = floor(2^32 (2^s - d) / d) + 1 (Granlund & Montgomery, 1994).
struct FastDiv {
    uint32_t d, m, s;
};

inline FastDiv make_fastdiv(uint32_t d)
{
    FastDiv f;
    f.d = d;
    uint32_t s = 0;
    while ((1ull << s) < d) ++s;
    f.s = s;
    f.m = (uint32_t)(((1ull << 32) * ((1ull << s) - d)) / d + 1);
    return f;
}

__device__ __forceinline__ uint32_t fdiv(uint32_t n, const FastDiv& f)
{
    return (__umulhi(n, f.m) + n) >> f.s;
}

// Raw buffer access.  Loads through a buffer descriptor return zeros for
// byte offsets at or past the buffer's size, which the kernels use for
// padding, halo and ragged edges: an invalid element gets offset kOOB.
// Buffers must be smaller than 2^31 bytes so that kOOB plus any in-range
// offset never wraps.
constexpr uint32_t kOOB = 0x80000000u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ uint4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t off)
{
    const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
    return make_uint4(v.x, v.y, v.z, v.w);
}

// Direct global-to-LDS copy of 16 bytes per lane: lane l's 16 bytes land at
// LDS byte address lds_base + 16*l (lds_base is wave-uniform); lanes with an
// out-of-range offset write zeros.  The copy is issued from inline assembly
// so that the compiler does not track it: its completion (vmcnt) is awaited
// explicitly with wait_vmem() before the barrier that publishes the data,
// which keeps the copy of the next step in flight during the MFMAs of the
// current one.  M0 is saved and restored around the copy.
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ u32x4_t make_rsrc_words(const void* p, uint32_t bytes)
{
    const uint64_t a = reinterpret_cast<uint64_t>(p);
    u32x4_t r;
    r.x = (uint32_t)a;
    r.y = (uint32_t)(a >> 32) & 0xffffu;  // stride 0
    r.z = bytes;
    r.w = 0x00020000u;
    return r;
}

__device__ __forceinline__ uint32_t lds_addr(const void* p)
{
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

__device__ __forceinline__ void buf_load16_lds(const u32x4_t& rsrc, uint32_t off, uint32_t lds_base)
{
    lds_base = __builtin_amdgcn_readfirstlane(lds_base);  // wave-uniform by contract
    uint32_t saved;
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %3\n\t"
        "s_nop 0\n\t"
        "buffer_load_dwordx4 %1, %2, 0 offen lds\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "v"(off), "s"(rsrc), "s"(lds_base));
}

// The same for 4 bytes per lane: lane l's word lands at lds_base + 4*l.
__device__ __forceinline__ void buf_load4_lds(const u32x4_t& rsrc, uint32_t off, uint32_t lds_base)
{
    lds_base = __builtin_amdgcn_readfirstlane(lds_base);  // wave-uniform by contract
    uint32_t saved;
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %3\n\t"
        "s_nop 0\n\t"
        "buffer_load_dword %1, %2, 0 offen lds\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "v"(off), "s"(rsrc), "s"(lds_base));
}

// Wait until all of this wave's vector memory operations have completed.
__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0f70); }
// Wait until at most n (0..7) of this wave's vector memory operations are
// outstanding: the oldest ones (copies complete in issue order) have landed.
__device__ __forceinline__ void wait_vmem_upto(int n)
{
    switch (n) {
    case 0: __builtin_amdgcn_s_waitcnt(0x0f70); break;
    case 1: __builtin_amdgcn_s_waitcnt(0x0f71); break;
    case 2: __builtin_amdgcn_s_waitcnt(0x0f72); break;
    case 3: __builtin_amdgcn_s_waitcnt(0x0f73); break;
    case 4: __builtin_amdgcn_s_waitcnt(0x0f74); break;
    case 5: __builtin_amdgcn_s_waitcnt(0x0f75); break;
    case 6: __builtin_amdgcn_s_waitcnt(0x0f76); break;
    default: __builtin_amdgcn_s_waitcnt(0x0f77); break;
    }
}
// vmcnt(0) and lgkmcnt(0): this wave's copies have landed and its LDS reads are done.
__device__ __forceinline__ void wait_vmem_lds() { __builtin_amdgcn_s_waitcnt(0x0070); }

// Reduction split of the data-gradient GEMM: with T tiles and `slots`
// resident workgroups, split every tile's `nsteps` reduction steps S ways
// when at least two tiles' worth of workgroups would otherwise sit idle.
__host__ __device__ inline int data_split(int T, int nsteps, int slots, int smax)
{
    if (T <= 0 || 2 * T > slots) return 1;
    int sp = slots / T;
    if (sp > smax) sp = smax;
    if (sp > nsteps) sp = nsteps;
    return sp < 1 ? 1 : sp;
}

// XCD-aware block order.  The dispatcher hands consecutive workgroups to the
// eight XCDs in turn; this maps the j-th workgroup an XCD receives to the
// j-th tile of a contiguous range owned by that XCD, so tiles that share
// operands share one L2.  A bijection on [0, nb) for any nb.
__device__ __forceinline__ int xcd_remap(int b, int nb)
{
    const int xcd = b & 7, j = b >> 3;
    const int per = nb >> 3, rem = nb & 7;
    return xcd * per + (xcd < rem ? xcd : rem) + j;
}

// Swizzle of a 16-byte chunk inside a 256-byte LDS row (16 chunks).  Chosen
// so that sixteen consecutive rows read at one logical chunk, and rows
// 8c + j for c = 0..15 written at one logical chunk, fall on sixteen
// different chunk positions.
__device__ __forceinline__ int swz16(int row)
{
    return (row & 15) ^ ((row >> 4) & 7);
}

}  // namespace cbw
