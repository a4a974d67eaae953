// common.hpp -- types and small device helpers shared by the libnnconv
// kernels (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace nnconv {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Operand element types.  Both are 16-bit storage formats; products are
// accumulated in fp32 by the matrix cores.
struct Half {
    static constexpr int id = 0;
};
struct BFloat {
    static constexpr int id = 1;
};

// D += A * B on a 32x32 output tile with a 16-deep reduction
// (v_mfma_f32_32x32x16_{f16,bf16}).  Each lane supplies 8 consecutive
// reduction elements of one row of A (row = lane % 32) and of one column of
// B (column = lane % 32); lanes 0-31 hold reduction slots 0-7, lanes 32-63
// slots 8-15.  Result: lane holds column lane % 32, rows
// 8*(i/4) + 4*(lane/32) + i%4 for i = 0..15.
template <class T>
__device__ __forceinline__ f32x16 mfma32(u32x4 a, u32x4 b, f32x16 c);

template <>
__device__ __forceinline__ f32x16 mfma32<Half>(u32x4 a, u32x4 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a),
                                                  __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}

template <>
__device__ __forceinline__ f32x16 mfma32<BFloat>(u32x4 a, u32x4 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// fp32 -> 16-bit storage, round to nearest even, overflow to +-inf.
template <class T>
__device__ __forceinline__ uint32_t to16(float v);

template <>
__device__ __forceinline__ uint32_t to16<Half>(float v) {
    _Float16 h = (_Float16)v;
    return (uint32_t)__builtin_bit_cast(uint16_t, h);
}

template <>
__device__ __forceinline__ uint32_t to16<BFloat>(float v) {
    __bf16 h = (__bf16)v;
    return (uint32_t)__builtin_bit_cast(uint16_t, h);
}

// 16-bit storage -> fp32 (exact).
template <class T>
__device__ __forceinline__ float from16(uint32_t bits);

template <>
__device__ __forceinline__ float from16<Half>(uint32_t bits) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)bits);
}

template <>
__device__ __forceinline__ float from16<BFloat>(uint32_t bits) {
    return __builtin_bit_cast(float, bits << 16);
}

// Buffer resources: raw (unswizzled) addressing with a byte range check.
// A load whose offset lies at or beyond num_records returns zero, which
// gives zero padding for free: masked lanes use OOB_OFFSET.
constexpr uint32_t OOB_OFFSET = 0x80000000u;
constexpr uint32_t MAX_BUFFER_BYTES = 0x7FFFFFF0u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes,
                                             0x00020000);
}

__device__ __forceinline__ u32x4 load16(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, 0);
}

// Unsigned division by a run-time constant d >= 1 for dividends below 2^31:
// q = (mulhi(n, m) + n) >> s with s = ceil(log2 d), m = floor(2^32 (2^s - d) / d) + 1.
struct FastDiv {
    uint32_t d, m, s;
};

inline FastDiv make_fastdiv(uint32_t d) {
    FastDiv f;
    f.d = d;
    uint32_t s = 0;
    while ((1ull << s) < d) ++s;
    f.s = s;
    f.m = (uint32_t)((((1ull << s) - d) << 32) / d + 1);
    return f;
}

__device__ __forceinline__ uint32_t fdiv(uint32_t n, const FastDiv &f) {
    return (__umulhi(n, f.m) + n) >> f.s;
}

// Workgroup ids are dealt round-robin to the 8 XCDs (each with its own L2).
// Renumber them so that consecutive logical tiles run on the same XCD.
__device__ __forceinline__ uint32_t xcd_remap(uint32_t bid, uint32_t nblocks) {
    const uint32_t nx = 8;
    uint32_t q = nblocks / nx, r = nblocks % nx;
    uint32_t x = bid % nx, i = bid / nx;
    uint32_t base = (x < r) ? x * (q + 1) : r * (q + 1) + (x - r) * q;
    return base + i;
}

// LDS row swizzle for tiles of 8 x 16-byte chunks per row: logical chunk c
// of row r lives at physical chunk c ^ swz(r).  Consecutive rows read at the
// same logical chunk, and rows 8 apart written at the same logical chunk,
// fall in different 16-byte bank groups.
__device__ __forceinline__ int swz(int row) { return (row ^ (row >> 3)) & 7; }

// ---------------------------------------------------------------------------
// Direct-to-LDS staging and LDS hand-offs (shared by the matrix-core kernels)
// ---------------------------------------------------------------------------

typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

// Wait until at most `n` vector-memory operations of this wave are
// outstanding.  Written as asm with a memory clobber so no load or store
// moves across it.
template <int n>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(n >= 0 && n < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(n) : "memory");
}

// Workgroup barrier for LDS hand-offs between waves: first wait until this
// wave's own LDS reads and writes have completed (s_barrier alone does not),
// so data written before the barrier is what other waves read after it.  The
// memory clobber also keeps the compiler from moving LDS accesses across it
// (the direct-to-LDS loads are invisible to its dependence tracking).
__device__ __forceinline__ void barrier_lds() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Buffer descriptor (gfx9 format, raw addressing) for the bytes
// [base + shift, base + bytes); empty when shift >= bytes.  The words are
// made wave-uniform so they live in scalar registers.
__device__ __forceinline__ i32x4 desc_at(const void *base, uint32_t bytes, uint32_t shift) {
    const uint64_t a = (uint64_t)base + shift;
    i32x4 d;
    d[0] = __builtin_amdgcn_readfirstlane((int32_t)(uint32_t)a);
    d[1] = __builtin_amdgcn_readfirstlane((int32_t)((uint32_t)(a >> 32) & 0xFFFFu));
    d[2] = __builtin_amdgcn_readfirstlane((int32_t)(shift < bytes ? bytes - shift : 0u));
    d[3] = 0x00020000;
    return d;
}

__device__ __forceinline__ i32x4 desc_of(const void *base, uint32_t bytes) {
    return desc_at(base, bytes, 0);
}

// buffer_load_dwordx4 ... lds: lane i's 16 bytes from desc + voff go to LDS
// byte address lds_addr + 16*i; offsets at or past the descriptor's range
// deliver zeros.
__device__ __forceinline__ void dma16(uint32_t lds_addr, uint32_t voff, i32x4 desc) {
    asm volatile(
        "s_mov_b32 m0, %0\n\t"
        "buffer_load_dwordx4 %1, %2, 0 offen lds"
        :
        : "s"(__builtin_amdgcn_readfirstlane(lds_addr)), "v"(voff), "s"(desc)
        : "memory");
}

}  // namespace nnconv
