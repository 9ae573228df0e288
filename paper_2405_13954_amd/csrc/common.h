// Device-side helpers shared by the LoGra HIP kernels (gfx950 / CDNA4).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace logra {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef double f64x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t bf16_bits;

constexpr int kWave = 64;

// 128-bit load as four dwords (the only global access width the streaming
// kernels use).
__device__ __forceinline__ u32x4 ld128(const void *p) {
    return *reinterpret_cast<const u32x4 *>(p);
}
// Streaming 128-bit load of data read exactly once (non-temporal hint).
__device__ __forceinline__ u32x4 ld128_nt(const void *p) {
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
}

// Raw buffer resource over [base, base + bytes): a lane whose byte offset is
// at or beyond `bytes` reads zeros and touches no memory (the hardware range
// check), which is how masked tokens and contraction tails are skipped
// without branches.
constexpr uint32_t kBufOOB = 0x80000000u;   // an offset beyond every range used here
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), static_cast<short>(0),
                                             static_cast<int>(bytes), 0x00020000);
}
// The same, for a base and size the compiler cannot prove wave-uniform
// although they are: both are taken from lane 0, so that the descriptor lives
// in scalar registers.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc_uniform(const void *base, uint32_t bytes) {
    const uint64_t p = reinterpret_cast<uint64_t>(base);
    const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(p));
    const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(p >> 32));
    const uint64_t q = (static_cast<uint64_t>(hi) << 32) | lo;
    return buf_rsrc(reinterpret_cast<const void *>(q), __builtin_amdgcn_readfirstlane(bytes));
}
__device__ __forceinline__ u32x4 buf_ld128(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, static_cast<int>(off), 0, 0);
}
// Same, marked non-temporal (nt): for data streamed once, so that it does not
// push reused data (projection matrices) out of L2.
__device__ __forceinline__ u32x4 buf_ld128_nt(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, static_cast<int>(off), 0, 2);
}

// gfx950 asynchronous copy: 16 bytes per lane from buffer offset `voff`
// straight into LDS at byte address lds + 16 * lane (lds is wave-uniform);
// offsets at or past the buffer's range store zeros.  The load reads M0 one
// wait state after the scalar write (s_nop 0), as the hardware requires.  It
// is tracked by vmcnt, which the callers wait on explicitly (s_waitcnt in
// inline asm): the compiler does not see this load.
__device__ __forceinline__ void copy_to_lds(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t lds) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                 :: "s"(lds), "v"(voff), "s"(r) : "memory");
}

// The same copy with the non-temporal hint (nt): the lines it brings in are
// the first to be evicted, for an operand that is streamed once.
__device__ __forceinline__ void copy_to_lds_nt(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t lds) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen nt lds"
                 :: "s"(lds), "v"(voff), "s"(r) : "memory");
}

// 32-bit LDS byte address of a __shared__ object (the address-space cast
// yields the offset within the workgroup's LDS allocation).
template <typename T>
__device__ __forceinline__ uint32_t lds_addr(T *p) {
    return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) T *)p));
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) {
    return __builtin_bit_cast(bf16x8, v);
}
__device__ __forceinline__ f32x4 as_f32x4(u32x4 v) { return __builtin_bit_cast(f32x4, v); }

__device__ __forceinline__ float bf16_to_f32(bf16_bits h) {
    return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

// fp32 -> bf16, round to nearest, ties to even; NaN stays a quiet NaN.
__device__ __forceinline__ bf16_bits f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<bf16_bits>((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return static_cast<bf16_bits>(u >> 16);
}

template <typename T>
__device__ __forceinline__ void store_out(T *p, float v);
template <>
__device__ __forceinline__ void store_out<float>(float *p, float v) { *p = v; }
template <>
__device__ __forceinline__ void store_out<bf16_bits>(bf16_bits *p, float v) {
    *p = f32_to_bf16_rne(v);
}

template <typename T>
__device__ __forceinline__ void store_out_d(T *p, double v);
template <>
__device__ __forceinline__ void store_out_d<float>(float *p, double v) { *p = static_cast<float>(v); }
template <>
__device__ __forceinline__ void store_out_d<bf16_bits>(bf16_bits *p, double v) {
    *p = f32_to_bf16_rne(static_cast<float>(v));
}
template <>
__device__ __forceinline__ void store_out_d<double>(double *p, double v) { *p = v; }

template <typename T>
__device__ __forceinline__ double load_in_d(const T *p);
template <>
__device__ __forceinline__ double load_in_d<float>(const float *p) { return static_cast<double>(*p); }
template <>
__device__ __forceinline__ double load_in_d<bf16_bits>(const bf16_bits *p) {
    return static_cast<double>(bf16_to_f32(*p));
}
template <>
__device__ __forceinline__ double load_in_d<double>(const double *p) { return *p; }

// Matrix-core products.  Operand layouts of the 16x16 shapes: lane l holds
// row (l % 16) of A and column (l % 16) of B, with the contraction slice
// selected by l / 16; the result holds rows 4*(l/16) + r, r < 4, of column
// l % 16.  Any assignment of contraction indices to (l/16, element) is valid
// as long as A and B use the same one.
// A double from lane `src` (a compile-time lane), as two 32-bit readlanes.
__device__ __forceinline__ double readlane_d(double v, int src) {
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(u), src));
    const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(u >> 32), src));
    return __builtin_bit_cast(double, (static_cast<uint64_t>(hi) << 32) | lo);
}

__device__ __forceinline__ f32x4 mfma16_bf16(bf16x8 a, bf16x8 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma16_f32(float a, float b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}
// fp64 16x16x4: same operand layout, but result register r of lane l holds
// row (l/16) + 4r of column l % 16 (rows interleaved, unlike the fp32 shapes).
__device__ __forceinline__ f64x4 mfma16_f64(double a, double b, f64x4 c) {
    return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
}
// 32x32x16: lane l holds row (l % 32) of A / column (l % 32) of B; result
// register r holds row 8*(r/4) + 4*(l/32) + (r%4) of column l % 32.
__device__ __forceinline__ f32x16 mfma32_bf16(bf16x8 a, bf16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

}  // namespace logra
