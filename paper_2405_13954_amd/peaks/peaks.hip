// Measured ceilings: a sustained bf16 MFMA loop and an HBM read stream (see
// include/logra_peaks.h).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "logra_peaks.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void k_peak_mfma(int64_t iters, float *sink, int64_t *cycles) {
    const int tid = threadIdx.x;
    // operands that the compiler cannot fold: small values from the thread index
    bf16x8 a, b;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        a[e] = static_cast<__bf16>(static_cast<float>((tid + e) & 7) * 0.125f);
        b[e] = static_cast<__bf16>(static_cast<float>((tid * 3 + e) & 7) * 0.0625f);
    }
    f32x16 c0 = {}, c1 = {}, c2 = {}, c3 = {};
    const long long t0 = clock64(), w0 = wall_clock64();
    for (int64_t i = 0; i < iters; ++i) {
        c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c0, 0, 0, 0);
        c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c1, 0, 0, 0);
        c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c2, 0, 0, 0);
        c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c3, 0, 0, 0);
    }
    const long long t1 = clock64(), w1 = wall_clock64();
    float s = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) s += c0[r] + c1[r] + c2[r] + c3[r];
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
    if (tid == 0) {
        sink[blockIdx.x] = s;
        if (cycles && blockIdx.x == 0) {
            cycles[0] = t1 - t0;
            cycles[1] = w1 - w0;
        }
    }
}

// The same loop on data: each lane holds 16 operand fragments read from
// `ops` (random bf16 values), and the MFMAs take them in the pattern of a
// register-tiled GEMM: one A fragment for four MFMAs in a row (one per
// accumulator), a different B fragment for each.  The multiplier inputs then
// change from one MFMA to the next as they do in a GEMM on real data.  (The
// loop above feeds every MFMA the same two fragments of short-mantissa
// values, which toggles far fewer bits.)
__global__ __launch_bounds__(256) void k_peak_mfma_data(const u32x4 *ops, int64_t iters, float *sink,
                                                        int64_t *cycles) {
    const int tid = threadIdx.x;
    const u32x4 *src = ops + static_cast<size_t>(blockIdx.x & 15) * (16 * 256) + tid;
    bf16x8 f[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) f[r] = __builtin_bit_cast(bf16x8, src[r * 256]);
    f32x16 c0 = {}, c1 = {}, c2 = {}, c3 = {};
    const long long t0 = clock64(), w0 = wall_clock64();
    for (int64_t i = 0; i < iters; i += 8) {
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[u], f[8 + u], c0, 0, 0, 0);
            c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[u], f[8 + ((u + 1) & 7)], c1, 0, 0, 0);
            c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[u], f[8 + ((u + 2) & 7)], c2, 0, 0, 0);
            c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[u], f[8 + ((u + 3) & 7)], c3, 0, 0, 0);
        }
    }
    const long long t1 = clock64(), w1 = wall_clock64();
    float s = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) s += c0[r] + c1[r] + c2[r] + c3[r];
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
    if (tid == 0) {
        sink[blockIdx.x] = s;
        if (cycles && blockIdx.x == 0) {
            cycles[0] = t1 - t0;
            cycles[1] = w1 - w0;
        }
    }
}

// Mode 0: grid-stride 128-bit loads, four in flight per thread.
__global__ __launch_bounds__(256) void k_peak_read(const u32x4 *buf, int64_t n, float *sink) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * 256;
    int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    uint32_t x = 0;
    for (; i + 3 * stride < n; i += 4 * stride) {
        const u32x4 v0 = buf[i], v1 = buf[i + stride], v2 = buf[i + 2 * stride], v3 = buf[i + 3 * stride];
        x ^= v0[0] ^ v0[1] ^ v0[2] ^ v0[3] ^ v1[0] ^ v1[1] ^ v1[2] ^ v1[3];
        x ^= v2[0] ^ v2[1] ^ v2[2] ^ v2[3] ^ v3[0] ^ v3[1] ^ v3[2] ^ v3[3];
    }
    for (; i < n; i += stride) {
        const u32x4 v = buf[i];
        x ^= v[0] ^ v[1] ^ v[2] ^ v[3];
    }
    for (int o = 32; o > 0; o >>= 1) x ^= __shfl_xor(x, o, 64);
    if (threadIdx.x == 0) sink[blockIdx.x] = static_cast<float>(x & 0xffff);
}

// Mode 1: each workgroup streams its own contiguous range, eight
// non-temporal 128-bit loads in flight per thread.
__global__ __launch_bounds__(256) void k_peak_read_blocked(const u32x4 *buf, int64_t n, float *sink) {
    const int64_t per = (n + gridDim.x - 1) / gridDim.x;
    const int64_t b0 = static_cast<int64_t>(blockIdx.x) * per;
    const int64_t b1 = b0 + per < n ? b0 + per : n;
    uint32_t x = 0;
    int64_t i = b0 + threadIdx.x;
    for (; i + 7 * 256 < b1; i += 8 * 256) {
        u32x4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = __builtin_nontemporal_load(buf + i + u * 256);
#pragma unroll
        for (int u = 0; u < 8; ++u) x ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
    }
    for (; i < b1; i += 256) {
        const u32x4 v = buf[i];
        x ^= v[0] ^ v[1] ^ v[2] ^ v[3];
    }
    for (int o = 32; o > 0; o >>= 1) x ^= __shfl_xor(x, o, 64);
    if (threadIdx.x == 0) sink[blockIdx.x] = static_cast<float>(x & 0xffff);
}

// Mode 2: each wave streams its own contiguous range into an LDS ring with
// asynchronous global-to-LDS copies of 1 KB (whole 128-byte lines), eight
// copies in flight, the way the projection streams its operands.
__global__ __launch_bounds__(256) void k_peak_read_lds(const uint8_t *buf, int64_t bytes, float *sink) {
    __shared__ __attribute__((aligned(1024))) uint8_t ring[4][16 * 1024];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t waves = static_cast<int64_t>(gridDim.x) * 4;
    const int64_t w = static_cast<int64_t>(blockIdx.x) * 4 + wave;
    const int64_t kb = bytes / 1024;                       // 1 KB copies in all
    const int64_t per = (kb + waves - 1) / waves;
    int64_t c0 = w * per, c1 = c0 + per < kb ? c0 + per : kb;
    const uint32_t lds = static_cast<uint32_t>(
        reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) uint8_t *)&ring[wave][0]));
    int slot = 0;
    for (int64_t c = c0; c < c1; ++c) {
        // a window of the buffer small enough for 32-bit offsets
        const uint8_t *base = buf + c * 1024;
        const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint8_t *>(base), static_cast<short>(0), 1024, 0x00020000);
        asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen nt lds"
                     :: "s"(lds + slot * 1024), "v"(static_cast<uint32_t>(lane * 16)), "s"(r) : "memory");
        slot = (slot + 1) & 15;
        asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (threadIdx.x == 0) sink[blockIdx.x] = static_cast<float>(ring[0][0] + ring[3][1023]);
}

}  // namespace

extern "C" int logra_peak_mfma_bf16(int groups, int64_t iters, float *sink, int64_t *cycles_out, void *stream) {
    if (groups <= 0 || iters <= 0 || sink == nullptr) return -1;
    hipLaunchKernelGGL(k_peak_mfma, dim3(groups), dim3(256), 0, static_cast<hipStream_t>(stream), iters, sink,
                       cycles_out);
    return hipGetLastError() == hipSuccess ? 0 : -3;
}

extern "C" int logra_peak_mfma_bf16_data(int groups, int64_t iters, const void *ops, float *sink,
                                         int64_t *cycles_out, void *stream) {
    if (groups <= 0 || iters <= 0 || iters % 8 != 0 || ops == nullptr || sink == nullptr ||
        (reinterpret_cast<uintptr_t>(ops) & 15) != 0)
        return -1;
    hipLaunchKernelGGL(k_peak_mfma_data, dim3(groups), dim3(256), 0, static_cast<hipStream_t>(stream),
                       static_cast<const u32x4 *>(ops), iters, sink, cycles_out);
    return hipGetLastError() == hipSuccess ? 0 : -3;
}

extern "C" int logra_peak_hbm_read(const void *buf, size_t bytes, int groups, int mode, float *sink, void *stream) {
    if (buf == nullptr || sink == nullptr || groups <= 0 || bytes == 0 || bytes % 1024 != 0 ||
        (reinterpret_cast<uintptr_t>(buf) & 1023) != 0 || mode < 0 || mode > 2)
        return -1;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    if (mode == 0)
        hipLaunchKernelGGL(k_peak_read, dim3(groups), dim3(256), 0, s, static_cast<const u32x4 *>(buf),
                           static_cast<int64_t>(bytes / 16), sink);
    else if (mode == 1)
        hipLaunchKernelGGL(k_peak_read_blocked, dim3(groups), dim3(256), 0, s, static_cast<const u32x4 *>(buf),
                           static_cast<int64_t>(bytes / 16), sink);
    else
        hipLaunchKernelGGL(k_peak_read_lds, dim3(groups), dim3(256), 0, s, static_cast<const uint8_t *>(buf),
                           static_cast<int64_t>(bytes), sink);
    return hipGetLastError() == hipSuccess ? 0 : -3;
}

extern "C" int logra_peak_wall_clock_khz(int *khz) {
    int dev = 0;
    if (khz == nullptr || hipGetDevice(&dev) != hipSuccess) return -1;
    return hipDeviceGetAttribute(khz, hipDeviceAttributeWallClockRate, dev) == hipSuccess ? 0 : -3;
}
