// Shared device helpers for the gfx950 kernels: vector types, buffer
// resources (out-of-range loads return zero), and conversions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pifa {

typedef __bf16 bf16;
typedef _Float16 f16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

// Raw buffer resource over [base, base + bytes).  Loads at a byte offset
// >= bytes return 0, which pads ragged tiles without branches.  Word 3 is
// the gfx9 raw-buffer format (32-bit data, no swizzle, range checked).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
    const uint32_t n = bytes <= 0 ? 0u : (bytes >= 0xFFFFFFFFll ? 0xFFFFFFFFu : (uint32_t)bytes);
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)n, 0x00020000);
}

__device__ __forceinline__ u32x4 load16(__amdgpu_buffer_rsrc_t rs, uint32_t byte_off) {
    return __builtin_amdgcn_raw_buffer_load_b128(rs, (int)byte_off, 0, 0);
}

__device__ __forceinline__ u32x4 zero16() {
    u32x4 z = {0u, 0u, 0u, 0u};
    return z;
}

// fp32 -> bf16, round to nearest even (NaN stays NaN).
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float v) {
    uint32_t u = __builtin_bit_cast(uint32_t, v);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t b) {
    return __builtin_bit_cast(float, (uint32_t)b << 16);
}

// Output element stores for the two storage dtypes.
template <typename T>
struct Store;
template <>
struct Store<bf16> {
    __device__ __forceinline__ static void put(bf16* p, float v) {
        *reinterpret_cast<uint16_t*>(p) = f32_to_bf16_bits(v);
    }
};
template <>
struct Store<float> {
    __device__ __forceinline__ static void put(float* p, float v) { *p = v; }
};

__host__ __device__ constexpr int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
__host__ __device__ constexpr int64_t round_up(int64_t a, int64_t b) { return ceil_div(a, b) * b; }

}  // namespace pifa
