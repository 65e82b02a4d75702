// Diagnostic kernels that confirm the chip's peaks on the machine at hand:
// the sustained matrix-core rate with the shader clock it runs at, and the
// HBM read rate.  Not part of any layer's path.
#pragma once

#include "common.hpp"
#include "gemm_mfma.hpp"

namespace pifa {

// Each wave issues `iters` rounds of four independent bf16 32x32x16 MFMAs on
// register operands (no memory traffic).  Lane 0 of wave 0 records the
// shader-clock cycles (s_memtime) and the 100 MHz real-time ticks
// (s_memrealtime) that the workgroup's loop took, so the host can derive the
// clock the matrix cores actually ran at.  `seed` keeps the operands unknown
// at compile time; the sum of the accumulators is stored only if it equals
// `seed` exactly (never, for seed = 0 and nonzero operands), which keeps the
// loop from being removed.
__global__ __launch_bounds__(256) void mfma_probe(int64_t iters, float seed, float* sink, uint64_t* clocks) {
    const int lane = threadIdx.x & (kWave - 1);
    const uint32_t bits = 0x3F803F80u ^ (uint32_t)(lane & 7) ^ __builtin_bit_cast(uint32_t, seed);
    const u32x4 a = {bits, bits ^ 1u, bits ^ 2u, bits ^ 3u};
    const u32x4 b = {bits ^ 4u, bits ^ 5u, bits ^ 6u, bits ^ 7u};
    f32x16 c0{}, c1{}, c2{}, c3{};
    const uint64_t cyc0 = __builtin_amdgcn_s_memtime();
    const uint64_t rt0 = __builtin_amdgcn_s_memrealtime();
    for (int64_t i = 0; i < iters; ++i) {
        c0 = Mfma<bf16>::mma32(a, b, c0);
        c1 = Mfma<bf16>::mma32(b, a, c1);
        c2 = Mfma<bf16>::mma32(a, a, c2);
        c3 = Mfma<bf16>::mma32(b, b, c3);
    }
    float s = 0.f;
#pragma unroll
    for (int v = 0; v < 16; ++v) s += c0[v] + c1[v] + c2[v] + c3[v];
    const uint64_t cyc1 = __builtin_amdgcn_s_memtime();
    const uint64_t rt1 = __builtin_amdgcn_s_memrealtime();
    if (s == seed) sink[blockIdx.x] = s;
    if (threadIdx.x == 0) {
        clocks[2 * blockIdx.x] = cyc1 - cyc0;
        clocks[2 * blockIdx.x + 1] = rt1 - rt0;
    }
}

// The same loop on operands that change with every MFMA, as a GEMM's do:
// each wave holds 8 register sets of random bf16 values (random sign and
// mantissa, magnitudes in [0.5, 1)) and each MFMA of a round of 8 takes a
// different pair.  Matrix-core power depends on how many operand bits toggle,
// so under the board's power limit this loop runs at a lower clock than
// mfma_probe's constant operands; the pair of rates brackets what a GEMM on
// real data can reach.  `iters` is a multiple of 8.
__device__ __forceinline__ uint32_t probe_mix(uint32_t x) {
    x ^= x >> 16;
    x *= 0x7FEB352Du;
    x ^= x >> 15;
    x *= 0x846CA68Bu;
    x ^= x >> 16;
    return x;
}

__global__ __launch_bounds__(256) void mfma_probe_random(int64_t iters, float seed, float* sink, uint64_t* clocks) {
    const uint32_t base = (uint32_t)(blockIdx.x * 256 + threadIdx.x) * 64u ^ __builtin_bit_cast(uint32_t, seed);
    u32x4 a[8], b[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            a[q][w] = (probe_mix(base + 8 * q + w) & 0x807F807Fu) | 0x3F003F00u;
            b[q][w] = (probe_mix(base + 8 * q + w + 4) & 0x807F807Fu) | 0x3F003F00u;
        }
    }
    f32x16 c0{}, c1{}, c2{}, c3{};
    const uint64_t cyc0 = __builtin_amdgcn_s_memtime();
    const uint64_t rt0 = __builtin_amdgcn_s_memrealtime();
    for (int64_t i = 0; i < iters; i += 8) {
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            c0 = Mfma<bf16>::mma32(a[q], b[q], c0);
            c1 = Mfma<bf16>::mma32(b[(q + 1) & 7], a[(q + 3) & 7], c1);
            c2 = Mfma<bf16>::mma32(a[(q + 5) & 7], b[(q + 2) & 7], c2);
            c3 = Mfma<bf16>::mma32(b[(q + 6) & 7], a[(q + 7) & 7], c3);
        }
    }
    float s = 0.f;
#pragma unroll
    for (int v = 0; v < 16; ++v) s += c0[v] + c1[v] + c2[v] + c3[v];
    const uint64_t cyc1 = __builtin_amdgcn_s_memtime();
    const uint64_t rt1 = __builtin_amdgcn_s_memrealtime();
    if (s == seed) sink[blockIdx.x] = s;
    if (threadIdx.x == 0) {
        clocks[2 * blockIdx.x] = cyc1 - cyc0;
        clocks[2 * blockIdx.x + 1] = rt1 - rt0;
    }
}

// Streams `n16` 16-byte words of a buffer, one load per thread per step of a
// grid-stride loop; a word is stored only if the XOR of what a thread read
// equals a fixed constant (which keeps the loads; the benchmark's zero-filled
// buffer never matches).
__global__ __launch_bounds__(256) void hbm_read_probe(const u32x4* __restrict__ buf, int64_t n16, uint32_t* sink) {
    uint32_t x = 0;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += (int64_t)gridDim.x * blockDim.x) {
        const u32x4 v = buf[i];
        x ^= v[0] ^ v[1] ^ v[2] ^ v[3];
    }
    if (x == 0x9E3779B9u) sink[blockIdx.x] = x;
}

}  // namespace pifa
