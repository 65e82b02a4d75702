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

// Streams `bytes` (a multiple of 16) of a buffer with 16-byte loads, four in
// flight per thread, and stores one word per workgroup (the XOR of what it
// read) so the loads are kept.
__global__ __launch_bounds__(256) void hbm_read_probe(const u32x4* __restrict__ buf, int64_t n16, uint32_t* sink) {
    uint32_t x = 0;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    for (; i + 3 * stride < n16; i += 4 * stride) {
        const u32x4 v0 = buf[i], v1 = buf[i + stride], v2 = buf[i + 2 * stride], v3 = buf[i + 3 * stride];
        x ^= v0[0] ^ v0[1] ^ v0[2] ^ v0[3] ^ v1[0] ^ v1[1] ^ v1[2] ^ v1[3];
        x ^= v2[0] ^ v2[1] ^ v2[2] ^ v2[3] ^ v3[0] ^ v3[1] ^ v3[2] ^ v3[3];
    }
    for (; i < n16; i += stride) {
        const u32x4 v = buf[i];
        x ^= v[0] ^ v[1] ^ v[2] ^ v[3];
    }
    __shared__ uint32_t red[4];
    for (int o = 32; o > 0; o >>= 1) x ^= __shfl_xor(x, o);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = x;
    __syncthreads();
    if (threadIdx.x == 0) sink[blockIdx.x] = red[0] ^ red[1] ^ red[2] ^ red[3];
}

}  // namespace pifa
