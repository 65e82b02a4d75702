// One-off weight preparation at layer creation.
#pragma once

#include "common.hpp"

namespace pifa {

// dst (rows_pad x cols_pad) = src (rows x cols, row stride ld) zero-padded.
template <typename T>
__global__ void pack_pad(const T* __restrict__ src, int64_t rows, int64_t cols, int64_t ld,
                         T* __restrict__ dst, int64_t rows_pad, int64_t cols_pad) {
    const int64_t total = rows_pad * cols_pad;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = e / cols_pad, j = e % cols_pad;
        dst[e] = (i < rows && j < cols) ? src[i * ld + j] : T(0);
    }
}

// Largest finite |x| of a bf16 array, as magnitude bits (monotone in |x|).
__global__ void absmax_bf16(const uint16_t* __restrict__ src, int64_t n, unsigned* __restrict__ out) {
    unsigned mx = 0;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n;
         e += (int64_t)gridDim.x * blockDim.x) {
        const unsigned b = src[e] & 0x7FFFu;
        if (b < 0x7F80u && b > mx) mx = b;
    }
    for (int off = kWave / 2; off > 0; off >>= 1) {
        const unsigned o = __shfl_down(mx, off);
        mx = o > mx ? o : mx;
    }
    if ((threadIdx.x & (kWave - 1)) == 0) atomicMax(out, mx);
}

// dst (rows_pad x cols_pad, fp16) = src (bf16, rows x cols) * scale, zero
// padded.  scale is a power of two chosen so the largest |x| * scale lies in
// [2^14, 2^15): bf16's 8 significant bits fit fp16's 11, so every entry not
// pushed below fp16's normal range (|x| < max|x| * 2^-28) converts exactly.
__global__ void bf16_to_f16_scaled(const uint16_t* __restrict__ src, int64_t rows, int64_t cols,
                                   f16* __restrict__ dst, int64_t rows_pad, int64_t cols_pad,
                                   float scale) {
    const int64_t total = rows_pad * cols_pad;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = e / cols_pad, j = e % cols_pad;
        const float v = (i < rows && j < cols) ? bf16_bits_to_f32(src[i * cols + j]) : 0.f;
        dst[e] = (f16)(v * scale);
    }
}

}  // namespace pifa
