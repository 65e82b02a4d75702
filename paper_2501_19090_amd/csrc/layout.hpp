// Weight layout of the matrices a layer handle owns.
//
// "MFMA-lane order": an N x K weight matrix (row n produces output column n,
// K is the reduction axis) is cut into blocks of 16 rows x 128 columns.
// Block (g, b) -- rows 16g..16g+15, columns 128b..128b+127 -- is 4 KB at
// block index g * KB + b (KB = ceil(K / 128)); inside it, the 16-byte chunk
// at position c * 64 + l (c = 0..3, l = 0..63) holds
//     row 16g + (l % 16), columns 128b + 32 (l / 16) + 8c ... +7.
// That is exactly what lane l of a wave feeds as the B operand of the c-th
// MFMA 16x16x32 when the wave covers 128 columns of the block, so the decode
// kernel streams each block with four fully coalesced 1 KB wave loads.  The
// prefill GEMM reads the same layout into its LDS tiles.  Rows past N and
// columns past K are zero.
#pragma once

#include "common.hpp"

namespace pifa {

constexpr int kPackRows = 16;
constexpr int kPackCols = 128;
constexpr int kPackChunks = kPackRows * kPackCols / 8;  // 256 chunks of 16 B per block

__host__ __device__ inline int64_t packed_groups(int64_t N) { return ceil_div(N, kPackRows); }
__host__ __device__ inline int64_t packed_kblocks(int64_t K) { return ceil_div(K, kPackCols); }
__host__ __device__ inline int64_t packed_elems(int64_t N, int64_t K) {
    return packed_groups(N) * packed_kblocks(K) * kPackChunks * 8;
}

// Pack src (rows x cols, row stride ld, bf16 bits or fp32 bits of width
// sizeof(TS)) into the lane-ordered layout of a (rows_log x cols_log) matrix
// with dtype TD; elements outside rows x cols are zero.  For TS = uint16_t
// (bf16) and TD = f16 every value is multiplied by `scale` (a power of two).
template <typename TS, typename TD>
__global__ void pack_lane_order(const TS* __restrict__ src, int64_t rows, int64_t cols, int64_t ld,
                                TD* __restrict__ dst, int64_t rows_log, int64_t cols_log,
                                float scale) {
    const int64_t KB = packed_kblocks(cols_log);
    const int64_t nchunks = packed_groups(rows_log) * KB * kPackChunks;
    for (int64_t ch = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; ch < nchunks;
         ch += (int64_t)gridDim.x * blockDim.x) {
        const int64_t blk = ch / kPackChunks;
        const int pos = (int)(ch % kPackChunks);
        const int c = pos / 64, l = pos % 64;
        const int64_t g = blk / KB, b = blk % KB;
        const int64_t n = g * kPackRows + (l % 16);
        const int64_t k0 = b * kPackCols + 32 * (l / 16) + 8 * c;
        TD* out = dst + ch * 8;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int64_t k = k0 + e;
            if (n < rows && k < cols) {
                if constexpr (sizeof(TS) == 2 && sizeof(TD) == 2 && !__is_same(TD, f16)) {
                    out[e] = src[n * ld + k];  // bf16 bits copied as-is
                } else if constexpr (__is_same(TD, f16)) {
                    out[e] = (f16)(bf16_bits_to_f32((uint16_t)src[n * ld + k]) * scale);
                } else {
                    out[e] = src[n * ld + k];
                }
            } else {
                out[e] = TD(0);
            }
        }
    }
}

}  // namespace pifa
