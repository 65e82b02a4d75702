// Kernels of the PIFA layer backward pass (bf16 layers).
//
// Forward (Algorithm "PIFA Layer", row-major):  Y_p = X W_p^T,
// Y_np = Y_p C^T, Y[:, I] = Y_p, Y[:, I^c] = Y_np.  With G = dL/dY the chain
// rule gives
//   G_p  = G[:, I] + G[:, I^c] C      (M x r)
//   dX   = G_p W_p                    (M x d_in)
//   dW_p = G_p^T X                    (r x d_in)
//   dC   = G[:, I^c]^T Y_p            (n_np x r)
// All four are products for the prefill GEMM (gemm_mfma.hpp), which wants
// both operands K-contiguous; this file holds the data movement that puts
// them in that form (gathers, tiled transposes, transposed weight packs) and
// the epilogue of the G_p product.
//
// Precision: G_p multiplies W_p in dX = G_p W_p with the same cancellation as
// Y_p C^T in the forward (C rebuilds W_np from W_p), so G_p is handed to that
// product as a bf16 pair hi + lo (about 16 significant bits) against W_p^T
// stored twice along K.  dW_p and dC have no such cancellation and use bf16
// operands; all products accumulate in fp32.
#pragma once

#include "common.hpp"
#include "layout.hpp"

namespace pifa {

// Element (n, k) of a lane-ordered matrix with KB 128-column blocks per row group.
__device__ __forceinline__ int64_t lane_order_index(int64_t n, int64_t k, int64_t KB) {
    const int64_t g = n / kPackRows, b = k / kPackCols;
    const int rr = (int)(n % kPackRows), cc = (int)(k % kPackCols);
    const int l = 16 * (cc / 32) + rr, c = (cc % 32) / 8, e = cc % 8;
    return ((g * KB + b) * kPackChunks + c * 64 + l) * 8 + e;
}

template <typename T>
__device__ __forceinline__ float to_f32(T v);
template <>
__device__ __forceinline__ float to_f32<bf16>(bf16 v) {
    return bf16_bits_to_f32(__builtin_bit_cast(uint16_t, v));
}
template <>
__device__ __forceinline__ float to_f32<f16>(f16 v) {
    return (float)v;
}

// dst = lane order of a (rows_log x cols_log) bf16 matrix whose element
// (i, c) is src(c mod period, i) * scale, where src is a lane-ordered matrix
// (src_kb column blocks per row group) of which rows < src_rows and columns
// < src_cols are valid; everything else is zero.  Used for W_p^T stored twice
// along K (period = r_pad) and for C^T in bf16 (period = cols_log, scale
// undoing C's fp16 scale, exact for bf16-representable C).
template <typename TS>
__global__ void pack_transposed(const TS* __restrict__ src, int64_t src_kb, int64_t src_rows, int64_t src_cols,
                                int64_t period, float scale, bf16* __restrict__ dst, int64_t rows_log,
                                int64_t cols_log) {
    const int64_t KB = packed_kblocks(cols_log);
    const int64_t nchunks = packed_groups(rows_log) * KB * kPackChunks;
    for (int64_t ch = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; ch < nchunks;
         ch += (int64_t)gridDim.x * blockDim.x) {
        const int64_t blk = ch / kPackChunks;
        const int pos = (int)(ch % kPackChunks);
        const int c = pos / 64, l = pos % 64;
        const int64_t g = blk / KB, b = blk % KB;
        const int64_t i = g * kPackRows + (l % 16);
        const int64_t k0 = b * kPackCols + 32 * (l / 16) + 8 * c;
        uint16_t* out = reinterpret_cast<uint16_t*>(dst) + ch * 8;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int64_t k = k0 + e;
            const int64_t s = k % period;
            float v = 0.f;
            if (i < rows_log && k < cols_log && s < src_rows && i < src_cols)
                v = to_f32<TS>(src[lane_order_index(s, i, src_kb)]) * scale;
            out[e] = f32_to_bf16_bits(v);
        }
    }
}

// out[m * ld_out + j] = in[m * ld_in + idx[j]] for j < ncols, zero for
// ncols <= j < ld_out (the K padding of a GEMM operand).
__global__ void gather_cols(const bf16* __restrict__ in, int64_t ld_in, int64_t M, const int32_t* __restrict__ idx,
                            int64_t ncols, bf16* __restrict__ out, int64_t ld_out) {
    const uint16_t* src = reinterpret_cast<const uint16_t*>(in);
    uint16_t* dst = reinterpret_cast<uint16_t*>(out);
    const int64_t total = M * ld_out;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t m = e / ld_out, j = e % ld_out;
        dst[e] = j < ncols ? src[m * ld_in + idx[j]] : (uint16_t)0;
    }
}

// out[j * ld_out + m] = in[m * ld_in + col(j)] for j < ncols and m < M, with
// col(j) = idx[j] (or j when idx is null); zero for M <= m < ld_out.  64 x 64
// tiles through LDS so both the reads (along j) and the writes (along m) are
// row-contiguous.  Grid: (ceil(ld_out / 64), ceil(ncols / 64)), 256 threads.
constexpr int kTrTile = 64;

__global__ __launch_bounds__(256) void gather_transpose(const bf16* __restrict__ in, int64_t ld_in, int64_t M,
                                                        const int32_t* __restrict__ idx, int64_t ncols,
                                                        bf16* __restrict__ out, int64_t ld_out) {
    __shared__ uint16_t tile[kTrTile][kTrTile + 1];
    const uint16_t* src = reinterpret_cast<const uint16_t*>(in);
    uint16_t* dst = reinterpret_cast<uint16_t*>(out);
    const int64_t m0 = (int64_t)blockIdx.x * kTrTile, j0 = (int64_t)blockIdx.y * kTrTile;
    const int tid = threadIdx.x;
#pragma unroll
    for (int i = 0; i < kTrTile * kTrTile / 256; ++i) {
        const int t = tid + 256 * i, mm = t / kTrTile, jj = t % kTrTile;
        const int64_t m = m0 + mm, j = j0 + jj;
        uint16_t v = 0;
        if (m < M && j < ncols) v = src[m * ld_in + (idx ? (int64_t)idx[j] : j)];
        tile[mm][jj] = v;
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kTrTile * kTrTile / 256; ++i) {
        const int t = tid + 256 * i, jj = t / kTrTile, mm = t % kTrTile;
        const int64_t m = m0 + mm, j = j0 + jj;
        if (j < ncols && m < ld_out) dst[j * ld_out + m] = tile[mm][jj];
    }
}

// Zero columns [c0, ld) of a rows x ld bf16 matrix.
__global__ void zero_cols(bf16* __restrict__ p, int64_t rows, int64_t ld, int64_t c0) {
    uint16_t* q = reinterpret_cast<uint16_t*>(p);
    const int64_t w = ld - c0, total = rows * w;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x)
        q[(e / w) * ld + c0 + e % w] = 0;
}

// Epilogue of G_p = G[:, I^c] C (+ G[:, I]): acc(m, j) for j < r_pad.
//   * adds G[m, piv[j]] for j < r;
//   * writes the bf16 pair hi = bf16(g), lo = bf16(g - hi) to
//     split[m * lds + j] and split[m * lds + r_pad + j] (the A operand of
//     dX = [hi | lo] [W_p^T | W_p^T]^T); padding columns j >= r get zeros;
//   * writes hi transposed to gpt[j * ldt + m] for j < r (the A operand of
//     dW_p = G_p^T X).
struct GradPivotEpi {
    const bf16* G;
    int64_t ldg;
    const int32_t* piv;
    int64_t r, r_pad;
    bf16* split;
    int64_t lds;
    bf16* gpt;
    int64_t ldt;
    int64_t M;

    struct Col {
        int64_t n;
        int64_t src;
        bool piv_ok;
    };
    __device__ __forceinline__ Col col(int64_t n) const {
        Col c;
        c.n = n;
        c.piv_ok = n < r;
        c.src = c.piv_ok ? (int64_t)piv[n] : 0;
        return c;
    }
    __device__ __forceinline__ void store(int64_t m, const Col& c, float v) const {
        if (m >= M || c.n >= r_pad) return;
        const uint16_t* g16 = reinterpret_cast<const uint16_t*>(G);
        const float g = c.piv_ok ? v + bf16_bits_to_f32(g16[m * ldg + c.src]) : 0.f;
        const uint16_t hi = f32_to_bf16_bits(g);
        const uint16_t lo = f32_to_bf16_bits(g - bf16_bits_to_f32(hi));
        uint16_t* s16 = reinterpret_cast<uint16_t*>(split);
        s16[m * lds + c.n] = hi;
        s16[m * lds + r_pad + c.n] = lo;
        if (c.piv_ok) reinterpret_cast<uint16_t*>(gpt)[c.n * ldt + m] = hi;
    }
};

}  // namespace pifa
