// Kernels of the PIFA layer backward pass (bf16 layers).
//
// Forward (Algorithm "PIFA Layer", row-major):  Y_p = X W_p^T,
// Y_np = Y_p C^T, Y[:, I] = Y_p, Y[:, I^c] = Y_np.  With G = dL/dY the chain
// rule gives
//   G_p  = G[:, I] + G[:, I^c] C      (M x r)
//   dX   = G_p W_p                    (M x d_in)
//   dW_p = G_p^T X                    (r x d_in)
//   dC   = G[:, I^c]^T Y_p            (n_np x r)
// All four are products for the prefill GEMM (gemm_mfma.hpp).  G_p and dX
// take K-contiguous operands; dW_p and dC reduce over the activation rows
// and read their operands K-major (rows of G_p, X, G[:, I^c], Y[:, I]).  This
// file holds the gathers of G[:, I^c] and Y[:, I] as rows, the transposed
// weight packs and the epilogue of the G_p product.
//
// Precision: G_p multiplies W_p in dX = G_p W_p with the same cancellation as
// Y_p C^T in the forward (C rebuilds W_np from W_p): a bf16 G_p misses the
// bf16 bar there (about 7e-3 measured on QR-pivoted layers), fp16 meets it
// (about 2e-3).  G_p is therefore kept in fp32 and converted row by row to
// fp16 times 2^s_m, s_m chosen from the row's largest |value|, against an
// fp16 copy of W_p^T scaled by 2^c; the product is multiplied back by
// 2^-(s_m + c), which is exact.  dW_p and dC have no such cancellation and
// use bf16 operands; all products accumulate in fp32.
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

// dst = lane order of a (rows_log x cols_log) matrix of type TD whose element
// (i, c) is src(c mod period, i) * scale, where src is a lane-ordered matrix
// (src_kb column blocks per row group) of which rows < src_rows and columns
// < src_cols are valid; everything else is zero.  Used for W_p^T in fp16
// times 2^c and for C^T in bf16 (scale undoing C's fp16 scale, exact for
// bf16-representable C); period = cols_log unless a copy repeats along K.
template <typename TS, typename TD>
__global__ void pack_transposed(const TS* __restrict__ src, int64_t src_kb, int64_t src_rows, int64_t src_cols,
                                int64_t period, float scale, TD* __restrict__ dst, int64_t rows_log,
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
        TD* out = dst + ch * 8;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int64_t k = k0 + e;
            const int64_t s = k % period;
            float v = 0.f;
            if (i < rows_log && k < cols_log && s < src_rows && i < src_cols)
                v = to_f32<TS>(src[lane_order_index(s, i, src_kb)]) * scale;
            if constexpr (__is_same(TD, f16)) out[e] = (f16)v;
            else reinterpret_cast<uint16_t*>(out)[e] = f32_to_bf16_bits(v);
        }
    }
}

// One pass over a 64 x 64 tile of in[m][col(j)] (col(j) = idx[j], or j when
// idx is null), for m < M and j < ncols, written
//   row-major:  out_r[m * ld_r + j]  (j < ld_r; zero for j >= ncols), and/or
//   transposed: out_t[j * ld_t + m]  (m < ld_t; zero for m >= M),
// with 16-byte stores (ld_r, ld_t multiples of 8).  The gathered loads are
// 2 bytes wide; with sorted indices neighbouring lanes read neighbouring
// columns of one row.  Grid: (ceil(max(M, ld_t) / 64), ceil(max(ncols, ld_r) / 64)).
constexpr int kTrTile = 64;

__global__ __launch_bounds__(256) void gather_tile(const bf16* __restrict__ in, int64_t ld_in, int64_t M,
                                                   const int32_t* __restrict__ idx, int64_t ncols,
                                                   bf16* __restrict__ out_r, int64_t ld_r, bf16* __restrict__ out_t,
                                                   int64_t ld_t) {
    __shared__ uint16_t tile[kTrTile][kTrTile + 2];
    const uint16_t* src = reinterpret_cast<const uint16_t*>(in);
    const int64_t m0 = (int64_t)blockIdx.x * kTrTile, j0 = (int64_t)blockIdx.y * kTrTile;
    const int tid = threadIdx.x;
    if (!idx && (ld_in & 7) == 0 && (reinterpret_cast<uintptr_t>(in) & 15) == 0) {
        // plain transpose of 16-byte aligned rows: 8 columns per load
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int ch = tid + 256 * i, mm = ch / 8, j8 = (ch % 8) * 8;
            const int64_t m = m0 + mm, j = j0 + j8;
            uint16_t v[8];
            if (m < M && j + 8 <= ncols) {
                const u32x4 w = *reinterpret_cast<const u32x4*>(src + m * ld_in + j);
                __builtin_memcpy(v, &w, 16);
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e) v[e] = (m < M && j + e < ncols) ? src[m * ld_in + j + e] : (uint16_t)0;
            }
#pragma unroll
            for (int e = 0; e < 8; ++e) tile[mm][j8 + e] = v[e];
        }
    } else {
        // every load is unconditional (clamped row, a valid column): under a
        // lane condition each would be a branch whose join waits for it, one
        // memory round trip per element
        const int jj = tid % kTrTile;
        const int64_t j = j0 + jj;
        const int64_t cj = j < ncols ? (idx ? (int64_t)idx[j] : j) : 0;
        constexpr int kPer = kTrTile * kTrTile / 256;
        uint16_t v[kPer];
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
            const int64_t m = m0 + tid / kTrTile + 4 * i;
            v[i] = src[(m < M ? m : M - 1) * ld_in + cj];
        }
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
            const int mm = tid / kTrTile + 4 * i;
            tile[mm][jj] = (m0 + mm < M && j < ncols) ? v[i] : (uint16_t)0;
        }
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int ch = tid + 256 * i;  // 512 chunks of 8 elements per tile
        const int a = ch / 8, b8 = (ch % 8) * 8;
        if (out_r) {  // row m0 + a, columns j0 + b8 .. +7
            const int64_t m = m0 + a, j = j0 + b8;
            if (m < M && j < ld_r) {
                uint16_t v[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) v[e] = tile[a][b8 + e];
                *reinterpret_cast<u32x4*>(reinterpret_cast<uint16_t*>(out_r) + m * ld_r + j) =
                    __builtin_bit_cast(u32x4, v);
            }
        }
        if (out_t) {  // row j0 + a of the transpose, columns m0 + b8 .. +7
            const int64_t j = j0 + a, m = m0 + b8;
            if (j < ncols && m < ld_t) {
                uint16_t v[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) v[e] = tile[b8 + e][a];
                *reinterpret_cast<u32x4*>(reinterpret_cast<uint16_t*>(out_t) + j * ld_t + m) =
                    __builtin_bit_cast(u32x4, v);
            }
        }
    }
}

// Epilogue of G_p = G[:, I^c] C (+ G[:, I]): acc(m, n) for n < r_pad.
//   * the accumulator starts from G[m, piv[n]] for n < r (init);
//   * writes G_p in fp32 to gp[m * r_pad + n] (padding columns n >= r get
//     zeros), for the row-wise fp16 conversion;
//   * writes bf16(G_p) to gpb[m * r_pad + n] (zeros at n >= r): the K-major
//     A operand of dW_p = G_p^T X.
// In a whole tile the fp32 rows go out element by element (store4_rows) and
// the bf16 rows through the staged 16-byte epilogue (staged()); the K-split
// reduction uses store().
struct GradPivotEpi {
    static constexpr bool kRowsPlusStaged = true;
    const bf16* G;
    int64_t ldg;
    const int32_t* piv;
    int64_t r, r_pad;
    float* gp;
    bf16* gpb;
    int64_t M;

    struct Col {
        int64_t n;
        int64_t src;
        bool piv_ok;
    };
    // The loads below are unconditional, from clamped (valid) addresses, with
    // the result selected afterwards: a load under a lane-dependent condition
    // is compiled as a branch that waits for it, which serialised the 64
    // starting-value loads of a lane (15 of the product's 63 us).
    __device__ __forceinline__ Col col(int64_t n) const {
        Col c;
        c.n = n;
        c.piv_ok = n < r;
        const int32_t p = piv[c.piv_ok ? n : 0];
        c.src = c.piv_ok ? (int64_t)p : 0;
        return c;
    }
    // the product starts from G[m, piv[n]] (the G[:, I] term)
    __device__ __forceinline__ float init(int64_t m, const Col& c) const {
        const uint16_t* g16 = reinterpret_cast<const uint16_t*>(G);
        const float g = bf16_bits_to_f32(g16[(m < M ? m : 0) * ldg + c.src]);
        return (c.piv_ok && m < M) ? g : 0.f;
    }
    __device__ __forceinline__ void store(int64_t m, const Col& c, float v) const {
        if (m >= M || c.n >= r_pad) return;
        const float g = c.piv_ok ? v : 0.f;
        gp[m * r_pad + c.n] = g;
        reinterpret_cast<uint16_t*>(gpb)[m * r_pad + c.n] = f32_to_bf16_bits(g);
    }
    // rows m .. m + 3 (m % 4 == 0) of column c, fp32 rows only
    __device__ __forceinline__ void store4_rows(int64_t m, const Col& c, const float (&v)[4]) const {
        if (c.n >= r_pad || m >= M) return;
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (m + e < M) gp[(m + e) * r_pad + c.n] = c.piv_ok ? v[e] : 0.f;
    }
    // the bf16 rows (the tile's padding columns n >= r hold zero products:
    // C^T's padding rows and their starting values are zero)
    __device__ __forceinline__ StagedEpi<bf16> staged() const {
        return StagedEpi<bf16>{reinterpret_cast<uint16_t*>(gpb), r_pad, r_pad, 1.f, nullptr, M};
    }
};

// Row m of gp (n = r_pad fp32 values, n % 4 == 0) -> fp16 out[m][:] times
// 2^s_m with the row's largest |value| in [2^14, 2^15) (s_m = 0 for a zero
// row), and inv[m] = 2^-s_m.  One workgroup of 256 threads per row.
__global__ __launch_bounds__(256) void rows_to_f16(const float* __restrict__ gp, int64_t n, f16* __restrict__ out,
                                                   float* __restrict__ inv) {
    __shared__ float red[256 / kWave];
    const int64_t m = blockIdx.x;
    const f32x4* row = reinterpret_cast<const f32x4*>(gp + m * n);
    const int64_t nq = n / 4;
    float mx = 0.f;
    for (int64_t q = threadIdx.x; q < nq; q += 256) {
        const f32x4 v = row[q];
        mx = fmaxf(mx, fmaxf(fmaxf(fabsf(v[0]), fabsf(v[1])), fmaxf(fabsf(v[2]), fabsf(v[3]))));
    }
    for (int off = kWave / 2; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
    if ((threadIdx.x & (kWave - 1)) == 0) red[threadIdx.x / kWave] = mx;
    __syncthreads();
    mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    int s = 0;
    if (mx > 0.f && __builtin_isfinite(mx)) {
        int e = 0;
        (void)frexpf(mx, &e);  // mx = f * 2^e, f in [0.5, 1)
        s = 15 - e;            // mx * 2^s in [2^14, 2^15)
        s = s < -100 ? -100 : (s > 100 ? 100 : s);
    }
    const float sc = ldexpf(1.f, s);
    for (int64_t q = threadIdx.x; q < nq; q += 256) {
        const f32x4 v = row[q];
        f16 h[4] = {(f16)(v[0] * sc), (f16)(v[1] * sc), (f16)(v[2] * sc), (f16)(v[3] * sc)};
        *reinterpret_cast<uint64_t*>(out + m * n + 4 * q) = __builtin_bit_cast(uint64_t, h);
    }
    if (threadIdx.x == 0) inv[m] = ldexpf(1.f, -s);
}

// Epilogue writing round(acc(m, n) * row_scale[m] * out_scale) to
// out[m * ldo + n] (bf16) for m < M, n < N.
struct RowScaleEpi {
    bf16* out;
    int64_t ldo, N;
    const float* row_scale;
    float out_scale;
    int64_t M;
    struct Col {
        int64_t n;
        bool ok;
    };
    __device__ __forceinline__ Col col(int64_t n) const { return Col{n, n < N}; }
    __device__ __forceinline__ void store(int64_t m, const Col& c, float v) const {
        if (m < M && c.ok) Store<bf16>::put(out + m * ldo + c.n, v * row_scale[m] * out_scale);
    }
    // rows m .. m + 3 (m % 4 == 0) of column c: one 16-byte load of their
    // scales (row_scale holds M rounded up to 4 values)
    __device__ __forceinline__ void store4(int64_t m, const Col& c, const float (&v)[4]) const {
        if (m >= M || !c.ok) return;
        const f32x4 s = *reinterpret_cast<const f32x4*>(row_scale + m);
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (m + e < M) Store<bf16>::put(out + (m + e) * ldo + c.n, v[e] * s[e] * out_scale);
    }
};

}  // namespace pifa
