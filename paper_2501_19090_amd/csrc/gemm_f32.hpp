// fp32 products on the vector ALUs: acc(m, n) = sum_k A[m, k] * B[n, k] with
// fp32 fused multiply-adds in K order.  gfx950 has no reduced-precision fp32
// matrix path, and fp32 layers are the small correctness configuration, so a
// plain LDS-tiled kernel (64 x 64 tile, 4 x 4 outputs per thread) serves all
// fp32 products; loads are bounds-checked so any shape and alignment work.
#pragma once

#include "common.hpp"
#include "epilogue.hpp"

namespace pifa {

template <typename Epi>
__global__ __launch_bounds__(256) void gemm_nt_f32(const float* __restrict__ A, int64_t lda,
                                                   int64_t M, const float* __restrict__ B,
                                                   int64_t ldb, int64_t N, int64_t K, Epi epi) {
    constexpr int BM = 64, BN = 64, BK = 16;
    __shared__ float As[BK][BM + 4];
    __shared__ float Bs[BK][BN + 4];
    const int tid = threadIdx.x;
    const int tx = tid % 16, ty = tid / 16;
    const int64_t m0 = (int64_t)blockIdx.y * BM, n0 = (int64_t)blockIdx.x * BN;

    float acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;

    for (int64_t k0 = 0; k0 < K; k0 += BK) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int idx = tid + e * 256;
            const int row = idx / BK, kk = idx % BK;
            const int64_t m = m0 + row, n = n0 + row, k = k0 + kk;
            As[kk][row] = (m < M && k < K) ? A[m * lda + k] : 0.f;
            Bs[kk][row] = (n < N && k < K) ? B[n * ldb + k] : 0.f;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < BK; ++kk) {
            float a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
#pragma unroll
            for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx * 4 + j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_fmaf(a[i], b[j], acc[i][j]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const auto c = epi.col(n0 + tx * 4 + j);
#pragma unroll
        for (int i = 0; i < 4; ++i) epi.store(m0 + ty * 4 + i, c, acc[i][j]);
    }
}

}  // namespace pifa
