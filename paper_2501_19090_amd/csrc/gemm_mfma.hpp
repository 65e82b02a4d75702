// Prefill GEMM on CDNA4 matrix cores: acc(m, n) = sum_k A[m, k] * B[n, k].
//
// Both operands are K-contiguous row-major (A: M x K activations, B: N x K
// weight rows), which is the layout the MFMA operand registers want: a lane
// supplies 8 consecutive K values of one row.  Used for X W_p^T (bf16),
// Y_p C^T (fp16 operands) and the dense / low-rank baselines.
//
// Block tile BM x BN, K step BK, staged through LDS with double buffering:
// global loads for step k+1 are in flight while step k runs on MFMA.  Rows
// are padded by 16 bytes in LDS so the 16-byte operand reads of 32 lanes
// (32 rows, same K offset) spread over all banks.  Ragged M / N / K are
// handled by buffer-resource range checks (out-of-range loads return 0) and
// a K mask, so any M, N and any K that is a multiple of 8 work.
#pragma once

#include "common.hpp"
#include "epilogue.hpp"

namespace pifa {

template <typename T>
struct Mfma;

template <>
struct Mfma<bf16> {
    __device__ __forceinline__ static f32x16 mma32(u32x4 a, u32x4 b, f32x16 c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                       __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
    }
    __device__ __forceinline__ static f32x4 mma16(u32x4 a, u32x4 b, f32x4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                       __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
    }
};

template <>
struct Mfma<f16> {
    __device__ __forceinline__ static f32x16 mma32(u32x4 a, u32x4 b, f32x16 c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a),
                                                      __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
    }
    __device__ __forceinline__ static f32x4 mma16(u32x4 a, u32x4 b, f32x4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                      __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
    }
};

// Map the linear workgroup id to an output tile.
//  1. The dispatcher sends consecutive workgroup ids round-robin to the 8
//     XCDs; undo that so each XCD gets a contiguous range of tiles (tiles
//     that share A rows then share that XCD's L2).
//  2. Within the range, walk tiles in bands of `kGroupM` tile rows so that
//     concurrently resident tiles reuse both A and B panels.
constexpr int kXcds = 8;
constexpr int kGroupM = 8;

__device__ __forceinline__ void tile_coords(int64_t bid, int64_t tiles_m, int64_t tiles_n,
                                            int64_t& tm, int64_t& tn) {
    const int64_t ntiles = tiles_m * tiles_n;
    int64_t t = bid;
    if (ntiles % kXcds == 0) t = (bid % kXcds) * (ntiles / kXcds) + bid / kXcds;
    const int64_t band = (int64_t)kGroupM * tiles_n;
    const int64_t first_m = (t / band) * kGroupM;
    const int64_t rows = (tiles_m - first_m) < kGroupM ? (tiles_m - first_m) : kGroupM;
    const int64_t in_band = t % band;
    tm = first_m + in_band % rows;
    tn = in_band / rows;
}

template <typename T, int BM, int BN, int BK, int WM, int WN, typename Epi>
__global__ __launch_bounds__(WM* WN* kWave) void gemm_nt_mfma(const T* __restrict__ A, int64_t lda,
                                                             int64_t M, const T* __restrict__ B,
                                                             int64_t ldb, int64_t N, int64_t K,
                                                             Epi epi) {
    constexpr int NT = WM * WN * kWave;
    constexpr int LDK = BK + 8;   // padded LDS row, in elements
    constexpr int CPR = BK / 8;   // 16-byte chunks per tile row
    constexpr int A_CH = BM * CPR / NT;
    constexpr int B_CH = BN * CPR / NT;
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int TM = WTM / 32, TN = WTN / 32;
    static_assert(BM * CPR % NT == 0 && BN * CPR % NT == 0, "tile does not split over threads");
    static_assert(WTM % 32 == 0 && WTN % 32 == 0 && BK % 16 == 0, "bad warp tile");

    __shared__ __attribute__((aligned(16))) T As[2][BM * LDK];
    __shared__ __attribute__((aligned(16))) T Bs[2][BN * LDK];

    const int64_t tiles_m = ceil_div(M, BM), tiles_n = ceil_div(N, BN);
    int64_t tm, tn;
    tile_coords(blockIdx.x, tiles_m, tiles_n, tm, tn);
    const int64_t m0 = tm * BM, n0 = tn * BN;

    const auto ars = make_rsrc(A + m0 * lda, ((M - m0 - 1) * lda + K) * (int64_t)sizeof(T));
    const auto brs = make_rsrc(B + n0 * ldb, ((N - n0 - 1) * ldb + K) * (int64_t)sizeof(T));

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = tid / kWave;
    const int wm = wave / WN, wn = wave % WN;

    u32x4 ra[A_CH], rb[B_CH];
    auto gload = [&](int64_t k0) {
#pragma unroll
        for (int i = 0; i < A_CH; ++i) {
            const int c = tid + i * NT;
            const int row = c / CPR;
            const int64_t k = k0 + (c % CPR) * 8;
            ra[i] = k < K ? load16(ars, (uint32_t)((row * lda + k) * (int64_t)sizeof(T))) : zero16();
        }
#pragma unroll
        for (int i = 0; i < B_CH; ++i) {
            const int c = tid + i * NT;
            const int row = c / CPR;
            const int64_t k = k0 + (c % CPR) * 8;
            rb[i] = k < K ? load16(brs, (uint32_t)((row * ldb + k) * (int64_t)sizeof(T))) : zero16();
        }
    };
    auto sstore = [&](int buf) {
#pragma unroll
        for (int i = 0; i < A_CH; ++i) {
            const int c = tid + i * NT;
            *reinterpret_cast<u32x4*>(&As[buf][(c / CPR) * LDK + (c % CPR) * 8]) = ra[i];
        }
#pragma unroll
        for (int i = 0; i < B_CH; ++i) {
            const int c = tid + i * NT;
            *reinterpret_cast<u32x4*>(&Bs[buf][(c / CPR) * LDK + (c % CPR) * 8]) = rb[i];
        }
    };

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    const int64_t nk = ceil_div(K, BK);
    gload(0);
    sstore(0);
    __syncthreads();

    const int frag_row = lane & 31;
    const int frag_k = (lane >> 5) * 8;
    for (int64_t kt = 0; kt < nk; ++kt) {
        const int cur = (int)(kt & 1);
        if (kt + 1 < nk) gload((kt + 1) * BK);
        const T* as = &As[cur][(wm * WTM + frag_row) * LDK + frag_k];
        const T* bs = &Bs[cur][(wn * WTN + frag_row) * LDK + frag_k];
#pragma unroll
        for (int kk = 0; kk < BK / 16; ++kk) {
            u32x4 af[TM], bfr[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i)
                af[i] = *reinterpret_cast<const u32x4*>(as + i * 32 * LDK + kk * 16);
#pragma unroll
            for (int j = 0; j < TN; ++j)
                bfr[j] = *reinterpret_cast<const u32x4*>(bs + j * 32 * LDK + kk * 16);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) acc[i][j] = Mfma<T>::mma32(af[i], bfr[j], acc[i][j]);
        }
        if (kt + 1 < nk) sstore(cur ^ 1);
        __syncthreads();
    }

    // 32x32 accumulator layout: lane holds column (lane % 32) and rows
    // 8*(v/4) + 4*(lane/32) + (v%4) for v = 0..15.
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const auto c = epi.col(n0 + wn * WTN + j * 32 + (lane & 31));
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            const int64_t mb = m0 + wm * WTM + i * 32 + 4 * (lane >> 5);
#pragma unroll
            for (int v = 0; v < 16; ++v) epi.store(mb + 8 * (v >> 2) + (v & 3), c, acc[i][j][v]);
        }
    }
}

}  // namespace pifa
