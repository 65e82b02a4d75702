// Decode-sized products (M <= 16 activation rows), bound by the weight stream.
//
// acc(m, n) = sum_k A[m, k] * B[n, k] for m < M <= 16, B = weight rows.
// Work is cut into 16-column groups (one MFMA 16x16x32 output tile) and
// K-splits.  Inside a workgroup each wave streams its own K slices of the 16
// weight rows with 16-byte loads (a row contributes 64 contiguous bytes per
// lane group per step), the activation rows ride in the MFMA A operand (rows
// >= M are zero), and the waves are summed in LDS.  Across K-splits, each
// workgroup writes its 16x16 partial to a scratch buffer; the last one to
// arrive (device-scope counter) sums all partials in split order --
// deterministic -- runs the epilogue and re-arms the counter for the next
// launch.
//
// The K order inside an MFMA is free as long as A and B use the same one, so
// a lane loads 32 consecutive K values of its row and feeds them to four
// MFMAs; the four lane groups cover 128 consecutive K per wave step.
#pragma once

#include "common.hpp"
#include "epilogue.hpp"
#include "gemm_mfma.hpp"

namespace pifa {

constexpr int kSkinnyRows = 16;
constexpr int kSkinnyStepK = 128;  // K covered by one wave step

// A operand from a bf16 / fp16 activation matrix (M x K, row stride lda).
template <typename T>
struct ALoad16 {
    const T* a;
    int64_t lda;
    int64_t M;
    static constexpr int kOps = 1;
    __device__ __forceinline__ void load(int m, int64_t k, int64_t kend, u32x4 (&out)[1]) const {
        out[0] = (m < M && k < kend)
                     ? *reinterpret_cast<const u32x4*>(a + (int64_t)m * lda + k)
                     : zero16();
    }
};

// A operand from an fp32 matrix, split into a hi and a lo part of type T
// (value * scale = hi + lo up to T's rounding of the remainder); the two
// MFMAs against the same weights recover close to fp32 precision.
template <typename T>
struct ASplit32 {
    const float* a;
    int64_t lda;
    int64_t M;
    float scale;
    static constexpr int kOps = 2;
    __device__ __forceinline__ void load(int m, int64_t k, int64_t kend, u32x4 (&out)[2]) const {
        if (!(m < M && k < kend)) {
            out[0] = zero16();
            out[1] = zero16();
            return;
        }
        const f32x4* p = reinterpret_cast<const f32x4*>(a + (int64_t)m * lda + k);
        const f32x4 x0 = p[0], x1 = p[1];
        T hi[8], lo[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const float v = (e < 4 ? x0[e] : x1[e - 4]) * scale;
            hi[e] = (T)v;
            lo[e] = (T)(v - (float)hi[e]);
        }
        out[0] = __builtin_bit_cast(u32x4, hi);
        out[1] = __builtin_bit_cast(u32x4, lo);
    }
};

template <typename TB, int WAVES, int UNROLL, typename AL, typename Epi>
__global__ __launch_bounds__(WAVES* kWave) void skinny_mfma(AL al, const TB* __restrict__ B,
                                                           int64_t ldb, int64_t N, int64_t K,
                                                           int64_t k_split,
                                                           float* __restrict__ partials,
                                                           int* __restrict__ counters, Epi epi) {
    constexpr int OPS = AL::kOps;
    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = tid / kWave;
    const int64_t g = blockIdx.x;
    const int64_t n0 = g * kSkinnyRows;
    const int s = blockIdx.y;
    const int S = gridDim.y;
    const int64_t kbeg = (int64_t)s * k_split;
    const int64_t kend = (kbeg + k_split) < K ? (kbeg + k_split) : K;

    const auto brs = make_rsrc(B + n0 * ldb, ((N - n0 - 1) * ldb + K) * (int64_t)sizeof(TB));
    const int row = lane & 15;       // weight row (output column) and activation row
    const int kq = (lane >> 4) * 32; // this lane's 32-wide K slice within a step

    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int64_t kb = kbeg + (int64_t)wave * kSkinnyStepK; kb < kend;
         kb += (int64_t)WAVES * kSkinnyStepK * UNROLL) {
        u32x4 bw[UNROLL][4];
        u32x4 aw[UNROLL][4][OPS];
#pragma unroll
        for (int u = 0; u < UNROLL; ++u)
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int64_t k = kb + (int64_t)u * WAVES * kSkinnyStepK + kq + c * 8;
                bw[u][c] = k < kend ? load16(brs, (uint32_t)((row * ldb + k) * (int64_t)sizeof(TB)))
                                    : zero16();
            }
#pragma unroll
        for (int u = 0; u < UNROLL; ++u)
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int64_t k = kb + (int64_t)u * WAVES * kSkinnyStepK + kq + c * 8;
                al.load(row, k, kend, aw[u][c]);
            }
#pragma unroll
        for (int u = 0; u < UNROLL; ++u)
#pragma unroll
            for (int c = 0; c < 4; ++c)
#pragma unroll
                for (int o = 0; o < OPS; ++o) acc = Mfma<TB>::mma16(aw[u][c][o], bw[u][c], acc);
    }

    // sum the waves of this workgroup (16x16 tile, 4 values per lane)
    __shared__ f32x4 red[WAVES][kWave];
    red[wave][lane] = acc;
    __syncthreads();
    if (wave != 0) return;
    f32x4 tot = red[0][lane];
#pragma unroll
    for (int w = 1; w < WAVES; ++w) tot += red[w][lane];

    if (S > 1) {
        f32x4* part = reinterpret_cast<f32x4*>(partials);
        part[(g * S + s) * kWave + lane] = tot;
        __threadfence();
        int prev = 0;
        if (lane == 0) prev = atomicAdd(&counters[g], 1);
        prev = __shfl(prev, 0);
        if (prev != S - 1) return;
        __threadfence();
        tot = part[(g * S) * kWave + lane];
        for (int t = 1; t < S; ++t) tot += part[(g * S + t) * kWave + lane];
        if (lane == 0) counters[g] = 0;
    }

    // 16x16 accumulator layout: lane holds column (lane % 16), rows 4*(lane/16) + v
    const auto c = epi.col(n0 + (lane & 15));
#pragma unroll
    for (int v = 0; v < 4; ++v) epi.store(4 * (lane >> 4) + v, c, tot[v]);
}

}  // namespace pifa
