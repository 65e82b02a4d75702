// Decode-sized products (M <= 16 * MT activation rows, MT <= 8), bound by the
// weight stream.
//
// acc(m, n) = sum_k A[m, k] * B[n, k] for m < M, B = weight rows.
// One workgroup owns 16 output columns (one MFMA 16x16x32 output tile per
// 16 activation rows) and the whole K range, so no workgroup waits on
// another: its waves take interleaved 128-wide K slices, stream the 16 weight
// rows of each slice once, feed every weight chunk to MT MFMAs (one per
// 16-row activation tile; rows >= M are zero), and are summed in LDS.
//
// The K order inside an MFMA is free as long as A and B use the same one, so
// a lane covers 32 consecutive K values of its row per slice and feeds them
// to four MFMAs; the four lane groups cover the slice's 128 K values.  With
// weights in the lane order of layout.hpp those are four contiguous 1 KB wave
// loads per slice; the row-major variant serves caller-owned weights.
#pragma once

#include "common.hpp"
#include "epilogue.hpp"
#include "gemm_mfma.hpp"
#include "layout.hpp"

namespace pifa {

constexpr int kSkinnyRows = 16;
constexpr int kSkinnyStepK = 128;  // K covered by one wave step

// The activation loads below are exec-masked (rows m >= M and K values past
// K keep zeros): at decode sizes most lanes hold rows past M, and a masked
// lane costs the load nothing.  The kernels issue them in a phase of their
// own, ahead of the MFMAs that use them.

// A operand from a bf16 / fp16 activation matrix (M x K, row stride lda).
template <typename T>
struct ALoad16 {
    const T* a;
    int64_t lda;
    int64_t M;
    static constexpr int kOps = 1;
    __device__ __forceinline__ void load(int m, int64_t k, int64_t K, u32x4 (&out)[1]) const {
        out[0] = zero16();
        if (m < M && k < K) out[0] = *reinterpret_cast<const u32x4*>(a + (int64_t)m * lda + k);
    }
};

// A operand from an fp16 pair hand-off (epilogue kWsF16Pair): hi plane at
// a, lo plane at a + M * lda; two MFMAs against the same weights.
struct ALoadPair16 {
    const f16* a;
    int64_t lda;
    int64_t M;
    static constexpr int kOps = 2;
    __device__ __forceinline__ void load(int m, int64_t k, int64_t K, u32x4 (&out)[2]) const {
        out[0] = zero16();
        out[1] = zero16();
        if (m < M && k < K) {
            out[0] = *reinterpret_cast<const u32x4*>(a + (int64_t)m * lda + k);
            out[1] = *reinterpret_cast<const u32x4*>(a + (M + (int64_t)m) * lda + k);
        }
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
    __device__ __forceinline__ void load(int m, int64_t k, int64_t K, u32x4 (&out)[2]) const {
        f32x4 x0 = {0.f, 0.f, 0.f, 0.f}, x1 = x0;
        if (m < M && k < K) {
            const f32x4* p = reinterpret_cast<const f32x4*>(a + (int64_t)m * lda + k);
            x0 = p[0];
            x1 = p[1];
        }
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

// Sum the per-wave 16x16 tiles in LDS and hand the result to the epilogue;
// wave t finishes activation tile t (t < MT).  Only weight rows n0 + [c_lo,
// c_lo + c_cnt) are stored (a workgroup may own part of a 16-row group).
// ecol: epi.col(n0 + lane % 16), taken before the K loop so its index load
// is not a dependent round trip after the reduction.
template <int WAVES, int MT, typename Epi, typename ECol>
__device__ __forceinline__ void skinny_finish(const f32x4 (&acc)[MT], const Epi& epi, const ECol& ecol, int c_lo = 0,
                                              int c_cnt = 16) {
    static_assert(MT <= WAVES, "one finishing wave per tile");
    __shared__ f32x4 red[WAVES][MT][kWave];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
#pragma unroll
    for (int t = 0; t < MT; ++t) red[wave][t][lane] = acc[t];
    __syncthreads();
    if (wave >= MT) return;
    f32x4 tot = red[0][wave][lane];
#pragma unroll
    for (int w = 1; w < WAVES; ++w) tot += red[w][wave][lane];
    // 16x16 accumulator layout: lane holds column (lane % 16), rows 4*(lane/16) + v
    if ((unsigned)((lane & 15) - c_lo) >= (unsigned)c_cnt) return;
#pragma unroll
    for (int v = 0; v < 4; ++v) epi.store(16 * wave + 4 * (lane >> 4) + v, ecol, tot[v]);
}

// Weights in lane order (layout.hpp): B holds packed_elems(N, K) elements;
// this workgroup owns rows [part * 16 / PARTS, (part + 1) * 16 / PARTS) of
// 16-row group g of B.  PARTS > 1 spreads a narrow product over more
// workgroups (the weight stream of each part is a set of 128-byte runs);
// the lanes of the other parts feed zeros to the MFMA.
template <typename TB, int WAVES, int UNROLL, int MT, int PARTS, typename AL, typename Epi>
__device__ __forceinline__ void skinny_packed_group(const AL& al, const TB* __restrict__ B, int64_t K,
                                                    const Epi& epi, int64_t g, int part = 0) {
    static_assert(PARTS == 1 || PARTS == 2 || PARTS == 4, "parts of a 16-row group");
    constexpr int OPS = AL::kOps;
    constexpr int PROWS = kSkinnyRows / PARTS;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int64_t KB = packed_kblocks(K);
    const u32x4* blk = reinterpret_cast<const u32x4*>(B) + g * KB * kPackChunks;
    const int row = lane & 15;
    const int kq = (lane >> 4) * 32;
    const bool mine = PARTS == 1 || row / PROWS == part;
    const auto ecol = epi.col(g * kSkinnyRows + row);

    f32x4 acc[MT];
#pragma unroll
    for (int t = 0; t < MT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    // Single activation operands (with registers for a whole step) are all
    // loaded right after the step's weights and before its MFMAs, so they
    // cost one round trip per step instead of one per MFMA (the dense and
    // pivot products at M = 16: 7% and 3% faster).  The two-operand forms
    // keep their loads next to the MFMAs, which measured 4% faster for them.
    constexpr bool kHoistA = OPS == 1 && MT * UNROLL * (WAVES > 8 ? 2 : 1) <= 8;
    for (int64_t kb = wave; kb < KB; kb += (int64_t)WAVES * UNROLL) {
        u32x4 bw[UNROLL][4];
        u32x4 aw[kHoistA ? UNROLL : 1][4][kHoistA ? MT : 1][OPS];
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) {
            const int64_t b = kb + (int64_t)u * WAVES;
#pragma unroll
            for (int c = 0; c < 4; ++c) {  // exec-masked: the other parts' lanes load nothing
                bw[u][c] = zero16();
                if (mine && b < KB) bw[u][c] = blk[b * kPackChunks + c * kWave + lane];
            }
        }
        if constexpr (kHoistA) {
#pragma unroll
            for (int u = 0; u < UNROLL; ++u)
#pragma unroll
                for (int c = 0; c < 4; ++c)
#pragma unroll
                    for (int t = 0; t < MT; ++t)
                        al.load(row + 16 * t, (kb + (int64_t)u * WAVES) * kSkinnyStepK + kq + c * 8, K, aw[u][c][t]);
        }
        // keep every load of the step ahead of its MFMAs (the scheduler would
        // otherwise interleave them to save registers, and each load issued
        // after an MFMA that waited is another memory round trip)
        if constexpr (kHoistA) __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < UNROLL; ++u)
#pragma unroll
            for (int c = 0; c < 4; ++c)
#pragma unroll
                for (int t = 0; t < MT; ++t) {
                    if constexpr (!kHoistA)
                        al.load(row + 16 * t, (kb + (int64_t)u * WAVES) * kSkinnyStepK + kq + c * 8, K, aw[0][c][0]);
                    const u32x4(&a)[OPS] = aw[kHoistA ? u : 0][c][kHoistA ? t : 0];
#pragma unroll
                    for (int o = 0; o < OPS; ++o) acc[t] = Mfma<TB>::mma16(a[o], bw[u][c], acc[t]);
                }
    }
    skinny_finish<WAVES, MT>(acc, epi, ecol, part * PROWS, PROWS);
}

// Grid: PARTS * packed_groups(N) workgroups.
template <typename TB, int WAVES, int UNROLL, int MT, int PARTS, typename AL, typename Epi>
__global__ __launch_bounds__(WAVES* kWave) void skinny_packed(AL al, const TB* __restrict__ B,
                                                             int64_t N, int64_t K, Epi epi) {
    (void)N;
    skinny_packed_group<TB, WAVES, UNROLL, MT, PARTS, AL, Epi>(al, B, K, epi, blockIdx.x / PARTS,
                                                               (int)(blockIdx.x % PARTS));
}

// Several weight streams with the same activation rows in one launch
// (grouped layers): problem p owns workgroups [start[p], start[p + 1]).
constexpr int kMaxSkinnyGroup = 8;

template <typename TB, typename AL, typename Epi>
struct SkinnyProblem {
    AL al;
    const TB* B;
    int64_t K;
    Epi epi;
};

template <typename TB, typename AL, typename Epi>
struct SkinnyGroup {
    SkinnyProblem<TB, AL, Epi> p[kMaxSkinnyGroup];
    int64_t start[kMaxSkinnyGroup + 1];
    int n;
};

template <typename TB, int WAVES, int UNROLL, int MT, typename AL, typename Epi>
__global__ __launch_bounds__(WAVES* kWave) void skinny_packed_grouped(SkinnyGroup<TB, AL, Epi> grp) {
    const int64_t b = blockIdx.x;
    int q = 0;
    while (q + 1 < grp.n && b >= grp.start[q + 1]) ++q;
    const SkinnyProblem<TB, AL, Epi>& p = grp.p[q];
    skinny_packed_group<TB, WAVES, UNROLL, MT, 1, AL, Epi>(p.al, p.B, p.K, p.epi, b - grp.start[q]);
}

// Streaming variant for long weight streams (many 16-row groups, or a deep
// K) and at most kStreamRows activation rows.  The problems of a SkinnyGroup
// (one, or the members of a grouped layer, each with its own K) are cut into
// units: a 16-row group, or 1 / PARTS of one as above; problem q owns units
// [start[q], start[q + 1]).  Workgroup b takes units b, b + gridDim.x, ... and
// walks them in passes of its waves over STEP = WAVES * UNROLL blocks of 128 K
// values, issuing the weight loads of the next pass before the MFMAs of the
// current one, so the stream stays in flight across passes, units, problems
// and reductions instead of restarting with every workgroup.
//
// Every problem's activation rows are staged in LDS first, as the MFMA
// operand chunks al.load produces, so the MFMA loop issues no global loads of
// its own: global loads complete in issue order as far as the wait counters
// go, and an activation load issued after the prefetch would make the MFMAs
// wait for the prefetch as well.  With 16 waves, UNROLL 1 and the same PARTS
// the sums run in the order of skinny_packed_group (bit-identical results).
//
// Dynamic LDS: skinny_stream_lds(M, sum of the problems' K rounded up to 128,
// OPS, WAVES) bytes.  Every problem has the same activation rows M.
constexpr int kStreamRows = 4;

__host__ __device__ inline int64_t skinny_stream_lds(int64_t M, int64_t k_blocks_total, int ops, int waves) {
    return M * k_blocks_total * (kSkinnyStepK / 8) * ops * 16 + 2 * (int64_t)waves * kWave * 16;
}

template <typename TB, int WAVES, int UNROLL, int PARTS, typename AL, typename Epi>
__global__ __launch_bounds__(WAVES* kWave) void skinny_stream(SkinnyGroup<TB, AL, Epi> grp) {
    static_assert(PARTS == 1 || PARTS == 2 || PARTS == 4, "parts of a 16-row group");
    constexpr int OPS = AL::kOps;
    constexpr int STEP = WAVES * UNROLL;
    constexpr int PROWS = kSkinnyRows / PARTS;
    constexpr int CPB = kSkinnyStepK / 8;  // 8-value chunks per 128-wide K block
    extern __shared__ u32x4 xs[];          // per problem [M][KB * CPB][OPS] chunks, then [2][WAVES][kWave] f32x4
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int M = (int)grp.p[0].al.M;
    const int64_t units = grp.start[grp.n];
    int64_t kb_total = 0;
    for (int q = 0; q < grp.n; ++q) kb_total += packed_kblocks(grp.p[q].K);
    f32x4* red = reinterpret_cast<f32x4*>(xs + M * kb_total * CPB * OPS);
    const int row = lane & 15;
    const bool live = row < M;

    // iteration state (uniform): unit u of problem q, pass p; u >= units ends
    struct It {
        int64_t u;
        int q;
        int64_t p;
    };
    auto settle = [&](It s) {
        while (s.q + 1 < grp.n && s.u >= grp.start[s.q + 1]) ++s.q;
        return s;
    };
    auto next = [&](It s) {
        if (s.p + 1 < ceil_div(packed_kblocks(grp.p[s.q].K), (int64_t)STEP)) {
            ++s.p;
            return s;
        }
        s.u += gridDim.x;
        s.p = 0;
        return settle(s);
    };
    // weights of one pass (zeros past the last unit: a masked lane's offset is
    // past the buffer range, so the load returns 0 without a memory access)
    auto fetch = [&](const It& s, u32x4(&bw)[UNROLL][4]) {
        const SkinnyProblem<TB, AL, Epi>& P = grp.p[s.q];
        const int64_t KB = packed_kblocks(P.K);
        const int64_t lu = s.u - grp.start[s.q];
        const bool mine = s.u < units && (PARTS == 1 || row / PROWS == (int)(lu % PARTS));
        const auto rs = make_rsrc31(P.B + (lu / PARTS) * KB * (kPackChunks * 8), KB * kPackChunks * 16);
        const int64_t kb0 = s.p * STEP + wave;
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) {
            const int64_t b = kb0 + (int64_t)u * WAVES;
            const uint32_t off = (mine && b < KB) ? (uint32_t)((b * kPackChunks + lane) * 16) : kMaskedOffset;
#pragma unroll
            for (int c = 0; c < 4; ++c) bw[u][c] = load16(rs, off + c * kWave * 16);
        }
    };
    f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
    int par = 0;
    auto step = [&](const It& s, const u32x4(&bw)[UNROLL][4]) {
        const SkinnyProblem<TB, AL, Epi>& P = grp.p[s.q];
        const int64_t KB = packed_kblocks(P.K);
        int64_t kb_before = 0;  // staged K blocks of the problems before q
        for (int q = 0; q < s.q; ++q) kb_before += packed_kblocks(grp.p[q].K);
        // chunk (row, K values 32 * (lane / 16) + 8 * c of block b): lds_lane + (CPB * b + c) * OPS
        const int lds_lane = (int)((M * kb_before * CPB + row * KB * CPB + (lane >> 4) * 4) * OPS);
        const int64_t kb0 = s.p * STEP + wave;
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) {
            const int64_t b = kb0 + (int64_t)u * WAVES;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                u32x4 aw[OPS];
#pragma unroll
                for (int o = 0; o < OPS; ++o)
                    aw[o] = (live && b < KB) ? xs[lds_lane + ((int)b * CPB + c) * OPS + o] : zero16();
#pragma unroll
                for (int o = 0; o < OPS; ++o) acc = Mfma<TB>::mma16(aw[o], bw[u][c], acc);
            }
        }
        if (s.u < units && s.p + 1 == ceil_div(KB, (int64_t)STEP)) {
            // the unit is complete: sum the waves and store (as skinny_finish)
            red[(par * WAVES + wave) * kWave + lane] = acc;
            __syncthreads();
            if (wave == 0) {
                f32x4 tot = red[par * WAVES * kWave + lane];
#pragma unroll
                for (int w = 1; w < WAVES; ++w) tot += red[(par * WAVES + w) * kWave + lane];
                const int64_t lu = s.u - grp.start[s.q];
                const int part = (int)(lu % PARTS);
                if ((unsigned)((lane & 15) - part * PROWS) < (unsigned)PROWS) {
                    const auto c = P.epi.col((lu / PARTS) * kSkinnyRows + (lane & 15));
#pragma unroll
                    for (int v = 0; v < 4; ++v) P.epi.store(4 * (lane >> 4) + v, c, tot[v]);
                }
            }
            acc = f32x4{0.f, 0.f, 0.f, 0.f};
            par ^= 1;
        }
    };

    // the first weights are in flight while the rows are staged
    It cur = settle(It{(int64_t)blockIdx.x, 0, 0});
    It nxt = next(cur);
    u32x4 w0[UNROLL][4], w1[UNROLL][4];
    fetch(cur, w0);
    for (int q = 0, off = 0; q < grp.n; ++q) {
        const SkinnyProblem<TB, AL, Epi>& P = grp.p[q];
        const int64_t KC = packed_kblocks(P.K) * CPB;
        for (int64_t i = threadIdx.x; i < M * KC; i += WAVES * kWave) {
            u32x4 v[OPS];
            P.al.load((int)(i / KC), (i % KC) * 8, P.K, v);
#pragma unroll
            for (int o = 0; o < OPS; ++o) xs[off + i * OPS + o] = v[o];
        }
        off += (int)(M * KC * OPS);
    }
    __syncthreads();  // staged rows visible
    while (cur.u < units) {
        fetch(nxt, w1);
        step(cur, w0);
        cur = nxt;
        nxt = next(nxt);
        if (cur.u >= units) break;
        fetch(nxt, w0);
        step(cur, w1);
        cur = nxt;
        nxt = next(nxt);
    }
}

// Row-major weights (row stride ldb), for caller-owned matrices.
template <typename TB, int WAVES, int UNROLL, int MT, typename AL, typename Epi>
__global__ __launch_bounds__(WAVES* kWave) void skinny_rowmajor(AL al, const TB* __restrict__ B,
                                                               int64_t ldb, int64_t N, int64_t K,
                                                               Epi epi) {
    constexpr int OPS = AL::kOps;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int64_t n0 = (int64_t)blockIdx.x * kSkinnyRows;
    // this workgroup's 16 rows (fewer at the end): rows past N and K values
    // past K lie past the range (masked offsets too stay below 2^31)
    const int64_t rows = (N - n0) < kSkinnyRows ? (N - n0) : kSkinnyRows;
    const auto brs = make_rsrc31(B + n0 * ldb, ((rows - 1) * ldb + K) * (int64_t)sizeof(TB));
    const int row = lane & 15;
    const int kq = (lane >> 4) * 32;
    const auto ecol = epi.col(n0 + row);

    f32x4 acc[MT];
#pragma unroll
    for (int t = 0; t < MT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int64_t kb = (int64_t)wave * kSkinnyStepK; kb < K; kb += (int64_t)WAVES * kSkinnyStepK * UNROLL) {
        u32x4 bw[UNROLL][4];
#pragma unroll
        for (int u = 0; u < UNROLL; ++u)
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int64_t k = kb + (int64_t)u * WAVES * kSkinnyStepK + kq + c * 8;
                bw[u][c] = load16(brs, k < K ? (uint32_t)((row * ldb + k) * (int64_t)sizeof(TB)) : kMaskedOffset);
            }
#pragma unroll
        for (int u = 0; u < UNROLL; ++u)
#pragma unroll
            for (int c = 0; c < 4; ++c)
#pragma unroll
                for (int t = 0; t < MT; ++t) {
                    u32x4 aw[OPS];
                    al.load(row + 16 * t, kb + (int64_t)u * WAVES * kSkinnyStepK + kq + c * 8, K, aw);
#pragma unroll
                    for (int o = 0; o < OPS; ++o) acc[t] = Mfma<TB>::mma16(aw[o], bw[u][c], acc[t]);
                }
    }
    skinny_finish<WAVES, MT>(acc, epi, ecol);
}

}  // namespace pifa
