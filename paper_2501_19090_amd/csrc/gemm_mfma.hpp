// Prefill GEMM on CDNA4 matrix cores: acc(m, n) = sum_k A[m, k] * B[n, k].
//
// Both operands are K-contiguous row-major (A: M x K activations, B: N x K
// weight rows), which is the layout the MFMA operand registers want: a lane
// supplies 8 consecutive K values of one row.  Used for X W_p^T (bf16),
// Y_p C^T (fp16 operands) and the dense / low-rank baselines.
//
// Block tile BM x BN, K step BK, staged through LDS with double buffering,
// 8 waves (2 per SIMD) each owning a 64 x 64 sub-tile of 32x32x16 MFMAs.
// Global loads run PGR tiles ahead through registers; the LDS write of the
// next tile is issued right after the first MFMA group of the current one,
// and operand fragments for MFMA step kk+1 are read from LDS while step kk
// runs, so the matrix cores rarely wait on memory.  Rows are padded by 16
// bytes in LDS so the 16-byte operand reads of 32 lanes (32 rows, same K
// offset) spread over all banks (no bank conflicts were counted).  Ragged M / N / K are
// handled by buffer-resource range checks (out-of-range loads return 0; a
// masked lane is given an offset past the range), so any M, N and any K that
// is a multiple of 8 work.  B is either
// row-major (row stride ldb) or in the lane order of layout.hpp (BPACK).
//
// K-major operands (KM bit 0: A, bit 1: B) are stored K x M (K x N) with
// row stride lda >= M rounded up to 8 (ldb likewise, 16-byte aligned rows):
// the transposed products of the backward pass, whose
// reduction runs over the activation rows.  Their tiles go to LDS as they
// are loaded (BK rows of the tile's M or N extent) and the MFMA fragments
// are read back with the transposing LDS read of gfx950 (ds_read_b64_tr_b16):
// within each group of 16 lanes, lane R reads 4 elements of K row R / 4 at
// column 4 (R % 4), and lane L receives the 4 elements of column L from those
// 4 rows, so two such reads give a lane the 8 consecutive K values of its row.
#pragma once

#include <type_traits>

#include "common.hpp"
#include "epilogue.hpp"
#include "layout.hpp"

namespace pifa {

// An epilogue with init(m, col) gives the starting value of acc(m, n) (the
// product is added to it): the GEMM loads it before its K loop, where the
// load latency hides behind the first tiles' loads, and split_reduce starts
// its sum with it.
template <typename E, typename = void>
struct InitEpi {
    static constexpr bool value = false;
};
template <typename E>
struct InitEpi<E, std::void_t<decltype(&E::init)>> {
    static constexpr bool value = true;
};

// An epilogue with store4(m, col, v[4]) takes the four consecutive rows
// m .. m + 3 of one column that a lane of the 32x32 layout holds at once.
template <typename E, typename = void>
struct Store4Epi {
    static constexpr bool value = false;
};
template <typename E>
struct Store4Epi<E, std::void_t<decltype(&E::store4)>> {
    static constexpr bool value = true;
};

// An epilogue with skip_tile(m0, n0, BM, BN) may drop whole output tiles
// (the workgroup exits before any work).
template <typename E, typename = void>
struct SkipEpi {
    static constexpr bool value = false;
};
template <typename E>
struct SkipEpi<E, std::void_t<decltype(&E::skip_tile)>> {
    static constexpr bool value = true;
};

// An epilogue with kStaged writes a contiguous output through LDS with
// 16-byte stores (StagedEpi).
template <typename E, typename = void>
struct StagedEpiT {
    static constexpr bool value = false;
};
template <typename E>
struct StagedEpiT<E, std::void_t<decltype(E::kStaged)>> {
    static constexpr bool value = true;
};

// An epilogue with kRowsPlusStaged stores one output element-wise
// (store4_rows) and a second, contiguous one through LDS (staged()).
template <typename E, typename = void>
struct RowsPlusStagedEpiT {
    static constexpr bool value = false;
};
template <typename E>
struct RowsPlusStagedEpiT<E, std::void_t<decltype(E::kRowsPlusStaged)>> {
    static constexpr bool value = true;
};

// An epilogue with kDual has a per-element part (y) and a staged part (ws).
template <typename E, typename = void>
struct DualEpiT {
    static constexpr bool value = false;
};
template <typename E>
struct DualEpiT<E, std::void_t<decltype(E::kDual)>> {
    static constexpr bool value = true;
};

// LDS bytes of a BM x BN tile of T with K step BK: the double-buffered
// operand tiles (the staged epilogues reuse them after the K loop).
// A K-major tile is stored as BK rows of BM (BN) elements with a pitch of
// BM + 32 (BN + 32): the 16 lanes of a transposing read cover 4 rows x 32
// bytes, and that pitch puts the 4 rows on disjoint bank groups.
template <int BM, int BK, bool KMAJ>
constexpr int tile_elems() {
    return KMAJ ? BK * (BM + 32) : BM * (BK + 8);
}
template <typename T, int BM, int BN, int BK, int KM = 0>
constexpr int gemm_lds_bytes() {
    return 2 * (tile_elems<BM, BK, (KM & 1) != 0>() + tile_elems<BN, BK, (KM & 2) != 0>()) * (int)sizeof(T);
}

typedef short v4i16 __attribute__((ext_vector_type(4)));

// 8 consecutive K values (k0 .. k0 + 7) of row r0 + lane % 32 of a K-major LDS
// tile with pitch P (elements), for the 32x32x16 operand layout: lane l
// holds row l % 32, K values 8 (l / 32) .. + 7 of the 16-deep step at k0.
template <typename T, int P>
__device__ __forceinline__ u32x4 frag_kmajor(const T* tile, int k0, int r0, int lane) {
    const int g = lane >> 4, R = lane & 15;
    const T* p = tile + (k0 + 8 * (g >> 1) + (R >> 2)) * P + r0 + 16 * (g & 1) + 4 * (R & 3);
    typedef __attribute__((address_space(3))) v4i16 lds_v4;
    const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4*)p);
    const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4*)(p + 4 * P));
    const uint2 a = __builtin_bit_cast(uint2, lo), b = __builtin_bit_cast(uint2, hi);
    return u32x4{a.x, a.y, b.x, b.y};
}

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
//     that share A rows then share that XCD's L2).  The even XCDs take the
//     first four ranges and the odd XCDs the last four, so the two XCDs
//     whose ranges form one band (and read the same A panels) are both even
//     or both odd: paired as 2i and 2i + 1, the odd XCD of each pair ran
//     about 9% more cycles per tile of a 2048-deep product, and the pairing
//     by parity measured 1.2 us faster on the 4096 x 2048 non-pivot product
//     (49.5 -> 48.3 us) and equal elsewhere.  Only the timing changes: every
//     tile computes the same sums wherever it runs.
//  2. Within the range, walk tiles in bands of `group` tile rows, column by
//     column, so that one XCD's range is a block of about group x (range /
//     group) tiles.  Its L2 then fills group A panels of BM rows and
//     range / group B panels of BN rows; `band_rows` picks the power of two
//     that makes the two byte counts about equal, which minimises their sum
//     (256 x 128 tiles of a 4096 x 2048 product: 4 x 8 tiles, 16 MB of
//     panels per XCD against 20 MB for 8 x 4).
constexpr int kXcds = 8;

// Step 1 on its own: consecutive ids of one XCD become a contiguous range.
__device__ __forceinline__ int64_t xcd_remap(int64_t bid, int64_t ntiles) {
    const int64_t x = bid % kXcds;
    const int64_t range = (x & 1) ? kXcds / 2 + (x >> 1) : (x >> 1);
    return ntiles % kXcds == 0 ? range * (ntiles / kXcds) + bid / kXcds : bid;
}

template <int BM, int BN>
__device__ __forceinline__ int64_t band_rows(int64_t tiles_m, int64_t ntiles) {
    const int64_t per_xcd = ntiles % kXcds == 0 ? ntiles / kXcds : ntiles;
    int64_t g = 1;
    while (2 * g <= tiles_m && 4 * g * g * BM <= per_xcd * BN) g *= 2;
    return g;
}

// Step 2 on its own: tile t of a tiles_m x tiles_n grid, in bands of `group` tile rows.
__device__ __forceinline__ void band_coords(int64_t t, int64_t tiles_m, int64_t tiles_n, int64_t group,
                                            int64_t& tm, int64_t& tn) {
    const int64_t band = group * tiles_n;
    const int64_t first_m = (t / band) * group;
    const int64_t rows = (tiles_m - first_m) < group ? (tiles_m - first_m) : group;
    const int64_t in_band = t % band;
    tm = first_m + in_band % rows;
    tn = in_band / rows;
}

template <int BM, int BN>
__device__ __forceinline__ void tile_coords(int64_t bid, int64_t tiles_m, int64_t tiles_n, int64_t& tm,
                                            int64_t& tn) {
    const int64_t ntiles = tiles_m * tiles_n;
    band_coords(xcd_remap(bid, ntiles), tiles_m, tiles_n, band_rows<BM, BN>(tiles_m, ntiles), tm, tn);
}

// Offset past every buffer range: the load returns 0 without a branch.
constexpr uint32_t kMaskedOffset = 0x80000000u;

// Buffer resource whose range stays below kMaskedOffset.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc31(const void* base, int64_t bytes) {
    const uint32_t n = bytes <= 0 ? 0u : (bytes >= 0x7FFFFFFFll ? 0x7FFFFFFFu : (uint32_t)bytes);
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)n, 0x00020000);
}

// Store tile (m0, n0) of a contiguous output (StagedEpi): each chunk of R
// rows is written to LDS as TOut rows of BN values (pitch BN + 8, which
// spreads the column-wise writes over the banks), then read back and stored 8
// values per 16-byte store; columns at or past N are not stored.
template <int BM, int BN, int WM, int WN, int TM, int TN, typename TOut>
__device__ __forceinline__ void staged_store(const f32x16 (&acc)[TM][TN], int64_t m0, int64_t n0,
                                             const StagedEpi<TOut>& e, char* smem, int lds_bytes) {
    constexpr int NT = WM * WN * kWave;
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int P = BN + 8;       // LDS row pitch in elements
    constexpr int G = BN / 8;       // 16-byte groups per row
    constexpr int R0 = (BM * P * 2 <= 163840) ? BM : 163840 / (2 * P);
    const int R = (lds_bytes / (2 * P)) < R0 ? (lds_bytes / (2 * P)) : R0;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int wm = wave / WN, wn = wave % WN;
    uint16_t* tile = reinterpret_cast<uint16_t*>(smem);
    int over = 0;
    for (int r0 = 0; r0 < BM && m0 + r0 < e.M; r0 += R) {
        __syncthreads();
#pragma unroll
        for (int i = 0; i < TM; ++i) {
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int nl = wn * WTN + j * 32 + (lane & 31);
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int ml = wm * WTM + i * 32 + 4 * (lane >> 5) + 8 * (v >> 2) + (v & 3) - r0;
                    if ((unsigned)ml < (unsigned)R && m0 + r0 + ml < e.M && n0 + nl < e.N)
                        tile[ml * P + nl] = e.bits(acc[i][j][v], over);
                }
            }
        }
        __syncthreads();
        const int RC = (BM - r0) < R ? (BM - r0) : R;  // rows of this chunk inside the tile
        for (int q = threadIdx.x; q < RC * G; q += NT) {
            const int rr = q / G, g = q % G;
            const int64_t m = m0 + r0 + rr, n = n0 + 8 * g;
            if (m >= e.M || n >= e.N) continue;
            const u32x4 v = *reinterpret_cast<const u32x4*>(tile + rr * P + 8 * g);
            uint16_t* dst = e.out + m * e.ldo + n;
            if (n + 8 <= e.N) {
                *reinterpret_cast<u32x4*>(dst) = v;
            } else {
                const uint16_t* hv = reinterpret_cast<const uint16_t*>(&v);
                for (int x = 0; x < 8 && n + x < e.N; ++x) dst[x] = hv[x];
            }
        }
    }
    if (over && e.overflow) atomicAdd(e.overflow, over);
}

// One output tile (tm, tn) over the K range [kbeg, kend); both operands are
// masked outside that range.
template <typename T, int BM, int BN, int BK, int WM, int WN, bool BPACK, int PGR, typename Epi, int KM = 0>
__device__ __forceinline__ void gemm_nt_tile(const T* __restrict__ A, int64_t lda, int64_t M,
                                             const T* __restrict__ B, int64_t ldb, int64_t N, int64_t K,
                                             int64_t kbeg, int64_t kend, int64_t tm, int64_t tn,
                                             const Epi& epi) {
    constexpr int NT = WM * WN * kWave;
    constexpr int LDK = BK + 8;  // padded LDS row, in elements
    constexpr int CPR = BK / 8;  // 16-byte chunks per tile row
    constexpr int A_CH = BM * CPR / NT;
    constexpr int B_CH = BN * CPR / NT;
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int TM = WTM / 32, TN = WTN / 32;
    constexpr int KK = BK / 16;
    constexpr int CPG = 2 * BK;  // packed: chunks of one 16-row group inside a tile
    constexpr int LPC = BK / 2;  // packed: lanes per MFMA slice inside a tile
    static_assert(BM * CPR % NT == 0 && BN * CPR % NT == 0, "tile does not split over threads");
    static_assert(WTM % 32 == 0 && WTN % 32 == 0 && KK >= 2, "bad warp tile");
    static_assert(!BPACK || ((BK == 64 || BK == 128) && BN % kPackRows == 0), "bad packed tile");
    static_assert(PGR >= 1 && PGR <= 4, "prefetch depth");
    constexpr bool AKM = (KM & 1) != 0, BKM = (KM & 2) != 0;
    static_assert(!(BPACK && BKM), "a packed B is K-contiguous");
    constexpr int PMA = BM + 32, PMB = BN + 32;  // K-major tile pitches
    constexpr int AEL = tile_elems<BM, BK, AKM>(), BEL = tile_elems<BN, BK, BKM>();

    constexpr int LDS_BYTES = gemm_lds_bytes<T, BM, BN, BK, KM>();
    __shared__ __attribute__((aligned(16))) char smem[LDS_BYTES];
    T(*As)[AEL] = reinterpret_cast<T(*)[AEL]>(smem);
    T(*Bs)[BEL] = reinterpret_cast<T(*)[BEL]>(smem + 2 * AEL * sizeof(T));

    const int64_t m0 = tm * BM, n0 = tn * BN;
    if constexpr (SkipEpi<Epi>::value) {
        if (epi.skip_tile(m0, n0, BM, BN)) return;
    }

    // K-major: element (k, m) at k * lda + m, with lda >= M rounded up to 8
    // (the last row's final chunk lies inside the row pitch, so it is read
    // whole: a range ending mid-chunk would zero the chunk's valid elements);
    // elements at m >= M only feed output rows >= M, which are not stored
    const auto ars = AKM ? make_rsrc31(A + m0, ((K - 1) * lda + round_up(M - m0, (int64_t)8)) * (int64_t)sizeof(T))
                         : make_rsrc31(A + m0 * lda, ((M - m0 - 1) * lda + K) * (int64_t)sizeof(T));
    const int64_t KB = packed_kblocks(K);
    const auto brs = BPACK ? make_rsrc31(B + (n0 / kPackRows) * KB * (kPackChunks * 8),
                                         (packed_groups(N) - n0 / kPackRows) * KB * kPackChunks * 16)
                     : BKM ? make_rsrc31(B + n0, ((K - 1) * ldb + round_up(N - n0, (int64_t)8)) * (int64_t)sizeof(T))
                           : make_rsrc31(B + n0 * ldb, ((N - n0 - 1) * ldb + K) * (int64_t)sizeof(T));

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = tid / kWave;
    const int wm = wave / WN, wn = wave % WN;

    struct Stage {
        u32x4 a[A_CH], b[B_CH];
        int blds[B_CH];  // LDS element offset of each B chunk
    };
    Stage S[PGR];
    auto gload = [&](int64_t k0, Stage& R) {
#pragma unroll
        for (int i = 0; i < A_CH; ++i) {
            const int c = tid + i * NT;
            if constexpr (AKM) {  // chunk: 8 consecutive rows m of K row k
                // rows k >= kend get bit 31 (past every range) without a
                // select: the per-chunk row makes the mask lane-dependent
                const int64_t k = k0 + c / (BM / 8);
                const int mc = c % (BM / 8);
                const uint32_t off = (uint32_t)((k * lda + 8 * mc) * (int64_t)sizeof(T));
                R.a[i] = load16(ars, off | ((uint32_t)(k >= kend) << 31));
            } else {
                const int row = c / CPR;
                const int64_t k = k0 + (c % CPR) * 8;
                R.a[i] = load16(ars, k < kend ? (uint32_t)((row * lda + k) * (int64_t)sizeof(T)) : kMaskedOffset);
            }
        }
        if constexpr (BKM) {
#pragma unroll
            for (int i = 0; i < B_CH; ++i) {
                const int c = tid + i * NT;
                const int kr = c / (BN / 8), nc = c % (BN / 8);
                const int64_t k = k0 + kr;
                const uint32_t off = (uint32_t)((k * ldb + 8 * nc) * (int64_t)sizeof(T));
                R.b[i] = load16(brs, off | ((uint32_t)(k >= kend) << 31));
                R.blds[i] = kr * PMB + 8 * nc;
            }
        } else if constexpr (BPACK) {
            const int64_t blk = k0 / kPackCols;
            const int hsel = (int)((k0 % kPackCols) / BK);
#pragma unroll
            for (int i = 0; i < B_CH; ++i) {
                const int cid = tid + i * NT, gl = cid / CPG, rem = cid % CPG;
                const int c = rem / LPC, l = hsel * LPC + rem % LPC;
                const int kc = 4 * ((l >> 4) - hsel * (LPC / 16)) + c;  // chunk index in the tile
                R.b[i] = load16(brs, k0 + kc * 8 < kend ? (uint32_t)((((gl * KB + blk) * 4 + c) * 64 + l) * 16)
                                                        : kMaskedOffset);
                R.blds[i] = (gl * kPackRows + (l & 15)) * LDK + kc * 8;
            }
        } else {
#pragma unroll
            for (int i = 0; i < B_CH; ++i) {
                const int c = tid + i * NT, row = c / CPR;
                const int64_t k = k0 + (c % CPR) * 8;
                R.b[i] = load16(brs, k < kend ? (uint32_t)((row * ldb + k) * (int64_t)sizeof(T)) : kMaskedOffset);
                R.blds[i] = row * LDK + (c % CPR) * 8;
            }
        }
    };
    auto sstore = [&](int buf, const Stage& R) {
#pragma unroll
        for (int i = 0; i < A_CH; ++i) {
            const int c = tid + i * NT;
            if constexpr (AKM)
                *reinterpret_cast<u32x4*>(&As[buf][(c / (BM / 8)) * PMA + (c % (BM / 8)) * 8]) = R.a[i];
            else
                *reinterpret_cast<u32x4*>(&As[buf][(c / CPR) * LDK + (c % CPR) * 8]) = R.a[i];
        }
#pragma unroll
        for (int i = 0; i < B_CH; ++i) *reinterpret_cast<u32x4*>(&Bs[buf][R.blds[i]]) = R.b[i];
    };

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f32x16{};
    // The epilogue's column descriptors (output index loads).  The epilogues
    // that start from loaded values or write two outputs take them before the
    // K loop on tiles with at most 4 accumulator blocks per wave, so the
    // loads are in flight with the first tiles (the pivot product: 82.4 ->
    // 80.4 us); the others take them after the loop (early, the non-pivot
    // product took 1 us longer), as do the wider tiles, which have no
    // registers to spare across the loop.
    const auto& ecol_src = [&]() -> decltype(auto) {
        if constexpr (DualEpiT<Epi>::value) return (epi.y);
        else return (epi);
    }();
    using ECol = decltype(ecol_src.col(0));
    constexpr bool kEarlyCols = InitEpi<Epi>::value || (DualEpiT<Epi>::value && TM * TN <= 4);
    ECol ecols[TN];
    auto fill_ecols = [&]() {
#pragma unroll
        for (int j = 0; j < TN; ++j) ecols[j] = ecol_src.col(n0 + wn * WTN + j * 32 + (lane & 31));
    };
    if constexpr (kEarlyCols) fill_ecols();
    if constexpr (InitEpi<Epi>::value) {
        // 32x32 accumulator layout (see the epilogue below)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const auto& c = ecols[j];
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const int64_t mb = m0 + wm * WTM + i * 32 + 4 * (lane >> 5);
#pragma unroll
                for (int v = 0; v < 16; ++v) acc[i][j][v] = epi.init(mb + 8 * (v >> 2) + (v & 3), c);
            }
        }
    }

    // 32x32x16 operands: lane supplies row (lane % 32), K values 8*(lane/32) .. +7
    const int frag_row = lane & 31, frag_k = (lane >> 5) * 8;
    u32x4 fa[2][TM], fb[2][TN];
    auto lds_frag = [&](int buf, int kk, int slot) {
        if constexpr (AKM) {
#pragma unroll
            for (int i = 0; i < TM; ++i) fa[slot][i] = frag_kmajor<T, PMA>(As[buf], kk * 16, wm * WTM + i * 32, lane);
        } else {
            const T* as = &As[buf][(wm * WTM + frag_row) * LDK + frag_k + kk * 16];
#pragma unroll
            for (int i = 0; i < TM; ++i) fa[slot][i] = *reinterpret_cast<const u32x4*>(as + i * 32 * LDK);
        }
        if constexpr (BKM) {
#pragma unroll
            for (int j = 0; j < TN; ++j) fb[slot][j] = frag_kmajor<T, PMB>(Bs[buf], kk * 16, wn * WTN + j * 32, lane);
        } else {
            const T* bs = &Bs[buf][(wn * WTN + frag_row) * LDK + frag_k + kk * 16];
#pragma unroll
            for (int j = 0; j < TN; ++j) fb[slot][j] = *reinterpret_cast<const u32x4*>(bs + j * 32 * LDK);
        }
    };

    const int64_t nk = ceil_div(kend - kbeg, BK);
    // Tile t is staged in S[t % PGR].  Before iteration kt the LDS buffer
    // (kt & 1) holds tile kt and tiles kt+1 .. kt+PGR are in flight.
    // The steady state has no data-dependent branches: loads past kend are
    // masked (they return zeros), and the LDS store and fragment reads of
    // the last iterations touch a buffer nobody reads again.  A branch here
    // would make the compiler wait for every outstanding load at the join,
    // which serialises the prefetch.
#pragma unroll
    for (int p = 0; p < PGR; ++p) gload(kbeg + (int64_t)p * BK, S[p]);
    sstore(0, S[0]);
    gload(kbeg + (int64_t)PGR * BK, S[0]);
    __syncthreads();
    lds_frag(0, 0, 0);
    // With EARLY, the one barrier per tile sits before the last MFMA step
    // (after every wave has read its last fragments of this tile and written
    // the next one), so the next tile's first fragments are read while the
    // last MFMA step runs instead of after the barrier.
    constexpr bool EARLY = PGR >= 2;
    auto body = [&](int64_t kt, Stage& nxt) {  // nxt = S[(kt + 1) % PGR]
        const int cur = (int)(kt & 1);
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
            const int slot = kk & 1;
            if (kk + 1 < KK) lds_frag(cur, kk + 1, slot ^ 1);
            else if (EARLY) lds_frag(cur ^ 1, 0, slot ^ 1);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) acc[i][j] = Mfma<T>::mma32(fa[slot][i], fb[slot][j], acc[i][j]);
            // the other LDS buffer was last read before the previous barrier
            if (kk == 0) sstore(cur ^ 1, nxt);
            if (kk == 1) gload(kbeg + (kt + 1 + PGR) * BK, nxt);
            if (EARLY && kk == KK - 2) __syncthreads();
        }
        if constexpr (EARLY) {
            __builtin_amdgcn_iglp_opt(0);
        } else {
            __syncthreads();
            lds_frag(cur ^ 1, 0, 0);
        }
    };
    // PGR iterations per trip so that every stage index is a constant
    int64_t kt = 0;
    for (; kt + PGR <= nk; kt += PGR) {
#pragma unroll
        for (int u = 0; u < PGR; ++u) body(kt + u, S[(u + 1) % PGR]);
    }
#pragma unroll
    for (int u = 0; u < PGR - 1; ++u)
        if (kt + u < nk) body(kt + u, S[(u + 1) % PGR]);

    // 256 x 128 tiles of the plain bf16 scatter (the non-pivot product) write
    // their outputs row by row through LDS: each store instruction of a wave
    // covers 64 consecutive tile columns of one output row, whose scattered
    // destinations span about two lines of Y, instead of 32 columns of two
    // rows.  Attention layer at M = 4096, three alternating passes: 47.6-47.9
    // -> 46.7-47.1 us per launch, bit-identical outputs.  The other tiles keep
    // the element-wise stores (staged this way the 256 x 192 and 256 x 256
    // tiles lost 10-15%, and the 128 x 128 tiles of M = 2048 about 0.8 us).
    constexpr bool kRowScatter = std::is_same<Epi, ScatterEpi<bf16, kWsNone>>::value && BM == 256 && BN == 128 &&
                                 WM * WN == 8;
    if constexpr (!kEarlyCols && !kRowScatter) fill_ecols();
    if constexpr (kRowScatter) {
        constexpr int P = BN + 8;  // LDS row pitch (elements)
        static_assert(BM * P * 2 <= LDS_BYTES, "row staging does not fit the tile's LDS");
        uint16_t* tile = reinterpret_cast<uint16_t*>(smem);
        const auto c_lo = epi.col(n0 + lane), c_hi = epi.col(n0 + kWave + lane);
        __syncthreads();  // every wave is done with the operand buffers
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int nl = wn * WTN + j * 32 + (lane & 31);
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int ml = wm * WTM + i * 32 + 4 * (lane >> 5) + 8 * (v >> 2) + (v & 3);
                    tile[ml * P + nl] = f32_to_bf16_bits(acc[i][j][v] * epi.out_scale);
                }
            }
        __syncthreads();
        uint16_t* out = reinterpret_cast<uint16_t*>(epi.out);
        for (int r = wave; r < BM; r += WM * WN) {
            const int64_t m = m0 + r;
            if (m >= epi.M) break;
            const uint16_t lo = tile[r * P + lane], hi = tile[r * P + kWave + lane];
            if (c_lo.out_ok) out[m * epi.ldo + c_lo.dst] = lo;
            if (c_hi.out_ok) out[m * epi.ldo + c_hi.dst] = hi;
        }
        return;
    } else if constexpr (StagedEpiT<Epi>::value) {
        staged_store<BM, BN, WM, WN, TM, TN>(acc, m0, n0, epi, smem, LDS_BYTES);
        return;
    } else if constexpr (RowsPlusStagedEpiT<Epi>::value) {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const auto& c = ecols[j];
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const int64_t mb = m0 + wm * WTM + i * 32 + 4 * (lane >> 5);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const float v4[4] = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                                         acc[i][j][4 * q + 3]};
                    epi.store4_rows(mb + 8 * q, c, v4);
                }
            }
        }
        staged_store<BM, BN, WM, WN, TM, TN>(acc, m0, n0, epi.staged(), smem, LDS_BYTES);
        return;
    } else if constexpr (DualEpiT<Epi>::value) {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const auto& c = ecols[j];
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const int64_t mb = m0 + wm * WTM + i * 32 + 4 * (lane >> 5);
#pragma unroll
                for (int v = 0; v < 16; ++v) epi.y.store(mb + 8 * (v >> 2) + (v & 3), c, acc[i][j][v]);
            }
        }
        staged_store<BM, BN, WM, WN, TM, TN>(acc, m0, n0, epi.ws, smem, LDS_BYTES);
        return;
    } else if constexpr (Store4Epi<Epi>::value && BM == 256) {
        // rows outer on the 256-row tiles too (the backward's dX = G_p W_p on
        // 256 x 256 tiles, three alternating passes: 77.9-78.7 -> 76.3-76.7 us)
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            const int64_t mb = m0 + wm * WTM + i * 32 + 4 * (lane >> 5);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    const float v4[4] = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                                         acc[i][j][4 * q + 3]};
                    epi.store4(mb + 8 * q, ecols[j], v4);
                }
            }
        }
    } else if constexpr (std::is_same<Epi, ScatterEpi<bf16, kWsNone>>::value && BM == 256) {
        // the wider tiles of the non-pivot product: rows outer, so that the
        // stores of one group of rows go out across all column blocks in turn
        // (M = 4096, three alternating passes, us per launch: the MLP up
        // projection's 256 x 192 tiles 167.5-169.9 -> 164.1-165.3, the
        // r = 10% layer's 256 x 256 tiles 31.1-31.4 -> 28.9-29.6)
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            const int64_t mb = m0 + wm * WTM + i * 32 + 4 * (lane >> 5);
#pragma unroll
            for (int v = 0; v < 16; ++v) {
#pragma unroll
                for (int j = 0; j < TN; ++j) epi.store(mb + 8 * (v >> 2) + (v & 3), ecols[j], acc[i][j][v]);
            }
        }
    } else {
    // 32x32 accumulator layout: lane holds column (lane % 32) and rows
    // 8*(v/4) + 4*(lane/32) + (v%4) for v = 0..15.
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const auto& c = ecols[j];
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            const int64_t mb = m0 + wm * WTM + i * 32 + 4 * (lane >> 5);
            if constexpr (Store4Epi<Epi>::value) {
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const float v4[4] = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                                         acc[i][j][4 * q + 3]};
                    epi.store4(mb + 8 * q, c, v4);
                }
            } else {
#pragma unroll
                for (int v = 0; v < 16; ++v) epi.store(mb + 8 * (v >> 2) + (v & 3), c, acc[i][j][v]);
            }
        }
    }
    }
}

struct SplitEpi;

// K splitting (partial products, Epi = SplitEpi): workgroup (tile,
// blockIdx.y = s) reduces K range [s * k_split, min(K, (s + 1) * k_split));
// k_split is a multiple of BK.  Every other epilogue covers all of K.
template <typename T, int BM, int BN, int BK, int WM, int WN, bool BPACK, int PGR, typename Epi, int KM = 0>
__global__ __launch_bounds__(WM* WN* kWave) void gemm_nt_mfma(const T* __restrict__ A, int64_t lda,
                                                             int64_t M, const T* __restrict__ B,
                                                             int64_t ldb, int64_t N, int64_t K,
                                                             int64_t k_split, Epi epi) {
    int64_t tm, tn;
    tile_coords<BM, BN>(blockIdx.x, ceil_div(M, BM), ceil_div(N, BN), tm, tn);
    if constexpr (std::is_same<Epi, SplitEpi>::value) {
        const int64_t kbeg = (int64_t)blockIdx.y * k_split;
        const int64_t kend = (kbeg + k_split) < K ? (kbeg + k_split) : K;
        gemm_nt_tile<T, BM, BN, BK, WM, WN, BPACK, PGR, Epi, KM>(A, lda, M, B, ldb, N, K, kbeg, kend, tm, tn, epi);
    } else {
        // only the partial products of a split launch cover part of K; with
        // the whole range fixed at compile time the K loop's addressing is
        // simpler (measured about 3% faster on the GEMM1 shape)
        gemm_nt_tile<T, BM, BN, BK, WM, WN, BPACK, PGR, Epi, KM>(A, lda, M, B, ldb, N, K, 0, K, tm, tn, epi);
    }
}

// Epilogue of a K-split launch: the fp32 partial tile of split s goes to
// P[s][m][n] (row-major M x N per split).
struct SplitEpi {
    float* P;
    int64_t M, N;
    struct Col {
        int64_t n;
        bool ok;
    };
    __device__ __forceinline__ Col col(int64_t n) const { return Col{n, n < N}; }
    __device__ __forceinline__ void store(int64_t m, const Col& c, float v) const {
        if (m < M && c.ok) P[((int64_t)blockIdx.y * M + m) * N + c.n] = v;
    }
};

// Sum the S partial products in split order (deterministic; after the
// epilogue's starting value, if it has one) and apply the real epilogue; one
// thread per 4 consecutive columns of a row.  When N is a
// multiple of 4 the four partial values of a split arrive in one 16-byte
// load and four splits are loaded before they are added, so that a thread
// keeps several loads in flight; the additions happen in the same order
// either way.
template <typename Epi>
__global__ __launch_bounds__(256) void split_reduce(const float* __restrict__ P, int S, int64_t M,
                                                    int64_t N, Epi epi) {
    const int64_t nq = ceil_div(N, 4);
    const bool vec = (N & 3) == 0;
    for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < M * nq;
         q += (int64_t)gridDim.x * blockDim.x) {
        const int64_t m = q / nq, n0 = (q % nq) * 4;
        float v[4] = {0.f, 0.f, 0.f, 0.f};
        if constexpr (InitEpi<Epi>::value) {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (n0 + e < N) v[e] = epi.init(m, epi.col(n0 + e));
        }
        if (vec) {
            const f32x4* p = reinterpret_cast<const f32x4*>(P + m * N + n0);
            const int64_t stride = M * N / 4;  // one split, in 16-byte units
            f32x4 acc = {v[0], v[1], v[2], v[3]};
            int s = 0;
            for (; s + 4 <= S; s += 4) {
                const f32x4 a = p[s * stride], b = p[(s + 1) * stride], c = p[(s + 2) * stride],
                            d = p[(s + 3) * stride];
                acc += a;
                acc += b;
                acc += c;
                acc += d;
            }
            for (; s < S; ++s) acc += p[s * stride];
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = acc[e];
        } else {
            for (int s = 0; s < S; ++s) {
                const float* p = P + ((int64_t)s * M + m) * N + n0;
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (n0 + e < N) v[e] += p[e];
            }
        }
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (n0 + e < N) epi.store(m, epi.col(n0 + e), v[e]);
    }
}

}  // namespace pifa
