// libpifa: C ABI for the PIFA layer forward on MI355X (gfx950).
//
// Algorithm "PIFA Layer" of arXiv 2501.19090 (Sec. 3.2) for row-major
// activations:
//   GEMM1  Y_p  = X W_p^T          -> Y[:, pivot_idx]    (+ Y_p hand-off)
//   GEMM2  Y_np = Y_p C^T          -> Y[:, nonpivot_idx]
// Both assignments are fused into the producing kernel's epilogue.  M > 16
// runs the LDS-tiled MFMA GEMM; M <= 16 runs the weight-streaming skinny
// MFMA kernel.  fp32 layers use the fp32 vector-ALU kernel.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "../../include/pifa.h"
#include "common.hpp"
#include "epilogue.hpp"
#include "gemm_f32.hpp"
#include "gemm_mfma.hpp"
#include "backward.hpp"
#include "build.hpp"
#include "gemv_skinny.hpp"
#include "layout.hpp"
#include "linalg64.hpp"
#include "prepack.hpp"
#include "probe.hpp"

using namespace pifa;

namespace {

// ------------------------------------------------------------------ config
constexpr int64_t kDecodeMaxM = 16;  // M at or below this takes the weight-streaming path
constexpr int kMaxGroup = kMaxSkinnyGroup;  // layers per pifa_group
constexpr int64_t kRowPad = 64;      // W_p rows / C columns padded to this multiple

constexpr int kGemmBK = 64;
constexpr int64_t kCus = 256;
constexpr int kSkinnyWaves = 8;

#define PIFA_HIP(call)                                  \
    do {                                                \
        if ((call) != hipSuccess) return PIFA_ERR_HIP;  \
    } while (0)

inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }
inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// A handle's memory lives on the device current at its creation; launching
// its kernels with another device current would touch that memory from the
// wrong GPU, so such calls are refused.
pifa_status check_device(int dev) {
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) return PIFA_ERR_HIP;
    return cur == dev ? PIFA_OK : PIFA_ERR_WRONG_DEVICE;
}

#define PIFA_ON_DEVICE(dev)                      \
    do {                                         \
        const pifa_status s_ = check_device(dev); \
        if (s_ != PIFA_OK) return s_;            \
    } while (0)
inline size_t esize(pifa_dtype dt) { return dt == PIFA_BF16 ? 2 : 4; }
inline bool valid_dtype(pifa_dtype dt) { return dt == PIFA_BF16 || dt == PIFA_F32; }

// A device buffer that only grows; growing waits for `st` (or, for a buffer
// shared by calls on any stream, the whole device) first so no kernel in
// flight still uses the old allocation.
struct GrowBuf {
    void* ptr = nullptr;
    size_t bytes = 0;
    pifa_status ensure(size_t need, hipStream_t st, bool any_stream = false) {
        if (need <= bytes) return PIFA_OK;
        PIFA_HIP(any_stream ? hipDeviceSynchronize() : hipStreamSynchronize(st));
        if (ptr) PIFA_HIP(hipFree(ptr));
        ptr = nullptr;
        bytes = 0;
        if (hipMalloc(&ptr, need) != hipSuccess) return PIFA_ERR_OOM;
        bytes = need;
        return PIFA_OK;
    }
    void release() {
        if (ptr) (void)hipFree(ptr);
        ptr = nullptr;
        bytes = 0;
    }
};

// ------------------------------------------------------------------ kernel timing
enum Site {
    kSitePifaGemm1 = 0,
    kSitePifaGemm2,
    kSitePifaGemv1,
    kSitePifaGemv2,
    kSitePifaF32Gemm1,
    kSitePifaF32Gemm2,
    kSiteDenseGemm,
    kSiteDenseGemv,
    kSiteDenseF32,
    kSiteLowrankGemm1,
    kSiteLowrankGemm2,
    kSiteLowrankGemv1,
    kSiteLowrankGemv2,
    kSiteLowrankF32,
    kSiteGroupGemm1,
    kSiteGroupGemm2,
    kSiteGroupGemv1,
    kSiteGroupGemv2,
    kSiteBwdData,
    kSiteBwdGp,
    kSiteBwdDx,
    kSiteBwdDwp,
    kSiteBwdDc,
    kSiteBwdRows,
    kSiteCalibGather,
    kSiteCalibGram,
    kSiteCalibSolve,
    kSiteCount
};

const char* const kSiteNames[kSiteCount] = {
    "pifa_gemm1_xwp",      "pifa_gemm2_ypc",      "pifa_gemv1_xwp",      "pifa_gemv2_ypc",
    "pifa_f32_gemm1",      "pifa_f32_gemm2",      "dense_gemm",          "dense_gemv",
    "dense_f32",           "lowrank_gemm1_xv",    "lowrank_gemm2_tu",    "lowrank_gemv1_xv",
    "lowrank_gemv2_tu",    "lowrank_f32",         "pifa_group_gemm1",    "pifa_group_gemm2",
    "pifa_group_gemv1",    "pifa_group_gemv2",    "pifa_bwd_gather",     "pifa_bwd_gp",
    "pifa_bwd_dx",         "pifa_bwd_dwp",        "pifa_bwd_dc",         "pifa_bwd_rows_f16",
    "pifa_calib_gather",   "pifa_calib_gram",     "pifa_calib_solve"};

struct Profiler {
    std::mutex mu;
    bool on = false;
    struct Rec {
        int site;
        hipEvent_t start, stop;
    };
    std::vector<Rec> pending;
    std::vector<hipEvent_t> pool;
    int64_t launches[kSiteCount] = {};
    double ms[kSiteCount] = {};

    hipEvent_t get() {
        if (!pool.empty()) {
            hipEvent_t e = pool.back();
            pool.pop_back();
            return e;
        }
        hipEvent_t e = nullptr;
        if (hipEventCreate(&e) != hipSuccess) return nullptr;
        return e;
    }
};

Profiler& profiler() {
    static Profiler p;
    return p;
}

// Set while a call runs that must create nothing (pifa_forward_noalloc):
// its launches are never bracketed by profiling events.
thread_local bool t_untimed = false;

// Brackets one launch with events when profiling is on.
struct TimedLaunch {
    int site;
    hipStream_t st;
    hipEvent_t start = nullptr, stop = nullptr;
    TimedLaunch(int s, hipStream_t stream) : site(s), st(stream) {
        Profiler& p = profiler();
        if (!p.on || t_untimed) return;
        std::lock_guard<std::mutex> g(p.mu);
        start = p.get();
        stop = p.get();
        if (start) (void)hipEventRecord(start, st);
    }
    ~TimedLaunch() {
        if (!start || !stop) return;
        Profiler& p = profiler();
        (void)hipEventRecord(stop, st);
        std::lock_guard<std::mutex> g(p.mu);
        p.pending.push_back({site, start, stop});
    }
};

// ------------------------------------------------------------------ launchers
enum TileCfg : int { kTile256x256 = 0, kTile256x192 = 1, kTile256x128 = 2, kTile128x128 = 3 };

// K splitting for launches that would leave CUs idle: at most kMaxSplit
// splits of at least four K tiles each, with the fp32 partials (s M N 4
// bytes, written and read back once) at most the operand bytes ((M + N) K 2)
// and capped at kMaxPartialBytes.  Measured on the LLaMA-7B attention
// products at M = 17..256: more splits than this fill more CUs but lose more
// to the partials and the short K loops than they gain.  No split when one
// split's partials (M N 4 bytes) exceed kMaxSplitSliceBytes: the tall, narrow
// products of the rank sweep at M = 4096 (N = 410..832 wide, 128..224 tiles
// of 128 x 128) ran 17-34% faster unsplit with CUs left idle than split in
// two (the r = 80% non-pivot product 38 against 57 us).
constexpr int64_t kMaxSplit = 16;
constexpr int64_t kMaxPartialBytes = 256ll << 20;
constexpr int64_t kMaxSplitSliceBytes = 6ll << 20;

struct SplitPlan {
    int64_t splits, k_split;
};

SplitPlan split_plan(int64_t tiles, int64_t M, int64_t N, int64_t K) {
    SplitPlan p{1, K};
    if (tiles >= kCus || M * N * 4 > kMaxSplitSliceBytes) return p;
    int64_t s = std::min<int64_t>({ceil_div(kCus, tiles), K / (4 * kGemmBK), kMaxSplit,
                                   std::max<int64_t>(1, K * (M + N) / (2 * std::max<int64_t>(1, M * N))),
                                   kMaxPartialBytes / std::max<int64_t>(1, M * N * 4)});
    if (s <= 1) return p;
    p.k_split = round_up(ceil_div(K, s), kGemmBK);
    p.splits = ceil_div(K, p.k_split);
    return p;
}

// Partial-product bytes a launch of this shape needs (0 if it does not split).
TileCfg pick_tile(int64_t M, int64_t N);

// No product with more rows than this splits K: its 128-row tiles alone
// fill the chip.  Reserving for every M up to it covers every split.
constexpr int64_t kSplitMaxM = 128 * kCus;

struct GemmPlan {
    int64_t bm, bn;
    SplitPlan split;
};
GemmPlan gemm_plan(int64_t M, int64_t N, int64_t K, bool wide_ok, bool can_split);

size_t split_bytes(int64_t M, int64_t N, int64_t K) {
    if (M == 0 || N == 0) return 0;
    const GemmPlan g = gemm_plan(M, N, K, true, true);
    return g.split.splits > 1 ? (size_t)(g.split.splits * M * N) * 4 : 0;
}

// Prefill tile configurations and a cost model to pick one: time ~ rounds
// of concurrently resident tiles x tile area x tiles sharing a CU / relative
// efficiency (measured: 256x256 and 256x192 tiles reach ~1.15x and 128x128
// ~0.9x the per-FLOP rate of 256x128).  128x128 fits two workgroups per CU.
// The 256x192 tile serves widths that leave the 256x128 grid just past a
// whole number of rounds (N = 2458 or 2867 at M = 4096: one round of
// 256x192 tiles instead of two of 256x128, 25% faster; N = 8960: 13%).
TileCfg pick_tile(int64_t M, int64_t N) {
    struct C { int64_t bm, bn, per_cu; double eff; };
    const C cfg[4] = {{256, 256, 1, 1.15}, {256, 192, 1, 1.15}, {256, 128, 1, 1.0}, {128, 128, 2, 0.9}};
    int best = 3;
    double best_t = 1e300;
    for (int i = 0; i < 4; ++i) {
        const int64_t tiles = ceil_div(M, cfg[i].bm) * ceil_div(N, cfg[i].bn);
        const int64_t rounds = ceil_div(tiles, kCus * cfg[i].per_cu);
        const int64_t sharing = std::min(cfg[i].per_cu, ceil_div(tiles, kCus));
        const double t = (double)rounds * cfg[i].bm * cfg[i].bn * sharing / cfg[i].eff;
        if (t < best_t * 0.999) {
            best_t = t;
            best = i;
        }
    }
    return (TileCfg)best;
}

// The tile and K split of a prefill product.  wide_ok: the epilogue fits the
// registers the 256 x 256 and 256 x 192 tiles leave; can_split: a partials
// buffer is available.
GemmPlan gemm_plan(int64_t M, int64_t N, int64_t K, bool wide_ok, bool can_split) {
    TileCfg cfg = pick_tile(M, N);
    if (!wide_ok && (cfg == kTile256x256 || cfg == kTile256x192)) cfg = kTile256x128;
    if (cfg == kTile256x256) return {256, 256, {1, K}};
    if (cfg == kTile256x192) return {256, 192, {1, K}};
    if (cfg == kTile256x128) return {256, 128, {1, K}};
    // at most 128 rows: split K over 64 x 64 tiles (4 waves), half the rows of
    // the smallest 8-wave tile, so no tile computes masked rows at M <= 64 and
    // twice the tiles need half the splits at M = 128, as long as each split
    // stays at most 1024 deep (one wave per SIMD cannot hide a longer loop:
    // the dense 4096^2 layer at M = 128 took 17.0 us with 2048-deep splits
    // against 15.1 us on 128 x 64 tiles).  Attention layer, HIP-graph replay:
    // PIFA M = 17 19.5 -> 18.0 us, M = 128 29.3 -> 26.5 us; dense M = 17-64
    // 12.4-13.2 -> 11.0-12.1 us.
    if (M <= 128 && can_split) {
        const SplitPlan p = split_plan(ceil_div(M, 64) * ceil_div(N, 64), M, N, K);
        if (p.splits > 1 && p.k_split <= 1024) return {64, 64, p};
    }
    // too few tiles for the chip even at 128 x 128: split K, or, when that
    // does not pay and 128 x 128 tiles keep at most half the chip busy, take
    // 128 x 64 tiles if they fill it in one round (the rank sweep's 410-wide
    // products at M = 4096: 224 tiles, 35 against 45 us)
    const int64_t t128x128 = ceil_div(M, 128) * ceil_div(N, 128);
    const int64_t t128x64 = ceil_div(M, 128) * ceil_div(N, 64);
    const SplitPlan p = can_split ? split_plan(t128x128, M, N, K) : SplitPlan{1, K};
    if (p.splits == 1 && 2 * t128x128 <= kCus && t128x64 <= kCus) return {128, 64, p};
    if (p.splits > 1) {
        // a product at most 2048 deep whose 64 x 64 tiles keep at least half
        // the chip busy runs them over its whole K: no partial sums and no
        // reduction launch (the attention layer's non-pivot product, K = 2048:
        // M = 256 17.6 -> 14.6 us, M = 512 20.8 -> 15.7 us).  Deeper products
        // keep the split (the pivot product, K = 4096, at M = 256: 19.2 us
        // split against 24.4 us unsplit on 64 x 64 tiles).
        if (K <= 2048 && 2 * ceil_div(M, 64) * ceil_div(N, 64) >= kCus) return {64, 64, {1, K}};
        // a split product: 128 x 64 tiles need half the splits for as many
        // workgroups, so half the partial sums (the attention layer at
        // M = 128..256: 10-15% faster per product)
        const SplitPlan q = split_plan(t128x64, M, N, K);
        if (q.splits > 1) return {128, 64, q};
    }
    return {128, 128, p};
}

template <typename T, bool BPACK, typename Epi, int KM = 0>
hipError_t launch_gemm(int site, const T* A, int64_t lda, int64_t M, const T* B, int64_t ldb,
                       int64_t N, int64_t K, Epi epi, float* partials, hipStream_t st) {
    if (M == 0 || N == 0) return hipSuccess;
    TimedLaunch timed(site, st);
    // epilogues that load the accumulators' starting values, or add into
    // fp64 / store fp32 outputs, need more registers than the 256 x 256 and
    // 256 x 192 tiles have left (they spill there)
    constexpr bool kWideOk = !InitEpi<Epi>::value && !std::is_same<Epi, AccF64Epi>::value &&
                             !std::is_same<Epi, ScatterEpi<float, kWsNone>>::value;
    const GemmPlan g = gemm_plan(M, N, K, kWideOk, partials != nullptr);
    const dim3 grid((unsigned)(ceil_div(M, g.bm) * ceil_div(N, g.bn)));
    if (g.bm == 256 && g.bn == 256) {
        if constexpr (DualEpiT<Epi>::value)
            hipLaunchKernelGGL((gemm_nt_mfma<T, 256, 256, kGemmBK, 2, 4, BPACK, 1, ScatterEpi<bf16, kWsF16>, KM>), grid,
                               dim3(8 * kWave), 0, st, A, lda, M, B, ldb, N, K, K, epi.elementwise());
        else if constexpr (kWideOk)
            hipLaunchKernelGGL((gemm_nt_mfma<T, 256, 256, kGemmBK, 2, 4, BPACK, 1, Epi, KM>), grid, dim3(8 * kWave), 0,
                               st, A, lda, M, B, ldb, N, K, K, epi);
    } else if (g.bm == 256 && g.bn == 192) {
        // the 256-row tiles write the pivot product's fp16 hand-off element by
        // element: staged through LDS it cost more than its stores save (M =
        // 4096, three alternating passes, us per launch: attention layer,
        // 256 x 128 tiles, 80.1-81.2 -> 76.3-76.4; r = 70% of 4096, 256 x 192
        // tiles, 103.9-104.2 -> 100.0-100.4).  The 128-row tiles keep it
        // staged (1-2 us faster there).
        if constexpr (DualEpiT<Epi>::value)
            hipLaunchKernelGGL((gemm_nt_mfma<T, 256, 192, kGemmBK, 4, 2, BPACK, 2, ScatterEpi<bf16, kWsF16>, KM>), grid,
                               dim3(8 * kWave), 0, st, A, lda, M, B, ldb, N, K, K, epi.elementwise());
        else if constexpr (kWideOk)
            hipLaunchKernelGGL((gemm_nt_mfma<T, 256, 192, kGemmBK, 4, 2, BPACK, 2, Epi, KM>), grid, dim3(8 * kWave), 0,
                               st, A, lda, M, B, ldb, N, K, K, epi);
    } else if (g.bm == 256) {
        if constexpr (DualEpiT<Epi>::value)
            hipLaunchKernelGGL((gemm_nt_mfma<T, 256, 128, kGemmBK, 4, 2, BPACK, 2, ScatterEpi<bf16, kWsF16>, KM>), grid,
                               dim3(8 * kWave), 0, st, A, lda, M, B, ldb, N, K, K, epi.elementwise());
        else
            hipLaunchKernelGGL((gemm_nt_mfma<T, 256, 128, kGemmBK, 4, 2, BPACK, 2, Epi, KM>), grid, dim3(8 * kWave), 0,
                               st, A, lda, M, B, ldb, N, K, K, epi);
    } else if (g.split.splits == 1) {
        if (g.bm == 64)
            hipLaunchKernelGGL((gemm_nt_mfma<T, 64, 64, kGemmBK, 2, 2, BPACK, 2, Epi, KM>), grid, dim3(4 * kWave), 0,
                               st, A, lda, M, B, ldb, N, K, K, epi);
        else if (g.bn == 64)
            hipLaunchKernelGGL((gemm_nt_mfma<T, 128, 64, kGemmBK, 4, 2, BPACK, 2, Epi, KM>), grid, dim3(8 * kWave), 0,
                               st, A, lda, M, B, ldb, N, K, K, epi);
        else
            hipLaunchKernelGGL((gemm_nt_mfma<T, 128, 128, kGemmBK, 4, 2, BPACK, 2, Epi, KM>), grid, dim3(8 * kWave), 0,
                               st, A, lda, M, B, ldb, N, K, K, epi);
    } else {
        SplitEpi se{partials, M, N};
        const dim3 sgrid(grid.x, (unsigned)g.split.splits);
        if (g.bm == 64)
            hipLaunchKernelGGL((gemm_nt_mfma<T, 64, 64, kGemmBK, 2, 2, BPACK, 2, SplitEpi, KM>), sgrid,
                               dim3(4 * kWave), 0, st, A, lda, M, B, ldb, N, K, g.split.k_split, se);
        else if (g.bn == 64)
            hipLaunchKernelGGL((gemm_nt_mfma<T, 128, 64, kGemmBK, 4, 2, BPACK, 2, SplitEpi, KM>), sgrid,
                               dim3(8 * kWave), 0, st, A, lda, M, B, ldb, N, K, g.split.k_split, se);
        else
            hipLaunchKernelGGL((gemm_nt_mfma<T, 128, 128, kGemmBK, 4, 2, BPACK, 2, SplitEpi, KM>), sgrid,
                               dim3(8 * kWave), 0, st, A, lda, M, B, ldb, N, K, g.split.k_split, se);
        const int64_t work = M * ceil_div(N, 4);
        hipLaunchKernelGGL((split_reduce<Epi>), dim3((unsigned)std::min<int64_t>(ceil_div(work, 256), 65536)),
                           dim3(256), 0, st, (const float*)partials, (int)g.split.splits, M, N, epi);
    }
    return hipGetLastError();
}

template <typename Epi>
hipError_t launch_gemm_f32(int site, const float* A, int64_t lda, int64_t M, const float* B,
                           int64_t ldb, int64_t N, int64_t K, Epi epi, hipStream_t st) {
    if (M == 0 || N == 0) return hipSuccess;
    TimedLaunch timed(site, st);
    hipLaunchKernelGGL((gemm_nt_f32<Epi>), dim3((unsigned)ceil_div(N, 64), (unsigned)ceil_div(M, 64)),
                       dim3(256), 0, st, A, lda, M, B, ldb, N, K, epi);
    return hipGetLastError();
}

// Launch shape of a weight-streaming product with one 16-row activation tile:
// waves per workgroup, 128-wide K blocks per wave step (unroll) and
// workgroups per 16-row weight group (parts).  Measured over every decode
// shape of the LLaMA-7B / 70B layers and the rank sweep on MI355X:
//  * few activation rows (M <= 4): the A operand costs almost nothing, so the
//    shape that puts the whole weight stream in flight at once wins -- 16
//    waves, enough unroll to cover K in about one step, and narrow products
//    (at most 128 groups) split over two workgroups;
//  * more rows: every workgroup re-reads the activation block, so fewer,
//    deeper workgroups (8 waves, unroll up to 4) win, and a group is split
//    only when the grid would be small or K is long.
struct SkinnyShape {
    int waves, unroll, parts;
};

SkinnyShape skinny_shape(int64_t M, int64_t groups, int64_t KB) {
    if (M <= 4) return {KB >= 8 ? 16 : 8, KB > 16 ? 2 : 1, groups <= 128 ? 2 : 1};
    return {8, KB <= 8 ? 1 : KB <= 16 ? 2 : 4, (groups < 128 || (groups < 256 && KB >= 64)) ? 2 : 1};
}

template <typename TB, int W, int U, int MT, int P, typename AL, typename Epi>
void skinny_launch(const AL& al, const TB* B, int64_t N, int64_t K, const Epi& epi, hipStream_t st) {
    hipLaunchKernelGGL((skinny_packed<TB, W, U, MT, P, AL, Epi>), dim3((unsigned)(P * packed_groups(N))),
                       dim3(W * kWave), 0, st, al, B, N, K, epi);
}

// B in lane order (layout.hpp), logical N x K.  Several activation tiles
// (MT > 1) use 8 waves without unrolling; a narrow product (few 16-row
// groups) splits each group over 2 or 4 workgroups so the weight stream is
// spread over the whole chip.
// Long weight streams (at least kStreamMinBlocks blocks of 16 rows x 128 K,
// about 25 MB) with at most kStreamRows activation rows take the streaming
// kernel: one 16-wave workgroup per CU walks its share of the units with the
// next pass's weights in flight (measured 6-19% faster from 33 MB up, 201 MB
// of the 70B up projection's C in 35 against 43 us; equal or slower on the
// 8-17 MB streams of the 4096 x 4096 layer, where a single round of
// workgroups already covers the stream).
constexpr int64_t kStreamMinBlocks = 6144;
constexpr int64_t kStreamMaxLds = 65536;

// grp.start[] counts 16-row groups per problem; the kernel's units are
// PARTS per group
template <typename TB, int PARTS, typename AL, typename Epi>
void skinny_stream_launch(SkinnyGroup<TB, AL, Epi> grp, int64_t k_blocks_total, hipStream_t st) {
    for (int q = 0; q <= grp.n; ++q) grp.start[q] *= PARTS;
    const int64_t units = grp.start[grp.n];
    const int64_t per_wg = ceil_div(units, (int64_t)kCus);
    hipLaunchKernelGGL((skinny_stream<TB, 16, 1, PARTS, AL, Epi>), dim3((unsigned)ceil_div(units, per_wg)),
                       dim3(16 * kWave), (size_t)skinny_stream_lds(grp.p[0].al.M, k_blocks_total, AL::kOps, 16), st,
                       grp);
}

// Whether a weight stream of `blocks` 16 x 128 blocks over k_blocks_total
// staged K blocks takes the streaming kernel.
inline bool use_stream(int64_t M, int64_t blocks, int64_t k_blocks_total, int ops) {
    return M <= kStreamRows && blocks >= kStreamMinBlocks &&
           skinny_stream_lds(M, k_blocks_total, ops, 16) <= kStreamMaxLds;
}

template <typename TB, int MT, typename AL, typename Epi>
void skinny_packed_mt(const AL& al, const TB* B, int64_t N, int64_t K, const Epi& epi, hipStream_t st) {
    const int64_t groups = packed_groups(N);
    if constexpr (MT == 1) {
        const int64_t KB = packed_kblocks(K);
        if (use_stream(al.M, groups * KB, KB, AL::kOps)) {
            SkinnyGroup<TB, AL, Epi> one;
            one.p[0] = SkinnyProblem<TB, AL, Epi>{al, B, K, epi};
            one.n = 1;
            one.start[0] = 0;
            one.start[1] = groups;
            if (groups <= 128) return skinny_stream_launch<TB, 2>(one, KB, st);
            return skinny_stream_launch<TB, 1>(one, KB, st);
        }
        const SkinnyShape c = skinny_shape(al.M, groups, packed_kblocks(K));
        const int key = c.waves * 100 + c.unroll * 10 + c.parts;
        switch (key) {
            case 811: return skinny_launch<TB, 8, 1, 1, 1>(al, B, N, K, epi, st);
            case 812: return skinny_launch<TB, 8, 1, 1, 2>(al, B, N, K, epi, st);
            case 821: return skinny_launch<TB, 8, 2, 1, 1>(al, B, N, K, epi, st);
            case 822: return skinny_launch<TB, 8, 2, 1, 2>(al, B, N, K, epi, st);
            case 841: return skinny_launch<TB, 8, 4, 1, 1>(al, B, N, K, epi, st);
            case 842: return skinny_launch<TB, 8, 4, 1, 2>(al, B, N, K, epi, st);
            case 1611: return skinny_launch<TB, 16, 1, 1, 1>(al, B, N, K, epi, st);
            case 1612: return skinny_launch<TB, 16, 1, 1, 2>(al, B, N, K, epi, st);
            case 1621: return skinny_launch<TB, 16, 2, 1, 1>(al, B, N, K, epi, st);
            default: return skinny_launch<TB, 16, 2, 1, 2>(al, B, N, K, epi, st);
        }
    } else {
        if (groups >= kCus) skinny_launch<TB, kSkinnyWaves, 1, MT, 1>(al, B, N, K, epi, st);
        else if (2 * groups >= kCus) skinny_launch<TB, kSkinnyWaves, 1, MT, 2>(al, B, N, K, epi, st);
        else skinny_launch<TB, kSkinnyWaves, 1, MT, 4>(al, B, N, K, epi, st);
    }
}

template <typename TB, typename AL, typename Epi>
hipError_t launch_skinny_packed(int site, AL al, const TB* B, int64_t N, int64_t K, Epi epi,
                                hipStream_t st) {
    if (packed_groups(N) == 0) return hipSuccess;
    TimedLaunch timed(site, st);
    if (al.M <= 16) skinny_packed_mt<TB, 1>(al, B, N, K, epi, st);
    else if (al.M <= 32) skinny_packed_mt<TB, 2>(al, B, N, K, epi, st);
    else if (al.M <= 64) skinny_packed_mt<TB, 4>(al, B, N, K, epi, st);
    else skinny_packed_mt<TB, 8>(al, B, N, K, epi, st);
    return hipGetLastError();
}

// Grouped weight streams for decode-sized M (at most 16 rows).
template <typename TB, typename AL, typename Epi>
hipError_t launch_skinny_grouped(int site, SkinnyGroup<TB, AL, Epi> grp, const int64_t* n_rows,
                                 hipStream_t st) {
    grp.start[0] = 0;
    for (int q = 0; q < grp.n; ++q) grp.start[q + 1] = grp.start[q] + packed_groups(n_rows[q]);
    if (grp.start[grp.n] == 0) return hipSuccess;
    int64_t KB = 0, kb_total = 0, blocks = 0;
    for (int q = 0; q < grp.n; ++q) {
        KB = std::max(KB, packed_kblocks(grp.p[q].K));
        kb_total += packed_kblocks(grp.p[q].K);
        blocks += (grp.start[q + 1] - grp.start[q]) * packed_kblocks(grp.p[q].K);
    }
    TimedLaunch timed(site, st);
    if (use_stream(grp.p[0].al.M, blocks, kb_total, AL::kOps)) {
        skinny_stream_launch<TB, 1>(grp, kb_total, st);
        return hipGetLastError();
    }
    const SkinnyShape c = skinny_shape(grp.p[0].al.M, grp.start[grp.n], KB);  // one workgroup per group
    const dim3 grid((unsigned)grp.start[grp.n]);
    if (c.waves == 16 && c.unroll == 2)
        hipLaunchKernelGGL((skinny_packed_grouped<TB, 16, 2, 1, AL, Epi>), grid, dim3(16 * kWave), 0, st, grp);
    else if (c.waves == 16)
        hipLaunchKernelGGL((skinny_packed_grouped<TB, 16, 1, 1, AL, Epi>), grid, dim3(16 * kWave), 0, st, grp);
    else if (c.unroll == 4)
        hipLaunchKernelGGL((skinny_packed_grouped<TB, 8, 4, 1, AL, Epi>), grid, dim3(8 * kWave), 0, st, grp);
    else if (c.unroll == 2)
        hipLaunchKernelGGL((skinny_packed_grouped<TB, 8, 2, 1, AL, Epi>), grid, dim3(8 * kWave), 0, st, grp);
    else
        hipLaunchKernelGGL((skinny_packed_grouped<TB, 8, 1, 1, AL, Epi>), grid, dim3(8 * kWave), 0, st, grp);
    return hipGetLastError();
}

// B row-major with row stride ldb.
template <typename TB, int MT, typename AL, typename Epi>
void skinny_rowmajor_mt(const AL& al, const TB* B, int64_t ldb, int64_t N, int64_t K, const Epi& epi,
                        hipStream_t st) {
    constexpr int U = MT == 1 ? 2 : 1;
    hipLaunchKernelGGL((skinny_rowmajor<TB, kSkinnyWaves, U, MT, AL, Epi>), dim3((unsigned)ceil_div(N, kSkinnyRows)),
                       dim3(kSkinnyWaves * kWave), 0, st, al, B, ldb, N, K, epi);
}

template <typename TB, typename AL, typename Epi>
hipError_t launch_skinny_rowmajor(int site, AL al, const TB* B, int64_t ldb, int64_t N, int64_t K,
                                  Epi epi, hipStream_t st) {
    if (N == 0) return hipSuccess;
    TimedLaunch timed(site, st);
    if (al.M <= 16) skinny_rowmajor_mt<TB, 1>(al, B, ldb, N, K, epi, st);
    else if (al.M <= 32) skinny_rowmajor_mt<TB, 2>(al, B, ldb, N, K, epi, st);
    else if (al.M <= 64) skinny_rowmajor_mt<TB, 4>(al, B, ldb, N, K, epi, st);
    else skinny_rowmajor_mt<TB, 8>(al, B, ldb, N, K, epi, st);
    return hipGetLastError();
}

unsigned grid_for(int64_t work) { return (unsigned)std::max<int64_t>(1, std::min<int64_t>(ceil_div(work, 256), 65536)); }

// Row-major copy with zero padding (fp32 layers keep row-major weights).
hipError_t pack_rowmajor_f32(const void* src, int64_t rows, int64_t cols, void* dst, int64_t rows_pad,
                             int64_t cols_pad) {
    if (rows_pad * cols_pad == 0) return hipSuccess;
    hipLaunchKernelGGL((pack_pad<float>), dim3(grid_for(rows_pad * cols_pad)), dim3(256), 0, 0,
                       (const float*)src, rows, cols, cols, (float*)dst, rows_pad, cols_pad);
    return hipGetLastError();
}

// bf16 rows x cols -> lane order of a rows_log x cols_log matrix (bf16).
hipError_t pack_lane_bf16(const void* src, int64_t rows, int64_t cols, void* dst, int64_t rows_log,
                          int64_t cols_log) {
    const int64_t chunks = packed_groups(rows_log) * packed_kblocks(cols_log) * kPackChunks;
    if (chunks == 0) return hipSuccess;
    hipLaunchKernelGGL((pack_lane_order<uint16_t, uint16_t>), dim3(grid_for(chunks)), dim3(256), 0, 0,
                       (const uint16_t*)src, rows, cols, cols, (uint16_t*)dst, rows_log, cols_log, 1.f);
    return hipGetLastError();
}

// Largest finite |x| of a bf16 device array (synchronous).
pifa_status absmax_bf16_host(const void* src, int64_t n, float* out) {
    unsigned* dmax = nullptr;
    if (hipMalloc(&dmax, sizeof(unsigned)) != hipSuccess) return PIFA_ERR_OOM;
    unsigned bits = 0;
    bool ok = hipMemset(dmax, 0, sizeof(unsigned)) == hipSuccess;
    if (ok && n > 0) {
        hipLaunchKernelGGL(absmax_bf16, dim3((unsigned)std::min<int64_t>(ceil_div(n, 256), 4096)), dim3(256),
                           0, 0, (const uint16_t*)src, n, dmax);
        ok = hipGetLastError() == hipSuccess;
    }
    ok = ok && hipMemcpy(&bits, dmax, sizeof(unsigned), hipMemcpyDeviceToHost) == hipSuccess;
    (void)hipFree(dmax);
    if (!ok) return PIFA_ERR_HIP;
    *out = __builtin_bit_cast(float, bits << 16);
    return PIFA_OK;
}

// ------------------------------------------------------------------ shared workspace
// Workspace of the stateless baselines, one per device.  Growing it waits
// for the whole device; the calls that use it must not overlap on the GPU
// (the same rule as for one handle used from several streams).
struct DeviceScratch {
    std::mutex mu;
    GrowBuf inter;  // intermediate X V^T of the stateless low-rank baseline
    GrowBuf part;   // K-split partial products of stateless calls
};

DeviceScratch& device_scratch(int dev) {
    static std::mutex table_mu;
    static std::vector<DeviceScratch*> table;
    std::lock_guard<std::mutex> g(table_mu);
    if ((size_t)dev >= table.size()) table.resize((size_t)dev + 1, nullptr);
    if (!table[(size_t)dev]) table[(size_t)dev] = new DeviceScratch();
    return *table[(size_t)dev];
}

pifa_status check_dims(const pifa_dims& d) {
    if (d.d_in < 1 || d.d_out < 1 || d.r < 1) return PIFA_ERR_INVALID_ARG;
    if (d.r > d.d_in || d.r > d.d_out) return PIFA_ERR_INVALID_ARG;
    if (d.d_in > INT32_MAX || d.d_out > INT32_MAX) return PIFA_ERR_UNSUPPORTED;
    return PIFA_OK;
}

pifa_status check_rows_aligned(pifa_dtype dt, int64_t d_in) {
    return (dt == PIFA_BF16 && d_in % 8 != 0) ? PIFA_ERR_UNSUPPORTED : PIFA_OK;
}

}  // namespace

// ===================================================================== handles
// bf16 layers keep their weights in lane order (layout.hpp); fp32 layers keep
// row-major copies for the vector-ALU kernels.
struct pifa_layer {
    int device = 0;
    pifa_dtype dtype = PIFA_BF16;
    int64_t d_in = 0, d_out = 0, r = 0, n_np = 0, r_pad = 0;
    void* Wp = nullptr;        // bf16: lane order of r_pad x d_in; f32: r x d_in
    void* C = nullptr;         // bf16: fp16 lane order of n_np x r_pad, times 2^c_log2; f32: n_np x r
    int32_t* piv = nullptr;    // r
    int32_t* npiv = nullptr;   // n_np
    int* overflow = nullptr;
    int c_log2 = 0, y_log2 = 0;
    GrowBuf ws;                // Y_p hand-off
    GrowBuf part;              // K-split partial products
    // backward, built on first use from the packed forward weights
    void* bwd_wpt = nullptr;   // lane order of d_in x r_pad: W_p^T in fp16 times 2^bwd_cw
    void* bwd_ct = nullptr;    // lane order of r_pad x ldc: C^T in bf16 (ldc = n_np rounded up to 8)
    int bwd_cw = 0;
    GrowBuf bws;               // backward operands and partial products
};

struct lowrank_layer {
    int device = 0;
    pifa_dtype dtype = PIFA_BF16;
    int64_t d_in = 0, d_out = 0, r = 0, r_pad = 0;
    void* U = nullptr;  // bf16: lane order of d_out x r_pad; f32: d_out x r
    void* V = nullptr;  // bf16: lane order of r_pad x d_in; f32: r x d_in
    GrowBuf ws;
    GrowBuf part;
};

struct dense_layer {
    int device = 0;
    pifa_dtype dtype = PIFA_BF16;
    int64_t d_in = 0, d_out = 0;
    void* W = nullptr;  // bf16: lane order of d_out x d_in; f32: d_out x d_in
    GrowBuf part;
};

// Layers that share X.  The members keep their C, non-pivot indices (already
// offset into the group's output) and C scale; their W_p blocks are moved
// into one concatenated lane-order W_p, so nothing is stored twice.
struct pifa_group {
    int device = 0;
    int n = 0;
    int64_t d_in = 0, d_out = 0, r_pad = 0;  // d_out, r_pad: sums over the members
    std::vector<pifa_layer*> layers;
    std::vector<int64_t> r_off;  // first W_p row (and Y_p column) of each member
    void* Wp = nullptr;          // lane order of r_pad x d_in
    int32_t* piv = nullptr;      // r_pad: output column of each W_p row, -1 on padding rows
    int* overflow = nullptr;
    int y_log2 = 0;
    GrowBuf ws;
    GrowBuf part;
};

namespace {

void free_layer(pifa_layer* h) {
    if (!h) return;
    if (h->Wp) (void)hipFree(h->Wp);
    if (h->C) (void)hipFree(h->C);
    if (h->piv) (void)hipFree(h->piv);
    if (h->npiv) (void)hipFree(h->npiv);
    if (h->overflow) (void)hipFree(h->overflow);
    if (h->bwd_wpt) (void)hipFree(h->bwd_wpt);
    if (h->bwd_ct) (void)hipFree(h->bwd_ct);
    h->ws.release();
    h->part.release();
    h->bws.release();
    delete h;
}

void free_lowrank(lowrank_layer* h) {
    if (!h) return;
    if (h->U) (void)hipFree(h->U);
    if (h->V) (void)hipFree(h->V);
    h->ws.release();
    h->part.release();
    delete h;
}

void free_group(pifa_group* g) {
    if (!g) return;
    for (pifa_layer* h : g->layers) free_layer(h);
    if (g->Wp) (void)hipFree(g->Wp);
    if (g->piv) (void)hipFree(g->piv);
    if (g->overflow) (void)hipFree(g->overflow);
    g->ws.release();
    g->part.release();
    delete g;
}

size_t group_ws_bytes(const pifa_group* g, int64_t M) {
    return (size_t)M * (size_t)g->r_pad * (M <= kDecodeMaxM ? 4 : 2);
}

size_t group_part_bytes(const pifa_group* g, int64_t M) {
    if (M <= kDecodeMaxM) return 0;
    size_t b = split_bytes(M, g->r_pad, g->d_in);
    for (const pifa_layer* h : g->layers) b = std::max(b, split_bytes(M, h->n_np, h->r_pad));
    return b;
}

void free_dense(dense_layer* h) {
    if (!h) return;
    if (h->W) (void)hipFree(h->W);
    h->part.release();
    delete h;
}

size_t pifa_ws_bytes(const pifa_layer* h, int64_t M) {
    if (h->dtype == PIFA_F32) return (size_t)M * (size_t)h->r * 4;
    if (M <= kDecodeMaxM) return (size_t)M * (size_t)h->r_pad * 4;
    return (size_t)M * (size_t)h->r_pad * 2;
}

size_t pifa_part_bytes(const pifa_layer* h, int64_t M) {
    if (h->dtype == PIFA_F32 || M <= kDecodeMaxM) return 0;
    return std::max(split_bytes(M, h->r_pad, h->d_in), split_bytes(M, h->n_np, h->r_pad));
}

size_t lowrank_part_bytes(pifa_dtype dt, int64_t M, int64_t d_in, int64_t d_out, int64_t r_cols) {
    if (dt == PIFA_F32 || M <= kDecodeMaxM) return 0;
    return std::max(split_bytes(M, r_cols, d_in), split_bytes(M, d_out, r_cols));
}

size_t dense_part_bytes(pifa_dtype dt, int64_t M, int64_t d_in, int64_t d_out) {
    if (dt == PIFA_F32 || M <= kDecodeMaxM) return 0;
    return split_bytes(M, d_out, d_in);
}

size_t lowrank_ws_bytes(pifa_dtype dt, int64_t M, int64_t r_cols) {
    if (dt == PIFA_F32 || M <= kDecodeMaxM) return (size_t)M * (size_t)r_cols * 4;
    return (size_t)M * (size_t)r_cols * 2;
}

// A contiguous output with rows of ld elements at p can take the staged
// 16-byte-store epilogue.
inline bool staged_ok(const void* p, int64_t ld) { return aligned16(p) && ld % 8 == 0; }

// Y = (X V^T) U^T.  V: r_cols x d_in, U: d_out x r_cols, both in lane order
// when PACKED (bf16 handle), else row-major (stateless call, fp32).
template <bool PACKED>
pifa_status lowrank_run(pifa_dtype dt, const void* U, const void* V, const void* X, void* Y,
                        int64_t M, int64_t d_in, int64_t d_out, int64_t r_cols, void* T,
                        float* partials, hipStream_t st) {
    hipError_t e;
    if (dt == PIFA_F32) {
        float* t = (float*)T;
        e = launch_gemm_f32(kSiteLowrankF32, (const float*)X, d_in, M, (const float*)V, d_in, r_cols,
                            d_in,
                            make_epi<float, kWsNone>(t, r_cols, nullptr, r_cols, 1.f, nullptr, 0, 0,
                                                     1.f, nullptr, M),
                            st);
        if (e != hipSuccess) return PIFA_ERR_HIP;
        e = launch_gemm_f32(kSiteLowrankF32, t, r_cols, M, (const float*)U, r_cols, d_out, r_cols,
                            make_epi<float, kWsNone>((float*)Y, d_out, nullptr, d_out, 1.f, nullptr,
                                                     0, 0, 1.f, nullptr, M),
                            st);
        return e == hipSuccess ? PIFA_OK : PIFA_ERR_HIP;
    }
    if (M <= kDecodeMaxM) {
        float* t = (float*)T;
        auto e1 = make_epi<float, kWsNone>(t, r_cols, nullptr, r_cols, 1.f, nullptr, 0, 0, 1.f, nullptr, M);
        auto e2 = make_epi<bf16, kWsNone>((bf16*)Y, d_out, nullptr, d_out, 1.f, nullptr, 0, 0, 1.f,
                                          nullptr, M);
        ALoad16<bf16> a1{(const bf16*)X, d_in, M};
        ASplit32<bf16> a2{t, r_cols, M, 1.f};
        if constexpr (PACKED) {
            e = launch_skinny_packed<bf16>(kSiteLowrankGemv1, a1, (const bf16*)V, r_cols, d_in, e1, st);
            if (e != hipSuccess) return PIFA_ERR_HIP;
            e = launch_skinny_packed<bf16>(kSiteLowrankGemv2, a2, (const bf16*)U, d_out, r_cols, e2, st);
        } else {
            e = launch_skinny_rowmajor<bf16>(kSiteLowrankGemv1, a1, (const bf16*)V, d_in, r_cols, d_in, e1, st);
            if (e != hipSuccess) return PIFA_ERR_HIP;
            e = launch_skinny_rowmajor<bf16>(kSiteLowrankGemv2, a2, (const bf16*)U, r_cols, d_out, r_cols, e2,
                                             st);
        }
        return e == hipSuccess ? PIFA_OK : PIFA_ERR_HIP;
    }
    bf16* t = (bf16*)T;
    // contiguous outputs with 16-byte rows take the staged 16-byte-store
    // epilogue, as the PIFA hand-off does
    if (staged_ok(t, r_cols))
        e = launch_gemm<bf16, PACKED>(kSiteLowrankGemm1, (const bf16*)X, d_in, M, (const bf16*)V, d_in, r_cols, d_in,
                                      StagedEpi<bf16>{(uint16_t*)t, r_cols, r_cols, 1.f, nullptr, M}, partials, st);
    else
        e = launch_gemm<bf16, PACKED>(kSiteLowrankGemm1, (const bf16*)X, d_in, M, (const bf16*)V, d_in,
                                      r_cols, d_in,
                                      make_epi<bf16, kWsNone>(t, r_cols, nullptr, r_cols, 1.f, nullptr, 0,
                                                              0, 1.f, nullptr, M),
                                      partials, st);
    if (e != hipSuccess) return PIFA_ERR_HIP;
    if (staged_ok(Y, d_out))
        e = launch_gemm<bf16, PACKED>(kSiteLowrankGemm2, t, r_cols, M, (const bf16*)U, r_cols, d_out, r_cols,
                                      StagedEpi<bf16>{(uint16_t*)Y, d_out, d_out, 1.f, nullptr, M}, partials, st);
    else
        e = launch_gemm<bf16, PACKED>(kSiteLowrankGemm2, t, r_cols, M, (const bf16*)U, r_cols, d_out, r_cols,
                                      make_epi<bf16, kWsNone>((bf16*)Y, d_out, nullptr, d_out, 1.f, nullptr,
                                                              0, 0, 1.f, nullptr, M),
                                      partials, st);
    return e == hipSuccess ? PIFA_OK : PIFA_ERR_HIP;
}

// Y = X W^T; W lane order (PACKED) or row-major.
template <bool PACKED>
pifa_status dense_run(pifa_dtype dt, const void* W, const void* X, void* Y, int64_t M, int64_t d_in,
                      int64_t d_out, float* partials, hipStream_t st) {
    hipError_t e;
    if (dt == PIFA_F32) {
        e = launch_gemm_f32(kSiteDenseF32, (const float*)X, d_in, M, (const float*)W, d_in, d_out, d_in,
                            make_epi<float, kWsNone>((float*)Y, d_out, nullptr, d_out, 1.f, nullptr,
                                                     0, 0, 1.f, nullptr, M),
                            st);
        return e == hipSuccess ? PIFA_OK : PIFA_ERR_HIP;
    }
    auto epi = make_epi<bf16, kWsNone>((bf16*)Y, d_out, nullptr, d_out, 1.f, nullptr, 0, 0, 1.f,
                                       nullptr, M);
    if (M <= kDecodeMaxM) {
        ALoad16<bf16> a{(const bf16*)X, d_in, M};
        if constexpr (PACKED)
            e = launch_skinny_packed<bf16>(kSiteDenseGemv, a, (const bf16*)W, d_out, d_in, epi, st);
        else
            e = launch_skinny_rowmajor<bf16>(kSiteDenseGemv, a, (const bf16*)W, d_in, d_out, d_in, epi, st);
        return e == hipSuccess ? PIFA_OK : PIFA_ERR_HIP;
    }
    if (staged_ok(Y, d_out))
        e = launch_gemm<bf16, PACKED>(kSiteDenseGemm, (const bf16*)X, d_in, M, (const bf16*)W, d_in, d_out, d_in,
                                      StagedEpi<bf16>{(uint16_t*)Y, d_out, d_out, 1.f, nullptr, M}, partials, st);
    else
        e = launch_gemm<bf16, PACKED>(kSiteDenseGemm, (const bf16*)X, d_in, M, (const bf16*)W, d_in, d_out,
                                      d_in, epi, partials, st);
    return e == hipSuccess ? PIFA_OK : PIFA_ERR_HIP;
}

}  // namespace

// ===================================================================== C ABI
extern "C" {

const char* pifa_status_string(pifa_status s) {
    switch (s) {
        case PIFA_OK: return "PIFA_OK";
        case PIFA_ERR_INVALID_ARG: return "PIFA_ERR_INVALID_ARG";
        case PIFA_ERR_BAD_INDEX: return "PIFA_ERR_BAD_INDEX";
        case PIFA_ERR_UNSUPPORTED: return "PIFA_ERR_UNSUPPORTED";
        case PIFA_ERR_HIP: return "PIFA_ERR_HIP";
        case PIFA_ERR_OOM: return "PIFA_ERR_OOM";
        case PIFA_ERR_NOT_RANK_R: return "PIFA_ERR_NOT_RANK_R";
        case PIFA_ERR_NOT_SPD: return "PIFA_ERR_NOT_SPD";
        case PIFA_ERR_WRONG_DEVICE: return "PIFA_ERR_WRONG_DEVICE";
        case PIFA_ERR_TOO_LARGE: return "PIFA_ERR_TOO_LARGE";
    }
    return "PIFA_ERR_UNKNOWN";
}

pifa_status pifa_gemm_plan(int64_t M, int64_t N, int64_t K, int wide_epilogue, int64_t* tile_m,
                           int64_t* tile_n, int64_t* k_splits) {
    if (M < 1 || N < 1 || K < 1 || !tile_m || !tile_n || !k_splits) return PIFA_ERR_INVALID_ARG;
    const GemmPlan g = gemm_plan(M, N, K, wide_epilogue != 0, true);
    *tile_m = g.bm;
    *tile_n = g.bn;
    *k_splits = g.split.splits;
    return PIFA_OK;
}

pifa_status pifa_validate_partition(const int32_t* pivot_idx, const int32_t* nonpivot_idx,
                                    pifa_dims dims) {
    pifa_status s = check_dims(dims);
    if (s != PIFA_OK) return s;
    const int64_t n_np = dims.d_out - dims.r;
    if (!pivot_idx || (n_np > 0 && !nonpivot_idx)) return PIFA_ERR_INVALID_ARG;
    std::vector<uint8_t> seen((size_t)dims.d_out, 0);
    auto mark = [&](const int32_t* idx, int64_t n) {
        for (int64_t i = 0; i < n; ++i) {
            const int64_t v = idx[i];
            if (v < 0 || v >= dims.d_out || seen[(size_t)v]) return false;
            seen[(size_t)v] = 1;
        }
        return true;
    };
    if (!mark(pivot_idx, dims.r)) return PIFA_ERR_BAD_INDEX;
    if (n_np > 0 && !mark(nonpivot_idx, n_np)) return PIFA_ERR_BAD_INDEX;
    return PIFA_OK;  // d_out distinct in-range values: an exact partition
}

}  // extern "C"

namespace {

// The forward of Algorithm "PIFA Layer" with caller-chosen workspace: ws
// holds pifa_ws_bytes(h, M) bytes (the Y_p hand-off), part
// pifa_part_bytes(h, M) bytes (K-split partial products; may be null when
// that is 0).  Arguments are already validated.
pifa_status forward_with(pifa_layer* h, const void* X, void* Y, int64_t M, void* ws, float* part,
                         hipStream_t st) {
    hipError_t e;
    if (h->dtype == PIFA_F32) {
        float* yp = (float*)ws;
        e = launch_gemm_f32(kSitePifaF32Gemm1, (const float*)X, h->d_in, M, (const float*)h->Wp, h->d_in,
                            h->r, h->d_in,
                            make_epi<float, kWsF32>((float*)Y, h->d_out, h->piv, h->r, 1.f, yp, h->r,
                                                    h->r, 1.f, nullptr, M),
                            st);
        if (e != hipSuccess) return PIFA_ERR_HIP;
        if (h->n_np > 0) {
            e = launch_gemm_f32(kSitePifaF32Gemm2, yp, h->r, M, (const float*)h->C, h->r, h->n_np, h->r,
                                make_epi<float, kWsNone>((float*)Y, h->d_out, h->npiv, h->n_np, 1.f,
                                                         nullptr, 0, 0, 1.f, nullptr, M),
                                st);
            if (e != hipSuccess) return PIFA_ERR_HIP;
        }
        return PIFA_OK;
    }

    const float y_scale = std::ldexp(1.0f, h->y_log2);
    const float out_scale = std::ldexp(1.0f, -(h->y_log2 + h->c_log2));
    if (M <= kDecodeMaxM) {
        f16* yp = (f16*)ws;  // hi plane, then lo plane, M x r_pad each
        e = launch_skinny_packed<bf16>(kSitePifaGemv1, ALoad16<bf16>{(const bf16*)X, h->d_in, M},
                                       (const bf16*)h->Wp, h->r_pad, h->d_in,
                                       make_epi<bf16, kWsF16Pair>((bf16*)Y, h->d_out, h->piv, h->r, 1.f, yp,
                                                                  h->r_pad, h->r_pad, y_scale, h->overflow, M),
                                       st);
        if (e != hipSuccess) return PIFA_ERR_HIP;
        if (h->n_np > 0) {
            e = launch_skinny_packed<f16>(kSitePifaGemv2, ALoadPair16{yp, h->r_pad, M}, (const f16*)h->C, h->n_np,
                                          h->r_pad,
                                          make_epi<bf16, kWsNone>((bf16*)Y, h->d_out, h->npiv, h->n_np,
                                                                  out_scale, nullptr, 0, 0, 1.f, nullptr, M),
                                          st);
            if (e != hipSuccess) return PIFA_ERR_HIP;
        }
        return PIFA_OK;
    }

    f16* yp = (f16*)ws;
    // pivot outputs scattered to their columns; the hand-off (contiguous,
    // 16-byte rows) staged and written 16 bytes at a time
    PivotHandoffEpi pe;
    pe.y = make_epi<bf16, kWsNone>((bf16*)Y, h->d_out, h->piv, h->r, 1.f, nullptr, 0, 0, 1.f, nullptr, M);
    pe.ws = StagedEpi<f16>{(uint16_t*)yp, h->r_pad, h->r_pad, y_scale, h->overflow, M};
    e = launch_gemm<bf16, true>(kSitePifaGemm1, (const bf16*)X, h->d_in, M, (const bf16*)h->Wp, 0, h->r_pad,
                                h->d_in, pe, part, st);
    if (e != hipSuccess) return PIFA_ERR_HIP;
    if (h->n_np > 0) {
        e = launch_gemm<f16, true>(kSitePifaGemm2, yp, h->r_pad, M, (const f16*)h->C, 0, h->n_np, h->r_pad,
                                   make_epi<bf16, kWsNone>((bf16*)Y, h->d_out, h->npiv, h->n_np, out_scale,
                                                           nullptr, 0, 0, 1.f, nullptr, M),
                                   part, st);
        if (e != hipSuccess) return PIFA_ERR_HIP;
    }
    return PIFA_OK;
}

// Copy n host indices to a new device array, adding `offset` to each.
pifa_status upload_indices(const int32_t* src, int64_t n, int64_t offset, int32_t** dst) {
    std::vector<int32_t> tmp((size_t)n);
    for (int64_t i = 0; i < n; ++i) tmp[(size_t)i] = (int32_t)(src[i] + offset);
    if (hipMalloc(dst, (size_t)n * sizeof(int32_t)) != hipSuccess) return PIFA_ERR_OOM;
    PIFA_HIP(hipMemcpy(*dst, tmp.data(), (size_t)n * sizeof(int32_t), hipMemcpyHostToDevice));
    return PIFA_OK;
}

// pifa_layer_create with every output index shifted by out_offset (the
// layer's column offset inside a group's output; 0 for a plain layer).
pifa_status create_layer(const void* W_p, const void* C, const int32_t* pivot_idx,
                         const int32_t* nonpivot_idx, pifa_dims dims, pifa_dtype dtype, int64_t out_offset,
                         pifa_layer** out) {
    if (!out) return PIFA_ERR_INVALID_ARG;
    *out = nullptr;
    if (!valid_dtype(dtype)) return PIFA_ERR_INVALID_ARG;
    pifa_status s = check_dims(dims);
    if (s != PIFA_OK) return s;
    const int64_t n_np = dims.d_out - dims.r;
    if (!W_p || (n_np > 0 && !C)) return PIFA_ERR_INVALID_ARG;
    s = check_rows_aligned(dtype, dims.d_in);
    if (s != PIFA_OK) return s;
    s = pifa_validate_partition(pivot_idx, nonpivot_idx, dims);
    if (s != PIFA_OK) return s;

    pifa_layer* h = new (std::nothrow) pifa_layer();
    if (!h) return PIFA_ERR_OOM;
    h->dtype = dtype;
    h->d_in = dims.d_in;
    h->d_out = dims.d_out;
    h->r = dims.r;
    h->n_np = n_np;
    const bool bf = dtype == PIFA_BF16;
    h->r_pad = bf ? round_up(dims.r, kRowPad) : dims.r;

    auto fail = [&](pifa_status st) {
        free_layer(h);
        return st;
    };
    if (hipGetDevice(&h->device) != hipSuccess) return fail(PIFA_ERR_HIP);
    if (hipDeviceSynchronize() != hipSuccess) return fail(PIFA_ERR_HIP);

    const size_t wp_bytes = bf ? (size_t)packed_elems(h->r_pad, h->d_in) * 2 : (size_t)h->r * h->d_in * 4;
    if (hipMalloc(&h->Wp, wp_bytes) != hipSuccess) return fail(PIFA_ERR_OOM);
    if ((bf ? pack_lane_bf16(W_p, h->r, h->d_in, h->Wp, h->r_pad, h->d_in)
            : pack_rowmajor_f32(W_p, h->r, h->d_in, h->Wp, h->r, h->d_in)) != hipSuccess)
        return fail(PIFA_ERR_HIP);

    s = upload_indices(pivot_idx, h->r, out_offset, &h->piv);
    if (s != PIFA_OK) return fail(s);
    if (hipMalloc(&h->overflow, sizeof(int)) != hipSuccess) return fail(PIFA_ERR_OOM);
    if (hipMemset(h->overflow, 0, sizeof(int)) != hipSuccess) return fail(PIFA_ERR_HIP);

    if (n_np > 0) {
        s = upload_indices(nonpivot_idx, n_np, out_offset, &h->npiv);
        if (s != PIFA_OK) return fail(s);
        if (!bf) {
            if (hipMalloc(&h->C, (size_t)n_np * h->r * 4) != hipSuccess) return fail(PIFA_ERR_OOM);
            if (pack_rowmajor_f32(C, n_np, h->r, h->C, n_np, h->r) != hipSuccess) return fail(PIFA_ERR_HIP);
        } else {
            float mx = 0.f;
            s = absmax_bf16_host(C, n_np * h->r, &mx);
            if (s != PIFA_OK) return fail(s);
            // scale so that max|C| * 2^c_log2 lies in [2^14, 2^15)
            int c_log2 = 0;
            if (mx > 0.f) c_log2 = std::max(-30, std::min(30, 14 - (int)std::floor(std::log2((double)mx))));
            h->c_log2 = c_log2;
            const int64_t chunks = packed_groups(n_np) * packed_kblocks(h->r_pad) * kPackChunks;
            if (hipMalloc(&h->C, (size_t)chunks * 16) != hipSuccess) return fail(PIFA_ERR_OOM);
            hipLaunchKernelGGL((pack_lane_order<uint16_t, f16>), dim3(grid_for(chunks)), dim3(256), 0, 0,
                               (const uint16_t*)C, n_np, h->r, h->r, (f16*)h->C, n_np, h->r_pad,
                               std::ldexp(1.0f, c_log2));
            if (hipGetLastError() != hipSuccess) return fail(PIFA_ERR_HIP);
        }
    }
    if (hipDeviceSynchronize() != hipSuccess) return fail(PIFA_ERR_HIP);
    *out = h;
    return PIFA_OK;
}

}  // namespace

extern "C" {

pifa_status pifa_layer_create(const void* W_p, const void* C, const int32_t* pivot_idx,
                              const int32_t* nonpivot_idx, pifa_dims dims, pifa_dtype dtype,
                              pifa_handle* out) {
    return create_layer(W_p, C, pivot_idx, nonpivot_idx, dims, dtype, 0, out);
}

pifa_status pifa_layer_destroy(pifa_handle h) {
    if (!h) return PIFA_OK;
    (void)hipDeviceSynchronize();
    free_layer(h);
    return PIFA_OK;
}

pifa_status pifa_layer_reserve(pifa_handle h, int64_t max_M) {
    if (!h || max_M < 0) return PIFA_ERR_INVALID_ARG;
    PIFA_ON_DEVICE(h->device);
    const size_t need = std::max(pifa_ws_bytes(h, max_M), pifa_ws_bytes(h, std::min<int64_t>(max_M, kDecodeMaxM)));
    pifa_status s = h->ws.ensure(need, 0);
    if (s != PIFA_OK) return s;
    // the split partials of every M up to max_M (they are not monotone in M)
    size_t part = 0;
    for (int64_t m = kDecodeMaxM + 1; m <= std::min(max_M, kSplitMaxM); ++m)
        part = std::max(part, pifa_part_bytes(h, m));
    s = h->part.ensure(part, 0);
    if (s != PIFA_OK) return s;
    return hipDeviceSynchronize() == hipSuccess ? PIFA_OK : PIFA_ERR_HIP;
}

size_t pifa_layer_weight_bytes(pifa_handle h) {
    if (!h) return 0;
    const size_t es = esize(h->dtype);
    return (size_t)(h->r * h->d_in + h->n_np * h->r) * es + (size_t)h->d_out * sizeof(int32_t);
}

pifa_status pifa_layer_set_intermediate_scale(pifa_handle h, int log2_scale) {
    if (!h || log2_scale < -30 || log2_scale > 30) return PIFA_ERR_INVALID_ARG;
    h->y_log2 = log2_scale;
    return PIFA_OK;
}

pifa_status pifa_layer_overflow_count(pifa_handle h, int64_t* count) {
    if (!h || !count) return PIFA_ERR_INVALID_ARG;
    int v = 0;
    PIFA_HIP(hipDeviceSynchronize());
    PIFA_HIP(hipMemcpy(&v, h->overflow, sizeof(int), hipMemcpyDeviceToHost));
    *count = v;
    return PIFA_OK;
}

pifa_status pifa_forward(pifa_handle h, const void* X, void* Y, int64_t M, void* stream) {
    if (!h || M < 0) return PIFA_ERR_INVALID_ARG;
    if (M == 0) return PIFA_OK;
    if (!X || !Y) return PIFA_ERR_INVALID_ARG;
    PIFA_ON_DEVICE(h->device);
    if (h->dtype == PIFA_BF16 && !aligned16(X)) return PIFA_ERR_UNSUPPORTED;
    hipStream_t st = as_stream(stream);
    pifa_status s = h->ws.ensure(pifa_ws_bytes(h, M), st);
    if (s != PIFA_OK) return s;
    s = h->part.ensure(pifa_part_bytes(h, M), st);
    if (s != PIFA_OK) return s;
    return forward_with(h, X, Y, M, h->ws.ptr, (float*)h->part.ptr, st);
}

pifa_status dense_forward(const void* W, const void* X, void* Y, int64_t M, int64_t d_in,
                          int64_t d_out, pifa_dtype dtype, void* stream) {
    if (!valid_dtype(dtype) || M < 0 || d_in < 1 || d_out < 1) return PIFA_ERR_INVALID_ARG;
    if (M == 0) return PIFA_OK;
    if (!W || !X || !Y) return PIFA_ERR_INVALID_ARG;
    pifa_status s = check_rows_aligned(dtype, d_in);
    if (s != PIFA_OK) return s;
    if (dtype == PIFA_BF16 && (!aligned16(X) || !aligned16(W))) return PIFA_ERR_UNSUPPORTED;
    hipStream_t st = as_stream(stream);
    int dev = 0;
    PIFA_HIP(hipGetDevice(&dev));
    DeviceScratch& ds = device_scratch(dev);
    std::lock_guard<std::mutex> g(ds.mu);
    s = ds.part.ensure(dense_part_bytes(dtype, M, d_in, d_out), st, true);
    if (s != PIFA_OK) return s;
    return dense_run<false>(dtype, W, X, Y, M, d_in, d_out, (float*)ds.part.ptr, st);
}

pifa_status dense_layer_create(const void* W, int64_t d_in, int64_t d_out, pifa_dtype dtype,
                               dense_handle* out) {
    if (!out) return PIFA_ERR_INVALID_ARG;
    *out = nullptr;
    if (!valid_dtype(dtype) || d_in < 1 || d_out < 1 || !W) return PIFA_ERR_INVALID_ARG;
    if (d_in > INT32_MAX || d_out > INT32_MAX) return PIFA_ERR_UNSUPPORTED;
    pifa_status s = check_rows_aligned(dtype, d_in);
    if (s != PIFA_OK) return s;
    dense_layer* h = new (std::nothrow) dense_layer();
    if (!h) return PIFA_ERR_OOM;
    h->dtype = dtype;
    h->d_in = d_in;
    h->d_out = d_out;
    auto fail = [&](pifa_status st) {
        free_dense(h);
        return st;
    };
    if (hipGetDevice(&h->device) != hipSuccess) return fail(PIFA_ERR_HIP);
    if (hipDeviceSynchronize() != hipSuccess) return fail(PIFA_ERR_HIP);
    const bool bf = dtype == PIFA_BF16;
    const size_t bytes = bf ? (size_t)packed_elems(d_out, d_in) * 2 : (size_t)d_out * d_in * 4;
    if (hipMalloc(&h->W, bytes) != hipSuccess) return fail(PIFA_ERR_OOM);
    if ((bf ? pack_lane_bf16(W, d_out, d_in, h->W, d_out, d_in)
            : pack_rowmajor_f32(W, d_out, d_in, h->W, d_out, d_in)) != hipSuccess)
        return fail(PIFA_ERR_HIP);
    if (hipDeviceSynchronize() != hipSuccess) return fail(PIFA_ERR_HIP);
    *out = h;
    return PIFA_OK;
}

pifa_status dense_layer_forward(dense_handle h, const void* X, void* Y, int64_t M, void* stream) {
    if (!h || M < 0) return PIFA_ERR_INVALID_ARG;
    if (M == 0) return PIFA_OK;
    if (!X || !Y) return PIFA_ERR_INVALID_ARG;
    PIFA_ON_DEVICE(h->device);
    if (h->dtype == PIFA_BF16 && !aligned16(X)) return PIFA_ERR_UNSUPPORTED;
    hipStream_t st = as_stream(stream);
    pifa_status s = h->part.ensure(dense_part_bytes(h->dtype, M, h->d_in, h->d_out), st);
    if (s != PIFA_OK) return s;
    if (h->dtype == PIFA_BF16)
        return dense_run<true>(h->dtype, h->W, X, Y, M, h->d_in, h->d_out, (float*)h->part.ptr, st);
    return dense_run<false>(h->dtype, h->W, X, Y, M, h->d_in, h->d_out, nullptr, st);
}

pifa_status dense_layer_reserve(dense_handle h, int64_t max_M) {
    if (!h || max_M < 0) return PIFA_ERR_INVALID_ARG;
    PIFA_ON_DEVICE(h->device);
    size_t part = 0;
    for (int64_t m = kDecodeMaxM + 1; m <= std::min(max_M, kSplitMaxM); ++m)
        part = std::max(part, dense_part_bytes(h->dtype, m, h->d_in, h->d_out));
    pifa_status s = h->part.ensure(part, 0);
    if (s != PIFA_OK) return s;
    return hipDeviceSynchronize() == hipSuccess ? PIFA_OK : PIFA_ERR_HIP;
}

pifa_status dense_layer_destroy(dense_handle h) {
    if (!h) return PIFA_OK;
    (void)hipDeviceSynchronize();
    free_dense(h);
    return PIFA_OK;
}

pifa_status lowrank_uv_forward(const void* U, const void* V, const void* X, void* Y, int64_t M,
                               pifa_dims dims, pifa_dtype dtype, void* stream) {
    if (!valid_dtype(dtype) || M < 0) return PIFA_ERR_INVALID_ARG;
    pifa_status s = check_dims(dims);
    if (s != PIFA_OK) return s;
    if (M == 0) return PIFA_OK;
    if (!U || !V || !X || !Y) return PIFA_ERR_INVALID_ARG;
    s = check_rows_aligned(dtype, dims.d_in);
    if (s != PIFA_OK) return s;
    if (dtype == PIFA_BF16 && (dims.r % 8 != 0 || !aligned16(X) || !aligned16(U) || !aligned16(V)))
        return PIFA_ERR_UNSUPPORTED;
    hipStream_t st = as_stream(stream);
    int dev = 0;
    PIFA_HIP(hipGetDevice(&dev));
    DeviceScratch& ds = device_scratch(dev);
    std::lock_guard<std::mutex> g(ds.mu);
    s = ds.inter.ensure(lowrank_ws_bytes(dtype, M, dims.r), st, true);
    if (s == PIFA_OK) s = ds.part.ensure(lowrank_part_bytes(dtype, M, dims.d_in, dims.d_out, dims.r), st, true);
    if (s != PIFA_OK) return s;
    return lowrank_run<false>(dtype, U, V, X, Y, M, dims.d_in, dims.d_out, dims.r, ds.inter.ptr,
                              (float*)ds.part.ptr, st);
}

pifa_status lowrank_layer_create(const void* U, const void* V, pifa_dims dims, pifa_dtype dtype,
                                 lowrank_handle* out) {
    if (!out) return PIFA_ERR_INVALID_ARG;
    *out = nullptr;
    if (!valid_dtype(dtype)) return PIFA_ERR_INVALID_ARG;
    pifa_status s = check_dims(dims);
    if (s != PIFA_OK) return s;
    if (!U || !V) return PIFA_ERR_INVALID_ARG;
    s = check_rows_aligned(dtype, dims.d_in);
    if (s != PIFA_OK) return s;
    lowrank_layer* h = new (std::nothrow) lowrank_layer();
    if (!h) return PIFA_ERR_OOM;
    h->dtype = dtype;
    h->d_in = dims.d_in;
    h->d_out = dims.d_out;
    h->r = dims.r;
    const bool bf = dtype == PIFA_BF16;
    h->r_pad = bf ? round_up(dims.r, kRowPad) : dims.r;
    auto fail = [&](pifa_status st) {
        free_lowrank(h);
        return st;
    };
    if (hipGetDevice(&h->device) != hipSuccess) return fail(PIFA_ERR_HIP);
    if (hipDeviceSynchronize() != hipSuccess) return fail(PIFA_ERR_HIP);
    if (bf) {
        if (hipMalloc(&h->U, (size_t)packed_elems(h->d_out, h->r_pad) * 2) != hipSuccess ||
            hipMalloc(&h->V, (size_t)packed_elems(h->r_pad, h->d_in) * 2) != hipSuccess)
            return fail(PIFA_ERR_OOM);
        if (pack_lane_bf16(U, h->d_out, h->r, h->U, h->d_out, h->r_pad) != hipSuccess ||
            pack_lane_bf16(V, h->r, h->d_in, h->V, h->r_pad, h->d_in) != hipSuccess)
            return fail(PIFA_ERR_HIP);
    } else {
        if (hipMalloc(&h->U, (size_t)h->d_out * h->r * 4) != hipSuccess ||
            hipMalloc(&h->V, (size_t)h->r * h->d_in * 4) != hipSuccess)
            return fail(PIFA_ERR_OOM);
        if (pack_rowmajor_f32(U, h->d_out, h->r, h->U, h->d_out, h->r) != hipSuccess ||
            pack_rowmajor_f32(V, h->r, h->d_in, h->V, h->r, h->d_in) != hipSuccess)
            return fail(PIFA_ERR_HIP);
    }
    if (hipDeviceSynchronize() != hipSuccess) return fail(PIFA_ERR_HIP);
    *out = h;
    return PIFA_OK;
}

pifa_status lowrank_layer_reserve(lowrank_handle h, int64_t max_M) {
    if (!h || max_M < 0) return PIFA_ERR_INVALID_ARG;
    PIFA_ON_DEVICE(h->device);
    const size_t need = std::max(lowrank_ws_bytes(h->dtype, max_M, h->r_pad),
                                 lowrank_ws_bytes(h->dtype, std::min<int64_t>(max_M, kDecodeMaxM), h->r_pad));
    pifa_status s = h->ws.ensure(need, 0);
    if (s != PIFA_OK) return s;
    size_t part = 0;
    for (int64_t m = kDecodeMaxM + 1; m <= std::min(max_M, kSplitMaxM); ++m)
        part = std::max(part, lowrank_part_bytes(h->dtype, m, h->d_in, h->d_out, h->r_pad));
    s = h->part.ensure(part, 0);
    if (s != PIFA_OK) return s;
    return hipDeviceSynchronize() == hipSuccess ? PIFA_OK : PIFA_ERR_HIP;
}

pifa_status lowrank_layer_forward(lowrank_handle h, const void* X, void* Y, int64_t M, void* stream) {
    if (!h || M < 0) return PIFA_ERR_INVALID_ARG;
    if (M == 0) return PIFA_OK;
    if (!X || !Y) return PIFA_ERR_INVALID_ARG;
    PIFA_ON_DEVICE(h->device);
    if (h->dtype == PIFA_BF16 && !aligned16(X)) return PIFA_ERR_UNSUPPORTED;
    hipStream_t st = as_stream(stream);
    pifa_status s = h->ws.ensure(lowrank_ws_bytes(h->dtype, M, h->r_pad), st);
    if (s == PIFA_OK) s = h->part.ensure(lowrank_part_bytes(h->dtype, M, h->d_in, h->d_out, h->r_pad), st);
    if (s != PIFA_OK) return s;
    if (h->dtype == PIFA_BF16)
        return lowrank_run<true>(h->dtype, h->U, h->V, X, Y, M, h->d_in, h->d_out, h->r_pad, h->ws.ptr,
                                 (float*)h->part.ptr, st);
    return lowrank_run<false>(h->dtype, h->U, h->V, X, Y, M, h->d_in, h->d_out, h->r, h->ws.ptr, nullptr, st);
}

pifa_status lowrank_layer_destroy(lowrank_handle h) {
    if (!h) return PIFA_OK;
    (void)hipDeviceSynchronize();
    free_lowrank(h);
    return PIFA_OK;
}

}  // extern "C"

// ===================================================================== backward
namespace {

inline int64_t align_elems(int64_t n) { return round_up(n, (int64_t)128); }  // 256-byte regions

// Transposed weight copies for the backward products (once per layer).
pifa_status prepare_backward(pifa_layer* h) {
    if (h->bwd_wpt) return PIFA_OK;
    const int64_t ldc = round_up(h->n_np, (int64_t)8);
    float mx = 0.f;
    pifa_status s = absmax_bf16_host(h->Wp, packed_elems(h->r_pad, h->d_in), &mx);
    if (s != PIFA_OK) return s;
    // scale so that max|W_p| * 2^cw lies in [2^14, 2^15), as for C
    const int cw = mx > 0.f ? std::max(-30, std::min(30, 14 - (int)std::floor(std::log2((double)mx)))) : 0;
    void* wpt = nullptr;
    void* ct = nullptr;
    if (hipMalloc(&wpt, (size_t)packed_elems(h->d_in, h->r_pad) * 2) != hipSuccess) return PIFA_ERR_OOM;
    if (h->n_np > 0 && hipMalloc(&ct, (size_t)packed_elems(h->r_pad, ldc) * 2) != hipSuccess) {
        (void)hipFree(wpt);
        return PIFA_ERR_OOM;
    }
    const int64_t c1 = packed_groups(h->d_in) * packed_kblocks(h->r_pad) * kPackChunks;
    hipLaunchKernelGGL((pack_transposed<bf16, f16>), dim3(grid_for(c1)), dim3(256), 0, 0, (const bf16*)h->Wp,
                       packed_kblocks(h->d_in), h->r, h->d_in, h->r_pad, std::ldexp(1.0f, cw), (f16*)wpt, h->d_in,
                       h->r_pad);
    bool ok = hipGetLastError() == hipSuccess;
    if (ok && ct) {
        const int64_t c2 = packed_groups(h->r_pad) * packed_kblocks(ldc) * kPackChunks;
        hipLaunchKernelGGL((pack_transposed<f16, bf16>), dim3(grid_for(c2)), dim3(256), 0, 0, (const f16*)h->C,
                           packed_kblocks(h->r_pad), h->n_np, h->r, ldc, std::ldexp(1.0f, -h->c_log2), (bf16*)ct,
                           h->r_pad, ldc);
        ok = hipGetLastError() == hipSuccess;
    }
    ok = ok && hipDeviceSynchronize() == hipSuccess;
    if (!ok) {
        (void)hipFree(wpt);
        if (ct) (void)hipFree(ct);
        return PIFA_ERR_HIP;
    }
    h->bwd_wpt = wpt;
    h->bwd_ct = ct;
    h->bwd_cw = cw;
    return PIFA_OK;
}

// gather_tile over all of in's needed tiles (see backward.hpp).
hipError_t launch_gather(const bf16* in, int64_t ld_in, int64_t M, const int32_t* idx, int64_t ncols, bf16* out_r,
                         int64_t ld_r, bf16* out_t, int64_t ld_t, hipStream_t st) {
    const int64_t mx = std::max(M, out_t ? ld_t : (int64_t)0);
    const int64_t nx = std::max(ncols, out_r ? ld_r : (int64_t)0);
    if (mx == 0 || nx == 0) return hipSuccess;
    hipLaunchKernelGGL(gather_tile, dim3((unsigned)ceil_div(mx, kTrTile), (unsigned)ceil_div(nx, kTrTile)), dim3(256),
                       0, st, in, ld_in, M, idx, ncols, out_r, ld_r, out_t, ld_t);
    return hipGetLastError();
}

}  // namespace

extern "C" {

pifa_status pifa_layer_backward(pifa_handle h, const void* X, const void* Y, const void* dY, int64_t M,
                                void* dX, float* dW_p, float* dC, void* stream) {
    if (!h || M < 0) return PIFA_ERR_INVALID_ARG;
    if (h->dtype != PIFA_BF16) return PIFA_ERR_UNSUPPORTED;
    PIFA_ON_DEVICE(h->device);
    hipStream_t st = as_stream(stream);
    const int64_t r = h->r, n_np = h->n_np, d_in = h->d_in, d_out = h->d_out, r_pad = h->r_pad;
    if (M == 0) {  // the gradient of an empty batch
        if (dW_p) PIFA_HIP(hipMemsetAsync(dW_p, 0, (size_t)r * d_in * 4, st));
        if (dC && n_np > 0) PIFA_HIP(hipMemsetAsync(dC, 0, (size_t)n_np * r * 4, st));
        return PIFA_OK;
    }
    if (!dY || (dX == nullptr && dW_p == nullptr && dC == nullptr)) return dY ? PIFA_OK : PIFA_ERR_INVALID_ARG;
    if ((dW_p && !X) || (dC && n_np > 0 && !Y)) return PIFA_ERR_INVALID_ARG;
    pifa_status s = prepare_backward(h);
    if (s != PIFA_OK) return s;

    const int64_t ldc = round_up(n_np, (int64_t)8), ldy = round_up(r, (int64_t)8);
    // workspace regions, in 2-byte elements (each a multiple of 256 bytes)
    const int64_t e_gic = align_elems(M * ldc), e_ypr = align_elems(M * ldy), e_gp32 = align_elems(2 * M * r_pad),
                  e_gp16 = align_elems(M * r_pad), e_inv = align_elems(2 * M), e_gpb = align_elems(M * r_pad);
    const size_t part = std::max({split_bytes(M, r_pad, ldc), split_bytes(M, d_in, r_pad), split_bytes(r, d_in, M),
                                  split_bytes(n_np, r, M)});
    const size_t main_bytes = (size_t)(e_gic + e_ypr + e_gp32 + e_gp16 + e_inv + e_gpb) * 2;
    s = h->bws.ensure(main_bytes + part, st);
    if (s != PIFA_OK) return s;
    bf16* gic = (bf16*)h->bws.ptr;
    bf16* ypr = gic + e_gic;
    float* gp32 = (float*)(ypr + e_ypr);
    f16* gp16 = (f16*)(ypr + e_ypr + e_gp32);
    float* inv = (float*)(ypr + e_ypr + e_gp32 + e_gp16);
    bf16* gpb = ypr + e_ypr + e_gp32 + e_gp16 + e_inv;
    float* partials = part ? (float*)((char*)h->bws.ptr + main_bytes) : nullptr;
    const bf16* G = (const bf16*)dY;
    hipError_t e = hipSuccess;

    {  // the gathered columns G[:, I^c] and Y[:, I] as rows
        TimedLaunch timed(kSiteBwdData, st);
        if (n_np > 0 && (e = launch_gather(G, d_out, M, h->npiv, n_np, gic, ldc, nullptr, 0, st)) != hipSuccess)
            return PIFA_ERR_HIP;
        if (n_np > 0 && dC &&
            (e = launch_gather((const bf16*)Y, d_out, M, h->piv, r, ypr, ldy, nullptr, 0, st)) != hipSuccess)
            return PIFA_ERR_HIP;
    }
    // G_p = G[:, I^c] C + G[:, I] in fp32, and bf16(G_p)
    e = launch_gemm<bf16, true>(kSiteBwdGp, gic, ldc, M, (const bf16*)h->bwd_ct, 0, r_pad, ldc,
                                GradPivotEpi{G, d_out, h->piv, r, r_pad, gp32, gpb, M}, partials, st);
    if (e != hipSuccess) return PIFA_ERR_HIP;
    if (dX) {  // dX = (G_p 2^s_m in fp16) (W_p^T 2^cw in fp16)^T 2^-(s_m + cw)
        {
            TimedLaunch timed(kSiteBwdRows, st);
            hipLaunchKernelGGL(rows_to_f16, dim3((unsigned)M), dim3(256), 0, st, gp32, r_pad, gp16, inv);
            if (hipGetLastError() != hipSuccess) return PIFA_ERR_HIP;
        }
        e = launch_gemm<f16, true>(kSiteBwdDx, gp16, r_pad, M, (const f16*)h->bwd_wpt, 0, d_in, r_pad,
                                   RowScaleEpi{(bf16*)dX, d_in, d_in, inv, std::ldexp(1.0f, -h->bwd_cw), M}, partials,
                                   st);
        if (e != hipSuccess) return PIFA_ERR_HIP;
    }
    // the transposed products reduce over the M activation rows: both
    // operands are read K-major (rows of G_p, X, G[:, I^c], Y[:, I])
    if (dW_p) {  // dW_p = G_p^T X
        e = launch_gemm<bf16, false, ScatterEpi<float, kWsNone>, 3>(
            kSiteBwdDwp, gpb, r_pad, r, (const bf16*)X, d_in, d_in, M,
            make_epi<float, kWsNone>(dW_p, d_in, nullptr, d_in, 1.f, nullptr, 0, 0, 1.f, nullptr, r), partials, st);
        if (e != hipSuccess) return PIFA_ERR_HIP;
    }
    if (dC && n_np > 0) {  // dC = G[:, I^c]^T Y_p
        e = launch_gemm<bf16, false, ScatterEpi<float, kWsNone>, 3>(
            kSiteBwdDc, gic, ldc, n_np, ypr, ldy, r, M,
            make_epi<float, kWsNone>(dC, r, nullptr, r, 1.f, nullptr, 0, 0, 1.f, nullptr, n_np), partials, st);
        if (e != hipSuccess) return PIFA_ERR_HIP;
    }
    return PIFA_OK;
}

}  // extern "C"

// ===================================================================== reconstruction
struct pifa_calib {
    int device = 0;
    int64_t n = 0;
    double* S = nullptr;  // sum x_u x_u^T
    double* P = nullptr;  // sum x_o x_u^T
    int* info = nullptr;  // Cholesky status
    GrowBuf ws;           // transposed batches and split partials
    GrowBuf work;         // reconstruction operands
};

namespace {

hipError_t gemm64_launch(hipStream_t st, int64_t Mr, int64_t Nc, int64_t K, double alpha, const double* A, int64_t sa0,
                         int64_t sa1, const double* B, int64_t sb0, int64_t sb1, double beta, double* C, int64_t sc0,
                         int64_t sc1, bool lower = false) {
    if (Mr <= 0 || Nc <= 0) return hipSuccess;
    // 128 x 128 tiles when they fill the chip and K is deep (about 60
    // TFLOP/s on the 4096-sized products, against 55 with 64 x 64 tiles);
    // 64 x 64 tiles otherwise, e.g. the blocked updates with K = 64
    if (!lower && K >= 512 && ceil_div(Mr, (int64_t)128) * ceil_div(Nc, (int64_t)128) >= kCus)
        hipLaunchKernelGGL((gemm64<128, 8>), dim3((unsigned)ceil_div(Nc, (int64_t)128), (unsigned)ceil_div(Mr, (int64_t)128)),
                           dim3(1024), 0, st, Mr, Nc, K, alpha, A, sa0, sa1, B, sb0, sb1, beta, C, sc0, sc1, 0);
    else
        hipLaunchKernelGGL((gemm64<64, 16>), dim3((unsigned)ceil_div(Nc, (int64_t)64), (unsigned)ceil_div(Mr, (int64_t)64)),
                           dim3(1024), 0, st, Mr, Nc, K, alpha, A, sa0, sa1, B, sb0, sb1, beta, C, sc0, sc1,
                           lower ? 1 : 0);
    return hipGetLastError();
}

// In-place lower Cholesky of the n x n matrix A (row stride ld); *info set on
// failure.  floor: one device double of scratch for the pivot threshold.
hipError_t cholesky64(double* A, int64_t n, int64_t ld, double* floor, int* info, hipStream_t st) {
    hipLaunchKernelGGL(pivot_floor64, dim3(1), dim3(256), 0, st, (const double*)A, n, ld, floor);
    for (int64_t kb = 0; kb < n; kb += kG64) {
        const int nb = (int)std::min<int64_t>(kG64, n - kb);
        double* Akk = A + kb * ld + kb;
        hipLaunchKernelGGL(chol_diag, dim3(1), dim3(256), 0, st, Akk, ld, nb, (const double*)floor, info);
        const int64_t rest = n - kb - nb;
        if (rest > 0) {
            double* L21 = A + (kb + nb) * ld + kb;
            // rest > 0: this block is a full one (nb == 64)
            hipLaunchKernelGGL(chol_panel, dim3((unsigned)ceil_div(rest, (int64_t)64)), dim3(64), 0, st, Akk, L21, ld,
                               rest);
            hipError_t e = gemm64_launch(st, rest, rest, nb, -1.0, L21, ld, 1, L21, 1, ld, 1.0,
                                         A + (kb + nb) * ld + kb + nb, ld, 1, true);
            if (e != hipSuccess) return e;
        }
    }
    return hipGetLastError();
}

// B (n x nrhs, row stride ldb) <- (L L^T)^-1 B for the lower factor L (row
// stride ld).  Linv: ceil(n / 64) * 64 * 64 doubles of scratch for the
// inverted diagonal blocks; X: n * nrhs doubles of scratch (row stride nrhs).
// Forward, L Y = B into X: Y_k = L_kk^-1 B_k, then the rows below lose
// L_ik Y_k.  Backward, L^T Z = Y into B: Z_k = L_kk^-T Y_k, then the rows
// above lose L_ki^T Z_k.  Multiplying by the inverted 64 x 64 blocks instead
// of substituting keeps every step on the MFMA GEMM; the blocks of a
// Cholesky factor of a matrix with condition number kappa have condition
// numbers of at most sqrt(kappa), which bounds what the explicit inverses add
// to the substitution's rounding error.
hipError_t spd_solve64(const double* L, int64_t n, int64_t ld, double* B, int64_t nrhs, int64_t ldb, double* Linv,
                       double* X, hipStream_t st) {
    const int64_t nblk = ceil_div(n, (int64_t)kG64);
    hipLaunchKernelGGL(tri_inv_blocks, dim3((unsigned)nblk), dim3(64), 0, st, L, ld, n, Linv);
    hipError_t e = hipGetLastError();
    for (int64_t kb = 0; kb < n && e == hipSuccess; kb += kG64) {
        const int64_t nb = std::min<int64_t>(kG64, n - kb), rest = n - kb - nb;
        const double* Li = Linv + (kb / kG64) * kG64 * kG64;
        e = gemm64_launch(st, nb, nrhs, nb, 1.0, Li, kG64, 1, B + kb * ldb, ldb, 1, 0.0, X + kb * nrhs, nrhs, 1);
        if (e == hipSuccess)
            e = gemm64_launch(st, rest, nrhs, nb, -1.0, L + (kb + nb) * ld + kb, ld, 1, X + kb * nrhs, nrhs, 1, 1.0,
                              B + (kb + nb) * ldb, ldb, 1);
    }
    for (int64_t kb = (nblk - 1) * kG64; kb >= 0 && e == hipSuccess; kb -= kG64) {
        const int64_t nb = std::min<int64_t>(kG64, n - kb);
        const double* Li = Linv + (kb / kG64) * kG64 * kG64;
        e = gemm64_launch(st, nb, nrhs, nb, 1.0, Li, 1, kG64, X + kb * nrhs, nrhs, 1, 0.0, B + kb * ldb, ldb, 1);
        if (e == hipSuccess)
            e = gemm64_launch(st, kb, nrhs, nb, -1.0, L + kb * ld, 1, ld, B + kb * ldb, ldb, 1, 1.0, X, nrhs, 1);
    }
    return e;
}

hipError_t transpose64_launch(const double* in, int64_t rows, int64_t cols, double* out, hipStream_t st) {
    if (rows == 0 || cols == 0) return hipSuccess;
    hipLaunchKernelGGL(transpose64, dim3((unsigned)ceil_div(cols, (int64_t)32), (unsigned)ceil_div(rows, (int64_t)32)),
                       dim3(256), 0, st, in, rows, cols, out);
    return hipGetLastError();
}

void free_calib(pifa_calib* c) {
    if (!c) return;
    if (c->S) (void)hipFree(c->S);
    if (c->P) (void)hipFree(c->P);
    if (c->info) (void)hipFree(c->info);
    c->ws.release();
    c->work.release();
    delete c;
}

}  // namespace

extern "C" {

pifa_status pifa_calib_create(int64_t d_in, pifa_calib_handle* out) {
    if (!out) return PIFA_ERR_INVALID_ARG;
    *out = nullptr;
    if (d_in < 1) return PIFA_ERR_INVALID_ARG;
    if (d_in > 65536) return PIFA_ERR_UNSUPPORTED;
    pifa_calib* c = new (std::nothrow) pifa_calib();
    if (!c) return PIFA_ERR_OOM;
    c->n = d_in;
    const size_t b = (size_t)d_in * d_in * sizeof(double);
    if (hipGetDevice(&c->device) != hipSuccess) { free_calib(c); return PIFA_ERR_HIP; }
    if (hipMalloc(&c->S, b) != hipSuccess || hipMalloc(&c->P, b) != hipSuccess ||
        hipMalloc(&c->info, sizeof(int)) != hipSuccess) {
        free_calib(c);
        return PIFA_ERR_OOM;
    }
    if (hipMemset(c->S, 0, b) != hipSuccess || hipMemset(c->P, 0, b) != hipSuccess ||
        hipDeviceSynchronize() != hipSuccess) {
        free_calib(c);
        return PIFA_ERR_HIP;
    }
    *out = c;
    return PIFA_OK;
}

pifa_status pifa_calib_destroy(pifa_calib_handle c) {
    if (!c) return PIFA_OK;
    (void)hipDeviceSynchronize();
    free_calib(c);
    return PIFA_OK;
}

pifa_status pifa_calib_reset(pifa_calib_handle c, void* stream) {
    if (!c) return PIFA_ERR_INVALID_ARG;
    PIFA_ON_DEVICE(c->device);
    const size_t b = (size_t)c->n * c->n * sizeof(double);
    PIFA_HIP(hipMemsetAsync(c->S, 0, b, as_stream(stream)));
    PIFA_HIP(hipMemsetAsync(c->P, 0, b, as_stream(stream)));
    return PIFA_OK;
}

pifa_status pifa_calib_accumulate(pifa_calib_handle c, const void* X_o, const void* X_u, int64_t B, void* stream) {
    if (!c || B < 0) return PIFA_ERR_INVALID_ARG;
    if (B == 0) return PIFA_OK;
    if (!X_o || !X_u) return PIFA_ERR_INVALID_ARG;
    PIFA_ON_DEVICE(c->device);
    hipStream_t st = as_stream(stream);
    const int64_t n = c->n, Bp = round_up(B, (int64_t)8);
    if (n % 8 == 0 && aligned16(X_o) && aligned16(X_u)) {
        // the batches' rows are the products' K-major operands (K = tokens)
        const size_t part = split_bytes(n, n, B);
        pifa_status s = c->ws.ensure(part, st);
        if (s != PIFA_OK) return s;
        float* partials = part ? (float*)c->ws.ptr : nullptr;
        const bf16* xu = (const bf16*)X_u;
        const bf16* xo = (const bf16*)X_o;
        // S is symmetric: only its lower tiles are accumulated (completed on read)
        if (launch_gemm<bf16, false, AccF64Epi, 3>(kSiteCalibGram, xu, n, n, xu, n, n, B,
                                                   AccF64Epi{c->S, n, n, n, true}, partials, st) != hipSuccess)
            return PIFA_ERR_HIP;
        if (launch_gemm<bf16, false, AccF64Epi, 3>(kSiteCalibGram, xo, n, n, xu, n, n, B,
                                                   AccF64Epi{c->P, n, n, n, false}, partials, st) != hipSuccess)
            return PIFA_ERR_HIP;
        return PIFA_OK;
    }
    // unaligned rows: transposed copies of the batches, then K-contiguous products
    const int64_t e_t = align_elems(n * Bp);
    const size_t part = split_bytes(n, n, Bp);
    pifa_status s = c->ws.ensure((size_t)(2 * e_t) * 2 + part, st);
    if (s != PIFA_OK) return s;
    bf16* xut = (bf16*)c->ws.ptr;
    bf16* xot = xut + e_t;
    float* partials = part ? (float*)((char*)c->ws.ptr + (size_t)(2 * e_t) * 2) : nullptr;
    {
        TimedLaunch timed(kSiteCalibGather, st);
        if (launch_gather((const bf16*)X_u, n, B, nullptr, n, nullptr, 0, xut, Bp, st) != hipSuccess) return PIFA_ERR_HIP;
        if (X_o != X_u &&
            launch_gather((const bf16*)X_o, n, B, nullptr, n, nullptr, 0, xot, Bp, st) != hipSuccess)
            return PIFA_ERR_HIP;
    }
    const bf16* xo = X_o == X_u ? xut : xot;
    // S += X_u^T X_u and P += X_o^T X_u: rows of the transposed batches, K = tokens
    // S is symmetric: only its lower tiles are accumulated (completed on read)
    if (launch_gemm<bf16, false>(kSiteCalibGram, xut, Bp, n, xut, Bp, n, Bp, AccF64Epi{c->S, n, n, n, true}, partials,
                                 st) != hipSuccess)
        return PIFA_ERR_HIP;
    if (launch_gemm<bf16, false>(kSiteCalibGram, xo, Bp, n, xut, Bp, n, Bp, AccF64Epi{c->P, n, n, n, false}, partials,
                                 st) != hipSuccess)
        return PIFA_ERR_HIP;
    return PIFA_OK;
}

pifa_status pifa_calib_read(pifa_calib_handle c, double* S, double* P, void* stream) {
    if (!c) return PIFA_ERR_INVALID_ARG;
    PIFA_ON_DEVICE(c->device);
    const size_t b = (size_t)c->n * c->n * sizeof(double);
    if (S) {
        hipLaunchKernelGGL(symmetrize_lower64, dim3(grid_for(c->n * c->n)), dim3(256), 0, as_stream(stream), c->S, c->n);
        PIFA_HIP(hipGetLastError());
    }
    if (S) PIFA_HIP(hipMemcpyAsync(S, c->S, b, hipMemcpyDeviceToDevice, as_stream(stream)));
    if (P) PIFA_HIP(hipMemcpyAsync(P, c->P, b, hipMemcpyDeviceToDevice, as_stream(stream)));
    return PIFA_OK;
}

pifa_status pifa_calib_reconstruct(pifa_calib_handle c, const double* W, int64_t d_out, const double* Vt, int64_t r,
                                   double lam, double alpha, double* U_r, double* Vt_r, void* stream) {
    if (!c || !W || !Vt || !U_r || !Vt_r || d_out < 1 || r < 1) return PIFA_ERR_INVALID_ARG;
    PIFA_ON_DEVICE(c->device);
    const int64_t n = c->n, m = d_out;
    if (r > n || r > m) return PIFA_ERR_INVALID_ARG;
    hipStream_t st = as_stream(stream);
    // work regions (fp64 elements, 32-element aligned)
    auto al = [](int64_t e) { return round_up(e, (int64_t)32); };
    const int64_t e_Z = al(n * n), e_T = al(m * n), e_SV = al(n * r), e_A = al(r * r), e_Bt = al(r * m),
                  e_G = al(r * r), e_H = al(r * n), e_QT = al(n * r), e_Sa = al(n * n),
                  e_X = al(std::max(r * m, r * n)), e_Li = ceil_div(n, (int64_t)kG64) * kG64 * kG64;
    pifa_status s = c->work.ensure(
        (size_t)(e_Z + e_T + e_SV + e_A + e_Bt + e_G + e_H + e_QT + e_Sa + e_X + e_Li + 32) * 8, st);
    if (s != PIFA_OK) return s;
    double* Z = (double*)c->work.ptr;
    double* T = Z + e_Z;
    double* SV = T + e_T;
    double* Ar = SV + e_SV;
    double* Ut = Ar + e_A;  // (T V)^T, then U_r^T (r x m)
    double* G = Ut + e_Bt;
    double* H = G + e_G;    // U_r^T (T + a W), then Q = G^-1 H (r x n)
    double* QT = H + e_H;   // Q^T, then V_r (n x r)
    double* Sa = QT + e_QT; // S + a I, then its factor
    double* X = Sa + e_Sa;  // scratch of the solves
    double* Linv = X + e_X; // their inverted diagonal blocks
    double* floor = Linv + e_Li;
    TimedLaunch timed(kSiteCalibSolve, st);
    hipError_t e;
#define PIFA_GO(call)                              \
    do {                                           \
        if ((e = (call)) != hipSuccess) return PIFA_ERR_HIP; \
    } while (0)
    PIFA_HIP(hipMemsetAsync(c->info, 0, sizeof(int), st));
    hipLaunchKernelGGL(symmetrize_lower64, dim3(grid_for(n * n)), dim3(256), 0, st, c->S, n);
    PIFA_GO(hipGetLastError());
    // T = W (lam P + (1 - lam) S)
    hipLaunchKernelGGL(axpby_diag64, dim3(grid_for(n * n)), dim3(256), 0, st, n, lam, (const double*)c->P, 1.0 - lam,
                       (const double*)c->S, 0.0, Z);
    PIFA_GO(hipGetLastError());
    PIFA_GO(gemm64_launch(st, m, n, n, 1.0, W, n, 1, Z, n, 1, 0.0, T, n, 1));
    // A_r = V^T S V with V = Vt^T;  (T V)^T
    PIFA_GO(gemm64_launch(st, n, r, n, 1.0, c->S, n, 1, Vt, 1, n, 0.0, SV, r, 1));
    PIFA_GO(gemm64_launch(st, r, r, n, 1.0, Vt, n, 1, SV, r, 1, 0.0, Ar, r, 1));
    PIFA_GO(gemm64_launch(st, r, m, n, 1.0, Vt, n, 1, T, 1, n, 0.0, Ut, m, 1));
    // U_r^T = A_r^-1 (T V)^T   (A_r symmetric)
    PIFA_GO(cholesky64(Ar, r, r, floor, c->info, st));
    PIFA_GO(spd_solve64(Ar, r, r, Ut, m, m, Linv, X, st));
    // G = U_r^T U_r;  H = U_r^T (T + a W)
    PIFA_GO(gemm64_launch(st, r, r, m, 1.0, Ut, m, 1, Ut, 1, m, 0.0, G, r, 1));
    PIFA_GO(gemm64_launch(st, r, n, m, 1.0, Ut, m, 1, T, n, 1, 0.0, H, n, 1));
    PIFA_GO(gemm64_launch(st, r, n, m, alpha, Ut, m, 1, W, n, 1, 1.0, H, n, 1));
    // Q = G^-1 H
    PIFA_GO(cholesky64(G, r, r, floor, c->info, st));
    PIFA_GO(spd_solve64(G, r, r, H, n, n, Linv, X, st));
    // V_r = (S + a I)^-1 Q^T  (n x r), i.e. V_r^T = Q (S + a I)^-1
    hipLaunchKernelGGL(axpby_diag64, dim3(grid_for(n * n)), dim3(256), 0, st, n, 1.0, (const double*)c->S, 0.0,
                       (const double*)nullptr, alpha, Sa);
    PIFA_GO(hipGetLastError());
    PIFA_GO(transpose64_launch(H, r, n, QT, st));
    PIFA_GO(cholesky64(Sa, n, n, floor, c->info, st));
    PIFA_GO(spd_solve64(Sa, n, n, QT, r, r, Linv, X, st));
    // outputs
    PIFA_GO(transpose64_launch(Ut, r, m, U_r, st));
    PIFA_GO(transpose64_launch(QT, n, r, Vt_r, st));
#undef PIFA_GO
    int info = 0;
    PIFA_HIP(hipMemcpyAsync(&info, c->info, sizeof(int), hipMemcpyDeviceToHost, st));
    PIFA_HIP(hipStreamSynchronize(st));
    return info ? PIFA_ERR_NOT_SPD : PIFA_OK;
}

}  // extern "C"

extern "C" {

pifa_status pifa_group_create(int n, const void* const* W_p, const void* const* C,
                              const int32_t* const* pivot_idx, const int32_t* const* nonpivot_idx,
                              const pifa_dims* dims, pifa_dtype dtype, pifa_group_handle* out) {
    if (!out) return PIFA_ERR_INVALID_ARG;
    *out = nullptr;
    if (n < 1 || n > kMaxGroup || !W_p || !pivot_idx || !dims || !valid_dtype(dtype)) return PIFA_ERR_INVALID_ARG;
    if (dtype != PIFA_BF16) return PIFA_ERR_UNSUPPORTED;
    for (int i = 0; i < n; ++i) {
        pifa_status s = check_dims(dims[i]);
        if (s != PIFA_OK) return s;
        if (dims[i].d_in != dims[0].d_in) return PIFA_ERR_INVALID_ARG;
        const int64_t n_np = dims[i].d_out - dims[i].r;
        if (!W_p[i] || (n_np > 0 && (!C || !C[i] || !nonpivot_idx || !nonpivot_idx[i])))
            return PIFA_ERR_INVALID_ARG;
        s = pifa_validate_partition(pivot_idx[i], n_np > 0 ? nonpivot_idx[i] : nullptr, dims[i]);
        if (s != PIFA_OK) return s;
    }
    pifa_group* g = new (std::nothrow) pifa_group();
    if (!g) return PIFA_ERR_OOM;
    auto fail = [&](pifa_status st) {
        free_group(g);
        return st;
    };
    if (hipGetDevice(&g->device) != hipSuccess) return fail(PIFA_ERR_HIP);
    g->n = n;
    g->d_in = dims[0].d_in;
    std::vector<int32_t> piv_host;
    for (int i = 0; i < n; ++i) {
        pifa_layer* h = nullptr;
        pifa_status s = create_layer(W_p[i], C ? C[i] : nullptr, pivot_idx[i],
                                     nonpivot_idx ? nonpivot_idx[i] : nullptr, dims[i], dtype, g->d_out, &h);
        if (s != PIFA_OK) return fail(s);
        g->layers.push_back(h);
        g->r_off.push_back(g->r_pad);
        for (int64_t j = 0; j < h->r_pad; ++j)
            piv_host.push_back(j < h->r ? (int32_t)(g->d_out + pivot_idx[i][j]) : -1);
        g->d_out += h->d_out;
        g->r_pad += h->r_pad;
    }
    if (g->d_out > INT32_MAX) return fail(PIFA_ERR_UNSUPPORTED);
    // concatenate the members' lane-order W_p blocks (16-row groups follow one another)
    const size_t wp_bytes = (size_t)packed_elems(g->r_pad, g->d_in) * 2;
    if (hipMalloc(&g->Wp, wp_bytes) != hipSuccess) return fail(PIFA_ERR_OOM);
    size_t off = 0;
    for (pifa_layer* h : g->layers) {
        const size_t b = (size_t)packed_elems(h->r_pad, h->d_in) * 2;
        if (hipMemcpy((char*)g->Wp + off, h->Wp, b, hipMemcpyDeviceToDevice) != hipSuccess)
            return fail(PIFA_ERR_HIP);
        off += b;
        (void)hipFree(h->Wp);
        h->Wp = nullptr;
    }
    if (hipMalloc(&g->piv, piv_host.size() * sizeof(int32_t)) != hipSuccess) return fail(PIFA_ERR_OOM);
    if (hipMemcpy(g->piv, piv_host.data(), piv_host.size() * sizeof(int32_t), hipMemcpyHostToDevice) != hipSuccess)
        return fail(PIFA_ERR_HIP);
    if (hipMalloc(&g->overflow, sizeof(int)) != hipSuccess) return fail(PIFA_ERR_OOM);
    if (hipMemset(g->overflow, 0, sizeof(int)) != hipSuccess) return fail(PIFA_ERR_HIP);
    if (hipDeviceSynchronize() != hipSuccess) return fail(PIFA_ERR_HIP);
    *out = g;
    return PIFA_OK;
}

pifa_status pifa_group_destroy(pifa_group_handle g) {
    if (!g) return PIFA_OK;
    (void)hipDeviceSynchronize();
    free_group(g);
    return PIFA_OK;
}

pifa_status pifa_group_reserve(pifa_group_handle g, int64_t max_M) {
    if (!g || max_M < 0) return PIFA_ERR_INVALID_ARG;
    PIFA_ON_DEVICE(g->device);
    pifa_status s = g->ws.ensure(std::max(group_ws_bytes(g, max_M),
                                          group_ws_bytes(g, std::min<int64_t>(max_M, kDecodeMaxM))), 0);
    if (s != PIFA_OK) return s;
    size_t part = 0;
    for (int64_t m = kDecodeMaxM + 1; m <= std::min(max_M, kSplitMaxM); ++m)
        part = std::max(part, group_part_bytes(g, m));
    s = g->part.ensure(part, 0);
    if (s != PIFA_OK) return s;
    return hipDeviceSynchronize() == hipSuccess ? PIFA_OK : PIFA_ERR_HIP;
}

size_t pifa_group_weight_bytes(pifa_group_handle g) {
    if (!g) return 0;
    size_t b = 0;
    for (pifa_layer* h : g->layers) b += pifa_layer_weight_bytes(h);
    return b;
}

pifa_status pifa_group_set_intermediate_scale(pifa_group_handle g, int log2_scale) {
    if (!g || log2_scale < -30 || log2_scale > 30) return PIFA_ERR_INVALID_ARG;
    g->y_log2 = log2_scale;
    return PIFA_OK;
}

pifa_status pifa_group_overflow_count(pifa_group_handle g, int64_t* count) {
    if (!g || !count) return PIFA_ERR_INVALID_ARG;
    int v = 0;
    PIFA_HIP(hipDeviceSynchronize());
    PIFA_HIP(hipMemcpy(&v, g->overflow, sizeof(int), hipMemcpyDeviceToHost));
    *count = v;
    return PIFA_OK;
}

pifa_status pifa_group_forward(pifa_group_handle g, const void* X, void* Y, int64_t M, void* stream) {
    if (!g || M < 0) return PIFA_ERR_INVALID_ARG;
    if (M == 0) return PIFA_OK;
    if (!X || !Y) return PIFA_ERR_INVALID_ARG;
    PIFA_ON_DEVICE(g->device);
    if (!aligned16(X)) return PIFA_ERR_UNSUPPORTED;
    hipStream_t st = as_stream(stream);
    pifa_status s = g->ws.ensure(group_ws_bytes(g, M), st);
    if (s != PIFA_OK) return s;
    const float y_scale = std::ldexp(1.0f, g->y_log2);
    bf16* y = (bf16*)Y;
    f16* yp = (f16*)g->ws.ptr;
    using EpiNP = ScatterEpi<bf16, kWsNone>;
    hipError_t e;
    if (M <= kDecodeMaxM) {
        // pivot outputs of every member from one weight stream; Y_p as fp16 hi + lo planes
        e = launch_skinny_packed<bf16>(kSiteGroupGemv1, ALoad16<bf16>{(const bf16*)X, g->d_in, M},
                                       (const bf16*)g->Wp, g->r_pad, g->d_in,
                                       make_epi<bf16, kWsF16Pair>(y, g->d_out, g->piv, g->r_pad, 1.f, yp, g->r_pad,
                                                                  g->r_pad, y_scale, g->overflow, M),
                                       st);
        if (e != hipSuccess) return PIFA_ERR_HIP;
        SkinnyGroup<f16, ALoadPair16, EpiNP> grp{};
        int64_t rows[kMaxSkinnyGroup] = {};
        for (int i = 0; i < g->n; ++i) {
            const pifa_layer* h = g->layers[(size_t)i];
            const float out_scale = std::ldexp(1.0f, -(g->y_log2 + h->c_log2));
            grp.p[grp.n] = {ALoadPair16{yp + g->r_off[(size_t)i], g->r_pad, M}, (const f16*)h->C, h->r_pad,
                            make_epi<bf16, kWsNone>(y, g->d_out, h->npiv, h->n_np, out_scale, nullptr, 0, 0, 1.f,
                                                    nullptr, M)};
            rows[grp.n++] = h->n_np;
        }
        e = launch_skinny_grouped(kSiteGroupGemv2, grp, rows, st);
        return e == hipSuccess ? PIFA_OK : PIFA_ERR_HIP;
    }
    s = g->part.ensure(group_part_bytes(g, M), st);
    if (s != PIFA_OK) return s;
    e = launch_gemm<bf16, true>(kSiteGroupGemm1, (const bf16*)X, g->d_in, M, (const bf16*)g->Wp, 0, g->r_pad,
                                g->d_in,
                                make_epi<bf16, kWsF16>(y, g->d_out, g->piv, g->r_pad, 1.f, yp, g->r_pad, g->r_pad,
                                                       y_scale, g->overflow, M),
                                (float*)g->part.ptr, st);
    if (e != hipSuccess) return PIFA_ERR_HIP;
    // The non-pivot products: one launch per member, as its own pifa_forward
    // runs it.  Both products are compute-bound at these sizes; one launch
    // over all members measured slower (372 against 2 x 165 us for the
    // LLaMA-7B gate and up projections at M = 4096).
    for (int i = 0; i < g->n; ++i) {
        const pifa_layer* h = g->layers[(size_t)i];
        if (h->n_np == 0) continue;
        const float out_scale = std::ldexp(1.0f, -(g->y_log2 + h->c_log2));
        e = launch_gemm<f16, true>(kSiteGroupGemm2, yp + g->r_off[(size_t)i], g->r_pad, M, (const f16*)h->C, 0,
                                   h->n_np, h->r_pad,
                                   make_epi<bf16, kWsNone>(y, g->d_out, h->npiv, h->n_np, out_scale, nullptr, 0, 0,
                                                           1.f, nullptr, M),
                                   (float*)g->part.ptr, st);
        if (e != hipSuccess) return PIFA_ERR_HIP;
    }
    return PIFA_OK;
}

pifa_status pifa_build_f64(const double* W, pifa_dims dims, double* W_p, double* C, int32_t* pivot_idx,
                           int32_t* nonpivot_idx, double* report, void* stream) {
    pifa_status s = check_dims(dims);
    if (s != PIFA_OK) return s;
    const int64_t d_in = dims.d_in, d_out = dims.d_out, r = dims.r, n_np = d_out - r;
    if (!W || !W_p || !pivot_idx || (n_np > 0 && (!C || !nonpivot_idx))) return PIFA_ERR_INVALID_ARG;
    hipStream_t st = as_stream(stream);

    struct Buf {
        void* p = nullptr;
        ~Buf() {
            if (p) (void)hipFree(p);
        }
    } A, norm2, perm, tau, status, RT, Csel, diag, idx, Fp, aux;
    auto alloc = [](Buf& b, size_t bytes) { return hipMalloc(&b.p, bytes < 16 ? 16 : bytes) == hipSuccess; };
    if (!alloc(A, (size_t)d_out * d_in * 8) || !alloc(norm2, (size_t)d_out * 8) ||
        !alloc(perm, (size_t)d_out * 4) || !alloc(tau, (size_t)r * 8) || !alloc(status, 4) ||
        !alloc(diag, (size_t)r * 8) || !alloc(idx, (size_t)(r + 2 * n_np + r) * 4) ||
        !alloc(Fp, (size_t)d_out * kPanel * 8) || !alloc(aux, (size_t)kPanel * 8))
        return PIFA_ERR_OOM;
    double* dA = (double*)A.p;
    double* dn = (double*)norm2.p;
    int32_t* dperm = (int32_t*)perm.p;
    double* dF = (double*)Fp.p;
    PIFA_HIP(hipMemsetAsync(status.p, 0, 4, st));

    // QR with column pivoting in panels of kPanel steps (build.hpp)
    hipLaunchKernelGGL(qr_init, dim3((unsigned)ceil_div(d_out, 4)), dim3(256), 0, st, W, dA, dn, dperm, d_out, d_in);
    for (int64_t k0 = 0; k0 < r; k0 += kPanel) {
        const int64_t nb = std::min<int64_t>(kPanel, r - k0);
        for (int64_t k = k0; k < k0 + nb; ++k) {
            // columns of up to kPivotLdsRows rows keep the updated pivot
            // column in LDS (fewer dependent memory round trips, bit-identical)
            if (d_in <= kPivotLdsRows)
                hipLaunchKernelGGL(qr_panel_pivot_lds, dim3(1), dim3(kBuildThreads), (size_t)(d_in - k) * 8, st, dA, dn,
                                   dperm, dF, (double*)tau.p, (double*)aux.p, (int*)status.p, k, k0, d_out, d_in);
            else
                hipLaunchKernelGGL(qr_panel_pivot, dim3(1), dim3(kBuildThreads), 0, st, dA, dn, dperm, dF,
                                   (double*)tau.p, (double*)aux.p, (int*)status.p, k, k0, d_out, d_in);
            if (k + 1 < d_out)
                hipLaunchKernelGGL(qr_panel_gemv, dim3((unsigned)ceil_div(d_out - k - 1, 4)), dim3(256), 0, st, dA, dn,
                                   dF, (const double*)tau.p, (const double*)aux.p, k, k0, d_out, d_in);
        }
        // the panel's reflections on the rest of the trailing matrix, then
        // its exact residual norms
        const int64_t ks = k0 + nb;
        if (ks < d_out) {
            if (ks < d_in &&
                gemm64_launch(st, d_in - ks, d_out - ks, nb, -1.0, dA + k0 * d_in + ks, 1, d_in, dF + ks * kPanel, 1,
                              kPanel, 1.0, dA + ks * d_in + ks, 1, d_in) != hipSuccess)
                return PIFA_ERR_HIP;
            hipLaunchKernelGGL(qr_norms, dim3((unsigned)ceil_div(d_out - ks, 4)), dim3(256), 0, st, (const double*)dA, dn,
                               ks, d_out, d_in);
        }
    }
    PIFA_HIP(hipGetLastError());

    // rank certification on the host: diagonal of R, residual norms
    std::vector<int32_t> hperm((size_t)d_out);
    std::vector<double> hdiag((size_t)r), hnorm((size_t)d_out);
    int hstatus = 0;
    hipLaunchKernelGGL(extract_diag, dim3(grid_for(r)), dim3(256), 0, st, (const double*)dA, (double*)diag.p, r, d_in);
    PIFA_HIP(hipGetLastError());
    PIFA_HIP(hipMemcpyAsync(hdiag.data(), diag.p, (size_t)r * 8, hipMemcpyDeviceToHost, st));
    PIFA_HIP(hipMemcpyAsync(hperm.data(), dperm, (size_t)d_out * 4, hipMemcpyDeviceToHost, st));
    PIFA_HIP(hipMemcpyAsync(hnorm.data(), dn, (size_t)d_out * 8, hipMemcpyDeviceToHost, st));
    PIFA_HIP(hipMemcpyAsync(&hstatus, status.p, 4, hipMemcpyDeviceToHost, st));
    PIFA_HIP(hipStreamSynchronize(st));
    const double r00 = std::fabs(hdiag[0]), rlast = std::fabs(hdiag[(size_t)r - 1]);
    double resid = 0.0;
    for (int64_t j = r; j < d_out; ++j) resid = std::max(resid, std::sqrt(std::max(hnorm[(size_t)j], 0.0)));
    const bool certified = hstatus == 0 && rlast >= 1e-8 * r00 && resid <= 1e-10 * r00;
    if (report) {
        report[0] = r00;
        report[1] = rlast;
        report[2] = resid;
        report[3] = certified ? 1.0 : 0.0;
    }
    if (!certified) return PIFA_ERR_NOT_RANK_R;

    // sorted index sets and the selection slot each came from
    std::vector<std::pair<int32_t, int32_t>> piv((size_t)r), npv((size_t)n_np);
    for (int64_t s2 = 0; s2 < r; ++s2) piv[(size_t)s2] = {hperm[(size_t)s2], (int32_t)s2};
    for (int64_t t = 0; t < n_np; ++t) npv[(size_t)t] = {hperm[(size_t)(r + t)], (int32_t)t};
    std::sort(piv.begin(), piv.end());
    std::sort(npv.begin(), npv.end());
    std::vector<int32_t> hidx((size_t)(r + 2 * n_np + r));
    int32_t* rows_p = hidx.data();            // r: sorted pivot rows
    int32_t* rows_np = rows_p + r;            // n_np: sorted non-pivot rows
    int32_t* row_src = rows_np + n_np;        // n_np: selection slot of each sorted non-pivot
    int32_t* col_src = row_src + n_np;        // r: selection slot of each sorted pivot
    for (int64_t i = 0; i < r; ++i) {
        rows_p[i] = piv[(size_t)i].first;
        col_src[i] = piv[(size_t)i].second;
        pivot_idx[i] = rows_p[i];
    }
    for (int64_t q = 0; q < n_np; ++q) {
        rows_np[q] = npv[(size_t)q].first;
        row_src[q] = npv[(size_t)q].second;
        nonpivot_idx[q] = rows_np[q];
    }
    int32_t* didx = (int32_t*)idx.p;
    PIFA_HIP(hipMemcpyAsync(didx, hidx.data(), hidx.size() * 4, hipMemcpyHostToDevice, st));

    hipLaunchKernelGGL(gather_rows, dim3(grid_for(r * d_in)), dim3(256), 0, st, W, didx, W_p, r, d_in);
    if (n_np > 0) {
        if (!alloc(RT, (size_t)r * r * 8) || !alloc(Csel, (size_t)n_np * r * 8)) return PIFA_ERR_OOM;
        hipLaunchKernelGGL(extract_r11, dim3(grid_for(r * r)), dim3(256), 0, st, (const double*)dA, (double*)RT.p, r,
                           d_in);
        // C R11^T = R12^T, right-looking blocks of kSolveBlock unknowns (build.hpp)
        double* X = (double*)Csel.p;
        const double* R11 = (const double*)RT.p;
        hipLaunchKernelGGL(coeff_rhs, dim3(grid_for(n_np * r)), dim3(256), 0, st, (const double*)dA, X, r, n_np, d_in);
        for (int64_t s0 = (ceil_div(r, (int64_t)kSolveBlock) - 1) * kSolveBlock; s0 >= 0; s0 -= kSolveBlock) {
            const int nb = (int)std::min<int64_t>(kSolveBlock, r - s0);
            hipLaunchKernelGGL(coeff_block_solve, dim3((unsigned)ceil_div(n_np, (int64_t)kSolveBlock)),
                               dim3(kSolveBlock), 0, st, R11, X, r, n_np, s0, nb);
            // X[:, 0:s0] -= X[:, s0:s0+nb] R11[0:s0, s0:s0+nb]^T
            if (s0 > 0 && gemm64_launch(st, n_np, s0, nb, -1.0, X + s0, r, 1, R11 + s0, 1, r, 1.0, X, r, 1) !=
                              hipSuccess)
                return PIFA_ERR_HIP;
        }
        hipLaunchKernelGGL(gather_coeffs, dim3(grid_for(n_np * r)), dim3(256), 0, st, (const double*)Csel.p,
                           didx + r + n_np, didx + r + 2 * n_np, C, n_np, r);
    }
    PIFA_HIP(hipGetLastError());
    PIFA_HIP(hipStreamSynchronize(st));
    return PIFA_OK;
}

pifa_status pifa_profile_enable(int on) {
    Profiler& p = profiler();
    std::lock_guard<std::mutex> g(p.mu);
    p.on = on != 0;
    return PIFA_OK;
}

pifa_status pifa_profile_reset(void) {
    Profiler& p = profiler();
    std::lock_guard<std::mutex> g(p.mu);
    for (auto& r : p.pending) {
        (void)hipEventSynchronize(r.stop);
        p.pool.push_back(r.start);
        p.pool.push_back(r.stop);
    }
    p.pending.clear();
    for (int i = 0; i < kSiteCount; ++i) {
        p.launches[i] = 0;
        p.ms[i] = 0.0;
    }
    return PIFA_OK;
}

pifa_status pifa_profile_read(const char** names, int64_t* launches, double* total_ms, int max_sites,
                              int* n_sites) {
    if (!names || !launches || !total_ms || !n_sites || max_sites < 0) return PIFA_ERR_INVALID_ARG;
    Profiler& p = profiler();
    std::lock_guard<std::mutex> g(p.mu);
    pifa_status status = PIFA_OK;
    for (auto& r : p.pending) {
        float ms = 0.f;
        if (hipEventSynchronize(r.stop) != hipSuccess ||
            hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess)
            status = PIFA_ERR_HIP;
        p.launches[r.site] += 1;
        p.ms[r.site] += ms;
        p.pool.push_back(r.start);
        p.pool.push_back(r.stop);
    }
    p.pending.clear();
    int n = 0;
    for (int i = 0; i < kSiteCount && n < max_sites; ++i) {
        if (p.launches[i] == 0) continue;
        names[n] = kSiteNames[i];
        launches[n] = p.launches[i];
        total_ms[n] = p.ms[i];
        ++n;
    }
    *n_sites = n;
    return status;
}

// ------------------------------------------------------------------ allocation-free forward
namespace {

// The workspace of pifa_forward_noalloc: one fixed array per GPU, held until
// the process ends.  In host code `scratch` names a host-side stand-in, not
// the device memory; its device address on each GPU comes from
// hipGetSymbolAddress, called once per device with that device current.
constexpr size_t kNoAllocScratchBytes = 32ull << 20;
static __device__ __align__(256) uint8_t scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

pifa_status scratch_address(int dev, void** out) {
    if (dev < 0 || dev >= kMaxDevices) return PIFA_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> g(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return PIFA_ERR_HIP;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return PIFA_OK;
}

}  // namespace

pifa_status pifa_forward_noalloc(pifa_handle h, const void* X, void* Y, int64_t M, void* stream) {
    if (!h || M < 0) return PIFA_ERR_INVALID_ARG;
    if (M == 0) return PIFA_OK;
    if (!X || !Y) return PIFA_ERR_INVALID_ARG;
    PIFA_ON_DEVICE(h->device);
    if (h->dtype == PIFA_BF16 && !aligned16(X)) return PIFA_ERR_UNSUPPORTED;
    const size_t ws = (size_t)round_up((int64_t)pifa_ws_bytes(h, M), 256);
    const size_t part = pifa_part_bytes(h, M);
    if (ws + part > kNoAllocScratchBytes) return PIFA_ERR_TOO_LARGE;
    void* base = nullptr;
    const pifa_status s = scratch_address(h->device, &base);
    if (s != PIFA_OK) return s;
    t_untimed = true;
    const pifa_status r = forward_with(h, X, Y, M, base, part ? (float*)((char*)base + ws) : nullptr,
                                       as_stream(stream));
    t_untimed = false;
    return r;
}

// ------------------------------------------------------------------ peak probes
namespace {

struct DevBuf {
    void* p = nullptr;
    ~DevBuf() {
        if (p) (void)hipFree(p);
    }
};

}  // namespace

namespace {

pifa_status probe_mfma(bool random, int64_t iters, double* tflops, double* sclk_mhz, void* stream) {
    if (iters < 1 || !tflops || !sclk_mhz) return PIFA_ERR_INVALID_ARG;
    if (random) iters = round_up(iters, 8);
    hipStream_t st = as_stream(stream);
    constexpr unsigned kGrid = 2048, kThreads = 256;
    DevBuf clocks, sink;
    if (hipMalloc(&clocks.p, (size_t)kGrid * 16) != hipSuccess) return PIFA_ERR_OOM;
    if (hipMalloc(&sink.p, (size_t)kGrid * 4) != hipSuccess) return PIFA_ERR_OOM;
    int dev = 0, wall_khz = 0;
    PIFA_HIP(hipGetDevice(&dev));
    PIFA_HIP(hipDeviceGetAttribute(&wall_khz, hipDeviceAttributeWallClockRate, dev));
    if (wall_khz <= 0) return PIFA_ERR_UNSUPPORTED;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    PIFA_HIP(hipEventCreate(&e0));
    if (hipEventCreate(&e1) != hipSuccess) {
        (void)hipEventDestroy(e0);
        return PIFA_ERR_HIP;
    }
    auto run = [&]() {
        if (random)
            hipLaunchKernelGGL(mfma_probe_random, dim3(kGrid), dim3(kThreads), 0, st, iters, 0.0f, (float*)sink.p,
                               (uint64_t*)clocks.p);
        else
            hipLaunchKernelGGL(mfma_probe, dim3(kGrid), dim3(kThreads), 0, st, iters, 0.0f, (float*)sink.p,
                               (uint64_t*)clocks.p);
        return hipGetLastError();
    };
    float ms = 0.f;
    bool ok = run() == hipSuccess && hipEventRecord(e0, st) == hipSuccess && run() == hipSuccess &&
              hipEventRecord(e1, st) == hipSuccess && hipEventSynchronize(e1) == hipSuccess &&
              hipEventElapsedTime(&ms, e0, e1) == hipSuccess;
    std::vector<uint64_t> h((size_t)kGrid * 2);
    ok = ok && hipMemcpy(h.data(), clocks.p, h.size() * 8, hipMemcpyDeviceToHost) == hipSuccess;
    (void)hipEventDestroy(e0);
    (void)hipEventDestroy(e1);
    if (!ok || ms <= 0.f) return PIFA_ERR_HIP;
    // 4 waves x 4 MFMAs of 32 x 32 x 16 (2 * 16384 FLOPs each) per iteration
    *tflops = (double)kGrid * 4 * 4 * 32768.0 * (double)iters / (ms * 1e9);
    double mhz = 0.0;
    int64_t n = 0;
    for (unsigned b = 0; b < kGrid; ++b) {
        if (h[2 * b + 1] == 0) continue;
        mhz += (double)h[2 * b] / (double)h[2 * b + 1] * (wall_khz / 1000.0);
        ++n;
    }
    *sclk_mhz = n ? mhz / n : 0.0;
    return PIFA_OK;
}

}  // namespace

pifa_status pifa_probe_mfma(int64_t iters, double* tflops, double* sclk_mhz, void* stream) {
    return probe_mfma(false, iters, tflops, sclk_mhz, stream);
}

pifa_status pifa_probe_mfma_random(int64_t iters, double* tflops, double* sclk_mhz, void* stream) {
    return probe_mfma(true, iters, tflops, sclk_mhz, stream);
}

pifa_status pifa_probe_hbm_read(const void* buf, int64_t bytes, int reps, double* gbps, void* stream) {
    if (!buf || bytes < 16 || bytes % 16 != 0 || reps < 1 || !gbps || !aligned16(buf)) return PIFA_ERR_INVALID_ARG;
    hipStream_t st = as_stream(stream);
    // the best of three grid sizes (8, 16 and 32 workgroups of 256 threads per CU)
    constexpr unsigned kThreads = 256;
    const unsigned grids[3] = {2048, 4096, 8192};
    DevBuf sink;
    if (hipMalloc(&sink.p, (size_t)8192 * 4) != hipSuccess) return PIFA_ERR_OOM;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    PIFA_HIP(hipEventCreate(&e0));
    if (hipEventCreate(&e1) != hipSuccess) {
        (void)hipEventDestroy(e0);
        return PIFA_ERR_HIP;
    }
    double best = 0.0;
    bool ok = true;
    for (unsigned grid : grids) {
        auto run = [&]() {
            hipLaunchKernelGGL(hbm_read_probe, dim3(grid), dim3(kThreads), 0, st, (const u32x4*)buf, bytes / 16,
                               (uint32_t*)sink.p);
            return hipGetLastError();
        };
        ok = ok && run() == hipSuccess && hipEventRecord(e0, st) == hipSuccess;
        for (int i = 0; ok && i < reps; ++i) ok = run() == hipSuccess;
        float ms = 0.f;
        ok = ok && hipEventRecord(e1, st) == hipSuccess && hipEventSynchronize(e1) == hipSuccess &&
             hipEventElapsedTime(&ms, e0, e1) == hipSuccess && ms > 0.f;
        if (ok) best = std::max(best, (double)bytes * reps / (ms * 1e6));
    }
    (void)hipEventDestroy(e0);
    (void)hipEventDestroy(e1);
    if (!ok) return PIFA_ERR_HIP;
    *gbps = best;
    return PIFA_OK;
}

}  // extern "C"
