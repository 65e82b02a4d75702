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
#include "gemv_skinny.hpp"
#include "prepack.hpp"

using namespace pifa;

namespace {

// ------------------------------------------------------------------ config
constexpr int64_t kDecodeMaxM = 16;  // M at or below this takes the skinny path
constexpr int64_t kRowPad = 64;      // W_p rows / C columns padded to this multiple

constexpr int kGemmBM = 128, kGemmBN = 128, kGemmBK = 64, kGemmWM = 2, kGemmWN = 2;
constexpr int kSkinnyWaves = 4, kSkinnyUnroll = 2;
constexpr int64_t kSkinnyTargetWgs = 1024;
constexpr int64_t kSkinnyMaxSplit = 16;

#define PIFA_HIP(call)                                  \
    do {                                                \
        if ((call) != hipSuccess) return PIFA_ERR_HIP;  \
    } while (0)

inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }
inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
inline size_t esize(pifa_dtype dt) { return dt == PIFA_BF16 ? 2 : 4; }
inline bool valid_dtype(pifa_dtype dt) { return dt == PIFA_BF16 || dt == PIFA_F32; }

// ------------------------------------------------------------------ skinny split
struct SkinnyPlan {
    int64_t groups, splits, k_split;
};

SkinnyPlan skinny_plan(int64_t N, int64_t K) {
    SkinnyPlan p;
    p.groups = ceil_div(N, kSkinnyRows);
    const int64_t step = (int64_t)kSkinnyWaves * kSkinnyStepK;
    int64_t s = ceil_div(kSkinnyTargetWgs, p.groups < 1 ? 1 : p.groups);
    const int64_t smax = ceil_div(K, step);
    if (s > smax) s = smax;
    if (s > kSkinnyMaxSplit) s = kSkinnyMaxSplit;
    if (s < 1) s = 1;
    p.k_split = round_up(ceil_div(K, s), step);
    p.splits = ceil_div(K, p.k_split);
    return p;
}

size_t skinny_partial_bytes(const SkinnyPlan& p) {
    return p.splits > 1 ? (size_t)(p.groups * p.splits) * kWave * sizeof(f32x4) : 0;
}

// Scratch for the split-K reduction of the skinny kernel.  Counters start at
// zero and every launch leaves them at zero.
struct SplitScratch {
    float* partials = nullptr;
    size_t partial_bytes = 0;
    int* counters = nullptr;
    size_t n_counters = 0;

    pifa_status ensure(const SkinnyPlan& p, hipStream_t st) {
        const size_t pb = skinny_partial_bytes(p);
        const size_t nc = (size_t)p.groups;
        if (pb <= partial_bytes && nc <= n_counters) return PIFA_OK;
        PIFA_HIP(hipStreamSynchronize(st));
        if (pb > partial_bytes) {
            if (partials) PIFA_HIP(hipFree(partials));
            partials = nullptr;
            partial_bytes = 0;
            if (hipMalloc(&partials, pb) != hipSuccess) return PIFA_ERR_OOM;
            partial_bytes = pb;
        }
        if (nc > n_counters) {
            if (counters) PIFA_HIP(hipFree(counters));
            counters = nullptr;
            n_counters = 0;
            if (hipMalloc(&counters, nc * sizeof(int)) != hipSuccess) return PIFA_ERR_OOM;
            PIFA_HIP(hipMemset(counters, 0, nc * sizeof(int)));
            PIFA_HIP(hipDeviceSynchronize());
            n_counters = nc;
        }
        return PIFA_OK;
    }
    void release() {
        if (partials) (void)hipFree(partials);
        if (counters) (void)hipFree(counters);
        partials = nullptr;
        counters = nullptr;
        partial_bytes = n_counters = 0;
    }
};

// A device buffer that only grows; growing waits for `st` first so no kernel
// in flight still uses the old allocation.
struct GrowBuf {
    void* ptr = nullptr;
    size_t bytes = 0;
    pifa_status ensure(size_t need, hipStream_t st) {
        if (need <= bytes) return PIFA_OK;
        PIFA_HIP(hipStreamSynchronize(st));
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

// ------------------------------------------------------------------ launchers
template <typename T, typename Epi>
hipError_t launch_gemm(const T* A, int64_t lda, int64_t M, const T* B, int64_t ldb, int64_t N,
                       int64_t K, Epi epi, hipStream_t st) {
    const int64_t tiles = ceil_div(M, kGemmBM) * ceil_div(N, kGemmBN);
    if (tiles == 0) return hipSuccess;
    hipLaunchKernelGGL((gemm_nt_mfma<T, kGemmBM, kGemmBN, kGemmBK, kGemmWM, kGemmWN, Epi>),
                       dim3((unsigned)tiles), dim3(kGemmWM * kGemmWN * kWave), 0, st, A, lda, M, B,
                       ldb, N, K, epi);
    return hipGetLastError();
}

template <typename Epi>
hipError_t launch_gemm_f32(const float* A, int64_t lda, int64_t M, const float* B, int64_t ldb,
                           int64_t N, int64_t K, Epi epi, hipStream_t st) {
    if (M == 0 || N == 0) return hipSuccess;
    hipLaunchKernelGGL((gemm_nt_f32<Epi>), dim3((unsigned)ceil_div(N, 64), (unsigned)ceil_div(M, 64)),
                       dim3(256), 0, st, A, lda, M, B, ldb, N, K, epi);
    return hipGetLastError();
}

template <typename TB, typename AL, typename Epi>
hipError_t launch_skinny(AL al, const TB* B, int64_t ldb, int64_t N, int64_t K,
                         const SplitScratch& sc, Epi epi, hipStream_t st) {
    const SkinnyPlan p = skinny_plan(N, K);
    if (p.groups == 0) return hipSuccess;
    hipLaunchKernelGGL((skinny_mfma<TB, kSkinnyWaves, kSkinnyUnroll, AL, Epi>),
                       dim3((unsigned)p.groups, (unsigned)p.splits), dim3(kSkinnyWaves * kWave), 0, st,
                       al, B, ldb, N, K, p.k_split, sc.partials, sc.counters, epi);
    return hipGetLastError();
}

hipError_t launch_pack_bits(const void* src, int64_t rows, int64_t cols, int64_t ld, void* dst,
                            int64_t rows_pad, int64_t cols_pad, size_t elem, hipStream_t st) {
    const int64_t total = rows_pad * cols_pad;
    if (total == 0) return hipSuccess;
    const unsigned blocks = (unsigned)std::min<int64_t>(ceil_div(total, 256), 65536);
    if (elem == 2)
        hipLaunchKernelGGL((pack_pad<uint16_t>), dim3(blocks), dim3(256), 0, st,
                           (const uint16_t*)src, rows, cols, ld, (uint16_t*)dst, rows_pad, cols_pad);
    else
        hipLaunchKernelGGL((pack_pad<float>), dim3(blocks), dim3(256), 0, st, (const float*)src, rows,
                           cols, ld, (float*)dst, rows_pad, cols_pad);
    return hipGetLastError();
}

// ------------------------------------------------------------------ shared workspace
struct DeviceScratch {
    std::mutex mu;
    GrowBuf inter;  // intermediate X V^T of the stateless low-rank baseline
    SplitScratch split;
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
struct pifa_layer {
    int device = 0;
    pifa_dtype dtype = PIFA_BF16;
    int64_t d_in = 0, d_out = 0, r = 0, n_np = 0, r_pad = 0;
    void* Wp = nullptr;        // bf16: r_pad x d_in, rows >= r zero; f32: r x d_in
    void* C = nullptr;         // bf16: fp16 n_np x r_pad times 2^c_log2; f32: n_np x r
    int32_t* piv = nullptr;    // r
    int32_t* npiv = nullptr;   // n_np
    int* overflow = nullptr;
    int c_log2 = 0, y_log2 = 0;
    GrowBuf ws;                // Y_p hand-off
    SplitScratch split;
};

struct lowrank_layer {
    int device = 0;
    pifa_dtype dtype = PIFA_BF16;
    int64_t d_in = 0, d_out = 0, r = 0, r_pad = 0;
    void* U = nullptr;  // d_out x r_pad, columns >= r zero
    void* V = nullptr;  // r_pad x d_in, rows >= r zero
    GrowBuf ws;
    SplitScratch split;
};

namespace {

void free_layer(pifa_layer* h) {
    if (!h) return;
    if (h->Wp) (void)hipFree(h->Wp);
    if (h->C) (void)hipFree(h->C);
    if (h->piv) (void)hipFree(h->piv);
    if (h->npiv) (void)hipFree(h->npiv);
    if (h->overflow) (void)hipFree(h->overflow);
    h->ws.release();
    h->split.release();
    delete h;
}

void free_lowrank(lowrank_layer* h) {
    if (!h) return;
    if (h->U) (void)hipFree(h->U);
    if (h->V) (void)hipFree(h->V);
    h->ws.release();
    h->split.release();
    delete h;
}

size_t pifa_ws_bytes(const pifa_layer* h, int64_t M) {
    if (h->dtype == PIFA_F32) return (size_t)M * (size_t)h->r * 4;
    if (M <= kDecodeMaxM) return (size_t)M * (size_t)h->r_pad * 4;
    return (size_t)M * (size_t)h->r_pad * 2;
}

pifa_status pifa_prepare(pifa_layer* h, int64_t M, hipStream_t st) {
    pifa_status s = h->ws.ensure(pifa_ws_bytes(h, M), st);
    if (s != PIFA_OK) return s;
    if (h->dtype == PIFA_BF16 && M <= kDecodeMaxM) {
        s = h->split.ensure(skinny_plan(h->r_pad, h->d_in), st);
        if (s != PIFA_OK) return s;
        if (h->n_np > 0) s = h->split.ensure(skinny_plan(h->n_np, h->r_pad), st);
    }
    return s;
}

size_t lowrank_ws_bytes(pifa_dtype dt, int64_t M, int64_t r_cols) {
    if (dt == PIFA_F32 || M <= kDecodeMaxM) return (size_t)M * (size_t)r_cols * 4;
    return (size_t)M * (size_t)r_cols * 2;
}

// Y = (X V^T) U^T with V: r_cols x d_in (ldv = d_in), U: d_out x r_cols (ldu = r_cols).
pifa_status lowrank_run(pifa_dtype dt, const void* U, const void* V, const void* X, void* Y,
                        int64_t M, int64_t d_in, int64_t d_out, int64_t r_cols, void* T,
                        const SplitScratch& sc, hipStream_t st) {
    hipError_t e;
    if (dt == PIFA_F32) {
        float* t = (float*)T;
        e = launch_gemm_f32((const float*)X, d_in, M, (const float*)V, d_in, r_cols, d_in,
                            make_epi<float, kWsNone>(t, r_cols, nullptr, r_cols, 1.f, nullptr, 0, 0,
                                                     1.f, nullptr, M),
                            st);
        if (e != hipSuccess) return PIFA_ERR_HIP;
        e = launch_gemm_f32(t, r_cols, M, (const float*)U, r_cols, d_out, r_cols,
                            make_epi<float, kWsNone>((float*)Y, d_out, nullptr, d_out, 1.f, nullptr,
                                                     0, 0, 1.f, nullptr, M),
                            st);
        return e == hipSuccess ? PIFA_OK : PIFA_ERR_HIP;
    }
    if (M <= kDecodeMaxM) {
        float* t = (float*)T;
        e = launch_skinny<bf16>(ALoad16<bf16>{(const bf16*)X, d_in, M}, (const bf16*)V, d_in,
                                r_cols, d_in, sc,
                                make_epi<float, kWsNone>(t, r_cols, nullptr, r_cols, 1.f, nullptr,
                                                         0, 0, 1.f, nullptr, M),
                                st);
        if (e != hipSuccess) return PIFA_ERR_HIP;
        e = launch_skinny<bf16>(ASplit32<bf16>{t, r_cols, M, 1.f}, (const bf16*)U, r_cols, d_out,
                                r_cols, sc,
                                make_epi<bf16, kWsNone>((bf16*)Y, d_out, nullptr, d_out, 1.f,
                                                        nullptr, 0, 0, 1.f, nullptr, M),
                                st);
        return e == hipSuccess ? PIFA_OK : PIFA_ERR_HIP;
    }
    bf16* t = (bf16*)T;
    e = launch_gemm<bf16>((const bf16*)X, d_in, M, (const bf16*)V, d_in, r_cols, d_in,
                          make_epi<bf16, kWsNone>(t, r_cols, nullptr, r_cols, 1.f, nullptr, 0, 0,
                                                  1.f, nullptr, M),
                          st);
    if (e != hipSuccess) return PIFA_ERR_HIP;
    e = launch_gemm<bf16>(t, r_cols, M, (const bf16*)U, r_cols, d_out, r_cols,
                          make_epi<bf16, kWsNone>((bf16*)Y, d_out, nullptr, d_out, 1.f, nullptr, 0,
                                                  0, 1.f, nullptr, M),
                          st);
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
    }
    return "PIFA_ERR_UNKNOWN";
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

pifa_status pifa_layer_create(const void* W_p, const void* C, const int32_t* pivot_idx,
                              const int32_t* nonpivot_idx, pifa_dims dims, pifa_dtype dtype,
                              pifa_handle* out) {
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
    h->r_pad = dtype == PIFA_BF16 ? round_up(dims.r, kRowPad) : dims.r;

    auto fail = [&](pifa_status st) {
        free_layer(h);
        return st;
    };
    if (hipGetDevice(&h->device) != hipSuccess) return fail(PIFA_ERR_HIP);
    if (hipDeviceSynchronize() != hipSuccess) return fail(PIFA_ERR_HIP);
    const size_t es = esize(dtype);

    if (hipMalloc(&h->Wp, (size_t)h->r_pad * h->d_in * es) != hipSuccess) return fail(PIFA_ERR_OOM);
    if (launch_pack_bits(W_p, h->r, h->d_in, h->d_in, h->Wp, h->r_pad, h->d_in, es, 0) != hipSuccess)
        return fail(PIFA_ERR_HIP);

    if (hipMalloc(&h->piv, (size_t)h->r * sizeof(int32_t)) != hipSuccess) return fail(PIFA_ERR_OOM);
    if (hipMemcpy(h->piv, pivot_idx, (size_t)h->r * sizeof(int32_t), hipMemcpyHostToDevice) != hipSuccess)
        return fail(PIFA_ERR_HIP);
    if (hipMalloc(&h->overflow, sizeof(int)) != hipSuccess) return fail(PIFA_ERR_OOM);
    if (hipMemset(h->overflow, 0, sizeof(int)) != hipSuccess) return fail(PIFA_ERR_HIP);

    if (n_np > 0) {
        if (hipMalloc(&h->npiv, (size_t)n_np * sizeof(int32_t)) != hipSuccess) return fail(PIFA_ERR_OOM);
        if (hipMemcpy(h->npiv, nonpivot_idx, (size_t)n_np * sizeof(int32_t), hipMemcpyHostToDevice) !=
            hipSuccess)
            return fail(PIFA_ERR_HIP);
        if (hipMalloc(&h->C, (size_t)n_np * h->r_pad * es) != hipSuccess) return fail(PIFA_ERR_OOM);
        if (dtype == PIFA_F32) {
            if (launch_pack_bits(C, n_np, h->r, h->r, h->C, n_np, h->r, 4, 0) != hipSuccess)
                return fail(PIFA_ERR_HIP);
        } else {
            unsigned* dmax = nullptr;
            if (hipMalloc(&dmax, sizeof(unsigned)) != hipSuccess) return fail(PIFA_ERR_OOM);
            unsigned bits = 0;
            bool ok = hipMemset(dmax, 0, sizeof(unsigned)) == hipSuccess;
            const int64_t n = n_np * h->r;
            if (ok) {
                hipLaunchKernelGGL(absmax_bf16, dim3((unsigned)std::min<int64_t>(ceil_div(n, 256), 4096)),
                                   dim3(256), 0, 0, (const uint16_t*)C, n, dmax);
                ok = hipGetLastError() == hipSuccess &&
                     hipMemcpy(&bits, dmax, sizeof(unsigned), hipMemcpyDeviceToHost) == hipSuccess;
            }
            (void)hipFree(dmax);
            if (!ok) return fail(PIFA_ERR_HIP);
            // scale so that max|C| * 2^c_log2 lies in [2^14, 2^15)
            int c_log2 = 0;
            if (bits != 0) {
                const float mx = __builtin_bit_cast(float, bits << 16);
                c_log2 = 14 - (int)std::floor(std::log2((double)mx));
                c_log2 = std::max(-30, std::min(30, c_log2));
            }
            h->c_log2 = c_log2;
            const int64_t total = n_np * h->r_pad;
            hipLaunchKernelGGL(bf16_to_f16_scaled,
                               dim3((unsigned)std::min<int64_t>(ceil_div(total, 256), 65536)), dim3(256),
                               0, 0, (const uint16_t*)C, n_np, h->r, (f16*)h->C, n_np, h->r_pad,
                               std::ldexp(1.0f, c_log2));
            if (hipGetLastError() != hipSuccess) return fail(PIFA_ERR_HIP);
        }
    }
    if (hipDeviceSynchronize() != hipSuccess) return fail(PIFA_ERR_HIP);
    *out = h;
    return PIFA_OK;
}

pifa_status pifa_layer_destroy(pifa_handle h) {
    if (!h) return PIFA_OK;
    (void)hipDeviceSynchronize();
    free_layer(h);
    return PIFA_OK;
}

pifa_status pifa_layer_reserve(pifa_handle h, int64_t max_M) {
    if (!h || max_M < 0) return PIFA_ERR_INVALID_ARG;
    pifa_status s = pifa_prepare(h, max_M, 0);
    if (s == PIFA_OK && max_M > kDecodeMaxM) s = pifa_prepare(h, kDecodeMaxM, 0);
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
    if (h->dtype == PIFA_BF16 && !aligned16(X)) return PIFA_ERR_UNSUPPORTED;
    hipStream_t st = as_stream(stream);
    pifa_status s = pifa_prepare(h, M, st);
    if (s != PIFA_OK) return s;
    hipError_t e;

    if (h->dtype == PIFA_F32) {
        float* yp = (float*)h->ws.ptr;
        e = launch_gemm_f32((const float*)X, h->d_in, M, (const float*)h->Wp, h->d_in, h->r, h->d_in,
                            make_epi<float, kWsF32>((float*)Y, h->d_out, h->piv, h->r, 1.f, yp, h->r,
                                                    h->r, 1.f, nullptr, M),
                            st);
        if (e != hipSuccess) return PIFA_ERR_HIP;
        if (h->n_np > 0) {
            e = launch_gemm_f32(yp, h->r, M, (const float*)h->C, h->r, h->n_np, h->r,
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
        float* yp = (float*)h->ws.ptr;
        e = launch_skinny<bf16>(ALoad16<bf16>{(const bf16*)X, h->d_in, M}, (const bf16*)h->Wp, h->d_in,
                                h->r_pad, h->d_in, h->split,
                                make_epi<bf16, kWsF32>((bf16*)Y, h->d_out, h->piv, h->r, 1.f, yp,
                                                       h->r_pad, h->r_pad, y_scale, h->overflow, M),
                                st);
        if (e != hipSuccess) return PIFA_ERR_HIP;
        if (h->n_np > 0) {
            e = launch_skinny<f16>(ASplit32<f16>{yp, h->r_pad, M, y_scale}, (const f16*)h->C, h->r_pad,
                                   h->n_np, h->r_pad, h->split,
                                   make_epi<bf16, kWsNone>((bf16*)Y, h->d_out, h->npiv, h->n_np,
                                                           out_scale, nullptr, 0, 0, 1.f, nullptr, M),
                                   st);
            if (e != hipSuccess) return PIFA_ERR_HIP;
        }
        return PIFA_OK;
    }

    f16* yp = (f16*)h->ws.ptr;
    e = launch_gemm<bf16>((const bf16*)X, h->d_in, M, (const bf16*)h->Wp, h->d_in, h->r_pad, h->d_in,
                          make_epi<bf16, kWsF16>((bf16*)Y, h->d_out, h->piv, h->r, 1.f, yp, h->r_pad,
                                                 h->r_pad, y_scale, h->overflow, M),
                          st);
    if (e != hipSuccess) return PIFA_ERR_HIP;
    if (h->n_np > 0) {
        e = launch_gemm<f16>(yp, h->r_pad, M, (const f16*)h->C, h->r_pad, h->n_np, h->r_pad,
                             make_epi<bf16, kWsNone>((bf16*)Y, h->d_out, h->npiv, h->n_np, out_scale,
                                                     nullptr, 0, 0, 1.f, nullptr, M),
                             st);
        if (e != hipSuccess) return PIFA_ERR_HIP;
    }
    return PIFA_OK;
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
    hipError_t e;
    if (dtype == PIFA_F32) {
        e = launch_gemm_f32((const float*)X, d_in, M, (const float*)W, d_in, d_out, d_in,
                            make_epi<float, kWsNone>((float*)Y, d_out, nullptr, d_out, 1.f, nullptr,
                                                     0, 0, 1.f, nullptr, M),
                            st);
        return e == hipSuccess ? PIFA_OK : PIFA_ERR_HIP;
    }
    auto epi = make_epi<bf16, kWsNone>((bf16*)Y, d_out, nullptr, d_out, 1.f, nullptr, 0, 0, 1.f,
                                       nullptr, M);
    if (M <= kDecodeMaxM) {
        int dev = 0;
        PIFA_HIP(hipGetDevice(&dev));
        DeviceScratch& ds = device_scratch(dev);
        std::lock_guard<std::mutex> g(ds.mu);
        s = ds.split.ensure(skinny_plan(d_out, d_in), st);
        if (s != PIFA_OK) return s;
        e = launch_skinny<bf16>(ALoad16<bf16>{(const bf16*)X, d_in, M}, (const bf16*)W, d_in, d_out,
                                d_in, ds.split, epi, st);
        return e == hipSuccess ? PIFA_OK : PIFA_ERR_HIP;
    }
    e = launch_gemm<bf16>((const bf16*)X, d_in, M, (const bf16*)W, d_in, d_out, d_in, epi, st);
    return e == hipSuccess ? PIFA_OK : PIFA_ERR_HIP;
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
    s = ds.inter.ensure(lowrank_ws_bytes(dtype, M, dims.r), st);
    if (s != PIFA_OK) return s;
    if (dtype == PIFA_BF16 && M <= kDecodeMaxM) {
        s = ds.split.ensure(skinny_plan(dims.r, dims.d_in), st);
        if (s == PIFA_OK) s = ds.split.ensure(skinny_plan(dims.d_out, dims.r), st);
        if (s != PIFA_OK) return s;
    }
    return lowrank_run(dtype, U, V, X, Y, M, dims.d_in, dims.d_out, dims.r, ds.inter.ptr, ds.split, st);
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
    h->r_pad = dtype == PIFA_BF16 ? round_up(dims.r, kRowPad) : dims.r;
    auto fail = [&](pifa_status st) {
        free_lowrank(h);
        return st;
    };
    if (hipGetDevice(&h->device) != hipSuccess) return fail(PIFA_ERR_HIP);
    if (hipDeviceSynchronize() != hipSuccess) return fail(PIFA_ERR_HIP);
    const size_t es = esize(dtype);
    if (hipMalloc(&h->U, (size_t)h->d_out * h->r_pad * es) != hipSuccess) return fail(PIFA_ERR_OOM);
    if (hipMalloc(&h->V, (size_t)h->r_pad * h->d_in * es) != hipSuccess) return fail(PIFA_ERR_OOM);
    if (launch_pack_bits(U, h->d_out, h->r, h->r, h->U, h->d_out, h->r_pad, es, 0) != hipSuccess ||
        launch_pack_bits(V, h->r, h->d_in, h->d_in, h->V, h->r_pad, h->d_in, es, 0) != hipSuccess)
        return fail(PIFA_ERR_HIP);
    if (hipDeviceSynchronize() != hipSuccess) return fail(PIFA_ERR_HIP);
    *out = h;
    return PIFA_OK;
}

pifa_status lowrank_layer_reserve(lowrank_handle h, int64_t max_M) {
    if (!h || max_M < 0) return PIFA_ERR_INVALID_ARG;
    const int64_t m = std::max<int64_t>(max_M, kDecodeMaxM);
    pifa_status s = h->ws.ensure(std::max(lowrank_ws_bytes(h->dtype, m, h->r_pad),
                                          lowrank_ws_bytes(h->dtype, kDecodeMaxM, h->r_pad)),
                                 0);
    if (s == PIFA_OK && h->dtype == PIFA_BF16) {
        s = h->split.ensure(skinny_plan(h->r_pad, h->d_in), 0);
        if (s == PIFA_OK) s = h->split.ensure(skinny_plan(h->d_out, h->r_pad), 0);
    }
    if (s != PIFA_OK) return s;
    return hipDeviceSynchronize() == hipSuccess ? PIFA_OK : PIFA_ERR_HIP;
}

pifa_status lowrank_layer_forward(lowrank_handle h, const void* X, void* Y, int64_t M, void* stream) {
    if (!h || M < 0) return PIFA_ERR_INVALID_ARG;
    if (M == 0) return PIFA_OK;
    if (!X || !Y) return PIFA_ERR_INVALID_ARG;
    if (h->dtype == PIFA_BF16 && !aligned16(X)) return PIFA_ERR_UNSUPPORTED;
    hipStream_t st = as_stream(stream);
    pifa_status s = h->ws.ensure(lowrank_ws_bytes(h->dtype, M, h->r_pad), st);
    if (s != PIFA_OK) return s;
    if (h->dtype == PIFA_BF16 && M <= kDecodeMaxM) {
        s = h->split.ensure(skinny_plan(h->r_pad, h->d_in), st);
        if (s == PIFA_OK) s = h->split.ensure(skinny_plan(h->d_out, h->r_pad), st);
        if (s != PIFA_OK) return s;
    }
    return lowrank_run(h->dtype, h->U, h->V, X, Y, M, h->d_in, h->d_out, h->r_pad, h->ws.ptr, h->split,
                       st);
}

pifa_status lowrank_layer_destroy(lowrank_handle h) {
    if (!h) return PIFA_OK;
    (void)hipDeviceSynchronize();
    free_lowrank(h);
    return PIFA_OK;
}

}  // extern "C"
