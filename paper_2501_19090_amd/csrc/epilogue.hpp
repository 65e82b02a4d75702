// Epilogues shared by every GEMM/GEMV kernel.
//
// A kernel produces fp32 values acc(m, n) of a product with N columns and
// hands each one to the epilogue, which
//   * writes round(acc * out_scale) to out[m * ldo + idx[n]] for n < n_out
//     (idx == nullptr means the identity map; idx[n] < 0 means no output for
//     column n, used for the padding rows of grouped layers) -- this is the pivot /
//     non-pivot assignment of Algorithm "PIFA Layer" (its last two steps),
//     fused into the producing kernel so there is no separate permutation pass;
//   * optionally keeps a workspace copy ws[m * ldws + n] for n < n_ws, as fp16
//     times ws_scale (the bf16 path's Y_p hand-off), as fp32, or as an fp16
//     pair hi = fp16(v * ws_scale), lo = fp16(v * ws_scale - hi) in two planes
//     of M * ldws elements (the decode hand-off, about 22 significant bits).
#pragma once

#include "common.hpp"

namespace pifa {

enum WsKind { kWsNone = 0, kWsF16 = 1, kWsF32 = 2, kWsF16Pair = 3 };

template <typename TOut, int WS>
struct ScatterEpi {
    TOut* out;
    int64_t ldo;
    const int32_t* idx;  // nullptr: column n goes to output column n
    int64_t n_out;
    float out_scale;
    void* ws;
    int64_t ldws;
    int64_t n_ws;
    float ws_scale;
    int* overflow;  // fp16 hand-off overflow counter
    int64_t M;

    struct Col {
        int64_t n;
        int64_t dst;
        bool out_ok;
        bool ws_ok;
    };

    __device__ __forceinline__ Col col(int64_t n) const {
        Col c;
        c.n = n;
        c.out_ok = n < n_out;
        // A load under a condition (the lane's, or idx == nullptr) becomes a
        // branch whose join waits for it, so the index is read unconditionally
        // through a buffer resource: a clamped offset, and an empty range
        // (the load returns 0 without an access) when there is no map.
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<int32_t*>(idx), (short)0, idx ? (int)(n_out * 4) : 0, 0x00020000);
        const int32_t v = (int32_t)__builtin_amdgcn_raw_buffer_load_b32(rs, (int)((c.out_ok ? n : 0) * 4), 0, 0);
        const int64_t d = idx ? (int64_t)v : n;
        c.dst = c.out_ok ? d : 0;
        if (c.dst < 0) {  // a padding column of a grouped layer: no output
            c.out_ok = false;
            c.dst = 0;
        }
        c.ws_ok = (WS != kWsNone) && n < n_ws;
        return c;
    }

    __device__ __forceinline__ void store(int64_t m, const Col& c, float v) const {
        if (m >= M) return;
        if (c.out_ok) Store<TOut>::put(out + m * ldo + c.dst, v * out_scale);
        if constexpr (WS == kWsF16) {
            if (c.ws_ok) {
                const float s = v * ws_scale;
                const f16 h = (f16)s;
                if (!__builtin_isfinite((float)h) && __builtin_isfinite(s)) atomicAdd(overflow, 1);
                reinterpret_cast<f16*>(ws)[m * ldws + c.n] = h;
            }
        } else if constexpr (WS == kWsF16Pair) {
            if (c.ws_ok) {
                const float s = v * ws_scale;
                const f16 hi = (f16)s;
                const f16 lo = (f16)(s - (float)hi);
                if (!__builtin_isfinite((float)hi) && __builtin_isfinite(s)) atomicAdd(overflow, 1);
                f16* w = reinterpret_cast<f16*>(ws);
                w[m * ldws + c.n] = hi;
                w[(M + m) * ldws + c.n] = lo;
            }
        } else if constexpr (WS == kWsF32) {
            if (c.ws_ok) {
                reinterpret_cast<float*>(ws)[m * ldws + c.n] = v;
                // the consumer splits v * ws_scale into fp16 hi + lo
                if (overflow) {
                    const float s = v * ws_scale;
                    if (!__builtin_isfinite((float)(f16)s) && __builtin_isfinite(s)) atomicAdd(overflow, 1);
                }
            }
        }
    }
};

// Contiguous-output epilogue with 16-byte stores: out[m * ldo + n] =
// TOut(acc(m, n) * scale) for m < M, n < N.  The tile is staged in LDS as
// whole row pieces and written 8 values per store (rows 16-byte aligned:
// ldo a multiple of 8, out 16-byte aligned).  TOut is bf16 (an output) or
// f16 (the Y_p hand-off, whose overflows are counted in *overflow when it
// is not null).
template <typename TOut>
struct StagedEpi {
    static constexpr bool kStaged = true;
    uint16_t* out;
    int64_t ldo;
    int64_t N;
    float scale;
    int* overflow;
    int64_t M;

    // element-wise form, for the K-split reduction
    struct Col {
        int64_t n;
        bool ok;
    };
    __device__ __forceinline__ Col col(int64_t n) const { return Col{n, n < N}; }
    __device__ __forceinline__ uint16_t bits(float v, int& over) const {
        const float s = v * scale;
        if constexpr (__is_same(TOut, f16)) {
            const f16 h = (f16)s;
            over += !__builtin_isfinite((float)h) && __builtin_isfinite(s);
            return __builtin_bit_cast(uint16_t, h);
        } else {
            return f32_to_bf16_bits(s);
        }
    }
    __device__ __forceinline__ void store(int64_t m, const Col& c, float v) const {
        if (m >= M || !c.ok) return;
        int over = 0;
        out[m * ldo + c.n] = bits(v, over);
        if (over && overflow) atomicAdd(overflow, over);
    }
};

// The pivot product's epilogue of a bf16 prefill: the pivot outputs go to
// their columns of Y element by element (scatter), and the fp16 hand-off,
// a contiguous M x ldws matrix, is staged in LDS and written with 16-byte
// stores (on the 128-row tiles; the 256-row tiles take elementwise()).
// col / store serve the K-split reduction, element by element.
struct PivotHandoffEpi {
    static constexpr bool kDual = true;
    ScatterEpi<bf16, kWsNone> y;
    StagedEpi<f16> ws;

    struct Col {
        typename ScatterEpi<bf16, kWsNone>::Col y;
        typename StagedEpi<f16>::Col ws;
    };
    __device__ __forceinline__ Col col(int64_t n) const { return Col{y.col(n), ws.col(n)}; }
    __device__ __forceinline__ void store(int64_t m, const Col& c, float v) const {
        y.store(m, c.y, v);
        ws.store(m, c.ws, v);
    }
    // the same outputs with the hand-off written element by element (the
    // 256-row tiles: faster there than staging it through LDS)
    __host__ ScatterEpi<bf16, kWsF16> elementwise() const {
        ScatterEpi<bf16, kWsF16> e;
        e.out = y.out;
        e.ldo = y.ldo;
        e.idx = y.idx;
        e.n_out = y.n_out;
        e.out_scale = y.out_scale;
        e.ws = ws.out;
        e.ldws = ws.ldo;
        e.n_ws = ws.N;
        e.ws_scale = ws.scale;
        e.overflow = ws.overflow;
        e.M = y.M;
        return e;
    }
};

template <typename TOut, int WS>
__host__ inline ScatterEpi<TOut, WS> make_epi(TOut* out, int64_t ldo, const int32_t* idx,
                                              int64_t n_out, float out_scale, void* ws,
                                              int64_t ldws, int64_t n_ws, float ws_scale,
                                              int* overflow, int64_t M) {
    ScatterEpi<TOut, WS> e;
    e.out = out;
    e.ldo = ldo;
    e.idx = idx;
    e.n_out = n_out;
    e.out_scale = out_scale;
    e.ws = ws;
    e.ldws = ldws;
    e.n_ws = n_ws;
    e.ws_scale = ws_scale;
    e.overflow = overflow;
    e.M = M;
    return e;
}

}  // namespace pifa
