// PIFA build on the GPU (Algorithm "Pivoting Factorization", Sec. 3.2), fp64.
//
// QR with column pivoting (Businger & Golub) on A = W'^T: column j of A is
// row j of W', so A is held as d_out contiguous columns of length d_in -- the
// bytes of W' in row-major order.  Step k picks the column of largest
// residual norm (ties to the lowest original row index), swaps it into
// position k and turns A[k:, k] into a Householder reflector H = I - tau v v^T
// (v[0] = 1 implicit, v[1:] stored below the diagonal, R[k][k] on it); the
// steps run in panels whose trailing update is one GEMM (qr_panel_* below).
// After r steps R11 (r x r, upper triangular) and R12 (r x (d_out - r)) sit in
// the first r entries of the columns.  The coefficient matrix solves
// W_p^T C^T = W_np^T in the least-squares sense through those factors:
// C R11^T = R12^T (row by row a back substitution), done by
// coeff_solve in blocks of 64 unknowns, each workgroup owning 64 rows of C.
#pragma once

#include "common.hpp"

namespace pifa {

constexpr int kBuildThreads = 1024;

// Cross-lane moves on the VALU (DPP) instead of the LDS crossbar that
// __shfl_xor uses.  dpp<CTRL, ROWS>(x, old): lane l gets x from the lane CTRL
// names; lanes of rows outside the ROWS mask get old.  Controls used:
// quad_perm [1,0,3,2] (0xB1) and [2,3,0,1] (0x4E), row_ror:4 (0x124) and
// :8 (0x128), row_bcast:15 (0x142) and :31 (0x143).
template <int CTRL, int ROWS = 0xF>
__device__ __forceinline__ uint32_t dpp32(uint32_t x, uint32_t old) {
    return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)x, CTRL, ROWS, 0xF, false);
}
template <int CTRL, int ROWS = 0xF>
__device__ __forceinline__ double dpp64(double x, double old) {
    const uint2 u = __builtin_bit_cast(uint2, x), o = __builtin_bit_cast(uint2, old);
    const uint2 r = {dpp32<CTRL, ROWS>(u.x, o.x), dpp32<CTRL, ROWS>(u.y, o.y)};
    return __builtin_bit_cast(double, r);
}
__device__ __forceinline__ double lane63(double x) {
    const uint2 u = __builtin_bit_cast(uint2, x);
    const uint2 r = {(uint32_t)__builtin_amdgcn_readlane((int)u.x, 63), (uint32_t)__builtin_amdgcn_readlane((int)u.y, 63)};
    return __builtin_bit_cast(double, r);
}

// The sum of x over the wave's 64 lanes (every lane active), returned to
// every lane: a butterfly within each quad and each row of 16 lanes, then the
// rows folded into lane 63.  A fixed order, so the result is deterministic,
// and equal inputs give equal sums.  (About 4x faster than the same
// reduction through __shfl_xor, which moves doubles through the LDS
// crossbar: the 17 sums of a pivot step took 22 K of its 49 K cycles.)
__device__ __forceinline__ double wave_sum(double x) {
    x += dpp64<0xB1>(x, 0.0);
    x += dpp64<0x4E>(x, 0.0);
    x += dpp64<0x124>(x, 0.0);
    x += dpp64<0x128>(x, 0.0);
    x += dpp64<0x142, 0xA>(x, 0.0);  // rows 1 and 3 add rows 0 and 2
    x += dpp64<0x143, 0xC>(x, 0.0);  // rows 2 and 3 add rows 0 + 1
    return lane63(x);
}

// A (d_out columns of length d_in) = W' rows; norm2[j] = ||A_j||^2; perm[j] = j.
__global__ __launch_bounds__(256) void qr_init(const double* __restrict__ W, double* __restrict__ A,
                                               double* __restrict__ norm2, int32_t* __restrict__ perm,
                                               int64_t d_out, int64_t d_in) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t j = (int64_t)blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
    if (j >= d_out) return;
    const double* w = W + j * d_in;
    double* a = A + j * d_in;
    double s = 0.0;
    for (int64_t i = lane; i < d_in; i += kWave) {
        const double x = w[i];
        a[i] = x;
        s += x * x;
    }
    s = wave_sum(s);
    if (lane == 0) {
        norm2[j] = s;
        perm[j] = (int32_t)j;
    }
}

// The pivoting runs in panels of at most kPanel steps (the blocked form of
// LAPACK's xGEQP3 / xLAQPS): inside a panel the trailing columns are not
// updated; each step k = k0 + j instead adds a column to
//   F (d_out x kPanel, row c at F + c * kPanel):  F[c, j] = tau_k a_c^(k)T v_k,
// where a_c^(k) = a_c - V[:, 0:j] F[c, 0:j]^T is column c after the panel's
// earlier reflections and V holds their Householder vectors (stored in
// A's columns k0 .. k-1 below the diagonal, with an implicit 1 on it).  Row k
// of every trailing column is brought up to date at its step (it becomes
// row k of R), and the residual norms are downdated by that row's squares.
// At the end of a panel one GEMM, A[rows >= k0+nb, cols >= k0+nb] -= V F^T,
// applies the panel's reflections to the rest of the trailing matrix, and
// the residual norms of the trailing columns are recomputed exactly, so every
// panel starts from exact norms.  The trailing matrix is read once per step
// and written once per panel, instead of read twice and written once per
// step.
constexpr int kPanel = 16;

// One step of a wave argmax over (value v, key k, index i): take the partner
// lane's triple (dpp64 / dpp32 with control CTRL, rows ROWS; lanes outside
// ROWS see their own) if its value is larger, or equal with a smaller key.
template <int CTRL, int ROWS>
__device__ __forceinline__ void argmax_step(double& v, int32_t& k, int32_t& i) {
    const double ov = dpp64<CTRL, ROWS>(v, v);
    const int32_t ok = (int32_t)dpp32<CTRL, ROWS>((uint32_t)k, (uint32_t)k);
    const int32_t oi = (int32_t)dpp32<CTRL, ROWS>((uint32_t)i, (uint32_t)i);
    if (ov > v || (ov == v && ok < k)) {
        v = ov;
        k = ok;
        i = oi;
    }
}

// The pivot of step k, for a workgroup of kBuildThreads threads (all of them
// call it): the column c in [k, d_out) of largest norm2[c], ties to the
// lowest original index perm[c].  The comparison is a total order, so the
// result is exact whatever the reduction order.
__device__ __forceinline__ int64_t block_pivot(const double* __restrict__ norm2, const int32_t* __restrict__ perm,
                                               int64_t k, int64_t d_out, double* s_val, int64_t* s_idx,
                                               int32_t* s_key) {
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    double bv = -1.0;
    int64_t bi = -1;
    int32_t bk = INT32_MAX;
    for (int64_t c = k + tid; c < d_out; c += kBuildThreads) {
        const double v = norm2[c];
        const int32_t key = perm[c];
        if (v > bv || (v == bv && key < bk)) {
            bv = v;
            bi = c;
            bk = key;
        }
    }
    {   // the wave's best (value, key, index), on the VALU; a total order
        // (larger value, then smaller key), so the result is exact
        int32_t bi32 = (int32_t)bi;
        argmax_step<0xB1, 0xF>(bv, bk, bi32);
        argmax_step<0x4E, 0xF>(bv, bk, bi32);
        argmax_step<0x124, 0xF>(bv, bk, bi32);
        argmax_step<0x128, 0xF>(bv, bk, bi32);
        argmax_step<0x142, 0xA>(bv, bk, bi32);
        argmax_step<0x143, 0xC>(bv, bk, bi32);
        bv = lane63(bv);
        bk = __builtin_amdgcn_readlane(bk, 63);
        bi = (int64_t)__builtin_amdgcn_readlane(bi32, 63);
    }
    if (lane == 0) {
        s_val[wave] = bv;
        s_idx[wave] = bi;
        s_key[wave] = bk;
    }
    __syncthreads();
    if (tid == 0) {
        for (int w = 1; w < kBuildThreads / kWave; ++w)
            if (s_val[w] > bv || (s_val[w] == bv && s_key[w] < bk)) {
                bv = s_val[w];
                bi = s_idx[w];
                bk = s_key[w];
            }
        s_idx[0] = bi;
    }
    __syncthreads();
    return s_idx[0];
}

// Step k = k0 + j, part 1 (a single workgroup of kBuildThreads threads):
//   * pivot: the column of largest (downdated) residual norm, ties to the
//     lowest original index; swap it into position k (A columns, F rows,
//     norms, perm);
//   * bring column k's rows [k, d_in) up to date: a_k -= V[:, 0:j] F[k, 0:j]^T;
//   * turn a_k[k:] into a Householder reflector (R[k][k] on the diagonal,
//     v[1:] below it, tau[k]);
//   * aux[t] = -tau_k V[k:, t]^T v_k for t < j (for F's recurrence).
// status[0] is set to 1 if the pivot column is zero.
__global__ __launch_bounds__(kBuildThreads) void qr_panel_pivot(double* __restrict__ A, double* __restrict__ norm2,
                                                                int32_t* __restrict__ perm, double* __restrict__ F,
                                                                double* __restrict__ tau, double* __restrict__ aux,
                                                                int* __restrict__ status, int64_t k, int64_t k0,
                                                                int64_t d_out, int64_t d_in) {
    __shared__ double s_val[kBuildThreads / kWave];
    __shared__ int64_t s_idx[kBuildThreads / kWave];
    __shared__ int32_t s_key[kBuildThreads / kWave];
    __shared__ double fk[kPanel];
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int j = (int)(k - k0);

    const int64_t p = block_pivot(norm2, perm, k, d_out, s_val, s_idx, s_key);

    // swap columns k and p, with their F rows, norms and original indices
    if (p != k) {
        double* ak = A + k * d_in;
        double* ap = A + p * d_in;
        for (int64_t i = tid; i < d_in; i += kBuildThreads) {
            const double t = ak[i];
            ak[i] = ap[i];
            ap[i] = t;
        }
        if (tid < j) {
            const double t = F[k * kPanel + tid];
            F[k * kPanel + tid] = F[p * kPanel + tid];
            F[p * kPanel + tid] = t;
        }
        if (tid == 0) {
            const int32_t tp = perm[k];
            perm[k] = perm[p];
            perm[p] = tp;
            const double tn = norm2[k];
            norm2[k] = norm2[p];
            norm2[p] = tn;
        }
    }
    __syncthreads();
    if (tid < kPanel) fk[tid] = tid < j ? F[k * kPanel + tid] : 0.0;
    __syncthreads();

    // One pass over rows [k, d_in) of column k and of the panel's earlier
    // reflectors V[:, 0:j] (a row's j values loaded together): the column
    // after those reflections, x[i] = a_k[i] - V[i, 0:j] fk, its squared
    // norm, and dot[t] = sum_{i > k} V[i, t] x[i] for the aux vector.
    double* x = A + k * d_in;
    double s = 0.0;
    double dot[kPanel];
#pragma unroll
    for (int t = 0; t < kPanel; ++t) dot[t] = 0.0;
    for (int64_t i = k + tid; i < d_in; i += kBuildThreads) {
        double vrow[kPanel];
#pragma unroll
        for (int t = 0; t < kPanel; ++t) vrow[t] = t < j ? A[(k0 + t) * d_in + i] : 0.0;
        double v = x[i];
#pragma unroll
        for (int t = 0; t < kPanel; ++t) v -= vrow[t] * fk[t];  // zero past j
        x[i] = v;
        s += v * v;
        if (i > k) {
#pragma unroll
            for (int t = 0; t < kPanel; ++t) dot[t] += vrow[t] * v;
        }
    }
    __shared__ double s_dot[kBuildThreads / kWave][kPanel + 1];
    s = wave_sum(s);
#pragma unroll
    for (int t = 0; t < kPanel; ++t) {
        const double d = wave_sum(dot[t]);
        if (lane == 0) s_dot[wave][t] = d;
    }
    if (lane == 0) s_val[wave] = s;
    __syncthreads();
    if (tid == 0) {
        double t = 0.0;
        for (int w = 0; w < kBuildThreads / kWave; ++w) t += s_val[w];
        s_val[0] = t;
    }
    if (tid < j) {
        double d = 0.0;
        for (int w = 0; w < kBuildThreads / kWave; ++w) d += s_dot[w][tid];
        s_dot[0][tid] = d;
    }
    __syncthreads();
    const double xnorm = sqrt(s_val[0]);
    const double alpha = x[k];
    if (xnorm == 0.0) {
        if (tid == 0) {
            status[0] = 1;
            tau[k] = 0.0;
        }
        if (tid < j) aux[tid] = 0.0;
        return;
    }
    const double beta = -copysign(xnorm, alpha);
    const double tk = (beta - alpha) / beta;
    const double inv = 1.0 / (alpha - beta);
    for (int64_t i = k + 1 + tid; i < d_in; i += kBuildThreads) x[i] *= inv;
    // aux[t] = -tau_k V[k:, t]^T v_k = -tau_k (V[k, t] + inv * dot[t]), v_k[k] = 1
    if (tid < j) aux[tid] = -tk * (A[(k0 + tid) * d_in + k] + inv * s_dot[0][tid]);
    __syncthreads();  // every thread read alpha = x[k] above
    if (tid == 0) {
        x[k] = beta;
        tau[k] = tk;
    }
}

// qr_panel_pivot with fewer dependent memory round trips, for columns of at
// most kPivotLdsRows rows (longer columns take qr_panel_pivot): the pivot
// column is read where it is (position p) in the same pass that moves the old
// column k there and brings the pivot column up to date; the updated rows
// wait in LDS (dynamic, (d_in - k) doubles) until they are scaled into the
// reflector, and alpha = x[k] is read from there.  The arithmetic and its
// order are those of qr_panel_pivot, so the results are bit-identical.
// (64 KB of dynamic LDS at most.)
constexpr int64_t kPivotLdsRows = 8192;

__global__ __launch_bounds__(kBuildThreads) void qr_panel_pivot_lds(double* __restrict__ A, double* __restrict__ norm2,
                                                                    int32_t* __restrict__ perm, double* __restrict__ F,
                                                                    double* __restrict__ tau, double* __restrict__ aux,
                                                                    int* __restrict__ status, int64_t k, int64_t k0,
                                                                    int64_t d_out, int64_t d_in) {
    __shared__ double s_val[kBuildThreads / kWave];
    __shared__ int64_t s_idx[kBuildThreads / kWave];
    __shared__ int32_t s_key[kBuildThreads / kWave];
    __shared__ double fk[kPanel];
    extern __shared__ double pcol[];  // rows [k, d_in) of the updated pivot column
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int j = (int)(k - k0);

    const int64_t p = block_pivot(norm2, perm, k, d_out, s_val, s_idx, s_key);

    // columns k and p trade F rows, norms and original indices; fk is the
    // pivot column's F row
    if (tid < kPanel) {
        const double fp = tid < j ? F[p * kPanel + tid] : 0.0;
        fk[tid] = fp;
        if (p != k && tid < j) {
            const double fo = F[k * kPanel + tid];
            F[k * kPanel + tid] = fp;
            F[p * kPanel + tid] = fo;
        }
    }
    if (tid == 0 && p != k) {
        const int32_t tp = perm[k];
        perm[k] = perm[p];
        perm[p] = tp;
        const double tn = norm2[k];
        norm2[k] = norm2[p];
        norm2[p] = tn;
    }
    double* x = A + k * d_in;
    double* ap = A + p * d_in;
    if (p != k) {  // rows above k (entries of R) swap as they are
        for (int64_t i = tid; i < k; i += kBuildThreads) {
            const double t = x[i];
            x[i] = ap[i];
            ap[i] = t;
        }
    }
    __syncthreads();  // fk

    // one pass over rows [k, d_in): the pivot column after the panel's
    // reflections, x[i] = a_p[i] - V[i, 0:j] fk (to LDS), its squared norm
    // and dot[t] = sum_{i > k} V[i, t] x[i]; the old column k moves to p
    double s = 0.0;
    double dot[kPanel];
#pragma unroll
    for (int t = 0; t < kPanel; ++t) dot[t] = 0.0;
    for (int64_t i = k + tid; i < d_in; i += kBuildThreads) {
        double vrow[kPanel];
#pragma unroll
        for (int t = 0; t < kPanel; ++t) vrow[t] = t < j ? A[(k0 + t) * d_in + i] : 0.0;
        double v = ap[i];
        if (p != k) ap[i] = x[i];
#pragma unroll
        for (int t = 0; t < kPanel; ++t) v -= vrow[t] * fk[t];  // zero past j
        pcol[i - k] = v;
        s += v * v;
        if (i > k) {
#pragma unroll
            for (int t = 0; t < kPanel; ++t) dot[t] += vrow[t] * v;
        }
    }
    __shared__ double s_dot[kBuildThreads / kWave][kPanel + 1];
    s = wave_sum(s);
#pragma unroll
    for (int t = 0; t < kPanel; ++t) {
        const double d = wave_sum(dot[t]);
        if (lane == 0) s_dot[wave][t] = d;
    }
    if (lane == 0) s_val[wave] = s;
    __syncthreads();
    if (tid == 0) {
        double t = 0.0;
        for (int w = 0; w < kBuildThreads / kWave; ++w) t += s_val[w];
        s_val[0] = t;
    }
    if (tid < j) {
        double d = 0.0;
        for (int w = 0; w < kBuildThreads / kWave; ++w) d += s_dot[w][tid];
        s_dot[0][tid] = d;
    }
    __syncthreads();
    const double xnorm = sqrt(s_val[0]);
    const double alpha = pcol[0];
    if (xnorm == 0.0) {
        for (int64_t i = k + tid; i < d_in; i += kBuildThreads) x[i] = pcol[i - k];
        if (tid == 0) {
            status[0] = 1;
            tau[k] = 0.0;
        }
        if (tid < j) aux[tid] = 0.0;
        return;
    }
    const double beta = -copysign(xnorm, alpha);
    const double tk = (beta - alpha) / beta;
    const double inv = 1.0 / (alpha - beta);
    for (int64_t i = k + 1 + tid; i < d_in; i += kBuildThreads) x[i] = pcol[i - k] * inv;
    // aux[t] = -tau_k V[k:, t]^T v_k = -tau_k (V[k, t] + inv * dot[t]), v_k[k] = 1
    if (tid < j) aux[tid] = -tk * (A[(k0 + tid) * d_in + k] + inv * s_dot[0][tid]);
    if (tid == 0) {
        x[k] = beta;
        tau[k] = tk;
    }
}

// Step k = k0 + j, part 2: one wave per trailing column c > k, read only
// except for three values per column:
//   F[c, j]  = tau_k a_c^T v_k + F[c, 0:j] aux[0:j]  (a_c as of the panel start)
//   R[k][c]  = a_c[k] - V[k, 0:j] F[c, 0:j]^T - F[c, j]   (written to a_c[k])
//   norm2[c] -= R[k][c]^2
__global__ __launch_bounds__(256) void qr_panel_gemv(double* __restrict__ A, double* __restrict__ norm2,
                                                     double* __restrict__ F, const double* __restrict__ tau,
                                                     const double* __restrict__ aux, int64_t k, int64_t k0,
                                                     int64_t d_out, int64_t d_in) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t c = k + 1 + (int64_t)blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
    if (c >= d_out) return;
    const int j = (int)(k - k0);
    const double* v = A + k * d_in;  // v[k] = 1 (implicit), v[k+1:] stored
    double* a = A + c * d_in;
    double d;
    if ((d_in & 1) == 0) {
        // 16-byte loads of rows [s2, d_in), s2 = k + 1 rounded up to even,
        // four pairs in flight per lane (clamped indices, masked products: no
        // branch per load); row k + 1 on its own when it is odd.  The order
        // depends only on k, so equal columns give equal sums.
        const int64_t s = k + 1, s2 = s + (s & 1), n2 = d_in / 2;
        const double2* v2 = reinterpret_cast<const double2*>(v);
        const double2* a2 = reinterpret_cast<const double2*>(a);
        double acc[8] = {0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0};
        for (int64_t q = s2 / 2 + lane; q < n2; q += 4 * kWave) {
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int64_t qu = q + u * kWave;
                const bool ok = qu < n2;
                const int64_t qc = ok ? qu : n2 - 1;
                const double2 vv = v2[qc], aa = a2[qc];
                acc[2 * u] += ok ? vv.x * aa.x : 0.0;
                acc[2 * u + 1] += ok ? vv.y * aa.y : 0.0;
            }
        }
        d = ((acc[0] + acc[1]) + (acc[2] + acc[3])) + ((acc[4] + acc[5]) + (acc[6] + acc[7]));
        if (lane == 0 && (s & 1) && s < d_in) d += v[s] * a[s];
    } else {
        double d1 = 0.0, d2 = 0.0;
        int64_t i = k + 1 + lane;
        for (; i + kWave < d_in; i += 2 * kWave) {
            d1 += v[i] * a[i];
            d2 += v[i + kWave] * a[i + kWave];
        }
        if (i < d_in) d1 += v[i] * a[i];
        d = d1 + d2;
    }
    const double akc = a[k];
    d = wave_sum(d) + akc;
    double* Fc = F + c * kPanel;
    double corr = 0.0, row = 0.0;
    if (lane < j) {
        const double f = Fc[lane];
        corr = f * aux[lane];
        row = A[(k0 + lane) * d_in + k] * f;
    }
    corr = wave_sum(corr);
    row = wave_sum(row);
    if (lane == 0) {
        const double f = tau[k] * d + corr;
        Fc[j] = f;
        const double rkc = akc - row - f;
        a[k] = rkc;
        norm2[c] = fmax(norm2[c] - rkc * rkc, 0.0);
    }
}

// Exact residual norms ||A_c[k:]||^2 of columns c >= k (one wave per column).
__global__ __launch_bounds__(256) void qr_norms(const double* __restrict__ A, double* __restrict__ norm2, int64_t k,
                                                int64_t d_out, int64_t d_in) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t c = k + (int64_t)blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
    if (c >= d_out) return;
    const double* a = A + c * d_in;
    double s = 0.0;
    for (int64_t i = k + lane; i < d_in; i += kWave) s += a[i] * a[i];
    s = wave_sum(s);
    if (lane == 0) norm2[c] = s;
}

// diag[k] = R[k][k] = A_k[k] for k < r.
__global__ void extract_diag(const double* __restrict__ A, double* __restrict__ diag, int64_t r, int64_t d_in) {
    for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < r; k += (int64_t)gridDim.x * blockDim.x)
        diag[k] = A[k * d_in + k];
}

// R11 in row-major form: RT[s][t] = A_t[s] for s <= t < r, 0 below.
__global__ void extract_r11(const double* __restrict__ A, double* __restrict__ RT, int64_t r, int64_t d_in) {
    const int64_t total = r * r;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t s = e / r, t = e % r;
        RT[e] = t >= s ? A[t * d_in + s] : 0.0;
    }
}

// C (n_np x r) with C R11^T = R12^T, i.e. for each row q of C:
//   sum_{t >= s} R11[s][t] c[t] = b[s],  b[s] = A_{r+q}[s]   (s < r),
// solved from the last unknown up in blocks of kSolveBlock unknowns,
// right-looking: X = the right-hand sides (coeff_rhs); for each block, from
// the last, coeff_block_solve finds the block's unknowns of every row by
// substitution against R11's diagonal block, and one fp64 MFMA GEMM (gemm64)
// subtracts their contribution from the right-hand sides of all earlier
// unknowns.  The GEMMs carry the n_np r^2 FLOPs over the whole chip, where a
// left-looking solve with one workgroup per 64 rows of C kept n_np / 64
// workgroups busy (32 at 4096 x 4096, r = 2048).
constexpr int kSolveBlock = 64;

__global__ void coeff_rhs(const double* __restrict__ A, double* __restrict__ X, int64_t r, int64_t n_np,
                          int64_t d_in) {
    const int64_t total = n_np * r;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t q = e / r, s = e % r;
        X[e] = A[(r + q) * d_in + s];
    }
}

// Unknowns [s0, s0 + nb) of rows [64 b, 64 b + 64) of X, in place: thread t
// substitutes row 64 b + t against the diagonal block of R11 (upper
// triangular, row-major in RT with row stride r).
__global__ __launch_bounds__(kSolveBlock) void coeff_block_solve(const double* __restrict__ RT, double* __restrict__ X,
                                                                  int64_t r, int64_t n_np, int64_t s0, int nb) {
    __shared__ double sD[kSolveBlock][kSolveBlock + 1];
    __shared__ double sB[kSolveBlock][kSolveBlock + 1];
    const int tid = threadIdx.x;
    const int64_t q0 = (int64_t)blockIdx.x * kSolveBlock;
    for (int e = tid; e < kSolveBlock * kSolveBlock; e += kSolveBlock) {
        const int a = e / kSolveBlock, b = e % kSolveBlock;
        sD[a][b] = (a < nb && b < nb) ? RT[(s0 + a) * r + s0 + b] : 0.0;
        const int64_t q = q0 + a;
        sB[a][b] = (q < n_np && b < nb) ? X[q * r + s0 + b] : 0.0;
    }
    __syncthreads();
    for (int a = nb - 1; a >= 0; --a) {
        double v = sB[tid][a];
        for (int b = a + 1; b < nb; ++b) v -= sD[a][b] * sB[tid][b];
        sB[tid][a] = v / sD[a][a];
    }
    __syncthreads();
    for (int e = tid; e < kSolveBlock * kSolveBlock; e += kSolveBlock) {
        const int row = e / kSolveBlock, col = e % kSolveBlock;
        const int64_t q = q0 + row;
        if (q < n_np && col < nb) X[q * r + s0 + col] = sB[row][col];
    }
}

// Outputs in sorted order: W_p[i] = W'[pivot_idx[i]], and
// C_out[q][i] = C_sel[row_src[q]][col_src[i]].
__global__ void gather_rows(const double* __restrict__ W, const int32_t* __restrict__ rows, double* __restrict__ out,
                            int64_t n_rows, int64_t n_cols) {
    const int64_t total = n_rows * n_cols;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = e / n_cols, c = e % n_cols;
        out[e] = W[(int64_t)rows[i] * n_cols + c];
    }
}

__global__ void gather_coeffs(const double* __restrict__ Csel, const int32_t* __restrict__ row_src,
                              const int32_t* __restrict__ col_src, double* __restrict__ out, int64_t n_np,
                              int64_t r) {
    const int64_t total = n_np * r;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t q = e / r, i = e % r;
        out[e] = Csel[(int64_t)row_src[q] * r + col_src[i]];
    }
}

}  // namespace pifa
