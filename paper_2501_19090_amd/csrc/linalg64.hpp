// fp64 dense linear algebra for the reconstruction solves of Sec. 4 (the
// closed-form U and V updates of Algorithm "MPIFA", Part 1).  These run once
// per layer on n x n and r x r systems; the hot part of the reconstruction is
// the accumulation of the calibration sums, which runs on the MFMA GEMM.
//
//   gemm64        C = alpha op(A) op(B) + beta C with arbitrary element strides
//                 (transposes are strides, no copies) on fp64 MFMA tiles;
//                 optional lower-triangle tiles only, for symmetric updates.
//   Cholesky      A = L L^T, right-looking in 64-column blocks: diagonal block
//                 in one workgroup's LDS, panel by forward substitution, trailing
//                 update by gemm64 (lower tiles only).
//   spd solve     L L^T X = B for many right-hand sides: blocked forward and
//                 backward substitution; each diagonal block is applied as its
//                 explicit inverse (tri_inv_blocks), so every step is a gemm64.
#pragma once

#include "common.hpp"

namespace pifa {

constexpr int kG64 = 64;  // block size of the factorisations and solves

typedef double f64x4 __attribute__((ext_vector_type(4)));

// C[i*sc0 + j*sc1] = alpha * sum_k A[i*sa0 + k*sa1] * B[k*sb0 + j*sb1] + beta * C[...]
// for i < Mr, j < Nc, on v_mfma_f64_16x16x4_f64.  LOWER: only tiles whose
// first row >= first column (tiles on the diagonal are computed whole).
// beta == 0 ignores C's old value.
// Tile BT x BT, K step BK, 16 waves in a 4 x 4 grid (1024 threads), each a
// (BT/4) x (BT/4) block of 16 x 16 MFMA outputs.  Both operands are staged
// k-major in LDS ([k][i] and [k][j]), so any stride pattern loads with the
// unit-stride axis across consecutive threads and every fragment read is
// unit-stride.  MFMA lane layout: lane l supplies A[l % 16][l / 16] and
// B[l / 16][l % 16]; element v of the result is D[4 v + l / 16][l % 16].
// Each output is one fp64 FMA chain over k in ascending order.
// Grid: (ceil(Nc / BT), ceil(Mr / BT)).
template <int BT, int BK>
__global__ __launch_bounds__(1024) void gemm64(int64_t Mr, int64_t Nc, int64_t K, double alpha,
                                               const double* __restrict__ A, int64_t sa0, int64_t sa1,
                                               const double* __restrict__ B, int64_t sb0, int64_t sb1, double beta,
                                               double* __restrict__ C, int64_t sc0, int64_t sc1, int lower) {
    constexpr int NT = 1024, LD = BT + 1, PT = BT * BK / NT;
    constexpr int WT = BT / 4, TT = WT / 16;
    static_assert(PT >= 1 && BT * BK % NT == 0 && WT % 16 == 0 && BK % 4 == 0, "bad fp64 tile");
    const int64_t i0 = (int64_t)blockIdx.y * BT, j0 = (int64_t)blockIdx.x * BT;
    if (lower && j0 > i0) return;
    __shared__ double As[2][BK * LD];
    __shared__ double Bs[2][BK * LD];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 2, wn = wave & 3;
    const bool a_k1 = sa1 == 1, b_j1 = sb1 == 1;
    // element e of a staged tile: (row ii, depth kk) of A, (depth kb, column jj) of B
    auto a_at = [&](int e, int& ii, int& kk) {
        ii = a_k1 ? e / BK : e % BT;
        kk = a_k1 ? e % BK : e / BT;
    };
    auto b_at = [&](int e, int& kb, int& jj) {
        jj = b_j1 ? e % BT : e / BK;
        kb = b_j1 ? e / BT : e % BK;
    };
    double ra[PT], rb[PT];
    auto gload = [&](int64_t k0) {
#pragma unroll
        for (int q = 0; q < PT; ++q) {
            int ii, kk, kb, jj;
            a_at(tid + NT * q, ii, kk);
            b_at(tid + NT * q, kb, jj);
            const int64_t i = i0 + ii, ka = k0 + kk, j = j0 + jj, kB = k0 + kb;
            ra[q] = (i < Mr && ka < K) ? A[i * sa0 + ka * sa1] : 0.0;
            rb[q] = (j < Nc && kB < K) ? B[kB * sb0 + j * sb1] : 0.0;
        }
    };
    auto sstore = [&](int buf) {
#pragma unroll
        for (int q = 0; q < PT; ++q) {
            int ii, kk, kb, jj;
            a_at(tid + NT * q, ii, kk);
            b_at(tid + NT * q, kb, jj);
            As[buf][kk * LD + ii] = ra[q];
            Bs[buf][kb * LD + jj] = rb[q];
        }
    };
    f64x4 acc[TT][TT];
#pragma unroll
    for (int a = 0; a < TT; ++a)
#pragma unroll
        for (int b = 0; b < TT; ++b) acc[a][b] = f64x4{0.0, 0.0, 0.0, 0.0};
    const int64_t nk = (K + BK - 1) / BK;
    gload(0);
    sstore(0);
    __syncthreads();
    const int fr = lane & 15, fk = lane >> 4;
    for (int64_t kt = 0; kt < nk; ++kt) {
        const int cur = (int)(kt & 1);
        if (kt + 1 < nk) gload((kt + 1) * BK);  // in flight during this tile's MFMAs
#pragma unroll
        for (int s = 0; s < BK / 4; ++s) {
            double fa[TT], fb[TT];
#pragma unroll
            for (int a = 0; a < TT; ++a) fa[a] = As[cur][(s * 4 + fk) * LD + wm * WT + a * 16 + fr];
#pragma unroll
            for (int b = 0; b < TT; ++b) fb[b] = Bs[cur][(s * 4 + fk) * LD + wn * WT + b * 16 + fr];
#pragma unroll
            for (int a = 0; a < TT; ++a)
#pragma unroll
                for (int b = 0; b < TT; ++b)
                    acc[a][b] = __builtin_amdgcn_mfma_f64_16x16x4f64(fa[a], fb[b], acc[a][b], 0, 0, 0);
        }
        // the other buffer was last read before the previous barrier
        if (kt + 1 < nk) sstore(cur ^ 1);
        __syncthreads();
    }
#pragma unroll
    for (int a = 0; a < TT; ++a)
#pragma unroll
        for (int b = 0; b < TT; ++b)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int64_t i = i0 + wm * WT + a * 16 + 4 * v + fk, j = j0 + wn * WT + b * 16 + fr;
                if (i < Mr && j < Nc) {
                    double* c = C + i * sc0 + j * sc1;
                    *c = beta == 0.0 ? alpha * acc[a][b][v] : fma(alpha, acc[a][b][v], beta * *c);
                }
            }
}

// *out = 1e-13 * max_i A[i][i] (n x n, row stride ld): the smallest pivot a
// factorisation accepts, i.e. a bound of about 1e13 on the condition number.
// One workgroup of 256 threads.
constexpr double kPivotTol = 1e-13;

__global__ __launch_bounds__(256) void pivot_floor64(const double* __restrict__ A, int64_t n, int64_t ld,
                                                     double* __restrict__ out) {
    __shared__ double red[256];
    double mx = 0.0;
    for (int64_t i = threadIdx.x; i < n; i += 256) mx = fmax(mx, A[i * ld + i]);
    red[threadIdx.x] = mx;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) red[threadIdx.x] = fmax(red[threadIdx.x], red[threadIdx.x + w]);
        __syncthreads();
    }
    if (threadIdx.x == 0) *out = kPivotTol * red[0];
}

// Unblocked Cholesky of the nb x nb (nb <= 64) block at A (row stride ld), in
// place (lower triangle; the upper part is left as is).  One workgroup of 256
// threads, block staged in LDS; thread (ty, tx) of a 16 x 16 grid owns rows
// ty + 16a and columns tx + 16b (a, b < 4) of the trailing update, so no
// index is divided.  Step j: every thread reads the pivot and the column
// values it needs, a barrier, then the scaled column and the rank-1 update
// are written.  *info is set to 1 on a pivot that is not finite or not above
// *floor (the matrix is not numerically positive definite).
__global__ __launch_bounds__(256) void chol_diag(double* __restrict__ A, int64_t ld, int nb,
                                                 const double* __restrict__ floor, int* __restrict__ info) {
    __shared__ double L[kG64][kG64 + 1];
    const int tid = threadIdx.x, tx = tid % 16, ty = tid / 16;
    {  // thread t loads column t % 64 of rows t / 64 + 4 k: 16 independent loads
        const int c = tid % kG64, r0 = tid / kG64;
#pragma unroll
        for (int k = 0; k < kG64 / 4; ++k) {
            const int i = r0 + 4 * k;
            if (i < nb && c < nb) L[i][c] = A[(int64_t)i * ld + c];
        }
    }
    __syncthreads();
    const double fl = *floor;
    for (int j = 0; j < nb; ++j) {
        const double d = L[j][j];
        const bool ok = d > fl && d > 0.0 && __builtin_isfinite(d);
        const double s = ok ? sqrt(d) : 1.0;
        const double inv = 1.0 / s;  // one division per step; the column is scaled by multiplication
        double li[4], lc[4];
#pragma unroll
        for (int a = 0; a < 4; ++a) {
            li[a] = L[ty + 16 * a][j] * inv;
            lc[a] = L[tx + 16 * a][j] * inv;
        }
        const double cj = tid > j && tid < nb ? L[tid][j] * inv : 0.0;
        __syncthreads();
        if (tid == 0) {
            L[j][j] = s;
            if (!ok) *info = 1;
        }
        if (tid > j && tid < nb) L[tid][j] = cj;
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                const int i = ty + 16 * a, c = tx + 16 * b;
                if (c > j && c <= i && i < nb) L[i][c] -= li[a] * lc[b];
            }
        __syncthreads();
    }
    {
        const int c = tid % kG64, r0 = tid / kG64;
#pragma unroll
        for (int k = 0; k < kG64 / 4; ++k) {
            const int i = r0 + 4 * k;
            if (i < nb && c <= i) A[(int64_t)i * ld + c] = L[i][c];
        }
    }
}

constexpr int kWin = 8;  // columns per pass of the windowed substitution

// Loads the nb x nb lower block at Ld (row stride ld) into rows [0, 64) of
// L, zero everywhere else (columns >= nb, rows >= nb up to 127), and the
// reciprocals of its diagonal into inv (zero past nb).  One wave, lane t
// loading column t (coalesced loads, all in flight at once); the caller
// synchronises.
__device__ __forceinline__ void load_lower_block(const double* __restrict__ Ld, int64_t ld, int nb,
                                                 double (&L)[2 * kG64][kG64 + 1], double (&inv)[kG64]) {
    const int t = threadIdx.x;
    const bool col_ok = t < nb;
#pragma unroll
    for (int i = 0; i < kG64; ++i) {
        const double v = Ld[(int64_t)(i < nb ? i : 0) * ld + (col_ok ? t : 0)];  // in bounds, no branch
        L[i][t] = (i < nb && col_ok) ? v : 0.0;
    }
#pragma unroll
    for (int i = kG64; i < 2 * kG64; ++i) L[i][t] = 0.0;
    inv[t] = t < nb ? 1.0 / Ld[(int64_t)t * ld + t] : 0.0;
}

// Forward substitution x <- L^-1 x for the lower block in LDS (as
// load_lower_block leaves it), one right-hand side per lane in w.  Columns
// are eliminated kWin at a time, each against every later row (the rows past
// the block read the zero padding); after a pass the kWin finished values
// go to out(j, value) and the window shifts down by kWin.  The loop body is
// the same for every pass, so its code stays in the instruction cache (a
// fully unrolled elimination is about 58 KB of straight-line code that each
// wave fetches once).  Each pass runs as (column, 16-row chunk) steps whose
// LDS reads are issued one step ahead of their FMAs, so the read latency
// hides behind the previous step (38 -> 24 us for a 4032-row panel).
template <typename Out>
__device__ __forceinline__ void lower_solve_window(const double (&L)[2 * kG64][kG64 + 1], const double (&inv)[kG64],
                                                   double (&w)[kG64], Out&& out) {
    constexpr int kSteps = kWin * 4;  // (column t, chunk c) = (s / 4, s % 4)
#pragma unroll 1
    for (int j0 = 0; j0 < kG64; j0 += kWin) {
        double buf[2][16];
        auto load = [&](int s, double (&dst)[16]) {
            const int t = s >> 2, c = s & 3;
#pragma unroll
            for (int ii = 0; ii < 16; ++ii) dst[ii] = L[j0 + 16 * c + ii][j0 + t];
        };
        load(0, buf[0]);
        double xt = 0.0;
#pragma unroll
        for (int s = 0; s < kSteps; ++s) {
            const int t = s >> 2, c = s & 3;
            if (s + 1 < kSteps) load(s + 1, buf[(s + 1) & 1]);
            if (c == 0) {
                xt = w[t] * inv[j0 + t];
                w[t] = xt;
            }
#pragma unroll
            for (int ii = 0; ii < 16; ++ii) {
                const int i = 16 * c + ii;
                if (i > t) w[i] -= buf[s & 1][ii] * xt;
            }
            // keeps the scheduler from hoisting every read of the pass above
            // the first FMA (hundreds of registers)
            __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int t = 0; t < kWin; ++t) out(j0 + t, w[t]);
#pragma unroll
        for (int i = 0; i < kG64 - kWin; ++i) w[i] = w[i + kWin];
#pragma unroll
        for (int i = kG64 - kWin; i < kG64; ++i) w[i] = 0.0;
    }
}

// Panel of a blocked Cholesky: rows [0, nrows) of P (row stride ld, 64
// columns) become P L11^-T, L11 being the 64 x 64 lower factor at Ld (row
// stride ld): row p solves L11 x = p^T.  One row per lane.  Only full
// diagonal blocks have a panel below them (a block narrower than 64 is the
// last one of its matrix).
__global__ __launch_bounds__(64) void chol_panel(const double* __restrict__ Ld, double* __restrict__ P, int64_t ld,
                                                 int64_t nrows) {
    __shared__ double L[2 * kG64][kG64 + 1];
    __shared__ double inv[kG64];
    load_lower_block(Ld, ld, kG64, L, inv);
    __syncthreads();
    const int64_t row = (int64_t)blockIdx.x * 64 + threadIdx.x;
    if (row >= nrows) return;
    double* p = P + row * ld;
    double w[kG64];
#pragma unroll
    for (int j = 0; j < kG64; ++j) w[j] = p[j];
    lower_solve_window(L, inv, w, [&](int j, double v) { p[j] = v; });
}

// Inverses of the diagonal blocks of a lower factor: block b (rows and
// columns [64 b, 64 b + nb)) of the n x n factor L (row stride ld) goes to
// Linv[b * 64 * 64 ...] as a dense 64 x 64 row-major block, zero above the
// diagonal and outside nb x nb.  One one-wave workgroup per block; lane t
// solves L_bb y = e_t, column t of the inverse.
__global__ __launch_bounds__(64) void tri_inv_blocks(const double* __restrict__ L, int64_t ld, int64_t n,
                                                     double* __restrict__ Linv) {
    __shared__ double Ls[2 * kG64][kG64 + 1];
    __shared__ double inv[kG64];
    const int64_t kb = (int64_t)blockIdx.x * kG64;
    const int nb = (int)(n - kb < kG64 ? n - kb : kG64);
    load_lower_block(L + kb * ld + kb, ld, nb, Ls, inv);
    __syncthreads();
    const int t = threadIdx.x;
    double w[kG64];
#pragma unroll
    for (int i = 0; i < kG64; ++i) w[i] = (i == t && t < nb) ? 1.0 : 0.0;
    double* out = Linv + (int64_t)blockIdx.x * kG64 * kG64;
    lower_solve_window(Ls, inv, w, [&](int j, double v) { out[j * kG64 + t] = v; });
}

// out = a * X + b * Y + d * I (n x n row-major; Y may be null, then b is ignored)
__global__ void axpby_diag64(int64_t n, double a, const double* __restrict__ X, double b, const double* __restrict__ Y,
                             double d, double* __restrict__ out) {
    const int64_t total = n * n;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
        double v = a * X[e];
        if (Y) v += b * Y[e];
        if (e / n == e % n) v += d;
        out[e] = v;
    }
}

// out (cols x rows) = in^T (rows x cols), fp64, 32 x 32 LDS tiles.
__global__ __launch_bounds__(256) void transpose64(const double* __restrict__ in, int64_t rows, int64_t cols,
                                                   double* __restrict__ out) {
    __shared__ double t[32][33];
    const int64_t r0 = (int64_t)blockIdx.y * 32, c0 = (int64_t)blockIdx.x * 32;
    const int tx = threadIdx.x % 32, ty = threadIdx.x / 32;
    for (int k = ty; k < 32; k += 8) {
        const int64_t r = r0 + k, c = c0 + tx;
        t[k][tx] = (r < rows && c < cols) ? in[r * cols + c] : 0.0;
    }
    __syncthreads();
    for (int k = ty; k < 32; k += 8) {
        const int64_t c = c0 + k, r = r0 + tx;
        if (c < cols && r < rows) out[c * rows + r] = t[tx][k];
    }
}

// Epilogue for the MFMA GEMM: out[m * ld + n] += acc (the running fp64 sums
// of the calibration statistics; fp32 products are accumulated in fp64).
// With lower_tiles, output tiles entirely above the diagonal are skipped (a
// symmetric sum; symmetrize_lower64 fills them afterwards).
struct AccF64Epi {
    double* out;
    int64_t ld, N, M;
    bool lower_tiles;
    __device__ __forceinline__ bool skip_tile(int64_t m0, int64_t n0, int BM, int BN) const {
        (void)BN;
        return lower_tiles && n0 >= m0 + BM;
    }
    struct Col {
        int64_t n;
        bool ok;
    };
    __device__ __forceinline__ Col col(int64_t n) const { return Col{n, n < N}; }
    __device__ __forceinline__ void store(int64_t m, const Col& c, float v) const {
        if (m < M && c.ok) out[m * ld + c.n] += (double)v;
    }
};


// S[i][j] = S[j][i] for i < j (n x n row-major): completes a sum of which only
// the lower triangle (and whole diagonal tiles) was accumulated.
__global__ void symmetrize_lower64(double* __restrict__ S, int64_t n) {
    const int64_t total = n * n;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = e / n, j = e % n;
        if (i < j) S[e] = S[j * n + i];
    }
}

}  // namespace pifa
