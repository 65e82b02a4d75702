/*
 * PIFA oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, fp64 CPU implementation of Pivoting Factorization
 * (Zhao, Zhang & Cannistraci, arXiv 2501.19090).  Only the test suite, the
 * smoke check and the benchmark's CPU-baseline leg may load this library.
 * It shares no code, header, table or helper with the GPU library and must
 * never be used as a fallback for it.
 *
 * What it computes, and where the paper defines it:
 *   oracle_pifa_build      -- Algorithm "Pivoting Factorization" (Sec. 3.2,
 *                             alg. pifa_build): pivot rows of a rank-r W' by
 *                             QR with column pivoting (Businger & Golub 1971)
 *                             applied to W'^T, the split of eq. (separate),
 *                             and the coefficient matrix C of eq. (wnp),
 *                             W_np = C W_p, obtained by a least-squares solve.
 *   oracle_pifa_forward    -- Algorithm "PIFA Layer" (alg. pifa), written for
 *                             row-major activations: Y = X W^T, so the
 *                             paper's row sets I / I^c become column sets of Y.
 *   oracle_dense_forward   -- the dense layer Y = X W^T whose cost the paper
 *                             gives as 2mnb FLOPs (Sec. 3.3).
 *   oracle_lowrank_forward -- the low-rank layer Y = (X V^T) U^T, i.e. the
 *                             paper's U (V^T X) in row-major form (Sec. 3.3).
 *   oracle_reconstruction_error -- the losslessness check
 *                             || P[W_p; C W_p] - W ||_F / ||W||_F.
 *   oracle_pifa_backward   -- gradients of Algorithm "PIFA Layer" (the layer
 *                             is differentiable end to end, Sec. 5 and 6):
 *                             the chain rule through its two products and
 *                             two column assignments.
 *
 * Readings of points the paper leaves open (each is listed in the design
 * notes of the repository):
 *   - indices are 0-based; I and I^c are returned sorted ascending, and the
 *     rows of W_p / columns of C follow that order;
 *   - pivot ties (equal residual norms) go to the lowest original row index;
 *   - residual column norms are recomputed exactly after every Householder
 *     step (no norm downdating), so the pivot sequence is deterministic;
 *   - the linear solve for C uses the QR factors of W_p^T that the pivoting
 *     already produced: with W'^T P = Q [R11 R12; 0 R22] and R22 = 0 for a
 *     rank-r input, the least-squares solution of W_p^T C^T = W_np^T is
 *     C^T = R11^{-1} R12 (no normal equations);
 *   - the input must have numerical rank exactly r: the build refuses a W'
 *     whose r-th pivot is tiny relative to the first, or whose residual after
 *     r steps is not negligible.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* rank certification thresholds (relative to |R_00|) */
#define ORACLE_MIN_PIVOT_RATIO 1e-8
#define ORACLE_MAX_RESIDUAL_RATIO 1e-10

enum {
    ORACLE_OK = 0,
    ORACLE_NOT_RANK_R = 1,
    ORACLE_BAD_ARGS = -1,
    ORACLE_NO_MEMORY = -2
};

static int clamp_threads(int nthreads) { return nthreads < 1 ? 1 : nthreads; }

/* Progress lines of long builds: every `oracle_progress_every` QRCP steps a
 * line goes to stderr (0 = silent).  Reporting only; no effect on results. */
static int64_t oracle_progress_every = 0;

void oracle_set_progress(int64_t every) { oracle_progress_every = every < 0 ? 0 : every; }

typedef struct {
    int32_t key;  /* original row index of W' */
    int64_t slot; /* position in the pivoted factorization */
} keyed_slot;

static int cmp_keyed_slot(const void* a, const void* b) {
    const keyed_slot* x = (const keyed_slot*)a;
    const keyed_slot* y = (const keyed_slot*)b;
    return (x->key > y->key) - (x->key < y->key);
}

/*
 * Pivoting Factorization of a rank-r matrix W' (d_out x d_in, row-major).
 *
 * QR with column pivoting runs on A = W'^T: column j of A is row j of W', so
 * A is held as d_out contiguous columns of length d_in (the same bytes as W'
 * in row-major order).  Step k picks the column with the largest residual
 * norm ||A[k:, j]||, swaps it into position k, and annihilates A[k+1:, k]
 * with a Householder reflector H = I - tau v v^T, v[0] = 1.
 *
 * Outputs (caller-allocated):
 *   pivot_idx     r        sorted original row indices of the pivot rows (I)
 *   nonpivot_idx  d_out-r  sorted complement (I^c)
 *   Wp            r x d_in        W'[I, :]
 *   C             (d_out-r) x r   W'[I^c, :] = C W_p
 *   select_order  r        pivot rows in the order QRCP selected them
 *   report        4        |R_00|, |R_{r-1,r-1}|, max residual column norm
 *                          after r steps, and 1.0 if the rank certification
 *                          passed (0.0 otherwise)
 * Returns ORACLE_OK, ORACLE_NOT_RANK_R, ORACLE_BAD_ARGS or ORACLE_NO_MEMORY.
 */
int oracle_pifa_build(const double* W, int64_t d_out, int64_t d_in, int64_t r,
                      int nthreads, int32_t* pivot_idx, int32_t* nonpivot_idx,
                      double* Wp, double* C, int32_t* select_order,
                      double* report) {
    if (!W || !pivot_idx || !Wp || !select_order || !report) return ORACLE_BAD_ARGS;
    if (d_out < 1 || d_in < 1 || r < 1 || r > d_out || r > d_in) return ORACLE_BAD_ARGS;
    if (r < d_out && (!nonpivot_idx || !C)) return ORACLE_BAD_ARGS;
    const int nt = clamp_threads(nthreads);
    const int64_t n_np = d_out - r;

    double* A = (double*)malloc((size_t)d_out * (size_t)d_in * sizeof(double));
    double* nrm2 = (double*)malloc((size_t)d_out * sizeof(double));
    int32_t* perm = (int32_t*)malloc((size_t)d_out * sizeof(int32_t));
    double* tmp = (double*)malloc((size_t)d_in * sizeof(double));
    if (!A || !nrm2 || !perm || !tmp) {
        free(A); free(nrm2); free(perm); free(tmp);
        return ORACLE_NO_MEMORY;
    }
    memcpy(A, W, (size_t)d_out * (size_t)d_in * sizeof(double));
    for (int64_t j = 0; j < d_out; ++j) perm[j] = (int32_t)j;

    /* initial squared column norms of A (= squared row norms of W') */
#pragma omp parallel for schedule(static) num_threads(nt)
    for (int64_t j = 0; j < d_out; ++j) {
        const double* a = A + j * d_in;
        double s = 0.0;
        for (int64_t i = 0; i < d_in; ++i) s += a[i] * a[i];
        nrm2[j] = s;
    }

    int status = ORACLE_OK;
    for (int64_t k = 0; k < r; ++k) {
        if (oracle_progress_every > 0 && k % oracle_progress_every == 0) {
            fprintf(stderr, "oracle build %lld x %lld, r = %lld: QRCP step %lld\n", (long long)d_out,
                    (long long)d_in, (long long)r, (long long)k);
            fflush(stderr);
        }
        /* pivot: largest residual norm, ties to the lowest original index */
        int64_t p = k;
        for (int64_t j = k + 1; j < d_out; ++j) {
            if (nrm2[j] > nrm2[p] || (nrm2[j] == nrm2[p] && perm[j] < perm[p])) p = j;
        }
        if (p != k) {
            memcpy(tmp, A + k * d_in, (size_t)d_in * sizeof(double));
            memcpy(A + k * d_in, A + p * d_in, (size_t)d_in * sizeof(double));
            memcpy(A + p * d_in, tmp, (size_t)d_in * sizeof(double));
            int32_t tp = perm[k]; perm[k] = perm[p]; perm[p] = tp;
            double tn = nrm2[k]; nrm2[k] = nrm2[p]; nrm2[p] = tn;
        }

        /* Householder reflector for x = A[k:, k] */
        double* x = A + k * d_in;
        double xnorm2 = 0.0;
        for (int64_t i = k; i < d_in; ++i) xnorm2 += x[i] * x[i];
        const double xnorm = sqrt(xnorm2);
        if (xnorm == 0.0) { status = ORACLE_NOT_RANK_R; break; }
        const double alpha = x[k];
        const double beta = -copysign(xnorm, alpha);
        const double tau = (beta - alpha) / beta;
        const double inv = 1.0 / (alpha - beta);
        for (int64_t i = k + 1; i < d_in; ++i) x[i] *= inv; /* v[1:], v[0] = 1 */
        x[k] = beta;                                         /* R[k][k] */

        /* apply H to the trailing columns; recompute their residual norms */
#pragma omp parallel for schedule(static) num_threads(nt)
        for (int64_t j = k + 1; j < d_out; ++j) {
            double* a = A + j * d_in;
            double w = a[k];
            for (int64_t i = k + 1; i < d_in; ++i) w += x[i] * a[i];
            w *= tau;
            a[k] -= w;
            double s = 0.0;
            for (int64_t i = k + 1; i < d_in; ++i) {
                a[i] -= w * x[i];
                s += a[i] * a[i];
            }
            nrm2[j] = s;
        }
    }

    if (status == ORACLE_OK) {
        const double r00 = fabs(A[0]);
        const double rlast = fabs(A[(r - 1) * d_in + (r - 1)]);
        double resid = 0.0;
        for (int64_t j = r; j < d_out; ++j) {
            const double nj = sqrt(nrm2[j]);
            if (nj > resid) resid = nj;
        }
        const int certified = (rlast >= ORACLE_MIN_PIVOT_RATIO * r00) &&
                              (resid <= ORACLE_MAX_RESIDUAL_RATIO * r00);
        report[0] = r00;
        report[1] = rlast;
        report[2] = resid;
        report[3] = certified ? 1.0 : 0.0;
        if (!certified) status = ORACLE_NOT_RANK_R;
    } else {
        report[0] = report[1] = report[2] = report[3] = 0.0;
    }

    if (status == ORACLE_OK) {
        for (int64_t s = 0; s < r; ++s) select_order[s] = perm[s];

        /* sorted pivot / non-pivot index sets and the slot each came from */
        keyed_slot* piv = (keyed_slot*)malloc((size_t)r * sizeof(keyed_slot));
        keyed_slot* npv = (keyed_slot*)malloc((size_t)(n_np > 0 ? n_np : 1) * sizeof(keyed_slot));
        int64_t* pos_of_slot = (int64_t*)malloc((size_t)r * sizeof(int64_t));
        double* R11 = (double*)malloc((size_t)r * (size_t)r * sizeof(double));
        if (!piv || !npv || !pos_of_slot || !R11) {
            status = ORACLE_NO_MEMORY;
        } else {
            for (int64_t s = 0; s < r; ++s) { piv[s].key = perm[s]; piv[s].slot = s; }
            for (int64_t t = 0; t < n_np; ++t) { npv[t].key = perm[r + t]; npv[t].slot = r + t; }
            qsort(piv, (size_t)r, sizeof(keyed_slot), cmp_keyed_slot);
            if (n_np > 0) qsort(npv, (size_t)n_np, sizeof(keyed_slot), cmp_keyed_slot);
            for (int64_t i = 0; i < r; ++i) {
                pivot_idx[i] = piv[i].key;
                pos_of_slot[piv[i].slot] = i;
            }
            for (int64_t q = 0; q < n_np; ++q) nonpivot_idx[q] = npv[q].key;

            /* W_p = W'[I, :] taken from the untouched input */
            for (int64_t i = 0; i < r; ++i)
                memcpy(Wp + i * d_in, W + (int64_t)pivot_idx[i] * d_in, (size_t)d_in * sizeof(double));

            /* R11 in row-major form: R11[s][t] = A[t][s] for s <= t < r */
            for (int64_t s = 0; s < r; ++s)
                for (int64_t t = 0; t < r; ++t)
                    R11[s * r + t] = (t >= s) ? A[t * d_in + s] : 0.0;

            if (oracle_progress_every > 0) {
                fprintf(stderr, "oracle build %lld x %lld, r = %lld: QRCP done, solving for C\n",
                        (long long)d_out, (long long)d_in, (long long)r);
                fflush(stderr);
            }
            /* C^T = R11^{-1} R12 by back substitution, one non-pivot row of
             * W' (one column of R12) at a time, scattered to sorted order */
#pragma omp parallel num_threads(nt)
            {
                double* y = (double*)malloc((size_t)r * sizeof(double));
#pragma omp for schedule(dynamic, 16)
                for (int64_t q = 0; q < n_np; ++q) {
                    const double* rhs = A + npv[q].slot * d_in; /* R12[:, col] */
                    for (int64_t s = r - 1; s >= 0; --s) {
                        const double* row = R11 + s * r;
                        double acc = rhs[s];
                        for (int64_t t = s + 1; t < r; ++t) acc -= row[t] * y[t];
                        y[s] = acc / row[s];
                    }
                    double* crow = C + q * r;
                    for (int64_t s = 0; s < r; ++s) crow[pos_of_slot[s]] = y[s];
                }
                free(y);
            }
        }
        free(piv); free(npv); free(pos_of_slot); free(R11);
    }

    free(A); free(nrm2); free(perm); free(tmp);
    return status;
}

/*
 * PIFA layer forward (alg. pifa) for row-major activations X (M x d_in):
 *   Y_p  = X W_p^T            (M x r)        -- pivot outputs
 *   Y_np = Y_p C^T            (M x (d_out-r)) -- non-pivot outputs
 *   Y[:, pivot_idx[j]]    = Y_p[:, j]
 *   Y[:, nonpivot_idx[t]] = Y_np[:, t]
 * No rounding of the intermediate Y_p.  Y is M x d_out row-major.
 */
void oracle_pifa_forward(const double* X, int64_t M, int64_t d_in, int64_t d_out,
                         int64_t r, const int32_t* pivot_idx,
                         const int32_t* nonpivot_idx, const double* Wp,
                         const double* C, double* Y, int nthreads) {
    const int nt = clamp_threads(nthreads);
    const int64_t n_np = d_out - r;
    double* Yp = (double*)malloc((size_t)(M > 0 ? M : 1) * (size_t)r * sizeof(double));
    if (!Yp) return;

#pragma omp parallel for collapse(2) schedule(static) num_threads(nt)
    for (int64_t m = 0; m < M; ++m)
        for (int64_t j = 0; j < r; ++j) {
            const double* x = X + m * d_in;
            const double* w = Wp + j * d_in;
            double s = 0.0;
            for (int64_t k = 0; k < d_in; ++k) s += x[k] * w[k];
            Yp[m * r + j] = s;
        }

#pragma omp parallel for collapse(2) schedule(static) num_threads(nt)
    for (int64_t m = 0; m < M; ++m)
        for (int64_t t = 0; t < n_np; ++t) {
            const double* yp = Yp + m * r;
            const double* c = C + t * r;
            double s = 0.0;
            for (int64_t j = 0; j < r; ++j) s += yp[j] * c[j];
            Y[m * d_out + nonpivot_idx[t]] = s;
        }

    for (int64_t m = 0; m < M; ++m)
        for (int64_t j = 0; j < r; ++j) Y[m * d_out + pivot_idx[j]] = Yp[m * r + j];

    free(Yp);
}

/* Dense layer: Y = X W^T, W is d_out x d_in row-major. */
void oracle_dense_forward(const double* X, const double* W, int64_t M, int64_t d_in,
                          int64_t d_out, double* Y, int nthreads) {
    const int nt = clamp_threads(nthreads);
#pragma omp parallel for collapse(2) schedule(static) num_threads(nt)
    for (int64_t m = 0; m < M; ++m)
        for (int64_t n = 0; n < d_out; ++n) {
            const double* x = X + m * d_in;
            const double* w = W + n * d_in;
            double s = 0.0;
            for (int64_t k = 0; k < d_in; ++k) s += x[k] * w[k];
            Y[m * d_out + n] = s;
        }
}

/* Low-rank layer: T = X V^T (M x r), Y = T U^T; U is d_out x r, V is r x d_in. */
void oracle_lowrank_forward(const double* X, const double* U, const double* V,
                            int64_t M, int64_t d_in, int64_t d_out, int64_t r,
                            double* Y, int nthreads) {
    const int nt = clamp_threads(nthreads);
    double* T = (double*)malloc((size_t)(M > 0 ? M : 1) * (size_t)r * sizeof(double));
    if (!T) return;
#pragma omp parallel for collapse(2) schedule(static) num_threads(nt)
    for (int64_t m = 0; m < M; ++m)
        for (int64_t s = 0; s < r; ++s) {
            const double* x = X + m * d_in;
            const double* v = V + s * d_in;
            double acc = 0.0;
            for (int64_t k = 0; k < d_in; ++k) acc += x[k] * v[k];
            T[m * r + s] = acc;
        }
#pragma omp parallel for collapse(2) schedule(static) num_threads(nt)
    for (int64_t m = 0; m < M; ++m)
        for (int64_t n = 0; n < d_out; ++n) {
            const double* t = T + m * r;
            const double* u = U + n * r;
            double acc = 0.0;
            for (int64_t s = 0; s < r; ++s) acc += t[s] * u[s];
            Y[m * d_out + n] = acc;
        }
    free(T);
}

/*
 * Losslessness of a PIFA layer: rebuild W from (I, W_p, C) -- pivot rows are
 * W_p, non-pivot rows are C W_p -- and return ||rebuilt - W||_F / ||W||_F.
 */
double oracle_reconstruction_error(const double* W, int64_t d_out, int64_t d_in,
                                   int64_t r, const int32_t* pivot_idx,
                                   const int32_t* nonpivot_idx, const double* Wp,
                                   const double* C, int nthreads) {
    const int nt = clamp_threads(nthreads);
    const int64_t n_np = d_out - r;
    double err2 = 0.0, ref2 = 0.0;

#pragma omp parallel for reduction(+ : err2, ref2) schedule(static) num_threads(nt)
    for (int64_t i = 0; i < r; ++i) {
        const double* w = W + (int64_t)pivot_idx[i] * d_in;
        const double* p = Wp + i * d_in;
        for (int64_t k = 0; k < d_in; ++k) {
            const double d = p[k] - w[k];
            err2 += d * d;
            ref2 += w[k] * w[k];
        }
    }

#pragma omp parallel num_threads(nt) reduction(+ : err2, ref2)
    {
        double* row = (double*)malloc((size_t)d_in * sizeof(double));
#pragma omp for schedule(dynamic, 8)
        for (int64_t q = 0; q < n_np; ++q) {
            for (int64_t k = 0; k < d_in; ++k) row[k] = 0.0;
            const double* c = C + q * r;
            for (int64_t j = 0; j < r; ++j) {
                const double cj = c[j];
                const double* p = Wp + j * d_in;
                for (int64_t k = 0; k < d_in; ++k) row[k] += cj * p[k];
            }
            const double* w = W + (int64_t)nonpivot_idx[q] * d_in;
            for (int64_t k = 0; k < d_in; ++k) {
                const double d = row[k] - w[k];
                err2 += d * d;
                ref2 += w[k] * w[k];
            }
        }
        free(row);
    }
    return ref2 > 0.0 ? sqrt(err2 / ref2) : sqrt(err2);
}

/* Number of threads an OpenMP region started by this library would use. */
int oracle_max_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/*
 * Gradients of Algorithm "PIFA Layer" for G = dL/dY (M x d_out).  Forward:
 * Y_p = X W_p^T, Y_np = Y_p C^T, Y[:, I] = Y_p, Y[:, I^c] = Y_np.  Backward,
 * step by step:
 *   G_p   = G[:, I] + G[:, I^c] C        (Y_p feeds both assignments)
 *   dC    = G[:, I^c]^T Y_p              (n_np x r)
 *   dX    = G_p W_p                      (M x d_in)
 *   dW_p  = G_p^T X                      (r x d_in)
 * Y_p is recomputed from X and W_p.  dX, dWp, dC are overwritten; dC may be
 * NULL when r = d_out.
 */
void oracle_pifa_backward(const double* X, const double* G, int64_t M, int64_t d_in,
                          int64_t d_out, int64_t r, const int32_t* pivot_idx,
                          const int32_t* nonpivot_idx, const double* Wp, const double* C,
                          double* dX, double* dWp, double* dC, int nthreads) {
    const int nt = clamp_threads(nthreads);
    const int64_t n_np = d_out - r;
    const size_t mr = (size_t)(M > 0 ? M : 1) * (size_t)r;
    double* Yp = (double*)malloc(mr * sizeof(double));
    double* Gp = (double*)malloc(mr * sizeof(double));
    if (!Yp || !Gp) {
        free(Yp);
        free(Gp);
        return;
    }

#pragma omp parallel for collapse(2) schedule(static) num_threads(nt)
    for (int64_t m = 0; m < M; ++m)
        for (int64_t j = 0; j < r; ++j) {
            double s = 0.0;
            for (int64_t k = 0; k < d_in; ++k) s += X[m * d_in + k] * Wp[j * d_in + k];
            Yp[m * r + j] = s;
        }

    /* G_p = G[:, I] + G[:, I^c] C */
#pragma omp parallel for collapse(2) schedule(static) num_threads(nt)
    for (int64_t m = 0; m < M; ++m)
        for (int64_t j = 0; j < r; ++j) {
            double s = G[m * d_out + pivot_idx[j]];
            for (int64_t k = 0; k < n_np; ++k) s += G[m * d_out + nonpivot_idx[k]] * C[k * r + j];
            Gp[m * r + j] = s;
        }

    /* dC = G[:, I^c]^T Y_p */
#pragma omp parallel for collapse(2) schedule(static) num_threads(nt)
    for (int64_t k = 0; k < n_np; ++k)
        for (int64_t j = 0; j < r; ++j) {
            double s = 0.0;
            for (int64_t m = 0; m < M; ++m) s += G[m * d_out + nonpivot_idx[k]] * Yp[m * r + j];
            dC[k * r + j] = s;
        }

    /* dX = G_p W_p */
#pragma omp parallel for collapse(2) schedule(static) num_threads(nt)
    for (int64_t m = 0; m < M; ++m)
        for (int64_t i = 0; i < d_in; ++i) {
            double s = 0.0;
            for (int64_t j = 0; j < r; ++j) s += Gp[m * r + j] * Wp[j * d_in + i];
            dX[m * d_in + i] = s;
        }

    /* dW_p = G_p^T X */
#pragma omp parallel for collapse(2) schedule(static) num_threads(nt)
    for (int64_t j = 0; j < r; ++j)
        for (int64_t i = 0; i < d_in; ++i) {
            double s = 0.0;
            for (int64_t m = 0; m < M; ++m) s += Gp[m * r + j] * X[m * d_in + i];
            dWp[j * d_in + i] = s;
        }

    free(Yp);
    free(Gp);
}
