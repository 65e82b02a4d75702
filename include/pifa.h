/*
 * libpifa -- PIFA (Pivoting Factorization) linear layer forward on MI355X.
 *
 * Method: Zhao, Zhang & Cannistraci, "Pivoting Factorization: A Compact Meta
 * Low-Rank Representation of Sparsity for Efficient Inference in Large
 * Language Models", arXiv 2501.19090.
 *
 * A rank-r weight W (d_out x d_in) is stored as its r pivot rows W_p
 * (r x d_in), the coefficient matrix C ((d_out - r) x r) with non-pivot rows
 * W_np = C W_p (Sec. 3.2, eq. wnp), and the pivot / non-pivot row index sets
 * I and I^c.  The layer forward (Algorithm "PIFA Layer") is
 *     Y_p = X W_p^T,   Y_np = Y_p C^T,   Y[:, I] = Y_p,   Y[:, I^c] = Y_np
 * written here for row-major activations X (M x d_in) and outputs Y
 * (M x d_out): the paper's row index sets of W become column positions of Y.
 *
 * Conventions for every entry point:
 *   - Matrices are dense, row-major, contiguous, with no padding between rows.
 *   - "device" pointers are HIP device memory on the current device;
 *     "host" pointers are ordinary host memory.
 *   - A handle belongs to the device that was current when it was created;
 *     every call taking it returns PIFA_ERR_WRONG_DEVICE if another device
 *     is current (destroy calls excepted).
 *   - Element type is given by a pifa_dtype: PIFA_BF16 (bfloat16 storage,
 *     fp32 accumulation) or PIFA_F32.  X, Y and the weights share the dtype.
 *   - bf16 requires d_in to be a multiple of 8 (16-byte rows); f32 accepts
 *     any d_in.
 *   - `stream` is a hipStream_t passed as void*; NULL means the default stream.
 *   - No entry point throws.  Arguments are validated synchronously and a
 *     status is returned; a kernel fault surfaces at the caller's next
 *     synchronisation.  NaN and Inf in the inputs propagate to the outputs.
 *   - Indices are 0-based int32 (the paper's are 1-based sets).
 */
#ifndef PIFA_H
#define PIFA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { PIFA_F32 = 0, PIFA_BF16 = 1 } pifa_dtype;

typedef enum {
    PIFA_OK = 0,
    PIFA_ERR_INVALID_ARG = -1, /* null pointer, bad size or dtype        */
    PIFA_ERR_BAD_INDEX = -2,   /* index out of range, duplicate, or the  */
                               /* two sets do not partition [0, d_out)   */
    PIFA_ERR_UNSUPPORTED = -3, /* a shape or alignment the kernels lack  */
    PIFA_ERR_HIP = -4,         /* a HIP runtime call or launch failed    */
    PIFA_ERR_OOM = -5,         /* device memory allocation failed        */
    PIFA_ERR_NOT_RANK_R = -6,  /* pifa_build_f64: W' is not numerically  */
                               /* of rank r                              */
    PIFA_ERR_NOT_SPD = -7,     /* pifa_calib_reconstruct: a normal-      */
                               /* equation matrix is not positive        */
                               /* definite (too few calibration rows)    */
    PIFA_ERR_WRONG_DEVICE = -8, /* a handle used while another device is */
                                /* current than the one it was created on*/
    PIFA_ERR_TOO_LARGE = -9     /* pifa_forward_noalloc: the call needs   */
                                /* more workspace than its fixed scratch */
} pifa_status;

/* Layer shape: W is d_out x d_in with rank r, 1 <= r <= min(d_in, d_out)
 * (Sec. 3.3 assumes r < min(m, n) for the memory saving; r = d_out is
 * accepted and gives an empty C). */
typedef struct {
    int64_t d_in;
    int64_t d_out;
    int64_t r;
} pifa_dims;

typedef struct pifa_layer* pifa_handle;
typedef struct lowrank_layer* lowrank_handle;
typedef struct dense_layer* dense_handle;
typedef struct pifa_group* pifa_group_handle;
typedef struct pifa_calib* pifa_calib_handle;

/* Human-readable name of a status code (static storage, never NULL). */
const char* pifa_status_string(pifa_status s);

/*
 * Host-only check that pivot_idx (r entries) and nonpivot_idx (d_out - r
 * entries) are in range, free of duplicates and together cover [0, d_out)
 * exactly (Algorithm "Pivoting Factorization": I^c = {1..m} \ I).  Any order
 * is accepted.  Needs no GPU.  Returns PIFA_OK, PIFA_ERR_INVALID_ARG (bad
 * dims or null pointer) or PIFA_ERR_BAD_INDEX.
 */
pifa_status pifa_validate_partition(const int32_t* pivot_idx, const int32_t* nonpivot_idx,
                                    pifa_dims dims);

/*
 * Host-only diagnostic: the output tile (tile_m x tile_n rows x columns of
 * Y) and the number of K splits (1 = none; otherwise fp32 partial products
 * summed by a second kernel) that a prefill product Y = A B^T of M x N
 * outputs over K runs with (more than 16 activation rows; the products of
 * pifa_forward, the baselines, the backward pass and the calibration sums
 * all take this plan).  wide_epilogue = 0 for epilogues that keep per-output
 * state (fp32 or fp64 outputs, starting values), which never take the 256 x
 * 256 and 256 x 192 tiles.  Needs no GPU.  Returns PIFA_OK or
 * PIFA_ERR_INVALID_ARG (a size below 1 or a null pointer).
 */
pifa_status pifa_gemm_plan(int64_t M, int64_t N, int64_t K, int wide_epilogue, int64_t* tile_m,
                           int64_t* tile_n, int64_t* k_splits);

/*
 * Create a PIFA layer from the output of Algorithm "Pivoting Factorization".
 *   W_p           device, r x d_in, dtype.  Row j is the weight row that
 *                 produces output column pivot_idx[j].
 *   C             device, (d_out - r) x r, dtype; may be NULL when r = d_out.
 *                 Row k produces output column nonpivot_idx[k]; its columns
 *                 follow the row order of W_p.
 *   pivot_idx     host, r entries; nonpivot_idx host, d_out - r entries
 *                 (may be NULL when r = d_out).  Validated as by
 *                 pifa_validate_partition.
 * The layer copies everything it needs into memory it owns, so the caller may
 * free its buffers on return.  bf16 layers reorder W_p and C into 16 x 128
 * blocks in MFMA operand order (rows padded to a multiple of 64 with zeros)
 * and convert C exactly to fp16 with a power-of-two scale.
 * Synchronises the device.  On success *out holds the handle.
 */
pifa_status pifa_layer_create(const void* W_p, const void* C, const int32_t* pivot_idx,
                              const int32_t* nonpivot_idx, pifa_dims dims, pifa_dtype dtype,
                              pifa_handle* out);

/* Release a layer and its device memory (synchronises the device). NULL is OK. */
pifa_status pifa_layer_destroy(pifa_handle h);

/*
 * Pre-size the layer's workspace for forwards of up to max_M rows, so that
 * later pifa_forward calls allocate nothing.  Synchronises the device.
 */
pifa_status pifa_layer_reserve(pifa_handle h, int64_t max_M);

/*
 * Algorithm "PIFA Layer": Y[:, I] = X W_p^T and Y[:, I^c] = (X W_p^T) C^T.
 *   X  device, M x d_in, dtype, borrowed (read only).
 *   Y  device, M x d_out, dtype; every element is written.
 * M = 0 returns PIFA_OK without launching.  Asynchronous on `stream`.
 * The layer's workspace holds the intermediate Y_p, so calls on one handle
 * must not overlap (use one handle per concurrent stream).  If M exceeds the
 * reserved size the workspace grows, which synchronises `stream`.
 * bf16: Y_p is handed from the first to the second product as fp16 times
 * 2^s (s = 0 unless set by pifa_layer_set_intermediate_scale); a |Y_p * 2^s|
 * above 65504 cannot be represented, is counted (pifa_layer_overflow_count)
 * and produces non-finite outputs in that row.
 */
pifa_status pifa_forward(pifa_handle h, const void* X, void* Y, int64_t M, void* stream);

/*
 * pifa_forward for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc).
 * Same arguments, results and stream semantics as pifa_forward, bit for bit,
 * but the workspace is a fixed 32 MiB array in the library's device memory
 * (one per GPU, held until the process ends) instead of the handle's: the
 * call allocates nothing, on the device or the host, and never synchronises.
 * The Y_p hand-off (M * r_pad * 4 bytes for M <= 16, M * r_pad * 2 above;
 * fp32 layers M * r * 4; r_pad = r rounded up to 64) rounded up to 256
 * bytes, plus the K-split partial products of small batches, must fit in
 * those 32 MiB, else PIFA_ERR_TOO_LARGE and nothing is launched (for the
 * 4096 x 4096, r = 2048 layer every M up to 8192 fits).  Every call on a GPU
 * shares that GPU's array: calls that overlap on one GPU, on any stream or
 * handle, race and give undefined results.  Nothing in the array needs to
 * start at zero (every call writes what it reads).  Launches are never
 * timed by pifa_profile_*.
 */
pifa_status pifa_forward_noalloc(pifa_handle h, const void* X, void* Y, int64_t M, void* stream);

/* Bytes of weights and indices a forward must read: r*d_in + (d_out-r)*r
 * elements of the dtype plus d_out int32 indices (Sec. 3.3 memory cost). */
size_t pifa_layer_weight_bytes(pifa_handle h);

/* Set the power-of-two exponent s applied to Y_p before its fp16 hand-off
 * (bf16 layers only; -30 <= s <= 30). */
pifa_status pifa_layer_set_intermediate_scale(pifa_handle h, int log2_scale);

/* Number of Y_p elements that overflowed fp16 since creation (synchronises
 * the device).  Always 0 for f32 layers. */
pifa_status pifa_layer_overflow_count(pifa_handle h, int64_t* count);

/*
 * Gradients of Algorithm "PIFA Layer" (the layer is differentiable end to
 * end, Sec. 5 and 6; the chain rule through its two products and two column
 * assignments).  With G = dL/dY:
 *   G_p  = G[:, I] + G[:, I^c] C,   dX = G_p W_p,
 *   dW_p = G_p^T X,                 dC = G[:, I^c]^T Y_p.
 *   X   device, M x d_in, bf16: the forward's input.
 *   Y   device, M x d_out, bf16: the forward's output for X; its pivot
 *       columns Y[:, I] supply Y_p for dC.
 *   dY  device, M x d_out, bf16: G.
 *   dX  device, M x d_in, bf16 (overwritten), or NULL to skip.
 *   dW_p device, r x d_in, fp32 (overwritten), rows in the layer's W_p order,
 *       or NULL to skip.
 *   dC  device, (d_out - r) x r, fp32 (overwritten), rows in the layer's C
 *       order, or NULL to skip (ignored when r = d_out).
 * No alignment is required of X, Y, dY.  M = 0 zeroes dW_p and dC.  bf16
 * layers only (PIFA_F32 returns PIFA_ERR_UNSUPPORTED).  The first call builds
 * transposed copies of W_p and C in the layer (synchronous); the handle's
 * backward workspace grows on demand (synchronising `stream`).  Calls on one
 * handle must not overlap.  G_p reaches dX in fp16 with a power-of-two
 * scale per row (C makes that product cancel, and bf16 is too coarse there);
 * the other products take bf16 operands; all accumulate in fp32.
 */
pifa_status pifa_layer_backward(pifa_handle h, const void* X, const void* Y, const void* dY, int64_t M,
                                void* dX, float* dW_p, float* dC, void* stream);

/*
 * Grouped PIFA layers that read the same activations X (for example a
 * transformer MLP's gate and up projections, or attention's q, k and v), with
 * a rank of their own each (MPIFA_NS sets a density per module: appendix
 * "Experiment Details", MPIFA_NS).  Evaluated together: one product X [W_p,1; W_p,2; ...]^T reads
 * X once for every layer's pivot outputs; for M <= 16 one launch also
 * streams every layer's C for Y_np,i = Y_p,i C_i^T, and for larger M each
 * layer's Y_np,i is its own launch.
 *   n             number of layers, 1 <= n <= 8.
 *   W_p[i], C[i]  device pointers as for pifa_layer_create (C[i] may be NULL
 *                 when r_i = d_out,i).
 *   pivot_idx[i], nonpivot_idx[i]  host arrays as for pifa_layer_create,
 *                 relative to layer i's own outputs [0, d_out,i).
 *   dims[i]       all with the same d_in.
 *   dtype         PIFA_BF16 only (PIFA_F32 returns PIFA_ERR_UNSUPPORTED).
 * Everything is copied into memory the group owns (one concatenated W_p; no
 * copy is kept twice).  Synchronises the device.
 */
pifa_status pifa_group_create(int n, const void* const* W_p, const void* const* C,
                              const int32_t* const* pivot_idx, const int32_t* const* nonpivot_idx,
                              const pifa_dims* dims, pifa_dtype dtype, pifa_group_handle* out);

/* Release a group (synchronises the device).  NULL is OK. */
pifa_status pifa_group_destroy(pifa_group_handle g);

/* Pre-size the group's workspace for forwards of up to max_M rows. */
pifa_status pifa_group_reserve(pifa_group_handle g, int64_t max_M);

/*
 * Y = [Y_1 | Y_2 | ... | Y_n]: layer i's Algorithm "PIFA Layer" output goes
 * to columns [o_i, o_i + d_out,i) of Y, o_i = d_out,1 + ... + d_out,i-1.
 *   X  device, M x d_in, bf16 (16-byte aligned), borrowed.
 *   Y  device, M x (sum of d_out,i), bf16; every element is written.
 * Each layer's result equals its own pifa_forward with the same intermediate
 * scale: bit for bit for M <= 16, and up to the fp32 summation order of
 * K-split products otherwise (the two calls may split K differently).  Same
 * stream, workspace and overflow rules as pifa_forward; M = 0 returns
 * PIFA_OK without launching.
 */
pifa_status pifa_group_forward(pifa_group_handle g, const void* X, void* Y, int64_t M, void* stream);

/* Sum of pifa_layer_weight_bytes over the group's layers. */
size_t pifa_group_weight_bytes(pifa_group_handle g);

/* Intermediate scale exponent s for every layer of the group (-30..30). */
pifa_status pifa_group_set_intermediate_scale(pifa_group_handle g, int log2_scale);

/* fp16 hand-off overflows of the group since creation (synchronises). */
pifa_status pifa_group_overflow_count(pifa_group_handle g, int64_t* count);

/*
 * Dense baseline (Sec. 3.3, 2 m n b FLOPs): Y = X W^T.
 *   W device d_out x d_in; X device M x d_in; Y device M x d_out.
 * Reads the caller's row-major W directly (no copy).  Products too small to
 * fill the GPU split K through the library's shared per-device workspace,
 * as lowrank_uv_forward does: calls on different streams must not overlap.
 */
pifa_status dense_forward(const void* W, const void* X, void* Y, int64_t M, int64_t d_in,
                          int64_t d_out, pifa_dtype dtype, void* stream);

/* Dense baseline with W prepacked once into the same weight layout the PIFA
 * layer uses (the like-for-like counterpart of pifa_layer_create).  W is a
 * device buffer as for dense_forward; it is copied.  Synchronises on create
 * and destroy. */
pifa_status dense_layer_create(const void* W, int64_t d_in, int64_t d_out, pifa_dtype dtype,
                               dense_handle* out);
pifa_status dense_layer_forward(dense_handle h, const void* X, void* Y, int64_t M, void* stream);
pifa_status dense_layer_reserve(dense_handle h, int64_t max_M);
pifa_status dense_layer_destroy(dense_handle h);

/*
 * Low-rank baseline (Sec. 3.3, 2 b r (m + n) FLOPs): Y = (X V^T) U^T, i.e. the
 * paper's U (V^T X) for row-major activations.
 *   U device d_out x r; V device r x d_in; X device M x d_in; Y device M x d_out.
 * The intermediate X V^T goes through the library's shared workspace (calls
 * on different streams must not overlap).  bf16 requires r to be a multiple
 * of 8 here (PIFA_ERR_UNSUPPORTED otherwise); lowrank_layer_create accepts
 * any r.
 */
pifa_status lowrank_uv_forward(const void* U, const void* V, const void* X, void* Y, int64_t M,
                               pifa_dims dims, pifa_dtype dtype, void* stream);

/* Low-rank baseline with weights prepacked once into the PIFA layer's weight
 * layout (r padded to a multiple of 64), the like-for-like counterpart of
 * pifa_layer_create.  U and V are
 * device buffers as for lowrank_uv_forward; they are copied. */
pifa_status lowrank_layer_create(const void* U, const void* V, pifa_dims dims, pifa_dtype dtype,
                                 lowrank_handle* out);
pifa_status lowrank_layer_forward(lowrank_handle h, const void* X, void* Y, int64_t M,
                                  void* stream);
pifa_status lowrank_layer_reserve(lowrank_handle h, int64_t max_M);
pifa_status lowrank_layer_destroy(lowrank_handle h);

/*
 * Online Error-Accumulation-Minimization reconstruction (Sec. 4; Part 1 of
 * Algorithm "MPIFA" in the appendix "Experiment Details").  A calibration
 * handle keeps the running sums of one layer with input width d_in = n:
 *   S = sum_i x_u^i x_u^i^T   and   P = sum_i x_o^i x_u^i^T   (n x n, fp64),
 * x_o from the dense data flow and x_u from the low-rank one.  The mixed
 * target sum of the paper is T = sum_i y_t^i x_u^i^T = W (lam P + (1 - lam) S)
 * (eq. mix_original_output, regrouped by associativity), so the dense
 * weight is not needed until the solve and one handle serves any mix ratio.
 */
pifa_status pifa_calib_create(int64_t d_in, pifa_calib_handle* out);
pifa_status pifa_calib_destroy(pifa_calib_handle c);

/* Zero the sums (asynchronous on `stream`). */
pifa_status pifa_calib_reset(pifa_calib_handle c, void* stream);

/*
 * Add one batch of B calibration rows (tokens): X_o and X_u device, bf16,
 * B x d_in row-major, no alignment required (X_o may equal X_u).  The
 * products run on the MFMA GEMM with fp32 accumulation over the batch; the
 * batch results are added to the fp64 sums.  Asynchronous on `stream`; calls
 * on one handle must not overlap.
 */
pifa_status pifa_calib_accumulate(pifa_calib_handle c, const void* X_o, const void* X_u, int64_t B,
                                  void* stream);

/* Copy the sums into device fp64 n x n buffers (either may be NULL). */
pifa_status pifa_calib_read(pifa_calib_handle c, double* S, double* P, void* stream);

/*
 * Steps 5 and 6 of Algorithm "MPIFA" with the regularised V update
 * (eq. lsq_v_reg), in fp64 on the device:
 *   T     = W (lam P + (1 - lam) S)
 *   U_r   = T V (V^T S V)^-1                                  (eq. lsq_online)
 *   V_r^T = (U_r^T U_r)^-1 U_r^T (T + alpha W) (S + alpha I)^-1
 * with the paper's V = Vt^T.  Squared Frobenius norms are read into the
 * objectives, the only reading under which these closed forms are minimisers.
 *   W     device fp64, d_out x d_in (the dense weight).
 *   Vt    device fp64, r x d_in (V^T of the low-rank start U V^T).
 *   U_r   device fp64, d_out x r (output).   Vt_r  device fp64, r x d_in (output).
 * 1 <= r <= min(d_in, d_out).  The three symmetric systems are solved by
 * Cholesky factorisation; a matrix that is not positive definite returns
 * PIFA_ERR_NOT_SPD (outputs undefined).  Synchronises `stream` (it reads the
 * factorisation status); work memory is owned by the handle.
 */
pifa_status pifa_calib_reconstruct(pifa_calib_handle c, const double* W, int64_t d_out, const double* Vt,
                                   int64_t r, double lam, double alpha, double* U_r, double* Vt_r,
                                   void* stream);

/*
 * Algorithm "Pivoting Factorization" (Sec. 3.2) on the GPU, in fp64: QR with
 * column pivoting (Businger-Golub) on W'^T picks r pivot rows (largest
 * residual norm first, ties to the lowest row index, residual norms
 * recomputed exactly after every step), then C solves W_np = C W_p by least
 * squares through the pivoted QR factors (C R11^T = R12^T).
 *   W            device, d_out x d_in fp64, the rank-r matrix W' (read only)
 *   W_p          device, r x d_in fp64 output: W'[pivot_idx, :]
 *   C            device, (d_out - r) x r fp64 output (may be NULL if r = d_out);
 *                columns follow pivot_idx
 *   pivot_idx    host, r int32 output, sorted ascending
 *   nonpivot_idx host, d_out - r int32 output, sorted ascending
 *   report       host, 4 doubles or NULL: |R_00|, |R_{r-1,r-1}|, largest
 *                residual column norm after r steps, 1.0 if certified
 * W' must have numerical rank exactly r: |R_{r-1,r-1}| >= 1e-8 |R_00| and
 * every residual norm <= 1e-10 |R_00|, else PIFA_ERR_NOT_RANK_R (outputs
 * other than report are then unspecified).  Synchronous on `stream`;
 * allocates and frees its own workspace (about (d_out + r) x max(d_in, r)
 * doubles).
 */
pifa_status pifa_build_f64(const double* W, pifa_dims dims, double* W_p, double* C, int32_t* pivot_idx,
                           int32_t* nonpivot_idx, double* report, void* stream);

/*
 * Per-kernel timing.  While enabled, every kernel the library launches for a
 * forward is bracketed by a pair of HIP events recorded on the launch stream
 * (they add no synchronisation).  pifa_profile_read synchronises on the
 * recorded events and returns, per launch site, the number of launches and
 * their summed duration in milliseconds since the last reset; sites with no
 * launches are omitted.  names[i] points to static storage.  Returns the
 * number of sites written through *n_sites (at most max_sites).
 * Not thread-safe against concurrent forwards on other host threads.
 */
pifa_status pifa_profile_enable(int on);
pifa_status pifa_profile_reset(void);
pifa_status pifa_profile_read(const char** names, int64_t* launches, double* total_ms, int max_sites,
                              int* n_sites);

/*
 * Peak probes (diagnostics; they allocate and free a few KB and synchronise).
 *
 * pifa_probe_mfma: the sustained bf16 matrix-core rate of the current device.
 * 2048 workgroups of 4 waves each issue `iters` rounds of four independent
 * v_mfma_f32_32x32x16_bf16 on register operands (no memory traffic); the
 * second of two launches is timed with HIP events.  *tflops is its dense
 * FLOP rate; *sclk_mhz is the shader clock the loop ran at, averaged over
 * the workgroups (shader-clock cycles over real-time-clock ticks).
 *
 * pifa_probe_mfma_random: the same on operands that change with every MFMA
 * (each wave cycles through 8 register sets of random bf16 values; `iters`
 * is rounded up to a multiple of 8).  Matrix-core power grows with the
 * operand bits that toggle, so under the board's power limit this rate and
 * clock are what a GEMM on real data can approach, while pifa_probe_mfma's
 * constant operands give the rate at the unthrottled clock.
 *
 * pifa_probe_hbm_read: `reps` back-to-back reads of the device buffer `buf`
 * (`bytes` a multiple of 16, 16-byte aligned; larger than the 256 MB
 * Infinity Cache to measure HBM) with 16-byte loads in a grid-stride loop;
 * *gbps = bytes * reps / the elapsed time of the `reps` launches (one
 * untimed launch first), the best of grids of 2048, 4096 and 8192
 * workgroups of 256 threads.
 * Both return PIFA_ERR_INVALID_ARG for a bad argument and PIFA_ERR_HIP if
 * a launch or event fails.
 */
pifa_status pifa_probe_mfma(int64_t iters, double* tflops, double* sclk_mhz, void* stream);
pifa_status pifa_probe_mfma_random(int64_t iters, double* tflops, double* sclk_mhz, void* stream);
pifa_status pifa_probe_hbm_read(const void* buf, int64_t bytes, int reps, double* gbps, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* PIFA_H */
