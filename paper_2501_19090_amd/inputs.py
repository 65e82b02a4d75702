"""Seeded synthetic inputs shared by the tests, the smoke check and the bench.

This module holds none of the PIFA arithmetic: it only draws random numbers
and rounds them once to the storage dtype, so that the GPU library and the
fp64 oracle consume identical bits.

Workload recipe (paper shapes, synthetic values):
  * U (d_out x r) and V (r x d_in) i.i.d. N(0, sigma^2) with sigma = r^-1/2,
    drawn in that order from numpy PCG64 seeded with ``seed``; W' = U V has
    rank r.  The second parameter of the configs' "N(0, 1/sqrt(128))" is read
    as the standard deviation.
  * X (M x d_in) i.i.d. N(0, 1) from PCG64 seeded with (seed, M).
  * Rounding to bf16 goes fp64 -> fp32 -> bf16, round-to-nearest-even at each
    step; the resulting bits are what both sides use.
"""
from __future__ import annotations

import numpy as np

# (config index) -> base seed; a layer's seed is base + its index in the config
SEED_BASE = 2501


def config_seed(config: int, layer: int = 0) -> int:
    return SEED_BASE + 100 * int(config) + int(layer)


# --------------------------------------------------------------------------
# rounding to storage dtypes
# --------------------------------------------------------------------------
def f32_bits_to_bf16_bits(x32: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (round-to-nearest-even); returns uint16 bits."""
    u = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32)
    nan = (u & 0x7FFFFFFF) > 0x7F800000
    lsb = (u >> 16) & 1
    rounded = ((u.astype(np.uint64) + 0x7FFF + lsb) >> 16).astype(np.uint16)
    return np.where(nan, ((u >> 16) | 0x40).astype(np.uint16), rounded)


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def round_bf16(a: np.ndarray):
    """fp64 -> (bf16 bits as uint16, the same values as fp64)."""
    bits = f32_bits_to_bf16_bits(np.asarray(a, dtype=np.float64).astype(np.float32))
    return bits, bf16_bits_to_f64(bits)


def round_f32(a: np.ndarray):
    """fp64 -> (fp32 array, the same values as fp64)."""
    a32 = np.ascontiguousarray(np.asarray(a, dtype=np.float64).astype(np.float32))
    return a32, a32.astype(np.float64)


def round_to(a: np.ndarray, dtype: str):
    """Round once to ``dtype`` ('bf16' or 'f32'): (storage array, fp64 values)."""
    if dtype == "bf16":
        return round_bf16(a)
    if dtype == "f32":
        return round_f32(a)
    raise ValueError("unknown dtype %r" % (dtype,))


# --------------------------------------------------------------------------
# Gaussian low-rank layers and activations
# --------------------------------------------------------------------------
def lowrank_factors(d_out: int, d_in: int, r: int, seed: int):
    """U (d_out x r), V (r x d_in), i.i.d. N(0, 1/r), fp64; W' = U V has rank r."""
    rng = np.random.default_rng(seed)
    sigma = float(r) ** -0.5
    U = rng.standard_normal((d_out, r)) * sigma
    V = rng.standard_normal((r, d_in)) * sigma
    return U, V


def activations(M: int, d_in: int, seed: int) -> np.ndarray:
    """X (M x d_in) i.i.d. N(0, 1), fp64."""
    rng = np.random.default_rng([int(seed), int(M)])
    return rng.standard_normal((M, d_in))


def random_partition(d_out: int, r: int, seed: int):
    """A seeded random r-subset of [0, d_out) and its complement, both sorted."""
    rng = np.random.default_rng([int(seed), 7])
    perm = rng.permutation(d_out)
    piv = np.sort(perm[:r]).astype(np.int32)
    npiv = np.sort(perm[r:]).astype(np.int32)
    return piv, npiv


# --------------------------------------------------------------------------
# exactness probes
# --------------------------------------------------------------------------
def layout_probe_layer(d_in: int, d_out: int, r: int):
    """W_p = [I_r | 0] and one-hot C rows, C[k, (7k + 3) mod r] = 1.

    With these weights every output element is a single product x * 1, exact in
    any summation order and any intermediate format, so Y[:, I[j]] = X[:, j]
    and Y[:, I^c[k]] = X[:, (7k+3) mod r] exactly.
    """
    Wp = np.zeros((r, d_in))
    Wp[np.arange(r), np.arange(r)] = 1.0
    C = np.zeros((d_out - r, r))
    if d_out > r:
        k = np.arange(d_out - r)
        C[k, (7 * k + 3) % r] = 1.0
    return Wp, C


def layout_probe_activations(M: int, d_in: int, seed: int) -> np.ndarray:
    """Values that are exact in bf16 and fp16: +-m * 2^e, m in [1, 2) with 3
    fraction bits, e in [-4, 7]."""
    rng = np.random.default_rng([int(seed), 13])
    mant = 1.0 + rng.integers(0, 8, size=(M, d_in)) / 8.0
    expo = rng.integers(-4, 8, size=(M, d_in)).astype(np.float64)
    sign = np.where(rng.integers(0, 2, size=(M, d_in)) == 0, -1.0, 1.0)
    return sign * mant * np.exp2(expo)


def integer_layer(d_in: int, d_out: int, r: int, M: int, seed: int, density: float = 0.05):
    """Integer-valued X in {-2..2}, W_p and C in {-1, 0, 1}, sparse enough that
    every partial sum stays small; all products and sums are then exact in
    fp32, bf16 and fp16, so any summation order gives the same bits.

    Returns (X, Wp, C) as fp64 arrays with integer values, plus the bound
    max|Y_p| and max|Y| (computed by the caller's oracle if needed).
    """
    rng = np.random.default_rng([int(seed), 17])
    X = rng.integers(-2, 3, size=(M, d_in)).astype(np.float64)
    # keep |Y_p| <= 2 * nnz(W_p row) small: at most ~density*d_in nonzeros
    nnz_p = max(1, min(d_in, int(round(density * d_in)), 16))
    Wp = np.zeros((r, d_in))
    for j in range(r):
        cols = rng.choice(d_in, size=nnz_p, replace=False)
        Wp[j, cols] = rng.choice([-1.0, 1.0], size=nnz_p)
    nnz_c = max(1, min(r, 8))
    C = np.zeros((d_out - r, r))
    for k in range(d_out - r):
        cols = rng.choice(r, size=nnz_c, replace=False)
        C[k, cols] = rng.choice([-1.0, 1.0], size=nnz_c)
    return X, Wp, C


# --------------------------------------------------------------------------
# the workloads: LLaMA layer shapes with synthetic values
# --------------------------------------------------------------------------
# name -> (config index, layer index, d_in, d_out, r, dtype, M values, layer kind)
# layer kind "built": (I, W_p, C) come from the PIFA build of W' = U V
# (every configuration, the LLaMA-70B shapes included).
RANK_SWEEP = (0.1, 0.2, 0.3, 0.4, 0.5, 0.6, 0.7, 0.8, 0.9)

CONFIGS = {
    "A_f32_256": (0, 0, 256, 256, 128, "f32", (32,), "built"),
    "B_attn_4096": (1, 0, 4096, 4096, 2048, "bf16", (1, 16, 128, 2048, 4096), "built"),
    "C_mlp_up_4096x11008": (2, 0, 4096, 11008, 2048, "bf16", (1, 4096), "built"),
    "C_mlp_down_11008x4096": (2, 1, 11008, 4096, 2048, "bf16", (1, 4096), "built"),
    "D_70b_sq_8192": (3, 0, 8192, 8192, 4096, "bf16", (1, 4096), "built"),
    "D_70b_up_8192x28672": (3, 1, 8192, 28672, 4096, "bf16", (1, 4096), "built"),
}
for _i, _rho in enumerate(RANK_SWEEP):
    CONFIGS["E_sweep_r%02d" % round(100 * _rho)] = (4, _i, 4096, 4096, int(round(_rho * 4096)), "bf16",
                                                    (1, 4096), "built")
