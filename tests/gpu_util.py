"""Helpers for the GPU parity tests: seeded layers built by the oracle,
upload of the rounded bits, and comparison metrics."""
from __future__ import annotations

import contextlib
import functools
import sys
import time

import numpy as np

import oracle
from paper_2501_19090_amd import inputs


def torch_mod():
    import torch
    return torch


def to_dev(storage: np.ndarray):
    """Upload bf16 bits (uint16) or fp32 values to cuda:0 as bf16 / fp32."""
    torch = torch_mod()
    if storage.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(storage).view(np.int16)).to("cuda:0").view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(storage, dtype=np.float32)).to("cuda:0")


def from_dev(t) -> np.ndarray:
    return t.float().cpu().numpy().astype(np.float64)


def rel_fro(got, ref) -> float:
    n = np.linalg.norm(ref)
    return float(np.linalg.norm(got - ref) / (n if n > 0 else 1.0))


# pytest's capture manager (set by conftest): long oracle builds print their
# progress past the capture, so a run shows it while the build is under way
CAPTURE_MANAGER = None
# builds of a W' with at least this many elements report progress
LARGE_BUILD_ELEMS = 1 << 26


def _uncaptured():
    if CAPTURE_MANAGER is None:
        return contextlib.nullcontext()
    return CAPTURE_MANAGER.global_and_fixture_disabled()


@functools.lru_cache(maxsize=None)
def gaussian_layer(d_in: int, d_out: int, r: int, seed: int):
    """(pivot_idx, nonpivot_idx, W_p, C, U, V) in fp64: the oracle's PIFA build
    of the Gaussian rank-r W' = U V.  Built once per process."""
    U, V = inputs.lowrank_factors(d_out, d_in, r, seed)
    if d_out * d_in < LARGE_BUILD_ELEMS:
        b = oracle.build_pifa(U @ V, r)
        return b["pivot_idx"], b["nonpivot_idx"], b["Wp"], b["C"], U, V
    with _uncaptured():
        t0 = time.perf_counter()
        print("oracle build of the %d x %d rank-%d layer (seed %d) ..." % (d_out, d_in, r, seed),
              file=sys.stderr, flush=True)
        b = oracle.build_pifa(U @ V, r, progress=512)
        print("oracle build of the %d x %d layer done in %.1f s" % (d_out, d_in, time.perf_counter() - t0),
              file=sys.stderr, flush=True)
    return b["pivot_idx"], b["nonpivot_idx"], b["Wp"], b["C"], U, V


def config_layer(name: str):
    cfg, lay, d_in, d_out, r, dt, Ms, kind = inputs.CONFIGS[name]
    assert kind == "built"
    return gaussian_layer(d_in, d_out, r, inputs.config_seed(cfg, lay))


class DeviceLayer:
    """A PIFA layer rounded once to `dtype`, on the GPU and as fp64 values."""

    def __init__(self, piv, npiv, Wp, C, dtype: str):
        from paper_2501_19090_amd import pifa
        self.piv, self.npiv = np.asarray(piv, np.int32), np.asarray(npiv, np.int32)
        self.r, self.d_in = Wp.shape
        self.d_out = self.r + self.npiv.size
        self.dtype = dtype
        wp_st, self.Wp = inputs.round_to(Wp, dtype)
        c_st, self.C = inputs.round_to(C, dtype)
        self.wp_dev = to_dev(wp_st)
        self.c_dev = to_dev(c_st) if C.size else None
        self.handle = pifa.pifa_layer_create(self.wp_dev, self.c_dev, self.piv, self.npiv,
                                             (self.d_in, self.d_out, self.r))

    def forward(self, x_dev, M=None):
        from paper_2501_19090_amd import pifa
        torch = torch_mod()
        M = x_dev.shape[0] if M is None else M
        y = torch.full((max(M, 1), self.d_out), float("nan"), dtype=x_dev.dtype, device=x_dev.device)
        pifa.pifa_forward(self.handle, x_dev, y, M)
        torch.cuda.synchronize()
        return y

    def oracle(self, x64):
        return oracle.pifa_forward(x64, self.piv, self.npiv, self.Wp, self.C, d_out=self.d_out)

    def close(self):
        from paper_2501_19090_amd import pifa
        if self.handle:
            pifa.pifa_layer_destroy(self.handle)
            self.handle = 0


# Rows of Y are independent, so a check may cover a subset of them; up to
# this many rows every row is compared with the oracle.
ALL_ROWS_MAX_M = 4096


def sample_rows(M: int, k: int | None = None, seed: int = 0) -> np.ndarray:
    """Rows to compare with the oracle.  By default every row up to
    ALL_ROWS_MAX_M rows; with k (or above that size) the first row, the last
    row and a seeded random subset, k + 2 >= 256 rows in all."""
    if k is None and M <= ALL_ROWS_MAX_M:
        return np.arange(M)
    k = 510 if k is None else k
    if M <= k + 2:
        return np.arange(M)
    rng = np.random.default_rng([seed, M])
    inner = rng.choice(np.arange(1, M - 1), size=k, replace=False)
    return np.unique(np.concatenate([[0, M - 1], inner]))


def activations(M: int, d_in: int, seed: int, dtype: str):
    st, x64 = inputs.round_to(inputs.activations(M, d_in, seed), dtype)
    return to_dev(st), x64
