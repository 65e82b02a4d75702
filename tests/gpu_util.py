"""Helpers for the GPU parity tests: seeded layers (built by the oracle or
drawn directly), upload of the rounded bits, and comparison metrics."""
from __future__ import annotations

import functools

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


@functools.lru_cache(maxsize=None)
def gaussian_layer(d_in: int, d_out: int, r: int, seed: int, kind: str = "built"):
    """(pivot_idx, nonpivot_idx, W_p, C) in fp64, plus U, V when built."""
    if kind == "built":
        U, V = inputs.lowrank_factors(d_out, d_in, r, seed)
        b = oracle.build_pifa(U @ V, r)
        return b["pivot_idx"], b["nonpivot_idx"], b["Wp"], b["C"], U, V
    piv, npiv, Wp, C = inputs.direct_layer(d_in, d_out, r, seed)
    return piv, npiv, Wp, C, None, None


def config_layer(name: str):
    cfg, lay, d_in, d_out, r, dt, Ms, kind = inputs.CONFIGS[name]
    return gaussian_layer(d_in, d_out, r, inputs.config_seed(cfg, lay), kind)


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


def sample_rows(M: int, k: int = 24, seed: int = 0) -> np.ndarray:
    """Rows to check against the oracle: all rows when few, else the first,
    the last and a seeded random subset."""
    if M <= 64:
        return np.arange(M)
    rng = np.random.default_rng([seed, M])
    return np.unique(np.concatenate([[0, M - 1], rng.choice(M, size=k, replace=False)]))


def activations(M: int, d_in: int, seed: int, dtype: str):
    st, x64 = inputs.round_to(inputs.activations(M, d_in, seed), dtype)
    return to_dev(st), x64
