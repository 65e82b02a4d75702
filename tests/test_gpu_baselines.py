"""GPU parity of the same-engine baselines: dense X W^T and low-rank
(X V^T) U^T, stateless and prepacked, against the fp64 oracle."""
import numpy as np
import pytest

import oracle
from paper_2501_19090_amd import inputs

from gpu_util import activations, from_dev, rel_fro, sample_rows, to_dev, torch_mod

pytestmark = pytest.mark.gpu
TOL = {"bf16": 5e-3, "f32": 1e-5}


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    if not torch_mod().cuda.is_available():
        pytest.skip("no GPU")


def _uv(d_in, d_out, r, seed, dtype):
    U, V = inputs.lowrank_factors(d_out, d_in, r, seed)
    u_st, U64 = inputs.round_to(U, dtype)
    v_st, V64 = inputs.round_to(V, dtype)
    return to_dev(u_st), U64, to_dev(v_st), V64


def _run_all(d_in, d_out, r, M, dtype, seed=1):
    """Run dense, stateless low-rank and prepacked low-rank; return errors."""
    torch = torch_mod()
    from paper_2501_19090_amd import pifa
    u_dev, U64, v_dev, V64 = _uv(d_in, d_out, r, seed, dtype)
    w_st, W64 = inputs.round_to(U64 @ V64, dtype)
    w_dev = to_dev(w_st)
    x_dev, x64 = activations(M, d_in, seed + 5, dtype)
    rows = sample_rows(M)
    errs = {}
    y = torch.full((M, d_out), float("nan"), dtype=x_dev.dtype, device="cuda:0")
    pifa.dense_forward(w_dev, x_dev, y)
    torch.cuda.synchronize()
    ref_d = oracle.dense_forward(x64[rows], W64)
    errs["dense"] = rel_fro(from_dev(y)[rows], ref_d)
    hd = pifa.dense_layer_create(w_dev)
    try:
        y.fill_(float("nan"))
        pifa.dense_layer_forward(hd, x_dev, y)
        torch.cuda.synchronize()
        errs["dense_layer"] = rel_fro(from_dev(y)[rows], ref_d)
    finally:
        pifa.dense_layer_destroy(hd)
    ref_lr = oracle.lowrank_forward(x64[rows], U64, V64)
    if dtype == "f32" or r % 8 == 0:
        y.fill_(float("nan"))
        pifa.lowrank_uv_forward(u_dev, v_dev, x_dev, y)
        torch.cuda.synchronize()
        errs["lowrank"] = rel_fro(from_dev(y)[rows], ref_lr)
    h = pifa.lowrank_layer_create(u_dev, v_dev)
    try:
        y.fill_(float("nan"))
        pifa.lowrank_layer_forward(h, x_dev, y)
        torch.cuda.synchronize()
        errs["lowrank_layer"] = rel_fro(from_dev(y)[rows], ref_lr)
    finally:
        pifa.lowrank_layer_destroy(h)
    return errs


@pytest.mark.parametrize("M", [1, 5, 16, 17, 200, 4096])
def test_baselines_config_b_shape(M):
    errs = _run_all(4096, 4096, 2048, M, "bf16")
    print("M=%d" % M, errs, flush=True)
    assert all(e <= TOL["bf16"] for e in errs.values()), errs


@pytest.mark.parametrize("dims", [(256, 256, 128), (136, 200, 33), (512, 1000, 410)])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("M", [1, 16, 40, 100, 128])
def test_baselines_ragged(dims, dtype, M):
    d_in, d_out, r = dims
    errs = _run_all(d_in, d_out, r, M, dtype, seed=d_out)
    assert all(e <= TOL[dtype] for e in errs.values()), errs


@pytest.mark.parametrize("M", [1, 16, 300])
def test_dense_integer_bitexact(M):
    torch = torch_mod()
    from paper_2501_19090_amd import pifa
    rng = np.random.default_rng(M)
    d_in, d_out = 1024, 776
    X = rng.integers(-2, 3, size=(M, d_in)).astype(np.float64)
    W = np.zeros((d_out, d_in))
    for n in range(d_out):
        W[n, rng.choice(d_in, 16, replace=False)] = rng.choice([-1.0, 1.0], 16)
    for dtype in ("bf16", "f32"):
        w_st, W64 = inputs.round_to(W, dtype)
        x_st, x64 = inputs.round_to(X, dtype)
        x_dev = to_dev(x_st)
        y = torch.full((M, d_out), float("nan"), dtype=x_dev.dtype, device="cuda:0")
        w_dev = to_dev(w_st)
        pifa.dense_forward(w_dev, x_dev, y)
        torch.cuda.synchronize()
        ref = oracle.dense_forward(x64, W64)
        assert np.array_equal(from_dev(y), ref)
        h = pifa.dense_layer_create(w_dev)
        try:
            y.fill_(float("nan"))
            pifa.dense_layer_forward(h, x_dev, y)
            torch.cuda.synchronize()
            assert np.array_equal(from_dev(y), ref)
        finally:
            pifa.dense_layer_destroy(h)
