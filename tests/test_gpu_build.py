"""GPU PIFA build (pifa_build_f64) against the fp64 oracle's build.

Both run QR with column pivoting with exact residual norms and the same
tie rule, so on generic inputs the pivot sets agree exactly; C agrees to
rounding, the layer must be lossless (reconstruction <= 1e-10), and the
hand-derived worked examples (exact ties) must come out as derived.
"""
import json
import os

import numpy as np
import pytest

import oracle
from paper_2501_19090_amd import inputs

from gpu_util import DeviceLayer, activations, config_layer, from_dev, rel_fro, sample_rows, torch_mod

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    if not torch_mod().cuda.is_available():
        pytest.skip("no GPU")


def _gpu_build(W, r):
    torch = torch_mod()
    from paper_2501_19090_amd import pifa
    Wd = torch.from_numpy(np.ascontiguousarray(W, dtype=np.float64)).to("cuda:0")
    piv, npiv, Wp, C, report = pifa.pifa_build_f64(Wd, r)
    return piv, npiv, Wp.cpu().numpy(), C.cpu().numpy(), report


@pytest.mark.parametrize("d_out,d_in,r", [(64, 48, 16), (48, 64, 16), (96, 96, 1), (32, 48, 32), (256, 256, 128),
                                          (333, 200, 150), (1024, 1024, 512), (2752, 1024, 512),
                                          (1024, 2752, 512), (4096, 4096, 2048),
                                          # columns longer than the LDS-held pivot column (8192 rows)
                                          (96, 9000, 48), (40, 8193, 40)])
def test_build_matches_oracle(d_out, d_in, r):
    U, V = inputs.lowrank_factors(d_out, d_in, r, seed=d_out + r)
    W = U @ V
    ref = oracle.build_pifa(W, r)
    piv, npiv, Wp, C, report = _gpu_build(W, r)
    assert np.array_equal(piv, ref["pivot_idx"]) and np.array_equal(npiv, ref["nonpivot_idx"])
    assert np.array_equal(Wp, ref["Wp"])
    if C.size:
        assert rel_fro(C, ref["C"]) <= 1e-10
    assert report[3] == 1.0
    assert oracle.reconstruction_error(W, piv, npiv, Wp, C) <= 1e-10


@pytest.mark.timeout(900)  # the oracle build of a LLaMA-70B shape takes minutes (then cached)
@pytest.mark.parametrize("name", ["D_70b_sq_8192", "D_70b_up_8192x28672"])
def test_build_matches_oracle_llama70b_shapes(name):
    """The GPU build of the LLaMA-70B layers (8192 x 8192 and 8192 -> 28672,
    r = 4096) selects exactly the oracle's pivots, and its C agrees."""
    cfg, lay_i, d_in, d_out, r, *_ = inputs.CONFIGS[name]
    piv_o, npiv_o, Wp_o, C_o, U, V = config_layer(name)
    W = U @ V
    piv, npiv, Wp, C, report = _gpu_build(W, r)
    assert np.array_equal(piv, piv_o) and np.array_equal(npiv, npiv_o)
    assert np.array_equal(Wp, Wp_o)
    err_c = rel_fro(C, C_o)
    rec = oracle.reconstruction_error(W, piv, npiv, Wp, C)
    print("%s: identical pivots, C rel_F %.2e, reconstruction %.2e" % (name, err_c, rec), flush=True)
    assert err_c <= 1e-10
    assert report[3] == 1.0
    assert rec <= 1e-10


def test_build_worked_examples():
    with open(os.path.join(GOLDEN, "qrcp_worked_examples.json")) as f:
        examples = json.load(f)["examples"]
    for ex in examples:
        W = np.array(ex["W"], dtype=np.float64)
        piv, npiv, Wp, C, _ = _gpu_build(W, ex["r"])
        assert piv.tolist() == ex["pivot_idx"], ex["name"]
        assert npiv.tolist() == ex["nonpivot_idx"], ex["name"]
        np.testing.assert_array_equal(Wp, np.array(ex["Wp"], dtype=np.float64))
        np.testing.assert_allclose(C, np.array(ex["C"], dtype=np.float64), rtol=0, atol=1e-14)


def test_build_rejects_wrong_rank():
    from paper_2501_19090_amd import pifa
    U, V = inputs.lowrank_factors(64, 64, 8, 3)
    U[:, 1] = U[:, 0]
    with pytest.raises(pifa.PifaError) as e:
        _gpu_build(U @ V, 8)
    assert e.value.status == pifa.PIFA_ERR_NOT_RANK_R
    W = np.random.default_rng(0).standard_normal((40, 30))
    with pytest.raises(pifa.PifaError):
        _gpu_build(W, 10)


def test_gpu_built_layer_forward():
    """Build on the GPU, round to bf16, run the forward: the result matches
    the oracle evaluated on the same rounded layer, and the dense product."""
    d_out, d_in, r = 1536, 1024, 512
    U, V = inputs.lowrank_factors(d_out, d_in, r, 31)
    W = U @ V
    piv, npiv, Wp, C, _ = _gpu_build(W, r)
    lay = DeviceLayer(piv, npiv, Wp, C, "bf16")
    try:
        for M in (1, 16, 300):
            x_dev, x64 = activations(M, d_in, 5, "bf16")
            y = from_dev(lay.forward(x_dev))
            assert rel_fro(y, lay.oracle(x64)) <= 5e-3
            assert rel_fro(y, x64 @ W.T) <= 2e-2
    finally:
        lay.close()
