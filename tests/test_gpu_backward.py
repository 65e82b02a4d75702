"""Backward pass of the PIFA layer (pifa_layer_backward) against the fp64
oracle's chain rule, through the C ABI.

The oracle evaluates the gradients on the same bf16 bits the GPU consumes
(X, dY, W_p, C); Y_p for dC comes from the GPU forward's output Y[:, I], whose
bf16 rounding is inside the bar.  Bar: rel_F <= 5e-3 for dX (bf16 out), dW_p
and dC (fp32 out).  At the benchmark size the oracle checks sampled rows of
dX and sampled pivot slots of dW_p and dC (a reduced problem that yields
exactly those gradient entries).
"""
import numpy as np
import pytest

import oracle
from paper_2501_19090_amd import inputs

from gpu_util import (DeviceLayer, activations, config_layer, from_dev, gaussian_layer, rel_fro, sample_rows,
                      to_dev, torch_mod)

pytestmark = pytest.mark.gpu
TOL = 5e-3


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    if not torch_mod().cuda.is_available():
        pytest.skip("no GPU")


def _grads(lay, x_dev, g_dev, M):
    from paper_2501_19090_amd import pifa
    torch = torch_mod()
    y = lay.forward(x_dev, M)
    dX = torch.full((max(M, 1), lay.d_in), float("nan"), dtype=torch.bfloat16, device="cuda:0")
    dWp = torch.full((lay.r, lay.d_in), float("nan"), dtype=torch.float32, device="cuda:0")
    dC = torch.full((max(lay.d_out - lay.r, 1), lay.r), float("nan"), dtype=torch.float32, device="cuda:0")
    pifa.pifa_layer_backward(lay.handle, x_dev, y, g_dev, dX, dWp, dC if lay.d_out > lay.r else None, M)
    torch.cuda.synchronize()
    return dX, dWp, dC


def _check_small(lay, M, seed):
    x_dev, x64 = activations(M, lay.d_in, seed, "bf16")
    g_dev, g64 = activations(M, lay.d_out, seed + 1000, "bf16")
    dX, dWp, dC = _grads(lay, x_dev, g_dev, M)
    rX, rW, rC = oracle.pifa_backward(x64, g64, lay.piv, lay.npiv, lay.Wp, lay.C)
    assert rel_fro(from_dev(dX), rX) <= TOL, ("dX", M)
    assert rel_fro(from_dev(dWp), rW) <= TOL, ("dWp", M)
    if rC.size:
        assert rel_fro(from_dev(dC), rC) <= TOL, ("dC", M)


@pytest.mark.parametrize("d_in,d_out,r", [(256, 320, 96), (136, 203, 72), (512, 1024, 300), (128, 96, 96)])
def test_backward_small_shapes(d_in, d_out, r):
    """Ragged r (not a multiple of 64), n_np not a multiple of 8, r = d_out."""
    piv, npiv, Wp, C, *_ = gaussian_layer(d_in, d_out, r, 50 + r)
    lay = DeviceLayer(piv, npiv, Wp, C, "bf16")
    try:
        for M in (1, 5, 17, 100, 300):
            _check_small(lay, M, seed=M)
    finally:
        lay.close()


def test_backward_full_size_sampled():
    """The LLaMA-7B attention shape (4096 x 4096, r = 2048) at M = 4096."""
    piv, npiv, Wp, C, *_ = config_layer("B_attn_4096")
    lay = DeviceLayer(piv, npiv, Wp, C, "bf16")
    try:
        M = 4096
        x_dev, x64 = activations(M, lay.d_in, 21, "bf16")
        g_dev, g64 = activations(M, lay.d_out, 22, "bf16")
        dX, dWp, dC = _grads(lay, x_dev, g_dev, M)
        # dX rows depend only on their own rows of X and G: the first, the
        # last and 510 seeded rows (the oracle's backward of all 4096 rows
        # takes minutes)
        rows = sample_rows(M, k=510)
        rX, _, _ = oracle.pifa_backward(x64[rows], g64[rows], lay.piv, lay.npiv, lay.Wp, lay.C)
        assert rel_fro(from_dev(dX)[rows], rX) <= TOL
        # dW_p[S, :] and dC[:, S] for a few pivot slots S: the same gradients
        # of the reduced layer whose pivot set is I[S] (outputs re-indexed)
        S = np.array([0, 1, 517, 1024, 2046, 2047])
        Gs = np.concatenate([g64[:, lay.piv[S]], g64[:, lay.npiv]], axis=1)
        piv_s = np.arange(S.size, dtype=np.int32)
        npiv_s = np.arange(S.size, S.size + lay.npiv.size, dtype=np.int32)
        _, rW, rC = oracle.pifa_backward(x64, Gs, piv_s, npiv_s, lay.Wp[S], lay.C[:, S])
        assert rel_fro(from_dev(dWp)[S], rW) <= TOL
        assert rel_fro(from_dev(dC)[:, S], rC) <= TOL
        assert torch_mod().isfinite(dWp).all() and torch_mod().isfinite(dC).all()
    finally:
        lay.close()


def test_backward_deterministic_and_optional_outputs():
    from paper_2501_19090_amd import pifa
    torch = torch_mod()
    piv, npiv, Wp, C, *_ = gaussian_layer(256, 320, 96, 146)
    lay = DeviceLayer(piv, npiv, Wp, C, "bf16")
    try:
        M = 77
        x_dev, _ = activations(M, 256, 3, "bf16")
        g_dev, _ = activations(M, 320, 4, "bf16")
        a = _grads(lay, x_dev, g_dev, M)
        b = _grads(lay, x_dev, g_dev, M)
        for u, v in zip(a, b):
            assert torch.equal(u, v)
        # outputs may be skipped one by one
        y = lay.forward(x_dev, M)
        dWp = torch.zeros((96, 256), dtype=torch.float32, device="cuda:0")
        pifa.pifa_layer_backward(lay.handle, x_dev, y, g_dev, None, dWp, None, M)
        torch.cuda.synchronize()
        assert torch.equal(dWp, a[1])
        # M = 0 is the zero gradient
        pifa.pifa_layer_backward(lay.handle, x_dev, y, g_dev, None, dWp, None, 0)
        torch.cuda.synchronize()
        assert not dWp.any()
    finally:
        lay.close()


def test_backward_rejects_f32_layer():
    from paper_2501_19090_amd import pifa
    piv, npiv, Wp, C, *_ = gaussian_layer(64, 80, 32, 7)
    lay = DeviceLayer(piv, npiv, Wp, C, "f32")
    try:
        x_dev, _ = activations(4, 64, 1, "f32")
        # the binding refuses fp32 activations for the (bf16-only) backward ...
        with pytest.raises(TypeError):
            pifa.pifa_layer_backward(lay.handle, x_dev, x_dev, x_dev, None, None, None, 4)
        # ... and the library itself refuses the fp32 layer
        st = pifa.lib().pifa_layer_backward(lay.handle, x_dev.data_ptr(), x_dev.data_ptr(), x_dev.data_ptr(), 4,
                                            None, None, None, None)
        assert st == pifa.PIFA_ERR_UNSUPPORTED
    finally:
        lay.close()
