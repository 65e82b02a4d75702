"""pifa_forward_noalloc (the library's fixed per-GPU scratch as workspace)
against pifa_forward on the same layer and inputs: the same kernels on the
same launch plan, so the outputs must agree bit for bit.  Two calls in a row
per layer, the second on a smaller batch (the scratch keeps the first call's
contents), and a batch whose workspace exceeds the scratch is refused."""
import numpy as np
import pytest

from paper_2501_19090_amd import inputs

from gpu_util import DeviceLayer, activations, config_layer, from_dev, torch_mod

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    if not torch_mod().cuda.is_available():
        pytest.skip("no GPU")


def _both(lay, x_dev, M):
    """(Y from pifa_forward, Y from pifa_forward_noalloc) for the first M rows."""
    torch = torch_mod()
    from paper_2501_19090_amd import pifa
    x = x_dev[:M].contiguous()
    y_ref = torch.full((M, lay.d_out), float("nan"), dtype=x.dtype, device="cuda:0")
    y_new = torch.full((M, lay.d_out), float("nan"), dtype=x.dtype, device="cuda:0")
    pifa.pifa_forward(lay.handle, x, y_ref, M)
    pifa.pifa_forward_noalloc(lay.handle, x, y_new, M)
    torch.cuda.synchronize()
    return from_dev(y_ref), from_dev(y_new)


@pytest.mark.parametrize("Ms", [(4096, 300), (2048, 16), (128, 1), (17, 5)])
def test_noalloc_matches_forward_attention_layer(Ms):
    """The LLaMA-7B attention layer (4096 x 4096, r = 2048): prefill, K-split
    and decode launch plans, each followed by a smaller batch."""
    piv, npiv, Wp, C, *_ = config_layer("B_attn_4096")
    lay = DeviceLayer(piv, npiv, Wp, C, "bf16")
    try:
        x_dev, _ = activations(max(Ms), lay.d_in, 77, "bf16")
        for M in Ms:
            ref, new = _both(lay, x_dev, M)
            assert np.isfinite(ref).all()
            assert np.array_equal(ref, new), (M, np.nanmax(np.abs(ref - new)))
    finally:
        lay.close()


def test_noalloc_matches_forward_f32_and_ragged():
    """fp32 layer (config A) and a ragged bf16 layer, two calls each."""
    piv, npiv, Wp, C, *_ = config_layer("A_f32_256")
    for dims, dt in (((256, 256, 128), "f32"), ((1024, 520, 410), "bf16")):
        d_in, d_out, r = dims
        if dt == "f32":
            lay = DeviceLayer(piv, npiv, Wp, C, dt)
        else:
            p2, n2 = inputs.random_partition(d_out, r, seed=9)
            U, V = inputs.lowrank_factors(r, d_in, r, 9)
            rng = np.random.default_rng(9)
            lay = DeviceLayer(p2, n2, U @ V, rng.standard_normal((d_out - r, r)) * 0.25, dt)
        try:
            x_dev, _ = activations(300, d_in, 5, dt)
            for M in (300, 7):
                ref, new = _both(lay, x_dev, M)
                assert np.array_equal(ref, new), (dt, M)
        finally:
            lay.close()


def test_noalloc_refuses_a_batch_beyond_its_scratch():
    torch = torch_mod()
    from paper_2501_19090_amd import pifa
    piv, npiv, Wp, C, *_ = config_layer("B_attn_4096")
    lay = DeviceLayer(piv, npiv, Wp, C, "bf16")
    try:
        M = 16384  # Y_p alone is 16384 x 2048 fp16 = 64 MiB
        x = torch.zeros((M, lay.d_in), dtype=torch.bfloat16, device="cuda:0")
        y = torch.full((M, lay.d_out), 7.0, dtype=torch.bfloat16, device="cuda:0")
        with pytest.raises(pifa.PifaError) as e:
            pifa.pifa_forward_noalloc(lay.handle, x, y, M)
        assert e.value.status == pifa.PIFA_ERR_TOO_LARGE
        torch.cuda.synchronize()
        assert bool((y == 7.0).all())  # nothing was launched
    finally:
        lay.close()
