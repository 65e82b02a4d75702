"""The peak probes return rates and clocks within physical bounds on the
device at hand (diagnostics beside the roofline; no layer's path uses them)."""
import pytest

from gpu_util import torch_mod

pytestmark = pytest.mark.gpu


def test_mfma_probes_are_plausible():
    torch_mod()
    from paper_2501_19090_amd import pifa
    tf_const, mhz_const = pifa.pifa_probe_mfma(4000)
    tf_rand, mhz_rand = pifa.pifa_probe_mfma_random(4003)  # rounded up to a multiple of 8
    # dense bf16 peak of the chip: 2516.6 TFLOP/s at 2400 MHz
    for tf, mhz in ((tf_const, mhz_const), (tf_rand, mhz_rand)):
        assert 100.0 < tf < 2516.6 * 1.05, tf
        assert 500.0 < mhz < 2600.0, mhz
        # the rate follows the clock: never above the peak at that clock
        assert tf <= 2516.6 * mhz / 2400.0 * 1.05, (tf, mhz)


def test_mfma_probe_rejects_bad_arguments():
    torch_mod()
    from paper_2501_19090_amd import pifa
    for fn in (pifa.pifa_probe_mfma, pifa.pifa_probe_mfma_random):
        with pytest.raises(pifa.PifaError) as e:
            fn(0)
        assert e.value.status == pifa.PIFA_ERR_INVALID_ARG


def test_hbm_read_probe_is_plausible():
    torch = torch_mod()
    from paper_2501_19090_amd import pifa
    buf = torch.zeros(1 << 28, dtype=torch.uint8, device="cuda:0")
    gbps = pifa.pifa_probe_hbm_read(buf, 3)
    assert 500.0 < gbps < 20000.0, gbps  # 256 MiB can sit in the 256 MB Infinity Cache
