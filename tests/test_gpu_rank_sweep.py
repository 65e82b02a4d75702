"""Rank sweep on 4096 x 4096 (r / d = 0.1 ... 0.9): PIFA parity at M = 1 and
M = 4096 on layers built by the oracle."""
import pytest

from paper_2501_19090_amd import inputs

from test_gpu_parity import _gaussian_case

pytestmark = pytest.mark.gpu

SWEEP = [n for n in inputs.CONFIGS if n.startswith("E_sweep")]


@pytest.mark.parametrize("name", SWEEP)
@pytest.mark.parametrize("M", [1, 4096])
def test_rank_sweep(name, M):
    _gaussian_case(name, M)
