"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Bars: the pivot / non-pivot layout is bit-exact (layout probe, integer-exact
layers); Gaussian layers meet rel_F <= 1e-5 (fp32) and <= 5e-3 (bf16 inputs,
fp32 accumulation).  Full-size configurations are run at their real M in the
launch configuration the benchmark times; the oracle checks a seeded subset
of rows there (rows of Y are independent).
"""
import numpy as np
import pytest

import oracle
from paper_2501_19090_amd import inputs

from gpu_util import (DeviceLayer, activations, config_layer, from_dev, gaussian_layer, rel_fro,
                      sample_rows, to_dev, torch_mod)

pytestmark = pytest.mark.gpu

TOL = {"bf16": 5e-3, "f32": 1e-5}
# 4 / 5 straddle the decode launch-shape switch (few activation rows vs many)
DECODE_AND_PREFILL_M = (1, 2, 4, 5, 7, 16, 17, 33, 64, 100, 128, 129, 300)


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    torch = torch_mod()
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield


def _check_layout(lay: DeviceLayer, M: int, seed: int):
    x64 = inputs.layout_probe_activations(M, lay.d_in, seed)
    st, x64 = inputs.round_to(x64, lay.dtype)
    y = from_dev(lay.forward(to_dev(st)))
    # closed form of the probe, for every row
    k = np.arange(lay.d_out - lay.r)
    assert np.array_equal(y[:, lay.piv], x64[:, : lay.r])
    assert np.array_equal(y[:, lay.npiv], x64[:, (7 * k + 3) % lay.r])
    # and the oracle, element by element, on sampled rows
    rows = sample_rows(M)
    assert np.array_equal(y[rows], lay.oracle(x64[rows]))


# ------------------------------------------------------------------ layout probe
PROBE_CONFIGS = ["B_attn_4096", "C_mlp_up_4096x11008", "C_mlp_down_11008x4096", "D_70b_sq_8192",
                 "D_70b_up_8192x28672", "E_sweep_r10", "E_sweep_r90"]


@pytest.mark.timeout(900)  # the first use of a LLaMA-70B shape runs its oracle build (minutes)
@pytest.mark.parametrize("name", PROBE_CONFIGS)
def test_layout_probe_bitexact_at_config_shapes(name):
    """The index sets of each configuration (the oracle's I for built layers)
    with probe weights: every output element must land exactly."""
    cfg, lay_i, d_in, d_out, r, dt, Ms, kind = inputs.CONFIGS[name]
    piv, npiv, *_ = config_layer(name)
    Wp, C = inputs.layout_probe_layer(d_in, d_out, r)
    lay = DeviceLayer(piv, npiv, Wp, C, dt)
    try:
        for M in (1, 16, 17, 300):
            _check_layout(lay, M, seed=M)
    finally:
        lay.close()


@pytest.mark.parametrize("dims", [(64, 64, 64), (72, 200, 1), (136, 96, 40), (1024, 520, 410),
                                  (256, 4096, 256), (4104, 130, 129)])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_layout_probe_ragged_shapes(dims, dtype):
    """Ragged r, d_out and d_in around tile edges; r = d_out (empty C) and r = 1."""
    d_in, d_out, r = dims
    piv, npiv = inputs.random_partition(d_out, r, seed=d_out + r)
    Wp, C = inputs.layout_probe_layer(d_in, d_out, r)
    lay = DeviceLayer(piv, npiv, Wp, C, dtype)
    try:
        for M in DECODE_AND_PREFILL_M:
            _check_layout(lay, M, seed=M + 1)
    finally:
        lay.close()


def test_layout_probe_unsorted_partition():
    """Any order of the index sets is accepted and honoured as given."""
    d_in, d_out, r = 256, 384, 136
    rng = np.random.default_rng(5)
    perm = rng.permutation(d_out).astype(np.int32)
    piv, npiv = perm[:r], perm[r:]
    Wp, C = inputs.layout_probe_layer(d_in, d_out, r)
    for dtype in ("bf16", "f32"):
        lay = DeviceLayer(piv, npiv, Wp, C, dtype)
        try:
            for M in (3, 16, 200):
                _check_layout(lay, M, seed=M)
        finally:
            lay.close()


# ------------------------------------------------------------------ integer exact
@pytest.mark.parametrize("dims", [(512, 768, 320), (1024, 1024, 512), (256, 2752, 200), (2048, 640, 448)])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_integer_layers_bitexact(dims, dtype):
    """Integer-valued X, W_p, C: every partial sum is exact, so the GPU must
    equal the oracle bit for bit whatever its tiling and K splitting."""
    d_in, d_out, r = dims
    piv, npiv = inputs.random_partition(d_out, r, seed=r)
    for M in DECODE_AND_PREFILL_M:
        X, Wp, C = inputs.integer_layer(d_in, d_out, r, M, seed=M)
        lay = DeviceLayer(piv, npiv, Wp, C, dtype)
        try:
            st, x64 = inputs.round_to(X, dtype)
            y = from_dev(lay.forward(to_dev(st)))
            ref = lay.oracle(x64)
            assert np.abs(ref).max() <= 256
            assert np.array_equal(y, ref), (M, np.abs(y - ref).max())
        finally:
            lay.close()


@pytest.mark.parametrize("dims", [(2048, 4096, 2048), (1536, 2752, 1536), (2560, 4096, 2458), (1280, 4096, 1229),
                                  (1024, 1024, 410)])
def test_integer_layers_bitexact_large_tiles(dims):
    """M = 4096 selects the large prefill tiles (256 x 128; 256 x 192 for the
    2496-wide pivot product of r = 2458 and the 2867-wide non-pivot product
    of r = 1229; 128 x 64 for the 448-wide pivot product of r = 410, which
    is not split); integer data keeps every element exact, checked on sampled
    rows against the oracle."""
    d_in, d_out, r = dims
    M = 4096
    piv, npiv = inputs.random_partition(d_out, r, seed=r + 1)
    X, Wp, C = inputs.integer_layer(d_in, d_out, r, M, seed=7)
    for dtype in ("bf16", "f32"):
        lay = DeviceLayer(piv, npiv, Wp, C, dtype)
        try:
            st, x64 = inputs.round_to(X, dtype)
            y = from_dev(lay.forward(to_dev(st)))
            rows = sample_rows(M, k=64, seed=3)
            assert np.array_equal(y[rows], lay.oracle(x64[rows]))
        finally:
            lay.close()


@pytest.mark.parametrize("dims", [(8192, 14336, 1536), (8200, 14336, 1500)])
@pytest.mark.parametrize("M", [1, 2, 3, 4, 5])
def test_integer_layers_bitexact_long_weight_streams(dims, M):
    """Decode rows against weight streams long enough for the streaming decode
    kernel: W_p 1536 x 8192 (96 groups of 16 rows, each split over two
    workgroups, x 64 blocks of 128 K) and C 12800 x 1536 (800 groups x 12
    blocks, fewer than one per wave); the second layer has a ragged last K
    block in W_p (d_in = 8200) and 1500 pivots padded to 1536.  M = 5 takes
    the kernel with one workgroup per group.  Integer data: bit-exact against
    the oracle."""
    d_in, d_out, r = dims
    piv, npiv = inputs.random_partition(d_out, r, seed=11)
    X, Wp, C = inputs.integer_layer(d_in, d_out, r, M, seed=M + 40)
    lay = DeviceLayer(piv, npiv, Wp, C, "bf16")
    try:
        st, x64 = inputs.round_to(X, "bf16")
        y = from_dev(lay.forward(to_dev(st)))
        ref = lay.oracle(x64)
        assert np.abs(ref).max() <= 256
        assert np.array_equal(y, ref), (M, np.abs(y - ref).max())
    finally:
        lay.close()


def test_layout_probe_large_m():
    """Probe weights at the attention shape with M = 4096 rows."""
    name = "B_attn_4096"
    cfg, lay_i, d_in, d_out, r, dt, Ms, kind = inputs.CONFIGS[name]
    piv, npiv, *_ = config_layer(name)
    Wp, C = inputs.layout_probe_layer(d_in, d_out, r)
    lay = DeviceLayer(piv, npiv, Wp, C, dt)
    try:
        for M in (2048, 4096):
            _check_layout(lay, M, seed=M)
    finally:
        lay.close()


# ------------------------------------------------------------------ Gaussian configs
# Configurations whose oracle forward at M = 4096 is checked on a seeded row
# subset (first, last and 510 more rows; rows of Y are independent): the
# LLaMA-70B shapes, about 1.1 TFLOP of fp64 work for all 4096 rows.
SUBSET_CONFIGS = ("D_70b_sq_8192", "D_70b_up_8192x28672")


def _gaussian_case(name: str, M: int):
    cfg, lay_i, d_in, d_out, r, dt, Ms, kind = inputs.CONFIGS[name]
    piv, npiv, Wp, C, _, _ = config_layer(name)
    lay = DeviceLayer(piv, npiv, Wp, C, dt)
    try:
        x_dev, x64 = activations(M, d_in, inputs.config_seed(cfg, lay_i), dt)
        y = from_dev(lay.forward(x_dev))
        assert np.isfinite(y).all()
        rows = sample_rows(M, k=510, seed=cfg) if (name in SUBSET_CONFIGS and M > 512) else sample_rows(M)
        ref = lay.oracle(x64[rows])
        got = y[rows]
        err = rel_fro(got, ref)
        err_p = rel_fro(got[:, lay.piv], ref[:, lay.piv])
        err_np = rel_fro(got[:, lay.npiv], ref[:, lay.npiv]) if lay.npiv.size else 0.0
        print("%s M=%d rows=%d rel_F=%.3e (pivot %.3e, non-pivot %.3e)"
              % (name, M, rows.size, err, err_p, err_np), flush=True)
        assert err <= TOL[dt]
        from paper_2501_19090_amd import pifa
        assert pifa.pifa_layer_overflow_count(lay.handle) == 0
    finally:
        lay.close()


def test_config_a_fp32():
    _gaussian_case("A_f32_256", 32)


def test_config_a_fp32_matches_dense():
    """Config A's check: Y against dense X W^T of the unrounded W."""
    piv, npiv, Wp, C, U, V = config_layer("A_f32_256")
    lay = DeviceLayer(piv, npiv, Wp, C, "f32")
    try:
        x_dev, x64 = activations(32, 256, inputs.config_seed(0), "f32")
        y = from_dev(lay.forward(x_dev))
        assert rel_fro(y, x64 @ (U @ V).T) <= 1e-5
    finally:
        lay.close()


@pytest.mark.parametrize("M", [1, 16, 128, 2048, 4096])
def test_config_b(M):
    _gaussian_case("B_attn_4096", M)


@pytest.mark.parametrize("name", ["C_mlp_up_4096x11008", "C_mlp_down_11008x4096"])
@pytest.mark.parametrize("M", [1, 4096])
def test_config_c(name, M):
    _gaussian_case(name, M)


@pytest.mark.timeout(900)  # the oracle build of a LLaMA-70B shape takes minutes
@pytest.mark.parametrize("name", ["D_70b_sq_8192", "D_70b_up_8192x28672"])
@pytest.mark.parametrize("M", [1, 4096])
def test_config_d(name, M):
    """Layers built by the oracle (QR with column pivoting of the Gaussian
    rank-4096 W' = U V), as for every other configuration."""
    _gaussian_case(name, M)


@pytest.mark.parametrize("M", [3, 16, 17, 33, 100, 255, 256, 257, 1000])
def test_config_b_ragged_m(M):
    _gaussian_case("B_attn_4096", M)


# ------------------------------------------------------------------ semantics
def test_m_zero_is_noop():
    torch = torch_mod()
    piv, npiv = inputs.random_partition(96, 40, 1)
    Wp, C = inputs.layout_probe_layer(64, 96, 40)
    lay = DeviceLayer(piv, npiv, Wp, C, "bf16")
    try:
        from paper_2501_19090_amd import pifa
        x = torch.zeros((1, 64), dtype=torch.bfloat16, device="cuda:0")
        y = torch.full((1, 96), 3.0, dtype=torch.bfloat16, device="cuda:0")
        pifa.pifa_forward(lay.handle, x, y, 0)
        torch.cuda.synchronize()
        assert bool((y == 3.0).all())
    finally:
        lay.close()


def test_deterministic_and_stream_ordered():
    """Same inputs give the same bits, also on a side stream."""
    torch = torch_mod()
    piv, npiv, Wp, C, _, _ = gaussian_layer(1024, 1536, 512, 3)
    lay = DeviceLayer(piv, npiv, Wp, C, "bf16")
    try:
        from paper_2501_19090_amd import pifa
        for M in (1, 9, 16, 700):
            x_dev, _ = activations(M, 1024, 11, "bf16")
            y1 = lay.forward(x_dev)
            s = torch.cuda.Stream()
            y2 = torch.empty_like(y1)
            s.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(s):
                pifa.pifa_forward(lay.handle, x_dev, y2, M, s)
            s.synchronize()
            assert torch.equal(y1, y2)
    finally:
        lay.close()


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_non_finite_inputs_stay_in_their_rows(dtype):
    """A NaN or an Inf in a row of X makes every output of that row non-finite
    (the products and the fp16 hand-off carry them), and leaves every other
    row bit-identical to the run without them (rows are independent), in the
    decode, split-K and prefill launch shapes."""
    torch = torch_mod()
    piv, npiv, Wp, C, _, _ = gaussian_layer(512, 768, 256, 8)
    lay = DeviceLayer(piv, npiv, Wp, C, dtype)
    try:
        for M in (1, 5, 16, 100, 700):
            x_dev, _ = activations(M, 512, 21 + M, dtype)
            y_clean = lay.forward(x_dev)
            x_bad = x_dev.clone()
            bad = {0: float("nan")} if M == 1 else {0: float("nan"), M - 1: float("inf")}
            for row, v in bad.items():
                x_bad[row, 5 + row % 7] = v
            y = lay.forward(x_bad)
            for row in bad:
                assert not bool(torch.isfinite(y[row]).any()), (M, row)
            keep = [m for m in range(M) if m not in bad]
            if keep:
                assert torch.equal(y[keep], y_clean[keep]), M
    finally:
        lay.close()


def test_short_buffers_are_rejected_before_the_call():
    """The binding checks buffer sizes against the handle's dimensions, so a
    tensor that is too small never reaches the kernels (which would access it
    past its end)."""
    torch = torch_mod()
    from paper_2501_19090_amd import pifa
    piv, npiv = inputs.random_partition(96, 40, 3)
    Wp, C = inputs.layout_probe_layer(64, 96, 40)
    lay = DeviceLayer(piv, npiv, Wp, C, "bf16")
    try:
        x = torch.zeros((8, 64), dtype=torch.bfloat16, device="cuda:0")
        y_short = torch.zeros((8, 95), dtype=torch.bfloat16, device="cuda:0")
        with pytest.raises(ValueError):
            pifa.pifa_forward(lay.handle, x, y_short)
        with pytest.raises(ValueError):
            pifa.pifa_forward(lay.handle, x[:4], torch.zeros((8, 96), dtype=torch.bfloat16, device="cuda:0"), 8)
        y = torch.zeros((8, 96), dtype=torch.bfloat16, device="cuda:0")
        pifa.pifa_forward(lay.handle, x, y)  # the right sizes still run
        torch.cuda.synchronize()
        w = torch.zeros((96, 64), dtype=torch.bfloat16, device="cuda:0")
        with pytest.raises(ValueError):
            pifa.dense_forward(w[:50], x, y, d_out=96)
    finally:
        lay.close()


def test_wrong_dtypes_are_rejected_before_the_call():
    """The library reads raw bytes, so the binding refuses activations, outputs
    or coefficients whose element type differs from the layer's."""
    torch = torch_mod()
    from paper_2501_19090_amd import pifa
    piv, npiv = inputs.random_partition(96, 40, 3)
    Wp, C = inputs.layout_probe_layer(64, 96, 40)
    lay = DeviceLayer(piv, npiv, Wp, C, "bf16")
    try:
        x = torch.zeros((8, 64), dtype=torch.bfloat16, device="cuda:0")
        y = torch.zeros((8, 96), dtype=torch.bfloat16, device="cuda:0")
        with pytest.raises(TypeError):
            pifa.pifa_forward(lay.handle, x.float(), y)
        with pytest.raises(TypeError):
            pifa.pifa_forward(lay.handle, x, y.float())
        with pytest.raises(ValueError):
            pifa.pifa_forward(lay.handle, x.cpu(), y)
        with pytest.raises(TypeError):
            pifa.pifa_layer_create(lay.wp_dev, lay.c_dev.float(), lay.piv, lay.npiv, (64, 96, 40))
        w = torch.zeros((96, 64), dtype=torch.bfloat16, device="cuda:0")
        with pytest.raises(TypeError):
            pifa.dense_forward(w, x.float(), y)
        pifa.pifa_forward(lay.handle, x, y)  # matching types still run
        torch.cuda.synchronize()
    finally:
        lay.close()


def _exchanged_pivot_set(W, piv, npiv, swaps: int):
    """A second valid pivot set: starting from QRCP's, repeatedly swap the
    pivot j and non-pivot k with the largest |C[k, j]| (a basis exchange that
    does not shrink the pivot rows' volume, so C stays bounded)."""
    piv, npiv = list(piv), list(npiv)
    for _ in range(swaps):
        C = np.linalg.lstsq(W[piv].T, W[npiv].T, rcond=None)[0].T
        k, j = np.unravel_index(np.argmax(np.abs(C)), C.shape)
        piv[j], npiv[k] = npiv[k], piv[j]
    piv, npiv = np.sort(np.array(piv, np.int32)), np.sort(np.array(npiv, np.int32))
    C = np.linalg.lstsq(W[piv].T, W[npiv].T, rcond=None)[0].T
    return piv, npiv, C


def test_pivot_set_invariance():
    """The same rank-r W with two different well-conditioned pivot sets gives
    the same Y (exactly so in exact arithmetic; Sec. 3.2 allows any r
    independent rows)."""
    U, V = inputs.lowrank_factors(1536, 1024, 384, 21)
    W = U @ V
    b = oracle.build_pifa(W, 384)
    piv2, npiv2, C2 = _exchanged_pivot_set(W, b["pivot_idx"], b["nonpivot_idx"], 12)
    assert not np.array_equal(piv2, b["pivot_idx"])
    x_dev, x64 = activations(200, 1024, 3, "bf16")
    l1 = DeviceLayer(b["pivot_idx"], b["nonpivot_idx"], b["Wp"], b["C"], "bf16")
    l2 = DeviceLayer(piv2, npiv2, W[piv2], C2, "bf16")
    try:
        for M in (5, 200):
            y1, y2 = from_dev(l1.forward(x_dev[:M])), from_dev(l2.forward(x_dev[:M]))
            assert rel_fro(y1, l1.oracle(x64[:M])) <= 5e-3
            assert rel_fro(y2, l2.oracle(x64[:M])) <= 5e-3
            # rounding the two layers' weights to bf16 perturbs them differently,
            # so the outputs agree to the weight-rounding level
            dense = x64[:M] @ W.T
            assert rel_fro(y1, y2) <= 2e-2
            assert rel_fro(y1, dense) <= 2e-2 and rel_fro(y2, dense) <= 2e-2
    finally:
        l1.close()
        l2.close()


def test_intermediate_overflow_is_counted():
    """|Y_p * 2^s| beyond fp16's range is reported, not silently wrong, on the
    weight-streaming path (M <= 128) and on the GEMM path alike."""
    from paper_2501_19090_amd import pifa
    piv, npiv, Wp, C, _, _ = gaussian_layer(512, 768, 256, 4)
    lay = DeviceLayer(piv, npiv, Wp, C, "bf16")
    try:
        assert pifa.pifa_layer_overflow_count(lay.handle) == 0
        pifa.pifa_layer_set_intermediate_scale(lay.handle, 20)
        seen = 0
        for M in (4, 100, 300):
            x_dev, _ = activations(M, 512, 2, "bf16")
            y = from_dev(lay.forward(x_dev))
            assert not np.isfinite(y[:, lay.npiv]).all()
            assert np.isfinite(y[:, lay.piv]).all()
            count = pifa.pifa_layer_overflow_count(lay.handle)
            assert count > seen, M
            seen = count
    finally:
        lay.close()


def test_intermediate_scale_keeps_parity():
    """A moderate power-of-two hand-off scale leaves results within the bar."""
    from paper_2501_19090_amd import pifa
    piv, npiv, Wp, C, _, _ = gaussian_layer(512, 768, 256, 4)
    lay = DeviceLayer(piv, npiv, Wp, C, "bf16")
    try:
        for s in (-6, 3):
            pifa.pifa_layer_set_intermediate_scale(lay.handle, s)
            for M in (5, 300):
                x_dev, x64 = activations(M, 512, 9, "bf16")
                assert rel_fro(from_dev(lay.forward(x_dev)), lay.oracle(x64)) <= 5e-3
        assert pifa.pifa_layer_overflow_count(lay.handle) == 0
    finally:
        lay.close()


def test_weight_bytes():
    from paper_2501_19090_amd import pifa
    piv, npiv = inputs.random_partition(300, 100, 2)
    Wp, C = inputs.layout_probe_layer(128, 300, 100)
    for dtype, es in (("bf16", 2), ("f32", 4)):
        lay = DeviceLayer(piv, npiv, Wp, C, dtype)
        try:
            assert pifa.pifa_layer_weight_bytes(lay.handle) == es * (100 * 128 + 200 * 100) + 4 * 300
        finally:
            lay.close()


def test_misaligned_activation_rejected():
    torch = torch_mod()
    from paper_2501_19090_amd import pifa
    piv, npiv = inputs.random_partition(64, 32, 1)
    Wp, C = inputs.layout_probe_layer(64, 64, 32)
    lay = DeviceLayer(piv, npiv, Wp, C, "bf16")
    try:
        buf = torch.zeros(4 * 64 + 1, dtype=torch.bfloat16, device="cuda:0")
        x = buf[1:].view(4, 64)  # 2-byte offset
        y = torch.empty((4, 64), dtype=torch.bfloat16, device="cuda:0")
        st = pifa.lib().pifa_forward(lay.handle, x.data_ptr(), y.data_ptr(), 4, None)
        assert st == pifa.PIFA_ERR_UNSUPPORTED
    finally:
        lay.close()
