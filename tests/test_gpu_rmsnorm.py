"""GPU parity of dg_rmsnorm against the CPU oracle, bit for bit (gfx950):
the descriptor-ordered sum of squares, then IEEE sqrt and division, then the
element step with its rounding points."""
import numpy as np
import pytest

import oracle
from paper_2609_11356_amd import inputs
from tests.gpu_util import assert_bits_equal, dev_bf16, dev_f32, host_bits

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dg():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_11356_amd import dg as _dg
    _dg.lib()
    return _dg


def run(dg, desc, X, w=None, eps=0.0):
    import torch
    d = dg.Desc(**dict(desc, reduce="sumsq"))
    out_bf16 = desc.get("out", "f32") == "bf16"
    Y = torch.full(X.shape, float("nan"), dtype=torch.bfloat16 if out_bf16 else torch.float32, device="cuda")
    dg.dg_rmsnorm(d, dev_f32(X), None if w is None else dev_bf16(w), eps, Y)
    torch.cuda.synchronize()
    return host_bits(Y)


DESCS = [dict(leaf_w=64), dict(leaf_w=7, fma=0), dict(leaf_w=256, leaf_layout="strided", lane_fold="down"),
         dict(leaf_w=32, leaf_layout="strided"), dict(leaf_w=256, leaf_layout="strided", out="bf16"),
         dict(leaf_w=64, out="bf16", norm_round="pre_weight"),
         dict(leaf_w=128, leaf_layout="strided", lane_fold="down", out="bf16", norm_round="pre_weight"),
         dict(leaf_w=64, leaf_layout="strided", fma=0)]


@pytest.mark.parametrize("di", range(len(DESCS)))
def test_rmsnorm_ragged(dg, di):
    """Widths that defeat the vector path (cols % 4 != 0), fewer elements
    than lanes, several leaves, the widest row the one-pass kernel holds in
    registers (8192) and one past it (two passes); with and without the
    weight; eps 0 and 1e-5."""
    desc = DESCS[di]
    for cols in (1, 3, 64, 100, 1000, 4099, 8192, 8193):
        X = inputs.lognormal_f32(cols + 7 * di, (21, cols))
        w = inputs.normal_bf16(cols + 3, (cols,), 1.0)
        for ww in (None, w):
            for eps in (0.0, 1e-5):
                got = run(dg, desc, X, ww, eps)
                want = oracle.rmsnorm(desc, X, ww, eps=eps)
                assert_bits_equal(got, want, "%s cols %d w %s eps %g" % (desc, cols, ww is not None, eps))


@pytest.mark.parametrize("desc", [dict(leaf_w=256, leaf_layout="strided", lane_fold="down", out="bf16"),
                                  dict(leaf_w=64, out="bf16", norm_round="pre_weight")])
def test_rmsnorm_full_config(dg, desc):
    """X 16384 x 8192 fp32 (log-normal magnitudes), a bf16 weight, eps 1e-5:
    every output against the oracle."""
    X = inputs.rowsum_input(8)
    w = inputs.normal_bf16(10, (X.shape[1],), 1.0)
    assert_bits_equal(run(dg, desc, X, w, 1e-5), oracle.rmsnorm(desc, X, w, eps=1e-5), "rmsnorm %s" % desc)


def test_rmsnorm_unaligned_rows_take_two_passes(dg):
    """X 4 bytes past a 16-byte boundary: the one-pass kernel's vector loads
    do not apply; same bits."""
    import torch
    X = inputs.lognormal_f32(51, (9, 1024))
    w = inputs.normal_bf16(52, (1024,), 1.0)
    desc = dict(leaf_w=256, leaf_layout="strided", lane_fold="down", out="bf16")
    want = oracle.rmsnorm(desc, X, w, eps=1e-5)
    buf = torch.empty(X.size + 1, dtype=torch.float32, device="cuda")
    buf[1:] = torch.from_numpy(X.reshape(-1)).cuda()
    Y = torch.full(X.shape, float("nan"), dtype=torch.bfloat16, device="cuda")
    dg.dg_rmsnorm(dg.Desc(**dict(desc, reduce="sumsq")), buf[1:].data_ptr(), dev_bf16(w).data_ptr(), 1e-5,
                  Y.data_ptr(), 9, 1024)
    torch.cuda.synchronize()
    assert_bits_equal(host_bits(Y), want)


def test_rmsnorm_root_and_division_over_exponents(dg):
    """One element per row: s = x^2, so the reciprocal root runs on 2^20
    values spread over the whole binary32 range (squares that underflow to
    subnormals or zero and overflow to infinity included) and the outputs
    carry every bit of it; eps 0 and a tiny eps."""
    rng = np.random.default_rng(12)
    n = 1 << 20
    X = (rng.uniform(1, 2, n) * np.exp2(rng.integers(-80, 70, n)) * rng.choice([-1, 1], n)).astype(np.float32)
    X[:4] = [0.0, -0.0, np.float32(2.0 ** -149), np.float32(3.0e38)]
    X = X[:, None]
    for eps in (0.0, 1e-30):
        assert_bits_equal(run(dg, dict(leaf_w=1), X, None, eps), oracle.rmsnorm(dict(leaf_w=1), X, eps=eps),
                          "eps %g" % eps)


def test_rmsnorm_close_to_torch(dg):
    """Sanity against the textbook formula in float64 (not a parity check)."""
    X = inputs.lognormal_f32(40, (64, 2048))
    w = inputs.normal_bf16(41, (2048,), 1.0)
    wf = inputs.bf16_bits_to_f32(w).astype(np.float64)
    X64 = X.astype(np.float64)
    ref = X64 / np.sqrt((X64 ** 2).mean(1, keepdims=True) + 1e-5) * wf
    got = run(dg, dict(leaf_w=64), X, w, 1e-5).astype(np.float64)
    assert np.all(np.abs(got - ref) <= 2.0 ** -17 * np.abs(ref) + 1e-30)
