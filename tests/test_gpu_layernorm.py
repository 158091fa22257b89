"""GPU parity of dg_layernorm against the CPU oracle, bit for bit (gfx950):
two descriptor-ordered row sums (mean, then squares of the centred values),
IEEE sqrt and division, then the element step with its rounding points."""
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


def run(dg, desc, X, w=None, b=None, eps=0.0):
    import torch
    d = dg.Desc(**desc)
    out_bf16 = desc.get("out", "f32") == "bf16"
    Y = torch.full(X.shape, float("nan"), dtype=torch.bfloat16 if out_bf16 else torch.float32, device="cuda")
    dg.dg_layernorm(d, dev_f32(X), None if w is None else dev_bf16(w), None if b is None else dev_bf16(b), eps, Y)
    torch.cuda.synchronize()
    return host_bits(Y)


DESCS = [dict(leaf_w=256, leaf_layout="strided", lane_fold="down"),
         dict(leaf_w=128, leaf_layout="strided", out="bf16", norm_round="pre_weight"),
         dict(leaf_w=64, leaf_layout="strided", lane_fold="down", fma=0, out="bf16"),
         dict(leaf_w=64), dict(leaf_w=7, out="bf16", fma=0), dict(leaf_w=32, leaf_layout="strided", lane_fold="down")]


@pytest.mark.parametrize("di", range(len(DESCS)))
def test_layernorm_ragged(dg, di):
    """One-pass and four-pass paths; widths off the vector path, fewer
    elements than lanes, one past the register limit; weight and bias each
    present or not; a large common offset."""
    desc = DESCS[di]
    for cols in (1, 3, 64, 100, 1000, 4099, 8192, 8193):
        X = (inputs.lognormal_f32(cols + 13 * di, (21, cols), sigma=1.0) + 30).astype(np.float32)
        w = inputs.normal_bf16(cols + 5, (cols,), 1.0)
        b = inputs.normal_bf16(cols + 6, (cols,), 1.0)
        for ww, bb in ((None, None), (w, None), (w, b), (None, b)):
            got = run(dg, desc, X, ww, bb, 1e-5)
            want = oracle.layernorm(desc, X, ww, bb, eps=1e-5)
            assert_bits_equal(got, want, "%s cols %d w %s b %s" % (desc, cols, ww is not None, bb is not None))


@pytest.mark.parametrize("desc", [dict(leaf_w=256, leaf_layout="strided", lane_fold="down", out="bf16"),
                                  dict(leaf_w=64, out="bf16", norm_round="pre_weight")])
def test_layernorm_full_config(dg, desc):
    """16384 x 8192 rows (log-normal magnitudes), bf16 weight and bias,
    eps 1e-5: every output against the oracle."""
    X = inputs.rowsum_input(8)
    w = inputs.normal_bf16(16, (8192,), 1.0)
    b = inputs.normal_bf16(17, (8192,), 1.0)
    assert_bits_equal(run(dg, desc, X, w, b, 1e-5), oracle.layernorm(desc, X, w, b, eps=1e-5), str(desc))


def test_layernorm_constant_rows(dg):
    """Constant rows: the centred values are exactly 0, so with eps 0 the
    root is 0 and 0 * inf is NaN on both sides; with eps > 0 the output is
    the bias."""
    X = np.full((5, 256), 3.25, dtype=np.float32)
    b = inputs.normal_bf16(18, (256,), 1.0)
    for desc in (DESCS[0], DESCS[3]):
        for eps in (0.0, 1e-5):
            assert_bits_equal(run(dg, desc, X, None, b, eps), oracle.layernorm(desc, X, None, b, eps=eps))
