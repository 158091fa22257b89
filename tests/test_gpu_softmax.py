"""GPU parity of dg_softmax against the CPU oracle, bit for bit (gfx950):
the exact max shift, the library's own exp, the row sum in the
descriptor's order, one reciprocal and one product per element."""
import numpy as np
import pytest

import oracle
from paper_2609_11356_amd import inputs
from tests.gpu_util import assert_bits_equal, dev_f32, host_bits

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dg():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_11356_amd import dg as _dg
    _dg.lib()
    return _dg


def run(dg, desc, X):
    import torch
    d = dg.Desc(**dict(desc, reduce="sum"))
    out_bf16 = desc.get("out", "f32") == "bf16"
    Y = torch.full(X.shape, float("nan"), dtype=torch.bfloat16 if out_bf16 else torch.float32, device="cuda")
    dg.dg_softmax(d, dev_f32(X), Y)
    torch.cuda.synchronize()
    return host_bits(Y)


DESCS = [dict(leaf_w=256, leaf_layout="strided", lane_fold="down"), dict(leaf_w=128, leaf_layout="strided", out="bf16"),
         dict(leaf_w=64, leaf_layout="strided", lane_fold="down", out="bf16"), dict(leaf_w=64),
         dict(leaf_w=7, out="bf16"), dict(leaf_w=32, leaf_layout="strided", lane_fold="down")]


@pytest.mark.parametrize("di", range(len(DESCS)))
def test_softmax_ragged(dg, di):
    """One-pass (strided lanes, rows up to 8192 in registers) and three-pass
    paths; widths off the vector path, fewer elements than lanes, and one
    past the register limit."""
    desc = DESCS[di]
    for cols in (1, 3, 64, 100, 1000, 4099, 8192, 8193):
        X = (inputs.lognormal_f32(cols + 11 * di, (21, cols), sigma=1.0) * 4).astype(np.float32)
        assert_bits_equal(run(dg, desc, X), oracle.softmax(desc, X), "%s cols %d" % (desc, cols))


@pytest.mark.parametrize("desc", [dict(leaf_w=256, leaf_layout="strided", lane_fold="down", out="bf16"),
                                  dict(leaf_w=64, out="bf16")])
def test_softmax_full_config(dg, desc):
    """16384 x 8192 logits (log-normal magnitudes, random signs): every
    output against the oracle."""
    X = inputs.lognormal_f32(13, (16384, 8192), sigma=1.0)
    assert_bits_equal(run(dg, desc, X), oracle.softmax(desc, X), "softmax %s" % desc)


def test_softmax_special_values(dg):
    """NaN and +inf rows are NaN everywhere, -inf entries give 0, wide
    exponent spreads underflow to 0 exactly as on the CPU."""
    X = inputs.lognormal_f32(14, (8, 512), sigma=1.0)
    X[0, 5] = np.nan
    X[1, 9] = np.inf
    X[2, ::3] = -np.inf
    X[3] *= 200.0
    X[4] = -np.inf
    for desc in (DESCS[0], DESCS[3]):
        assert_bits_equal(run(dg, desc, X), oracle.softmax(desc, X), str(desc))


def test_softmax_close_to_torch(dg):
    """Sanity against float64 (not a parity check)."""
    X = inputs.lognormal_f32(15, (64, 2048), sigma=1.0)
    X64 = X.astype(np.float64)
    E = np.exp(X64 - X64.max(1, keepdims=True))
    ref = E / E.sum(1, keepdims=True)
    got = run(dg, DESCS[0], X).astype(np.float64)
    assert np.all(np.abs(got - ref) <= 2.0 ** -17 * ref + 1e-45)
