"""GPU parity of dg_rowsum against the CPU oracle, bit for bit (gfx950)."""
import numpy as np
import pytest

import oracle
from paper_2609_11356_amd import inputs
from tests.gpu_util import assert_bits_equal, dev_f32

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
    d = dg.Desc(**desc)
    Xd = dev_f32(X)
    out = torch.full((X.shape[0],), float("nan"), dtype=torch.float32, device="cuda")
    dg.dg_rowsum(d, Xd, out)
    torch.cuda.synchronize()
    return out.cpu().numpy()


@pytest.mark.parametrize("desc", [dict(leaf_w=64, reduce="sum"), dict(leaf_w=64, reduce="sumsq", fma=1),
                                  dict(leaf_w=64, reduce="sumsq", fma=0)])
def test_rowsum_full_config(dg, desc):
    """X 16384 x 8192 fp32, log-normal magnitudes (sigma 2), random signs:
    every row against the oracle."""
    X = inputs.rowsum_input(8)
    got = run(dg, desc, X)
    want = oracle.rowsum(desc, X)
    assert_bits_equal(got, want, "rowsum %s" % desc)


@pytest.mark.parametrize("cols", [0, 1, 3, 63, 64, 65, 100, 4095, 4096, 4097, 8191, 12288, 70000])
@pytest.mark.parametrize("leaf_w", [1, 7, 64, 100])
def test_rowsum_ragged(dg, cols, leaf_w):
    """Ragged widths (partial leaves, leaf counts that are not powers of
    two, more than 64 leaves), unaligned rows (cols % 4 != 0), leaves wider
    than 64 (read straight from HBM), and row counts that leave a workgroup
    partly idle."""
    rows = 7
    X = inputs.lognormal_f32(cols * 31 + leaf_w, (rows, cols))
    for desc in (dict(leaf_w=leaf_w), dict(leaf_w=leaf_w, reduce="sumsq", fma=1)):
        assert_bits_equal(run(dg, desc, X), oracle.rowsum(desc, X), "rowsum %s cols %d" % (desc, cols))


def test_rowsum_zero_rows_and_negzero(dg):
    X = np.full((5, 300), -0.0, dtype=np.float32)
    got = run(dg, dict(leaf_w=64), X)
    assert_bits_equal(got, oracle.rowsum(dict(leaf_w=64), X))
    assert np.all(np.signbit(got))  # a row of -0 sums to -0


def test_rowsum_independent_of_row_count(dg):
    X = inputs.rowsum_input(9, rows=1000, cols=2048)
    a = run(dg, dict(leaf_w=64), X)
    b = run(dg, dict(leaf_w=64), X[:37].copy())
    assert np.array_equal(a[:37].view(np.uint32), b.view(np.uint32))
