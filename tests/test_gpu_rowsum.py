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


# ------------------------------------- strided leaves, count-up / count-down fold

STRIDED_W = [1, 2, 4, 8, 16, 32, 64, 128, 256]


@pytest.mark.parametrize("W", STRIDED_W)
@pytest.mark.parametrize("fold", ["up", "down"])
def test_rowsum_strided_ragged(dg, W, fold):
    """W lanes each taking every W-th element, folded by the count-up or the
    count-down butterfly: fewer elements than lanes, partial last steps,
    widths that defeat the vector loads (cols % 4 != 0), row counts that
    leave a wave's row groups partly idle; SUM and both SUMSQ rules."""
    for cols in (0, 1, 3, 5, W - 1, W, W + 1, 3 * W + 7, 1000, 4099):
        if cols < 0:
            continue
        rows = 37
        X = inputs.lognormal_f32(cols * 17 + W, (rows, cols))
        for extra in (dict(), dict(reduce="sumsq", fma=1), dict(reduce="sumsq", fma=0)):
            desc = dict(leaf_w=W, leaf_layout="strided", lane_fold=fold, **extra)
            assert_bits_equal(run(dg, desc, X), oracle.rowsum(desc, X), "%s cols %d" % (desc, cols))


@pytest.mark.parametrize("fold", ["up", "down"])
def test_rowsum_strided_full_config(dg, fold):
    """The 16384 x 8192 reduction with 256 strided lanes (the vector path),
    every row against the oracle, and the count-down order differing from
    the count-up one on this data."""
    X = inputs.rowsum_input(8)
    desc = dict(leaf_w=256, leaf_layout="strided", lane_fold=fold)
    got = run(dg, desc, X)
    assert_bits_equal(got, oracle.rowsum(desc, X), "rowsum %s" % desc)
    if fold == "down":
        up = oracle.rowsum(dict(desc, lane_fold="up"), X)
        assert not np.array_equal(got.view(np.uint32), up.view(np.uint32))


def test_rowsum_strided_unaligned_rows(dg):
    """A row base 4 bytes past a 16-byte boundary takes the scalar loads and
    gives the same bits."""
    import torch
    X = inputs.lognormal_f32(77, (9, 1024))
    desc = dict(leaf_w=256, leaf_layout="strided", lane_fold="down")
    want = oracle.rowsum(desc, X)
    buf = torch.empty(X.size + 1, dtype=torch.float32, device="cuda")
    buf[1:] = torch.from_numpy(X.reshape(-1)).cuda()
    out = torch.full((9,), float("nan"), dtype=torch.float32, device="cuda")
    d = dg.Desc(**desc)
    dg.dg_rowsum(d, buf[1:].data_ptr(), out.data_ptr(), 9, 1024)
    torch.cuda.synchronize()
    assert_bits_equal(out.cpu().numpy(), want)


def test_rowsum_strided_independent_of_row_count(dg):
    X = inputs.rowsum_input(9, rows=1000, cols=2048)
    for W in (32, 256):
        desc = dict(leaf_w=W, leaf_layout="strided", lane_fold="down")
        a = run(dg, desc, X)
        b = run(dg, desc, X[:37].copy())
        assert np.array_equal(a[:37].view(np.uint32), b.view(np.uint32)), W


@pytest.mark.parametrize("seed", range(64))
def test_rowsum_random_descriptor(dg, seed):
    """Seeded random descriptors (leaf width and layout, the fold direction of
    strided lanes, SUM or SUMSQ under either fma rule) on ragged row and
    column counts, every row compared with the oracle."""
    rng = np.random.default_rng(70_000 + seed)
    desc = {}
    if rng.random() < 0.5:
        desc.update(leaf_layout="strided", leaf_w=int(rng.choice([1, 2, 8, 32, 64, 128, 256])),
                    lane_fold=str(rng.choice(["up", "down"])))
    else:
        desc["leaf_w"] = int(rng.choice([1, 3, 16, 64, 100, 257]))
    if rng.random() < 0.5:
        desc.update(reduce="sumsq", fma=int(rng.integers(2)))
    rows = int(rng.choice([1, 5, 64, 300]))
    cols = int(rng.choice([0, 1, 31, 64, 255, 1000, 4099, 9000]))
    X = inputs.lognormal_f32(90_000 + seed, (rows, cols))
    print("seed %d rows %d cols %d desc %s" % (seed, rows, cols, desc), flush=True)
    assert_bits_equal(run(dg, desc, X), oracle.rowsum(desc, X), "rowsum %s %dx%d" % (desc, rows, cols))
