"""GPU parity of dg_gemm_colsum: C as dg_gemm writes it, and the column
sums bit for bit against the oracle's balanced tree down each column of
the oracle's C (gfx950)."""
import numpy as np
import pytest

import oracle
from paper_2609_11356_amd import inputs
from tests.gpu_util import assert_bits_equal, dev_bf16, host_bits

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dg():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_11356_amd import dg as _dg
    _dg.lib()
    return _dg


def run(dg, desc, A, B, bias=None):
    import torch
    M, K = A.shape
    N = B.shape[1]
    d = dg.Desc(**desc)
    out_bf16 = desc.get("out", "f32") == "bf16"
    C = torch.full((M, N), float("nan"), dtype=torch.bfloat16 if out_bf16 else torch.float32, device="cuda")
    cs = torch.full((N,), float("nan"), dtype=torch.float32, device="cuda")
    dg.dg_gemm_colsum(d, dev_bf16(A), dev_bf16(B), None if bias is None else dev_bf16(bias), C, cs)
    torch.cuda.synchronize()
    return host_bits(C), cs.cpu().numpy()


@pytest.mark.parametrize("desc", [dict(tile_k=64), dict(tile_k=64, out="bf16", epilogue="bias_silu"),
                                  dict(tile_k=64, split_k=4, split_combine="tree")])
@pytest.mark.parametrize("shape", [(1, 40, 256), (37, 72, 512), (256, 64, 256), (300, 520, 1032), (777, 96, 512)])
def test_colsum_ragged(dg, desc, shape):
    """Row counts below, at and across the 256-row runs, ragged columns."""
    M, N, K = shape
    A = inputs.spread_bf16(M + 1, (M, K))
    B = inputs.spread_bf16(N + 2, (K, N))
    bias = inputs.normal_bf16(3, (N,), 0.5)
    use_bias = desc.get("epilogue", "none") != "none"
    C, cs = run(dg, desc, A, B, bias if use_bias else None)
    Cw = oracle.gemm(desc, A, B, bias if use_bias else None)
    assert_bits_equal(C, Cw, "C %s %s" % (desc, shape))
    assert_bits_equal(cs, oracle.colsum(Cw), "colsum %s %s" % (desc, shape))


def test_colsum_mlp_shape(dg):
    """The MLP shape 2048 x 14336 x 4096 with fp32 output: the column sums
    of the whole output against the oracle's tree over the GPU's C (C itself
    is checked against the oracle on sampled outputs by the GEMM tests)."""
    A, B, bias = inputs.mlp()
    desc = dict(mma="16x16x32", tile_k=64)
    C, cs = run(dg, desc, A, B)
    assert_bits_equal(cs, oracle.colsum(C), "colsum of the MLP-shape output")
    rng = np.random.default_rng(5)
    ii, jj = rng.integers(0, 2048, 300), rng.integers(0, 14336, 300)
    assert_bits_equal(C[ii, jj], oracle.gemm_at(desc, A, B, None, ii, jj), "sampled C")


def test_colsum_no_rows(dg):
    import torch
    d = dg.Desc(tile_k=64)
    C = torch.empty((0, 48), dtype=torch.float32, device="cuda")
    cs = torch.full((48,), float("nan"), dtype=torch.float32, device="cuda")
    A = torch.empty((0, 64), dtype=torch.bfloat16, device="cuda")
    B = torch.zeros((64, 48), dtype=torch.bfloat16, device="cuda")
    dg.dg_gemm_colsum(d, A, B, None, C, cs)
    torch.cuda.synchronize()
    assert np.all(cs.cpu().numpy() == 0.0) and not np.any(np.signbit(cs.cpu().numpy()))


@pytest.mark.parametrize("M,desc", [(1000, dict(tile_k=64, out="bf16", epilogue="bias_silu")),
                                    (769, dict(tile_k=64)), (256, dict(tile_k=64, out="bf16"))])
def test_colsum_folded_in_epilogue(dg, M, desc):
    """Shapes large enough for the 256-row-block kernels, whose epilogue folds
    each 256-row run of the stored values (rows past M as -0) before the
    runs meet: a partial last run, bf16 output with bias and SiLU, a single
    run.  The sums against the oracle's tree over the GPU's C, and sampled C
    against the oracle."""
    N, K = 12288, 128
    A = inputs.spread_bf16(M + 5, (M, K))
    B = inputs.spread_bf16(N + 6, (K, N))
    bias = inputs.normal_bf16(7, (N,), 0.5)
    use_bias = desc.get("epilogue", "none") != "none"
    C, cs = run(dg, desc, A, B, bias if use_bias else None)
    assert_bits_equal(cs, oracle.colsum(C), "colsum %s M %d" % (desc, M))
    rng = np.random.default_rng(M)
    ii, jj = rng.integers(0, M, 200), rng.integers(0, N, 200)
    assert_bits_equal(C[ii, jj], oracle.gemm_at(desc, A, B, bias if use_bias else None, ii, jj), "sampled C")
