"""GPU parity of dg_gemm with binary16 operands (in_dtype = "f16") against
the CPU oracle, bit for bit (gfx950): the fp16 instruction folds its chunks
by the same rules as the bf16 one, with binary16 exponents."""
import numpy as np
import pytest

import oracle
from paper_2609_11356_amd import inputs
from tests.gpu_util import assert_bits_equal, dev_bf16, dev_f16, host_bits

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dg():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_11356_amd import dg as _dg
    _dg.lib()
    return _dg


def run(dg, desc, A, B, bias=None, knobs=None):
    import torch
    M, K = A.shape
    N = B.shape[1]
    d = dg.Desc(**desc)
    out_bf16 = desc.get("out", "f32") == "bf16"
    C = torch.full((M, N), float("nan"), dtype=torch.bfloat16 if out_bf16 else torch.float32, device="cuda")
    dg.dg_gemm(d, dev_f16(A), dev_f16(B), None if bias is None else dev_bf16(bias), C, knobs=knobs)
    torch.cuda.synchronize()
    return host_bits(C)


DESCS = [dict(tile_k=64), dict(tile_k=64, out="bf16", epilogue="bias_silu"),
         dict(tile_k=32, tile_combine="tree", fma=0), dict(tile_k=64, split_k=3, split_combine="tree"),
         dict(tile_k=96, tile_combine="seq", tail="first"), dict(mma="32x32x16", tile_k=48, fma=0)]
KNOBS = [None, dict(kernel=1), dict(kernel=3, tile_m=64, tile_n=128, occupancy=2, order=3),
         dict(kernel=3, tile_m=256, tile_n=128), dict(kernel=4, tile_m=16, tile_n=64, depth=4),
         dict(kernel=4, tile_m=64, tile_n=32, depth=2, slab_k=128), dict(kernel=5, tile_m=256, tile_n=256),
         dict(kernel=5, tile_m=128, tile_n=128), dict(kernel=6)]


@pytest.mark.parametrize("shape", [(1, 64, 512), (37, 200, 1000), (300, 520, 1032), (513, 264, 2048)])
@pytest.mark.parametrize("d", range(len(DESCS)))
def test_f16_descriptors_every_kernel(dg, shape, d):
    """Ragged shapes across the kernels that take binary16 operands; each
    knob that accepts the descriptor gives the oracle's bits."""
    M, N, K = shape
    desc = dict(DESCS[d], in_dtype="f16")
    A = inputs.spread_f16(M + d, (M, K), -8, 8)
    B = inputs.normal_f16(N + 2 * d, (K, N), 0.5)
    bias = inputs.normal_bf16(3, (N,), 0.5)
    use_bias = desc.get("epilogue", "none") != "none"
    want = oracle.gemm(desc, A, B, bias if use_bias else None)
    ran = 0
    for kn in KNOBS:
        try:
            got = run(dg, desc, A, B, bias if use_bias else None, knobs=kn)
        except dg.DgError as e:
            assert e.status == dg.DG_ERR_UNSUPPORTED, (kn, e)
            continue
        assert_bits_equal(got, want, "%s %s knobs %s" % (desc, shape, kn))
        ran += 1
    assert ran >= 2


def test_f16_scalar_path(dg):
    """Groups of one (the scalar path) with binary16 operands, chained chunks."""
    desc = dict(mma="scalar", tile_k=16, split_k=8, split_combine="tree", tile_combine="seq", in_dtype="f16")
    A = inputs.normal_f16(5, (3, 4096))
    B = inputs.normal_f16(6, (4096, 260), 0.1)
    assert_bits_equal(run(dg, desc, A, B), oracle.gemm(desc, A, B), "scalar f16")


def test_f16_wide_exponents_and_subnormals(dg):
    """Operands across the whole binary16 range, subnormals included, where
    the chunk grid and the window decide the bits."""
    rng = np.random.default_rng(12)
    M, N, K = 64, 128, 512
    A = (rng.choice([-1, 1], (M, K)) * (1 + rng.random((M, K))) * np.exp2(rng.integers(-24, 15, (M, K)))).astype(np.float16).view(np.uint16)
    B = (rng.choice([-1, 1], (K, N)) * (1 + rng.random((K, N))) * np.exp2(rng.integers(-24, 15, (K, N)))).astype(np.float16).view(np.uint16)
    for desc in (dict(tile_k=64, in_dtype="f16"), dict(tile_k=32, fma=0, tile_combine="tree", in_dtype="f16")):
        want = oracle.gemm(desc, A, B)
        for kn in (dict(kernel=1), dict(kernel=5, tile_m=128, tile_n=128), dict(kernel=4, tile_m=64, tile_n=32, depth=2, slab_k=128)):
            try:
                got = run(dg, desc, A, B, knobs=kn)
            except dg.DgError:
                continue
            assert_bits_equal(got, want, "wide f16 %s %s" % (desc, kn))


def test_f16_mlp_shape_sampled_and_batch_invariant(dg):
    """2048 x 14336 x 4096 with binary16 operands, bias and SiLU (the mixed
    256-row-block kernel): sampled outputs against the oracle, and row 0
    unchanged when the batch shrinks to 1, 37 and 512 rows."""
    desc = dict(tile_k=64, out="bf16", epilogue="bias_silu", in_dtype="f16")
    A = inputs.normal_f16(5, (2048, 4096))
    B = inputs.normal_f16(6, (4096, 14336), 0.02)
    bias = inputs.normal_bf16(7, (14336,), 0.02)
    C = run(dg, desc, A, B, bias)
    rng = np.random.default_rng(3)
    ii, jj = rng.integers(0, 2048, 300), rng.integers(0, 14336, 300)
    assert_bits_equal(C[ii, jj], oracle.gemm_at(desc, A, B, bias, ii, jj), "sampled f16 MLP")
    for m in (1, 37, 512):
        Cm = run(dg, desc, A[:m].copy(), B, bias)
        assert np.array_equal(Cm[0], C[0]), m


def test_f16_column_sums_and_strided_split(dg):
    """Binary16 operands through dg_gemm_colsum (the epilogue-folded runs on
    the 256-row-block kernel, fp32 out) and through a strided split on the
    few-row kernel."""
    import torch
    desc = dict(tile_k=64, in_dtype="f16")
    M, N, K = 1000, 12288, 128
    A = inputs.normal_f16(21, (M, K))
    B = inputs.normal_f16(22, (K, N), 0.5)
    d = dg.Desc(**desc)
    C = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    cs = torch.full((N,), float("nan"), dtype=torch.float32, device="cuda")
    dg.dg_gemm_colsum(d, dev_f16(A), dev_f16(B), None, C, cs)
    torch.cuda.synchronize()
    Ch = host_bits(C)
    assert_bits_equal(cs.cpu().numpy(), oracle.colsum(Ch), "f16 colsum")
    rng = np.random.default_rng(4)
    ii, jj = rng.integers(0, M, 200), rng.integers(0, N, 200)
    assert_bits_equal(Ch[ii, jj], oracle.gemm_at(desc, A, B, None, ii, jj), "f16 colsum C")
    sdesc = dict(tile_k=64, split_k=4, split_layout="strided", split_tile=64, split_combine="tree", in_dtype="f16")
    A = inputs.normal_f16(23, (7, 4096))
    B = inputs.normal_f16(24, (4096, 520), 0.1)
    assert_bits_equal(run(dg, sdesc, A, B), oracle.gemm(sdesc, A, B), "f16 strided split")
