"""dg_gemm_noalloc against dg_gemm through the C ABI (GPU): the entry point
that allocates nothing puts split-K partials in the library's fixed
per-device scratch; its outputs must equal dg_gemm's bit for bit, call after
call, including a smaller call after a larger one (the scratch keeps the
earlier call's partials), and a request larger than the scratch is refused
before any launch."""
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


DESCS = [
    dict(mma="16x16x32", tile_k=64, split_k=4, split_combine="seq"),
    dict(mma="16x16x32", tile_k=64, split_k=8, split_combine="tree", partial="bf16", merge="bf16",
         out="bf16", epilogue="bias_silu"),
    dict(mma="16x16x32", tile_k=32, split_k=3, tile_combine="tree", split_combine="tree", fma=0),
    dict(mma="16x16x32", tile_k=64, split_k=4, split_layout="strided", split_tile=64, out="bf16"),
    dict(mma="scalar", tile_k=16, split_k=5, tile_combine="seq", split_combine="tree"),
]


def _pair(dg, desc, A, B, bias):
    """Both entry points on the same device operands; NaN-filled outputs."""
    import torch
    d = dg.Desc(**desc)
    M, N = A.shape[0], B.shape[1]
    dt = torch.bfloat16 if desc.get("out", "f32") == "bf16" else torch.float32
    Ad, Bd = dev_bf16(A), dev_bf16(B)
    bd = None if bias is None else dev_bf16(bias)
    C0 = torch.full((M, N), float("nan"), dtype=dt, device="cuda")
    C1 = torch.full((M, N), float("nan"), dtype=dt, device="cuda")
    dg.dg_gemm(d, Ad, Bd, bd, C0)
    dg.dg_gemm_noalloc(d, Ad, Bd, bd, C1)
    torch.cuda.synchronize()
    return host_bits(C0), host_bits(C1)


@pytest.mark.parametrize("i", range(len(DESCS)))
def test_noalloc_equals_dg_gemm_large_then_small(dg, i):
    desc = DESCS[i]
    shapes = [(100, 1000, 3000), (7, 520, 1000)]   # the second call smaller than the first
    for n, (M, N, K) in enumerate(shapes):
        print("noalloc case", i, desc, (M, N, K), flush=True)
        A = inputs.normal_bf16(300 + 10 * i + n, (M, K))
        B = inputs.normal_bf16(400 + 10 * i + n, (K, N), 0.02)
        bias = inputs.normal_bf16(500 + i, (N,), 0.02) if desc.get("epilogue", "none") != "none" else None
        ref, got = _pair(dg, desc, A, B, bias)
        assert_bits_equal(got, ref, "noalloc vs dg_gemm %s %s" % (desc, (M, N, K)))
        if n == 1:   # the small call also against the oracle
            assert_bits_equal(got, oracle.gemm(desc, A, B, bias), "noalloc vs oracle %s" % desc)


def test_noalloc_at_the_scratch_limit(dg):
    """S * M * N * 4 bytes equal to the scratch size runs (the decode shape's
    parts at M = 128); one more row is refused before any launch."""
    import torch
    desc = dict(mma="16x16x32", tile_k=64, split_k=8, out="bf16")
    M, N, K = 128, 4096, 2048
    assert 8 * M * N * 4 == dg.NOALLOC_SCRATCH_BYTES
    print("noalloc limit", (M, N, K), flush=True)
    A = inputs.normal_bf16(601, (M, K))
    B = inputs.normal_bf16(602, (K, N), 0.02)
    ref, got = _pair(dg, desc, A, B, None)
    assert_bits_equal(got, ref, "noalloc at the limit")
    d = dg.Desc(**desc)
    Ad, Bd = dev_bf16(inputs.normal_bf16(603, (M + 1, K))), dev_bf16(B)
    C = torch.empty((M + 1, N), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(dg.DgError) as e:
        dg.dg_gemm_noalloc(d, Ad, Bd, None, C)
    assert e.value.status == dg.DG_ERR_SCRATCH
    # the library still works after the refusal
    ref, got = _pair(dg, desc, A[:9], B, None)
    assert_bits_equal(got, ref, "noalloc after a refusal")


def test_noalloc_single_part_uses_no_scratch(dg):
    desc = dict(mma="16x16x32", tile_k=64, out="bf16", epilogue="bias_silu")
    A = inputs.normal_bf16(701, (300, 520))
    B = inputs.normal_bf16(702, (520, 264), 0.02)
    bias = inputs.normal_bf16(703, (264,), 0.02)
    ref, got = _pair(dg, desc, A, B, bias)
    assert_bits_equal(got, ref, "noalloc S = 1")
    assert np.array_equal(got, oracle.gemm(desc, A, B, bias))
