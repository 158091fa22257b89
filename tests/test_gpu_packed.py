"""GPU parity of dg_gemm_packed (B in the packed form of dg_pack_b) through
the C ABI: the packed layout against its definition, every output against
the CPU oracle on ragged shapes under every descriptor the packed kernel
takes, and bit equality with dg_gemm on the row-major B at the few-row
shapes the bench times.  Inputs: seeded bf16 (or binary16) draws, normal or
exponent-spread."""
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


def packed_reference(B):
    """The packed form written out from its definition (layout only)."""
    K, N = B.shape
    KB, NP = -(-K // 32), -(-N // 16)
    Bz = np.zeros((KB * 32, NP * 16), np.uint16)
    Bz[:K, :N] = B
    out = np.zeros((NP, KB, 64, 8), np.uint16)
    for l in range(64):
        for e in range(8):
            out[:, :, l, e] = Bz[np.arange(KB)[None, :] * 32 + 8 * (l // 16) + e,
                                 np.arange(NP)[:, None] * 16 + l % 16]
    return out.reshape(-1)


def run_packed(dg, desc, A, B, bias=None, f16=False, knobs=None, offset_a=False):
    import torch
    dev = dev_f16 if f16 else dev_bf16
    dA = dev(A)
    if offset_a:
        # A at a 2-byte offset (its 16-byte runs unaligned)
        buf = dev(np.concatenate([np.zeros(1, np.uint16), A.reshape(-1)]))
        dA = buf[1:].view(A.shape)
    Bp = dg.dg_pack_b(dev(B))
    out_bf16 = desc.get("out", "f32") == "bf16"
    C = torch.full((A.shape[0], B.shape[1]), float("nan"), device="cuda",
                   dtype=torch.bfloat16 if out_bf16 else torch.float32)
    db = None if bias is None else dev_bf16(bias)
    dg.dg_gemm_packed(dg.Desc(**desc), dA, Bp, db, C, knobs=knobs)
    torch.cuda.synchronize()
    return host_bits(C)


@pytest.mark.parametrize("K,N", [(100, 37), (256, 16), (1000, 160), (31, 5)])
def test_pack_layout(dg, K, N):
    import torch
    B = inputs.normal_bf16(K + N, (K, N))
    Bp = dg.dg_pack_b(dev_bf16(B))
    torch.cuda.synchronize()
    got = Bp.data.cpu().numpy().view(np.uint16)[:dg.dg_packed_b_bytes(K, N) // 2]
    assert np.array_equal(got, packed_reference(B))


DESCS = [
    dict(tile_k=64),
    dict(tile_k=64, out="bf16"),
    dict(tile_k=64, out="bf16", epilogue="bias_silu"),
    dict(tile_k=64, out="bf16", epilogue="bias_silu", epi_round="pre_act"),
    dict(tile_k=64, epilogue="bias"),
    dict(tile_k=64, split_k=3),
    dict(tile_k=64, split_k=4, split_combine="tree", out="bf16"),
    dict(tile_k=64, split_k=2, k_cuts=[96]),
    dict(tile_k=64, split_k=3, partial="bf16", merge="bf16", out="bf16"),
    dict(tile_k=64, split_k=4, split_layout="strided", split_tile=64),
    dict(tile_k=32, split_k=4, split_layout="strided", split_tile=32, out="bf16"),
    dict(tile_k=64, split_k=2, split_layout="strided", split_tile=128, split_combine="tree"),
    dict(tile_k=64, split_k=8, split_layout="strided", split_tile=64, split_combine="tree"),
]
SHAPES = [(1, 37, 1000), (7, 160, 256), (16, 64, 1000), (33, 50, 512), (64, 21, 320), (5, 16, 100)]


@pytest.mark.parametrize("di", range(len(DESCS)))
def test_packed_matches_oracle_ragged(dg, di):
    desc = DESCS[di]
    for (M, N, K) in SHAPES:
        if desc.get("split_k", 1) > 1 and desc.get("split_layout") != "strided" and "k_cuts" not in desc:
            span = -(-(-(-K // desc["split_k"])) // desc["tile_k"]) * desc["tile_k"]
            if (desc["split_k"] - 1) * span >= K:
                continue               # the span rule would leave a part empty
        if "k_cuts" in desc and desc["k_cuts"][-1] >= K:
            continue
        for spread in (False, True):
            seed = 100 * di + M + N + K + spread
            A = inputs.spread_bf16(seed, (M, K)) if spread else inputs.normal_bf16(seed, (M, K))
            B = inputs.spread_bf16(seed + 1, (K, N)) if spread else inputs.normal_bf16(seed + 1, (K, N))
            bias = inputs.normal_bf16(seed + 2, (N,)) if desc.get("epilogue", "none") != "none" else None
            print("packed", desc, (M, N, K), "spread" if spread else "normal", flush=True)
            want = oracle.gemm(desc, A, B, bias)
            assert_bits_equal(run_packed(dg, desc, A, B, bias), want, "%s %s" % (desc, (M, N, K)))


@pytest.mark.parametrize("offset_a", [False, True])
def test_unaligned_a_rows(dg, offset_a):
    """K % 8 != 0 (A's rows are not 16-byte runs) and A itself at a 2-byte
    offset: the element-load path."""
    for (M, N, K) in [(3, 40, 203), (20, 48, 77), (64, 16, 1001)]:
        A, B = inputs.normal_bf16(M + K, (M, K)), inputs.normal_bf16(N + K, (K, N))
        desc = dict(tile_k=64, out="bf16")
        print("packed unaligned", (M, N, K), offset_a, flush=True)
        assert_bits_equal(run_packed(dg, desc, A, B, offset_a=offset_a), oracle.gemm(desc, A, B), str((M, N, K)))


def test_binary16_operands(dg):
    for (M, N, K) in [(1, 37, 1000), (16, 64, 256), (40, 48, 512)]:
        A, B = inputs.spread_f16(M + K, (M, K), -8, 8), inputs.normal_f16(N + K, (K, N), 0.5)
        desc = dict(tile_k=64, in_dtype="f16", out="bf16")
        print("packed f16", (M, N, K), flush=True)
        assert_bits_equal(run_packed(dg, desc, A, B, f16=True), oracle.gemm(desc, A, B), str((M, N, K)))


@pytest.mark.parametrize("knobs", [dict(kernel=11, depth=8), dict(kernel=11, depth=32), dict(kernel=11, tile_m=64),
                                   dict(kernel=11, tile_m=32, depth=8)])
def test_knobs_do_not_change_bits(dg, knobs):
    M, N, K = 7, 80, 1000
    A, B = inputs.spread_bf16(5, (M, K)), inputs.spread_bf16(6, (K, N))
    desc = dict(tile_k=64, out="bf16")
    assert_bits_equal(run_packed(dg, desc, A, B, knobs=knobs), oracle.gemm(desc, A, B), str(knobs))


@pytest.mark.parametrize("case", ["M1", "M7", "M32", "M64", "decode_seq", "decode_tree", "strided_M1", "strided_dec"])
def test_equals_row_major_at_bench_shapes(dg, case):
    """Every output equal to dg_gemm on the row-major B at the few-row bench
    shapes (4096 x 4096 weight; the 8 x 4096 x 14336 decode), and sampled
    outputs equal to the oracle's."""
    import torch
    if case.startswith("M"):
        M, N, K = int(case[1:]), 4096, 4096
        desc = dict(tile_k=64, out="bf16")
    elif case.startswith("decode"):
        M, N, K = 8, 4096, 14336
        desc = dict(tile_k=64, split_k=8, split_combine=case.split("_")[1], out="bf16")
    elif case == "strided_M1":
        M, N, K = 1, 4096, 4096
        desc = dict(tile_k=64, split_k=4, split_layout="strided", split_tile=64, out="bf16")
    else:
        M, N, K = 8, 4096, 14336
        desc = dict(tile_k=64, split_k=4, split_layout="strided", split_tile=128, out="bf16")
    A, B = inputs.spread_bf16(11, (M, K)), inputs.spread_bf16(12, (K, N))
    print("packed vs row-major", case, flush=True)
    got = run_packed(dg, desc, A, B)
    C = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    dg.dg_gemm(dg.Desc(**desc), dev_bf16(A), dev_bf16(B), None, C)
    torch.cuda.synchronize()
    assert np.array_equal(got, host_bits(C))
    rng = np.random.default_rng(1)
    ii, jj = rng.integers(0, M, 256), rng.integers(0, N, 256)
    want = inputs.f32_to_bf16_bits(oracle.gemm_at(desc, A, B, None, ii, jj))
    assert_bits_equal(got[ii, jj], want, case)
