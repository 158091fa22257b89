"""GPU parity of dg_gemm against the CPU oracle, bit for bit (gfx950).

Every case runs through the C ABI (paper_2609_11356_amd.dg) on seeded
synthetic inputs from paper_2609_11356_amd.inputs, and compares every output
(or, at full LLM sizes, a sample the oracle computes one by one) with the
oracle under the gfx950 MFMA model.  The bar is bit equality: the descriptor
fixes one correct byte pattern per output.
"""
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


def run(dg, desc, A, B, bias=None, knobs=None):
    import torch
    M, K = A.shape
    N = B.shape[1]
    d = dg.Desc(**desc)
    out_bf16 = desc.get("out", "f32") == "bf16"
    C = torch.empty((M, N), dtype=torch.bfloat16 if out_bf16 else torch.float32, device="cuda")
    C.fill_(float("nan"))
    dg.dg_gemm(d, dev_bf16(A), dev_bf16(B), None if bias is None else dev_bf16(bias), C, knobs=knobs)
    torch.cuda.synchronize()
    return host_bits(C)


def check_full(dg, desc, A, B, bias=None, knobs=None, what=""):
    got = run(dg, desc, A, B, bias, knobs)
    want = oracle.gemm(desc, A, B, bias)
    assert_bits_equal(got, want, what or str(desc))
    return got


TINY = dict(mma="16x16x32", tile_k=32, split_k=2, tile_combine="tree", split_combine="tree", fma=1)


@pytest.mark.parametrize("seed", range(10))
def test_tiny_config(dg, seed):
    """A 16x256, B 256x64, split 2 at k = 128, tiles of 32 combined by the
    balanced tree, parts by the balanced tree, fp32 out: ten normal draws and
    ten exponent-spread draws."""
    A, B = inputs.tiny(seed)
    check_full(dg, TINY, A, B, what="tiny normal seed %d" % seed)
    As, Bs = inputs.tiny(seed, spread=True)
    check_full(dg, TINY, As, Bs, what="tiny spread seed %d" % seed)


DESCS = [
    dict(mma="16x16x32", tile_k=64),
    dict(mma="32x32x16", tile_k=64),
    dict(mma="16x16x32", tile_k=64, fma=0),
    dict(mma="32x32x16", tile_k=32, fma=0, tile_combine="seq"),
    dict(mma="16x16x32", tile_k=32, tile_combine="tree"),
    dict(mma="16x16x32", tile_k=64, split_k=3),
    dict(mma="16x16x32", tile_k=64, split_k=4, split_combine="tree"),
    dict(mma="16x16x32", tile_k=64, split_k=4, split_combine="tree", partial="bf16", merge="bf16"),
    dict(mma="16x16x32", tile_k=64, split_k=3, partial="bf16"),
    dict(mma="16x16x32", tile_k=64, split_k=3, k_cuts=[100, 333]),
    dict(mma="16x16x32", tile_k=64, split_k=2, tail="first", tile_combine="tree"),
    dict(mma="16x16x32", tile_k=64, tail="first"),
    dict(mma="16x16x32", tile_k=64, out="bf16"),
    dict(mma="16x16x32", tile_k=64, out="bf16", epilogue="bias"),
    dict(mma="16x16x32", tile_k=64, out="bf16", epilogue="bias_silu"),
    dict(mma="16x16x32", tile_k=64, out="bf16", epilogue="bias_silu", epi_round="pre_act"),
    dict(mma="16x16x32", tile_k=64, split_k=4, out="bf16", epilogue="bias_silu"),
    # the scalar path: chained chunks (groups of one, FMA chains)
    dict(mma="scalar", tile_k=64),
    dict(mma="scalar", tile_k=16, split_k=4, tile_combine="seq", split_combine="tree"),
    dict(mma="scalar", tile_k=5, split_k=3, tile_combine="tree", tail="first"),
    dict(mma="scalar", tile_k=8, split_k=2, tile_combine="tree", out="bf16", epilogue="bias_silu"),
    dict(mma="scalar", tile_k=1, out="bf16", epilogue="bias"),
]


@pytest.mark.parametrize("shape", [(33, 72, 456), (5, 40, 203), (64, 128, 512), (1, 8, 8), (17, 16, 1)])
@pytest.mark.parametrize("di", range(len(DESCS)))
def test_descriptor_matrix_ragged(dg, di, shape):
    """Every descriptor field on ragged shapes (partial tiles, M and N not
    multiples of the block, K not a multiple of 8 or of the tile), normal and
    exponent-spread operands."""
    desc = DESCS[di]
    M, N, K = shape
    rng_seed = 100 * di + M
    A = inputs.normal_bf16(rng_seed, (M, K))
    B = inputs.normal_bf16(rng_seed + 1, (K, N), 0.05)
    bias = inputs.normal_bf16(rng_seed + 2, (N,), 0.5)
    S = desc.get("split_k", 1)
    span = -(-K // S)
    span = -(-span // desc["tile_k"]) * desc["tile_k"]
    cuts_outside = bool(desc.get("k_cuts")) and not desc["k_cuts"][-1] < K
    empty_part = S > 1 and not desc.get("k_cuts") and (S - 1) * span >= K
    if cuts_outside or empty_part:
        # a plan the descriptor cannot make for this K: both sides refuse it
        with pytest.raises(dg.DgError) as e:
            run(dg, desc, A, B, bias)
        assert e.value.status == dg.DG_ERR_SHAPE
        with pytest.raises(oracle.OracleError):
            oracle.gemm(desc, A, B, bias)
        return
    check_full(dg, desc, A, B, bias, what="%s %s normal" % (desc, shape))
    As = inputs.spread_bf16(rng_seed + 3, (M, K))
    Bs = inputs.spread_bf16(rng_seed + 4, (K, N))
    check_full(dg, desc, As, Bs, bias, what="%s %s spread" % (desc, shape))


@pytest.mark.parametrize("K,S", [(1, 1), (7, 1), (576, 3), (8648, 9), (8648, 1), (100000, 1)])
def test_all_ones_count(dg, K, S):
    """Every output of an all-ones product is exactly K (App. D's count)."""
    M, N = 3, 24
    ones = np.uint16(0x3F80)
    got = run(dg, dict(tile_k=64, split_k=S), np.full((M, K), ones), np.full((K, N), ones))
    assert np.all(got == K), np.unique(got)


@pytest.mark.parametrize("desc", [dict(tile_k=64, split_k=64, split_combine="tree"),
                                  dict(tile_k=32, split_k=64, split_combine="seq", partial="bf16", merge="bf16",
                                       out="bf16"),
                                  dict(tile_k=64, split_k=64, split_layout="strided", split_tile=64,
                                       split_combine="tree")])
def test_maximum_split(dg, desc):
    """The largest split a descriptor holds (64 parts, DG_MAX_SPLIT) on the
    MFMA path, row-major and packed B, against the oracle on every output."""
    import torch
    M, N, K = 5, 40, 4088       # 64 parts of 64 k under the span rule, the last one 56
    A, B = inputs.spread_bf16(51, (M, K)), inputs.spread_bf16(52, (K, N))
    want = oracle.gemm(desc, A, B)
    print("maximum split", desc, flush=True)
    assert_bits_equal(run(dg, desc, A, B), want, "row-major %s" % desc)
    if desc.get("split_layout") == "strided" or desc["tile_k"] % 32 == 0:
        out_bf16 = desc.get("out") == "bf16"
        C = torch.full((M, N), float("nan"), dtype=torch.bfloat16 if out_bf16 else torch.float32, device="cuda")
        dg.dg_gemm_packed(dg.Desc(**desc), dev_bf16(A), dg.dg_pack_b(dev_bf16(B)), None, C)
        torch.cuda.synchronize()
        assert_bits_equal(host_bits(C), want, "packed %s" % desc)


def test_k_zero_gives_epilogue_of_zero(dg):
    import torch
    bias = inputs.normal_bf16(1, (16,), 1.0)
    d = dg.Desc(epilogue="bias_silu", out="bf16")
    C = torch.empty((4, 16), dtype=torch.bfloat16, device="cuda")
    A = torch.empty((4, 0), dtype=torch.bfloat16, device="cuda")
    B = torch.empty((0, 16), dtype=torch.bfloat16, device="cuda")
    dg.dg_gemm(d, A, B, dev_bf16(bias), C)
    torch.cuda.synchronize()
    want = oracle.gemm(dict(epilogue="bias_silu", out="bf16"), np.zeros((4, 0), np.uint16),
                       np.zeros((0, 16), np.uint16), bias)
    assert_bits_equal(host_bits(C), want)


KNOBS = [dict(kernel=1), dict(kernel=2, tile_m=16, tile_n=64), dict(kernel=2, tile_m=16, tile_n=128),
         dict(kernel=2, tile_m=32, tile_n=128), dict(kernel=2, tile_m=64, tile_n=128),
         dict(kernel=2, tile_m=128, tile_n=128), dict(kernel=2, tile_m=256, tile_n=256),
         dict(kernel=2, tile_m=256, tile_n=128), dict(kernel=2, tile_m=128, tile_n=256),
         dict(kernel=3, tile_m=256, tile_n=128),
         dict(kernel=3, tile_m=128, tile_n=256), dict(kernel=3, tile_m=128, tile_n=128),
         dict(kernel=3, tile_m=64, tile_n=128), dict(kernel=3, tile_m=32, tile_n=256),
         dict(kernel=3, tile_m=32, tile_n=128), dict(kernel=3, tile_m=128, tile_n=128, occupancy=2, order=2),
         dict(kernel=3, tile_m=64, tile_n=128, occupancy=2, order=3), dict(kernel=3, tile_m=256, tile_n=128, order=3),
         dict(kernel=4, tile_m=16, tile_n=16, depth=4), dict(kernel=4, tile_m=32, tile_n=32, depth=8),
         dict(kernel=4, tile_m=64, tile_n=64, depth=4), dict(kernel=4, tile_m=16, tile_n=64, depth=8),
         dict(kernel=4, tile_m=16, tile_n=32, depth=4, slab_k=256), dict(kernel=4, tile_m=32, tile_n=64, depth=2, slab_k=256),
         dict(kernel=4, tile_m=64, tile_n=32, depth=4, slab_k=128),
         dict(kernel=5, tile_m=256, tile_n=128, order=1), dict(kernel=5, tile_m=256, tile_n=256),
         dict(kernel=5, tile_m=128, tile_n=128, order=2),
         dict(kernel=5, tile_m=128, tile_n=256, order=2),
         dict(kernel=6), dict(kernel=6, split_n=256), dict(kernel=6, split_n=512, order=3),
         dict(kernel=7), dict(kernel=7, split_n=256), dict(kernel=7, split_n=512, order=3),
         dict(kernel=10), dict(kernel=10, split_n=256), dict(kernel=10, split_n=512, order=3), dict(kernel=14),
         dict(kernel=8), dict(kernel=8, tile_m=16, tile_n=32, depth=6, slab_k=256),
         dict(kernel=8, tile_m=32, tile_n=32, depth=4, slab_k=128), dict(kernel=8, tile_m=64, tile_n=32, depth=3, slab_k=128),
         dict(kernel=8, tile_m=16, tile_n=64, depth=6, slab_k=128), None]


def test_scalar_path_strided_and_many_chunks(dg):
    """Chained chunks with many parts (the GEMV shape), strided dealing, and
    more rows than one thread carries."""
    for desc, shape in ((dict(mma="scalar", tile_k=16, split_k=64, tile_combine="seq", split_combine="tree"),
                         (1, 300, 4096)),
                        (dict(mma="scalar", tile_k=16, split_k=4, split_layout="strided", split_tile=32,
                              split_combine="tree"), (9, 72, 1000)),
                        (dict(mma="scalar", tile_k=32, split_k=8, out="bf16"), (8, 4096, 2048))):
        M, N, K = shape
        A = inputs.spread_bf16(M + 7, (M, K))
        B = inputs.spread_bf16(N + 8, (K, N))
        check_full(dg, desc, A, B, what="%s %s" % (desc, shape))


@pytest.mark.parametrize("desc", [dict(tile_k=64, out="bf16"), dict(tile_k=64, split_k=4, split_combine="tree"),
                                  dict(tile_k=64, out="bf16", epilogue="bias_silu")])
def test_speed_knobs_do_not_change_bits(dg, desc):
    """Kernel choice and block shape are speed knobs: identical bytes."""
    M, N, K = 300, 520, 1032
    A = inputs.spread_bf16(7, (M, K))
    B = inputs.spread_bf16(8, (K, N))
    bias = inputs.normal_bf16(9, (N,), 0.5)
    outs = [run(dg, desc, A, B, bias, knobs=k) for k in KNOBS]
    for o, k in zip(outs[1:], KNOBS[1:]):
        assert_bits_equal(o, outs[0], "knobs %s" % k)
    assert_bits_equal(outs[0], oracle.gemm(desc, A, B, bias))


def test_misaligned_operands_take_the_general_path(dg):
    """Operands offset by one element (2-byte aligned only) give the same bits."""
    import torch
    M, N, K = 20, 48, 256
    A = inputs.spread_bf16(11, (M, K))
    B = inputs.spread_bf16(12, (K, N))
    want = oracle.gemm(dict(tile_k=64), A, B)
    Ab = dev_bf16(np.concatenate([[0], A.reshape(-1)]))[1:]
    Bb = dev_bf16(np.concatenate([[0], B.reshape(-1)]))[1:]
    C = torch.empty((M, N), dtype=torch.float32, device="cuda")
    d = dg.Desc(tile_k=64)
    dg.dg_gemm(d, Ab.data_ptr(), Bb.data_ptr(), None, C.data_ptr(), M, N, K)
    torch.cuda.synchronize()
    assert_bits_equal(C.cpu().numpy(), want)


def test_silu_epilogue_exhaustive_over_bf16(dg):
    """The device exp/SiLU equals the oracle's on every bf16 input: with
    A = B = 0 the pre-activation is exactly the bias, so a 1 x 65536 GEMM
    whose bias holds every bf16 pattern evaluates SiLU at all of them."""
    N = 1 << 16
    bias = np.arange(N, dtype=np.uint32).astype(np.uint16)
    A = np.zeros((1, 8), np.uint16)
    B = np.zeros((8, N), np.uint16)
    for out in ("f32", "bf16"):
        desc = dict(tile_k=64, epilogue="bias_silu", out=out)
        got = run(dg, desc, A, B, bias)
        # z = (+0) (+) bias: the -0 bias gives +0
        assert_bits_equal(got[0], oracle.gemm(desc, A, B, bias)[0], "silu exhaustive " + out)


def test_silu_epilogue_random_fp32(dg):
    """SiLU at pre-activations with 16 significant bits (products of two bf16
    values plus a bf16 bias), over a wide exponent range."""
    M, N, K = 64, 1024, 8
    A = inputs.spread_bf16(21, (M, K), -20, 5)
    B = np.zeros((K, N), np.uint16)
    B[0] = inputs.spread_bf16(22, (N,), -8, 3)
    bias = inputs.normal_bf16(23, (N,), 2.0)
    desc = dict(tile_k=64, epilogue="bias_silu", out="f32")
    check_full(dg, desc, A, B, bias, what="silu random")


# ------------------------------------------------------ LLM-shaped configs


def test_batch_invariance_sweep(dg):
    """B 4096x4096 ~ N(0, 0.02); A = the first M rows of one 4096x4096 N(0,1)
    draw; one descriptor (tile_k 64, no split, bf16 out).  Row r is
    byte-identical for every M > r, the M = 7 product matches the oracle in
    full, and sampled outputs of the larger ones match it too."""
    import torch
    B = inputs.sweep_weight(2)
    Afull = inputs.sweep_activations(1, rows=4096)
    desc = dict(mma="16x16x32", tile_k=64, out="bf16")
    d = dg.Desc(**desc)
    Bd = dev_bf16(B)
    Ad = dev_bf16(Afull)
    outs = {}
    for M in inputs.SWEEP_M:
        C = torch.empty((M, 4096), dtype=torch.bfloat16, device="cuda")
        dg.dg_gemm(d, Ad[:M].contiguous(), Bd, None, C)
        torch.cuda.synchronize()
        outs[M] = host_bits(C)
    for M in inputs.SWEEP_M:
        for M2 in inputs.SWEEP_M:
            if M2 > M:
                assert np.array_equal(outs[M], outs[M2][:M]), (M, M2)
    assert_bits_equal(outs[7], oracle.gemm(desc, Afull[:7], B), "sweep M=7 full")
    rng = np.random.default_rng(5)
    ii = rng.integers(0, 4096, 3000)
    jj = rng.integers(0, 4096, 3000)
    want = oracle.gemm_at(desc, Afull, B, None, ii, jj)
    assert_bits_equal(outs[4096][ii, jj], inputs.f32_to_bf16_bits(want), "sweep M=4096 sampled")


@pytest.mark.parametrize("combine", ["seq", "tree"])
@pytest.mark.parametrize("out", ["bf16", "f32"])
def test_splitk_decode(dg, combine, out):
    """A 8x14336, B 14336x4096 ~ N(0, 0.02), split 8 at equal cuts, fp32
    partials in the workspace, merged by the chain or the balanced tree."""
    A, B = inputs.decode()
    desc = dict(mma="16x16x32", tile_k=64, split_k=8, split_combine=combine, out=out)
    got = run(dg, desc, A, B)
    # every one of the 32768 outputs
    assert_bits_equal(got, oracle.gemm(desc, A, B), "decode %s %s" % (combine, out))


def test_splitk_decode_spread(dg):
    """The decode shape on exponent-spread operands (where a regrouping of
    the parts or of the chunks flips output bits), every output."""
    A = inputs.spread_bf16(31, (8, 14336))
    B = inputs.spread_bf16(32, (14336, 4096))
    for combine in ("seq", "tree"):
        desc = dict(mma="16x16x32", tile_k=64, split_k=8, split_combine=combine, out="bf16")
        assert_bits_equal(run(dg, desc, A, B), oracle.gemm(desc, A, B), "decode spread %s" % combine)


@pytest.mark.parametrize("epi_round", ["final", "pre_act"])
def test_fused_mlp(dg, epi_round):
    """C = SiLU(A.B + bias) for A 2048x4096, B 4096x14336 ~ N(0, 0.02), bias
    14336 ~ N(0, 0.02), bf16 out, rounding point from the descriptor."""
    A, B, bias = inputs.mlp()
    desc = dict(mma="16x16x32", tile_k=64, out="bf16", epilogue="bias_silu", epi_round=epi_round)
    got = run(dg, desc, A, B, bias)
    rng = np.random.default_rng(7)
    ii = rng.integers(0, 2048, 2500)
    jj = rng.integers(0, 14336, 2500)
    want = inputs.f32_to_bf16_bits(oracle.gemm_at(desc, A, B, bias, ii, jj))
    assert_bits_equal(got[ii, jj], want, "mlp %s" % epi_round)
    # and the full first rows
    want_rows = oracle.gemm(desc, A[:2], B, bias)
    assert_bits_equal(got[:2], want_rows, "mlp rows 0-1")


def test_full_size_spread_draws(dg):
    """One exponent-spread draw at the fused-MLP shape and at the sweep's
    M = 4096 shape, compared with the oracle on sampled outputs and whole
    rows (narrow exponents can hide a regrouping; spread ones do not)."""
    rng = np.random.default_rng(8)
    A = inputs.spread_bf16(51, (2048, 4096))
    B = inputs.spread_bf16(52, (4096, 14336))
    bias = inputs.spread_bf16(53, (14336,))
    desc = dict(mma="16x16x32", tile_k=64, out="bf16", epilogue="bias_silu")
    got = run(dg, desc, A, B, bias)
    ii = rng.integers(0, 2048, 2500)
    jj = rng.integers(0, 14336, 2500)
    want = inputs.f32_to_bf16_bits(oracle.gemm_at(desc, A, B, bias, ii, jj))
    assert_bits_equal(got[ii, jj], want, "mlp spread sampled")
    assert_bits_equal(got[[0, 1337, 2047]], oracle.gemm(desc, A[[0, 1337, 2047]], B, bias), "mlp spread rows")
    A = inputs.spread_bf16(54, (4096, 4096))
    B = inputs.spread_bf16(55, (4096, 4096))
    desc = dict(mma="16x16x32", tile_k=64, out="bf16")
    got = run(dg, desc, A, B)
    ii = rng.integers(0, 4096, 3000)
    jj = rng.integers(0, 4096, 3000)
    want = inputs.f32_to_bf16_bits(oracle.gemm_at(desc, A, B, None, ii, jj))
    assert_bits_equal(got[ii, jj], want, "sweep M=4096 spread sampled")
    assert_bits_equal(got[[5, 4095]], oracle.gemm(desc, A[[5, 4095]], B), "sweep M=4096 spread rows")


def test_error_bound_vs_fp64(dg):
    """|C - C_fp64| <= 2^-8 * sum_k |a_ik b_kj| at an LLM shape."""
    A = inputs.sweep_activations(1, rows=64)
    B = inputs.sweep_weight(2)
    got = run(dg, dict(tile_k=64, out="bf16"), A, B)
    Af = inputs.bf16_bits_to_f32(A).astype(np.float64)
    Bf = inputs.bf16_bits_to_f32(B).astype(np.float64)
    ref = Af @ Bf
    mag = np.abs(Af) @ np.abs(Bf)
    err = np.abs(inputs.bf16_bits_to_f32(got).astype(np.float64) - ref)
    assert np.all(err <= 2.0 ** -8 * mag)


# ------------------------------------------------ strided layout of the split

STRIDED = [dict(tile_k=64, split_k=4, split_layout="strided", split_tile=64, out="bf16"),
           dict(tile_k=64, split_k=4, split_layout="strided", split_tile=128),
           dict(tile_k=32, split_k=2, split_layout="strided", split_tile=64, split_combine="tree"),
           dict(tile_k=64, split_k=8, split_layout="strided", split_tile=256, partial="bf16", merge="bf16"),
           dict(tile_k=32, split_k=3, split_layout="strided", split_tile=32, tile_combine="tree",
                fma=0, out="bf16"),
           dict(tile_k=64, split_k=4, split_layout="strided", split_tile=64, out="bf16",
                epilogue="bias_silu")]


@pytest.mark.parametrize("desc", STRIDED)
@pytest.mark.parametrize("shape", [(33, 72, 1032), (5, 40, 100), (70, 136, 4160)])
def test_strided_split_matches_oracle(dg, desc, shape):
    """Parts dealt every S-th tile (the cut's strided layout): identical
    bytes to the oracle on the default path and on the generic kernel,
    including ragged K and parts left empty (K = 100 < S w)."""
    M, N, K = shape
    A = inputs.spread_bf16(41, (M, K))
    B = inputs.spread_bf16(42, (K, N))
    bias = inputs.normal_bf16(43, (N,), 0.5)
    want = oracle.gemm(desc, A, B, bias)
    assert_bits_equal(run(dg, desc, A, B, bias), want, "default path")
    assert_bits_equal(run(dg, desc, A, B, bias, knobs=dict(kernel=1)), want, "generic kernel")
