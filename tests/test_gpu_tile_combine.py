"""GPU parity of the tiled kernel for the descriptors whose accumulator is not
one carried chain (Sec. 3.2.2): the tile chain (seq) and the balanced tile
tree, and fma = 0 (each 32-k instruction from zero, its result added to the
tile's accumulator).  Every output against the CPU oracle bit for bit, through
the C ABI, on shapes the tiled path takes (K and N multiples of 8, several
128 x 64 blocks, ragged M and N edges, tree parts of 2 to 128 tiles: every
stack depth and both sides of each power of two), normal and
exponent-spread draws; the kernel knob 12
against the generic kernel 1; the M = 1024 bench descriptors on sampled
outputs at 1024 x 4096 x 4096."""
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


def run(dg, desc, A, B, bias=None, knobs=None, f16=False):
    import torch
    M, K = A.shape
    N = B.shape[1]
    out_bf16 = desc.get("out", "f32") == "bf16"
    C = torch.full((M, N), float("nan"), dtype=torch.bfloat16 if out_bf16 else torch.float32, device="cuda")
    dev = dev_f16 if f16 else dev_bf16
    dg.dg_gemm(dg.Desc(**desc), dev(A), dev(B), None if bias is None else dev_bf16(bias), C, knobs=knobs)
    torch.cuda.synchronize()
    return host_bits(C)


def parts(desc, K):
    """The parts' lengths under the span rule (contiguous split, no explicit cuts)."""
    S = desc.get("split_k", 1)
    if S == 1:
        return [K]
    span = -(-(-(-K // S)) // desc["tile_k"]) * desc["tile_k"]
    cuts = [min(s * span, K) for s in range(S)] + [K]
    return [cuts[s + 1] - cuts[s] for s in range(S)]


def takes_tiled_path(desc, K, N):
    """Whether the library runs desc on the tile-combine kernel (the rule the
    host applies: 8-aligned K and N, tile boundaries on 32-k steps, at most
    128 tiles per part for the tree)."""
    tk = desc["tile_k"]
    if K % 8 or N % 8 or tk % 32 or (desc.get("fma", 1) == 0 and desc.get("mma", "16x16x32") != "16x16x32"):
        return False
    for ln in parts(desc, K):
        if desc.get("tail") == "first" and (ln % tk) % 32:
            return False
        if desc.get("tile_combine") == "tree" and -(-ln // tk) > 128:
            return False
    return True


DESCS = [
    dict(tile_k=64, tile_combine="tree"),
    dict(tile_k=32, tile_combine="tree"),
    dict(tile_k=128, tile_combine="seq"),
    dict(tile_k=64, fma=0),
    dict(tile_k=96, fma=0, tile_combine="seq"),
    dict(tile_k=64, fma=0, tile_combine="tree", out="bf16", epilogue="bias_silu"),
    dict(tile_k=64, tile_combine="tree", split_k=3),
    dict(tile_k=64, tile_combine="tree", split_k=2, tail="first"),
    dict(tile_k=32, tile_combine="seq", split_k=2, tail="first", out="bf16"),
    dict(tile_k=256, tile_combine="tree", split_k=2, partial="bf16", merge="bf16", out="bf16"),
    dict(mma="32x32x16", tile_k=64, tile_combine="tree"),
    dict(tile_k=64, tile_combine="tree", out="bf16", epilogue="bias"),
]
SHAPES = [(130, 200, 1000), (7, 264, 512), (64, 72, 96), (129, 136, 224), (40, 80, 1088), (9, 16, 320)]


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("di", range(len(DESCS)))
def test_matches_oracle(dg, di, shape):
    desc = DESCS[di]
    M, N, K = shape
    if any(ln == 0 for ln in parts(desc, K)):
        # the span rule leaves a part empty: the oracle and the library both refuse
        A, B = inputs.normal_bf16(7, (M, K)), inputs.normal_bf16(8, (K, N))
        bias = inputs.normal_bf16(9, (N,)) if desc.get("epilogue", "none") != "none" else None
        with pytest.raises(oracle.OracleError, match="status 3"):
            oracle.gemm(desc, A, B, bias)
        with pytest.raises(dg.DgError) as ei:
            run(dg, desc, A, B, bias)
        assert ei.value.status == dg.DG_ERR_SHAPE
        return
    seed = 1000 + 37 * di + M + K
    bias = inputs.normal_bf16(seed + 2, (N,), 0.5) if desc.get("epilogue", "none") != "none" else None
    tiled = takes_tiled_path(desc, K, N)
    for spread in (False, True):
        A = inputs.spread_bf16(seed, (M, K)) if spread else inputs.normal_bf16(seed, (M, K))
        B = inputs.spread_bf16(seed + 1, (K, N)) if spread else inputs.normal_bf16(seed + 1, (K, N), 0.05)
        print("tile combine", desc, shape, "spread" if spread else "normal", "tiled" if tiled else "generic",
              flush=True)
        want = oracle.gemm(desc, A, B, bias)
        assert_bits_equal(run(dg, desc, A, B, bias), want, "%s %s" % (desc, shape))
        if tiled:
            assert_bits_equal(run(dg, desc, A, B, bias, knobs=dict(kernel=12)), want, "kernel 12 %s" % desc)


def test_refusals(dg):
    """Kernel 12 refuses what it cannot order: a tree of more than 128 tiles
    per part, tile boundaries off the 32-k grid, a misaligned N, and the
    descriptors with one carried chain (fma = 1, carry)."""
    A = inputs.normal_bf16(1, (16, 4160))
    for desc, shape in [(dict(tile_k=32, tile_combine="tree"), (16, 64, 4160)),      # 130 tiles
                        (dict(tile_k=64, tile_combine="tree", tail="first"), (16, 64, 1000)),   # 1000 % 64 = 40
                        (dict(tile_k=64, tile_combine="seq"), (16, 60, 512)),         # N % 8
                        (dict(tile_k=64), (16, 64, 512))]:
        M, N, K = shape
        with pytest.raises(dg.DgError) as e:
            run(dg, desc, A[:M, :K], inputs.normal_bf16(3, (K, N)), knobs=dict(kernel=12))
        assert e.value.status == dg.DG_ERR_UNSUPPORTED, desc


@pytest.mark.parametrize("K", [2048, 2080, 4096])
def test_deep_trees(dg, K):
    """Tree parts of 64, 65 and 128 tiles (stacks of six and seven levels)."""
    desc = dict(tile_k=32, tile_combine="tree")
    M, N = 40, 72
    A, B = inputs.spread_bf16(41 + K, (M, K)), inputs.spread_bf16(42 + K, (K, N))
    print("deep tree", K, flush=True)
    want = oracle.gemm(desc, A, B)
    assert_bits_equal(run(dg, desc, A, B, knobs=dict(kernel=12)), want, "tree K=%d" % K)


@pytest.mark.parametrize("desc", [dict(tile_k=64, tile_combine="tree"), dict(tile_k=128, tile_combine="seq", split_k=2),
                                  dict(tile_k=64, fma=0, out="bf16")])
def test_kernel_12_equals_generic(dg, desc):
    M, N, K = 200, 264, 1024
    A, B = inputs.spread_bf16(21, (M, K)), inputs.spread_bf16(22, (K, N))
    print("kernel 12 vs 1", desc, flush=True)
    assert np.array_equal(run(dg, desc, A, B, knobs=dict(kernel=12)), run(dg, desc, A, B, knobs=dict(kernel=1)))


def test_binary16_operands(dg):
    desc = dict(tile_k=64, tile_combine="tree", in_dtype="f16", out="bf16")
    M, N, K = 130, 136, 512
    A, B = inputs.spread_f16(5, (M, K), -8, 8), inputs.normal_f16(6, (K, N), 0.5)
    print("tile tree f16", flush=True)
    assert_bits_equal(run(dg, desc, A, B, f16=True), oracle.gemm(desc, A, B), "f16 tree")


@pytest.mark.parametrize("desc", [dict(tile_k=256, tile_combine="tree", out="bf16"), dict(tile_k=64, fma=0, out="bf16")])
def test_bench_shapes_sampled(dg, desc):
    """The M = 1024 descriptors the bench times, 1024 x 4096 x 4096 on
    exponent-spread draws, sampled outputs against the oracle."""
    M, N, K = 1024, 4096, 4096
    A, B = inputs.spread_bf16(31, (M, K), -12, 12), inputs.spread_bf16(32, (K, N), -12, 12)
    print("tile combine bench shape", desc, flush=True)
    got = run(dg, dict(desc, mma="16x16x32"), A, B)
    rng = np.random.default_rng(9)
    ii = np.concatenate([rng.integers(0, M, 400), [0, M - 1]])
    jj = np.concatenate([rng.integers(0, N, 400), [N - 1, 0]])
    want = inputs.f32_to_bf16_bits(oracle.gemm_at(dict(desc, mma="16x16x32"), A, B, None, ii, jj))
    assert_bits_equal(got[ii, jj], want, str(desc))
