"""GPU parity of e4m3 x e4m3 GEMMs on the fp8 instructions (in_dtype
"e4m3"; Sec. 3.2.1: the fp8 instructions have their own semantics, which
the oracle models) against the CPU oracle, bit for bit, through the C ABI:

  * the four fp8 instruction names under fma = 1 (one chain of 16-k chunks:
    the same bits), on the fp8 tiled kernel (13) and the generic kernel (1);
  * fma = 0 with each instruction's group (16, 32, 64, 128 k from +0), tile
    chains and trees, strided splits, a leading short tile: the generic
    kernel;
  * split-K (span rule, explicit cuts on and off the 16-k grid), bf16
    partials and merges, the bias and bias + SiLU epilogues, bf16 output;
  * ragged shapes (M, N, K not multiples of the block, K and N off the
    16-byte grid), every finite code and an LLM-like weight draw;
  * the SiLU MLP shape 2048 x 14336 x 4096 on sampled outputs, in the
    launch configuration the bench times.
"""
import numpy as np
import pytest

import oracle
from paper_2609_11356_amd import inputs
from tests.gpu_util import assert_bits_equal, dev_bf16, host_bits

pytestmark = pytest.mark.gpu
FP8 = ("16x16x32_fp8", "32x32x16_fp8", "16x16x128_f8f6f4", "32x32x64_f8f6f4")


@pytest.fixture(scope="module")
def dg():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_11356_amd import dg as _dg
    _dg.lib()
    return _dg


def dev_u8(codes):
    import torch
    return torch.from_numpy(np.ascontiguousarray(codes, dtype=np.uint8)).cuda()


def run(dg, desc, A8, B8, bias=None, knobs=None):
    import torch
    desc = dict(desc, in_dtype="e4m3")
    out_bf16 = desc.get("out", "f32") == "bf16"
    C = torch.full((A8.shape[0], B8.shape[1]), float("nan"), device="cuda",
                   dtype=torch.bfloat16 if out_bf16 else torch.float32)
    dg.dg_gemm(dg.Desc(**desc), dev_u8(A8), dev_u8(B8), None if bias is None else dev_bf16(bias), C, knobs=knobs)
    torch.cuda.synchronize()
    return host_bits(C)


def f8_tiled(desc, M, N, K):
    """Whether the library takes desc to the fp8 tiled kernel at this shape."""
    if desc.get("tile_combine", "carry") != "carry" or desc.get("fma", 1) != 1:
        return False
    if desc.get("split_layout") == "strided" or K % 16 or N % 16:
        return False
    S, tk = desc.get("split_k", 1), desc["tile_k"]
    if desc.get("k_cuts"):
        cuts = [0] + list(desc["k_cuts"]) + [K]
    else:
        span = -(-(-(-K // S)) // tk) * tk
        cuts = [min(s * span, K) for s in range(S)] + [K]
    for s in range(S):
        ln = cuts[s + 1] - cuts[s]
        if cuts[s] % 16 or (desc.get("tail") == "first" and (ln % tk) % 16):
            return False
    return True


DESCS = [
    dict(mma="16x16x128_f8f6f4", tile_k=128),
    dict(mma="16x16x32_fp8", tile_k=32),
    dict(mma="32x32x16_fp8", tile_k=64, out="bf16", epilogue="bias_silu"),
    dict(mma="32x32x64_f8f6f4", tile_k=64, split_k=3),
    dict(mma="16x16x128_f8f6f4", tile_k=128, split_k=2, split_combine="tree", partial="bf16", merge="bf16",
         out="bf16", epilogue="bias"),
    dict(mma="16x16x32_fp8", tile_k=64, tail="first", split_k=2),
    dict(mma="16x16x32_fp8", tile_k=32, fma=0),
    dict(mma="32x32x16_fp8", tile_k=16, fma=0, out="bf16"),
    dict(mma="16x16x128_f8f6f4", tile_k=128, fma=0),
    dict(mma="32x32x64_f8f6f4", tile_k=128, fma=0, tile_combine="tree"),
    dict(mma="16x16x32_fp8", tile_k=64, tile_combine="seq"),
    dict(mma="16x16x32_fp8", tile_k=32, split_k=4, split_layout="strided", split_tile=64, out="bf16"),
]
SHAPES = [(130, 160, 1024), (64, 128, 512), (7, 48, 2048), (200, 272, 640), (33, 40, 1000), (5, 37, 100)]


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("di", range(len(DESCS)))
def test_matches_oracle(dg, di, shape):
    desc = DESCS[di]
    M, N, K = shape
    S = desc.get("split_k", 1)
    if S > 1 and desc.get("split_layout") != "strided":
        span = -(-(-(-K // S)) // desc["tile_k"]) * desc["tile_k"]
        if (S - 1) * span >= K:
            # the span rule leaves a part empty: the oracle and the library both refuse
            A8, B8 = inputs.e4m3_uniform(7, (M, K)), inputs.e4m3_uniform(8, (K, N))
            bias = inputs.normal_bf16(9, (N,)) if desc.get("epilogue", "none") != "none" else None
            with pytest.raises(oracle.OracleError, match="status 3"):
                oracle.gemm(dict(desc, in_dtype="e4m3"), A8, B8, bias)
            with pytest.raises(dg.DgError) as ei:
                run(dg, desc, A8, B8, bias)
            assert ei.value.status == dg.DG_ERR_SHAPE
            return
    seed = 100 + 31 * di + M + K
    bias = inputs.normal_bf16(seed + 2, (N,), 0.5) if desc.get("epilogue", "none") != "none" else None
    tiled = f8_tiled(desc, M, N, K)
    for draw in ("uniform", "weights"):
        A8 = inputs.e4m3_uniform(seed, (M, K)) if draw == "uniform" else inputs.e4m3_weights(seed, (M, K))
        B8 = inputs.e4m3_uniform(seed + 1, (K, N)) if draw == "uniform" else inputs.e4m3_weights(seed + 1, (K, N))
        print("fp8 gemm", desc, shape, draw, "tiled" if tiled else "generic", flush=True)
        want = oracle.gemm(dict(desc, in_dtype="e4m3"), A8, B8, bias)
        assert_bits_equal(run(dg, desc, A8, B8, bias), want, "%s %s %s" % (desc, shape, draw))
        assert_bits_equal(run(dg, desc, A8, B8, bias, knobs=dict(kernel=1)), want, "generic %s" % desc)
        if tiled:
            for tm, tn in ((128, 128), (256, 256), (256, 128)):
                assert_bits_equal(run(dg, desc, A8, B8, bias, knobs=dict(kernel=13, tile_m=tm, tile_n=tn)), want,
                                  "kernel 13 tile %dx%d %s" % (tm, tn, desc))


def test_instruction_names_give_the_same_bits_under_fma(dg):
    M, N, K = 96, 144, 1536
    A8, B8 = inputs.e4m3_uniform(1, (M, K)), inputs.e4m3_uniform(2, (K, N))
    print("fp8 instruction names", flush=True)
    outs = [run(dg, dict(mma=m, tile_k=128), A8, B8) for m in FP8]
    for o in outs[1:]:
        assert np.array_equal(o, outs[0])


def test_explicit_cuts_on_and_off_the_16k_grid(dg):
    """Cuts on multiples of 16 take the tiled kernel; a cut at 72 moves the
    chunk grid, so the library runs the generic kernel (and kernel 13 is
    refused); both equal the oracle."""
    M, N, K = 40, 64, 480
    A8, B8 = inputs.e4m3_uniform(3, (M, K)), inputs.e4m3_uniform(4, (K, N))
    for cuts, tiled in (([160, 320], True), ([72, 300], False)):
        desc = dict(mma="16x16x32_fp8", tile_k=32, split_k=3, k_cuts=cuts)
        print("fp8 cuts", cuts, flush=True)
        want = oracle.gemm(dict(desc, in_dtype="e4m3"), A8, B8)
        assert_bits_equal(run(dg, desc, A8, B8), want, str(cuts))
        if tiled:
            for tm, tn in ((128, 128), (256, 256), (256, 128)):
                assert_bits_equal(run(dg, desc, A8, B8, knobs=dict(kernel=13, tile_m=tm, tile_n=tn)), want,
                                  "kernel 13 %s" % cuts)
        else:
            with pytest.raises(dg.DgError) as e:
                run(dg, desc, A8, B8, knobs=dict(kernel=13))
            assert e.value.status == dg.DG_ERR_UNSUPPORTED


def test_refusals(dg):
    A8, B8 = inputs.e4m3_uniform(5, (16, 256)), inputs.e4m3_uniform(6, (256, 64))
    for desc, knobs in [(dict(mma="16x16x32_fp8", tile_k=32, fma=0), dict(kernel=13)),
                        (dict(mma="16x16x32_fp8", tile_k=64, tile_combine="tree"), dict(kernel=13)),
                        (dict(mma="16x16x32_fp8", tile_k=64), dict(kernel=3)),
                        (dict(mma="16x16x32_fp8", tile_k=64), dict(kernel=13, tile_m=64)),
                        (dict(mma="16x16x32_fp8", tile_k=64), dict(kernel=13, tile_m=256, tile_n=64))]:
        with pytest.raises(dg.DgError) as e:
            run(dg, desc, A8, B8, knobs=knobs)
        assert e.value.status == dg.DG_ERR_UNSUPPORTED, (desc, knobs)
    with pytest.raises(dg.DgError) as e:
        dg.Desc(mma="16x16x32", in_dtype="e4m3")
    assert e.value.status == dg.DG_ERR_INVALID
    with pytest.raises(dg.DgError) as e:
        dg.Desc(mma="16x16x128_f8f6f4", tile_k=128)
    assert e.value.status == dg.DG_ERR_INVALID


def test_special_codes(dg):
    """NaN codes give NaN in their row and column only; -0 and zero codes
    give +0 sums; the largest products (448 x 448) stay finite."""
    M, N, K = 32, 32, 256
    A8 = inputs.e4m3_uniform(7, (M, K))
    B8 = inputs.e4m3_uniform(8, (K, N))
    A8[3, 17] = 0x7F
    B8[200, 5] = 0xFF
    A8[4] = 0x80
    A8[5] = 0x7E
    B8[:, 6] = 0x7E
    desc = dict(mma="16x16x128_f8f6f4", tile_k=128)
    want = oracle.gemm(dict(desc, in_dtype="e4m3"), A8, B8)
    for knobs in (dict(kernel=13, tile_m=256, tile_n=256), dict(kernel=13, tile_m=256, tile_n=128),
                  dict(kernel=13, tile_m=128), dict(kernel=1)):
        got = run(dg, desc, A8, B8, knobs=knobs)
        assert_bits_equal(got, want, str(knobs))
    assert np.isnan(want[3]).all() and np.isnan(want[:, 5]).all()
    assert np.isfinite(np.delete(np.delete(want, 3, 0), 5, 1)).all()


@pytest.mark.parametrize("knobs", [dict(kernel=13, tile_m=256, tile_n=256), dict(kernel=13, tile_m=256, tile_n=128),
                                   dict(kernel=13, tile_m=128), dict(kernel=1)],
                         ids=["k13-256", "k13-256x128", "k13-128", "k1"])
def test_mlp_shape_sampled(dg, knobs):
    """2048 x 14336 x 4096 with the fused bias + SiLU and bf16 output (the
    bench's fp8 MLP launch: kernel 13 on 256 x 256 blocks; also its 128 x 128
    blocks and the generic kernel), sampled outputs against the oracle."""
    M, N, K = 2048, 14336, 4096
    A8 = inputs.e4m3_weights(41, (M, K), e_mid=4.0)
    B8 = inputs.e4m3_weights(42, (K, N))
    bias = inputs.normal_bf16(43, (N,))
    desc = dict(mma="16x16x128_f8f6f4", tile_k=128, out="bf16", epilogue="bias_silu")
    print("fp8 MLP shape", knobs, flush=True)
    got = run(dg, desc, A8, B8, bias, knobs=knobs)
    rng = np.random.default_rng(12)
    ii = np.concatenate([rng.integers(0, M, 500), [0, M - 1, M - 1]])
    jj = np.concatenate([rng.integers(0, N, 500), [N - 1, 0, N - 1]])
    want = inputs.f32_to_bf16_bits(oracle.gemm_at(dict(desc, in_dtype="e4m3"), A8, B8, bias, ii, jj))
    assert_bits_equal(got[ii, jj], want, "fp8 MLP %s" % knobs)


def test_other_entry_points(dg):
    """e4m3 x e4m3 through the entry point that allocates nothing (split-K
    partials in its fixed scratch: equal to dg_gemm, also on a second,
    smaller call) and through dg_gemm_colsum (C as dg_gemm writes it, the
    column sums as the oracle's tree over that C)."""
    import torch
    for desc, (M, N, K) in ((dict(mma="16x16x128_f8f6f4", tile_k=128, split_k=4, split_combine="tree"), (300, 272, 2048)),
                            (dict(mma="16x16x32_fp8", tile_k=32, split_k=3, fma=0, out="bf16"), (40, 96, 1000))):
        A8, B8 = inputs.e4m3_uniform(M + K, (M, K)), inputs.e4m3_uniform(N + K, (K, N))
        d = dg.Desc(**dict(desc, in_dtype="e4m3"))
        out_bf16 = desc.get("out") == "bf16"
        dt = torch.bfloat16 if out_bf16 else torch.float32
        for m in (M, M // 2):
            dA, dB = dev_u8(A8[:m]), dev_u8(B8)
            C1 = torch.full((m, N), float("nan"), device="cuda", dtype=dt)
            C2 = torch.full((m, N), float("nan"), device="cuda", dtype=dt)
            print("fp8 noalloc", desc, (m, N, K), flush=True)
            dg.dg_gemm(d, dA, dB, None, C1)
            dg.dg_gemm_noalloc(d, dA, dB, None, C2)
            torch.cuda.synchronize()
            assert_bits_equal(host_bits(C2), host_bits(C1), "noalloc %s m=%d" % (desc, m))
        want = oracle.gemm(dict(desc, in_dtype="e4m3"), A8, B8)
        assert_bits_equal(host_bits(C1), want[:M // 2], "dg_gemm %s" % desc)
    desc = dict(mma="16x16x128_f8f6f4", tile_k=128)
    M, N, K = 520, 264, 768
    A8, B8 = inputs.e4m3_weights(61, (M, K)), inputs.e4m3_weights(62, (K, N))
    d = dg.Desc(**dict(desc, in_dtype="e4m3"))
    C = torch.full((M, N), float("nan"), device="cuda", dtype=torch.float32)
    cs = torch.full((N,), float("nan"), device="cuda", dtype=torch.float32)
    print("fp8 colsum", flush=True)
    dg.dg_gemm_colsum(d, dev_u8(A8), dev_u8(B8), None, C, cs)
    torch.cuda.synchronize()
    want = oracle.gemm(dict(desc, in_dtype="e4m3"), A8, B8)
    assert_bits_equal(host_bits(C), want, "colsum GEMM")
    assert_bits_equal(cs.cpu().numpy(), oracle.colsum(want), "column sums")
