"""GPU parity of GEMMs with OCP e4m3 weights (in_dtype "bf16_e4m3": bf16 A,
one byte per element of B, widened exactly to bf16 and folded by the bf16
instruction) against the CPU oracle, bit for bit, through the C ABI: every
code widened exactly on both kernels that take it (row-major and packed),
ragged shapes under the descriptors they take, the few-row bench shapes
(packed) and the MLP shape (row-major, sampled)."""
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


def dev_u8(codes):
    import torch
    return torch.from_numpy(np.ascontiguousarray(codes, dtype=np.uint8)).cuda()


def run(dg, desc, A, B8, bias=None, packed=False, knobs=None):
    import torch
    desc = dict(desc, in_dtype="bf16_e4m3")
    out_bf16 = desc.get("out", "f32") == "bf16"
    C = torch.full((A.shape[0], B8.shape[1]), float("nan"), device="cuda",
                   dtype=torch.bfloat16 if out_bf16 else torch.float32)
    db = None if bias is None else dev_bf16(bias)
    if packed:
        dg.dg_gemm_packed(dg.Desc(**desc), dev_bf16(A), dg.dg_pack_b(dev_u8(B8)), db, C, knobs=knobs)
    else:
        dg.dg_gemm(dg.Desc(**desc), dev_bf16(A), dev_u8(B8), db, C, knobs=knobs)
    torch.cuda.synchronize()
    return host_bits(C)


@pytest.mark.parametrize("K,N", [(100, 37), (64, 16), (1000, 160), (31, 5)])
def test_pack_layout(dg, K, N):
    """dg_pack_b8 against the layout written out from its definition: every
    64 x 16 block one 1 KB run, lane l's 8 k of the first 32-k block, then
    its 8 k of the second."""
    B8 = inputs.e4m3_uniform(K + N, (K, N))
    Bp = dg.dg_pack_b(dev_u8(B8))
    got = Bp.data.cpu().numpy()[:dg.dg_packed_b8_bytes(K, N)]
    KR, NP = -(-K // 64), -(-N // 16)
    Bz = np.zeros((KR * 64, NP * 16), np.uint8)
    Bz[:K, :N] = B8
    want = np.zeros((NP, KR, 64, 2, 8), np.uint8)
    for l in range(64):
        for h in range(2):
            for e in range(8):
                want[:, :, l, h, e] = Bz[np.arange(KR)[None, :] * 64 + 32 * h + 8 * (l // 16) + e,
                                         np.arange(NP)[:, None] * 16 + l % 16]
    assert np.array_equal(got, want.reshape(-1))


def test_packed_refuses_parts_off_the_64k_runs(dg):
    """e4m3 runs hold 64 k: parts must start on one (bf16's 32-k parts are
    refused for an e4m3 B)."""
    A, B8 = inputs.normal_bf16(1, (4, 256)), inputs.e4m3_uniform(2, (256, 32))
    for desc in (dict(tile_k=32, split_k=2, k_cuts=[96]), dict(tile_k=32, split_k=2, split_layout="strided",
                                                               split_tile=32)):
        with pytest.raises(dg.DgError) as e:
            run(dg, desc, A, B8, packed=True)
        assert e.value.status == dg.DG_ERR_UNSUPPORTED, desc
    got = run(dg, dict(tile_k=32, split_k=2, k_cuts=[128]), A, B8, packed=True)
    assert_bits_equal(got, oracle.gemm(dict(tile_k=32, split_k=2, k_cuts=[128], in_dtype="bf16_e4m3"), A, B8), "cut 128")


@pytest.mark.parametrize("packed", [False, True])
def test_every_code_widens_exactly(dg, packed):
    """Row k0 of B holds the 256 codes (one per column), every other row
    zeros, and A = the unit vector at k0: each output is the single product
    1.0 x code, so the 256 outputs are the 256 decoded values (the
    accumulator starts at +0: -0 gives +0; a NaN code gives NaN).  k0 runs
    over the 32 k of a block: every byte of a lane's 8-byte run."""
    K = 32
    want = inputs.bf16_bits_to_f32(oracle.e4m3_to_bf16_bits(np.arange(256, dtype=np.uint8)))
    fin = ~np.isnan(want)
    for k0 in range(K):
        A = np.zeros((1, K), np.uint16)
        A[0, k0] = 0x3F80
        B8 = np.zeros((K, 256), np.uint8)
        B8[k0] = np.arange(256, dtype=np.uint8)
        got = run(dg, dict(tile_k=64), A, B8, packed=packed)[0]
        assert np.array_equal(got[fin], want[fin]), k0
        assert np.isnan(got[~fin]).all(), k0


DESCS = [
    dict(tile_k=64),
    dict(tile_k=64, out="bf16", epilogue="bias_silu"),
    dict(tile_k=64, split_k=3, split_combine="tree"),
    dict(tile_k=64, split_k=4, split_layout="strided", split_tile=64, out="bf16"),
    dict(tile_k=64, split_k=2, split_layout="strided", split_tile=256),
    dict(tile_k=32, tile_combine="tree", fma=0),                 # row-major only
]


@pytest.mark.parametrize("di", range(len(DESCS)))
@pytest.mark.parametrize("packed", [False, True])
def test_ragged_shapes(dg, di, packed):
    desc = DESCS[di]
    if packed and (desc.get("fma", 1) == 0 or desc.get("tile_combine", "carry") != "carry"):
        # the packed kernel takes a carried, fused accumulator only: refused
        A, B8 = inputs.normal_bf16(7, (5, 256)), inputs.e4m3_uniform(8, (256, 16))
        with pytest.raises(dg.DgError) as ei:
            run(dg, desc, A, B8, packed=True)
        assert ei.value.status == dg.DG_ERR_UNSUPPORTED
        return
    for (M, N, K), draw in [((1, 37, 1000), "uniform"), ((7, 160, 256), "weights"), ((33, 50, 512), "uniform"),
                            ((64, 21, 320), "weights"), ((5, 16, 100), "uniform")]:
        if packed and K % 8:
            continue
        S = desc.get("split_k", 1)
        if S > 1 and desc.get("split_layout") != "strided":
            span = -(-(-(-K // S)) // desc["tile_k"]) * desc["tile_k"]
            if (S - 1) * span >= K:
                continue               # the span rule would leave a part empty
        seed = 13 * di + M + N + K
        A = inputs.normal_bf16(seed, (M, K))
        B8 = inputs.e4m3_uniform(seed + 1, (K, N)) if draw == "uniform" else inputs.e4m3_weights(seed + 1, (K, N))
        bias = inputs.normal_bf16(seed + 2, (N,)) if desc.get("epilogue", "none") != "none" else None
        print("e4m3", desc, (M, N, K), draw, "packed" if packed else "row-major", flush=True)
        want = oracle.gemm(dict(desc, in_dtype="bf16_e4m3"), A, B8, bias)
        assert_bits_equal(run(dg, desc, A, B8, bias, packed=packed), want, "%s %s" % (desc, (M, N, K)))


@pytest.mark.parametrize("case", ["M1", "M7", "M32", "decode_seq", "decode_strided"])
def test_packed_bench_shapes(dg, case):
    """The few-row bench shapes with e4m3 weights: the packed kernel equals
    the row-major one on every output, and the oracle on sampled ones."""
    if case.startswith("M"):
        M, N, K = int(case[1:]), 4096, 4096
        desc = dict(tile_k=64, out="bf16")
    elif case == "decode_seq":
        M, N, K = 8, 4096, 14336
        desc = dict(tile_k=64, split_k=8, out="bf16")
    else:
        M, N, K = 8, 4096, 14336
        desc = dict(tile_k=64, split_k=4, split_layout="strided", split_tile=128, out="bf16")
    A, B8 = inputs.spread_bf16(21, (M, K), -12, 12), inputs.e4m3_uniform(22, (K, N))
    print("e4m3 bench shape", case, flush=True)
    got = run(dg, desc, A, B8, packed=True)
    assert np.array_equal(got, run(dg, desc, A, B8))
    rng = np.random.default_rng(5)
    ii, jj = rng.integers(0, M, 256), rng.integers(0, N, 256)
    want = inputs.f32_to_bf16_bits(oracle.gemm_at(dict(desc, in_dtype="bf16_e4m3"), A, B8, None, ii, jj))
    assert_bits_equal(got[ii, jj], want, case)


def test_mlp_shape_sampled(dg):
    """2048 x 14336 x 4096 with e4m3 weights and the fused bias + SiLU
    (row-major B, the generic kernel): sampled outputs against the oracle."""
    M, N, K = 2048, 14336, 4096
    A = inputs.normal_bf16(31, (M, K))
    B8 = inputs.e4m3_weights(32, (K, N), e_mid=4.0)
    bias = inputs.normal_bf16(33, (N,))
    desc = dict(tile_k=64, out="bf16", epilogue="bias_silu")
    print("e4m3 MLP shape", flush=True)
    got = run(dg, desc, A, B8, bias)
    rng = np.random.default_rng(6)
    ii = np.concatenate([rng.integers(0, M, 600), [0, M - 1]])
    jj = np.concatenate([rng.integers(0, N, 600), [N - 1, 0]])
    want = inputs.f32_to_bf16_bits(oracle.gemm_at(dict(desc, in_dtype="bf16_e4m3"), A, B8, bias, ii, jj))
    assert_bits_equal(got[ii, jj], want, "e4m3 MLP")
