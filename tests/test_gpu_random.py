"""Randomised GPU parity of dg_gemm against the CPU oracle (gfx950).

Each case draws, from its own seed, a descriptor (instruction group, tile
length, split count and merge, tile combine, short-tile position, the fma
rule, partial / merge / output types, epilogue and rounding point, operand
format), a ragged shape, inputs from the seeded generators, and one of the
speed knobs the knob test uses, among those the descriptor admits (the tiled
MFMA kernels take a carried accumulator with the fused rule; binary16
operands are not taken by the tiled, direct-to-LDS and four-wave kernels; the
scalar instruction runs on its own kernel).  A knob the drawn shape still
cannot run on is refused with DG_ERR_UNSUPPORTED; the case then runs the
library's own choice, so that every case compares all of its outputs with the
oracle, bit for bit, and the last test requires that most drawn knobs ran.  A draw whose K the descriptor's cut plan cannot split is one
the oracle refuses; the library must then refuse it as well (DG_ERR_SHAPE).
Most draws keep to what the tiled MFMA kernels accept (the 16x16x32 group, a
carried accumulator, the fused rule, K a multiple of 8) so that the knobs
reach those kernels.
"""
import numpy as np
import pytest

import oracle
from paper_2609_11356_amd import inputs
from tests.gpu_util import assert_bits_equal, dev_bf16, dev_f16, host_bits
from tests.test_gpu_gemm import KNOBS

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dg():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_11356_amd import dg as _dg
    _dg.lib()
    return _dg


def draw(seed):
    rng = np.random.default_rng(50_000 + seed)
    tiled = rng.random() < 0.6
    mma = "16x16x32" if tiled else str(rng.choice(["16x16x32", "32x32x16", "32x32x16", "scalar"]))
    g = {"16x16x32": 32, "32x32x16": 16, "scalar": 1}[mma]
    tile_k = int(g * rng.choice([1, 2, 4])) if mma != "scalar" else int(rng.choice([4, 8, 16, 64]))
    S = int(rng.choice([1, 1, 1, 2, 3, 4, 8]))
    desc = dict(mma=mma, tile_k=tile_k)
    if S > 1:
        desc.update(split_k=S, split_combine=str(rng.choice(["seq", "tree"])))
        if rng.random() < 0.3:
            desc["partial"] = "bf16"
            if rng.random() < 0.5:
                desc["merge"] = "bf16"
    if not tiled:
        if rng.random() < 0.4:
            desc["tile_combine"] = str(rng.choice(["seq", "tree"]))
        if mma != "scalar" and rng.random() < 0.3:
            desc["fma"] = 0
    if rng.random() < 0.2:
        desc["tail"] = "first"
    if rng.random() < 0.5:
        desc["out"] = "bf16"
    epi = str(rng.choice(["none", "none", "bias", "bias_silu"]))
    if epi != "none":
        desc["epilogue"] = epi
        if epi == "bias_silu" and rng.random() < 0.3:
            desc["epi_round"] = "pre_act"
    f16 = mma == "16x16x32" and rng.random() < 0.2
    if f16:
        desc["in_dtype"] = "f16"
    M = int(rng.choice([1, 7, 16, 33, 64, 100, 129, 160, 257]))
    N = int(rng.choice([8, 24, 64, 136, 200, 256, 264, 320]))
    K = int(rng.integers(max(1, S), 1200))
    if tiled:
        K = max(8 * S, K - K % 8)
    if f16:
        A = inputs.spread_f16(2 * seed, (M, K))
        B = inputs.spread_f16(2 * seed + 1, (K, N))
    elif rng.random() < 0.5:
        A = inputs.spread_bf16(2 * seed, (M, K))
        B = inputs.spread_bf16(2 * seed + 1, (K, N))
    else:
        A = inputs.normal_bf16(2 * seed, (M, K))
        B = inputs.normal_bf16(2 * seed + 1, (K, N), 0.05)
    bias = inputs.normal_bf16(7 * seed + 3, (N,), 1.0) if epi != "none" else None
    if mma == "scalar":
        pool = [dict(kernel=9)]
    elif not tiled:
        pool = [dict(kernel=1)]
    elif f16:
        pool = [k for k in KNOBS if k is not None and k["kernel"] not in (2, 7, 8, 10)]
    else:
        pool = [k for k in KNOBS if k is not None]
    knobs = pool[int(rng.integers(len(pool)))] if rng.random() < 0.8 else None
    return desc, A, B, bias, knobs, f16


KNOB_RUNS = {"ran": 0, "refused": 0}


@pytest.mark.parametrize("seed", range(192))
def test_random_descriptor_and_knob(dg, seed):
    import torch
    desc, A, B, bias, knobs, f16 = draw(seed)
    M, K = A.shape
    N = B.shape[1]
    print("seed %d M %d N %d K %d desc %s knobs %s" % (seed, M, N, K, desc, knobs), flush=True)
    d = dg.Desc(**desc)
    try:
        want = oracle.gemm(desc, A, B, bias)
    except oracle.OracleError as ex:
        # a K the descriptor's cut plan cannot split: the library refuses it too
        assert "status 3" in str(ex), ex
        want = None
    C = torch.empty((M, N), dtype=torch.bfloat16 if desc.get("out") == "bf16" else torch.float32, device="cuda")
    C.fill_(float("nan"))
    dev = dev_f16 if f16 else dev_bf16
    dA, dB = dev(A), dev(B)
    db = None if bias is None else dev_bf16(bias)
    if want is None:
        with pytest.raises(dg.DgError) as ei:
            dg.dg_gemm(d, dA, dB, db, C)
        assert ei.value.status == dg.DG_ERR_SHAPE
        return
    try:
        dg.dg_gemm(d, dA, dB, db, C, knobs=knobs)
        if knobs is not None:
            KNOB_RUNS["ran"] += 1
    except dg.DgError as ex:
        assert ex.status == dg.DG_ERR_UNSUPPORTED, ex
        KNOB_RUNS["refused"] += 1
        dg.dg_gemm(d, dA, dB, db, C)
    torch.cuda.synchronize()
    assert_bits_equal(host_bits(C), want, "seed %d %s %s" % (seed, desc, knobs))


def test_drawn_knobs_mostly_ran(dg):
    """The speed-knob coverage is measured: of the drawn knobs, at least 85 %
    ran as drawn (the rest hit a shape limit and ran the library's choice)."""
    n = KNOB_RUNS["ran"] + KNOB_RUNS["refused"]
    if n < 100:
        pytest.skip("needs the whole seed range in this session (%d knob cases ran)" % n)
    assert KNOB_RUNS["ran"] >= 0.85 * n, KNOB_RUNS
