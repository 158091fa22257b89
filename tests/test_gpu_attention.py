"""GPU parity of dg_attention against the CPU oracle's attention order (App.
F), bit for bit, through the C ABI.

Ragged heads (lengths not multiples of the key or query block, a single key,
cross attention with Lq != Lk) are compared in full under every descriptor
field; the LLM-shaped head (32 heads x 4096 tokens x 128, causal and not) on
rows the oracle computes one by one.  Inputs: seeded bf16 draws, Q and K
scaled so that scores spread over several binades, V normal or
exponent-spread; qk_scale = RN32(log2(e) / sqrt(d)).
"""
import itertools
import math

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


def scale(d):
    return float(np.float32(math.log2(math.e) / math.sqrt(d)))


def qkv(seed, H, Lq, Lk, d, spread_v=False):
    Q = inputs.normal_bf16(seed, (H, Lq, d), 1.5)
    K = inputs.normal_bf16(seed + 1, (H, Lk, d), 1.5)
    V = inputs.spread_bf16(seed + 2, (H, Lk, d), -8, 8) if spread_v else inputs.normal_bf16(seed + 2, (H, Lk, d))
    return Q, K, V


def run(dg, desc, Q, K, V, qs):
    import torch
    H, Lq, d = Q.shape
    out_bf16 = desc.get("out", "bf16") == "bf16"
    O = torch.full((H, Lq, d), float("nan"), dtype=torch.bfloat16 if out_bf16 else torch.float32, device="cuda")
    dg.dg_attention(dg.AttnDesc(**desc), dev_bf16(Q), dev_bf16(K), dev_bf16(V), O, qs)
    torch.cuda.synchronize()
    return host_bits(O)


UNMASKED = [dict(key_block=w, block_sum=bs, pv_fma=pf, l_fma=lf, final=fi, out=o)
            for w, bs, pf, lf, fi, o in itertools.product([32, 64, 128], ["tree", "seq"], [1, 0], [0, 1],
                                                         ["div", "recip"], ["bf16", "f32"])]
CAUSAL = [dict(key_block=w, causal=1, q_block=bm, block_sum=bs, pv_fma=pf, l_fma=lf, final=fi, out=o)
          for (w, bm), bs, pf, lf, fi, o in itertools.product(
              [(32, 16), (32, 48), (64, 64), (64, 80), (64, 128), (128, 64), (32, 96)], ["tree", "seq"],
              [1, 0], [0, 1], ["div"], ["bf16", "f32"])]


@pytest.mark.parametrize("di", range(0, len(UNMASKED), 2))
def test_unmasked_ragged(dg, di):
    desc = UNMASKED[di]
    for (H, Lq, Lk, d), spread in (((2, 100, 100, 64), False), ((1, 37, 257, 128), True), ((3, 1, 1, 64), False),
                                   ((1, 130, 19, 128), True)):
        print("attention", desc, (H, Lq, Lk, d), flush=True)
        Q, K, V = qkv(10 * di + Lq, H, Lq, Lk, d, spread)
        want = oracle.attention(desc, Q, K, V, scale(d))
        assert_bits_equal(run(dg, desc, Q, K, V, scale(d)), want, "%s %s" % (desc, (H, Lq, Lk, d)))


@pytest.mark.parametrize("di", range(len(CAUSAL)))
def test_causal_ragged(dg, di):
    """Causal heads whose length is not a multiple of the key or query
    block, including BLOCK_M off the key grid (80 with w = 64, 48 with
    w = 32): the split at the multiples of BLOCK_M is part of the answer."""
    desc = CAUSAL[di]
    for (H, L, d), spread in (((2, 150, 64), False), ((1, 257, 128), True), ((1, 1, 64), False)):
        print("attention", desc, (H, L, d), flush=True)
        Q, K, V = qkv(7 * di + L, H, L, L, d, spread)
        want = oracle.attention(desc, Q, K, V, scale(d))
        assert_bits_equal(run(dg, desc, Q, K, V, scale(d)), want, "%s %s" % (desc, (H, L, d)))


def test_query_block_changes_causal_bits_off_the_key_grid(dg):
    """With w = 64, BLOCK_M = 80 and BLOCK_M = 64 walk different boundaries;
    the library follows each (and BLOCK_M = 128 equals 64)."""
    Q, K, V = qkv(5, 1, 300, 300, 64, True)
    base = dict(key_block=64, causal=1, out="f32")
    o64 = run(dg, dict(base, q_block=64), Q, K, V, scale(64))
    o80 = run(dg, dict(base, q_block=80), Q, K, V, scale(64))
    o128 = run(dg, dict(base, q_block=128), Q, K, V, scale(64))
    assert np.array_equal(o64, o128)
    assert not np.array_equal(o64, o80)
    assert_bits_equal(o80, oracle.attention(dict(base, q_block=80), Q, K, V, scale(64)), "BLOCK_M 80")


@pytest.mark.parametrize("causal", [0, 1])
def test_llm_head_sampled(dg, causal):
    """32 heads x 4096 tokens x 128 (a Llama-style head set), the launch the
    bench times: 96 sampled rows (every head, early, middle and late rows)
    against the oracle row by row."""
    H, L, d = 32, 4096, 128
    Q, K, V = qkv(100 + causal, H, L, L, d)
    desc = dict(key_block=64, causal=causal, q_block=128, out="bf16")
    got = run(dg, desc, Q, K, V, scale(d))
    rng = np.random.default_rng(3 + causal)
    hh = np.concatenate([np.arange(H), rng.integers(0, H, 64)])
    ii = np.concatenate([rng.integers(0, 64, H), rng.integers(0, L, 64)])
    want = inputs.f32_to_bf16_bits(oracle.attention_rows(desc, Q, K, V, scale(d), hh, ii))
    assert_bits_equal(got[hh, ii], want, "llm head causal=%d" % causal)
    assert np.all(np.isfinite(inputs.bf16_bits_to_f32(got)))


def test_shape_and_descriptor_refusals(dg):
    import torch
    with pytest.raises(dg.DgError) as e:
        dg.AttnDesc(key_block=16)
    assert e.value.status == dg.DG_ERR_UNSUPPORTED
    with pytest.raises(dg.DgError) as e:
        dg.AttnDesc(causal=1, q_block=40)
    assert e.value.status == dg.DG_ERR_UNSUPPORTED
    Q = torch.zeros((1, 8, 64), dtype=torch.bfloat16, device="cuda")
    K = torch.zeros((1, 9, 64), dtype=torch.bfloat16, device="cuda")
    O = torch.zeros((1, 8, 64), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(dg.DgError) as e:
        dg.dg_attention(dg.AttnDesc(causal=1), Q, K, K, O, 0.1)
    assert e.value.status == dg.DG_ERR_SHAPE
    Q96 = torch.zeros((1, 8, 96), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(dg.DgError) as e:
        dg.dg_attention(dg.AttnDesc(), Q96, Q96, Q96, Q96.clone(), 0.1)
    assert e.value.status == dg.DG_ERR_UNSUPPORTED
