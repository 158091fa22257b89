"""Pins of the CPU oracle to facts other than itself (CPU only).

Each test ties one part of the oracle to something it does not compute:
values the paper prints for its worked examples (tests/golden), closed forms,
library routines (numpy's correctly rounded conversions and sequential
accumulation, torch's bf16 conversion, Python's exact rationals), textbook
special cases, invariants, and error bounds against float64.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2609_11356_amd import inputs
from tests.exact import bf, f, rn32, rn32_sqrt, rnbf

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
ONE = np.uint16(0x3F80)


def bits(x):
    return inputs.f32_to_bf16_bits(np.asarray(x, dtype=np.float32))


def exact_desc(g, **kw):
    d = dict(model="exact", g=g, tile_k=kw.pop("tile_k", max(g, 64)))
    d.update(kw)
    return d


# --------------------------------------------------------------- rounding


def test_rn32_helper_matches_numpy_conversion():
    """The exact-rational RN32 used by later pins agrees with numpy's
    correctly rounded float64 -> float32 conversion, ties and subnormals
    included."""
    rng = np.random.default_rng(11)
    d = rng.standard_normal(4000) * np.exp2(rng.integers(-160, 128, 4000))
    # exact binary32 midpoints: x.5 ulp
    mids = []
    for _ in range(500):
        v = np.float32(rng.standard_normal() * 2.0 ** rng.integers(-140, 100))
        nxt = np.nextafter(v, np.float32(np.inf))
        mids.append((float(v) + float(nxt)) / 2)
    for x in list(d) + mids + [2.0 ** -150, 3 * 2.0 ** -151, 2.0 ** -149 * 1.5]:
        assert rn32(Fraction(x)).view(np.uint32) == np.float32(x).view(np.uint32), x


def test_bf16_rounding_matches_torch():
    """Oracle bf16 RNE == torch's fp32 -> bf16 conversion over every high half
    and the low halves that decide rounding."""
    torch = pytest.importorskip("torch")
    hi = np.arange(0, 1 << 16, dtype=np.uint32) << 16
    lows = np.array([0, 1, 0x7FFF, 0x8000, 0x8001, 0xFFFF, 0x4000, 0xC000], dtype=np.uint32)
    u = (hi[:, None] | lows[None, :]).reshape(-1)
    x = u.view(np.float32)
    ref = torch.from_numpy(x.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    ours = np.array([oracle.f32_to_bf16(v) for v in x[::7]], dtype=np.uint16)
    refs = ref[::7]
    nan = np.isnan(x[::7])
    assert np.array_equal(ours[~nan], refs[~nan])
    assert np.all((ours[nan] & 0x7FFF) > 0x7F80)
    # the input generator's packer agrees too
    gen = inputs.f32_to_bf16_bits(x)
    assert np.array_equal(gen[~np.isnan(x)], ref[~np.isnan(x)])


# ------------------------------------------------------ exact group sums


@pytest.mark.parametrize("mode", ["normal", "spread", "wide"])
def test_exact_dot_matches_rationals(mode):
    """One rounding of the exact sum of bf16 products plus an fp32 seed
    (the paper's instruction hypothesis, Sec. 3.2.1) == Python's exact
    rational sum rounded by the IEEE definition."""
    rng = np.random.default_rng({"normal": 1, "spread": 2, "wide": 3}[mode])
    for t in range(300):
        n = int(rng.integers(1, 40))
        if mode == "normal":
            a, b = bits(rng.standard_normal(n)), bits(rng.standard_normal(n))
        elif mode == "spread":
            a = inputs.spread_bf16(1000 + t, n)
            b = inputs.spread_bf16(5000 + t, n)
        else:
            a = inputs.spread_bf16(1000 + t, n, -120, 120)
            b = inputs.spread_bf16(5000 + t, n, -10, 10)
        c = np.float32(rng.standard_normal() * 2.0 ** rng.integers(-30, 30))
        want = rn32(sum(bf(x) * bf(y) for x, y in zip(a, b)) + f(c))
        got = oracle.exact_dot_rn32(c, a, b)
        assert got.view(np.uint32) == want.view(np.uint32)
        # fma = 0: the group rounds on its own, then a second rounding
        got0 = oracle.group_update(c, a, b, g=64, fma=0, model="exact")
        want0 = np.float32(c) + rn32(sum(bf(x) * bf(y) for x, y in zip(a, b)))
        assert got0.view(np.uint32) == np.float32(want0).view(np.uint32)


# ------------------------------------------------ order: textbook cases


@pytest.mark.parametrize("fma", [0, 1])
def test_group_of_one_is_sequential_fp32_dot(fma):
    """g = 1, no split, carried accumulator: the descriptor's order is the
    plain left-to-right binary32 dot product (a product of two bf16 values is
    exact in binary32), i.e. numpy's sequential accumulation."""
    rng = np.random.default_rng(5)
    K, N = 300, 5
    A = bits(rng.standard_normal((3, K)))
    B = bits(rng.standard_normal((K, N)) * 0.1)
    C = oracle.gemm(exact_desc(1, tile_k=8, fma=fma), A, B)
    Af, Bf = inputs.bf16_bits_to_f32(A), inputs.bf16_bits_to_f32(B)
    for i in range(3):
        for j in range(N):
            prods = (Af[i] * Bf[:, j]).astype(np.float32)
            ref = np.add.accumulate(prods, dtype=np.float32)[-1]
            assert C[i, j].view(np.uint32) == ref.view(np.uint32)


DESCS = [
    dict(model="gfx950", mma="16x16x32", tile_k=64),
    dict(model="gfx950", mma="32x32x16", tile_k=64, fma=0),
    dict(model="gfx950", mma="16x16x32", tile_k=32, split_k=2, tile_combine="tree", split_combine="tree"),
    dict(model="gfx950", mma="16x16x32", tile_k=64, split_k=3, tile_combine="seq", split_combine="seq"),
    dict(model="gfx950", mma="16x16x32", tile_k=64, split_k=9, split_combine="tree", tail="first"),
    dict(model="gfx950", mma="16x16x32", tile_k=64, split_k=4, partial="bf16", merge="bf16"),
    dict(model="exact", g=16, tile_k=32, split_k=2, tile_combine="tree"),
    dict(model="exact", g=1, tile_k=4, tile_combine="seq", fma=0),
]


@pytest.mark.parametrize("desc", DESCS)
@pytest.mark.parametrize("K", [1, 7, 64, 257, 576, 8648])
def test_all_ones_counts_terms(desc, K):
    """All-ones A and B: every output is exactly K (binary32 holds every
    integer below 2^24), so any dropped or doubled term shows (the paper's
    App. D count test, including K = 8648 split nine ways)."""
    S = desc.get("split_k", 1)
    if desc.get("merge") == "bf16" and K > 256:
        pytest.skip("bf16 merge cannot hold K > 256 exactly")
    span = -(-K // S)
    tk = desc["tile_k"]
    span = -(-span // tk) * tk
    if S > 1 and (S - 1) * span >= K:
        with pytest.raises(oracle.OracleError):
            oracle.gemm(desc, np.full((2, K), ONE), np.full((K, 3), ONE))
        return
    C = oracle.gemm(desc, np.full((2, K), ONE), np.full((K, 3), ONE))
    assert np.all(C == K)


@pytest.mark.parametrize("desc", DESCS)
def test_small_integers_are_exact(desc):
    """Integer operands whose partial sums stay below 2^24 make every order
    exact: the oracle must return the integer matrix product."""
    rng = np.random.default_rng(9)
    K = 1152
    Ai = rng.integers(-8, 9, (4, K))
    Bi = rng.integers(-8, 9, (K, 6))
    C = oracle.gemm(desc, bits(Ai), bits(Bi))
    if desc.get("partial") == "bf16":
        pytest.skip("bf16 partials round integers above 256")
    assert np.array_equal(C.astype(np.int64), Ai @ Bi)


# ---------------------------------------------- the paper's worked walks


def _golden():
    with open(os.path.join(GOLDEN, "paper_walks.json")) as fh:
        return json.load(fh)


def _splitk_zero_set(desc):
    g = _golden()
    w = g["splitk_walk"]
    K, L, r = w["K"], g["L"], g["r"]
    rows = []
    for m in range(1, K - 1):
        v = np.zeros(K, dtype=np.float32)
        v[0], v[m], v[m + 1] = r, L, -L
        rows.append(v)
    A = bits(np.stack(rows))
    B = np.full((K, 1), ONE)
    C = oracle.gemm(desc, A, B)[:, 0]
    assert set(np.unique(C)) <= {0.0, np.float32(r)}
    return {m for m, v in zip(range(1, K - 1), C) if v == 0.0}


def test_splitk_walk_gfx950_matches_paper():
    """Sec. 4 split-K walk: r at k = 0, +L/-L at (m, m+1), K = 576 cut into
    three parts of 192.  The paper reads zeros for m = 1..191 and at 383 only.
    Under the gfx950 chunk arithmetic every placement inside r's part floors r
    away, so the measured set is exactly the printed one, for either
    instruction shape."""
    w = _golden()["splitk_walk"]
    want = set(range(w["zero_from"], w["zero_to"] + 1)) | set(w["zero_also"])
    for mma in ("16x16x32", "32x32x16"):
        desc = dict(model="gfx950", mma=mma, tile_k=64, split_k=w["parts"])
        assert list(oracle.plan_cuts(desc, w["K"])) == [0, 192, 384, 576]
        assert _splitk_zero_set(desc) == want


@pytest.mark.parametrize("g", [1, 16, 32])
def test_splitk_walk_exact_groups(g):
    """The same walk under the paper's exact-group hypothesis (Sec. 3.2.1).
    With g = 1 it reproduces the printed set.  With wider exact groups a pair
    inside one group cancels before r is seen, so only placements whose +L
    closes a group (m = g-1 mod g) or straddles a part boundary absorb r."""
    w = _golden()["splitk_walk"]
    desc = exact_desc(g, tile_k=64, split_k=w["parts"])
    got = _splitk_zero_set(desc)
    if g == 1:
        want = set(range(1, 192)) | {383}
    else:
        want = {m for m in range(1, 191) if m % g == g - 1} | {191, 383}
    assert got == want


def test_contiguous_walk_matches_paper():
    """Sec. 4 contiguous walk: eight terms summed in two groups of four, each
    group a left fold; r at 0; the pair at (1,2), (2,3), (3,4) gives 0 and the
    first placement returning r is (4,5)."""
    g = _golden()
    w = g["contiguous_walk"]
    desc = exact_desc(1, tile_k=w["group"], tile_combine="seq")
    for pair in w["pairs_zero"] + [w["first_pair_returning_r"]]:
        v = np.zeros(w["terms"], dtype=np.float32)
        v[w["r_at"]], v[pair[0]], v[pair[1]] = g["r"], g["L"], -g["L"]
        c = oracle.gemm(desc, bits(v[None, :]), np.full((w["terms"], 1), ONE))[0, 0]
        want = g["r"] if pair == w["first_pair_returning_r"] else 0.0
        assert c == np.float32(want), pair


# -------------------------------------------------------- trees and folds


def test_nonassociativity_hand_examples():
    """[2^24, 1, 1, -2^24]: chain 0, balanced tree 1, exact 2.
    [2^24, 1, -2^24, 1]: the count-up (natural-order) tree gives 1 while the
    count-down butterfly -- a tree over bit-reversed lanes (Sec. 3.2.2, GEMV)
    -- gives 2; the pinned order is the first."""
    v = np.array([2.0 ** 24, 1, 1, -2.0 ** 24], dtype=np.float32)
    assert oracle.tree(v) == 1.0
    X = v[None, :]
    assert oracle.rowsum(dict(leaf_w=4), X)[0] == 0.0
    assert oracle.rowsum(dict(leaf_w=1), X)[0] == 1.0
    w = np.array([2.0 ** 24, 1, -2.0 ** 24, 1], dtype=np.float32)
    assert oracle.tree(w) == 1.0
    assert oracle.tree(w[[0, 2, 1, 3]]) == 2.0


def _halving(v):
    v = np.asarray(v, dtype=np.float32)
    if len(v) == 1:
        return v[0]
    h = len(v) // 2
    return np.float32(_halving(v[:h]) + _halving(v[h:]))


def test_tree_is_recursive_halving_over_negzero_padding():
    """The balanced tree equals textbook recursive halving for a power-of-two
    count, and for any count equals it over the values padded on the right
    with -0 (the exact identity of binary32 addition)."""
    rng = np.random.default_rng(3)
    for n in list(range(1, 70)) + [127, 128, 129, 1000]:
        v = (rng.standard_normal(n) * np.exp2(rng.integers(-20, 20, n))).astype(np.float32)
        p = 1 << (n - 1).bit_length()
        padded = np.concatenate([v, np.full(p - n, -0.0, dtype=np.float32)])
        assert oracle.tree(v).view(np.uint32) == _halving(padded).view(np.uint32), n


def test_rowsum_special_cases():
    rng = np.random.default_rng(4)
    X = inputs.lognormal_f32(4, (6, 300))
    # one leaf covering the row: plain sequential accumulation
    seq = oracle.rowsum(dict(leaf_w=512), X)
    for r in range(6):
        assert seq[r] == np.add.accumulate(X[r], dtype=np.float32)[-1]
    # leaves of one element: the balanced tree of the elements
    tr = oracle.rowsum(dict(leaf_w=1), X)
    for r in range(6):
        assert tr[r] == oracle.tree(X[r])
    # leaves of 64: tree over the sequential leaves (SUM)
    lw = oracle.rowsum(dict(leaf_w=64), X)
    for r in range(6):
        leaves = [np.add.accumulate(X[r, i:i + 64], dtype=np.float32)[-1] for i in range(0, 300, 64)]
        assert lw[r] == oracle.tree(np.array(leaves, dtype=np.float32))
    # SUMSQ without fma: sequential sum of binary32 squares
    sq = oracle.rowsum(dict(leaf_w=512, reduce="sumsq", fma=0), X)
    for r in range(6):
        assert sq[r] == np.add.accumulate((X[r] * X[r]).astype(np.float32), dtype=np.float32)[-1]
    # SUMSQ with fma: s = RN32(x0^2), then s = RN32(x_i^2 + s) (one rounding)
    Y = X[:, :40]
    sf = oracle.rowsum(dict(leaf_w=64, reduce="sumsq", fma=1), Y)
    for r in range(6):
        s = rn32(f(Y[r, 0]) ** 2)
        for x in Y[r, 1:]:
            s = rn32(f(x) ** 2 + f(s))
        assert sf[r].view(np.uint32) == s.view(np.uint32)
    # comparable magnitudes, where one rounding and two roundings part ways
    U = np.random.default_rng(41).uniform(1, 2, (4, 200)).astype(np.float32)
    su = oracle.rowsum(dict(leaf_w=256, reduce="sumsq", fma=1), U)
    sd = oracle.rowsum(dict(leaf_w=256, reduce="sumsq", fma=0), U)
    for r in range(4):
        s = rn32(f(U[r, 0]) ** 2)
        for x in U[r, 1:]:
            s = rn32(f(x) ** 2 + f(s))
        assert su[r].view(np.uint32) == s.view(np.uint32)
    assert not np.array_equal(su, sd)
    # empty rows sum to +0
    assert oracle.rowsum(dict(leaf_w=64), np.zeros((3, 0), np.float32)).tolist() == [0.0] * 3


# ------------------------------------- strided leaves and the count-down fold


def _butterfly(lanes, down):
    """An xor butterfly simulated lane by lane in binary32 over len(lanes) (a
    power of two) lanes: at each step every lane adds its partner's value, a
    lane holding nothing (None) taking its partner's value as it is.  Offsets
    run 1, 2, 4, .. (up) or in the reverse order (down).  Returns lane 0."""
    P = len(lanes)
    v = list(lanes)
    offs = [1 << k for k in range(P.bit_length() - 1)]
    for d in (offs[::-1] if down else offs):
        nv = []
        for lane in range(P):
            a, b = v[lane], v[lane ^ d]
            nv.append(b if a is None else a if b is None else np.float32(np.float32(a) + np.float32(b)))
        v = nv
    return v[0]


def test_fold_down_hand_example():
    """[2^24, 1, -2^24, 1] as four lanes: the count-up butterfly pairs 0-1
    and 2-3 and gives 1; the count-down butterfly pairs 0-2 and 1-3 (a tree
    over the lanes in bit-reversed order, Sec. 3.2.2 GEMV) and gives 2."""
    X = np.array([[2.0 ** 24, 1, -2.0 ** 24, 1]], dtype=np.float32)
    for layout, w in (("strided", 4), ("contiguous", 1)):
        assert oracle.rowsum(dict(leaf_w=w, leaf_layout=layout), X)[0] == 1.0
        assert oracle.rowsum(dict(leaf_w=w, leaf_layout=layout, lane_fold="down"), X)[0] == 2.0


def test_folds_match_simulated_butterflies():
    """The oracle's two trees equal the two butterflies simulated lane by lane,
    for every lane count up to 256 and every number of occupied lanes (a -0
    lane next to an empty one keeps its sign: nothing is added to it)."""
    rng = np.random.default_rng(17)
    for P in (1, 2, 4, 8, 16, 32, 64, 128, 256):
        for n in sorted({1, 2, 3, P // 2 + 1, P - 1, P} - {0}):
            if n > P:
                continue
            v = (rng.standard_normal(n) * np.exp2(rng.integers(-30, 30, n))).astype(np.float32)
            lanes = list(v) + [None] * (P - n)
            assert oracle.tree_bitrev(v, P).view(np.uint32) == _butterfly(lanes, True).view(np.uint32), (P, n)
            assert oracle.tree(v).view(np.uint32) == _butterfly(lanes, False).view(np.uint32), (P, n)
    negz = np.array([-0.0], dtype=np.float32)
    assert oracle.tree_bitrev(negz, 4).view(np.uint32) == np.float32(-0.0).view(np.uint32)


def test_strided_leaves_take_every_count_th_element():
    """Two lanes over six elements: lane 0 folds x0, x2, x4 = 2^24, 1, 1 (each
    1 lost to rounding) and lane 1 folds -2^24, 0, 0, so the row sums to 0;
    contiguous leaves of three give (2^24 - 2^24 + 1) + (0 + 1 + 0) = 2."""
    X = np.array([[2.0 ** 24, -2.0 ** 24, 1, 0, 1, 0]], dtype=np.float32)
    for fold in ("up", "down"):
        assert oracle.rowsum(dict(leaf_w=2, leaf_layout="strided", lane_fold=fold), X)[0] == 0.0
    assert oracle.rowsum(dict(leaf_w=3), X)[0] == 2.0


def test_strided_special_cases():
    """One lane is plain sequential accumulation; as many lanes as elements is
    the butterfly over the elements; small integers are exact in every order."""
    X = inputs.lognormal_f32(5, (5, 300))
    for fold in ("up", "down"):
        one = oracle.rowsum(dict(leaf_w=1, leaf_layout="strided", lane_fold=fold), X)
        for r in range(5):
            assert one[r] == np.add.accumulate(X[r], dtype=np.float32)[-1]
    Y = X[:, :200]
    for fold, down in (("up", False), ("down", True)):
        got = oracle.rowsum(dict(leaf_w=256, leaf_layout="strided", lane_fold=fold), Y)
        for r in range(5):
            assert got[r].view(np.uint32) == _butterfly(list(Y[r]) + [None] * 56, down).view(np.uint32)
    # each lane a sequential chain over its own elements, then the butterfly
    for W in (2, 8, 64):
        for fold, down in (("up", False), ("down", True)):
            got = oracle.rowsum(dict(leaf_w=W, leaf_layout="strided", lane_fold=fold), X)
            for r in range(5):
                lanes = [np.add.accumulate(X[r, j::W], dtype=np.float32)[-1] for j in range(W)]
                assert got[r].view(np.uint32) == _butterfly(lanes, down).view(np.uint32), (W, fold)
    Z = np.random.default_rng(6).integers(-1000, 1000, (4, 777)).astype(np.float32)
    for W in (1, 4, 32, 64, 256):
        for fold in ("up", "down"):
            got = oracle.rowsum(dict(leaf_w=W, leaf_layout="strided", lane_fold=fold), Z)
            assert got.tolist() == Z.sum(1, dtype=np.float64).tolist()


# ------------------------------------------- structural identities of order


def _spread(seed, M=3, K=576, N=4):
    return inputs.spread_bf16(seed, (M, K)), inputs.spread_bf16(seed + 1, (K, N))


@pytest.mark.parametrize("model,g", [("exact", 16), ("gfx950", 32), ("gfx950", 16)])
def test_tiles_of_one_group_seq_equals_carry_without_fma(model, g):
    """Closing every tile after one group and chaining the tiles is the same
    tree as carrying the accumulator with the group rounded on its own."""
    A, B = _spread(21)
    kw = dict(model=model, g=g) if model == "exact" else dict(model=model, mma={32: "16x16x32", 16: "32x32x16"}[g])
    c1 = oracle.gemm(dict(kw, tile_k=g, tile_combine="seq", fma=1), A, B)
    c2 = oracle.gemm(dict(kw, tile_k=g, tile_combine="carry", fma=0), A, B)
    assert np.array_equal(c1.view(np.uint32), c2.view(np.uint32))


def test_single_tile_tree_and_seq_equal_carry():
    A, B = _spread(22)
    base = oracle.gemm(dict(tile_k=576), A, B)
    for tc in ("seq", "tree"):
        assert np.array_equal(oracle.gemm(dict(tile_k=576, tile_combine=tc), A, B).view(np.uint32),
                              base.view(np.uint32))


def test_fma_on_ignores_instruction_shape_on_gfx950():
    """With the accumulator carried through every chunk, the 16x16x32 and
    32x32x16 instructions (groups of 32 and 16) fold the same 8-product chunks
    in the same order."""
    A, B = _spread(23)
    for tc in ("carry", "tree"):
        c1 = oracle.gemm(dict(mma="16x16x32", tile_k=64, tile_combine=tc), A, B)
        c2 = oracle.gemm(dict(mma="32x32x16", tile_k=64, tile_combine=tc), A, B)
        assert np.array_equal(c1.view(np.uint32), c2.view(np.uint32))
    # ... but not with fma = 0, where the instruction's group is rounded alone
    c1 = oracle.gemm(dict(mma="16x16x32", tile_k=64, fma=0), A, B)
    c2 = oracle.gemm(dict(mma="32x32x16", tile_k=64, fma=0), A, B)
    assert not np.array_equal(c1.view(np.uint32), c2.view(np.uint32))


def test_explicit_cuts_equal_span_rule_and_tail_position():
    A, B = _spread(24)
    d = dict(tile_k=64, split_k=3)
    assert np.array_equal(oracle.gemm(d, A, B).view(np.uint32),
                          oracle.gemm(dict(d, k_cuts=[192, 384]), A, B).view(np.uint32))
    # K a multiple of tile_k: the short-tile position is moot
    assert np.array_equal(oracle.gemm(dict(d, tail="first"), A, B).view(np.uint32),
                          oracle.gemm(d, A, B).view(np.uint32))
    # a 40-element tail inside each tree-combined part changes the tree
    A2, B2 = _spread(25, K=3 * 232)
    d2 = dict(d, k_cuts=[232, 464], tile_combine="tree")
    t1 = oracle.gemm(d2, A2, B2)
    t2 = oracle.gemm(dict(d2, tail="first"), A2, B2)
    assert not np.array_equal(t1.view(np.uint32), t2.view(np.uint32))


def test_merge_trees_of_two_and_three_are_chains():
    """A balanced tree over 2 or 3 parts is the sequential chain; over 4 it
    is not."""
    A, B = _spread(26, K=768, N=16)
    for S in (2, 3):
        seq = oracle.gemm(dict(tile_k=64, split_k=S), A, B)
        tre = oracle.gemm(dict(tile_k=64, split_k=S, split_combine="tree"), A, B)
        assert np.array_equal(seq.view(np.uint32), tre.view(np.uint32))
    seq = oracle.gemm(dict(tile_k=64, split_k=4), A, B)
    tre = oracle.gemm(dict(tile_k=64, split_k=4, split_combine="tree"), A, B)
    assert not np.array_equal(seq.view(np.uint32), tre.view(np.uint32))


def test_rows_do_not_depend_on_M():
    """Each output follows its own order: the rows of a 7-row product equal
    the first 7 rows of a 64-row product (batch invariance is structural)."""
    A, B = _spread(27, M=64, K=256, N=8)
    full = oracle.gemm(dict(tile_k=64, out="bf16"), A, B)
    part = oracle.gemm(dict(tile_k=64, out="bf16"), A[:7], B)
    assert np.array_equal(full[:7], part)
    at = oracle.gemm_at(dict(tile_k=64, out="bf16"), A, B, None, [0, 5, 63], [1, 7, 3])
    assert np.array_equal(inputs.f32_to_bf16_bits(at), full[[0, 5, 63], [1, 7, 3]])


# ------------------------------------------------------------ error bounds


def _bound_check(desc, A, B, bias=None, rel=2.0 ** -8):
    C = oracle.gemm(desc, A, B, bias)
    Af = inputs.bf16_bits_to_f32(A).astype(np.float64)
    Bf = inputs.bf16_bits_to_f32(B).astype(np.float64)
    ref = Af @ Bf
    mag = np.abs(Af) @ np.abs(Bf)
    Cf = inputs.bf16_bits_to_f32(C) if C.dtype == np.uint16 else C
    err = np.abs(Cf.astype(np.float64) - ref)
    assert np.all(err <= rel * mag), float(np.max(err / np.maximum(mag, 1e-300)))
    return err, mag


def test_error_bound_tiny_config():
    """|C - C_fp64| <= 2^-8 * sum|a_ik b_kj| for the tiny descriptor, and the
    fp32 result is far tighter: one rounding per chunk update and merge."""
    A, B = inputs.tiny(0)
    desc = dict(mma="16x16x32", tile_k=32, split_k=2, tile_combine="tree", split_combine="tree")
    _bound_check(desc, A, B)
    updates = 256 // 8 + 8 + 2
    _bound_check(desc, A, B, rel=(2.0 ** -20 + updates * 2.0 ** -23))
    As, Bs = inputs.tiny(0, spread=True)
    _bound_check(desc, As, Bs, rel=(2.0 ** -20 + updates * 2.0 ** -23))


def test_error_bound_bf16_output_sweep_rows():
    A = inputs.sweep_activations(1, rows=4)[:, :1024]
    B = inputs.sweep_weight(2)[:1024, :256]
    _bound_check(dict(tile_k=64, out="bf16"), A, B)


# ------------------------------------------------------------- epilogue


def test_exp_accuracy_dense_sweep():
    """Our binary32 exp stays within 2 ulp of the real exponential."""
    xs = np.concatenate([np.linspace(-103.9, 88.7, 60001, dtype=np.float32),
                         np.float32(np.random.default_rng(6).uniform(-20, 20, 20000))])
    worst = 0.0
    for x in xs:
        y = oracle.exp(x)
        t = math.exp(float(x))
        if t < 2.0 ** -126:
            ulp = 2.0 ** -149
        else:
            ulp = 2.0 ** (math.floor(math.log2(t)) - 23)
        worst = max(worst, abs(float(y) - t) / ulp)
    assert worst <= 2.0, worst
    assert oracle.exp(-200.0) == 0.0 and oracle.exp(200.0) == np.inf
    assert np.isnan(oracle.exp(np.nan))


def test_silu_accuracy():
    """z / (1 + exp(-z)) within 4 ulp of the real SiLU while exp(-z) is
    finite in binary32 (z > -88.7); below that 1 + exp(-z) overflows and the
    result is a zero whose distance to the true value is below 2^-120."""
    rng = np.random.default_rng(7)
    for z in np.concatenate([rng.standard_normal(5000) * 4, rng.uniform(-95, 90, 2000)]).astype(np.float32):
        t = float(z) / (1.0 + math.exp(-float(z)))
        y = float(oracle.silu(z))
        if z > -88.7:
            assert abs(y - t) <= 4 * 2.0 ** -24 * abs(t) + 2.0 ** -149, (z, y, t)
        else:
            assert y == 0.0 and abs(t) < 2.0 ** -120


def test_epilogue_rounding_points():
    """FINAL: one bf16 rounding of silu(y + bias).  PRE_ACT: the
    pre-activation is rounded to bf16 first (an unfused Linear -> SiLU
    pair).  Both equal the helpers applied to the fp32 GEMM result."""
    A, B = inputs.tiny(0)
    bias = inputs.normal_bf16(7, (64,), 0.5)
    y = oracle.gemm(dict(tile_k=64), A, B)
    fin = oracle.gemm(dict(tile_k=64, epilogue="bias_silu", out="bf16"), A, B, bias)
    pre = oracle.gemm(dict(tile_k=64, epilogue="bias_silu", out="bf16", epi_round="pre_act"), A, B, bias)
    bb = inputs.bf16_bits_to_f32(bias)
    for i in range(0, 16, 5):
        for j in range(0, 64, 9):
            z = np.float32(y[i, j] + bb[j])
            assert fin[i, j] == oracle.f32_to_bf16(oracle.silu(z))
            zr = inputs.bf16_bits_to_f32(np.array([oracle.f32_to_bf16(z)]))[0]
            assert pre[i, j] == oracle.f32_to_bf16(oracle.silu(zr))
    plain = oracle.gemm(dict(tile_k=64, epilogue="bias"), A, B, bias)
    assert np.array_equal(plain, (y + bb[None, :]).astype(np.float32))


# --------------------------------------- the gfx950 chunk model by hand


def _chunk(acc, prods):
    a = bits([p[0] for p in prods])
    b = bits([p[1] for p in prods])
    return oracle.chunk8(np.float32(acc), a, b)


def test_chunk_model_hand_examples():
    """Worked cases of the gfx950 chunk arithmetic, each derived by hand from
    its definition (anchor E = largest exponent sum, products truncated
    toward zero onto 2^(E-24), T floored onto 2^max(E-24, x(T)-31, -157),
    one RNE rounding)."""
    # window: +2^e - 2^e + 1 keeps the 1 exactly when 2^0 >= 2^(e-24)
    for e in range(0, 40):
        got = _chunk(0, [(2.0 ** e, 1), (-(2.0 ** e), 1), (1, 1)])
        assert got == (1.0 if e <= 24 else 0.0), e
    # the Sec. 4 pair absorbs r inside one chunk ...
    assert _chunk(0, [(2.0 ** -15, 1), (1024, 1), (-1024, 1)]) == 0.0
    # ... and r survives when the pair cancels in an earlier chunk
    a = bits([1024, -1024] + [0] * 6 + [2.0 ** -15] + [0] * 7)
    assert oracle.group_update(0, a, np.full(16, ONE), 16, 1) == np.float32(2.0 ** -15)
    # ties to even on the product sum, tail below the grid dropped
    assert _chunk(0, [(1, 1), (2.0 ** -24, 1)]) == 1.0
    assert _chunk(0, [(1, 1), (2.0 ** -23, 1), (2.0 ** -24, 1)]) == np.float32(1 + 2.0 ** -22)
    assert _chunk(0, [(1, 1), (2.0 ** -24, 1), (2.0 ** -30, 1)]) == 1.0
    # the result-relative grid 2^(x(T)-31) keeps a tail the product grid drops
    assert _chunk(1.0, [(2.0 ** -24, 1), (2.0 ** -30, 1)]) == np.float32(1 + 2.0 ** -23)
    assert _chunk(1.0, [(2.0 ** -24, 1), (2.0 ** -31, 1)]) == np.float32(1 + 2.0 ** -23)
    assert _chunk(1.0, [(2.0 ** -24, 1), (2.0 ** -32, 1)]) == 1.0
    # products truncate toward zero, the sum floors toward -inf
    assert _chunk(0, [(1, 1), (-(2.0 ** -24), 1), (-(2.0 ** -30), 1)]) == np.float32(1 - 2.0 ** -24)
    assert _chunk(-1.0, [(-(2.0 ** -24), 1), (-(2.0 ** -40), 1)]) == np.float32(-(1 + 2.0 ** -23))
    # a small accumulator is floored onto the product grid
    assert _chunk(-(2.0 ** -30), [(1, 1)]) == np.float32(1 - 2.0 ** -24)
    assert _chunk(2.0 ** -30, [(1, 1)]) == 1.0
    # exactly zero results are +0, even from -0 inputs
    z = _chunk(-0.0, [(-0.0, 1), (0.0, -1)])
    assert z == 0.0 and not np.signbit(z)
    # products of 2^128 overflow to infinity before they can cancel
    assert np.isnan(_chunk(0, [(2.0 ** 127, 2), (-(2.0 ** 127), 2), (1, 1)]))
    assert _chunk(0, [(2.0 ** 127, 1.9921875), (-(2.0 ** 127), 1.9921875), (2.0 ** 103, 1)]) == np.float32(2.0 ** 103)
    assert _chunk(0, [(2.0 ** 127, 1.9921875), (-(2.0 ** 127), 1.9921875), (2.0 ** 102, 1)]) == 0.0
    # subnormal bf16 factors anchor at exponent -126
    assert _chunk(0, [(2.0 ** -133, 2.0 ** 100), (1.5 * 2.0 ** -26, 2.0 ** -25)]) == np.float32(2.0 ** -33)
    # the grid never goes below 2^-157
    assert _chunk(0, [(2.0 ** -75, 2.0 ** -75), (2.0 ** -75, 2.0 ** -82)]) == np.float32(2.0 ** -149)
    assert _chunk(0, [(2.0 ** -75, 2.0 ** -75), (2.0 ** -75, 2.0 ** -83)]) == 0.0
    assert _chunk(0, [(-(2.0 ** -75), 2.0 ** -75), (-(2.0 ** -75), 2.0 ** -83)]) == np.float32(-(2.0 ** -149))


def test_chunk_model_equals_exact_when_window_holds_everything():
    """When every term of every chunk sits on the chunk's grid (integers with a
    narrow spread), the chunk model is the exact-group hypothesis with groups
    of 8."""
    rng = np.random.default_rng(8)
    A = bits(rng.integers(-64, 65, (4, 256)))
    B = bits(rng.integers(-64, 65, (256, 5)))
    c1 = oracle.gemm(dict(model="gfx950", tile_k=64), A, B)
    c2 = oracle.gemm(dict(model="exact", g=8, tile_k=64), A, B)
    assert np.array_equal(c1, c2)


# ------------------------------------------------ strided layout of the split
#
# Sec. 3.2.2 (GEMV): a cut may deal the axis to its parts in tiles, part s
# taking every S-th tile, instead of giving each part a contiguous slice; the
# descriptor records which (layout).  Part s is then every k whose tile index
# floor(k / split_tile) is s mod S, in increasing k.


def _walk_operands(vals, K=32):
    """Row vector a with the given {k: value} entries (zero elsewhere) and an
    all-ones column: the products are the a entries themselves."""
    a = np.zeros((1, K), np.float32)
    for k, v in vals.items():
        a[0, k] = v
    return bits(a), np.full((K, 1), ONE)


@pytest.mark.parametrize("model", ["exact", "gfx950"])
def test_strided_layout_hand_walk(model):
    """A cancelling pair L, -L and a small r: which partial each lands in
    decides whether r survives (worked by hand; L = 2^30, r = 1, so that
    L + r rounds back to L in binary32)."""
    L = 2.0 ** 30
    base = dict(model=model, g=8, tile_k=8)
    a, b = _walk_operands({0: L, 16: -L, 8: 1.0})
    # contiguous halves [0,16) [16,32): (L (+) 1) = L, then L (+) -L = 0
    assert oracle.gemm(dict(base, split_k=2), a, b)[0, 0] == 0.0
    # strided, tiles of 8: part 0 = k 0-7, 16-23 (L then -L: exact 0),
    # part 1 = k 8-15, 24-31 (= 1): 0 (+) 1 = 1
    st = dict(base, split_k=2, split_layout="strided", split_tile=8)
    assert oracle.gemm(st, a, b)[0, 0] == 1.0
    # four parts, one tile each: L, 1, -L, 1.  Chain: ((L (+) 1) (+) -L) (+) 1
    # = 0 (+) 1 = 1; tree: (L (+) 1) (+) (-L (+) 1) = L (+) -L = 0
    a, b = _walk_operands({0: L, 8: 1.0, 16: -L, 24: 1.0})
    st4 = dict(base, split_k=4, split_layout="strided", split_tile=8)
    assert oracle.gemm(dict(st4, split_combine="seq"), a, b)[0, 0] == 1.0
    assert oracle.gemm(dict(st4, split_combine="tree"), a, b)[0, 0] == 0.0


@pytest.mark.parametrize("S,w,tile_k,K", [(2, 64, 64, 1032), (4, 64, 32, 4096), (4, 128, 64, 4160),
                                          (3, 32, 32, 1000), (4, 64, 64, 100), (8, 32, 32, 40)])
def test_strided_small_integers_are_exact(S, w, tile_k, K):
    """Integer operands keep every order exact, so a dropped, repeated or
    misplaced k shows as a wrong integer -- including ragged K and parts
    left empty (K < S w), whose value is +0."""
    rng = np.random.default_rng(S * 1000 + K)
    Ai = rng.integers(-8, 9, (3, K))
    Bi = rng.integers(-8, 9, (K, 5))
    for comb in ("seq", "tree"):
        d = dict(tile_k=tile_k, split_k=S, split_layout="strided", split_tile=w, split_combine=comb)
        C = oracle.gemm(d, bits(Ai), bits(Bi))
        assert np.array_equal(C.astype(np.int64), Ai @ Bi)


def test_strided_parts_are_gathered_chains():
    """Each strided part equals the one-part product over its own k, taken in
    increasing order; the split's merge chains those parts in part order."""
    A, B = _spread(21, M=2, K=1100, N=3)
    S, w = 4, 64
    ks = np.arange(1100)
    parts = []
    for s in range(S):
        idx = ks[(ks // w) % S == s]
        parts.append(oracle.gemm(dict(tile_k=64), np.ascontiguousarray(A[:, idx]),
                                 np.ascontiguousarray(B[idx])))
    y = parts[0]
    for p in parts[1:]:
        y = (y + p).astype(np.float32)
    got = oracle.gemm(dict(tile_k=64, split_k=S, split_layout="strided", split_tile=w), A, B)
    assert np.array_equal(got.view(np.uint32), y.view(np.uint32))
    one = oracle.gemm(dict(tile_k=64, split_layout="strided", split_tile=w), A, B)
    assert np.array_equal(one.view(np.uint32), oracle.gemm(dict(tile_k=64), A, B).view(np.uint32))


def test_strided_layout_rejects_what_it_cannot_express():
    A, B = np.full((1, 64), ONE), np.full((64, 1), ONE)
    for bad in (dict(split_tile=48, tile_k=32), dict(split_tile=0), dict(k_cuts=[32], split_tile=32),
                dict(tail="first", split_tile=32)):
        d = dict(tile_k=32, split_k=2, split_layout="strided")
        d.update(bad)
        with pytest.raises(oracle.OracleError):
            oracle.gemm(d, A, B)


# ------------------------------------------------------ RMS normalisation


def test_rn32_sqrt_helper_matches_numpy():
    """The exact-comparison root used below against numpy's binary32 sqrt
    (correctly rounded) over values of every exponent."""
    rng = np.random.default_rng(29)
    v = (rng.uniform(1, 2, 3000) * np.exp2(rng.integers(-140, 120, 3000))).astype(np.float32)
    for x in v:
        assert rn32_sqrt(f(x)).view(np.uint32) == np.sqrt(x).view(np.uint32), x


def test_rmsnorm_hand_example():
    """Row [3, 4]: s = 9 + 16 = 25 and the mean 12.5 are exact; the root and
    the reciprocal are each the exact value rounded once (exact rationals);
    eps joins before the root."""
    X = np.array([[3.0, 4.0]], dtype=np.float32)
    for eps, v in ((0.0, Fraction(25, 2)), (0.5, Fraction(13))):
        Y, rinv = oracle.rmsnorm(dict(leaf_w=64), X, eps=eps, with_rinv=True)
        q = rn32_sqrt(v)
        r = rn32(1 / f(q))
        assert rinv[0].view(np.uint32) == r.view(np.uint32), eps
        assert Y[0, 0] == rn32(3 * f(r)) and Y[0, 1] == rn32(4 * f(r))


def test_rmsnorm_closed_forms():
    """Rows of +-2^e over a power-of-two width: mean square 4^e, root 2^e,
    so the normalised values are +-1 exactly and the output is +-w; with
    eps = 3 * 4^e the root doubles and the output is +-w/2."""
    rng = np.random.default_rng(23)
    for cols in (1, 2, 64, 256, 4096):
        for e in (-20, -3, 0, 7, 20):
            sign = rng.choice([-1.0, 1.0], (3, cols)).astype(np.float32)
            X = (sign * np.float32(2.0 ** e)).astype(np.float32)
            w = inputs.normal_bf16(cols + e + 100, (cols,), 1.0)
            wf = (w.astype(np.uint32) << 16).view(np.float32)
            for layout, lw in (("contiguous", 64), ("strided", 256), ("strided", 1)):
                d = dict(leaf_w=lw, leaf_layout=layout)
                assert np.array_equal(oracle.rmsnorm(d, X), sign), (cols, e, layout)
                assert np.array_equal(oracle.rmsnorm(d, X, w), sign * wf)
                assert np.array_equal(oracle.rmsnorm(d, X, w, eps=3 * 4.0 ** e), sign * wf / 2)
                assert np.array_equal(oracle.rmsnorm(dict(d, out="bf16"), X, w),
                                      np.where(sign > 0, w, w ^ 0x8000).astype(np.uint16))


def test_rmsnorm_within_fp64_bound():
    """Log-normal rows against float64: the sum of squares of positive terms
    carries a relative error below 70 * 2^-24 (leaf of 64 plus the tree over
    128 leaves), the mean, root and reciprocal three more roundings, the two
    products two more: everything well inside 2^-17 relative."""
    X = inputs.lognormal_f32(31, (64, 8192))
    w = inputs.normal_bf16(32, (8192,), 1.0)
    wf = (w.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    eps = 1e-6
    X64 = X.astype(np.float64)
    ref = X64 / np.sqrt((X64 ** 2).mean(1, keepdims=True) + np.float64(np.float32(eps))) * wf
    for d in (dict(leaf_w=64), dict(leaf_w=256, leaf_layout="strided", lane_fold="down"),
              dict(leaf_w=64, fma=0)):
        got = oracle.rmsnorm(d, X, w, eps=eps).astype(np.float64)
        assert np.all(np.abs(got - ref) <= 2.0 ** -17 * np.abs(ref) + 1e-38), d


def test_rmsnorm_follows_the_rowsum_order_and_rounding_points():
    """The reciprocal root is taken from exactly the row sum of squares the
    descriptor fixes (dg_rowsum's order), and the bf16 rounding sits before
    the weight multiply only when asked (norm_round = pre_weight); the
    element step recomputed with numpy binary32 products and torch's bf16
    conversion."""
    import torch
    X = inputs.lognormal_f32(33, (16, 1000))
    w = inputs.normal_bf16(34, (1000,), 1.0)
    wf = (w.astype(np.uint32) << 16).view(np.float32)
    d = dict(leaf_w=128, leaf_layout="strided", lane_fold="down", fma=0)
    s = oracle.rowsum(dict(d, reduce="sumsq"), X)
    Y, rinv = oracle.rmsnorm(d, X, w, eps=1e-5, with_rinv=True)
    for r in range(16):
        v = rn32(f(rn32(f(s[r]) / 1000)) + f(np.float32(1e-5)))
        assert rinv[r] == rn32(1 / f(rn32_sqrt(f(v))))
    y = (X * rinv[:, None]).astype(np.float32)
    assert np.array_equal(Y, (y * wf).astype(np.float32))
    bf = lambda a: torch.from_numpy(a).to(torch.bfloat16).float().numpy()
    P = oracle.rmsnorm(dict(d, norm_round="pre_weight"), X, w, eps=1e-5)
    assert np.array_equal(P, (bf(y) * wf).astype(np.float32))
    assert not np.array_equal(P, Y)
    Pb = oracle.rmsnorm(dict(d, norm_round="pre_weight", out="bf16"), X, w, eps=1e-5)
    want = torch.from_numpy((bf(y) * wf).astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy()
    assert np.array_equal(Pb.view(np.int16), want)


# ---------------------------------------------------------------- softmax


def test_softmax_closed_forms():
    """Constant rows: every shifted value is 0, exp(0) = 1, the sum is the
    width exactly and each output is 1/width (a power of two here); the
    shift by the maximum keeps rows of +-1000 finite."""
    for cols in (1, 2, 64, 256, 4096):
        for c in (-1000.0, -3.5, 0.0, 2.0, 1000.0):
            X = np.full((3, cols), c, dtype=np.float32)
            for d in (dict(leaf_w=64), dict(leaf_w=256, leaf_layout="strided", lane_fold="down")):
                got = oracle.softmax(d, X)
                assert np.all(got == np.float32(1.0 / cols)), (cols, c, d)
                gb = oracle.softmax(dict(d, out="bf16"), X)
                assert np.all(gb == inputs.f32_to_bf16_bits(np.float32(1.0 / cols))), (cols, c, d)


def test_softmax_steps_and_rounding_points():
    """Each row: the maximum, the oracle's exp of the exact-order shifted
    values, the row sum in the descriptor's order (dg_rowsum's value), one
    reciprocal, one product per element (not a division)."""
    X = inputs.lognormal_f32(61, (6, 300), sigma=1.0)
    for d in (dict(leaf_w=64), dict(leaf_w=32, leaf_layout="strided", lane_fold="down"),
              dict(leaf_w=1, leaf_layout="strided")):
        got = oracle.softmax(d, X)
        for r in range(6):
            m = X[r].max()
            e = np.array([oracle.exp(np.float32(x - m)) for x in X[r]], dtype=np.float32)
            s = oracle.rowsum(dict(d, reduce="sum"), e[None, :])[0]
            rinv = np.float32(np.float32(1.0) / s)
            assert np.array_equal(got[r], (e * rinv).astype(np.float32)), (d, r)
    # a reciprocal multiply and a division part ways somewhere on these rows
    e = np.array([oracle.exp(np.float32(x - X[0].max())) for x in X[0]], dtype=np.float32)
    s = oracle.rowsum(dict(leaf_w=64), e[None, :])[0]
    assert not np.array_equal((e * np.float32(np.float32(1.0) / s)).astype(np.float32), (e / s).astype(np.float32))


def test_softmax_within_fp64_bound():
    """Against float64: exp within 2 ulp, a sum of positive terms within
    70 * 2^-24 relative, the reciprocal and the product one rounding each."""
    X = inputs.lognormal_f32(62, (32, 8192), sigma=1.0)
    X64 = X.astype(np.float64)
    E = np.exp(X64 - X64.max(1, keepdims=True))
    ref = E / E.sum(1, keepdims=True)
    for d in (dict(leaf_w=64), dict(leaf_w=256, leaf_layout="strided", lane_fold="down")):
        got = oracle.softmax(d, X).astype(np.float64)
        assert np.all(np.abs(got - ref) <= 2.0 ** -17 * ref + 1e-45), d


def test_softmax_special_values():
    """IEEE cases: a NaN anywhere, or +inf (inf - inf), makes the row NaN;
    -inf entries get exactly 0 beside finite ones."""
    X = np.array([[1.0, np.nan, 2.0], [1.0, np.inf, 2.0], [0.0, -np.inf, 0.0]], dtype=np.float32)
    got = oracle.softmax(dict(leaf_w=64), X)
    assert np.all(np.isnan(got[0])) and np.all(np.isnan(got[1]))
    assert got[2].tolist() == [0.5, 0.0, 0.5]


# ----------------------------------------------------- layer normalisation


def test_layernorm_closed_forms():
    """Rows c + a, c - a, c + a, ... over a power-of-two width, a a power of
    two: the sum, mean c, centred values +-a, their squares and the variance
    a^2 are all exact, so the normalised values are +-1 and the output is
    +-w + b rounded once."""
    rng = np.random.default_rng(71)
    for cols in (2, 64, 256, 4096):
        for c, a in ((0.0, 1.0), (3.0, 0.25), (-1000.0, 8.0), (2.0 ** 20, 2.0 ** -3)):
            sign = np.tile(np.array([1.0, -1.0], dtype=np.float32), (3, cols // 2))
            X = (np.float32(c) + sign * np.float32(a)).astype(np.float32)
            w = inputs.normal_bf16(cols + 1, (cols,), 1.0)
            b = inputs.normal_bf16(cols + 2, (cols,), 1.0)
            wf, bf_ = inputs.bf16_bits_to_f32(w), inputs.bf16_bits_to_f32(b)
            for d in (dict(leaf_w=64), dict(leaf_w=256, leaf_layout="strided", lane_fold="down"), dict(leaf_w=1)):
                assert np.array_equal(oracle.layernorm(d, X), sign), (cols, c, a, d)
                want = (sign * wf + bf_).astype(np.float32)
                assert np.array_equal(oracle.layernorm(d, X, w, b), want), (cols, c, a, d)


def test_layernorm_steps_and_rounding_points():
    """Each row: the mean from the descriptor-ordered sum, the centred values,
    their descriptor-ordered sum of squares, IEEE sqrt and reciprocal, then
    the products and the bias; with pre_weight the normalised value is
    rounded to bf16 (torch's conversion) before the weight."""
    import torch
    X = (inputs.lognormal_f32(72, (6, 300), sigma=1.0) + 5).astype(np.float32)
    w = inputs.normal_bf16(73, (300,), 1.0)
    b = inputs.normal_bf16(74, (300,), 1.0)
    wf, bf_ = inputs.bf16_bits_to_f32(w), inputs.bf16_bits_to_f32(b)
    for d in (dict(leaf_w=64), dict(leaf_w=32, leaf_layout="strided", lane_fold="down", fma=0)):
        for nr in ("final", "pre_weight"):
            got = oracle.layernorm(dict(d, norm_round=nr), X, w, b, eps=1e-5)
            for r in range(6):
                s1 = oracle.rowsum(dict(d, reduce="sum"), X[r:r + 1])[0]
                mean = np.float32(s1 / np.float32(300))
                dd = (X[r] - mean).astype(np.float32)
                s2 = oracle.rowsum(dict(d, reduce="sumsq"), dd[None, :])[0]
                v = rn32(f(rn32(f(s2) / 300)) + f(np.float32(1e-5)))
                rinv = rn32(1 / f(rn32_sqrt(f(v))))
                y = (dd * rinv).astype(np.float32)
                if nr == "pre_weight":
                    y = torch.from_numpy(y).to(torch.bfloat16).float().numpy()
                want = ((y * wf).astype(np.float32) + bf_).astype(np.float32)
                assert np.array_equal(got[r], want), (d, nr, r)


def test_layernorm_within_fp64_bound():
    """Against float64 on rows with a large common offset (the centred form
    keeps the variance accurate)."""
    X = (inputs.lognormal_f32(75, (32, 4096), sigma=1.0) + 100).astype(np.float32)
    X64 = X.astype(np.float64)
    mu = X64.mean(1, keepdims=True)
    ref = (X64 - mu) / np.sqrt(((X64 - mu) ** 2).mean(1, keepdims=True) + np.float64(np.float32(1e-5)))
    for d in (dict(leaf_w=64), dict(leaf_w=256, leaf_layout="strided", lane_fold="down")):
        got = oracle.layernorm(d, X, eps=1e-5).astype(np.float64)
        assert np.all(np.abs(got - ref) <= 2.0 ** -12 * (np.abs(ref) + 1)), d


# ------------------------------------------------- GEMM column-sum epilogue


def test_colsum_is_the_tree_down_each_column():
    """The hand walk down a column ([2^24, 1, -2^24, 1]: count-up tree 1,
    where a chain gives 0 and the exact sum 2), bf16 outputs widened
    exactly, small integers exact, and recursive halving over -0 padding
    for any row count."""
    C = np.array([[2.0 ** 24], [1.0], [-2.0 ** 24], [1.0]], dtype=np.float32)
    assert oracle.colsum(C)[0] == 1.0
    rng = np.random.default_rng(81)
    Z = rng.integers(-1000, 1000, (777, 33)).astype(np.float32)
    assert oracle.colsum(Z).tolist() == Z.sum(0, dtype=np.float64).tolist()
    W = rng.integers(-250, 250, (777, 33)).astype(np.float32)      # bf16 holds these exactly
    assert oracle.colsum(inputs.f32_to_bf16_bits(W)).tolist() == W.sum(0, dtype=np.float64).tolist()
    X = inputs.lognormal_f32(82, (100, 5))
    got = oracle.colsum(X)
    for j in range(5):
        p = 128
        padded = np.concatenate([X[:, j], np.full(p - 100, -0.0, dtype=np.float32)])
        assert got[j].view(np.uint32) == _halving(padded).view(np.uint32)


# ------------------------------------- the scalar path: chained chunks


def _chained_chunks_rational(a, b, S, T, tile_combine, split_combine):
    """Sec. 3.2.2 chained chunks written out in exact rationals: K cut into S
    contiguous chunks by the span rule (span rounded up to whole sub-blocks),
    each chunk into sub-blocks of T from its start, each sub-block an FMA
    chain from +0 (one rounding per product), the sub-blocks chained or
    met in the balanced tree, the chunks chained or met in the tree."""
    K = len(a)
    span = -(-K // S)
    span = -(-span // T) * T
    def tree(v):
        while len(v) > 1:
            w = [rn32(f(v[2 * i]) + f(v[2 * i + 1])) for i in range(len(v) // 2)]
            if len(v) % 2:
                w.append(v[-1])
            v = w
        return v[0]
    def chain(v):
        s = v[0]
        for x in v[1:]:
            s = rn32(f(s) + f(x))
        return s
    parts = []
    for s in range(S):
        lo, hi = s * span, min((s + 1) * span, K)
        tiles = []
        acc = np.float32(0.0)
        for t0 in range(lo, hi, T):
            if tile_combine != "carry":
                acc = np.float32(0.0)
            for k in range(t0, min(t0 + T, hi)):
                acc = rn32(f(acc) + bf(a[k]) * bf(b[k]))
            tiles.append(acc)
        part = tiles[-1] if tile_combine == "carry" else (chain(tiles) if tile_combine == "seq" else tree(tiles))
        parts.append(part)
    return chain(parts) if split_combine == "seq" else tree(parts)


@pytest.mark.parametrize("S,T,tc,sc", [(1, 1024, "carry", "seq"), (4, 16, "seq", "tree"), (8, 8, "tree", "seq"),
                                       (3, 32, "tree", "tree"), (16, 1, "seq", "seq")])
def test_scalar_chained_chunks_match_rationals(S, T, tc, sc):
    """The descriptor with the scalar instruction (groups of one) against the
    chained-chunk walk in exact rationals, on exponent-spread operands."""
    K = 290
    A = inputs.spread_bf16(91, (2, K))
    B = inputs.spread_bf16(92, (K, 3))
    d = dict(mma="scalar", tile_k=T, split_k=S, tile_combine=tc, split_combine=sc)
    C = oracle.gemm(d, A, B)
    for i in range(2):
        for j in range(3):
            want = _chained_chunks_rational(A[i], B[:, j], S, T, tc, sc)
            assert C[i, j].view(np.uint32) == np.float32(want).view(np.uint32), (i, j)


# ------------------------------------- parts and merges at bf16 (Sec. 3.2.2)
#
# partial_dtype: a finished part is stored at bf16; merge_dtype: the running
# merge sum is held at bf16, so every merge addition is rounded to bf16.  For
# two bf16 addends RNbf(RN32(x + y)) = RNbf(x + y) (a sum whose addends are
# more than 16 binades apart lies far from any bf16 midpoint), so the walk
# below rounds each merge's exact sum straight to bf16.


def _split_bf16_rational(a, b, S, split_combine, partial_bf16, merge_bf16):
    """Split-K over the scalar instruction written out in exact rationals:
    parts of span ceil(K/S) (tile_k = 1), each an FMA chain from +0 (one
    binary32 rounding per product), each part value rounded to bf16 when
    partial_bf16, the parts chained or met in the balanced tree with every
    merge addition rounded to bf16 when merge_bf16 (else to binary32)."""
    K = len(a)
    span = -(-K // S)
    parts = []
    for s in range(S):
        acc = Fraction(0)
        for k in range(s * span, min((s + 1) * span, K)):
            acc = f(rn32(acc + bf(a[k]) * bf(b[k])))
        parts.append(rnbf(acc) if partial_bf16 else acc)
    add = (lambda x, y: rnbf(x + y)) if merge_bf16 else (lambda x, y: f(rn32(x + y)))
    if split_combine == "seq":
        y = parts[0]
        for v in parts[1:]:
            y = add(y, v)
        return y
    while len(parts) > 1:
        nxt = [add(parts[2 * i], parts[2 * i + 1]) for i in range(len(parts) // 2)]
        if len(parts) % 2:
            nxt.append(parts[-1])
        parts = nxt
    return parts[0]


@pytest.mark.parametrize("S,sc,partial,merge", [(4, "seq", "bf16", "bf16"), (4, "tree", "bf16", "bf16"),
                                                (5, "seq", "bf16", "f32"), (7, "tree", "bf16", "bf16"),
                                                (8, "tree", "bf16", "f32"), (3, "seq", "f32", "f32")])
def test_bf16_parts_and_merges_match_rationals(S, sc, partial, merge):
    """Parts and merges at bf16 against the exact-rational walk, on normal
    and exponent-spread operands (the scalar instruction, so the parts are
    plain FMA chains)."""
    K = 210
    for A, B in ((bits(np.random.default_rng(41).standard_normal((3, K))),
                  bits(np.random.default_rng(42).standard_normal((K, 4)))),
                 (inputs.spread_bf16(43, (3, K)), inputs.spread_bf16(44, (K, 4)))):
        d = dict(mma="scalar", tile_k=1, split_k=S, split_combine=sc, partial=partial, merge=merge)
        C = oracle.gemm(d, A, B)
        for i in range(3):
            for j in range(4):
                want = _split_bf16_rational(A[i], B[:, j], S, sc, partial == "bf16", merge == "bf16")
                assert C[i, j].view(np.uint32) == np.float32(float(want)).view(np.uint32), (i, j)


def test_bf16_parts_and_merges_hand_examples():
    """Cases worked by hand where the bf16 rounding of a part or of a merge
    decides the result (bf16 keeps 8 significant bits: 1 + 2^-8 is a tie and
    goes to 1, 1 + 2^-7 is exact)."""
    one = dict(mma="scalar", tile_k=1)
    # four parts of one product each: 1, 2^-8, 2^-8, 2^-8
    A = bits([[1.0, 2.0 ** -8, 2.0 ** -8, 2.0 ** -8]])
    B = bits(np.ones((4, 1)))
    want = {("seq", "f32"): 1 + 3 * 2.0 ** -8,     # binary32 holds the sum
            ("tree", "f32"): 1 + 3 * 2.0 ** -8,
            ("seq", "bf16"): 1.0,                  # (1 + 2^-8) ties to 1, twice
            ("tree", "bf16"): 1 + 2.0 ** -7}       # 1 + 2^-8 -> 1; 2^-8 + 2^-8 = 2^-7; 1 + 2^-7 exact
    for (sc, merge), v in want.items():
        C = oracle.gemm(dict(one, split_k=4, split_combine=sc, partial="bf16", merge=merge), A, B)
        assert C[0, 0] == np.float32(v), (sc, merge, C[0, 0])
    # two parts: (1 + 2^-7)^2 = 1 + 2^-6 + 2^-14 and 2^-9
    A = bits([[1 + 2.0 ** -7, 1.0]])
    B = bits([[1 + 2.0 ** -7], [2.0 ** -9]])
    cases = {("f32", "f32"): 1 + 2.0 ** -6 + 2.0 ** -9 + 2.0 ** -14,
             ("bf16", "f32"): 1 + 2.0 ** -6 + 2.0 ** -9,   # the part loses its 2^-14
             ("bf16", "bf16"): 1 + 2.0 ** -6}              # and the merge its 2^-9
    for (partial, merge), v in cases.items():
        C = oracle.gemm(dict(one, split_k=2, partial=partial, merge=merge), A, B)
        assert C[0, 0] == np.float32(v), (partial, merge, C[0, 0])
    # the gfx950 instruction path takes the same part and merge roundings
    g = dict(model="gfx950", mma="16x16x32", tile_k=32, split_k=2, partial="bf16", merge="bf16")
    A = np.zeros((1, 64), dtype=np.uint16)
    B = np.zeros((64, 1), dtype=np.uint16)
    A[0, 0], B[0, 0] = bits(1 + 2.0 ** -7), bits(1 + 2.0 ** -7)
    A[0, 32], B[32, 0] = bits(1.0), bits(2.0 ** -9)
    assert oracle.gemm(g, A, B)[0, 0] == np.float32(1 + 2.0 ** -6)
    assert oracle.gemm(dict(g, merge="f32"), A, B)[0, 0] == np.float32(1 + 2.0 ** -6 + 2.0 ** -9)


# ------------------------------------------------- binary16 operands
#
# The fp16 MFMAs (v_mfma_f32_16x16x32_f16, 32x32x16_f16) fold their chunks by
# the same rules, with exponents read from the binary16 fields.


def h16(x):
    """Values -> binary16 bits (numpy's conversion, exact for the values used)."""
    return np.asarray(x, dtype=np.float16).view(np.uint16)


def test_f16_decoding_matches_numpy_on_every_pattern():
    """The oracle's binary16 decoding against numpy's float16 -> float32
    conversion on all 65536 bit patterns (NaNs compared as a class)."""
    hs = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    want = hs.view(np.float16).astype(np.float32)
    got = np.array([oracle.f16_to_f32(h) for h in hs], dtype=np.float32)
    nan = np.isnan(want)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan].view(np.uint32), want[~nan].view(np.uint32))


def test_f16_exact_dot_is_the_rational_sum_rounded_once():
    """exact_dot_rn32 on binary16 operands against the rational sum of the
    same values (numpy's float16 values as Fractions) rounded once."""
    rng = np.random.default_rng(16)
    for _ in range(200):
        n = int(rng.integers(1, 33))
        a = h16(rng.choice([-1, 1], n) * (1 + rng.random(n)) * np.exp2(rng.integers(-24, 15, n)))
        b = h16(rng.choice([-1, 1], n) * (1 + rng.random(n)) * np.exp2(rng.integers(-24, 15, n)))
        c = np.float32(rng.standard_normal() * 2.0 ** int(rng.integers(-30, 30)))
        q = Fraction(float(c)) + sum(Fraction(float(x)) * Fraction(float(y))
                                     for x, y in zip(a.view(np.float16), b.view(np.float16)))
        got = oracle.exact_dot_rn32(c, a, b, in_dtype="f16")
        assert got.view(np.uint32) == rn32(q).view(np.uint32) or (got == 0 and rn32(q) == 0)


def _chunk16(acc, prods):
    a = h16([p[0] for p in prods])
    b = h16([p[1] for p in prods])
    return oracle.chunk8(np.float32(acc), a, b, in_dtype="f16")


def test_f16_chunk_model_hand_examples():
    """Worked binary16 cases of the chunk rules, derived by hand: anchor E =
    the largest binary16 exponent sum (-14 for a subnormal factor), products
    truncated toward zero onto 2^(E-24), T floored onto 2^max(E-24, x(T)-31),
    one RNE rounding."""
    # a tie on the product sum: 1 + 2^-24 rounds to even; 2^-30 (a product of
    # two subnormal factors 2^-15) sits below the grid 2^-24 of anchor 0
    assert _chunk16(0, [(1, 1), (2.0 ** -12, 2.0 ** -12)]) == 1.0
    assert _chunk16(0, [(1, 1), (2.0 ** -12, 2.0 ** -12), (2.0 ** -15, 2.0 ** -15)]) == 1.0
    # ... whereas the exact sum rounds up
    a, b = h16([1, 2.0 ** -12, 2.0 ** -15]), h16([1, 2.0 ** -12, 2.0 ** -15])
    assert oracle.exact_dot_rn32(0, a, b, in_dtype="f16") == np.float32(1 + 2.0 ** -23)
    # the accumulator's own grid keeps a tail the product grid would drop
    assert _chunk16(1.0, [(2.0 ** -12, 2.0 ** -12), (2.0 ** -15, 2.0 ** -15)]) == np.float32(1 + 2.0 ** -23)
    # window: +2^e - 2^e + 1 keeps the 1 while 2^0 is on the grid 2^(e-24)
    for e in range(0, 31):
        ea, eb = min(e, 15), e - min(e, 15)
        got = _chunk16(0, [(2.0 ** ea, 2.0 ** eb), (-(2.0 ** ea), 2.0 ** eb), (1, 1)])
        assert got == (1.0 if e <= 24 else 0.0), e
    # products truncate toward zero, the sum floors toward -inf
    assert _chunk16(0, [(1, 1), (-(2.0 ** -12), 2.0 ** -12), (-(2.0 ** -15), 2.0 ** -15)]) == np.float32(1 - 2.0 ** -24)
    # a product of the largest binary16 values is finite
    assert _chunk16(0, [(65504, 65504)]) == np.float32(65504.0 * 65504.0)


def test_f16_chunk_model_equals_exact_when_window_holds_everything():
    """Integer binary16 operands of narrow spread: the chunk model is the
    exact-group model with groups of 8, and both equal the integer product."""
    rng = np.random.default_rng(9)
    Ai = rng.integers(-64, 65, (4, 256))
    Bi = rng.integers(-64, 65, (256, 5))
    c1 = oracle.gemm(dict(model="gfx950", tile_k=64, in_dtype="f16"), h16(Ai), h16(Bi))
    c2 = oracle.gemm(dict(model="exact", g=8, tile_k=64, in_dtype="f16"), h16(Ai), h16(Bi))
    assert np.array_equal(c1, c2)
    assert np.array_equal(c1, (Ai @ Bi).astype(np.float32))


@pytest.mark.parametrize("fma", [1, 0])
def test_f16_scalar_groups_are_a_binary32_chain(fma):
    """Groups of one with binary16 operands: each product is exact in binary32
    (22 significant bits), so the exact model is the binary32 chain acc + a*b,
    computed here with numpy float32 arithmetic (fma or not)."""
    rng = np.random.default_rng(11)
    a = h16(rng.standard_normal(300) * 3)
    b = h16(rng.standard_normal(300))
    acc = np.float32(0.0)
    for x, y in zip(a.view(np.float16).astype(np.float32), b.view(np.float16).astype(np.float32)):
        acc = np.float32(acc + np.float32(x * y))
    got = oracle.gemm(dict(model="exact", g=1, tile_k=300, fma=fma, in_dtype="f16"),
                      a.reshape(1, -1), b.reshape(-1, 1))
    assert got[0, 0].view(np.uint32) == acc.view(np.uint32)
