"""Pins of the oracle's gfx950 fp8 MFMA model (dgo_chunk16_e4m3; the fp8
instructions have their own semantics, Sec. 3.2.1) to facts other than its
own code (CPU only):

  * hand-worked chunks, each value derived on paper from the model's stated
    rules (group truncation onto 2^(E_g - 13), the chunk grid 2^(E - 24),
    the accumulator left out below 2^(E - 25), the result grid
    2^(x(T) - 31), one RNE rounding, the special values);
  * the Sec. 4 walk (+L, -L, r at every placement in one 32-k instruction)
    against the placement rule written out by hand in
    ``walk_prediction``;
  * exact rational arithmetic: where every term sits on the grids (narrow
    exponent spread) the model is the exact sum rounded once, and elsewhere
    it stays within the error the rules allow;
  * invariants: under fma = 1 the four fp8 instruction shapes give the same
    bits (the same chain of 16-k chunks);
  * planted mistakes: a transcription of the rules with one constant or one
    rounding direction changed fails these pins.
The model's agreement with the hardware itself is tests/test_gpu_fp8_mfma.py.
"""
import itertools
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2609_11356_amd import inputs
from tests.exact import rn32

FP8 = oracle.FP8_MMA


def val(code):
    return float(inputs.bf16_bits_to_f32(oracle.e4m3_to_bf16_bits(np.array([code], np.uint8)))[0])


def chunk(acc, prods):
    """prods: {k: (a code, b code)} within one 16-k chunk."""
    a = np.zeros(16, np.uint8)
    b = np.zeros(16, np.uint8)
    for k, (x, y) in prods.items():
        a[k], b[k] = x, y
    return oracle.chunk16_e4m3(np.float32(acc), a, b)


ONE, TWO, L8, NL8, R6, N448 = 0x38, 0x40, 0x78, 0xF8, 0x08, 0x7E
# (accumulator, products, expected): each worked by hand from the rules
HAND = [
    # one product is exact, the largest one too
    (0.0, {0: (N448, N448)}, 448.0 * 448.0),
    (0.0, {3: (0x01, 0x01)}, 2.0 ** -18),
    # inside a group, 2^-6 is truncated onto 2^(8 - 13): lost, also when negative
    (0.0, {0: (L8, ONE), 1: (R6, ONE)}, 256.0),
    (0.0, {0: (L8, ONE), 7: (R6 ^ 0x80, ONE)}, 256.0),
    # 2.25 x 1.125 = 81 x 2^-5 keeps its last bit, 2^(8 - 13), in the same group
    (0.0, {0: (L8, ONE), 1: (0x41, 0x39)}, 256.0 + 81.0 / 32.0),
    # in the other group of the chunk it is kept (the chunk grid is 2^-16)
    (0.0, {0: (L8, ONE), 8: (R6, ONE)}, 256.0 + 2.0 ** -6),
    # a group sum below the chunk grid is floored: -2^-17 becomes -2^-16, +2^-17 vanishes
    (0.0, {0: (L8, ONE), 8: (0x82, 0x01)}, 256.0 - 2.0 ** -16),
    (0.0, {0: (L8, ONE), 8: (0x02, 0x01)}, 256.0),
    # an accumulator below 2^(8 - 25) takes no part; at 2^-17 it is floored onto 2^-16
    (-(2.0 ** -18), {0: (L8, ONE)}, 256.0),
    (-(2.0 ** -17), {0: (L8, ONE)}, 256.0 - 2.0 ** -16),
    (2.0 ** -17, {0: (L8, ONE)}, 256.0),
    # ... and when the products cancel, a left-out accumulator gives +0
    (-(2.0 ** -18), {0: (L8, ONE), 9: (NL8, ONE)}, 0.0),
    (-(2.0 ** -17), {0: (L8, ONE), 9: (NL8, ONE)}, -(2.0 ** -16)),
    # the result grid 2^(x(T) - 31): 2^25 + 2 + 2^-18 is floored to the tie 2^25 + 2,
    # which rounds to even (exact rounding would give 2^25 + 4) ...
    (2.0 ** 25, {0: (TWO, ONE), 8: (0x01, 0x01)}, 2.0 ** 25),
    # ... while a tail on that grid (2^-6 >= 2^(25 - 31)) breaks the tie upward
    (2.0 ** 25, {0: (TWO, ONE), 8: (R6, ONE)}, 2.0 ** 25 + 4.0),
    # ... and one a bit below it (2^-7 < 2^(25 - 31)) does not
    (2.0 ** 25, {0: (TWO, ONE), 8: (R6, 0x30)}, 2.0 ** 25),
    # the chunk result is one RNE rounding of the floored sum
    (1.0, {0: (0x39, 0x39)}, 1.0 + 1.265625),
    (0.0, {0: (ONE, ONE), 8: (0x01, 0x01)}, 1.0 + 2.0 ** -18),
    # ties of the product sum itself: 2^24 + 1 rounds to even
    (2.0 ** 24, {0: (ONE, ONE)}, 2.0 ** 24),
    (2.0 ** 24, {0: (ONE, ONE), 8: (ONE, ONE), 1: (ONE, ONE)}, 2.0 ** 24 + 4.0),
    # zeros: no product leaves the accumulator (a -0 comes back +0); exact zero is +0
    (-0.0, {}, 0.0),
    (-0.0, {0: (0x80, ONE)}, 0.0),
    (-0.0, {0: (ONE, ONE), 1: (0xB8, ONE)}, 0.0),
    (-3.0, {}, -3.0),
    # special values
    (0.0, {0: (0x7F, ONE)}, np.nan),
    (0.0, {2: (0x7F, 0x00)}, np.nan),
    (1.0, {2: (0x00, 0xFF)}, np.nan),
    (np.nan, {}, np.nan),
    (np.inf, {0: (N448, N448)}, np.inf),
    (-np.inf, {}, -np.inf),
    (float(np.finfo(np.float32).max), {0: (N448, N448)}, float(np.finfo(np.float32).max)),
]


def same_bits(x, y):
    x, y = np.float32(x), np.float32(y)
    return (np.isnan(x) and np.isnan(y)) or x.view(np.uint32) == y.view(np.uint32)


@pytest.mark.parametrize("case", range(len(HAND)))
def test_hand_examples(case):
    acc, prods, want = HAND[case]
    assert same_bits(chunk(acc, prods), want), (acc, prods, chunk(acc, prods), want)


def walk_prediction(i, j, m, rv):
    """The model's value for +L (k = i), -L (k = j) and r (k = m) in one
    32-k instruction, L = 2^8 (anchor 8), r = rv far below it, the
    accumulator zero -- written out from the rules: r in a group of the
    pair is truncated onto 2^(8 - 13) (lost); r in a chunk with a member of
    the pair is floored onto 2^(8 - 24); a chunk's result is rounded to
    binary32; r in the chunk before the pair's becomes the accumulator and
    is left out of the pair's update when it lies below 2^(8 - 25), else
    floored onto 2^(8 - 24); r in the chunk after it stays as it is."""
    g = lambda k: k // 8
    c = lambda k: k // 16
    f32 = lambda x: float(np.float32(x))
    floor16 = np.floor(rv * 2.0 ** 16) / 2.0 ** 16
    if g(m) in (g(i), g(j)):
        return 0.0
    if c(i) == c(j):                   # the pair cancels within one chunk
        if c(m) == c(i):
            return floor16
        if c(m) > c(i):
            return rv
        return floor16 if abs(rv) >= 2.0 ** -17 else 0.0
    # the pair's members in different chunks, r beside one of them
    mine = 256.0 if c(m) == c(i) else -256.0
    if c(m) == 0:
        return f32(f32(mine + floor16) - mine)
    return floor16


WALK_R = [(0x08, 0x38), (0x82, 0x01), (0x81, 0x01)]       # 2^-6, -2^-17, -2^-18


def walk_operands(r):
    trips = list(itertools.permutations(range(32), 3))
    A = np.zeros((len(trips), 32), np.uint8)
    B = np.full((len(trips), 32), ONE, np.uint8)
    for c, (i, j, m) in enumerate(trips):
        A[c, i], A[c, j], A[c, m] = L8, NL8, r[0]
        B[c, m] = r[1]
    return trips, A, B


@pytest.mark.parametrize("r", WALK_R, ids=["2^-6", "-2^-17", "-2^-18"])
def test_walk_matches_the_placement_rule(r):
    trips, A, B = walk_operands(r)
    got = oracle.group_update_batch(np.zeros(len(trips)), A, B, 32, 1, in_dtype="e4m3")
    rv = val(r[0]) * val(r[1])
    want = np.array([walk_prediction(i, j, m, rv) for i, j, m in trips], np.float32)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


def exact_gemm(A, B):
    """Exact rational dot products of e4m3 codes, rounded once to binary32."""
    va = inputs.bf16_bits_to_f32(oracle.e4m3_to_bf16_bits(A)).astype(np.float64)
    vb = inputs.bf16_bits_to_f32(oracle.e4m3_to_bf16_bits(B)).astype(np.float64)
    out = np.zeros((A.shape[0], B.shape[1]), np.float32)
    for i in range(A.shape[0]):
        for j in range(B.shape[1]):
            out[i, j] = rn32(sum((Fraction(x) * Fraction(y) for x, y in zip(va[i], vb[:, j])), Fraction(0)))
    return out


@pytest.mark.parametrize("mma", FP8)
def test_equals_exact_when_the_grids_hold_everything(mma):
    """Operands with exponent fields in 6..9 and no subnormal: every product
    is an integer times 2^(E_max - 6 - 6), on every grid the model applies,
    and every partial sum too, so each output is the exact dot product
    rounded once (here exact, the sums staying below 2^24 units)."""
    rng = np.random.default_rng(3)
    K = 256
    A = (rng.integers(6, 10, (5, K)) << 3 | rng.integers(0, 8, (5, K)) | rng.integers(0, 2, (5, K)) << 7).astype(np.uint8)
    B = (rng.integers(6, 10, (K, 6)) << 3 | rng.integers(0, 8, (K, 6)) | rng.integers(0, 2, (K, 6)) << 7).astype(np.uint8)
    d = dict(mma=mma, in_dtype="e4m3", tile_k=128 if "128" in mma else 64)
    got = oracle.gemm(d, A, B)
    assert np.array_equal(got.view(np.uint32), exact_gemm(A, B).view(np.uint32))


def test_within_the_error_the_rules_allow():
    """Exponent-spread random chunks against the exact sum: each product
    loses less than 2^(E_g - 13), each group sum less than 2^(E - 24), a
    left-out accumulator less than 2^(E - 25), the result floor less than
    2^(x(T) - 31) and the rounding half a unit of binary32."""
    rng = np.random.default_rng(4)
    n = 3000
    a = inputs.e4m3_uniform(5, (n, 16))
    b = inputs.e4m3_uniform(6, (n, 16))
    acc = (rng.standard_normal(n) * np.exp2(rng.integers(-30, 30, n))).astype(np.float32)
    got = oracle.group_update_batch(acc, a, b, 16, 1, in_dtype="e4m3").astype(np.float64)
    va = inputs.bf16_bits_to_f32(oracle.e4m3_to_bf16_bits(a)).astype(np.float64)
    vb = inputs.bf16_bits_to_f32(oracle.e4m3_to_bf16_bits(b)).astype(np.float64)
    x = lambda c: np.where(((c >> 3) & 15) == 0, -6, ((c >> 3) & 15).astype(int) - 7)
    nz = ((a & 0x7F) != 0) & ((b & 0x7F) != 0)
    Ek = np.where(nz, x(a) + x(b), -999)
    Eg = np.stack([Ek[:, :8].max(1), Ek[:, 8:].max(1)], 1)
    E = Eg.max(1)
    exact = (va * vb).sum(1) + acc          # float64 is exact here: spread < 53 bits except the accumulator
    bound = (8 * np.exp2(Eg[:, 0] - 13.0) + 8 * np.exp2(Eg[:, 1] - 13.0) + 2 * np.exp2(E - 24.0) +
             np.exp2(E - 25.0) + np.abs(exact) * 2.0 ** -30 + np.abs(got) * 2.0 ** -24 + 2.0 ** -60 * np.abs(acc))
    ok = np.abs(got - exact) <= bound
    assert ok.all(), np.flatnonzero(~ok)[:5]


def test_fma_on_ignores_the_instruction_shape():
    """Under fma = 1 every fp8 instruction is the same chain of 16-k chunks,
    so the four shapes give the same bits (tile_k a multiple of all four
    instruction widths)."""
    A = inputs.e4m3_uniform(7, (4, 640))
    B = inputs.e4m3_uniform(8, (640, 5))
    outs = [oracle.gemm(dict(mma=m, in_dtype="e4m3", tile_k=128), A, B) for m in FP8]
    for o in outs[1:]:
        assert np.array_equal(o.view(np.uint32), outs[0].view(np.uint32))
    # with fma = 0 the group width shows: 16-k groups from zero differ from 128-k ones
    g16 = oracle.gemm(dict(mma="32x32x16_fp8", in_dtype="e4m3", tile_k=128, fma=0), A, B)
    g128 = oracle.gemm(dict(mma="16x16x128_f8f6f4", in_dtype="e4m3", tile_k=128, fma=0), A, B)
    assert not np.array_equal(g16.view(np.uint32), g128.view(np.uint32))


def test_descriptors_pair_operands_and_instructions():
    with pytest.raises(ValueError):
        oracle.params(dict(in_dtype="e4m3"))                       # a bf16 instruction
    with pytest.raises(ValueError):
        oracle.params(dict(mma="16x16x32_fp8"))                    # bf16 operands
    p, _ = oracle.params(dict(mma="16x16x128_f8f6f4", in_dtype="e4m3", tile_k=128))
    assert p.g == 128 and p.in_f16 == 2


# ------------------------------------------------------ planted mistakes


def rules(acc, a, b, GW=13, W=24, F=31, DROP=25, CW=16, GROUP_FLOOR=True, ACC_RULE=True):
    """The rules transcribed with exact rationals, one chunk of CW products
    (groups of 8), for planting mistakes (GW, W, F, DROP the grid offsets)."""
    a, b = [int(c) for c in a], [int(c) for c in b]
    if np.isnan(acc) or any((c & 0x7F) == 0x7F for c in list(a) + list(b)):
        return np.float32(np.nan)
    if np.isinf(acc):
        return np.float32(acc)
    x = lambda c: -6 if ((c >> 3) & 15) == 0 else ((c >> 3) & 15) - 7
    prods = [(Fraction(val(p)) * Fraction(val(q)), x(p) + x(q), t // 8)
             for t, (p, q) in enumerate(zip(a, b)) if (p & 0x7F) and (q & 0x7F)]
    if not prods:
        return np.float32(0.0) if acc == 0 else np.float32(acc)
    def onto(v, e, down):
        q = Fraction(2) ** e
        n = v / q
        i = n.numerator // n.denominator if down or v >= 0 else -((-n.numerator) // n.denominator)
        return i * q
    E = max(e for _, e, _ in prods)
    S = Fraction(0)
    for g in sorted(set(g for _, _, g in prods)):
        Eg = max(e for _, e, gg in prods if gg == g)
        T = sum((onto(p, Eg - GW, False) for p, _, gg in prods if gg == g), Fraction(0))
        S += onto(T, E - W, GROUP_FLOOR)
    A = Fraction(float(acc))
    if ACC_RULE and A != 0 and abs(A) < Fraction(2) ** (E - DROP):
        A = Fraction(0)
    T = S + A
    if T == 0:
        return np.float32(0.0)
    from tests.exact import ilog2
    T = onto(T, max(E - W, ilog2(T) - F), True)
    r = rn32(T)
    return np.float32(0.0) if r == 0 else r


def rules_walk(r, **kw):
    """The walk through the transcribed rules: two 16-k chunks in order."""
    trips, A, B = walk_operands(r)
    cw = kw.get("CW", 16)
    out = []
    for c in range(0, len(trips), 97):                 # a spread sample of the placements
        acc = np.float32(0.0)
        for s in range(0, 32, cw):
            acc = rules(acc, A[c, s:s + cw], B[c, s:s + cw], **kw)
        out.append((trips[c], acc))
    return out


def fails_a_pin(**kw):
    for acc, prods, want in HAND:
        a = np.zeros(16, np.uint8)
        b = np.zeros(16, np.uint8)
        for k, (p, q) in prods.items():
            a[k], b[k] = p, q
        if kw.get("CW", 16) == 16:
            got = rules(np.float32(acc), a, b, **kw)
        else:
            got = np.float32(acc)
            for s in range(0, 16, kw["CW"]):
                got = rules(got, a[s:s + kw["CW"]], b[s:s + kw["CW"]], **kw)
        if not same_bits(got, want):
            return True
    for r in WALK_R:
        rv = val(r[0]) * val(r[1])
        for (i, j, m), got in rules_walk(r, **kw):
            if not same_bits(got, walk_prediction(i, j, m, rv)):
                return True
    return False


def test_transcription_is_faithful():
    """The transcription with the model's constants reproduces the C oracle
    on random exponent-spread chunks and passes every pin."""
    rng = np.random.default_rng(9)
    a = inputs.e4m3_uniform(10, (400, 16))
    b = inputs.e4m3_uniform(11, (400, 16))
    acc = (rng.standard_normal(400) * np.exp2(rng.integers(-30, 20, 400))).astype(np.float32)
    for t in range(400):
        assert same_bits(rules(acc[t], a[t], b[t]), oracle.chunk16_e4m3(acc[t], a[t], b[t])), t
    assert not fails_a_pin()


@pytest.mark.parametrize("mutant", [dict(GW=12), dict(GW=14), dict(W=23), dict(W=25), dict(F=30), dict(F=32),
                                    dict(DROP=24), dict(DROP=26), dict(CW=8), dict(GROUP_FLOOR=False),
                                    dict(ACC_RULE=False)], ids=str)
def test_planted_mistakes_fail_a_pin(mutant):
    assert fails_a_pin(**mutant)
