"""Pins of the CPU oracle's attention order (App. F) to facts other than
itself (CPU only).

* dgo_exp2, the base-two exponential both sides evaluate with the same fixed
  steps: within 2 ulp of 2^x in float64 over a dense sweep, exact on the
  integers, the special values and the underflow / overflow edges.
* The recurrence (key blocks, running maximum, rescale roundings, the block
  row-sum tree, bf16 narrowing of the probabilities, the two matrix
  multiplications' groups, the place of the final division, the causal split
  at the multiples of BLOCK_M) written out again in exact rationals with one
  rounding per step, against the oracle under the exact instruction model.
* Closed forms that hold for every descriptor: equal scores give the mean of
  the visible value rows; one dominant key returns its value row exactly.
* Invariances the reading implies: BLOCK_M does not enter an unmasked
  answer, nor a causal one when it is a multiple of the key block.
* The float64 attention bound.
"""
import itertools
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2609_11356_amd import inputs
from tests.exact import bf, f, rn32, rnbf

MASK = np.float32(-1.0e6)


# ------------------------------------------------------------------- exp2


def _ulps(got, want64):
    """Distance in binary32 ulps of want64 (float64) from got (float32)."""
    w = np.float32(want64)
    ulp = np.spacing(np.abs(w)).astype(np.float64)
    return np.abs(got.astype(np.float64) - want64) / ulp


def test_exp2_accuracy_dense_sweep():
    """Within 2 ulp of 2^x (float64) over the normal-result range, and on
    every binary32 input of [-1, -1/2) and [1/2, 1)."""
    x = np.linspace(-125.0, 127.9, 5001).astype(np.float32)
    got = np.array([oracle.exp2(v) for v in x], dtype=np.float32)
    assert np.max(_ulps(got, np.exp2(x.astype(np.float64)))) <= 2.0
    for lo in (np.float32(0.5), np.float32(-1.0)):
        start = int(lo.view(np.uint32))
        xs = (np.arange(1 << 23, dtype=np.uint64) + start).astype(np.uint32).view(np.float32)
        got = oracle.exp2_range(start, 1 << 23)
        assert np.max(_ulps(got, np.exp2(xs.astype(np.float64)))) <= 2.0


def test_exp2_exact_points_and_edges():
    for n in range(-149, 128):
        assert oracle.exp2(float(n)) == np.float32(2.0 ** n), n
    assert oracle.exp2(0.0) == 1.0 and oracle.exp2(-0.0) == 1.0
    assert oracle.exp2(float("inf")) == np.inf and oracle.exp2(float("-inf")) == 0.0
    assert np.isnan(oracle.exp2(float("nan")))
    assert oracle.exp2(128.0) == np.inf and oracle.exp2(-151.5) == 0.0
    # the subnormal results are the correctly rounded 2^x (the scaling rounds once)
    for x in (-149.4, -149.6, -140.3, -126.5, -127.01):
        x = np.float32(x)
        want = np.float32(2.0 ** float(x))
        assert abs(int(oracle.exp2(x).view(np.uint32)) - int(want.view(np.uint32))) <= 1, x


def test_exp2_range_matches_scalar():
    start = int(np.float32(-3.0).view(np.uint32))
    got = oracle.exp2_range(start, 5000)
    want = np.array([oracle.exp2(np.uint32(start + i).view(np.float32)) for i in range(5000)], np.float32)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


# ------------------------------------------------- the recurrence, in rationals


def _blocks(desc, i, Lk):
    w = desc["key_block"]
    if not desc.get("causal"):
        return [(t, min(t + w, Lk), False) for t in range(0, Lk, w)]
    bm = desc["q_block"]
    q0 = i // bm * bm
    q1 = min(q0 + bm, Lk)
    return ([(t, min(t + w, q0), False) for t in range(0, q0, w)] +
            [(t, min(t + w, q1), True) for t in range(q0, q1, w)])


def _tree(vals):
    v = list(vals)
    while len(v) > 1:
        nxt = [rn32(f(v[2 * k]) + f(v[2 * k + 1])) for k in range(len(v) // 2)]
        if len(v) % 2:
            nxt.append(v[-1])
        v = nxt
    return v[0]


def _chain(vals):
    s = vals[0]
    for x in vals[1:]:
        s = rn32(f(s) + f(x))
    return s


def _attn_row_rational(desc, q, K, V, i, scale):
    """One query row in exact rationals, one rounding per step, groups of 32
    products summed exactly and rounded once (the exact instruction model)."""
    Lk, d = K.shape
    m = None                      # None = minus infinity
    l = np.float32(0.0)
    O = [np.float32(0.0)] * d
    for kb, ke, masked in _blocks(desc, i, Lk):
        s = []
        for t in range(kb, ke):
            acc = np.float32(0.0)
            for c0 in range(0, d, 32):
                acc = rn32(f(acc) + sum(bf(q[c]) * bf(K[t, c]) for c in range(c0, min(c0 + 32, d))))
            v = rn32(f(acc) * f(scale))
            if masked and t > i:
                v = rn32(f(v) + f(MASK))
            s.append(v)
        mn = max(s) if m is None else max(m, max(s))
        alpha = np.float32(0.0) if m is None else oracle.exp2(rn32(f(m) - f(mn)))
        p = [oracle.exp2(rn32(f(x) - f(mn))) for x in s]
        rs = _tree(p) if desc["block_sum"] == "tree" else _chain(p)
        if desc["l_fma"]:
            l = rn32(f(alpha) * f(l) + f(rs))
        else:
            l = rn32(f(rn32(f(alpha) * f(l))) + f(rs))
        pb = [rnbf(f(x)) for x in p]          # narrowed before P.V
        n = ke - kb
        for c in range(d):
            base = rn32(f(alpha) * f(O[c]))
            acc = base if desc["pv_fma"] else np.float32(0.0)
            for u0 in range(0, n, 32):
                acc = rn32(f(acc) + sum(pb[u] * bf(V[kb + u, c]) for u in range(u0, min(u0 + 32, n))))
            O[c] = acc if desc["pv_fma"] else rn32(f(base) + f(acc))
        m = mn
    if desc["final"] == "recip":
        r = rn32(Fraction(1) / f(l))
        out = [rn32(f(o) * f(r)) for o in O]
    else:
        out = [rn32(f(o) / f(l)) for o in O]
    return np.array(out, dtype=np.float32)


DESCS = [dict(key_block=w, causal=c, q_block=bm, block_sum=bs, pv_fma=pf, l_fma=lf, final=fi, out="f32")
         for (w, c, bm), bs, pf, lf, fi in itertools.product(
             [(1, 0, 1), (3, 0, 1), (8, 0, 1), (4, 1, 4), (4, 1, 6), (3, 1, 2), (8, 1, 5), (32, 1, 32)],
             ["tree", "seq"], [1, 0], [0, 1], ["div", "recip"])]


@pytest.mark.parametrize("di", range(0, len(DESCS), 3))
def test_recurrence_matches_rationals(di):
    """The oracle (exact instruction model) against the walk in exact
    rationals on a small head: every descriptor field, ragged blocks, both
    causal splits."""
    desc = DESCS[di]
    rng = np.random.default_rng(700 + di)
    Lk, d = 13, 40
    Q = inputs.normal_bf16(int(rng.integers(1 << 30)), (1, Lk, d), 0.6)
    K = inputs.normal_bf16(int(rng.integers(1 << 30)), (1, Lk, d), 0.6)
    V = inputs.spread_bf16(int(rng.integers(1 << 30)), (1, Lk, d), -6, 6)
    scale = np.float32(0.9)
    got = oracle.attention(dict(desc, model="exact"), Q, K, V, scale)
    rows = range(Lk) if desc["causal"] else (0, 6, 12)
    for i in rows:
        want = _attn_row_rational(desc, Q[0, i], K[0], V[0], i, scale)
        assert np.array_equal(got[0, i].view(np.uint32), want.view(np.uint32)), (desc, i)


def test_recurrence_bf16_output_and_wide_head():
    desc = dict(key_block=16, causal=1, q_block=24, block_sum="tree", pv_fma=1, l_fma=0, final="div", out="bf16")
    Lk, d = 40, 72
    Q = inputs.normal_bf16(31, (1, Lk, d), 0.3)
    K = inputs.normal_bf16(32, (1, Lk, d), 0.3)
    V = inputs.normal_bf16(33, (1, Lk, d))
    got = oracle.attention(dict(desc, model="exact"), Q, K, V, np.float32(1.3))
    for i in (0, 17, 23, 24, 39):
        want = _attn_row_rational(dict(desc, out="f32"), Q[0, i], K[0], V[0], i, np.float32(1.3))
        assert np.array_equal(got[0, i], inputs.f32_to_bf16_bits(want)), i


# --------------------------------------------------------------- closed forms


ALL = [dict(key_block=w, causal=c, q_block=bm, block_sum=bs, pv_fma=pf, l_fma=lf, final=fi, out="f32")
       for (w, c, bm), bs, pf, lf, fi in itertools.product(
           [(1, 0, 1), (5, 0, 1), (64, 0, 1), (4, 1, 4), (8, 1, 12), (64, 1, 128)],
           ["tree", "seq"], [1, 0], [0, 1], ["div", "recip"])]


@pytest.mark.parametrize("di", range(0, len(ALL), 4))
def test_equal_scores_give_the_mean_of_the_visible_values(di):
    """K = 0 makes every score 0: every visible key gets p = 1 exactly, every
    rescale is exp2(0) = 1, masked keys underflow to 0, so the output is the
    sum of the visible value rows (exact for small integers) divided by their
    count: one correctly rounded division (or the rounded reciprocal times
    the sum)."""
    desc = ALL[di]
    Lk, d = 70, 24
    rng = np.random.default_rng(di)
    Q = inputs.normal_bf16(di + 1, (1, Lk, d))
    K = np.zeros((1, Lk, d), np.uint16)
    Vi = rng.integers(-20, 21, (Lk, d))
    V = inputs.f32_to_bf16_bits(Vi.astype(np.float32)).reshape(1, Lk, d)
    got = oracle.attention(dict(desc, model="gfx950"), Q, K, V, np.float32(0.7))[0]
    for i in range(Lk):
        n = i + 1 if desc["causal"] else Lk
        tot = Vi[:n].sum(axis=0)
        if desc["final"] == "div":
            want = [rn32(Fraction(int(t), n)) for t in tot]
        else:
            r = rn32(Fraction(1, n))
            want = [rn32(int(t) * f(r)) for t in tot]
        assert np.array_equal(got[i].view(np.uint32), np.array(want, np.float32).view(np.uint32)), i


@pytest.mark.parametrize("di", range(1, len(ALL), 4))
def test_one_dominant_key_returns_its_value_row(di):
    """One key whose score exceeds every other by 256 (base-two units): every
    other probability underflows to 0 and the dominant one is 1, whichever
    block it falls in, so the output is that key's value row exactly."""
    desc = ALL[di]
    Lk, d = 50, 16
    Q = np.zeros((1, Lk, d), np.uint16)
    K = np.zeros((1, Lk, d), np.uint16)
    SIXTEEN = np.uint16(0x4180)   # 16.0 as bf16
    Q[0, :, 0] = SIXTEEN
    V = inputs.normal_bf16(di + 3, (1, Lk, d))
    for star in (0, 13, 31, 49):
        K2 = K.copy()
        K2[0, star, 0] = SIXTEEN
        got = oracle.attention(dict(desc, model="gfx950"), Q, K2, V, np.float32(1.0))[0]
        rows = [i for i in range(Lk) if not desc["causal"] or i >= star]
        want = inputs.bf16_bits_to_f32(V[0, star])
        for i in rows:
            assert np.array_equal(got[i], want), (star, i)


def test_query_block_enters_only_causal_answers_off_the_key_grid():
    """Unmasked: BLOCK_M is not part of the arithmetic.  Causal with BLOCK_M a
    multiple of the key block: the masked stage's boundaries are multiples of
    the key block and the blocks it adds past a row's last visible key are
    exact identities (rescale exp2(0) = 1, zero probabilities), so BLOCK_M
    drops out.  Causal with BLOCK_M off that grid moves the boundaries."""
    Lk, d = 96, 32
    Q = inputs.normal_bf16(61, (2, Lk, d))
    K = inputs.normal_bf16(62, (2, Lk, d))
    V = inputs.normal_bf16(63, (2, Lk, d))
    base = dict(key_block=16, block_sum="tree", out="f32")
    un = [oracle.attention(dict(base, causal=0, q_block=bm), Q, K, V, 0.5) for bm in (1, 16, 48)]
    assert all(np.array_equal(un[0], u) for u in un[1:])
    ca = [oracle.attention(dict(base, causal=1, q_block=bm), Q, K, V, 0.5) for bm in (16, 32, 64)]
    assert all(np.array_equal(ca[0], c) for c in ca[1:])
    off = oracle.attention(dict(base, causal=1, q_block=24), Q, K, V, 0.5)
    assert not np.array_equal(ca[0], off)


def test_within_float64_bound():
    """|out - attention64| <= 2^-7 max|v| + 2^-7 |attention64| per element:
    the bf16 narrowing of each probability moves the weighted sum by at most
    2^-8 of sum p |v| (relative to sum p: 2^-8 max|v|), the binary32 steps
    and the exp2 (2 ulp) by far less."""
    H, L, d = 2, 96, 64
    Q = inputs.normal_bf16(71, (H, L, d))
    K = inputs.normal_bf16(72, (H, L, d))
    V = inputs.normal_bf16(73, (H, L, d))
    scale = np.float32(1.0 / math.sqrt(d) * math.log2(math.e))
    for causal in (0, 1):
        desc = dict(key_block=32, causal=causal, q_block=64, out="f32")
        got = oracle.attention(desc, Q, K, V, scale).astype(np.float64)
        q, k, v = (inputs.bf16_bits_to_f32(x).astype(np.float64) for x in (Q, K, V))
        s = np.einsum("hid,hjd->hij", q, k) * float(scale)
        if causal:
            s = np.where(np.tril(np.ones((L, L), bool)), s, -np.inf)
        p = np.exp2(s - s.max(-1, keepdims=True))
        ref = np.einsum("hij,hjd->hid", p / p.sum(-1, keepdims=True), v)
        vmax = np.abs(v).max(axis=1, keepdims=True)
        assert np.all(np.abs(got - ref) <= 2.0 ** -7 * vmax + 2.0 ** -7 * np.abs(ref))


def test_rows_routine_equals_full_routine():
    Q = inputs.normal_bf16(81, (3, 33, 16))
    K = inputs.normal_bf16(82, (3, 33, 16))
    V = inputs.normal_bf16(83, (3, 33, 16))
    desc = dict(key_block=8, causal=1, q_block=12, out="bf16")
    full = oracle.attention(desc, Q, K, V, 0.8)
    hh, ii = [0, 2, 1, 2], [0, 32, 11, 12]
    rows = oracle.attention_rows(desc, Q, K, V, 0.8, hh, ii)
    assert np.array_equal(inputs.f32_to_bf16_bits(rows), full[hh, ii])


def test_invalid_shapes_refused():
    Q = inputs.normal_bf16(1, (1, 4, 8))
    K = inputs.normal_bf16(2, (1, 5, 8))
    with pytest.raises(oracle.OracleError):
        oracle.attention(dict(causal=1), Q, K, K, 1.0)       # causal needs Lq = Lk
    with pytest.raises(oracle.OracleError):
        oracle.attention(dict(key_block=0), Q, K, K, 1.0)
