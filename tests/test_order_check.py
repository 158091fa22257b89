"""The static order checker (Sec. 6) on gfx950 assembly built here: the
wave-level sums of tests/checker/lane_trees.hip, compiled with hipcc to
assembly (no GPU), walked, and compared with trees written from their
definitions; kernels that share a signature give the same bits, and kernels
in different classes differ on some input (checked by evaluating the walked
trees in binary32 on the CPU)."""
import os
import shutil

import numpy as np
import pytest

from paper_2609_11356_amd import order_check as oc

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "checker", "lane_trees.hip")
Y0 = [(8, 0)]                       # y[0]: the second pointer argument, byte 0


@pytest.fixture(scope="module")
def asm():
    if not os.path.exists(oc.HIPCC) and shutil.which("hipcc") is None:
        pytest.skip("no hipcc")
    return oc.compile_asm(SRC)


def leaf(i):
    """The leaf of x[i] (x the first pointer argument, 4-byte elements)."""
    return oc.Node("load", leaf=repr(oc.Aff(4 * i, {"arg0": 1})))


def add(a, b):
    return oc.Node("add", [a, b])


def butterfly(steps, n=64):
    """Every lane's value after the butterfly steps (lane i adds lane i ^ m),
    from the definition of the count-up and count-down trees."""
    v = [leaf(i) for i in range(n)]
    for m in steps:
        v = [add(v[i], v[i ^ m]) for i in range(n)]
    return v


def root(asm, name, outputs=Y0):
    w = oc.Walk(asm, name)
    r = w.roots(outputs)
    assert len(r) == len(outputs), (name, r)
    return r


def test_functions_found(asm):
    fns = set(oc.functions(asm))
    assert {"up_library", "up_shfl", "up_four", "up_two", "up_reversed", "down_library", "down_shfl",
            "up_steps_swapped", "chain", "groups16", "rcp_then_up", "branch_on_data"} <= fns


def test_count_up_read_off_the_assembly_is_the_perfect_tree(asm):
    """The library's lane steps (DPP quad_perm, half-row and row mirrors,
    ds_swizzle, ds_bpermute) give every lane the perfect tree over x[0..63]
    in element order."""
    want = oc.canon(butterfly([1, 2, 4, 8, 16, 32])[0])
    w = oc.Walk(asm, "up_library")
    assert len(w.stores) == 64 and not w.opaque
    assert all(t == want for _, t in w.roots())


def test_count_down_and_chain_match_their_definitions(asm):
    assert root(asm, "down_library")[0][1] == oc.canon(butterfly([32, 16, 8, 4, 2, 1])[0])
    v = leaf(0)
    for i in range(1, 64):
        v = add(v, leaf(i))
    assert root(asm, "chain")[0][1] == oc.canon(v)


def test_groups_of_sixteen(asm):
    """tree_sum_lanes<4>: four roots, each the perfect tree over its group."""
    r = root(asm, "groups16", [(8, 4 * g) for g in range(4)])
    for g in range(4):
        v = [leaf(16 * g + i) for i in range(16)]
        for m in (1, 2, 4, 8):
            v = [add(v[i], v[i ^ m]) for i in range(16)]
        assert r[g][1] == oc.canon(v[0])


def test_layouts_of_one_tree_share_a_signature(asm):
    """One element per lane over 64 lanes (DPP steps or shuffles), two or four
    consecutive elements per lane folded in the lane first, or the lanes
    reading the elements in reverse: one logical tree, one signature."""
    sigs = {k: oc.Walk(asm, k).signature(Y0) for k in ("up_library", "up_shfl", "up_two", "up_four", "up_reversed")}
    assert len(set(sigs.values())) == 1, sigs


def test_classes(asm):
    names = ["up_library", "up_shfl", "up_four", "up_two", "up_reversed", "down_library", "down_shfl",
             "up_steps_swapped", "chain"]
    got = oc.classes({k: oc.Walk(asm, k).signature(Y0) for k in names})
    assert got == [["chain"], ["down_library", "down_shfl"], ["up_library", "up_shfl", "up_four", "up_two", "up_reversed"],
                   ["up_steps_swapped"]]


def evaluate(n, x, memo):
    """A walked tree in binary32 (numpy, one rounding per add)."""
    k = id(n)
    if k not in memo:
        if n.op == "load":
            memo[k] = x[int(n.leaf.split("+")[-1]) // 4]
        elif n.op == "add":
            memo[k] = np.float32(evaluate(n.kids[0], x, memo) + evaluate(n.kids[1], x, memo))
        else:
            raise AssertionError(n.op)
    return memo[k]


def test_the_classes_are_real(asm):
    """Trees in one class give equal bits on every draw; every pair of classes
    differs on some draw of exponent-spread binary32 inputs."""
    reps = {"up": "up_library", "down": "down_library", "swapped": "up_steps_swapped", "chain": "chain"}
    trees = {}
    for k, name in list(reps.items()) + [("up_four", "up_four"), ("up_reversed", "up_reversed")]:
        w = oc.Walk(asm, name)
        trees[k] = [n for a, n in sorted(w.stores.values(), key=lambda an: an[0].key()) if a.key() == oc.Aff(0, {"arg8": 1}).key()][0]
    rng = np.random.default_rng(3)
    differ = set()
    for _ in range(200):
        x = (rng.standard_normal(64) * np.exp2(rng.integers(-20, 20, 64))).astype(np.float32)
        out = {k: evaluate(t, x, {}) for k, t in trees.items()}
        assert out["up"].view(np.uint32) == out["up_four"].view(np.uint32) == out["up_reversed"].view(np.uint32)
        for a in reps:
            for b in reps:
                if a < b and out[a].view(np.uint32) != out[b].view(np.uint32):
                    differ.add((a, b))
    assert differ == {(a, b) for a in reps for b in reps if a < b}


def test_unmodelled_instruction_is_a_function_of_its_operands(asm):
    """v_rcp_f32 is not modelled: it becomes an uninterpreted node over each
    lane's own leaf, so the 64 leaves stay distinct and the tree keeps its
    shape."""
    w = oc.Walk(asm, "rcp_then_up")
    assert any("v_rcp_f32" in t for t in w.opaque)
    r = w.roots(Y0)[0][1]
    assert r.count("opaque[v_rcp_f32") == 64 and len({r.find("L(%r)" % repr(oc.Aff(4 * i, {"arg0": 1}))) for i in range(64)}) == 64
    assert oc.Walk(asm, "rcp_then_up").signature(Y0) != oc.Walk(asm, "up_library").signature(Y0)


def test_data_dependent_control_flow_is_refused(asm):
    with pytest.raises(oc.Unsupported):
        oc.Walk(asm, "branch_on_data")


def test_parser_pieces():
    assert oc.parse_line("\tv_add_f32_dpp v1, v1, v1 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf bound_ctrl:1") == \
        ("v_add_f32_dpp", ["v1", "v1", "v1"], ["quad_perm:[1,0,3,2]", "row_mask:0xf", "bank_mask:0xf", "bound_ctrl:1"])
    assert oc.parse_line("\tglobal_load_dword v1, v[2:3], off offset:252") == \
        ("global_load_dword", ["v1", "v[2:3]", "off"], ["offset:252"])
    assert oc.parse_line(".LBB2_3:") is None and oc.parse_line("\t; comment") is None
    # DPP and swizzle lane maps against their definitions
    assert [oc._dpp_src(["quad_perm:[1,0,3,2]"], l) for l in range(4)] == [1, 0, 3, 2]
    assert [oc._dpp_src(["row_mirror"], l) for l in (0, 5, 16, 31)] == [15, 10, 31, 16]
    assert [oc._dpp_src(["row_half_mirror"], l) for l in (0, 7, 8, 15)] == [7, 0, 15, 8]
    assert [oc._dpp_src(["row_ror:8"], l) for l in (0, 8, 17)] == [8, 0, 25]
    assert oc._dpp_src(["row_shr:1"], 16) is None and oc._dpp_src(["row_shr:1"], 17) == 16
    assert [oc._swizzle_src(["offset:swizzle(SWAP,16)"], l) for l in (0, 16, 33, 63)] == [16, 0, 49, 47]
    assert [oc._swizzle_src(["offset:0x401f"], l) for l in (0, 16, 33)] == [16, 0, 49]   # bit mode, xor 16
    assert [oc._swizzle_src(["offset:0x101f"], l) for l in (0, 4, 35)] == [4, 0, 39]     # bit mode, xor 4


def perfect(lo, n):
    """The perfect tree over x[lo .. lo + n) in element order."""
    v = [leaf(lo + i) for i in range(n)]
    while len(v) > 1:
        v = [add(v[2 * i], v[2 * i + 1]) for i in range(len(v) // 2)]
    return v[0]


def test_cross_wave_exchange_through_lds(asm):
    """Waves of one workgroup meet through LDS (a store, a barrier, a load:
    one exchange that combines nothing).  256 threads with one element each
    and 128 threads with two consecutive elements each reach the perfect tree
    over x[0..255] and share its signature; chaining the four wave sums is
    another tree."""
    a = oc.Walk(asm, "block_256", block=(256, 1, 1))
    b = oc.Walk(asm, "block_128x2", block=(128, 1, 1))
    c = oc.Walk(asm, "block_256_chain", block=(256, 1, 1))
    assert a.roots(Y0)[0][1] == oc.canon(perfect(0, 256))
    assert a.signature(Y0) == b.signature(Y0)
    chained = add(add(add(perfect(0, 64), perfect(64, 64)), perfect(128, 64)), perfect(192, 64))
    assert c.roots(Y0)[0][1] == oc.canon(chained)
    assert c.signature(Y0) != a.signature(Y0)
    # the two classes are real: some draw separates them
    y0 = oc.Aff(0, {"arg8": 1}).key()
    ta, tc = a.stores[y0][1], c.stores[y0][1]
    rng = np.random.default_rng(4)
    x = (rng.standard_normal((50, 256)) * np.exp2(rng.integers(-20, 20, (50, 256)))).astype(np.float32)
    assert any(evaluate(ta, r, {}).view(np.uint32) != evaluate(tc, r, {}).view(np.uint32) for r in x)


@pytest.mark.parametrize("n", [512, 448])
def test_loops_walked_for_a_bound_configuration(asm, n):
    """With n bound (the third argument, byte 16) the loops are walked
    exactly: lane l's chain x[l], x[l + 64], ... then the count-up tree.
    Unrolling the chain by two with one accumulator keeps the tree; two
    accumulators (even and odd steps) regroup it.  Unbound, the trip count
    is data and the walk refuses."""
    fold = oc.Walk(asm, "strided_fold", args={16: n})
    lanes = []
    for l in range(64):
        v = leaf(l)
        for k in range(l + 64, n, 64):
            v = add(v, leaf(k))
        lanes.append(v)
    for m in (1, 2, 4, 8, 16, 32):
        lanes = [add(lanes[i], lanes[i ^ m]) for i in range(64)]
    assert fold.roots(Y0)[0][1] == oc.canon(lanes[0])
    assert oc.Walk(asm, "strided_fold_unroll2", args={16: n}).signature(Y0) == fold.signature(Y0)
    two = oc.Walk(asm, "strided_fold_two_acc", args={16: n})
    assert two.signature(Y0) != fold.signature(Y0)
    y0 = oc.Aff(0, {"arg8": 1}).key()
    rng = np.random.default_rng(5)
    x = (rng.standard_normal((50, n)) * np.exp2(rng.integers(-20, 20, (50, n)))).astype(np.float32)
    assert any(evaluate(fold.stores[y0][1], r, {}).view(np.uint32) != evaluate(two.stores[y0][1], r, {}).view(np.uint32)
               for r in x)
    with pytest.raises(oc.Unsupported):
        oc.Walk(asm, "strided_fold")


def test_pruning_predicate(asm):
    """A search over ways of summing 512 elements keeps the configurations
    with the reference's signature: the one-accumulator chain and its unroll
    by two, not the two-accumulator variant or a count-down lane fold."""
    space = {"fold": ("strided_fold", {16: 512}), "fold_unroll2": ("strided_fold_unroll2", {16: 512}),
             "fold_two_acc": ("strided_fold_two_acc", {16: 512}), "up_library": ("up_library", None)}
    sigs = {k: oc.Walk(asm, name, args=args).signature(Y0) for k, (name, args) in space.items()}
    assert oc.prune(sigs, "fold") == ["fold", "fold_unroll2"]
    assert oc.prune(sigs, sigs["up_library"]) == ["up_library"]


@pytest.mark.parametrize("mutant", ["no_commutative_sort", "leaf_by_lane", "lds_store_lost", "swizzle_xor_ignored"])
def test_planted_checker_mistakes_change_an_answer(asm, monkeypatch, mutant):
    """Each plausible slip in the walk changes a result the tests above pin:
    the one-class answer for the count-up layouts, or a tree against its
    definition."""
    if mutant == "no_commutative_sort":
        monkeypatch.setattr(oc, "COMMUTATIVE", set())
    elif mutant == "leaf_by_lane":
        real = oc.Walk.leaf
        monkeypatch.setattr(oc.Walk, "leaf", lambda self, addr: real(self, oc.Aff(addr.c % 256, addr.t)))
    elif mutant == "lds_store_lost":
        monkeypatch.setattr(oc.Walk, "_lds", lambda self, op, ops, mods: None)
    else:
        real_src = oc._swizzle_src
        monkeypatch.setattr(oc, "_swizzle_src", lambda mods, lane: lane if "SWAP" in " ".join(mods) else real_src(mods, lane))
    ok = True
    try:
        sigs = {k: oc.Walk(asm, k).signature(Y0) for k in ("up_library", "up_four", "up_reversed")}
        ok &= len(set(sigs.values())) == 1
        ok &= root(asm, "up_library")[0][1] == oc.canon(butterfly([1, 2, 4, 8, 16, 32])[0])
        a = oc.Walk(asm, "block_256", block=(256, 1, 1))
        ok &= a.roots(Y0)[0][1] == oc.canon(perfect(0, 256))
    except (oc.Unsupported, AssertionError, KeyError):
        ok = False
    assert not ok, mutant


MMA_SRC = os.path.join(HERE, "checker", "mma_chains.hip")


@pytest.fixture(scope="module")
def mma_asm():
    if not os.path.exists(oc.HIPCC) and shutil.which("hipcc") is None:
        pytest.skip("no hipcc")
    return oc.compile_asm(MMA_SRC)


def mma_chain(i, j, K):
    """Output (i, j) of A . B on the 16x16x32 bf16 instruction, from the chunk
    rule: the accumulator starts at +0 and each 8-k chunk, in increasing k,
    updates it once with its eight exact products."""
    acc = oc.Node("const", leaf="0")
    for c in range(K // 8):
        prods = [oc.Node("prod", [oc.Node("load", leaf=repr(oc.Aff(2 * (i * K + k), {"arg0": 1}))),
                                  oc.Node("load", leaf=repr(oc.Aff(2 * (j * K + k), {"arg8": 1})))])
                 for k in range(8 * c, 8 * c + 8)]
        acc = oc.Node("chunk", [acc] + prods)
    return acc


@pytest.mark.parametrize("K", [64, 128])
def test_mfma_k_loops(mma_asm, K):
    """The K loop's step (32 or 64, unrolled or not) leaves the signature: the
    same products reach the same accumulator in the same chunk order.  Two
    accumulators, or the k halves in reverse order, are other trees."""
    loop32 = oc.Walk(mma_asm, "mma_loop32", args={24: K})
    loop64 = oc.Walk(mma_asm, "mma_loop64", args={24: K})
    assert len(loop32.stores) == 256 and not loop32.opaque
    assert loop32.signature() == loop64.signature()
    for i, j in ((0, 0), (5, 11), (15, 15)):
        got = [t for a, t in loop32.roots() if a == repr(oc.Aff(4 * (i * 16 + j), {"arg16": 1}))]
        assert got == [oc.canon(mma_chain(i, j, K))], (i, j)
    if K == 64:
        sigs = {k: oc.Walk(mma_asm, k).signature() for k in ("mma_unrolled", "mma_two_acc", "mma_reversed")}
        assert sigs["mma_unrolled"] == loop32.signature()
        assert len(set(sigs.values())) == 3


def test_command_line(asm, capsys):
    """python -m paper_2609_11356_amd.order_check: one line per class."""
    assert oc.main([SRC, "up_library", "up_shfl", "down_library", "strided_fold", "--arg", "16=512"]) == 0
    lines = capsys.readouterr().out.strip().splitlines()
    assert sorted(l.split()[1:] for l in lines) == [["down_library"], ["strided_fold"], ["up_library", "up_shfl"]]
    assert oc.main([SRC, "branch_on_data"]) == 0
    assert "not walked" in capsys.readouterr().out
