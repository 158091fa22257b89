"""The Sec. 4 reconstruction procedure (tests/reconstruct.py) on the CPU,
with the oracle standing in for the vendor library: a planted descriptor
from every candidate family must come back as the one survivor, and a
vendor whose order changes between output columns must be reported as
having no single order."""
import numpy as np
import pytest

import oracle
from tests import reconstruct as r

PLANTED = [
    (2880, 256, 4, dict(tile_k=64, split_k=4, split_layout="strided", split_tile=128, split_combine="seq")),
    (2688, 256, 8, dict(tile_k=32, split_k=4, split_layout="strided", split_tile=32, split_combine="seq")),
    (2048, 128, 8, dict(tile_k=64, split_k=6, k_cuts=r._balanced_cuts(2048, 6, 128), split_combine="tree")),
    (768, 128, 16, dict(tile_k=64)),
    (4096, 256, 1, dict(tile_k=64, split_k=4, split_layout="strided", split_tile=64, split_combine="tree")),
    (2688, 256, 1, dict(mma="32x32x16", tile_k=64, fma=0)),
    (2688, 256, 1, dict(tile_k=64, fma=0)),
    (4096, 256, 2, dict(tile_k=64, split_k=3, k_cuts=r._span_cuts(4096, 3, 256), split_combine="seq")),
]


@pytest.mark.parametrize("case", range(len(PLANTED)))
def test_planted_descriptor_is_the_one_survivor(case):
    K, N, M, planted = PLANTED[case]
    planted = dict(planted, mma=planted.get("mma", "16x16x32"), out="bf16")
    pool, hist, uniform = r.reconstruct(M, N, K, draws=4, seed=case, log=lambda s: None,
                                        vendor=lambda A, B: oracle.gemm(planted, A, B))
    assert uniform
    assert len(pool) == 1, [r.describe(d) for d in pool]
    assert r._key(pool[0], K) == r._key(planted, K)


def test_candidates_are_distinct_orders():
    for K in (512, 768, 1856, 2880, 4096):
        keys = [r._key(d, K) for d in r.candidates(K)]
        assert len(keys) == len(set(keys))
        # every part is non-empty and the parts tile [0, K)
        for key in keys:
            covered = sorted(x for part in key[2] for x in part)
            assert all(b < e for b, e in covered)
            assert covered[0][0] == 0 and covered[-1][1] == K
            assert all(covered[i][1] == covered[i + 1][0] for i in range(len(covered) - 1))


def test_walk_reads_a_split_boundary():
    """The walk's own semantics on a contiguous split at 1024 with the parts
    merged in order: r survives exactly while the pair sits wholly in the
    second part, and is absorbed when the pair straddles the cut."""
    K = 2048
    desc = dict(mma="16x16x32", tile_k=64, split_k=2, k_cuts=[1024], out="bf16")
    ms = r.walk_positions(K)
    out = r.oracle_probe(desc, r.walk_columns(K, ms))
    assert set(np.unique(out)) <= {0, r.SMALL}
    assert np.array_equal(out == r.SMALL, ms >= 1024)


def test_order_varying_by_column_is_reported():
    K, N = 2048, 256
    first = dict(mma="16x16x32", tile_k=64, out="bf16")
    second = dict(mma="16x16x32", tile_k=64, split_k=2, k_cuts=[1024], out="bf16")

    def vendor(A, B):
        C = oracle.gemm(first, A, B)
        C[:, N // 2:] = oracle.gemm(second, A, B[:, N // 2:])
        return C
    pool, hist, uniform = r.reconstruct(1, N, K, vendor=vendor, log=lambda s: None)
    assert not uniform and pool == []
