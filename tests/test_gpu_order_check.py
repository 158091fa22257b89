"""The order checker's classes confirmed on the part (Sec. 6: equivalence
the checker certifies must be equivalence the hardware shows): the fixture
kernels of tests/checker run on seeded exponent-spread inputs; kernels the
checker puts in one class give the same bits on every draw, and every pair
of classes differs on some draw."""
import ctypes
import os
import shutil

import numpy as np
import pytest

from paper_2609_11356_amd import inputs, order_check as oc

pytestmark = pytest.mark.gpu
HERE = os.path.dirname(os.path.abspath(__file__))

LANE = {"up_library": None, "up_shfl": None, "up_four": None, "up_two": None, "up_reversed": None,
        "down_library": None, "down_shfl": None, "up_steps_swapped": None, "chain": None}
BLOCK = {"block_256": (256, 1, 1), "block_128x2": (128, 1, 1), "block_256_chain": (256, 1, 1)}
FOLD = ("strided_fold", "strided_fold_unroll2", "strided_fold_two_acc")
MMA = ("mma_unrolled", "mma_loop32", "mma_loop64", "mma_two_acc", "mma_reversed")


@pytest.fixture(scope="module")
def lib():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    if not os.path.exists(oc.HIPCC) and shutil.which("hipcc") is None:
        pytest.skip("no hipcc for the checker")
    from tests.probe import build
    if not os.path.exists(build.CHECK_LIB):
        build.build()
    L = ctypes.CDLL(build.CHECK_LIB)
    L.run_lane.argtypes = [ctypes.c_char_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int]
    L.run_mma.argtypes = [ctypes.c_char_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int]
    return L


def spread(rng, n):
    return (rng.standard_normal(n) * np.exp2(rng.integers(-20, 20, n))).astype(np.float32)


def confirm(classes, run, draws):
    """run(name, draw) -> output bits; same class -> equal on every draw,
    different classes -> some draw differs."""
    outs = {k: [run(k, d) for d in draws] for c in classes for k in c}
    for c in classes:
        for k in c[1:]:
            for d, (a, b) in enumerate(zip(outs[c[0]], outs[k])):
                assert np.array_equal(a, b), (c[0], k, d)
    for i in range(len(classes)):
        for j in range(i + 1, len(classes)):
            a, b = classes[i][0], classes[j][0]
            assert any(not np.array_equal(x, y) for x, y in zip(outs[a], outs[b])), (a, b)


def test_lane_and_block_classes_on_the_part(lib):
    import torch
    asm = oc.compile_asm(os.path.join(HERE, "checker", "lane_trees.hip"))
    y0 = [(8, 0)]
    sig = {k: oc.Walk(asm, k).signature(y0) for k in LANE}
    sig.update({k: oc.Walk(asm, k, block=b).signature(y0) for k, b in BLOCK.items()})
    sig.update({k: oc.Walk(asm, k, args={16: 512}).signature(y0) for k in FOLD})
    classes = oc.classes(sig)
    print("classes:", classes, flush=True)
    rng = np.random.default_rng(11)
    draws = [spread(rng, 512) for _ in range(100)]
    x = torch.empty(512, dtype=torch.float32, device="cuda")
    y = torch.empty(64, dtype=torch.float32, device="cuda")

    def run(name, d):
        # the 64-element trees read x[0..63], the blocks x[0..255], the folds x[0..511]
        x.copy_(torch.from_numpy(d))
        y.fill_(float("nan"))
        assert lib.run_lane(name.encode(), x.data_ptr(), y.data_ptr(), 512) == 0, name
        return y[:1].cpu().numpy().view(np.uint32).copy()
    # compare only kernels that sum the same elements: group the classes by element count
    groups = [[c for c in classes if c[0] in names] for names in (set(LANE), set(BLOCK), set(FOLD))]
    for g in groups:
        confirm(g, run, draws)


def test_mfma_classes_on_the_part(lib):
    import torch
    asm = oc.compile_asm(os.path.join(HERE, "checker", "mma_chains.hip"))
    sig = {k: oc.Walk(asm, k, args={24: 64} if "loop" in k else None).signature() for k in MMA}
    classes = oc.classes(sig)
    print("classes:", classes, flush=True)
    assert len(classes) == 3
    draws = [(inputs.spread_bf16(100 + s, (16, 64)), inputs.spread_bf16(200 + s, (16, 64))) for s in range(40)]
    A = torch.empty((16, 64), dtype=torch.int16, device="cuda")
    B = torch.empty((16, 64), dtype=torch.int16, device="cuda")
    C = torch.empty((16, 16), dtype=torch.float32, device="cuda")

    def run(name, d):
        A.copy_(torch.from_numpy(d[0].view(np.int16)))
        B.copy_(torch.from_numpy(d[1].view(np.int16)))
        C.fill_(float("nan"))
        assert lib.run_mma(name.encode(), A.data_ptr(), B.data_ptr(), C.data_ptr(), 64) == 0, name
        return C.cpu().numpy().view(np.uint32).copy()
    confirm(classes, run, draws)
