"""The oracle's model of one gfx950 bf16 or fp16 MFMA, checked against the hardware
on crafted and random single-instruction cases (compared at run time; no
hardware output is stored).  Operand slot layouts: 16x16x32 -- lane l holds
A[l%16][8(l/16)+e], B[8(l/16)+e][l%16], and rows 4(l/16)+r of column l%16 of
C; 32x32x16 -- A[l%32][8(l/32)+e], B[8(l/32)+e][l%32], C rows
8(r/4)+4(l/32)+r%4 of column l%32."""
import ctypes
import itertools
import os

import numpy as np
import pytest

import oracle
from paper_2609_11356_amd import inputs

pytestmark = pytest.mark.gpu
GEO = {0: (16, 32, 16), 1: (32, 16, 32), 2: (16, 32, 16), 3: (32, 16, 32)}   # 2, 3: fp16 operands


@pytest.fixture(scope="module")
def probe():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from tests.probe import build
    if not os.path.exists(build.LIB):
        build.build()
    L = ctypes.CDLL(build.LIB)
    L.mfma_probe.argtypes = [ctypes.c_int, ctypes.c_int] + [ctypes.c_void_p] * 5
    L.mfma_probe.restype = ctypes.c_int
    return L


def to_slots(instr, A, B, C):
    instr %= 2
    n = A.shape[0]
    l = np.arange(64)
    As = np.zeros((n, 64, 8), np.uint16)
    Bs = np.zeros((n, 64, 8), np.uint16)
    if instr == 0:
        for e in range(8):
            As[:, :, e] = A[:, l % 16, 8 * (l // 16) + e]
            Bs[:, :, e] = B[:, 8 * (l // 16) + e, l % 16]
        Cs = np.stack([C[:, 4 * (l // 16) + r, l % 16] for r in range(4)], -1)
    else:
        for e in range(8):
            As[:, :, e] = A[:, l % 32, 8 * (l // 32) + e]
            Bs[:, :, e] = B[:, 8 * (l // 32) + e, l % 32]
        Cs = np.stack([C[:, 8 * (r // 4) + 4 * (l // 32) + r % 4, l % 32] for r in range(16)], -1)
    return As, Bs, np.ascontiguousarray(Cs, dtype=np.float32)


def from_slots(instr, Ds):
    instr %= 2
    R, _, Cc = GEO[instr]
    n = Ds.shape[0]
    D = np.zeros((n, R, Cc), np.float32)
    l = np.arange(64)
    if instr == 0:
        for r in range(4):
            D[:, 4 * (l // 16) + r, l % 16] = Ds[:, :, r]
    else:
        for r in range(16):
            D[:, 8 * (r // 4) + 4 * (l // 32) + r % 4, l % 32] = Ds[:, :, r]
    return D


def run_probe(probe, instr, A, B, C):
    import torch
    As, Bs, Cs = to_slots(instr, A, B, C)
    dA = torch.from_numpy(As.view(np.int16)).cuda()
    dB = torch.from_numpy(Bs.view(np.int16)).cuda()
    dC = torch.from_numpy(Cs).cuda()
    dD = torch.empty_like(dC)
    st = probe.mfma_probe(instr, A.shape[0], dA.data_ptr(), dB.data_ptr(), dC.data_ptr(), dD.data_ptr(),
                          torch.cuda.current_stream().cuda_stream)
    assert st == 0
    torch.cuda.synchronize()
    return from_slots(instr, dD.cpu().numpy())


def model(instr, A, B, C):
    R, Kc, Cc = GEO[instr]
    n = A.shape[0]
    a = np.broadcast_to(A[:, :, None, :], (n, R, Cc, Kc)).reshape(-1, Kc)
    b = np.broadcast_to(np.transpose(B, (0, 2, 1))[:, None, :, :], (n, R, Cc, Kc)).reshape(-1, Kc)
    out = oracle.group_update_batch(C.reshape(-1), a, b, g=Kc, fma=1, in_dtype="f16" if instr >= 2 else "bf16")
    return out.reshape(n, R, Cc)


def compare(got, want, what):
    g = got.reshape(-1)
    w = want.reshape(-1)
    same = (g.view(np.uint32) == w.view(np.uint32)) | (np.isnan(g) & np.isnan(w))
    assert same.all(), "%s: %d of %d differ (first at %d: gpu %r oracle %r)" % (
        what, (~same).sum(), same.size, np.argmin(same), g[np.argmin(same)], w[np.argmin(same)])


def bits(x):
    return inputs.f32_to_bf16_bits(np.asarray(x, np.float32))


@pytest.mark.parametrize("instr", [0, 1])
@pytest.mark.parametrize("mode", ["normal", "spread", "wide", "accdom", "sparse", "cancel"])
def test_random_single_instructions(probe, instr, mode):
    R, Kc, Cc = GEO[instr]
    n = 3000 if instr == 0 else 800
    rng = np.random.default_rng(1000 * instr + hash(mode) % 997)
    seed = int(rng.integers(1 << 30))
    if mode == "normal":
        A = inputs.normal_bf16(seed, (n, R, Kc))
        B = inputs.normal_bf16(seed + 1, (n, Kc, Cc))
        C = rng.standard_normal((n, R, Cc)).astype(np.float32)
    else:
        lo, hi = (-120, 120) if mode == "wide" else (-30, 30)
        A = inputs.spread_bf16(seed, (n, R, Kc), lo, hi)
        B = inputs.spread_bf16(seed + 1, (n, Kc, Cc), -30, 30)
        C = (rng.standard_normal((n, R, Cc)) * np.exp2(rng.integers(-40, 40, (n, R, Cc)))).astype(np.float32)
        if mode == "accdom":
            C = (rng.choice([-1, 1], (n, R, Cc)) * np.exp2(rng.integers(20, 60, (n, R, Cc))) *
                 (1 + rng.random((n, R, Cc)))).astype(np.float32)
        if mode == "sparse":
            A[rng.random(A.shape) < 0.7] = 0
        if mode == "cancel":
            A[:, :, 1] = A[:, :, 0] ^ 0x8000
            B[:, 1, :] = B[:, 0, :]
    compare(run_probe(probe, instr, A, B, C), model(instr, A, B, C), "%d %s" % (instr, mode))


def test_triple_walk_all_placements(probe):
    """r = 2^-15 with +L/-L (L = 1024) at every ordered triple of distinct k
    positions of one 16x16x32 instruction (Sec. 4's walks, exhaustively)."""
    trips = list(itertools.permutations(range(32), 3))
    n = (len(trips) + 15) // 16
    A = np.zeros((n, 16, 32), np.float32)
    for t, (pr, p1, p2) in enumerate(trips):
        c, i = divmod(t, 16)
        A[c, i, pr], A[c, i, p1], A[c, i, p2] = 2.0 ** -15, 1024.0, -1024.0
    Ab = bits(A)
    B = np.full((n, 32, 16), 0x3F80, np.uint16)
    C = np.zeros((n, 16, 16), np.float32)
    compare(run_probe(probe, 0, Ab, B, C), model(0, Ab, B, C), "triple walk")


def test_edge_values(probe):
    """Window width, ties, grid floor, subnormal anchors, overflow, zeros."""
    cases = []
    for e in range(0, 40):
        cases.append(([(2.0 ** e, 1), (-(2.0 ** e), 1), (1, 1)], 0.0))
    for d in range(24, 40):
        cases.append(([(2.0 ** -24, 1), (2.0 ** -d, 1)], 1.0))
        cases.append(([(-(2.0 ** -24), 1), (-(2.0 ** -d), 1)], -1.0))
    for d in range(0, 12):
        cases.append(([(2.0 ** -75, 2.0 ** -75), (2.0 ** -75, 2.0 ** -(75 + d))], 0.0))
        cases.append(([(-(2.0 ** -75), 2.0 ** -75), (-(2.0 ** -75), 2.0 ** -(75 + d))], 0.0))
    for d in range(-4, 8):
        cases.append(([(2.0 ** -133, 2.0 ** 100), (1.5 * 2.0 ** -26, 2.0 ** (-26 - d))], 0.0))
    cases += [([(2.0 ** 127, 2), (-(2.0 ** 127), 2), (1, 1)], 0.0), ([(np.inf, 1)], 0.0),
              ([(np.inf, 0)], 0.0), ([(-0.0, 1), (0.0, -1)], -0.0), ([(1, 1)], np.inf),
              ([(1, 1), (2.0 ** -24, 1)], 0.0), ([(1, 1), (2.0 ** -23, 1), (2.0 ** -24, 1)], 0.0)]
    n = (len(cases) + 15) // 16
    A = np.zeros((n, 16, 32), np.float32)
    B = np.zeros((n, 32, 16), np.float32)
    C = np.zeros((n, 16, 16), np.float32)
    for t, (prods, acc) in enumerate(cases):
        c, i = divmod(t, 16)
        for q, (x, y) in enumerate(prods):
            A[c, i, q], B[c, q, i] = x, y
        C[c, i, i] = acc
    Ab, Bb = bits(A), bits(B)
    compare(run_probe(probe, 0, Ab, Bb, C), model(0, Ab, Bb, C), "edge values")


def h16(x):
    return np.asarray(x, dtype=np.float16).view(np.uint16)


@pytest.mark.parametrize("instr", [2, 3])
@pytest.mark.parametrize("mode", ["normal", "spread", "wide", "subnormal", "accdom", "cancel"])
def test_random_single_instructions_f16(probe, instr, mode):
    """fp16 operands: the same chunk model with binary16 exponents."""
    R, Kc, Cc = GEO[instr]
    n = 2000 if instr == 2 else 500
    rng = np.random.default_rng(77 * instr + hash(mode) % 991)
    sp = lambda shape, lo, hi: h16(rng.choice([-1, 1], shape) * (1 + rng.random(shape)) *
                                   np.exp2(rng.integers(lo, hi, shape)))
    C = (rng.standard_normal((n, R, Cc)) * np.exp2(rng.integers(-20, 20, (n, R, Cc)))).astype(np.float32)
    if mode == "normal":
        A, B = h16(rng.standard_normal((n, R, Kc))), h16(rng.standard_normal((n, Kc, Cc)))
        C = rng.standard_normal((n, R, Cc)).astype(np.float32)
    elif mode == "spread":
        A, B = sp((n, R, Kc), -12, 12), sp((n, Kc, Cc), -12, 12)
    elif mode == "wide":
        A, B = sp((n, R, Kc), -24, 15), sp((n, Kc, Cc), -24, 15)
    elif mode == "subnormal":
        A, B = sp((n, R, Kc), -24, -13), sp((n, Kc, Cc), -24, 4)
        C = (rng.standard_normal((n, R, Cc)) * np.exp2(rng.integers(-50, -20, (n, R, Cc)))).astype(np.float32)
    elif mode == "accdom":
        A, B = sp((n, R, Kc), -8, 8), sp((n, Kc, Cc), -8, 8)
        C = (rng.choice([-1, 1], (n, R, Cc)) * np.exp2(rng.integers(10, 40, (n, R, Cc))) *
             (1 + rng.random((n, R, Cc)))).astype(np.float32)
    else:
        A, B = sp((n, R, Kc), -6, 6), sp((n, Kc, Cc), -6, 6)
        A[:, :, 1] = A[:, :, 0] ^ 0x8000
        B[:, 1, :] = B[:, 0, :]
    compare(run_probe(probe, instr, A, B, C), model(instr, A, B, C), "f16 %d %s" % (instr, mode))


def test_edge_values_f16(probe):
    """Binary16 window width, ties, subnormal factors, the largest values,
    infinities and zeros in one 16x16x32 fp16 instruction each."""
    cases = []
    for e in range(0, 31):
        ea, eb = min(e, 15), e - min(e, 15)
        cases.append(([(2.0 ** ea, 2.0 ** eb), (-(2.0 ** ea), 2.0 ** eb), (1, 1)], 0.0))
    for d in range(12, 25):
        cases.append(([(2.0 ** -12, 2.0 ** -12), (2.0 ** -d, 1)], 1.0))
        cases.append(([(-(2.0 ** -12), 2.0 ** -12), (-(2.0 ** -d), 1)], -1.0))
    cases += [([(1, 1), (2.0 ** -12, 2.0 ** -12), (2.0 ** -15, 2.0 ** -15)], 0.0),
              ([(65504, 65504), (-65504, 65504), (2.0 ** -24, 1)], 0.0),
              ([(np.inf, 1)], 0.0), ([(np.inf, 0)], 0.0), ([(-0.0, 1), (0.0, -1)], -0.0),
              ([(1, 1)], np.inf), ([(2.0 ** -24, 2.0 ** -24)], 0.0), ([(2.0 ** -24, 2.0 ** -24)], 2.0 ** -60)]
    n = (len(cases) + 15) // 16
    A = np.zeros((n, 16, 32), np.float32)
    B = np.zeros((n, 32, 16), np.float32)
    C = np.zeros((n, 16, 16), np.float32)
    for t, (prods, acc) in enumerate(cases):
        c, i = divmod(t, 16)
        for q, (x, y) in enumerate(prods):
            A[c, i, q], B[c, q, i] = x, y
        C[c, i, i] = acc
    Ah, Bh = h16(A), h16(B)
    compare(run_probe(probe, 2, Ah, Bh, C), model(2, Ah, Bh, C), "f16 edge values")
