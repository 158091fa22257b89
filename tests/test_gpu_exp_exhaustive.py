"""The library's device exp and SiLU (the functions the fused epilogue and
the softmax kernels call) and exp2 (the attention kernel's) against the CPU
oracle's dgo_exp / dgo_silu / dgo_exp2 on every binary32 input, bit for bit (NaNs compared as a class).  The exp is
the library's own fixed sequence of steps (Cody-Waite reduction, degree-7
Taylor polynomial, exact power-of-two scaling), so its bits have no external
reference: the oracle's plain C version of the same steps is what fixes
them.  Four tests of 2^30 inputs each, in slabs of 2^26."""
import ctypes

import numpy as np
import pytest

import oracle

pytestmark = pytest.mark.gpu

SLAB = 1 << 26


@pytest.fixture(scope="module")
def probe():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from tests.probe import build
    L = ctypes.CDLL(build.MATH_LIB)
    L.math_probe_exp_silu.argtypes = [ctypes.c_uint64, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                      ctypes.c_void_p]
    L.math_probe_exp_silu.restype = ctypes.c_int
    L.math_probe_exp2.argtypes = [ctypes.c_uint64, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p]
    L.math_probe_exp2.restype = ctypes.c_int
    return L


def _same(got, want):
    g, w = got.view(np.uint32), want.view(np.uint32)
    ok = (g == w) | (np.isnan(got) & np.isnan(want))
    return ok


@pytest.mark.parametrize("quarter", range(4))
def test_exp_and_silu_equal_the_oracle_on_every_binary32(probe, quarter):
    import torch
    e_d = torch.empty(SLAB, dtype=torch.float32, device="cuda")
    s_d = torch.empty(SLAB, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    lo = quarter << 30
    for start in range(lo, lo + (1 << 30), SLAB):
        st = probe.math_probe_exp_silu(start, SLAB, e_d.data_ptr(), s_d.data_ptr(), stream)
        assert st == 0, "probe launch failed (%d)" % st
        ge, gs = e_d.cpu().numpy(), s_d.cpu().numpy()
        we, ws = oracle.exp_silu_range(start, SLAB)
        for name, got, want in (("exp", ge, we), ("silu", gs, ws)):
            ok = _same(got, want)
            if not ok.all():
                i = int(np.nonzero(~ok)[0][0])
                x = np.uint32(start + i).view(np.float32)
                raise AssertionError("%s differs on %d inputs of slab 0x%08x; first x = %r (0x%08x): "
                                     "device %r, oracle %r" % (name, int((~ok).sum()), start, x, start + i,
                                                               got[i], want[i]))
        print("slab 0x%08x ok" % start, flush=True)


@pytest.mark.parametrize("half", range(2))
def test_exp2_equals_the_oracle_on_every_binary32(probe, half):
    import torch
    e_d = torch.empty(SLAB, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    lo = half << 31
    for start in range(lo, lo + (1 << 31), SLAB):
        st = probe.math_probe_exp2(start, SLAB, e_d.data_ptr(), stream)
        assert st == 0, "probe launch failed (%d)" % st
        got = e_d.cpu().numpy()
        want = oracle.exp2_range(start, SLAB)
        ok = _same(got, want)
        if not ok.all():
            i = int(np.nonzero(~ok)[0][0])
            raise AssertionError("exp2 differs on %d inputs of slab 0x%08x; first bits 0x%08x: device %r, oracle %r"
                                 % (int((~ok).sum()), start, start + i, got[i], want[i]))
        print("exp2 slab 0x%08x ok" % start, flush=True)
