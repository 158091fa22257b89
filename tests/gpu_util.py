"""Helpers for GPU tests: device transfer of bf16 bit patterns and
bitwise comparison (NaNs compared as a class)."""
import numpy as np


def dev_bf16(bits):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits, dtype=np.uint16).view(np.int16)).view(torch.bfloat16).cuda()


def dev_f16(bits):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits, dtype=np.uint16).view(np.int16)).view(torch.float16).cuda()


def dev_f32(x):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda()


def host_bits(t):
    import torch
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def as_u32(x):
    """Output values as comparable bit patterns (bf16 widened to fp32 bits);
    every NaN maps to one pattern."""
    x = np.asarray(x)
    if x.dtype == np.uint16:
        x = (x.astype(np.uint32) << 16).view(np.float32)
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).copy()
    u[np.isnan(x)] = 0x7FC00000
    return u


def assert_bits_equal(got, want, what=""):
    g, w = as_u32(got), as_u32(want)
    assert g.shape == w.shape, (g.shape, w.shape)
    bad = np.nonzero(g.reshape(-1) != w.reshape(-1))[0]
    if len(bad):
        i = bad[0]
        gv = g.reshape(-1)[i:i + 1].view(np.float32)[0]
        wv = w.reshape(-1)[i:i + 1].view(np.float32)[0]
        raise AssertionError("%s: %d of %d outputs differ; first at flat index %d: got %r (0x%08x) want %r (0x%08x)"
                             % (what, len(bad), g.size, i, gv, g.reshape(-1)[i], wv, w.reshape(-1)[i]))
