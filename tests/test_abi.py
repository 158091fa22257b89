"""The C ABI on the host: the library loads, exports every entry point
include/dg.h declares, and validates descriptors and arguments before any
launch (CPU only: no call here reaches a kernel)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def dg():
    from paper_2609_11356_amd import dg as _dg
    if not os.path.exists(_dg.LIB_PATH):
        from paper_2609_11356_amd import build
        build.build()
    return _dg


def declared_functions():
    src = open(os.path.join(ROOT, "include", "dg.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(dg_[a-z0-9_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported(dg):
    lib = dg.lib()
    names = declared_functions()
    assert set(names) == set(dg.exported_symbols())
    for n in names:
        assert hasattr(lib, n), n


def test_version_and_strerror(dg):
    assert dg.dg_version() == 600
    for s in range(8):
        assert dg.dg_strerror(s)


@pytest.mark.parametrize("bad", [
    dict(tile_k=24), dict(tile_k=0), dict(mma="8x8"), dict(split_k=0), dict(split_k=65),
    dict(split_k=3, k_cuts=[5]), dict(split_k=3, k_cuts=[10, 5]), dict(split_k=2, k_cuts=[0]),
    dict(leaf_w=0), dict(fma=2),
    dict(split_k=4, split_layout="strided", split_tile=48),              # not whole accumulator tiles
    dict(split_k=4, split_layout="strided", split_tile=0),
    dict(split_k=3, split_layout="strided", split_tile=64, k_cuts=[64, 128]),
    dict(split_k=4, split_layout="strided", split_tile=64, tail="first"),
    dict(split_k=4, split_tile=64),                                      # a tile without the layout
    dict(leaf_layout="diagonal"), dict(lane_fold="sideways"), dict(norm_round="never")])
def test_invalid_descriptors_rejected(dg, bad):
    with pytest.raises((dg.DgError, KeyError)):
        dg.Desc(**bad)


def test_raw_field_values_checked(dg):
    """Out-of-range enum values of the new fields are rejected at create."""
    lib = dg.lib()
    for field, value in (("leaf_layout", 2), ("lane_fold", -1), ("norm_round", 5)):
        p = dg.dg_desc_params()
        p.struct_size = ctypes.sizeof(p)
        p.mma, p.tile_k, p.split_k, p.leaf_w = 1, 64, 1, 64
        setattr(p, field, value)
        h = ctypes.c_void_p()
        assert lib.dg_desc_create(ctypes.byref(p), ctypes.byref(h)) == dg.DG_ERR_INVALID


def test_strided_leaf_limits(dg):
    """Strided leaves: a power of two up to 256 lanes; the count-down fold
    needs strided lanes."""
    for w in (3, 48, 512):
        with pytest.raises(dg.DgError) as e:
            dg.Desc(leaf_w=w, leaf_layout="strided")
        assert e.value.status == dg.DG_ERR_UNSUPPORTED
    with pytest.raises(dg.DgError) as e:
        dg.Desc(leaf_w=64, lane_fold="down")
    assert e.value.status == dg.DG_ERR_UNSUPPORTED
    for w in (1, 2, 32, 64, 256):
        dg.Desc(leaf_w=w, leaf_layout="strided", lane_fold="down")


def test_unsupported_combinations(dg):
    with pytest.raises(dg.DgError) as e:
        dg.Desc(merge="bf16", partial="f32")
    assert e.value.status == dg.DG_ERR_UNSUPPORTED
    with pytest.raises(dg.DgError) as e:
        dg.Desc(epi_round="pre_act", epilogue="bias")
    assert e.value.status == dg.DG_ERR_UNSUPPORTED


def test_signature_canonical(dg):
    a = dg.Desc(mma="16x16x32", tile_k=64).signature()
    b = dg.Desc(mma="32x32x16", tile_k=64).signature()
    assert a == b  # fma = 1: the same 8-k chunks
    c = dg.Desc(mma="16x16x32", tile_k=64, fma=0).signature()
    d = dg.Desc(mma="32x32x16", tile_k=64, fma=0).signature()
    assert c != d and c != a
    assert dg.Desc(split_k=3, k_cuts=[100, 200]).signature().endswith("cuts:100:200")
    st = dg.Desc(split_k=4, split_layout="strided", split_tile=64).signature()
    assert st.endswith("strided:64") and st != dg.Desc(split_k=4).signature()
    # the scalar path: fma cannot change bits, so it is normalised away
    assert dg.Desc(mma="scalar", tile_k=7, fma=0).signature() == dg.Desc(mma="scalar", tile_k=7).signature()
    assert dg.Desc(mma="scalar", tile_k=64).signature() != dg.Desc(tile_k=64).signature()
    # one strided part is the whole axis: the same order as one contiguous part
    assert dg.Desc(split_layout="strided", split_tile=64).signature() == dg.Desc().signature()
    # leaf layout and fold appear when they are not the defaults; one lane has no fold
    up = dg.Desc(leaf_w=256, leaf_layout="strided").signature()
    down = dg.Desc(leaf_w=256, leaf_layout="strided", lane_fold="down").signature()
    assert up.endswith("leaf-strided") and down.endswith("leaf-strided/fold-down")
    assert dg.Desc(leaf_w=1, leaf_layout="strided", lane_fold="down").signature() == \
        dg.Desc(leaf_w=1, leaf_layout="strided").signature()
    assert up != dg.Desc(leaf_w=256).signature()
    assert dg.Desc(norm_round="pre_weight").signature().endswith("norm-pre-weight")


def test_signature_writes_every_cut(dg):
    """Sixty-four parts with explicit cuts that differ only in the last one
    give different signatures (the text is never cut short), and a buffer one
    byte too small is refused without being written."""
    cuts = [1000 * (i + 1) for i in range(63)]
    other = cuts[:-1] + [cuts[-1] + 1]
    a = dg.Desc(split_k=64, tile_k=64, k_cuts=cuts).signature()
    b = dg.Desc(split_k=64, tile_k=64, k_cuts=other).signature()
    assert a != b
    assert a.endswith(":" + str(cuts[-1])) and b.endswith(":" + str(other[-1]))
    assert a.count(":") == 63 and len(a) + 1 <= dg.SIGNATURE_MAX
    # the widest fields and cuts still fit
    big = [2 ** 62 - 63 + i for i in range(63)]
    w = dg.Desc(split_k=64, tile_k=2 ** 30, k_cuts=big, tile_combine="tree", split_combine="tree",
                tail="first", partial="bf16", merge="bf16", out="bf16", epilogue="bias_silu",
                epi_round="pre_act", leaf_w=256, reduce="sumsq", leaf_layout="strided", lane_fold="down",
                norm_round="pre_weight", in_dtype="f16").signature()
    assert w.endswith(":" + str(big[-1])) and len(w) + 1 <= dg.SIGNATURE_MAX
    lib = dg.lib()
    d = dg.Desc(split_k=64, tile_k=64, k_cuts=cuts)
    buf = ctypes.create_string_buffer(b"x" * len(a), len(a) + 1)
    assert lib.dg_desc_signature(d.handle, buf, len(a)) == dg.DG_ERR_INVALID
    assert buf.value == b"x" * len(a)
    assert lib.dg_desc_signature(d.handle, buf, len(a) + 1) == dg.DG_OK and buf.value.decode() == a


def test_attention_descriptor_validation(dg):
    """Attention descriptors: fields out of range are invalid; orders this
    build cannot run are unsupported; calls are checked before any launch."""
    for bad in (dict(key_block=0), dict(causal=2), dict(block_sum="carry"), dict(pv_fma=2), dict(final="half")):
        with pytest.raises((dg.DgError, KeyError)) as e:
            dg.AttnDesc(**bad)
        if isinstance(e.value, dg.DgError):
            assert e.value.status == dg.DG_ERR_INVALID, bad
    for bad in (dict(key_block=16), dict(key_block=96), dict(p_dtype="f32"), dict(causal=1, q_block=40)):
        with pytest.raises(dg.DgError) as e:
            dg.AttnDesc(**bad)
        assert e.value.status == dg.DG_ERR_UNSUPPORTED, bad
    for ok in (dict(key_block=32, causal=1, q_block=48), dict(key_block=128, q_block=1)):
        dg.AttnDesc(**ok)
    import torch
    if torch.cuda.is_available():
        return
    lib = dg.lib()
    a = dg.AttnDesc()
    c = dg.AttnDesc(causal=1, q_block=64)
    assert lib.dg_attention(a.handle, 16, 16, 16, 16, 0, 8, 8, 64, 1.0, None) == dg.DG_OK
    assert lib.dg_attention(a.handle, 16, 16, 16, 16, 2, 8, 0, 64, 1.0, None) == dg.DG_ERR_SHAPE
    assert lib.dg_attention(a.handle, 16, 16, 16, 16, 2, 8, 8, 96, 1.0, None) == dg.DG_ERR_UNSUPPORTED
    assert lib.dg_attention(c.handle, 16, 16, 16, 16, 2, 8, 9, 64, 1.0, None) == dg.DG_ERR_SHAPE
    assert lib.dg_attention(a.handle, 16, 24, 16, 16, 2, 8, 8, 64, 1.0, None) == dg.DG_ERR_ALIGN
    assert lib.dg_attention(a.handle, None, 16, 16, 16, 2, 8, 8, 64, 1.0, None) == dg.DG_ERR_INVALID
    assert lib.dg_attention(None, 16, 16, 16, 16, 2, 8, 8, 64, 1.0, None) == dg.DG_ERR_INVALID
    assert lib.dg_attention(a.handle, 16, 16, 16, 16, 65536, 8, 8, 64, 1.0, None) == dg.DG_ERR_SHAPE


def test_binding_refuses_inconsistent_tensors(dg):
    """The binding checks shapes, dtypes and layout with ValueError (not
    assert, so python -O keeps them) before the library is called; CPU
    tensors reach these checks first, so no GPU is needed."""
    import torch
    bf, f32 = torch.bfloat16, torch.float32
    A, B = torch.zeros(8, 16, dtype=bf), torch.zeros(16, 24, dtype=bf)
    cases = [
        (dg.dg_gemm, (dg.Desc(), A, B, None, torch.zeros(8, 24, dtype=bf))),            # C dtype
        (dg.dg_gemm, (dg.Desc(), A, torch.zeros(12, 24, dtype=bf), None, torch.zeros(8, 24))),
        (dg.dg_gemm, (dg.Desc(), A.float(), B, None, torch.zeros(8, 24))),
        (dg.dg_gemm, (dg.Desc(), A, B.t(), None, torch.zeros(8, 16))),                    # shape
        (dg.dg_gemm, (dg.Desc(), A, B.t().contiguous().t(), None, torch.zeros(8, 24))),   # layout
        (dg.dg_gemm, (dg.Desc(epilogue="bias"), A, B, None, torch.zeros(8, 24))),         # bias missing
        (dg.dg_gemm, (dg.Desc(epilogue="bias"), A, B, torch.zeros(23, dtype=bf), torch.zeros(8, 24))),
        (dg.dg_gemm_colsum, (dg.Desc(), A, torch.zeros(12, 24, dtype=bf), None, torch.zeros(8, 24),
                             torch.zeros(24))),
        (dg.dg_gemm_colsum, (dg.Desc(), A, B, None, torch.zeros(8, 24, dtype=bf), torch.zeros(24))),
        (dg.dg_gemm_colsum, (dg.Desc(), A, B, None, torch.zeros(8, 24), torch.zeros(23))),
        (dg.dg_gemm_colsum, (dg.Desc(epilogue="bias_silu"), A, B, None, torch.zeros(8, 24), torch.zeros(24))),
        (dg.dg_rmsnorm, (dg.Desc(reduce="sumsq"), torch.zeros(4, 8), None, 1e-6,
                         torch.zeros(4, 8, dtype=bf))),                                    # Y dtype
        (dg.dg_rmsnorm, (dg.Desc(reduce="sumsq", out="bf16"), torch.zeros(4, 8), None, 1e-6,
                         torch.zeros(4, 8))),
        (dg.dg_rmsnorm, (dg.Desc(reduce="sumsq"), torch.zeros(4, 8), torch.zeros(7, dtype=bf), 1e-6,
                         torch.zeros(4, 8))),
        (dg.dg_softmax, (dg.Desc(), torch.zeros(4, 8), torch.zeros(4, 8, dtype=bf))),
        (dg.dg_softmax, (dg.Desc(), torch.zeros(4, 8), torch.zeros(4, 9))),
        (dg.dg_layernorm, (dg.Desc(), torch.zeros(4, 8), None, None, 1e-6, torch.zeros(4, 8, dtype=bf))),
        (dg.dg_layernorm, (dg.Desc(), torch.zeros(4, 8), None, torch.zeros(8), 1e-6, torch.zeros(4, 8))),
        (dg.dg_rowsum, (dg.Desc(), torch.zeros(4, 8), torch.zeros(3))),
        (dg.dg_rowsum, (dg.Desc(), torch.zeros(4, 8, dtype=torch.float64), torch.zeros(4))),
    ]
    for fn, args in cases:
        with pytest.raises(ValueError):
            fn(*args)
    # consistent CPU tensors pass the shape checks and stop at the device check
    with pytest.raises(ValueError, match="GPU"):
        dg.dg_gemm(dg.Desc(), A, B, None, torch.zeros(8, 24))
    with pytest.raises(ValueError, match="GPU"):
        dg.dg_softmax(dg.Desc(), torch.zeros(4, 8), torch.zeros(4, 8))


def test_argument_errors_need_no_gpu(dg):
    # Every call below must be rejected before any launch: the pointers are
    # not device addresses.  Run where no GPU is visible, so that a
    # validation gap can never turn into a launch on bogus addresses.
    import torch
    if torch.cuda.is_available():
        pytest.skip("runs without a GPU: the calls pass host integers as pointers")
    d = dg.Desc()
    lib = dg.lib()
    # M = 0 / N = 0: no-op, no launch
    assert lib.dg_gemm(d.handle, 16, 16, None, 16, 0, 8, 8, None) == dg.DG_OK
    assert lib.dg_gemm(d.handle, 16, 16, None, 16, 8, 0, 8, None) == dg.DG_OK
    # negative sizes, NULL operands, misalignment, missing bias: rejected first
    assert lib.dg_gemm(d.handle, 16, 16, None, 16, -1, 8, 8, None) == dg.DG_ERR_SHAPE
    assert lib.dg_gemm(d.handle, None, 16, None, 16, 8, 8, 8, None) == dg.DG_ERR_INVALID
    assert lib.dg_gemm(d.handle, 17, 16, None, 16, 8, 8, 8, None) == dg.DG_ERR_ALIGN
    assert lib.dg_gemm(d.handle, 16, 16, None, 18, 8, 8, 8, None) == dg.DG_ERR_ALIGN  # fp32 C
    assert lib.dg_gemm(None, 16, 16, None, 16, 8, 8, 8, None) == dg.DG_ERR_INVALID
    e = dg.Desc(epilogue="bias")
    assert lib.dg_gemm(e.handle, 16, 16, None, 16, 8, 8, 8, None) == dg.DG_ERR_INVALID
    # a plan that leaves a part empty
    s = dg.Desc(split_k=8, tile_k=64)
    assert lib.dg_gemm(s.handle, 16, 16, None, 16, 8, 8, 100, None) == dg.DG_ERR_SHAPE
    c = dg.Desc(split_k=2, k_cuts=[300])
    assert lib.dg_gemm(c.handle, 16, 16, None, 16, 8, 8, 256, None) == dg.DG_ERR_SHAPE
    k0 = dg.Desc(split_k=2)
    assert lib.dg_gemm(k0.handle, 16, 16, None, 16, 8, 8, 0, None) == dg.DG_ERR_SHAPE
    # the no-allocation entry point: partials beyond its fixed scratch are
    # refused before any HIP call; its other checks are dg_gemm's
    s8 = dg.Desc(split_k=8, tile_k=64)
    assert lib.dg_gemm_noalloc(s8.handle, 16, 16, None, 16, 128, 8192, 4096, None) == dg.DG_ERR_SCRATCH
    assert 8 * 128 * 8192 * 4 > dg.NOALLOC_SCRATCH_BYTES
    assert lib.dg_gemm_noalloc(s8.handle, 16, 16, None, 16, 0, 8192, 4096, None) == dg.DG_OK
    assert lib.dg_gemm_noalloc(s8.handle, 16, 16, None, 16, 8, 8, 100, None) == dg.DG_ERR_SHAPE
    assert lib.dg_gemm_noalloc(d.handle, 17, 16, None, 16, 8, 8, 8, None) == dg.DG_ERR_ALIGN
    assert lib.dg_gemm_noalloc(None, 16, 16, None, 16, 8, 8, 8, None) == dg.DG_ERR_INVALID
    # knobs the build lacks
    kn = dg.dg_knobs(2, 48, 128, 0, 0, 0)
    assert lib.dg_gemm_knobs(d.handle, 16, 16, None, 16, 8, 8, 8, ctypes.byref(kn), None) == dg.DG_ERR_UNSUPPORTED
    kn = dg.dg_knobs(4, 16, 64, 0, 0, 5)
    assert lib.dg_gemm_knobs(d.handle, 16, 16, None, 16, 8, 8, 8, ctypes.byref(kn), None) == dg.DG_ERR_UNSUPPORTED
    kn = dg.dg_knobs(4, 64, 64, 0, 0, 4, 256)      # a combination the build lacks
    assert lib.dg_gemm_knobs(d.handle, 16, 16, None, 16, 8, 8, 8, ctypes.byref(kn), None) == dg.DG_ERR_UNSUPPORTED
    kn = dg.dg_knobs(3, 0, 0, 0, 0, 0, 128)        # slab_k is a kernel-4 knob
    assert lib.dg_gemm_knobs(d.handle, 16, 16, None, 16, 8, 8, 8, ctypes.byref(kn), None) == dg.DG_ERR_UNSUPPORTED
    kn = dg.dg_knobs(3, 256, 256, 0, 0, 0)         # kernel 3 has no 256 x 256 block
    assert lib.dg_gemm_knobs(d.handle, 16, 16, None, 16, 8, 8, 8, ctypes.byref(kn), None) == dg.DG_ERR_UNSUPPORTED
    # kernels 6, 7 and 10 take no tile shape; split_n is a multiple of 256 within N, and only for them
    for k in (6, 7, 10):
        for kn in (dg.dg_knobs(k, 256, 256, 0, 0, 0, 0, 0), dg.dg_knobs(k, 0, 0, 0, 0, 0, 0, 100),
                   dg.dg_knobs(k, 0, 0, 0, 0, 0, 0, 512), dg.dg_knobs(k, 0, 0, 0, 0, 0, 0, -256)):
            assert lib.dg_gemm_knobs(d.handle, 16, 16, None, 16, 8, 304, 8, ctypes.byref(kn), None) == \
                dg.DG_ERR_UNSUPPORTED
    sc = dg.Desc(mma="scalar", tile_k=16)
    for kn in (dg.dg_knobs(5, 0, 0, 0, 0, 0, 0, 0), dg.dg_knobs(1, 0, 0, 0, 0, 0, 0, 0),
               dg.dg_knobs(9, 16, 0, 0, 0, 0, 0, 0)):
        assert lib.dg_gemm_knobs(sc.handle, 16, 16, None, 16, 8, 304, 8, ctypes.byref(kn), None) == \
            dg.DG_ERR_UNSUPPORTED
    for kn in (dg.dg_knobs(5, 256, 256, 0, 0, 0, 0, 256), dg.dg_knobs(9, 0, 0, 0, 0, 0, 0, 0),
               dg.dg_knobs(8, 16, 16, 0, 0, 5, 256, 0), dg.dg_knobs(8, 48, 16, 0, 0, 0, 0, 0)):
        assert lib.dg_gemm_knobs(d.handle, 16, 16, None, 16, 8, 304, 8, ctypes.byref(kn), None) == \
            dg.DG_ERR_UNSUPPORTED
    # binary16 operands: not on the tiled, direct-to-LDS or four-wave kernels
    hd = dg.Desc(in_dtype="f16")
    for k in (2, 7, 8, 10):
        kn = dg.dg_knobs(k, 0, 0, 0, 0, 0, 0, 0)
        assert lib.dg_gemm_knobs(hd.handle, 16, 16, None, 16, 8, 304, 8, ctypes.byref(kn), None) == \
            dg.DG_ERR_UNSUPPORTED
    assert "/in-f16" in hd.signature() and "/in-f16" not in d.signature()
    # a strided split runs on the generic kernel or on kernel 4 with one dealt tile per slab
    sd = dg.Desc(split_k=4, split_layout="strided", split_tile=64)
    for kn in (dg.dg_knobs(3, 0, 0, 0, 0, 0, 0), dg.dg_knobs(5, 0, 0, 0, 0, 0, 0),
               dg.dg_knobs(4, 16, 32, 0, 0, 4, 128)):
        assert lib.dg_gemm_knobs(sd.handle, 16, 16, None, 16, 8, 8, 64, ctypes.byref(kn), None) == \
            dg.DG_ERR_UNSUPPORTED
    # kernel 12 (tile chain or tree, or fma = 0, on the tiled layout): no
    # other knob, no carried chain, no strided split, scalar path or e4m3 B,
    # tile boundaries on 32-k steps, at most 128 tiles per tree part
    tree = dg.Desc(tile_k=64, tile_combine="tree")
    k12 = dg.dg_knobs(12, 0, 0, 0, 0, 0, 0, 0)
    for desc, K in [(d, 512), (sd, 512), (sc, 512), (dg.Desc(tile_k=64, in_dtype="bf16_e4m3", fma=0), 512),
                    (dg.Desc(tile_k=32, tile_combine="tree"), 8192), (dg.Desc(tile_k=64, tile_combine="seq",
                                                                              tail="first"), 1000),
                    (dg.Desc(mma="32x32x16", tile_k=64, fma=0), 512)]:
        assert lib.dg_gemm_knobs(desc.handle, 16, 16, None, 16, 8, 64, K, ctypes.byref(k12), None) == \
            dg.DG_ERR_UNSUPPORTED, desc.signature()
    for kn in (dg.dg_knobs(12, 128, 128, 0, 0, 0, 0, 0), dg.dg_knobs(12, 0, 0, 1, 0, 0, 0, 0),
               dg.dg_knobs(12, 0, 0, 0, 0, 4, 0, 0), dg.dg_knobs(13, 0, 0, 0, 0, 0, 0, 0)):
        assert lib.dg_gemm_knobs(tree.handle, 16, 16, None, 16, 8, 64, 512, ctypes.byref(kn), None) == \
            dg.DG_ERR_UNSUPPORTED
    assert lib.dg_gemm_knobs(tree.handle, 16, 16, None, 16, 8, 60, 512, ctypes.byref(k12), None) == \
        dg.DG_ERR_UNSUPPORTED                                            # N % 8
    # RMS normalisation: the descriptor must name the sum of squares
    q = dg.Desc(reduce="sumsq")
    assert lib.dg_rmsnorm(d.handle, 16, None, 0.0, 16, 4, 5, None) == dg.DG_ERR_INVALID
    assert lib.dg_rmsnorm(q.handle, 16, None, 0.0, 16, 0, 5, None) == dg.DG_OK
    assert lib.dg_rmsnorm(q.handle, 16, None, 0.0, 16, 4, 0, None) == dg.DG_OK
    assert lib.dg_rmsnorm(q.handle, 16, None, 0.0, 16, -1, 5, None) == dg.DG_ERR_SHAPE
    assert lib.dg_rmsnorm(q.handle, None, None, 0.0, 16, 4, 5, None) == dg.DG_ERR_INVALID
    assert lib.dg_rmsnorm(q.handle, 18, None, 0.0, 16, 4, 5, None) == dg.DG_ERR_ALIGN
    assert lib.dg_rmsnorm(q.handle, 16, 17, 0.0, 16, 4, 5, None) == dg.DG_ERR_ALIGN
    assert lib.dg_rmsnorm(None, 16, None, 0.0, 16, 4, 5, None) == dg.DG_ERR_INVALID
    # softmax: the descriptor must name a plain sum
    assert lib.dg_softmax(q.handle, 16, 16, 4, 5, None) == dg.DG_ERR_INVALID
    assert lib.dg_softmax(d.handle, 16, 16, 0, 5, None) == dg.DG_OK
    assert lib.dg_softmax(d.handle, 16, 16, 4, 0, None) == dg.DG_OK
    assert lib.dg_softmax(d.handle, 16, 16, -1, 5, None) == dg.DG_ERR_SHAPE
    assert lib.dg_softmax(d.handle, None, 16, 4, 5, None) == dg.DG_ERR_INVALID
    assert lib.dg_softmax(d.handle, 18, 16, 4, 5, None) == dg.DG_ERR_ALIGN
    # GEMM with column sums: a NULL or misaligned colsum is rejected before any launch
    assert lib.dg_gemm_colsum(d.handle, 16, 16, None, 16, None, 8, 8, 8, None) == dg.DG_ERR_INVALID
    assert lib.dg_gemm_colsum(d.handle, 16, 16, None, 16, 18, 8, 8, 8, None) == dg.DG_ERR_ALIGN
    assert lib.dg_gemm_colsum(d.handle, 16, 16, None, 16, 16, 65536 * 256, 8, 8, None) == dg.DG_ERR_SHAPE
    assert lib.dg_gemm_colsum(d.handle, 16, 16, None, 16, None, 8, 0, 8, None) == dg.DG_OK
    # layer normalisation
    assert lib.dg_layernorm(d.handle, 16, None, None, 0.0, 16, 0, 5, None) == dg.DG_OK
    assert lib.dg_layernorm(d.handle, 16, None, None, 0.0, 16, 4, 0, None) == dg.DG_OK
    assert lib.dg_layernorm(d.handle, 16, None, None, 0.0, 16, -1, 5, None) == dg.DG_ERR_SHAPE
    assert lib.dg_layernorm(d.handle, 16, None, None, 0.0, None, 4, 5, None) == dg.DG_ERR_INVALID
    assert lib.dg_layernorm(d.handle, 16, None, 19, 0.0, 16, 4, 5, None) == dg.DG_ERR_ALIGN
    assert lib.dg_layernorm(None, 16, None, None, 0.0, 16, 4, 5, None) == dg.DG_ERR_INVALID
    # row reduction
    assert lib.dg_rowsum(d.handle, 16, 16, 0, 5, None) == dg.DG_OK
    assert lib.dg_rowsum(d.handle, 16, 18, 4, 5, None) == dg.DG_ERR_ALIGN
    assert lib.dg_rowsum(d.handle, 16, None, 4, 5, None) == dg.DG_ERR_INVALID
    assert lib.dg_rowsum(d.handle, 16, 16, -1, 5, None) == dg.DG_ERR_SHAPE


def test_fp8_descriptors_need_no_gpu(dg):
    """e4m3 x e4m3 pairs with the fp8 instructions only; under fma = 1 the
    four fp8 shapes share one signature (one chunk chain), under fma = 0
    each its own group; the kernels that may run it, and kernel 13's
    conditions, are checked before any launch."""
    lib = dg.lib()
    fp8 = ("16x16x32_fp8", "32x32x16_fp8", "16x16x128_f8f6f4", "32x32x64_f8f6f4")
    for bad in (dict(mma="16x16x32", in_dtype="e4m3"), dict(mma="16x16x32_fp8", tile_k=64),
                dict(mma="scalar", in_dtype="e4m3"), dict(mma="16x16x128_f8f6f4", tile_k=64, in_dtype="e4m3"),
                dict(mma="16x16x32_fp8", tile_k=64, in_dtype="bf16_e4m3")):
        with pytest.raises(dg.DgError) as e:
            dg.Desc(**bad)
        assert e.value.status == dg.DG_ERR_INVALID, bad
    sigs = {dg.Desc(mma=m, tile_k=128, in_dtype="e4m3").signature() for m in fp8}
    assert len(sigs) == 1 and next(iter(sigs)).startswith("gfx950-e4m3-mfma/chunk16/"), sigs
    assert len({dg.Desc(mma=m, tile_k=128, in_dtype="e4m3", fma=0).signature() for m in fp8}) == 4
    d = dg.Desc(mma="16x16x32_fp8", tile_k=64, in_dtype="e4m3")
    for k in (2, 3, 4, 5, 6, 7, 8, 9, 10, 11, 12):
        kn = dg.dg_knobs(k, 0, 0, 0, 0, 0, 0, 0)
        assert lib.dg_gemm_knobs(d.handle, 16, 16, None, 16, 16, 64, 512, ctypes.byref(kn), None) == \
            dg.DG_ERR_UNSUPPORTED, k
    k13 = dg.dg_knobs(13, 0, 0, 0, 0, 0, 0, 0)
    for desc, N, K in [(dg.Desc(mma="16x16x32_fp8", tile_k=64, in_dtype="e4m3", fma=0), 64, 512),
                       (dg.Desc(mma="16x16x32_fp8", tile_k=64, in_dtype="e4m3", tile_combine="tree"), 64, 512),
                       (dg.Desc(mma="16x16x32_fp8", tile_k=64, in_dtype="e4m3", split_k=2, split_layout="strided",
                                split_tile=64), 64, 512),
                       (dg.Desc(mma="16x16x32_fp8", tile_k=64, in_dtype="e4m3", tail="first"), 64, 520),
                       (dg.Desc(mma="16x16x32_fp8", tile_k=64, in_dtype="e4m3", split_k=2, k_cuts=[72]), 64, 512),
                       (d, 56, 512), (d, 64, 520)]:
        assert lib.dg_gemm_knobs(desc.handle, 16, 16, None, 16, 16, N, K, ctypes.byref(k13), None) == \
            dg.DG_ERR_UNSUPPORTED, (desc.signature(), N, K)
    for kn in (dg.dg_knobs(13, 128, 256, 0, 0, 0, 0, 0), dg.dg_knobs(13, 0, 0, 1, 0, 0, 0, 0),
               dg.dg_knobs(13, 0, 128, 0, 0, 0, 0, 0), dg.dg_knobs(13, 64, 0, 0, 0, 0, 0, 0)):
        assert lib.dg_gemm_knobs(d.handle, 16, 16, None, 16, 16, 64, 512, ctypes.byref(kn), None) == \
            dg.DG_ERR_UNSUPPORTED
    # the packed entry point takes a bf16 A only
    assert lib.dg_gemm_packed(d.handle, 16, 16, None, 16, 16, 64, 512, None) == dg.DG_ERR_UNSUPPORTED
    # byte operands need no alignment of their own; kernel 13 needs 16-byte rows
    assert lib.dg_gemm_knobs(d.handle, 17, 16, None, 16, 16, 64, 512, ctypes.byref(k13), None) == \
        dg.DG_ERR_UNSUPPORTED
    assert lib.dg_gemm(d.handle, 17, 16, None, 16, 0, 64, 512, None) == dg.DG_OK


def test_packed_b_size_and_refusals_need_no_gpu(dg):
    """The packed form's size, and dg_pack_b / dg_gemm_packed refusing what
    they do not take before any launch (host integers as pointers)."""
    import torch
    if torch.cuda.is_available():
        pytest.skip("runs without a GPU: the calls pass host integers as pointers")
    lib = dg.lib()
    assert dg.dg_packed_b_bytes(0, 16) == 0 and dg.dg_packed_b_bytes(32, 0) == 0
    assert dg.dg_packed_b_bytes(32, 16) == 1024
    assert dg.dg_packed_b_bytes(33, 17) == 2 * 2 * 1024
    assert dg.dg_packed_b_bytes(4096, 4096) == 4096 * 4096 * 2      # whole blocks: no padding
    assert dg.dg_packed_b_bytes(-1, 16) == 2 ** 64 - 1
    assert dg.dg_packed_b_bytes(1 << 62, 1 << 62) == 2 ** 64 - 1    # overflow
    assert lib.dg_pack_b(16, 16, -1, 8, None) == dg.DG_ERR_SHAPE
    assert lib.dg_pack_b(16, 16, 0, 8, None) == dg.DG_OK
    assert lib.dg_pack_b(None, 16, 8, 8, None) == dg.DG_ERR_INVALID
    assert lib.dg_pack_b(17, 16, 8, 8, None) == dg.DG_ERR_ALIGN
    assert lib.dg_pack_b(16, 8, 8, 8, None) == dg.DG_ERR_ALIGN       # Bp needs 16 bytes
    d = dg.Desc()
    ok = dict(A=16, B=16, C=16)
    gp = lambda desc, M, N, K, A=16, B=16, C=16: lib.dg_gemm_packed(desc.handle, A, B, None, C, M, N, K, None)
    assert gp(d, 0, 8, 8) == dg.DG_OK
    assert gp(d, 65, 8, 8) == dg.DG_ERR_UNSUPPORTED                 # few rows only
    assert gp(d, 8, 8, 8, B=8) == dg.DG_ERR_ALIGN
    assert gp(d, 8, 8, 8, A=None) == dg.DG_ERR_INVALID
    for bad in (dict(tile_combine="tree", tile_k=64), dict(fma=0), dict(tail="first", tile_k=64),
                dict(split_k=2, k_cuts=[48]), dict(split_k=4, split_layout="strided", split_tile=96, tile_k=32),
                dict(mma="scalar")):
        assert gp(dg.Desc(**bad), 8, 64, 256) == dg.DG_ERR_UNSUPPORTED, bad
    kn = dg.dg_knobs(4, 16, 64, 0, 0, 4, 64)       # a row-major kernel on packed B
    assert lib.dg_gemm_packed_knobs(d.handle, 16, 16, None, 16, 8, 8, 8, ctypes.byref(kn), None) == \
        dg.DG_ERR_UNSUPPORTED
    kn = dg.dg_knobs(11, 16, 0, 0, 0, 7)           # a ring depth the build lacks
    assert lib.dg_gemm_packed_knobs(d.handle, 16, 16, None, 16, 8, 8, 8, ctypes.byref(kn), None) == \
        dg.DG_ERR_UNSUPPORTED
    kn = dg.dg_knobs(11, 0, 0, 1, 0, 0)            # no block order on kernel 11
    assert lib.dg_gemm_packed_knobs(d.handle, 16, 16, None, 16, 8, 8, 8, ctypes.byref(kn), None) == \
        dg.DG_ERR_UNSUPPORTED
    kn = dg.dg_knobs(11, 0, 0, 0, 0, 0)            # kernel 11 only reads packed B
    assert lib.dg_gemm_knobs(d.handle, 16, 16, None, 16, 8, 8, 8, ctypes.byref(kn), None) == dg.DG_ERR_UNSUPPORTED


def test_build_rejects_register_spills():
    """The build fails when a kernel's resource remark reports spilled VGPRs."""
    from paper_2609_11356_amd import build
    remarks = "\n".join([
        "a.hip:1:1: remark: Function Name: _Zk1 [-Rpass-analysis=kernel-resource-usage]",
        "a.hip:1:1: remark:     SGPRs Spill: 2 [-Rpass-analysis=kernel-resource-usage]",
        "a.hip:1:1: remark:     VGPRs Spill: 0 [-Rpass-analysis=kernel-resource-usage]",
        "   12 | __global__ void k1() {",
        "      | ^",
        "a.hip:9:1: remark: Function Name: _Zk2 [-Rpass-analysis=kernel-resource-usage]",
        "a.hip:9:1: remark:     VGPRs Spill: 154 [-Rpass-analysis=kernel-resource-usage]",
    ])
    assert build.spilling_kernels(remarks) == ["_Zk2 (154 VGPRs)"]
    assert build.spilling_kernels(remarks.replace("154", "0")) == []
