"""Thin ctypes binding of libdg.so (include/dg.h): argument marshalling only.

Every step of the computation runs in the library's HIP kernels; this module
checks shapes and dtypes, turns torch tensors into device pointers and the
current HIP stream, and raises :class:`DgError` on a non-zero status.  It
never computes a result itself: if libdg.so is missing it raises.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdg.so")

DG_OK, DG_ERR_INVALID, DG_ERR_UNSUPPORTED, DG_ERR_SHAPE, DG_ERR_ALIGN, DG_ERR_NOMEM, DG_ERR_HIP, DG_ERR_SCRATCH = range(8)
MMA = {"16x16x32": 1, "32x32x16": 2, "scalar": 3,
       # the fp8 instructions (in_dtype "e4m3"; the f8f6f4 shapes at unit scales)
       "16x16x32_fp8": 4, "32x32x16_fp8": 5, "16x16x128_f8f6f4": 6, "32x32x64_f8f6f4": 7}
COMBINE = {"carry": 0, "seq": 1, "tree": 2}
TAIL = {"last": 0, "first": 1}
DTYPE = {"f32": 0, "bf16": 1}
EPILOGUE = {"none": 0, "bias": 1, "bias_silu": 2}
EPI_ROUND = {"final": 0, "pre_act": 1}
REDUCE = {"sum": 0, "sumsq": 1}
MAX_SPLIT = 64
SIGNATURE_MAX = 2048
NOALLOC_SCRATCH_BYTES = 16 << 20


class DgError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        super().__init__("%s: %s (status %d)" % (where, dg_strerror(status), status))


class dg_desc_params(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_uint32), ("mma", ctypes.c_int32), ("tile_k", ctypes.c_int32),
                ("split_k", ctypes.c_int32), ("n_cuts", ctypes.c_int32),
                ("k_cuts", ctypes.POINTER(ctypes.c_int64))] + [
        (n, ctypes.c_int32) for n in ("tile_combine", "split_combine", "tail", "fma", "partial_dtype",
                                      "merge_dtype", "out_dtype", "epilogue", "epi_round", "leaf_w",
                                      "reduce_op", "split_layout", "split_tile", "leaf_layout",
                                      "lane_fold", "norm_round", "in_dtype")]


class dg_knobs(ctypes.Structure):
    _fields_ = [("kernel", ctypes.c_int32), ("tile_m", ctypes.c_int32), ("tile_n", ctypes.c_int32),
                ("order", ctypes.c_int32), ("occupancy", ctypes.c_int32), ("depth", ctypes.c_int32),
                ("slab_k", ctypes.c_int32), ("split_n", ctypes.c_int32)]


class dg_attn_params(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_uint32)] + [
        (n, ctypes.c_int32) for n in ("key_block", "causal", "q_block", "block_sum", "p_dtype", "pv_fma", "l_fma",
                                      "final_div", "out_dtype")]


_lib = None


def lib():
    """The loaded libdg.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        # torch's HIP runtime first: libdg.so then binds to the runtime already
        # in the process instead of loading a second one beside it (two
        # runtimes in one process do not share the device)
        import torch  # noqa: F401
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libdg.so is not built (run __graft_entry__.build() or "
                               "python -m paper_2609_11356_amd.build)")
        L = ctypes.CDLL(LIB_PATH)
        vp, i64 = ctypes.c_void_p, ctypes.c_int64
        L.dg_desc_create.argtypes = [ctypes.POINTER(dg_desc_params), ctypes.POINTER(vp)]
        L.dg_desc_destroy.argtypes = [vp]
        L.dg_desc_destroy.restype = None
        L.dg_desc_signature.argtypes = [vp, ctypes.c_char_p, ctypes.c_size_t]
        L.dg_gemm.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, vp]
        L.dg_gemm_noalloc.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, vp]
        L.dg_gemm_knobs.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, ctypes.POINTER(dg_knobs), vp]
        L.dg_packed_b_bytes.argtypes = [i64, i64]
        L.dg_packed_b_bytes.restype = ctypes.c_size_t
        L.dg_pack_b.argtypes = [vp, vp, i64, i64, vp]
        L.dg_packed_b8_bytes.argtypes = [i64, i64]
        L.dg_packed_b8_bytes.restype = ctypes.c_size_t
        L.dg_pack_b8.argtypes = [vp, vp, i64, i64, vp]
        L.dg_gemm_packed.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, vp]
        L.dg_gemm_packed_knobs.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, ctypes.POINTER(dg_knobs), vp]
        L.dg_rowsum.argtypes = [vp, vp, vp, i64, i64, vp]
        L.dg_rmsnorm.argtypes = [vp, vp, vp, ctypes.c_float, vp, i64, i64, vp]
        L.dg_softmax.argtypes = [vp, vp, vp, i64, i64, vp]
        L.dg_layernorm.argtypes = [vp, vp, vp, vp, ctypes.c_float, vp, i64, i64, vp]
        L.dg_gemm_colsum.argtypes = [vp, vp, vp, vp, vp, vp, i64, i64, i64, vp]
        L.dg_attn_desc_create.argtypes = [ctypes.POINTER(dg_attn_params), ctypes.POINTER(vp)]
        L.dg_attn_desc_create.restype = ctypes.c_int
        L.dg_attn_desc_destroy.argtypes = [vp]
        L.dg_attn_desc_destroy.restype = None
        L.dg_attention.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, i64, ctypes.c_float, vp]
        L.dg_attention.restype = ctypes.c_int
        L.dg_strerror.argtypes = [ctypes.c_int]
        L.dg_strerror.restype = ctypes.c_char_p
        L.dg_version.restype = ctypes.c_int32
        for f in ("dg_desc_create", "dg_desc_signature", "dg_gemm", "dg_gemm_noalloc", "dg_gemm_knobs",
                  "dg_pack_b", "dg_pack_b8", "dg_gemm_packed", "dg_gemm_packed_knobs", "dg_rowsum", "dg_rmsnorm", "dg_softmax", "dg_layernorm", "dg_gemm_colsum"):
            getattr(L, f).restype = ctypes.c_int
        _lib = L
    return _lib


def dg_strerror(status: int) -> str:
    return lib().dg_strerror(int(status)).decode()


def dg_version() -> int:
    return int(lib().dg_version())


class Desc:
    """An immutable descriptor (dg_desc_create / dg_desc_destroy).

    Fields (strings as in the header's enums): mma ("16x16x32" | "32x32x16" |
    "scalar", or with e4m3 operands "16x16x32_fp8" | "32x32x16_fp8" |
    "16x16x128_f8f6f4" | "32x32x64_f8f6f4"),
    tile_k, split_k, k_cuts (None or S-1 ints), tile_combine ("carry" |
    "seq" | "tree"), split_combine ("seq" | "tree"), tail ("last" | "first"),
    fma (0/1), partial / merge / out ("f32" | "bf16"), epilogue ("none" |
    "bias" | "bias_silu"), epi_round ("final" | "pre_act"), leaf_w,
    reduce ("sum" | "sumsq"), split_layout ("contiguous" | "strided"),
    split_tile (the dealt tile of a strided split), leaf_layout ("contiguous" |
    "strided": leaf_w lanes each taking every leaf_w-th element), lane_fold
    ("up" | "down": the butterfly's offsets counting up or down), norm_round
    ("final" | "pre_weight": dg_rmsnorm rounds the normalised value to bf16
    before the weight), in_dtype ("bf16" | "f16" | "bf16_e4m3" | "e4m3": the
    GEMM operands; "bf16_e4m3" is a bf16 A with a B of OCP e4m3 bytes,
    "e4m3" both A and B OCP e4m3 bytes, folded by an fp8 instruction)."""

    DEFAULTS = dict(mma="16x16x32", tile_k=64, split_k=1, k_cuts=None, tile_combine="carry",
                    split_combine="seq", tail="last", fma=1, partial="f32", merge="f32", out="f32",
                    epilogue="none", epi_round="final", leaf_w=64, reduce="sum",
                    split_layout="contiguous", split_tile=0, leaf_layout="contiguous", lane_fold="up",
                    norm_round="final", in_dtype="bf16")

    def __init__(self, **fields):
        unknown = set(fields) - set(self.DEFAULTS) - {"model"}
        if unknown:
            raise ValueError("unknown descriptor fields: %s" % sorted(unknown))
        if fields.get("model", "gfx950") != "gfx950":
            raise ValueError("libdg realises the gfx950 MFMA arithmetic only")
        f = dict(self.DEFAULTS)
        f.update({k: v for k, v in fields.items() if k != "model"})
        self.fields = f
        p = dg_desc_params()
        p.struct_size = ctypes.sizeof(dg_desc_params)
        p.mma = MMA[f["mma"]]
        p.tile_k = int(f["tile_k"])
        p.split_k = int(f["split_k"])
        cuts = f["k_cuts"]
        self._cuts = None
        if cuts is not None:
            self._cuts = (ctypes.c_int64 * len(cuts))(*[int(c) for c in cuts])
            p.n_cuts = len(cuts)
            p.k_cuts = ctypes.cast(self._cuts, ctypes.POINTER(ctypes.c_int64))
        p.tile_combine = COMBINE[f["tile_combine"]]
        p.split_combine = COMBINE[f["split_combine"]]
        p.tail = TAIL[f["tail"]]
        p.fma = int(f["fma"])
        p.partial_dtype = DTYPE[f["partial"]]
        p.merge_dtype = DTYPE[f["merge"]]
        p.out_dtype = DTYPE[f["out"]]
        p.epilogue = EPILOGUE[f["epilogue"]]
        p.epi_round = EPI_ROUND[f["epi_round"]]
        p.leaf_w = int(f["leaf_w"])
        p.reduce_op = REDUCE[f["reduce"]]
        p.split_layout = {"contiguous": 0, "strided": 1}[f["split_layout"]]
        p.split_tile = int(f["split_tile"])
        p.leaf_layout = {"contiguous": 0, "strided": 1}[f["leaf_layout"]]
        p.lane_fold = {"up": 0, "down": 1}[f["lane_fold"]]
        p.norm_round = {"final": 0, "pre_weight": 1}[f["norm_round"]]
        p.in_dtype = {"bf16": 0, "f16": 1, "bf16_e4m3": 2, "e4m3": 3}[f["in_dtype"]]
        h = ctypes.c_void_p()
        st = lib().dg_desc_create(ctypes.byref(p), ctypes.byref(h))
        if st != DG_OK:
            raise DgError(st, "dg_desc_create")
        self.handle = h

    def signature(self) -> str:
        buf = ctypes.create_string_buffer(SIGNATURE_MAX)
        st = lib().dg_desc_signature(self.handle, buf, len(buf))
        if st != DG_OK:
            raise DgError(st, "dg_desc_signature")
        return buf.value.decode()

    def __del__(self):
        h = getattr(self, "handle", None)
        if h and _lib is not None:
            _lib.dg_desc_destroy(h)
            self.handle = None


def dg_desc_create(**fields) -> Desc:
    return Desc(**fields)


def _stream(stream):
    if stream is not None:
        return int(stream)
    import torch
    return int(torch.cuda.current_stream().cuda_stream)


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return int(t.data_ptr())


def _need(cond, msg):
    """Refuse a call before anything reaches the library (kept under python -O)."""
    if not cond:
        raise ValueError(msg)


def _out_dtype(desc):
    import torch
    return torch.bfloat16 if desc.fields["out"] == "bf16" else torch.float32


def _on_device(*ts):
    _need(all(t.is_cuda for t in ts if t is not None), "tensors must be on the GPU")


def _in_dtypes(desc):
    """The torch dtypes A and B must have under desc (an e4m3 B as raw bytes
    or torch's float8_e4m3fn)."""
    import torch
    f = desc.fields["in_dtype"]
    if f == "f16":
        return (torch.float16,), (torch.float16,)
    if f == "bf16_e4m3":
        return (torch.bfloat16,), (torch.uint8, getattr(torch, "float8_e4m3fn", torch.uint8))
    if f == "e4m3":
        e = (torch.uint8, getattr(torch, "float8_e4m3fn", torch.uint8))
        return e, e
    return (torch.bfloat16,), (torch.bfloat16,)


def _check_gemm(desc, A, B, bias, C):
    """Shapes, dtypes and layout of a GEMM call; returns (M, N, K)."""
    import torch
    want_a, want_b = _in_dtypes(desc)
    _need(A.dtype in want_a and B.dtype in want_b, "A must be %s and B %s" % (want_a[0], want_b[0]))
    _need(A.dim() == 2 and B.dim() == 2 and C.dim() == 2, "A, B and C must be matrices")
    M, K = A.shape
    K2, N = B.shape
    _need(K2 == K, "inner dimensions differ (%d, %d)" % (K, K2))
    _need(tuple(C.shape) == (M, N), "C must be %d x %d" % (M, N))
    _need(C.dtype == _out_dtype(desc), "C dtype must match the descriptor's output type")
    _need(A.is_contiguous() and B.is_contiguous() and C.is_contiguous(), "A, B and C must be row-major")
    if desc.fields["epilogue"] != "none":
        _need(bias is not None, "the descriptor's epilogue needs a bias")
    if bias is not None:
        _need(bias.dtype == torch.bfloat16 and bias.numel() == N and bias.is_contiguous(),
              "bias must be %d contiguous bf16 values" % N)
    _on_device(A, B, C, bias)
    return M, N, K


def _check_rows(desc, X, Y, *vecs):
    """An fp32 row-major X, a Y of X's shape and the descriptor's output type,
    and optional bf16 per-column vectors; returns (rows, cols)."""
    import torch
    _need(X.dtype == torch.float32 and X.dim() == 2, "X must be an fp32 matrix")
    _need(tuple(Y.shape) == tuple(X.shape), "Y must have X's shape")
    _need(Y.dtype == _out_dtype(desc), "Y dtype must match the descriptor's output type")
    _need(X.is_contiguous() and Y.is_contiguous(), "X and Y must be row-major")
    for t in vecs:
        _need(t is None or (t.dtype == torch.bfloat16 and t.is_contiguous() and t.numel() == X.shape[1]),
              "weight and bias must be %d contiguous bf16 values" % X.shape[1])
    _on_device(X, Y, *vecs)
    return X.shape


def dg_gemm(desc: Desc, A, B, bias, C, M=None, N=None, K=None, stream=None, knobs=None):
    """C = epilogue(A . B) in desc's order.  A (M,K) and B (K,N) bf16 (float16
    when the descriptor's in_dtype is "f16"), bias (N,) bf16 or None, C (M,N)
    of the descriptor's output type, all contiguous on the GPU (or raw device
    addresses with M, N, K given).  Inconsistent tensors raise ValueError
    before the library is called."""
    import torch
    if isinstance(A, torch.Tensor):
        M, N, K = _check_gemm(desc, A, B, bias, C)
    if knobs is not None:
        kp = _knobs(knobs)
        st = lib().dg_gemm_knobs(desc.handle, _ptr(A), _ptr(B), _ptr(bias), _ptr(C), M, N, K,
                                 ctypes.byref(kp), _stream(stream))
    else:
        st = lib().dg_gemm(desc.handle, _ptr(A), _ptr(B), _ptr(bias), _ptr(C), M, N, K, _stream(stream))
    if st != DG_OK:
        raise DgError(st, "dg_gemm")
    return C


def _knobs(knobs):
    return dg_knobs(int(knobs.get("kernel", 0)), int(knobs.get("tile_m", 0)), int(knobs.get("tile_n", 0)),
                    int(knobs.get("order", 0)), int(knobs.get("occupancy", 0)), int(knobs.get("depth", 0)),
                    int(knobs.get("slab_k", 0)), int(knobs.get("split_n", 0)))


def dg_packed_b_bytes(K: int, N: int) -> int:
    """Bytes of the packed form of a K x N matrix: ceil(N/16) ceil(K/32) 1 KB."""
    return int(lib().dg_packed_b_bytes(int(K), int(N)))


class PackedB:
    """B (K x N, bf16 or float16, or e4m3 bytes) in the packed form
    dg_gemm_packed reads: every 32 x 16 block (64 x 16 for e4m3) one 1 KB
    run in the 16x16x32 MFMA's B operand layout, runs by column panel then
    k.  data is a uint8 device tensor; dtype the element type."""

    def __init__(self, data, K: int, N: int, dtype):
        self.data, self.K, self.N, self.dtype = data, int(K), int(N), dtype


def dg_packed_b8_bytes(K: int, N: int) -> int:
    """Bytes of the packed form of a K x N e4m3 matrix: ceil(N/16) ceil(K/64) 1024."""
    return int(lib().dg_packed_b8_bytes(int(K), int(N)))


def dg_pack_b(B, out=None, stream=None) -> PackedB:
    """The packed form of B (K, N) (contiguous, on the GPU: bf16 or float16,
    or e4m3 as uint8 / float8_e4m3fn), into out (a uint8 device tensor of
    dg_packed_b_bytes(K, N), or dg_packed_b8_bytes for e4m3, bytes) or a
    new one."""
    import torch
    b8 = B.dtype in (torch.uint8, getattr(torch, "float8_e4m3fn", torch.uint8))
    _need(B.dim() == 2 and B.is_contiguous() and (b8 or B.dtype in (torch.bfloat16, torch.float16)),
          "B must be a contiguous bf16, float16 or e4m3 matrix")
    _on_device(B)
    K, N = B.shape
    n = dg_packed_b8_bytes(K, N) if b8 else dg_packed_b_bytes(K, N)
    if out is None:
        out = torch.empty(max(n, 16), dtype=torch.uint8, device=B.device)
    _need(out.dtype == torch.uint8 and out.numel() >= n and out.is_contiguous(), "out must hold %d bytes" % n)
    fn = lib().dg_pack_b8 if b8 else lib().dg_pack_b
    st = fn(_ptr(B), _ptr(out), K, N, _stream(stream))
    if st != DG_OK:
        raise DgError(st, "dg_pack_b8" if b8 else "dg_pack_b")
    return PackedB(out, K, N, torch.uint8 if b8 else B.dtype)


def dg_gemm_packed(desc: Desc, A, Bp, bias, C, M=None, N=None, K=None, stream=None, knobs=None):
    """dg_gemm with B packed by dg_pack_b (the same bits); Bp a PackedB, or a
    raw device address with M, N, K given."""
    import torch
    if isinstance(A, torch.Tensor):
        _need(isinstance(Bp, PackedB), "Bp must come from dg_pack_b")
        want_a, want_b = _in_dtypes(desc)
        _need(A.dtype in want_a and Bp.dtype in want_b, "A must be %s and B %s" % (want_a[0], want_b[0]))
        _need(A.dim() == 2 and C.dim() == 2 and A.is_contiguous() and C.is_contiguous(), "A and C must be row-major")
        M, K = A.shape
        N = Bp.N
        _need(Bp.K == K, "inner dimensions differ (%d, %d)" % (K, Bp.K))
        _need(tuple(C.shape) == (M, N), "C must be %d x %d" % (M, N))
        _need(C.dtype == _out_dtype(desc), "C dtype must match the descriptor's output type")
        if desc.fields["epilogue"] != "none":
            _need(bias is not None, "the descriptor's epilogue needs a bias")
        if bias is not None:
            _need(bias.dtype == torch.bfloat16 and bias.numel() == N and bias.is_contiguous(),
                  "bias must be %d contiguous bf16 values" % N)
        _on_device(A, C, bias, Bp.data)
        bptr = _ptr(Bp.data)
    else:
        bptr = _ptr(Bp)
    if knobs is not None:
        kp = _knobs(knobs)
        st = lib().dg_gemm_packed_knobs(desc.handle, _ptr(A), bptr, _ptr(bias), _ptr(C), M, N, K,
                                        ctypes.byref(kp), _stream(stream))
    else:
        st = lib().dg_gemm_packed(desc.handle, _ptr(A), bptr, _ptr(bias), _ptr(C), M, N, K, _stream(stream))
    if st != DG_OK:
        raise DgError(st, "dg_gemm_packed")
    return C


def dg_gemm_noalloc(desc: Desc, A, B, bias, C, M=None, N=None, K=None, stream=None):
    """dg_gemm through the entry point that allocates nothing: split-K
    partials go to the library's fixed per-device scratch (at most
    NOALLOC_SCRATCH_BYTES); calls that overlap on one device race."""
    import torch
    if isinstance(A, torch.Tensor):
        M, N, K = _check_gemm(desc, A, B, bias, C)
    st = lib().dg_gemm_noalloc(desc.handle, _ptr(A), _ptr(B), _ptr(bias), _ptr(C), M, N, K, _stream(stream))
    if st != DG_OK:
        raise DgError(st, "dg_gemm_noalloc")
    return C


def dg_rowsum(desc: Desc, X, out, rows=None, cols=None, stream=None):
    """out[r] = balanced-tree reduction of row r of X (fp32, row-major)."""
    import torch
    if isinstance(X, torch.Tensor):
        _need(X.dtype == torch.float32 and out.dtype == torch.float32 and X.dim() == 2, "X and out must be fp32")
        rows, cols = X.shape
        _need(out.numel() == rows, "out must hold one value per row")
        _need(X.is_contiguous() and out.is_contiguous(), "X and out must be contiguous")
        _on_device(X, out)
    st = lib().dg_rowsum(desc.handle, _ptr(X), _ptr(out), rows, cols, _stream(stream))
    if st != DG_OK:
        raise DgError(st, "dg_rowsum")
    return out


def dg_rmsnorm(desc: Desc, X, w, eps, Y, rows=None, cols=None, stream=None):
    """Y = RMS normalisation of the rows of X (fp32) scaled by w (bf16 or
    None), in the descriptor's order (its reduce must be "sumsq")."""
    import torch
    if isinstance(X, torch.Tensor):
        rows, cols = _check_rows(desc, X, Y, w)
    st = lib().dg_rmsnorm(desc.handle, _ptr(X), _ptr(w), ctypes.c_float(eps), _ptr(Y), rows, cols, _stream(stream))
    if st != DG_OK:
        raise DgError(st, "dg_rmsnorm")
    return Y


def dg_gemm_colsum(desc: Desc, A, B, bias, C, colsum, M=None, N=None, K=None, stream=None):
    """dg_gemm, then colsum[j] = the balanced tree down column j of C (fp32)."""
    import torch
    if isinstance(A, torch.Tensor):
        M, N, K = _check_gemm(desc, A, B, bias, C)
        _need(colsum.dtype == torch.float32 and colsum.numel() == N and colsum.is_contiguous(),
              "colsum must be %d contiguous fp32 values" % N)
        _on_device(colsum)
    st = lib().dg_gemm_colsum(desc.handle, _ptr(A), _ptr(B), _ptr(bias), _ptr(C), _ptr(colsum), M, N, K,
                              _stream(stream))
    if st != DG_OK:
        raise DgError(st, "dg_gemm_colsum")
    return C


def dg_layernorm(desc: Desc, X, w, b, eps, Y, rows=None, cols=None, stream=None):
    """Y = layer normalisation of the rows of X (fp32), both row sums in the
    descriptor's order, then the bf16 weight and bias (each may be None)."""
    import torch
    if isinstance(X, torch.Tensor):
        rows, cols = _check_rows(desc, X, Y, w, b)
    st = lib().dg_layernorm(desc.handle, _ptr(X), _ptr(w), _ptr(b), ctypes.c_float(eps), _ptr(Y), rows, cols,
                            _stream(stream))
    if st != DG_OK:
        raise DgError(st, "dg_layernorm")
    return Y


def dg_softmax(desc: Desc, X, Y, rows=None, cols=None, stream=None):
    """Y = softmax of the rows of X (fp32), the row sum in the descriptor's
    order (its reduce must be "sum")."""
    import torch
    if isinstance(X, torch.Tensor):
        rows, cols = _check_rows(desc, X, Y)
    st = lib().dg_softmax(desc.handle, _ptr(X), _ptr(Y), rows, cols, _stream(stream))
    if st != DG_OK:
        raise DgError(st, "dg_softmax")
    return Y


class AttnDesc:
    """An immutable attention descriptor (dg_attn_desc_create /
    dg_attn_desc_destroy).  Fields: key_block (BLOCK_N), causal (0/1), q_block
    (BLOCK_M, causal only), block_sum ("seq" | "tree"), p_dtype ("bf16"),
    pv_fma (0/1), l_fma (0/1), final ("div" | "recip"), out ("f32" | "bf16")."""

    DEFAULTS = dict(key_block=64, causal=0, q_block=64, block_sum="tree", p_dtype="bf16", pv_fma=1, l_fma=0,
                    final="div", out="bf16")

    def __init__(self, **fields):
        unknown = set(fields) - set(self.DEFAULTS) - {"model"}
        if unknown:
            raise ValueError("unknown attention fields: %s" % sorted(unknown))
        if fields.get("model", "gfx950") != "gfx950":
            raise ValueError("libdg realises the gfx950 MFMA arithmetic only")
        f = dict(self.DEFAULTS)
        f.update({k: v for k, v in fields.items() if k != "model"})
        self.fields = f
        p = dg_attn_params()
        p.struct_size = ctypes.sizeof(dg_attn_params)
        p.key_block = int(f["key_block"])
        p.causal = int(f["causal"])
        p.q_block = int(f["q_block"])
        p.block_sum = COMBINE[f["block_sum"]]
        p.p_dtype = DTYPE[f["p_dtype"]]
        p.pv_fma = int(f["pv_fma"])
        p.l_fma = int(f["l_fma"])
        p.final_div = {"div": 0, "recip": 1}[f["final"]]
        p.out_dtype = DTYPE[f["out"]]
        h = ctypes.c_void_p()
        st = lib().dg_attn_desc_create(ctypes.byref(p), ctypes.byref(h))
        if st != DG_OK:
            raise DgError(st, "dg_attn_desc_create")
        self.handle = h

    def __del__(self):
        h = getattr(self, "handle", None)
        if h and _lib is not None:
            _lib.dg_attn_desc_destroy(h)
            self.handle = None


def dg_attention(desc: AttnDesc, Q, K, V, O, qk_scale, H=None, Lq=None, Lk=None, dim=None, stream=None):
    """O = attention in the descriptor's order: Q (H, Lq, d), K and V (H, Lk,
    d) bf16, O (H, Lq, d) of the descriptor's output type, contiguous on the
    GPU (or raw device addresses with the sizes given)."""
    import torch
    if isinstance(Q, torch.Tensor):
        _need(Q.dtype == torch.bfloat16 and K.dtype == torch.bfloat16 and V.dtype == torch.bfloat16,
              "Q, K and V must be bf16")
        _need(Q.dim() == 3 and K.dim() == 3 and V.dim() == 3 and O.dim() == 3, "Q, K, V and O are (H, L, d)")
        H, Lq, dim = Q.shape
        Lk = K.shape[1]
        _need(tuple(K.shape) == (H, Lk, dim) and tuple(V.shape) == (H, Lk, dim), "K and V must be (H, Lk, d)")
        _need(tuple(O.shape) == (H, Lq, dim), "O must be (H, Lq, d)")
        _need(O.dtype == _out_dtype(desc), "O dtype must match the descriptor's output type")
        _need(all(t.is_contiguous() for t in (Q, K, V, O)), "Q, K, V and O must be contiguous")
        _on_device(Q, K, V, O)
    st = lib().dg_attention(desc.handle, _ptr(Q), _ptr(K), _ptr(V), _ptr(O), H, Lq, Lk, dim,
                            ctypes.c_float(qk_scale), _stream(stream))
    if st != DG_OK:
        raise DgError(st, "dg_attention")
    return O


def exported_symbols():
    """Names of the entry points include/dg.h declares."""
    return ["dg_desc_create", "dg_desc_destroy", "dg_desc_signature", "dg_gemm", "dg_gemm_noalloc",
            "dg_gemm_knobs", "dg_rowsum", "dg_rmsnorm", "dg_softmax", "dg_layernorm", "dg_gemm_colsum", "dg_strerror",
            "dg_version", "dg_attn_desc_create", "dg_attn_desc_destroy", "dg_attention",
            "dg_packed_b_bytes", "dg_pack_b", "dg_gemm_packed", "dg_gemm_packed_knobs", "dg_packed_b8_bytes",
            "dg_pack_b8"]
