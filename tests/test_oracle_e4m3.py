"""The oracle's OCP e4m3 decoding (the e4m3 B of in_dtype "bf16_e4m3" is
widened exactly to bf16, Sec. 3.2.1: the instruction is the bf16 one), pinned
to torch's own float8_e4m3fn conversion on every code and to the format's
defining values; the seeded e4m3 input draws; the library's acceptance and
refusal of e4m3 descriptors (host only)."""
import numpy as np
import pytest

import oracle
from paper_2609_11356_amd import inputs

ALL = np.arange(256, dtype=np.uint8)


def torch_decode(codes):
    """bf16 bits of each code by torch's float8_e4m3fn -> float32 (CPU), an
    implementation independent of the oracle's."""
    import torch
    f8 = getattr(torch, "float8_e4m3fn", None)
    if f8 is None:
        pytest.skip("torch has no float8_e4m3fn")
    v = torch.from_numpy(np.asarray(codes, np.uint8).copy()).view(f8).float().numpy()
    return v


def agrees_with_torch(decode):
    got = inputs.bf16_bits_to_f32(decode(ALL))
    want = torch_decode(ALL)
    nan = np.isnan(want)
    return bool(np.array_equal(np.isnan(got), nan) and np.array_equal(got[~nan].view(np.uint32),
                                                                          want[~nan].view(np.uint32)))


def test_every_code_matches_torch():
    assert agrees_with_torch(oracle.e4m3_to_bf16_bits)


def test_defining_values():
    b = oracle.e4m3_to_bf16_bits(ALL)
    f = inputs.bf16_bits_to_f32(b)
    assert f[0x00] == 0 and not np.signbit(f[0x00])
    assert f[0x80] == 0 and np.signbit(f[0x80])
    assert f[0x01] == 2.0 ** -9 and f[0x07] == 7 * 2.0 ** -9        # subnormals
    assert f[0x08] == 2.0 ** -6                                        # smallest normal
    assert f[0x38] == 1.0 and f[0xB8] == -1.0
    assert f[0x7E] == 448.0 and f[0xFE] == -448.0                      # largest finite
    assert np.isnan(f[0x7F]) and np.isnan(f[0xFF])
    assert np.isfinite(f[[c for c in range(256) if c & 0x7F != 0x7F]]).all()
    # the positive codes are ordered by value, strictly (no two codes alike)
    pos = f[:0x7F]
    assert np.all(np.diff(pos) > 0)


@pytest.mark.parametrize("mutant", ["bias8", "subnormal_as_normal", "no_nan", "sign_dropped"])
def test_planted_decoding_mistakes_are_caught(mutant):
    """Each plausible slip in the decoder fails the torch pin."""
    def bad(codes):
        c = np.asarray(codes, np.uint8)
        s, e, m = (c >> 7).astype(np.int64), ((c >> 3) & 15).astype(np.int64), (c & 7).astype(np.int64)
        bias = 8 if mutant == "bias8" else 7
        if mutant == "subnormal_as_normal":
            mag = np.ldexp(1.0 + m / 8.0, (e - bias).astype(np.int32))
        else:
            mag = np.where(e == 0, np.ldexp(m.astype(np.float64), 1 - bias - 3),
                           np.ldexp(1.0 + m / 8.0, (e - bias).astype(np.int32)))
        val = (mag if mutant == "sign_dropped" else np.where(s == 1, -mag, mag)).astype(np.float32)
        bits = (val.view(np.uint32) >> 16).astype(np.uint16)
        if mutant != "no_nan":
            nan = (e == 15) & (m == 7)
            bits[nan] = 0x7FC0
        return bits
    assert not agrees_with_torch(bad)


def test_gemm_on_e4m3_is_the_bf16_gemm_on_widened_b():
    """The oracle's e4m3 GEMM is its bf16 GEMM on the widened B, and the
    small cases it reduces to hold: one product per output is exact."""
    A = inputs.normal_bf16(1, (3, 40))
    B8 = inputs.e4m3_uniform(2, (40, 9))
    d = dict(tile_k=64, out="f32", in_dtype="bf16_e4m3")
    got = oracle.gemm(d, A, B8)
    want = oracle.gemm(dict(d, in_dtype="bf16"), A, oracle.e4m3_to_bf16_bits(B8))
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))
    one = np.zeros((1, 1), np.uint16)
    one[0, 0] = 0x3F80                                                 # A = 1.0
    exact = oracle.gemm(d, one, ALL[None, :])
    ref = torch_decode(ALL)
    fin = ~np.isnan(ref)
    # values equal (the accumulator starts at +0, so the -0 product gives +0)
    assert np.array_equal(exact[0][fin], ref[fin])
    assert not np.signbit(exact[0][0x80])
    assert np.isnan(exact[0][~fin]).all()


def test_input_draws():
    u = inputs.e4m3_uniform(3, (4096,))
    assert u.dtype == np.uint8 and not np.any((u & 0x7F) == 0x7F)
    assert len(np.unique(u)) > 240                                     # nearly every finite code
    w = inputs.e4m3_weights(4, (100000,))
    assert not np.any((w & 0x7F) == 0x7F)
    f = inputs.bf16_bits_to_f32(oracle.e4m3_to_bf16_bits(w))
    assert 0.3 < np.median(np.abs(f)) < 1.5                            # around 2^-1 .. 2^0
    assert np.array_equal(inputs.e4m3_uniform(3, (4096,)), u)          # seeded


def test_library_accepts_and_refuses_e4m3_descriptors():
    import ctypes
    from paper_2609_11356_amd import dg
    d = dg.Desc(tile_k=64, in_dtype="bf16_e4m3")
    assert "in-bf16xe4m3" in d.signature()
    with pytest.raises(dg.DgError) as e:
        dg.Desc(mma="scalar", in_dtype="bf16_e4m3")
    assert e.value.status == dg.DG_ERR_UNSUPPORTED
    import torch
    if torch.cuda.is_available():
        return
    lib = dg.lib()
    for kern in (2, 3, 4, 5, 6, 7, 8, 10):
        kn = dg.dg_knobs(kern, 0, 0, 0, 0, 0)
        assert lib.dg_gemm_knobs(d.handle, 16, 16, None, 16, 8, 8, 8, ctypes.byref(kn), None) == \
            dg.DG_ERR_UNSUPPORTED, kern
    # a row-major e4m3 B needs no 2-byte alignment; misaligned A is still refused
    assert lib.dg_gemm(d.handle, 17, 16, None, 16, 8, 8, 8, None) == dg.DG_ERR_ALIGN
    assert dg.dg_packed_b8_bytes(32, 16) == 1024 and dg.dg_packed_b8_bytes(64, 16) == 1024
    assert dg.dg_packed_b8_bytes(33, 17) == 2048 and dg.dg_packed_b8_bytes(65, 17) == 4096
    assert dg.dg_packed_b8_bytes(-1, 16) == 2 ** 64 - 1
    assert lib.dg_pack_b8(16, 8, 8, 8, None) == dg.DG_ERR_ALIGN        # Bp needs 16 bytes
    assert lib.dg_pack_b8(None, 16, 8, 8, None) == dg.DG_ERR_INVALID
