"""Seeded synthetic inputs shared by the tests, the benchmark and the smoke check.

This module holds no arithmetic of the method: it only draws random numbers
and packs them into bf16 / fp32 storage.  Both the GPU path and the CPU oracle
consume what it returns; neither is imported here.

Recipe (the paper evaluates on LLM-shaped GEMMs whose shape list is not
reproduced; these draws stand in for it):
  * RNG: ``numpy.random.default_rng(seed)`` (PCG64);
  * bf16 operands: standard normals drawn in float64, scaled, rounded to fp32
    (round-to-nearest-even), then to bf16 by round-to-nearest-even on the bits;
  * "spread" operands: bf16 values with exponents uniform in [-30, 30], a
    uniform 7-bit fraction and a random sign -- narrow exponent ranges hide a
    regrouping, so every parity case is also drawn this way;
  * row-reduction input: |x| = exp(2 Z), Z ~ N(0, 1) (log-normal, sigma = 2),
    random sign, fp32.
"""
from __future__ import annotations

import numpy as np


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Pack fp32 values into bf16 bit patterns (round-to-nearest-even)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    nan = (u & 0x7FFFFFFF) > 0x7F800000
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    if nan.any():
        r[nan] = ((u[nan] >> 16) | 0x40).astype(np.uint16)
    return r


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def normal_bf16(seed: int, shape, scale: float = 1.0) -> np.ndarray:
    rng = np.random.default_rng(seed)
    x = rng.standard_normal(shape) * scale
    return f32_to_bf16_bits(x.astype(np.float32))


def spread_bf16(seed: int, shape, emin: int = -30, emax: int = 30) -> np.ndarray:
    rng = np.random.default_rng(seed)
    e = rng.integers(emin, emax + 1, size=shape, dtype=np.int64)
    frac = rng.integers(0, 128, size=shape, dtype=np.int64)
    sign = rng.integers(0, 2, size=shape, dtype=np.int64)
    return ((sign << 15) | ((e + 127) << 7) | frac).astype(np.uint16)


def normal_f16(seed: int, shape, scale: float = 1.0) -> np.ndarray:
    """N(0, scale^2) draws as IEEE binary16 bits (numpy's nearest-even conversion)."""
    rng = np.random.default_rng(seed)
    return (rng.standard_normal(shape) * scale).astype(np.float16).view(np.uint16)


def spread_f16(seed: int, shape, emin: int = -14, emax: int = 14) -> np.ndarray:
    """Binary16 bits with uniform exponent fields in [emin, emax] (normal
    range), random fraction and sign."""
    rng = np.random.default_rng(seed)
    e = rng.integers(emin, emax + 1, size=shape, dtype=np.int64)
    frac = rng.integers(0, 1024, size=shape, dtype=np.int64)
    sign = rng.integers(0, 2, size=shape, dtype=np.int64)
    return ((sign << 15) | ((e + 15) << 10) | frac).astype(np.uint16)


def e4m3_uniform(seed: int, shape) -> np.ndarray:
    """OCP e4m3 codes (uint8) drawn uniformly over the 254 non-NaN codes:
    both zeros, every subnormal and normal, up to +-448."""
    rng = np.random.default_rng(seed)
    c = rng.integers(0, 254, size=shape).astype(np.uint8)
    # skip 0x7F (and, shifted by one more, 0xFF): codes 0..126 -> 0x00..0x7E,
    # 127..253 -> 0x80..0xFE
    return np.where(c >= 127, c + 1, c).astype(np.uint8)


def e4m3_weights(seed: int, shape, e_mid: float = 6.0, e_sd: float = 1.5) -> np.ndarray:
    """OCP e4m3 codes shaped like quantised weights: a random sign, a
    mantissa field uniform over 0..7, and an exponent field drawn around
    e_mid (values near 2^(e_mid - 7)), clipped to 0..15; NaN codes redrawn
    as the largest finite magnitude."""
    rng = np.random.default_rng(seed)
    e = np.clip(np.rint(rng.normal(e_mid, e_sd, size=shape)), 0, 15).astype(np.uint8)
    m = rng.integers(0, 8, size=shape).astype(np.uint8)
    sgn = rng.integers(0, 2, size=shape).astype(np.uint8)
    c = (sgn << 7) | (e << 3) | m
    nan = (c & 0x7F) == 0x7F
    c[nan] = c[nan] - 1
    return c.astype(np.uint8)


def lognormal_f32(seed: int, shape, sigma: float = 2.0) -> np.ndarray:
    rng = np.random.default_rng(seed)
    mag = np.exp(sigma * rng.standard_normal(shape))
    sign = np.where(rng.integers(0, 2, size=shape) == 1, -1.0, 1.0)
    return (sign * mag).astype(np.float32)


# ----------------------------------------------------------- named workloads

TINY = dict(M=16, N=64, K=256)
SWEEP_K = SWEEP_N = 4096
SWEEP_M = (1, 7, 32, 128, 1024, 4096)
DECODE = dict(M=8, N=4096, K=14336)
MLP = dict(M=2048, N=14336, K=4096)
ROWS = dict(rows=16384, cols=8192)


def tiny(seed: int = 0, spread: bool = False):
    """A 16x256, B 256x64: N(0,1)/sqrt(K) rounded to bf16."""
    M, N, K = TINY["M"], TINY["N"], TINY["K"]
    if spread:
        return spread_bf16(seed, (M, K)), spread_bf16(seed + 1000, (K, N))
    rng = np.random.default_rng(seed)
    a = (rng.standard_normal((M, K)) / np.sqrt(K)).astype(np.float32)
    b = (rng.standard_normal((K, N)) / np.sqrt(K)).astype(np.float32)
    return f32_to_bf16_bits(a), f32_to_bf16_bits(b)


def sweep_weight(seed: int = 2):
    """B 4096x4096 bf16 ~ N(0, 0.02)."""
    return normal_bf16(seed, (SWEEP_K, SWEEP_N), 0.02)


def sweep_activations(seed: int = 1, rows: int = 4096):
    """The first `rows` rows of one 4096x4096 N(0,1) bf16 draw (row r is the
    same for every M > r)."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((rows, SWEEP_K))
    return f32_to_bf16_bits(x.astype(np.float32))


def decode(seed_a: int = 3, seed_b: int = 4):
    M, N, K = DECODE["M"], DECODE["N"], DECODE["K"]
    return normal_bf16(seed_a, (M, K), 1.0), normal_bf16(seed_b, (K, N), 0.02)


def mlp(seed_a: int = 5, seed_b: int = 6, seed_bias: int = 7, rows: int | None = None):
    M, N, K = MLP["M"], MLP["N"], MLP["K"]
    a = normal_bf16(seed_a, (M, K), 1.0)
    if rows is not None:
        a = a[:rows].copy()
    return a, normal_bf16(seed_b, (K, N), 0.02), normal_bf16(seed_bias, (N,), 0.02)


def rowsum_input(seed: int = 8, rows: int | None = None, cols: int | None = None):
    return lognormal_f32(seed, (rows or ROWS["rows"], cols or ROWS["cols"]))
