"""Exact decoding and round-to-nearest-even encoding of the 16-bit storage formats.

The paper stores codebooks and scales in 16 bits (App. C, "Estimating Model
Size": 16 bits per codebook entry and per scale); activations are fp16 or bf16.
Decoding is exact in fp64. Encoding rounds to nearest, ties to even.
"""
from __future__ import annotations

import math

import numpy as np


def f16_bits_to_f64(bits) -> np.ndarray:
    """IEEE binary16 bit patterns -> exact fp64 values (subnormals included)."""
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float64)


def bf16_bits_to_f64(bits) -> np.ndarray:
    """bfloat16 bit patterns -> exact fp64 values.

    A bf16 number is the upper half of a binary32 number, so its value is the
    binary32 whose high 16 bits are the pattern and whose low 16 bits are zero.
    """
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def f16_bits_to_f32(bits) -> np.ndarray:
    """fp16 patterns -> float32 values (exact: binary16 is a subset of binary32)."""
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float32)


def f32_to_f16_bits(x32) -> np.ndarray:
    """float32 -> fp16 bits, round to nearest even (numpy's conversion)."""
    return np.asarray(x32, dtype=np.float32).astype(np.float16).view(np.uint16)


def f32_to_bf16_bits(x32) -> np.ndarray:
    """float32 -> bf16 bits, round to nearest even, by bit manipulation.

    Adding 0x7FFF plus the lowest kept bit to the 32-bit pattern and dropping the
    low half rounds the magnitude to nearest with ties to even; the carry moves
    into the exponent when the significand overflows, and a value that rounds
    past the largest finite bf16 becomes infinity, as round-to-nearest requires.
    NaN inputs map to a quiet NaN.
    """
    f = np.asarray(x32, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    keep_lsb = (u >> np.uint64(16)) & np.uint64(1)
    out = ((u + np.uint64(0x7FFF) + keep_lsb) >> np.uint64(16)).astype(np.uint16)
    nan = np.isnan(f)
    if np.any(nan):
        out = np.where(nan, np.uint16(0x7FC0), out).astype(np.uint16)
    return out


def round_to_format(x, fmt: str) -> np.ndarray:
    """Round fp64 values to nearest-even in ``fmt`` ("f16", "bf16", "f32"); return fp64.

    Format-generic definition used to pin the bit-level encoders: a binary
    format with p significand bits, minimum normal exponent emin and largest
    finite value xmax represents, near |x| in [2^e, 2^(e+1)), the multiples of
    2^(max(e, emin) - p + 1). Rounding is ``rint`` (ties to even) of x divided
    by that quantum, which is exact in fp64 because the quantum is a power of
    two. Values whose rounded magnitude exceeds xmax become infinity.
    """
    p, emin, xmax = {"f16": (11, -14, 65504.0),
                     "bf16": (8, -126, float(np.finfo(np.float32).max) * (1 - 2.0 ** -8) / (1 - 2.0 ** -24)),
                     "f32": (24, -126, float(np.finfo(np.float32).max))}[fmt]
    x = np.asarray(x, dtype=np.float64)
    out = np.empty_like(x)
    for idx, v in np.ndenumerate(x):
        if not math.isfinite(v) or v == 0.0:
            out[idx] = v
            continue
        e = math.frexp(abs(v))[1] - 1          # |v| in [2^e, 2^(e+1))
        q = max(e, emin) - p + 1
        r = float(np.rint(math.ldexp(v, -q)))
        r = math.ldexp(r, q)
        if abs(r) > xmax:
            r = math.copysign(math.inf, v)
        out[idx] = r
    return out


def ulp_of(x, fmt: str) -> np.ndarray:
    """Spacing of ``fmt`` numbers at the magnitude of each fp64 value (one unit in the last place)."""
    p, emin = {"f16": (11, -14), "bf16": (8, -126), "f32": (24, -126)}[fmt]
    x = np.abs(np.asarray(x, dtype=np.float64))
    e = np.where(x > 0, np.floor(np.log2(np.where(x > 0, x, 1.0))), emin)
    e = np.maximum(e, emin)
    return np.exp2(e - p + 1)
