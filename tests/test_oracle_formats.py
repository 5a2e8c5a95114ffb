"""Pins for the oracle's 16-bit encodings and decodings (CPU only).

The oracle's bf16 encoder is its own bit manipulation and its fp16 encoder is
numpy's conversion; both are pinned against hand-derived IEEE cases, against a
format-generic rounding definition, and against torch's conversions (an
independent library routine for the same operation).
"""
import json
import os

import numpy as np
import pytest
import torch

from oracle import formats

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _f32_from_hex(h):
    return np.array([int(h, 16)], dtype=np.uint32).view(np.float32)


def test_rne_hand_cases():
    cases = json.load(open(os.path.join(GOLD, "rne_cases.json")))["cases"]
    for f32hex, bf16hex, f16hex, why in cases:
        x = _f32_from_hex(f32hex)
        assert int(formats.f32_to_bf16_bits(x)[0]) == int(bf16hex, 16), why
        assert int(formats.f32_to_f16_bits(x)[0]) == int(f16hex, 16), why


def _random_f32(n, seed):
    rng = np.random.default_rng(seed)
    bits = rng.integers(0, 2 ** 32, size=n, dtype=np.uint64).astype(np.uint32)
    x = bits.view(np.float32)
    x = x[np.isfinite(x)]
    # add values concentrated near rounding boundaries and in the fp16 range
    near = (rng.normal(0, 1, n) * 2.0 ** rng.integers(-30, 20, n)).astype(np.float32)
    ties = (np.float32(1) + np.arange(n, dtype=np.float32) * np.float32(2.0 ** -8)).astype(np.float32)
    return np.concatenate([x, near, ties])


def test_bf16_encoder_matches_torch():
    x = _random_f32(200000, 1)
    ours = formats.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_f16_encoder_matches_torch():
    x = _random_f32(200000, 2)
    ours = formats.f32_to_f16_bits(x)
    ref = torch.from_numpy(x).to(torch.float16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


@pytest.mark.parametrize("fmt", ["f16", "bf16"])
def test_encoders_match_generic_rounding(fmt):
    rng = np.random.default_rng(3)
    x = (rng.normal(0, 1, 4000) * 2.0 ** rng.integers(-28, 17, 4000)).astype(np.float32)
    x = np.concatenate([x, np.float32([65504, 65519, 65520, 2 ** -24, 2 ** -25, 3 * 2 ** -26, -0.0, 0.0])])
    enc = formats.f32_to_bf16_bits(x) if fmt == "bf16" else formats.f32_to_f16_bits(x)
    dec = formats.bf16_bits_to_f64(enc) if fmt == "bf16" else formats.f16_bits_to_f64(enc)
    generic = formats.round_to_format(x.astype(np.float64), fmt)
    assert np.array_equal(dec, generic)


def test_decoders_exact():
    # every fp16 pattern decodes to the value sign * 2^(e-15) * (1 + f/1024) (normal) or f * 2^-24 (subnormal)
    bits = np.arange(0, 2 ** 16, dtype=np.uint32).astype(np.uint16)
    v = formats.f16_bits_to_f64(bits)
    sign = np.where(bits >> 15, -1.0, 1.0)
    e = (bits >> 10) & 0x1F
    f = (bits & 0x3FF).astype(np.float64)
    expect = np.where(e == 0, f * 2.0 ** -24, (1 + f / 1024) * np.exp2(e.astype(np.float64) - 15)) * sign
    finite = e != 31
    assert np.array_equal(v[finite], expect[finite])
    # bf16: value = sign * 2^(e-127) * (1 + f/128) for normal patterns, f * 2^-133 for subnormal ones
    vb = formats.bf16_bits_to_f64(bits)
    eb = (bits >> 7) & 0xFF
    fb = (bits & 0x7F).astype(np.float64)
    expb = np.where(eb == 0, fb * 2.0 ** -133, (1 + fb / 128) * np.exp2(eb.astype(np.float64) - 127)) * sign
    finb = eb != 255
    assert np.array_equal(vb[finb], expb[finb])


def test_ulp_of():
    assert formats.ulp_of(1.0, "bf16") == 2.0 ** -7
    assert formats.ulp_of(1.0, "f16") == 2.0 ** -10
    assert formats.ulp_of(1.999, "f16") == 2.0 ** -10
    assert formats.ulp_of(2.0 ** -20, "f16") == 2.0 ** -24   # subnormal spacing
    assert formats.ulp_of(0.0, "f16") == 2.0 ** -24
