"""Seeded synthetic inputs for the multi-bitwidth additive-codebook linear layer.

This module only draws random inputs and encodes them into the storage formats
(fp16 / bf16 bit patterns, uint8 / uint16 code planes). It holds none of the
method's arithmetic: no reconstruction, no product, no rounding of results.
Both the CPU oracle and the GPU path take their inputs from here, so the two
sides see the same bytes; neither side imports the other.

Recipe (one ``numpy.random.Generator(PCG64(seed))`` per layer, draws in this
order):

1. codebooks ``normal(0, 0.02/sqrt(M), (M, 2**B, g))`` -> fp16, the standard
   deviation is ``0.02/sqrt(M)`` so that a full sum of M codewords has a
   standard deviation near 0.02, a typical LLM weight scale;
2. codes ``integers(0, 2**B, (M, d_out, d_in/g))`` -> uint8 (B=8) or uint16
   (B=16), plane-major: plane m holds codebook m's index for every
   (output row, input group);
3. scales ``uniform(0.5, 1.5, d_out)`` -> fp16, one per output row;
4. activations ``normal(0, 1, (batch, d_in))`` -> fp16 or bf16 (round to
   nearest even); the heavy-tailed variant multiplies
   ``round(0.001*batch*d_in)`` positions, chosen without replacement, by 20
   before the cast. Calibration inputs of the distortion evaluator are drawn
   the same way (fp16, one input per row);
5. dense weights (distortion evaluator) ``normal(0, 0.02, (d_out, d_in))`` -> fp16.

Integer-valued variant (exactness tests of the distortion evaluator): the same
steps with codebook entries ``integers(-4, 5)``, scales drawn from {0.5, 1, 2},
inputs ``integers(-4, 5)`` and weights ``integers(-16, 17)``. Every product and
every partial sum of products of such values is an integer (or half-integer)
far below 2^24, so it is exact in fp32 whatever the summation order.

The shapes stand in for the projections of Llama-7B-class models (4096x4096,
11008x4096, 4096x11008, 14336x4096) quantized with M codebooks of 2**B
codewords of g=8 weights each, the setting of the paper's experiments (§6).
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional

import numpy as np

__all__ = ["Layer", "LayerSpec", "make_layer", "make_activations", "make_weights", "make_integer_layer",
           "make_integer_rows", "float_to_bf16_bits", "float_to_f16_bits", "CONFIGS", "config"]


def float_to_f16_bits(a: np.ndarray) -> np.ndarray:
    """fp64/fp32 values -> IEEE binary16 bit patterns (numpy's round-to-nearest-even)."""
    return np.asarray(a, dtype=np.float64).astype(np.float16).view(np.uint16)


def float_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """fp64 values -> bfloat16 bit patterns, rounding to nearest even.

    The value is first rounded to binary32 (exact for the draws used here up to
    one rounding; draws are then rounded once more), then the low 16 bits are
    rounded away with ties to even. NaN stays NaN.
    """
    f = np.asarray(a, dtype=np.float64).astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)
    nan = np.isnan(f)
    if nan.any():
        r = r.copy()
        r[nan] = 0x7FC0
    return r


@dataclasses.dataclass(frozen=True)
class LayerSpec:
    name: str
    d_out: int
    d_in: int
    g: int = 8
    M: int = 4
    B: int = 8
    seed: int = 0
    act_dtype: str = "f16"          # "f16" | "bf16"
    batches: tuple = (1,)
    ks: tuple = (1, 2, 3, 4)
    heavy_tail: bool = False
    n_tokens: int = 0               # >0: prefill GEMM workload


@dataclasses.dataclass
class Layer:
    spec: LayerSpec
    codes: np.ndarray      # [M][d_out][d_in/g] uint8 | uint16
    codebooks: np.ndarray  # [M][2**B][g] uint16 (fp16 bits)
    scales: np.ndarray     # [d_out] uint16 (fp16 bits)
    rng: np.random.Generator  # continues after the layer draws (activations come next)


def make_layer(spec: LayerSpec, seed: Optional[int] = None) -> Layer:
    """Draw codebooks, codes and scales for ``spec`` (steps 1-3 of the recipe)."""
    rng = np.random.Generator(np.random.PCG64(spec.seed if seed is None else seed))
    M, B, g = spec.M, spec.B, spec.g
    if spec.d_in % g:
        raise ValueError("d_in must be a multiple of g")
    cb = rng.normal(0.0, 0.02 / np.sqrt(M), size=(M, 1 << B, g))
    codebooks = float_to_f16_bits(cb)
    code_dt = np.uint8 if B <= 8 else np.uint16
    codes = rng.integers(0, 1 << B, size=(M, spec.d_out, spec.d_in // g), dtype=np.int64).astype(code_dt)
    scales = float_to_f16_bits(rng.uniform(0.5, 1.5, size=spec.d_out))
    return Layer(spec, codes, codebooks, scales, rng)


def make_activations(layer: Layer, rows: int, dtype: Optional[str] = None,
                     heavy_tail: Optional[bool] = None) -> np.ndarray:
    """Draw ``rows`` activation vectors of length d_in (step 4 of the recipe).

    Returns the bit patterns as uint16 in the requested storage dtype.
    """
    spec = layer.spec
    dtype = dtype or spec.act_dtype
    heavy = spec.heavy_tail if heavy_tail is None else heavy_tail
    x = layer.rng.normal(0.0, 1.0, size=(rows, spec.d_in))
    if heavy:
        n_out = int(round(0.001 * rows * spec.d_in))
        pos = layer.rng.choice(rows * spec.d_in, size=n_out, replace=False)
        x.reshape(-1)[pos] *= 20.0
    if dtype == "f16":
        return float_to_f16_bits(x)
    if dtype == "bf16":
        return float_to_bf16_bits(x)
    raise ValueError(dtype)


def make_calibration_inputs(layer: Layer, n: int) -> np.ndarray:
    """Draw n calibration inputs as the columns of X [d_in][n] in fp64 (step 6 of the recipe):
    normal(0, 1) scaled per input channel by exp(normal(0, 0.5)), with 0.5 % of the channels
    (at least one) scaled by 10 more (the outlier channels of LLM activations), so that the
    diagonal blocks of X X^T / n differ from group to group and are far from the identity."""
    spec = layer.spec
    sigma = np.exp(layer.rng.normal(0.0, 0.5, size=spec.d_in))
    n_big = max(1, int(round(0.005 * spec.d_in)))
    sigma[layer.rng.choice(spec.d_in, size=n_big, replace=False)] *= 10.0
    return layer.rng.normal(0.0, 1.0, size=(spec.d_in, n)) * sigma[:, None]


def make_weights(layer: Layer, std: float = 0.02) -> np.ndarray:
    """Draw a dense weight matrix [d_out][d_in], normal(0, std), as fp16 bits (step 5)."""
    spec = layer.spec
    return float_to_f16_bits(layer.rng.normal(0.0, std, size=(spec.d_out, spec.d_in)))


def make_integer_layer(spec: LayerSpec, seed: Optional[int] = None) -> Layer:
    """Integer-valued layer: codebook entries in [-4, 4], codes uniform, scales in {0.5, 1, 2}."""
    rng = np.random.Generator(np.random.PCG64(spec.seed if seed is None else seed))
    M, B, g = spec.M, spec.B, spec.g
    if spec.d_in % g:
        raise ValueError("d_in must be a multiple of g")
    codebooks = float_to_f16_bits(rng.integers(-4, 5, size=(M, 1 << B, g)).astype(np.float64))
    code_dt = np.uint8 if B <= 8 else np.uint16
    codes = rng.integers(0, 1 << B, size=(M, spec.d_out, spec.d_in // g), dtype=np.int64).astype(code_dt)
    scales = float_to_f16_bits(rng.choice(np.array([0.5, 1.0, 2.0]), size=spec.d_out))
    return Layer(spec, codes, codebooks, scales, rng)


def make_integer_rows(layer: Layer, rows: int, lim: int) -> np.ndarray:
    """``rows`` x d_in integers in [-lim, lim] as fp16 bits (inputs: lim 4, weights: lim 16)."""
    return float_to_f16_bits(layer.rng.integers(-lim, lim + 1, size=(rows, layer.spec.d_in)).astype(np.float64))


# The workloads: a small and a square layer, the up and down projections of a Llama-7B MLP, a
# layer with 2^16-entry codebooks, and a 2048-token prefill.
CONFIGS: List[LayerSpec] = [
    LayerSpec("tiny_1024x1024", 1024, 1024, seed=1, act_dtype="f16", batches=(1,)),
    LayerSpec("square_4096x4096", 4096, 4096, seed=2, act_dtype="f16", batches=(1, 4)),
    LayerSpec("mlp_up_11008x4096", 11008, 4096, seed=31, act_dtype="bf16", batches=(1, 8, 16), heavy_tail=True),
    LayerSpec("mlp_down_4096x11008", 4096, 11008, seed=32, act_dtype="bf16", batches=(1, 8, 16), heavy_tail=True),
    LayerSpec("b16_14336x4096", 14336, 4096, M=2, B=16, seed=4, act_dtype="f16", batches=(1,), ks=(1, 2)),
    LayerSpec("prefill_2048x4096x4096", 4096, 4096, seed=5, act_dtype="bf16", n_tokens=2048),
]


def config(name: str) -> LayerSpec:
    for c in CONFIGS:
        if c.name == name or c.name.startswith(name + "_"):
            return c
    raise KeyError(name)
