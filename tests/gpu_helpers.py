"""Shared helpers for the GPU parity tests: upload a seeded layer through the C ABI, and the
tolerance check the parity tests apply.

Tolerance (floating-point outputs): for every element,
    |y_gpu - y_ref| <= 2e-3 * max|y_ref| + 0.5 * ulp_out(y_ref)
where y_ref is the oracle's fp64 value and ulp_out the spacing of the output format at
|y_ref|. The first term is the stated bound on accumulated error, normalised by the largest
output (normwise, infinity norm); the second is the one rounding of the result into the
output format, which for bf16 alone can reach 2^-8 of a value, more than 2e-3. For F32
outputs the second term is negligible and the check is the plain normwise bound.
"""
from __future__ import annotations

import numpy as np
import torch

import oracle  # noqa: F401
from oracle import formats
import paper_2606_12876_amd as A

TOL = 2e-3

NP_TO_TORCH = {np.uint8: torch.uint8, np.uint16: torch.int16, np.int16: torch.int16}


def to_dev(a: np.ndarray) -> torch.Tensor:
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).cuda()


class GpuLayer:
    def __init__(self, codes, codebooks, scales, B=None):
        M, d_out, G = codes.shape
        if B is None:          # from the codebook size: 16, 256 or 65536 codewords
            B = {16: 4, 256: 8, 65536: 16}[codebooks.shape[1]]
        self.desc = A.make_desc(d_out, G * 8, M, B)
        self.codes, self.codebooks, self.scales = codes, codebooks, scales
        c, cb, s = to_dev(codes), to_dev(codebooks), to_dev(scales)
        self.handle = A.create(self.desc, c, cb, s)
        torch.cuda.synchronize()

    def close(self):
        if self.handle:
            A.destroy(self.handle)
            self.handle = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


def out_values(y: torch.Tensor) -> np.ndarray:
    """Device output -> exact fp64 numpy values."""
    y = y.cpu()
    if y.dtype == torch.float32:
        return y.numpy().astype(np.float64)
    bits = y.view(torch.int16).numpy().view(np.uint16)
    return formats.f16_bits_to_f64(bits) if y.dtype == torch.float16 else formats.bf16_bits_to_f64(bits)


def check_close(y_gpu: np.ndarray, y_ref: np.ndarray, fmt: str, what: str = ""):
    assert y_gpu.shape == y_ref.shape, (y_gpu.shape, y_ref.shape)
    assert np.all(np.isfinite(y_gpu)), f"{what}: non-finite output"
    scale = float(np.max(np.abs(y_ref))) if y_ref.size else 0.0
    bound = TOL * scale + 0.5 * formats.ulp_of(y_ref, fmt)
    err = np.abs(y_gpu - y_ref)
    worst = float(np.max(err / np.maximum(bound, 1e-300))) if err.size else 0.0
    normwise = float(np.max(err) / scale) if scale > 0 else 0.0
    assert np.all(err <= bound), f"{what}: max err/bound = {worst:.3f}, normwise err = {normwise:.3e}"
    return normwise


TORCH_DT = {"f16": torch.float16, "bf16": torch.bfloat16, "f32": torch.float32}
A_DT = {"f16": A.DType.F16, "bf16": A.DType.BF16, "f32": A.DType.F32}


def act_values(bits: np.ndarray, dt: str) -> np.ndarray:
    return formats.f16_bits_to_f64(bits) if dt == "f16" else formats.bf16_bits_to_f64(bits)
