"""Shared helpers for the GPU parity tests: upload a seeded layer through the C ABI, and the
tolerance checks the parity tests apply.

Tolerance (floating-point outputs), three checks on every element i, all required:
  1. normwise (the stated "max relative error 2e-3", read against the largest output):
       |y_gpu - y_ref| <= 2e-3 * max|y_ref| + 0.5 * ulp_out(y_ref)
  2. per element, above a floor: where |y_ref_i| >= 1e-2 * max|y_ref|,
       |y_gpu_i - y_ref_i| <= 2e-3 * |y_ref_i| + 0.5 * ulp_out(y_ref_i)
     so that an error confined to small outputs cannot hide under the largest one;
  3. fp32 outputs, when the caller gives the sum of absolute products T_i = sum |x_t w_t| over
     the n terms the kernel adds (every product of the method's fp16 / bf16 operands is exact in
     fp32): the rounding bound of fp32 summation in any order,
       |y_gpu_i - y_ref_i| <= 2 n u T_i + 2 u |y_ref_i|,   u = 2^-24
     (twice the classical (n - 1) u, leaving room for the matrix cores' internal order; the
     second term is the row scale's multiply).
y_ref is the oracle's fp64 value and ulp_out the spacing of the output format at |y_ref|; the
half-ulp term is the one rounding of the result into the output format, which for bf16 alone
can reach 2^-8 of a value, more than 2e-3.
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


U32 = 2.0 ** -24
FLOOR = 1e-2


def check_close(y_gpu: np.ndarray, y_ref: np.ndarray, fmt: str, what: str = "", terms=None, n_terms=None):
    assert y_gpu.shape == y_ref.shape, (y_gpu.shape, y_ref.shape)
    assert np.all(np.isfinite(y_gpu)), f"{what}: non-finite output"
    scale = float(np.max(np.abs(y_ref))) if y_ref.size else 0.0
    half_ulp = 0.5 * formats.ulp_of(y_ref, fmt)
    bound = TOL * scale + half_ulp
    err = np.abs(y_gpu - y_ref)
    worst = float(np.max(err / np.maximum(bound, 1e-300))) if err.size else 0.0
    normwise = float(np.max(err) / scale) if scale > 0 else 0.0
    assert np.all(err <= bound), f"{what}: max err/bound = {worst:.3f}, normwise err = {normwise:.3e}"
    big = np.abs(y_ref) >= FLOOR * scale
    if scale > 0 and np.any(big):
        eb = TOL * np.abs(y_ref[big]) + half_ulp[big]
        rel = float(np.max(err[big] / np.abs(y_ref[big])))
        assert np.all(err[big] <= eb), f"{what}: per-element error above the floor, max relative {rel:.3e}"
    if terms is not None and fmt == "f32":
        assert n_terms is not None
        tb = 2.0 * n_terms * U32 * np.asarray(terms) + 2.0 * U32 * np.abs(y_ref)
        ratio = float(np.max(err / np.maximum(tb, 1e-300))) if err.size else 0.0
        assert np.all(err <= tb), f"{what}: fp32 summation bound exceeded, max err/bound = {ratio:.3f}"
    return normwise


def abs_terms(x, codes, codebooks_f64, scales_f64, k):
    """T[b][i] = sum_t sum_{m<k} |x[b][t]| |s_i C_m[codes[m,i,j(t)]][t]|: the absolute products a
    GEMV adds (one per input, plane and output); n = k d_in of them per output."""
    import oracle
    return oracle.linear(np.abs(x), codes, np.abs(codebooks_f64), np.abs(scales_f64), k)


TORCH_DT = {"f16": torch.float16, "bf16": torch.bfloat16, "f32": torch.float32}
A_DT = {"f16": A.DType.F16, "bf16": A.DType.BF16, "f32": A.DType.F32}


def act_values(bits: np.ndarray, dt: str) -> np.ndarray:
    return formats.f16_bits_to_f64(bits) if dt == "f16" else formats.bf16_bits_to_f64(bits)
