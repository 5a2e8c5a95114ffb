"""Every GEMV kernel and every GEMM tiling, whatever the default dispatch picks (GPU).

aqmb_gemv_select runs a named kernel (direct gathers, matrix cores, lookup tables) and
aqmb_gemm_select a named tiling (16-row tiles; 256 x 128, 128 x 128, 128 x 64 tiles), so each one
is parity-tested against the oracle at every batch and token count, including the shapes the
default dispatch sends elsewhere. A kernel that cannot serve a case must refuse it with
EUNSUPPORTED and write nothing. Oracle and tolerance as in the other GEMV / GEMM tests.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from oracle import formats
from workloads import LayerSpec, make_layer, make_activations

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU hosts too; every test here is marked gpu
    pytest.skip("no GPU", allow_module_level=True)

import paper_2606_12876_amd as A  # noqa: E402
from gpu_helpers import GpuLayer, abs_terms, act_values, check_close, out_values, to_dev, TORCH_DT, A_DT  # noqa: E402

K = A.GemvKernel


def _serves(kernel, B, k, d_in, batch):
    """Which kernel serves which case (the header's aqmb_gemv_kernel table)."""
    if kernel == K.DIRECT:
        return B != 8 or (k <= 4 and d_in <= 16384)
    if kernel == K.MMA:
        return B != 16
    if kernel == K.LUT:
        return B == 8
    return True


CASES = [LayerSpec("ragged", 1000, 1032, seed=31), LayerSpec("M8", 520, 520, M=8, seed=34),
         LayerSpec("wide", 130, 16392, M=4, seed=38), LayerSpec("b4", 300, 1032, M=4, B=4, seed=51),
         LayerSpec("b16", 1030, 328, M=2, B=16, seed=35), LayerSpec("b16_M5", 70, 4104, M=5, B=16, seed=52),
         # 16-bit codes on rows longer than the LDS holds in x (20 blocks of 512 groups): x restaged per chunk
         LayerSpec("b16_long", 9, 81920, M=2, B=16, seed=54)]


@pytest.mark.parametrize("kernel", [K.DIRECT, K.MMA, K.LUT], ids=lambda k: k.name)
@pytest.mark.parametrize("spec", CASES, ids=lambda s: s.name)
def test_named_gemv_kernel_matches_oracle(kernel, spec):
    L = make_layer(spec)
    C, s = formats.f16_bits_to_f64(L.codebooks), formats.f16_bits_to_f64(L.scales)
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        for b in (1, 2, 3, 16):
            for xdt in ("f16", "bf16"):
                xbits = make_activations(L, b, xdt, heavy_tail=(b % 2 == 1))
                x = act_values(xbits, xdt)
                xd = to_dev(xbits).view(TORCH_DT[xdt])
                for k in sorted({1, 2, spec.M}):
                    y = torch.full((b, spec.d_out), 7.0, dtype=torch.float32, device="cuda")
                    if not _serves(kernel, spec.B, k, spec.d_in, b):
                        with pytest.raises(A.AqmbError) as ei:
                            A.gemv_select(gl.handle, k, xd, A_DT[xdt], b, y, A.DType.F32, kernel)
                        assert ei.value.status == A.Status.EUNSUPPORTED
                        torch.cuda.synchronize()
                        assert torch.all(y == 7.0)
                        continue
                    A.gemv_select(gl.handle, k, xd, A_DT[xdt], b, y, A.DType.F32, kernel)
                    torch.cuda.synchronize()
                    ref = oracle.linear(x, L.codes, C, s, k)
                    check_close(out_values(y), ref, "f32", f"{kernel.name} {spec.name} b={b} k={k} {xdt}",
                                terms=abs_terms(x, L.codes, C, s, k), n_terms=k * spec.d_in)


def test_named_gemv_kernel_rejects_unknown():
    L = make_layer(LayerSpec("u", 64, 64, seed=53))
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        x = torch.zeros((1, 64), dtype=torch.float16, device="cuda")
        y = torch.zeros((1, 64), dtype=torch.float32, device="cuda")
        with pytest.raises(A.AqmbError) as ei:
            A.gemv_select(gl.handle, 1, x, A.DType.F16, 1, y, A.DType.F32, 9)
        assert ei.value.status == A.Status.EINVAL


GEMM_CASES = [(1, 40, 264, 2, 8), (17, 257, 520, 3, 8), (300, 200, 264, 4, 8), (600, 130, 1032, 8, 8),
              (17, 257, 520, 3, 4), (300, 200, 264, 4, 4), (600, 130, 1032, 8, 4)]


@pytest.mark.parametrize("tiling", list(A.GemmTiling), ids=lambda t: t.name)
def test_named_gemm_tiling_matches_oracle(tiling):
    """Each tiling at token counts the default dispatch sends to another one, every shape."""
    for (n, d_out, d_in, M, B) in GEMM_CASES:
        L = make_layer(LayerSpec("g", d_out, d_in, M=M, B=B, seed=41 + n + B, act_dtype="bf16"))
        Xbits = make_activations(L, n, "bf16", heavy_tail=True)
        X = act_values(Xbits, "bf16")
        with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
            for k in sorted({1, M}):
                ref = oracle.gemm_reference(X, L.codes, L.codebooks, L.scales, k)
                Y = torch.empty((n, d_out), dtype=torch.float32, device="cuda")
                A.gemm_select(gl.handle, k, to_dev(Xbits).view(torch.bfloat16), n, Y, A.DType.F32, tiling)
                torch.cuda.synchronize()
                check_close(out_values(Y), ref, "f32", f"{tiling.name} n={n} {d_out}x{d_in} B={B} k={k}")
