"""Layers with 4-bit codes (codebooks of 16 codewords): create, dequant, decode GEMV, prefill GEMM
and the prefix distortions on the GPU against the oracle.

The 4 x 4-bit configuration is the one the paper's ablation on codebook precision against
codebook count compares with 2 x 8 bits. The oracle is the same fp64 reconstruction and product
for any codebook size; dequant must be bit-exact under the canonical rounding, the GEMV within
the normwise tolerance of the other GEMV tests.
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
from gpu_helpers import GpuLayer, out_values, check_close, to_dev, TORCH_DT, A_DT, act_values  # noqa: E402


def _vals(L):
    return formats.f16_bits_to_f64(L.codebooks), formats.f16_bits_to_f64(L.scales)


@pytest.mark.parametrize("shape", [(77, 360, 4), (256, 1024, 4), (33, 8, 2), (130, 20000, 3), (64, 512, 8)])
def test_dequant_bit_exact(shape):
    d_out, d_in, M = shape
    L = make_layer(LayerSpec("b4", d_out, d_in, M=M, B=4, seed=300 + d_out))
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        for k in range(1, M + 1):
            for dt in ("bf16", "f16", "f32"):
                W = torch.empty((d_out, d_in), dtype=TORCH_DT[dt], device="cuda")
                A.dequant(gl.handle, k, W, A_DT[dt])
                torch.cuda.synchronize()
                ref = oracle.dequant_canonical(L.codes, L.codebooks, L.scales, k, dt)
                if dt == "f32":                              # binary32 values: compare their bits
                    got, ref = W.cpu().numpy().view(np.uint32), np.asarray(ref, dtype=np.float32).view(np.uint32)
                else:
                    got = W.cpu().view(torch.int16).numpy().view(np.uint16)
                assert np.array_equal(got, ref), f"{shape} k={k} {dt}"


@pytest.mark.parametrize("shape,batches", [((77, 360, 4), (1, 3, 16)), ((4096, 4096, 4), (1, 4)),
                                           ((130, 20000, 3), (1, 5)), ((64, 512, 8), (1, 8)),
                                           ((5000, 520, 4), (1, 2, 8))])
def test_gemv_matches_oracle(shape, batches):
    """Ragged rows and groups (360 = 45 groups: one partial 32-group slice), the benchmarked shape,
    a row longer than one 2048-group stage of x (20000 = 2500 groups), M = 8, and 313 blocks of 16
    rows (more than one per compute unit). Batch 1 on the 4-bit kernel, 2 and more on the matrix
    cores."""
    d_out, d_in, M = shape
    L = make_layer(LayerSpec("b4g", d_out, d_in, M=M, B=4, seed=310 + d_in))
    C, s = _vals(L)
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        for b in batches:
            for xdt in ("f16", "bf16"):
                xbits = make_activations(L, b, xdt, heavy_tail=(b % 2 == 1))
                x = to_dev(xbits).view(TORCH_DT[xdt])
                xv = act_values(xbits, xdt)
                for k in sorted({1, M // 2 or 1, M}):
                    ref = oracle.linear(xv, L.codes, C, s, k)
                    for ydt in ("f32", "f16") if xdt == "f16" else ("bf16",):
                        y = torch.full((b, d_out), 7.0, dtype=TORCH_DT[ydt], device="cuda")
                        A.gemv(gl.handle, k, x, A_DT[xdt], b, y, A_DT[ydt])
                        torch.cuda.synchronize()
                        check_close(out_values(y), ref, ydt, f"{shape} b={b} k={k} {xdt}->{ydt}")


def test_codes_above_15_rejected():
    L = make_layer(LayerSpec("bad", 8, 64, M=2, B=4, seed=320))
    codes = L.codes.copy()
    codes[1, 5, 3] = 16
    desc = A.make_desc(8, 64, 2, 4)
    with pytest.raises(A.AqmbError) as ei:
        A.create(desc, to_dev(codes), to_dev(L.codebooks), to_dev(L.scales))
    assert ei.value.status == A.Status.EINVAL and "15" in A.last_error()


@pytest.mark.parametrize("n", [1, 70, 300, 1100])
def test_gemm_matches_oracle(n):
    """Both tilings (16-row up to 192 tokens, large tiles above: 300 and 1100 tokens span ragged
    token and row tiles and a ragged last K step); same weight rounding (the binary32 fold rounded
    to bf16) as the reference."""
    L = make_layer(LayerSpec("g4", 200, 1032, M=4, B=4, seed=340 + n, act_dtype="bf16"))
    Xbits = make_activations(L, n, "bf16", heavy_tail=True)
    X = act_values(Xbits, "bf16")
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        for k in (1, 2, 4):
            ref = oracle.gemm_reference(X, L.codes, L.codebooks, L.scales, k)
            for ydt in ("f32", "bf16"):
                Y = torch.empty((n, 200), dtype=TORCH_DT[ydt], device="cuda")
                A.gemm(gl.handle, k, to_dev(Xbits).view(torch.bfloat16), n, Y, A_DT[ydt])
                torch.cuda.synchronize()
                check_close(out_values(Y), ref, ydt, f"gemm n={n} k={k} {ydt}")


def test_gemm_full_size():
    """The prefill shape (2048 tokens x 4096 x 4096, 4 codebooks of 16 codewords): every output
    against the reference, at k = 1 and 4."""
    L = make_layer(LayerSpec("g4full", 4096, 4096, M=4, B=4, seed=345, act_dtype="bf16"))
    n = 2048
    Xbits = make_activations(L, n, "bf16")
    X = act_values(Xbits, "bf16")
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        Xd = to_dev(Xbits).view(torch.bfloat16)
        for k in (1, 4):
            Y = torch.empty((n, 4096), dtype=torch.bfloat16, device="cuda")
            A.gemm(gl.handle, k, Xd, n, Y, A.DType.BF16)
            torch.cuda.synchronize()
            ref = oracle.gemm_reference(X, L.codes, L.codebooks, L.scales, k)
            check_close(out_values(Y), ref, "bf16", f"gemm 2048x4096x4096 B=4 k={k}")


@pytest.mark.parametrize("M", [4, 6, 8])
def test_prefix_distortion_matches_oracle(M):
    """4-bit codes through the distortion kernel's layouts (two sample blocks per wave up to M = 5,
    one beyond)."""
    from workloads import make_weights
    L = make_layer(LayerSpec("d4", 257, 520, M=M, B=4, seed=350 + M))
    Wb = make_weights(L)
    Xb = make_activations(L, 150, "f16")
    C, s = _vals(L)
    ref = oracle.prefix_distortions(formats.f16_bits_to_f64(Wb), L.codes, C, s, formats.f16_bits_to_f64(Xb))
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        D = torch.empty(M, dtype=torch.float64, device="cuda")
        A.prefix_distortion(gl.handle, to_dev(Wb).view(torch.float16), A.DType.F16, to_dev(Xb).view(torch.float16),
                            A.DType.F16, 150, D)
        torch.cuda.synchronize()
        np.testing.assert_allclose(D.cpu().numpy(), ref, rtol=1e-5)


def test_multi_layer_calls_mix_code_widths():
    """aqmb_gemv_multi runs 4-bit layers one launch each, with results equal to aqmb_gemv."""
    L4 = make_layer(LayerSpec("m4", 96, 256, M=2, B=4, seed=330))
    L8 = make_layer(LayerSpec("m8", 40, 256, M=2, B=8, seed=331))
    with GpuLayer(L4.codes, L4.codebooks, L4.scales) as g4, GpuLayer(L8.codes, L8.codebooks, L8.scales) as g8:
        for b in (1, 2, 5):
            xbits = make_activations(L4, b, "f16")
            x = to_dev(xbits).view(torch.float16)
            ys = [torch.empty((b, 96), dtype=torch.float32, device="cuda"), torch.empty((b, 40), dtype=torch.float32, device="cuda")]
            A.gemv_multi([g4.handle, g8.handle], 2, x, A.DType.F16, b, ys, A.DType.F32)
            y1 = [torch.empty_like(t) for t in ys]
            A.gemv(g4.handle, 2, x, A.DType.F16, b, y1[0], A.DType.F32)
            A.gemv(g8.handle, 2, x, A.DType.F16, b, y1[1], A.DType.F32)
            torch.cuda.synchronize()
            assert torch.equal(ys[0], y1[0]) and torch.equal(ys[1], y1[1])
