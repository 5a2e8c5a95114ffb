"""The Python layer QuantLinear against the oracle (GPU).

QuantLinear serves y = x . W_k^T at any level k from one stored set of codes (section 5): up to
16 input rows through aqmb_gemv (fp16 or bf16 x), more through aqmb_gemm (bf16 x only; other
dtypes are refused, never converted). Both sides of the 16-row switch, both activation dtypes,
leading batch dimensions and the three code widths (B inferred from the codebook size).
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
from gpu_helpers import act_values, check_close, out_values, to_dev, TORCH_DT  # noqa: E402


def _module(L):
    codes = to_dev(L.codes)
    return A.QuantLinear(codes, to_dev(L.codebooks).view(torch.float16), to_dev(L.scales).view(torch.float16))


@pytest.mark.parametrize("B", [8, 4])
@pytest.mark.parametrize("xdt", ["f16", "bf16"])
def test_quantlinear_both_sides_of_the_row_switch(B, xdt):
    spec = LayerSpec("ql", 300, 520, M=4, B=B, seed=600 + B)
    L = make_layer(spec)
    C, s = formats.f16_bits_to_f64(L.codebooks), formats.f16_bits_to_f64(L.scales)
    q = _module(L)
    try:
        assert q.code_bits == B and (q.M, q.d_out, q.d_in) == (4, 300, 520)
        for n in (1, 16, 17, 300):
            xbits = make_activations(L, n, xdt, heavy_tail=True)
            x = to_dev(xbits).view(TORCH_DT[xdt])
            if n > 16 and xdt != "bf16":
                with pytest.raises(A.AqmbError) as ei:
                    q(x, 2)
                assert ei.value.status == A.Status.EUNSUPPORTED
                continue
            xv = act_values(xbits, xdt)
            for k in (1, 4):
                for out in (None, torch.float32):
                    y = q(x, k, out_dtype=out)
                    torch.cuda.synchronize()
                    assert y.shape == (n, 300) and y.dtype == (out or x.dtype)
                    if n <= 16:
                        ref = oracle.linear(xv, L.codes, C, s, k)
                    else:
                        ref = oracle.gemm_reference(xv, L.codes, L.codebooks, L.scales, k)
                    fmt = {torch.float16: "f16", torch.bfloat16: "bf16", torch.float32: "f32"}[y.dtype]
                    check_close(out_values(y), ref, fmt, f"QuantLinear B={B} n={n} k={k} {xdt} -> {fmt}")
    finally:
        q.close()


def test_quantlinear_leading_dims_and_dequant():
    spec = LayerSpec("ql3", 130, 264, M=3, seed=610, act_dtype="bf16")
    L = make_layer(spec)
    q = _module(L)
    try:
        xbits = make_activations(L, 2 * 3 * 5, "bf16")           # [2, 3, 5, d_in]: 30 rows -> GEMM
        x = to_dev(xbits).view(torch.bfloat16).reshape(2, 3, 5, 264)
        y = q(x, 3)
        torch.cuda.synchronize()
        assert y.shape == (2, 3, 5, 130)
        ref = oracle.gemm_reference(act_values(xbits, "bf16"), L.codes, L.codebooks, L.scales, 3)
        check_close(out_values(y.reshape(30, 130)), ref, "bf16", "leading dims")
        for k in (1, 3):
            W = q.dequant(k, torch.bfloat16)
            torch.cuda.synchronize()
            assert np.array_equal(W.cpu().view(torch.int16).numpy().view(np.uint16),
                                  oracle.dequant_canonical(L.codes, L.codebooks, L.scales, k, "bf16"))
    finally:
        q.close()


def test_quantlinear_16bit_codes():
    spec = LayerSpec("ql16", 200, 264, M=2, B=16, seed=620)
    L = make_layer(spec)
    C, s = formats.f16_bits_to_f64(L.codebooks), formats.f16_bits_to_f64(L.scales)
    q = _module(L)
    try:
        assert q.code_bits == 16
        xbits = make_activations(L, 5, "f16")
        for k in (1, 2):
            y = q(to_dev(xbits).view(torch.float16), k, out_dtype=torch.float32)
            torch.cuda.synchronize()
            check_close(out_values(y), oracle.linear(act_values(xbits, "f16"), L.codes, C, s, k), "f32", f"B=16 k={k}")
        X = to_dev(make_activations(L, 20, "bf16")).view(torch.bfloat16)
        with pytest.raises(A.AqmbError) as ei:                    # 20 rows: the GEMM has no 16-bit codes
            q(X, 1)
        assert ei.value.status == A.Status.EUNSUPPORTED
    finally:
        q.close()


def test_quantlinear_refuses_unknown_codebook_size():
    codes = torch.zeros((2, 8, 1), dtype=torch.uint8, device="cuda")
    with pytest.raises(A.AqmbError):
        A.QuantLinear(codes, torch.zeros((2, 32, 8), dtype=torch.float16, device="cuda"),
                      torch.ones(8, dtype=torch.float16, device="cuda"))
