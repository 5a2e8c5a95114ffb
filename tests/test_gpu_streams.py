"""Calls on one layer from two streams at once (GPU).

A layer is the stored format (C, b, s) that Alg. 1 returns and is read-only after creation: every
compute call reads it and writes only the caller's outputs, and the kernels that need scratch
(the lookup-table GEMV, the prefix distortion) take it per call from the stream-ordered pool. So
GEMV (every kernel), GEMM, dequant and the distortion may run on two streams at the same time
on one layer; every result must still match the oracle and the single-stream result. Both
streams have the default priority.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from oracle import formats
from workloads import LayerSpec, make_layer, make_activations, make_weights

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU hosts too; every test here is marked gpu
    pytest.skip("no GPU", allow_module_level=True)

import paper_2606_12876_amd as A  # noqa: E402
from gpu_helpers import GpuLayer, act_values, check_close, out_values, to_dev  # noqa: E402


def test_two_streams_on_one_layer_match_the_oracle():
    spec = LayerSpec("streams", 2000, 2048, M=4, seed=700)
    L = make_layer(spec)
    C, s = formats.f16_bits_to_f64(L.codebooks), formats.f16_bits_to_f64(L.scales)
    xs = [make_activations(L, b, "f16") for b in (1, 3)]
    Xbits = make_activations(L, 200, "bf16")
    Wbits = make_weights(L)
    Cal = make_activations(L, 64, "f16")
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        h = gl.handle
        W = to_dev(Wbits).view(torch.float16)
        Xc = to_dev(Cal).view(torch.float16)
        X = to_dev(Xbits).view(torch.bfloat16)
        out = []
        reps = 6
        for i in range(2 * reps):                     # both streams queue their calls before any sync
            st = streams[i % 2]
            xb = xs[i % 2]
            b = xb.shape[0]
            k = 1 + i % 4
            x = to_dev(xb).view(torch.float16)
            torch.cuda.synchronize()                  # inputs uploaded before the streams read them
            o = {"k": k, "b": b, "x": xb}
            with torch.cuda.stream(st):
                o["y"] = {kern: torch.empty((b, spec.d_out), dtype=torch.float32, device="cuda")
                          for kern in (A.GemvKernel.AUTO, A.GemvKernel.LUT, A.GemvKernel.MMA)}
                for kern, y in o["y"].items():
                    A.gemv_select(h, k, x, A.DType.F16, b, y, A.DType.F32, kern, stream=st)
                o["Y"] = torch.empty((200, spec.d_out), dtype=torch.float32, device="cuda")
                A.gemm(h, k, X, 200, o["Y"], A.DType.F32, stream=st)
                o["W"] = torch.empty((spec.d_out, spec.d_in), dtype=torch.bfloat16, device="cuda")
                A.dequant(h, k, o["W"], A.DType.BF16, stream=st)
                o["D"] = torch.empty((4,), dtype=torch.float64, device="cuda")
                A.prefix_distortion(h, W, A.DType.F16, Xc, A.DType.F16, 64, o["D"], stream=st)
            o["xdev"] = x
            out.append(o)
        torch.cuda.synchronize()
        Dref = oracle.prefix_distortions(formats.f16_bits_to_f64(Wbits), L.codes, C, s, formats.f16_bits_to_f64(Cal))
        D0 = out[0]["D"].cpu().numpy()
        for o in out:
            k, xv = o["k"], formats.f16_bits_to_f64(o["x"])
            ref = oracle.linear(xv, L.codes, C, s, k)
            for kern, y in o["y"].items():
                check_close(out_values(y), ref, "f32", f"stream gemv {kern.name} k={k} b={o['b']}")
            gref = oracle.gemm_reference(act_values(Xbits, "bf16"), L.codes, L.codebooks, L.scales, k)
            check_close(out_values(o["Y"]), gref, "f32", f"stream gemm k={k}")
            wref = oracle.dequant_canonical(L.codes, L.codebooks, L.scales, k, "bf16")
            assert np.array_equal(o["W"].cpu().view(torch.int16).numpy().view(np.uint16), wref)
            d = o["D"].cpu().numpy()
            assert np.array_equal(d, D0)                 # fixed reduction order: identical on every call
            np.testing.assert_allclose(d, Dref, rtol=1e-5)
        # the same GEMV issued alone gives the same bits
        for o in out[:2]:
            y = torch.empty_like(o["y"][A.GemvKernel.LUT])
            A.gemv_select(h, o["k"], o["xdev"], A.DType.F16, o["b"], y, A.DType.F32, A.GemvKernel.LUT)
            torch.cuda.synchronize()
            assert torch.equal(y, o["y"][A.GemvKernel.LUT])
