"""The allocation-free prefix distortion against the allocating one (GPU).

aqmb_prefix_distortion_noalloc runs the same kernels as aqmb_prefix_distortion with the library's
fixed per-device scratch instead of per-call scratch, so on the same inputs the two must agree bit
for bit, on consecutive calls that reuse the fixed scratch (the second with a smaller layer and
fewer calibration inputs, so fewer workgroups write it), and under HIP graph capture, the case it
exists for (replayed several times with other work in between).
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
from gpu_helpers import GpuLayer, to_dev  # noqa: E402


def _case(spec, n):
    L = make_layer(spec)
    Wb = make_weights(L)
    Xb = make_activations(L, n, "f16")
    return L, Wb, Xb


def _both(gl, Wb, Xb, n, M):
    W = to_dev(Wb).view(torch.float16)
    X = to_dev(Xb).view(torch.float16)
    D0 = torch.full((M,), -1.0, dtype=torch.float64, device="cuda")
    D1 = torch.full((M,), -2.0, dtype=torch.float64, device="cuda")
    A.prefix_distortion(gl.handle, W, A.DType.F16, X, A.DType.F16, n, D0)
    A.prefix_distortion_noalloc(gl.handle, W, A.DType.F16, X, A.DType.F16, n, D1)
    torch.cuda.synchronize()
    return D0.cpu().numpy(), D1.cpu().numpy()


def test_noalloc_matches_allocating_entry_point_twice():
    big = LayerSpec("na_big", 1500, 1032, M=4, seed=800)
    small = LayerSpec("na_small", 130, 264, M=3, seed=801)
    for spec, n in ((big, 300), (small, 40)):            # the second call: fewer rows, inputs and levels
        L, Wb, Xb = _case(spec, n)
        with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
            d_alloc, d_fixed = _both(gl, Wb, Xb, n, spec.M)
        assert np.array_equal(d_alloc, d_fixed), (spec.name, d_alloc, d_fixed)
        C, s = formats.f16_bits_to_f64(L.codebooks), formats.f16_bits_to_f64(L.scales)
        ref = oracle.prefix_distortions(formats.f16_bits_to_f64(Wb), L.codes, C, s, formats.f16_bits_to_f64(Xb))
        np.testing.assert_allclose(d_fixed, ref, rtol=1e-5)


def test_noalloc_under_graph_capture():
    spec = LayerSpec("na_graph", 700, 520, M=4, seed=802)
    n = 96
    L, Wb, Xb = _case(spec, n)
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        d_alloc, _ = _both(gl, Wb, Xb, n, spec.M)
        W = to_dev(Wb).view(torch.float16)
        X = to_dev(Xb).view(torch.float16)
        D = torch.zeros((spec.M,), dtype=torch.float64, device="cuda")
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            A.prefix_distortion_noalloc(gl.handle, W, A.DType.F16, X, A.DType.F16, n, D)
        torch.cuda.synchronize()
        for rep in range(4):
            D.fill_(-3.0)                                   # eager work between replays
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            assert np.array_equal(D.cpu().numpy(), d_alloc), f"replay {rep}"
        del g


def test_noalloc_rejects_like_the_allocating_call():
    spec = LayerSpec("na_rej", 64, 64, M=2, seed=803)
    L = make_layer(spec)
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        W = torch.zeros((64, 64), dtype=torch.float16, device="cuda")
        X = torch.zeros((4, 64), dtype=torch.float16, device="cuda")
        D = torch.zeros((2,), dtype=torch.float64, device="cuda")
        for args in ((W, A.DType.F16, X, A.DType.F16, 0), (W, A.DType.BF16, X, A.DType.F16, 4)):
            with pytest.raises(A.AqmbError):
                A.prefix_distortion_noalloc(gl.handle, args[0], args[1], args[2], args[3], args[4], D)
