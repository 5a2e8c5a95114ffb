"""Run-time loading and dropping of code planes (GPU).

A layer created with only its first r planes, then grown and shrunk, must at every resident level
match the oracle (dequant bit-exact to the canonical rounding, GEMV and GEMM within the parity
tolerance) and give bit-identical results to a layer created with all planes, and it must refuse
levels that need planes it does not hold (the multi-bitwidth property: level k reads planes
0..k-1 only).
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
from gpu_helpers import GpuLayer, abs_terms, check_close, out_values, to_dev  # noqa: E402


def _outputs(h, k, x, d_out, d_in, X):
    y = torch.empty((x.shape[0], d_out), dtype=torch.float32, device="cuda")
    A.gemv(h, k, x, A.DType.F16, x.shape[0], y, A.DType.F32)
    W = torch.empty((d_out, d_in), dtype=torch.bfloat16, device="cuda")
    A.dequant(h, k, W, A.DType.BF16)
    out = [y, W]
    if X is not None:
        Y = torch.empty((X.shape[0], d_out), dtype=torch.float32, device="cuda")
        A.gemm(h, k, X, X.shape[0], Y, A.DType.F32)
        out.append(Y)
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("B", [8, 4, 16])
def test_grow_and_shrink_match_full_layer(B):
    spec = LayerSpec("planes", 200, 264, M=4 if B != 16 else 2, B=B, seed=400 + B)
    L = make_layer(spec)
    M = spec.M
    desc = A.make_desc(spec.d_out, spec.d_in, M, B)
    xb = make_activations(L, 3, "f16")
    x = to_dev(xb).view(torch.float16)
    Xbits = make_activations(L, 70, "bf16") if B != 16 else None
    X = to_dev(Xbits).view(torch.bfloat16) if B != 16 else None
    C, s = formats.f16_bits_to_f64(L.codebooks), formats.f16_bits_to_f64(L.scales)
    x64 = formats.f16_bits_to_f64(xb)

    def oracle_check(got, k):
        """The prefix layer's outputs at level k against the oracle."""
        ref = oracle.linear(x64, L.codes, C, s, k)
        check_close(out_values(got[0]), ref, "f32", f"prefix B={B} gemv k={k}",
                    terms=abs_terms(x64, L.codes, C, s, k), n_terms=k * spec.d_in)
        wref = oracle.dequant_canonical(L.codes, L.codebooks, L.scales, k, "bf16")
        assert np.array_equal(got[1].cpu().view(torch.int16).numpy().view(np.uint16), wref), f"prefix B={B} dequant k={k}"
        if X is not None:
            gref = oracle.gemm_reference(formats.bf16_bits_to_f64(Xbits), L.codes, L.codebooks, L.scales, k)
            check_close(out_values(got[2]), gref, "f32", f"prefix B={B} gemm k={k}")
    cb, sc = to_dev(L.codebooks), to_dev(L.scales)
    with GpuLayer(L.codes, L.codebooks, L.scales) as full:
        ref = {k: _outputs(full.handle, k, x, spec.d_out, spec.d_in, X) for k in range(1, M + 1)}
        h = A.create_prefix(desc, 1, to_dev(L.codes[:1]), cb, sc)
        try:
            assert A.resident_planes(h) == 1
            def same(k):
                got = _outputs(h, k, x, spec.d_out, spec.d_in, X)
                oracle_check(got, k)
                for a, b in zip(got, ref[k]):
                    assert torch.equal(a, b), f"B={B} k={k}"
            def refused(k):
                y = torch.empty((3, spec.d_out), dtype=torch.float32, device="cuda")
                with pytest.raises(A.AqmbError) as ei:
                    A.gemv(h, k, x, A.DType.F16, 3, y, A.DType.F32)
                assert ei.value.status == A.Status.EINVAL and "resident" in A.last_error()
            same(1)
            if M > 1:
                refused(2)
                A.load_planes(h, M - 1, to_dev(L.codes[1:]))
                assert A.resident_planes(h) == M
                for k in range(1, M + 1):
                    same(k)
                A.drop_planes(h, 1)
                assert A.resident_planes(h) == 1
                same(1)
                refused(M)
                A.load_planes(h, 1, to_dev(L.codes[1:2]))
                same(2)
        finally:
            A.destroy(h)


def test_distortion_covers_resident_levels():
    spec = LayerSpec("dist", 130, 136, M=4, seed=410)
    L = make_layer(spec)
    desc = A.make_desc(spec.d_out, spec.d_in, 4, 8)
    Wb = make_weights(L)
    Xb = make_activations(L, 40, "f16")
    C = formats.f16_bits_to_f64(L.codebooks)
    s = formats.f16_bits_to_f64(L.scales)
    ref = oracle.prefix_distortions(formats.f16_bits_to_f64(Wb), L.codes, C, s, formats.f16_bits_to_f64(Xb))
    h = A.create_prefix(desc, 2, to_dev(L.codes[:2]), to_dev(L.codebooks), to_dev(L.scales))
    try:
        D = torch.full((4,), -1.0, dtype=torch.float64, device="cuda")
        A.prefix_distortion(h, to_dev(Wb).view(torch.float16), A.DType.F16, to_dev(Xb).view(torch.float16),
                            A.DType.F16, 40, D)
        torch.cuda.synchronize()
        d = D.cpu().numpy()
        np.testing.assert_allclose(d[:2], ref[:2], rtol=1e-5)
        assert np.all(d[2:] == -1.0)                 # only the resident levels are written
    finally:
        A.destroy(h)


def test_plane_calls_reject_bad_arguments():
    spec = LayerSpec("rej", 64, 64, M=3, seed=420)
    L = make_layer(spec)
    desc = A.make_desc(64, 64, 3, 8)
    cb, sc = to_dev(L.codebooks), to_dev(L.scales)
    for r in (0, 4):
        with pytest.raises(A.AqmbError):
            A.create_prefix(desc, r, to_dev(L.codes), cb, sc)
    h = A.create_prefix(desc, 2, to_dev(L.codes[:2]), cb, sc)
    try:
        with pytest.raises(A.AqmbError):
            A.load_planes(h, 2, to_dev(L.codes[:2]))     # would exceed M
        with pytest.raises(A.AqmbError):
            A.drop_planes(h, 3)                          # more than resident
        with pytest.raises(A.AqmbError):
            A.drop_planes(h, 0)
        assert A.resident_planes(h) == 2
        L4 = make_layer(LayerSpec("b4", 64, 64, M=2, B=4, seed=421))
        codes4 = L4.codes.copy()
        codes4[1, 0, 0] = 20
        h4 = A.create_prefix(A.make_desc(64, 64, 2, 4), 1, to_dev(codes4[:1]), to_dev(L4.codebooks), to_dev(L4.scales))
        try:
            with pytest.raises(A.AqmbError):
                A.load_planes(h4, 1, to_dev(codes4[1:]))  # a 4-bit code above 15
            assert A.resident_planes(h4) == 1
        finally:
            A.destroy(h4)
    finally:
        A.destroy(h)
