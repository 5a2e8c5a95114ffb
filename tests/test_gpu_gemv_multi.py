"""aqmb_gemv_multi: several layers on one input in one call (GPU).

Each output must equal, bit for bit, the output of aqmb_gemv on that layer alone (the one-launch
kernels run the same per-row arithmetic in the same order), and the fp64 oracle within the GEMV
tolerance. Covers both one-launch paths (the direct-gather multi-layer kernel at batch 1; the
matrix-core grid over all layers' row blocks from batch 2, also with 4-bit codes), layers of
different heights, and the paths that fall back to one launch per layer.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from workloads import LayerSpec, make_layer, make_activations

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU hosts too; every test here is marked gpu
    pytest.skip("no GPU", allow_module_level=True)

import paper_2606_12876_amd as A  # noqa: E402
from gpu_helpers import GpuLayer, out_values, check_close, to_dev, TORCH_DT, A_DT, act_values  # noqa: E402


def _f64(L):
    from oracle import formats
    return formats.f16_bits_to_f64(L.codebooks), formats.f16_bits_to_f64(L.scales)


def _run(gls, k, xbits, xdt, ydt, multi=True):
    b = xbits.shape[0]
    x = to_dev(xbits).view(TORCH_DT[xdt])
    ys = [torch.full((b, gl.desc.d_out), 3.0, dtype=TORCH_DT[ydt], device="cuda") for gl in gls]
    if multi:
        A.gemv_multi([gl.handle for gl in gls], k, x, A_DT[xdt], b, ys, A_DT[ydt])
    else:
        for gl, y in zip(gls, ys):
            A.gemv(gl.handle, k, x, A_DT[xdt], b, y, A_DT[ydt])
    torch.cuda.synchronize()
    return [out_values(y) for y in ys]


def _check(specs, batches, ks, xdt="f16", ydts=("f32", "f16")):
    layers = [make_layer(s) for s in specs]
    gls = [GpuLayer(L.codes, L.codebooks, L.scales) for L in layers]
    try:
        for b in batches:
            xbits = make_activations(layers[0], b, xdt, heavy_tail=(b % 2 == 1))
            x = act_values(xbits, xdt)
            for k in ks:
                for ydt in ydts:
                    got = _run(gls, k, xbits, xdt, ydt)
                    one = _run(gls, k, xbits, xdt, ydt, multi=False)
                    for i, (L, g, o) in enumerate(zip(layers, got, one)):
                        assert np.array_equal(g, o), f"layer {i} b={b} k={k} {ydt}: differs from aqmb_gemv"
                        C, s = _f64(L)
                        check_close(g, oracle.linear(x, L.codes, C, s, k), ydt, f"layer {i} b={b} k={k} {ydt}")
    finally:
        for gl in gls:
            gl.close()


def test_fused_projections_full_size():
    """Three 4096 x 4096 layers on one input (the shape of fused q/k/v projections), every k."""
    specs = [LayerSpec(f"qkv{i}", 4096, 4096, seed=60 + i) for i in range(3)]
    _check(specs, (1, 4), (1, 2, 3, 4), ydts=("f16",))


def test_layers_of_different_heights():
    """Row blocks that some layers do not have are skipped; ragged groups (65 per row)."""
    specs = [LayerSpec("h300", 300, 520, M=3, seed=64), LayerSpec("h1000", 1000, 520, M=3, seed=65),
             LayerSpec("h17", 17, 520, M=3, seed=66), LayerSpec("h1", 1, 520, M=3, seed=67)]
    _check(specs, (1, 2, 3, 4), (1, 2, 3), xdt="bf16", ydts=("f32", "bf16"))


def test_single_layer_and_wide_rows():
    """One layer; rows of 1376 groups (d_in 11008, three 512-group blocks per thread)."""
    _check([LayerSpec("one", 700, 264, M=2, seed=68)], (1, 3), (1, 2))
    _check([LayerSpec("w0", 64, 11008, M=4, seed=69), LayerSpec("w1", 200, 11008, M=4, seed=70)], (1, 4), (2, 4),
           xdt="bf16", ydts=("bf16",))


def test_fallback_paths():
    """k > 4 at batch 1 and 16-bit codes take one launch per layer; k > 4 at batch 8 the
    matrix-core grid; results are the same."""
    _check([LayerSpec("m6a", 130, 136, M=6, seed=71), LayerSpec("m6b", 77, 136, M=6, seed=72)], (1, 8), (5, 6))
    _check([LayerSpec("b16a", 90, 64, M=2, B=16, seed=73), LayerSpec("b16b", 33, 64, M=2, B=16, seed=74)], (1, 2),
           (1, 2))


def test_mismatched_inputs_rejected_and_nothing_written():
    La = make_layer(LayerSpec("a", 64, 64, M=2, seed=75))
    Lb = make_layer(LayerSpec("b", 64, 128, M=2, seed=76))
    with GpuLayer(La.codes, La.codebooks, La.scales) as ga, GpuLayer(Lb.codes, Lb.codebooks, Lb.scales) as gb:
        x = torch.zeros((1, 128), dtype=torch.float16, device="cuda")
        ys = [torch.full((1, 64), 7.0, dtype=torch.float32, device="cuda") for _ in range(2)]
        with pytest.raises(A.AqmbError):
            A.gemv_multi([ga.handle, gb.handle], 1, x, A.DType.F16, 1, ys, A.DType.F32)   # d_in differs
        with pytest.raises(A.AqmbError):
            A.gemv_multi([ga.handle, ga.handle], 3, x, A.DType.F16, 1, ys, A.DType.F32)   # k > M
        torch.cuda.synchronize()
        assert all(torch.all(y == 7.0) for y in ys)


def test_matrix_core_grid_4bit_and_tall_layers():
    """4-bit layers from batch 2 share one matrix-core launch; a layer with more 16-row blocks than
    compute units (5000 rows: 313 blocks) next to a small one makes the call fall back to one
    launch per layer (the tall one on its persistent kernel)."""
    _check([LayerSpec("f4a", 300, 520, M=4, B=4, seed=77), LayerSpec("f4b", 64, 520, M=4, B=4, seed=78)],
           (2, 5), (1, 3, 4))
    _check([LayerSpec("tall", 5000, 520, M=4, seed=79), LayerSpec("small", 100, 520, M=4, seed=80)], (3, 16),
           (1, 4), xdt="bf16", ydts=("bf16",))


def test_matrix_core_grid_sixteen_layers():
    """AQMB_MAX_MULTI layers of ragged heights (1 to 481 rows) in one matrix-core launch: every
    slot of the launch's layer table in use, blocks of different layers interleaved in the grid."""
    assert A.MAX_MULTI == 16
    specs = [LayerSpec(f"s{i}", 1 + 32 * i, 264, M=3, seed=90 + i) for i in range(16)]
    _check(specs, (2, 9), (1, 3), ydts=("f32",))
