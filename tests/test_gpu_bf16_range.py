"""bf16 activations far outside fp16's range and 8-value groups with a wide dynamic range: the
decode GEMV (direct-gather and 4-bit kernels at batch 1, matrix-core kernel from batch 2, in
both its bf16 forms: the exact codeword split at low k, the per-run conversion above; and its
persistent variant on a layer with more row blocks than compute units, x held across blocks or
reloaded with every item) against the fp64 oracle, fp32 output.

The direct-gather and 4-bit kernels represent each bf16 group as fp16 values times a power of two
that puts the group maximum in [2^14, 2^15), the matrix-core kernel each batch row's 128 inputs of
a run; values more than 2^29 below that maximum are rounded. The outputs must stay within the
usual tolerance and, at fp32 output, close to fp32 summation accuracy.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from oracle import formats
from workloads import LayerSpec, make_layer, float_to_bf16_bits

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU hosts too; every test here is marked gpu
    pytest.skip("no GPU", allow_module_level=True)

import paper_2606_12876_amd as A  # noqa: E402
from gpu_helpers import GpuLayer, out_values, check_close, to_dev, act_values  # noqa: E402


def _x(kind: str, b: int, d_in: int, seed: int) -> np.ndarray:
    rng = np.random.default_rng(seed)
    x = rng.normal(0.0, 1.0, size=(b, d_in))
    if kind == "huge":
        x *= 1e30
    elif kind == "tiny":
        x *= 1e-30
    elif kind == "wide":                                   # 24 decades inside every group
        x *= 10.0 ** rng.uniform(-12.0, 12.0, size=(b, d_in))
    elif kind == "over_fp16":                              # beyond 65504, next to ordinary values
        x[:, ::8] *= 1e6
    return float_to_bf16_bits(x)


@pytest.mark.parametrize("B", [8, 4])
@pytest.mark.parametrize("kind", ["huge", "tiny", "wide", "over_fp16"])
def test_bf16_range(kind, B):
    L = make_layer(LayerSpec("rng", 96, 1032, M=4, B=B, seed=400 + B, act_dtype="bf16"))
    C, s = formats.f16_bits_to_f64(L.codebooks), formats.f16_bits_to_f64(L.scales)
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        for b in (1, 2, 4, 8, 16):
            xbits = _x(kind, b, 1032, seed=410 + b)
            xv = act_values(xbits, "bf16")
            x = to_dev(xbits).view(torch.bfloat16)
            for k in (1, 2, 3, 4):
                ref = oracle.linear(xv, L.codes, C, s, k)
                y = torch.empty((b, 96), dtype=torch.float32, device="cuda")
                A.gemv(gl.handle, k, x, A.DType.BF16, b, y, A.DType.F32)
                torch.cuda.synchronize()
                got = out_values(y)
                normwise = check_close(got, ref, "f32", f"{kind} B={B} b={b} k={k}")
                assert normwise < 1e-5, f"{kind} B={B} b={b} k={k}: normwise error {normwise:.2e}"


@pytest.mark.parametrize("kind", ["wide", "over_fp16", "huge"])
def test_bf16_range_persistent(kind):
    """The persistent matrix-core kernel (4400 rows: 275 blocks of 16, more than the compute units
    of the chip) on rows of 545 groups (35 runs: three items per wave and block, so x is reloaded
    and converted with every item) and of 65 groups (x loaded and converted once, held for every
    block); batch 8 and 16 (two and four x loads per run), k = 1 (split form) and 2, 4 (converted)."""
    for d_in, seed in ((4360, 450), (520, 451)):
        L = make_layer(LayerSpec("pers", 4400, d_in, M=4, seed=seed, act_dtype="bf16"))
        C, s = formats.f16_bits_to_f64(L.codebooks), formats.f16_bits_to_f64(L.scales)
        with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
            for b in (8, 16):
                xbits = _x(kind, b, d_in, seed=460 + b)
                xv = act_values(xbits, "bf16")
                x = to_dev(xbits).view(torch.bfloat16)
                for k in (1, 2, 4):
                    ref = oracle.linear(xv, L.codes, C, s, k)
                    y = torch.empty((b, 4400), dtype=torch.float32, device="cuda")
                    A.gemv(gl.handle, k, x, A.DType.BF16, b, y, A.DType.F32)
                    torch.cuda.synchronize()
                    got = out_values(y)
                    what = f"persistent {kind} d_in={d_in} b={b} k={k}"
                    normwise = check_close(got, ref, "f32", what)
                    assert normwise < 1e-5, f"{what}: normwise error {normwise:.2e}"
