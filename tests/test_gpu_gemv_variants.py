"""Every GEMV kernel for 8-bit codes and both GEMM tilings (8- and 4-bit codes), whatever the default dispatch picks.

By default batch 1 runs the direct-gather kernel (fp16 x: on rows of at most 512 groups) and
larger batches the matrix-core kernel; the AQMB_GEMV variable (read once per process) forces one of them for every
batch. A child process
with the variable set runs the small GEMV cases against the oracle, so both kernels stay
parity-tested at every batch. Oracle and tolerance as in the other GEMV tests.
"""
from __future__ import annotations

import os
import subprocess
import sys

import pytest
import torch

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU hosts too; every test here is marked gpu
    pytest.skip("no GPU", allow_module_level=True)

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CHILD = r"""
import sys
sys.path.insert(0, {root!r}); sys.path.insert(0, {tests!r})
import numpy as np, torch
import oracle
from oracle import formats
from workloads import LayerSpec, make_layer, make_activations
from gpu_helpers import GpuLayer, check_close, act_values, to_dev, out_values, TORCH_DT, A_DT
import paper_2606_12876_amd as A
for spec in [LayerSpec("ragged", 1000, 1032, seed=31), LayerSpec("M8", 520, 520, M=8, seed=34),
             LayerSpec("wide", 130, 16392, M=4, seed=38)]:
    L = make_layer(spec)
    C, s = formats.f16_bits_to_f64(L.codebooks), formats.f16_bits_to_f64(L.scales)
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        for b in (1, 2, 3, 16):
            for xdt in ("f16", "bf16"):
                xbits = make_activations(L, b, xdt, heavy_tail=(b % 2 == 1))
                x = act_values(xbits, xdt)
                for k in sorted({{1, spec.M}}):
                    ref = oracle.linear(x, L.codes, C, s, k)
                    y = torch.empty((b, spec.d_out), dtype=torch.float32, device="cuda")
                    A.gemv(gl.handle, k, to_dev(xbits).view(TORCH_DT[xdt]), A_DT[xdt], b, y, A.DType.F32)
                    torch.cuda.synchronize()
                    check_close(out_values(y), ref, "f32", f"{{spec.name}} b={{b}} k={{k}} {{xdt}}")
print("variant ok", flush=True)
"""


@pytest.mark.parametrize("variant", ["mma", "cw"])
def test_forced_variant_matches_oracle(variant):
    env = dict(os.environ, AQMB_GEMV=variant)
    code = CHILD.format(root=ROOT, tests=os.path.join(ROOT, "tests"))
    r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0 and "variant ok" in r.stdout, f"AQMB_GEMV={variant}:\n{r.stdout[-2000:]}\n{r.stderr[-3000:]}"


GEMM_CHILD = r"""
import sys
sys.path.insert(0, {root!r}); sys.path.insert(0, {tests!r})
import numpy as np, torch
import oracle
from workloads import LayerSpec, make_layer, make_activations
from gpu_helpers import GpuLayer, check_close, act_values, to_dev, out_values
import paper_2606_12876_amd as A
for (n, d_out, d_in, M, B) in [(1, 40, 264, 2, 8), (17, 257, 520, 3, 8), (300, 200, 264, 4, 8), (600, 130, 1032, 8, 8),
                               (17, 257, 520, 3, 4), (300, 200, 264, 4, 4), (600, 130, 1032, 8, 4)]:
    L = make_layer(LayerSpec("g", d_out, d_in, M=M, B=B, seed=41 + n + B, act_dtype="bf16"))
    Xbits = make_activations(L, n, "bf16", heavy_tail=True)
    X = act_values(Xbits, "bf16")
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        for k in sorted({{1, M}}):
            ref = oracle.gemm_reference(X, L.codes, L.codebooks, L.scales, k)
            Y = torch.empty((n, d_out), dtype=torch.float32, device="cuda")
            A.gemm(gl.handle, k, to_dev(Xbits).view(torch.bfloat16), n, Y, A.DType.F32)
            torch.cuda.synchronize()
            check_close(out_values(Y), ref, "f32", f"gemm n={{n}} {{d_out}}x{{d_in}} B={{B}} k={{k}}")
print("variant ok", flush=True)
"""


@pytest.mark.parametrize("variant", ["small", "big", "big:256", "big:128", "big:64"])
def test_forced_gemm_tiling_matches_oracle(variant):
    """Both GEMM tilings at token counts the default dispatch sends to the other one, and each tile
    shape of the large-tile kernel (256 x 128, 128 x 128, 128 x 64) at every test shape."""
    tiling, _, tile = variant.partition(":")
    env = dict(os.environ, AQMB_GEMM=tiling)
    if tile:
        env["AQMB_GEMM_TILE"] = tile
    code = GEMM_CHILD.format(root=ROOT, tests=os.path.join(ROOT, "tests"))
    r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0 and "variant ok" in r.stdout, f"AQMB_GEMM {variant}:\n{r.stdout[-2000:]}\n{r.stderr[-3000:]}"
