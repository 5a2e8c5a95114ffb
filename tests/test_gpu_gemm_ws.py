"""aqmb_gemm_ws: the prefill GEMM with a caller workspace (two passes: bf16 weight tiles, then a
dense matrix-core kernel), against the oracle's GEMM reference and bit for bit against aqmb_gemm.

The two-pass path forms the same bf16 weight tile (binary32 left fold over the first k planes,
round to nearest even) and adds the same products in the same order as aqmb_gemm's 256 x 128
tiling, so outputs must be identical; the oracle check (gemm_reference, the definition with the
explicit bf16 weight rounding) pins both. Shapes: the full prefill workload at every k >= 3, 4-bit
codes, ragged rows / inputs / tokens with and without an XCD placement of the workgroups, both
output dtypes, and the cases that fall back to aqmb_gemm.
"""
import numpy as np
import pytest
import torch

import oracle
from workloads import LayerSpec, make_layer, make_activations, config

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU hosts too; every test here is marked gpu
    pytest.skip("no GPU", allow_module_level=True)

import paper_2606_12876_amd as A  # noqa: E402
from gpu_helpers import GpuLayer, out_values, check_close, to_dev, TORCH_DT, A_DT, act_values  # noqa: E402


def _run(gl, k, X, n, ydt, ws=None, fill=3.0):
    Y = torch.full((n, gl.desc.d_out), fill, dtype=TORCH_DT[ydt], device="cuda")
    if ws is False:
        A.gemm(gl.handle, k, X, n, Y, A_DT[ydt])
    else:
        A.gemm_ws(gl.handle, k, X, n, Y, A_DT[ydt], ws)
    torch.cuda.synchronize()
    return out_values(Y)


def _workspace(gl, k, n):
    nb = A.gemm_workspace_bytes(gl.handle, k, n)
    assert nb > 0, f"two-pass path not taken for k={k} n={n}"
    d = gl.desc
    assert nb == ((d.d_out + 31) // 32) * ((d.d_in + 63) // 64) * 4096   # 4 KiB per 32 rows x 64 inputs
    # filled with a pattern: every value the GEMM reads must have been written by its first pass
    return torch.full((nb // 2,), 0x7FC0, dtype=torch.int16, device="cuda")


def _check(spec, n, ks, ydts=("bf16",), oracle_rows=None):
    L = make_layer(spec)
    Xbits = make_activations(L, n, "bf16", heavy_tail=True)
    X = to_dev(Xbits).view(torch.bfloat16)
    Xv = act_values(Xbits, "bf16")
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        for k in ks:
            ws = _workspace(gl, k, n)
            rows = np.arange(n) if oracle_rows is None else np.asarray(oracle_rows)
            ref = oracle.gemm_reference(Xv[rows], L.codes, L.codebooks, L.scales, k)
            for ydt in ydts:
                got = _run(gl, k, X, n, ydt, ws)
                one = _run(gl, k, X, n, ydt, False)
                assert np.array_equal(got, one), f"{spec.name} k={k} {ydt}: differs from aqmb_gemm"
                check_close(got[rows], ref, ydt, f"{spec.name} k={k} {ydt}")


def test_prefill_workload_every_k():
    """2048 tokens x 4096 x 4096, M = 4: k = 3, 4 against the full oracle product."""
    spec = config("prefill")
    _check(spec, spec.n_tokens, (3, 4), ydts=("bf16", "f32"))


def test_ragged_everywhere_xcd_blocks():
    """d_out = 4000 (the last 32-row tile half empty), d_in = 4040 (505 groups: a ragged last
    K-step), 2000 tokens (a ragged last token tile); 8 x 32 workgroups in XCD blocks."""
    _check(LayerSpec("rg", 4000, 4040, M=3, seed=301), 2000, (3,), oracle_rows=np.r_[0:40, 1950:2000])


def test_two_rounds_of_workgroups():
    """4096 tokens (16 token tiles x 32 column blocks: two workgroups per compute unit in turn)."""
    spec = config("prefill")
    _check(spec, 4096, (4,), oracle_rows=np.r_[0:16, 2040:2056, 4080:4096])


def test_plain_workgroup_order():
    """9 token tiles x 31 column blocks: no XCD blocking divides the grid (plain order)."""
    _check(LayerSpec("po", 3900, 1024, M=3, seed=302), 2100, (3,), ydts=("f32",),
           oracle_rows=np.r_[0:32, 2048:2100])


def test_four_bit_codes_and_eight_planes():
    """16-codeword books (nibble codes) and k up to 8."""
    _check(LayerSpec("b4", 4096, 2048, M=4, B=4, seed=303), 2048, (3, 4), oracle_rows=np.r_[0:24, 2024:2048])
    _check(LayerSpec("m8", 4096, 1024, M=8, seed=304), 2048, (5, 8), oracle_rows=np.r_[0:16, 2040:2048])


def test_fallbacks_and_rejections():
    """k <= 2, few tokens or a small / absent workspace: exactly aqmb_gemm. A workspace that is not
    256-byte aligned is refused and nothing is written."""
    spec = config("prefill")
    L = make_layer(spec)
    n = spec.n_tokens
    Xbits = make_activations(L, n, "bf16")
    X = to_dev(Xbits).view(torch.bfloat16)
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        assert A.gemm_workspace_bytes(gl.handle, 1, n) == 0
        assert A.gemm_workspace_bytes(gl.handle, 2, n) == 0
        assert A.gemm_workspace_bytes(gl.handle, 4, 100) == 0          # 16-row tiling
        assert A.gemm_workspace_bytes(gl.handle, 4, 512) == 0          # smaller tiles
        nb = A.gemm_workspace_bytes(gl.handle, 4, n)
        one = _run(gl, 4, X, n, "bf16", False)
        small = torch.zeros((nb // 2 - 128,), dtype=torch.int16, device="cuda")
        assert np.array_equal(_run(gl, 4, X, n, "bf16", small), one)
        assert np.array_equal(_run(gl, 4, X, n, "bf16", None), one)
        assert np.array_equal(_run(gl, 1, X, n, "bf16", small), _run(gl, 1, X, n, "bf16", False))
        ws = torch.zeros((nb // 2 + 256,), dtype=torch.int16, device="cuda")
        Y = torch.full((n, gl.desc.d_out), 5.0, dtype=torch.bfloat16, device="cuda")
        with pytest.raises(A.AqmbError):
            _misaligned(gl, X, n, Y, ws, nb)
        torch.cuda.synchronize()
        assert torch.all(Y == 5.0)
        with pytest.raises(A.AqmbError):
            A.gemm_workspace_bytes(gl.handle, 5, n)                   # k > M


def _misaligned(gl, X, n, Y, ws, nb):
    import ctypes
    st = A.lib.aqmb_gemm_ws(gl.handle, 4, X.data_ptr(), n, Y.data_ptr(), int(A.DType.BF16),
                            ctypes.c_void_p(ws.data_ptr() + 16), nb, ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    if st != A.Status.OK:
        raise A.AqmbError(st, "aqmb_gemm_ws", "")
