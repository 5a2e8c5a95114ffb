"""GPU parity: the HIP path through the C ABI against the CPU oracle, on seeded inputs.

Dequantization is compared bit for bit with the oracle's stated evaluation order; GEMV and
GEMM outputs are compared element by element under the tolerance in tests/gpu_helpers.py.
Shapes cover several tiles with ragged tails in every dimension, batch 1..16, every k, the
degenerate layers (one group, one row, one codebook) and the workload shapes.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import formats
from workloads import CONFIGS, LayerSpec, make_layer, make_activations, config

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU hosts too; every test here is marked gpu
    pytest.skip("no GPU", allow_module_level=True)

import paper_2606_12876_amd as A  # noqa: E402
from gpu_helpers import GpuLayer, abs_terms, out_values, check_close, to_dev, TORCH_DT, A_DT, act_values  # noqa: E402


def _f64(L):
    return formats.f16_bits_to_f64(L.codebooks), formats.f16_bits_to_f64(L.scales)


def run_dequant(gl, k, dt):
    d = gl.desc
    W = torch.empty((d.d_out, d.d_in), dtype=TORCH_DT[dt], device="cuda")
    A.dequant(gl.handle, k, W, A_DT[dt])
    torch.cuda.synchronize()
    W = W.cpu()
    return W.numpy() if dt == "f32" else W.view(torch.int16).numpy().view(np.uint16)


def run_gemv(gl, k, xbits, xdt, ydt):
    b = xbits.shape[0]
    x = to_dev(xbits).view(TORCH_DT[xdt])
    y = torch.empty((b, gl.desc.d_out), dtype=TORCH_DT[ydt], device="cuda")
    A.gemv(gl.handle, k, x, A_DT[xdt], b, y, A_DT[ydt])
    torch.cuda.synchronize()
    return out_values(y)


def run_gemm(gl, k, Xbits, ydt):
    n = Xbits.shape[0]
    X = to_dev(Xbits).view(torch.bfloat16)
    Y = torch.empty((n, gl.desc.d_out), dtype=TORCH_DT[ydt], device="cuda")
    A.gemm(gl.handle, k, X, n, Y, A_DT[ydt])
    torch.cuda.synchronize()
    return out_values(Y)


# ------------------------------------------------------------------------------------ dequant

@pytest.mark.parametrize("spec", [
    LayerSpec("ragged", 1000, 1032, seed=21),           # 129 groups: 9 slices, the last with 1 group
    LayerSpec("M1", 37, 8, M=1, seed=22),               # one group per row, one codebook
    LayerSpec("b16", 300, 136, M=2, B=16, seed=23),      # 16-bit codes, 17 groups
    # more 64-row tiles than two per compute unit: 32-row tiles walked by each workgroup, a last
    # row tile of 4 rows and a last slice of one group
    LayerSpec("tiles32", 4100, 4104, M=2, seed=24),
    LayerSpec("g125", 70, 1000, M=3, seed=25),          # 125 groups: 32-row x 128-group tiles
    LayerSpec("g300", 40, 2400, M=2, seed=26),          # 300 groups: 8-row x 512-group tiles
], ids=lambda s: s.name)
@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_dequant_bit_exact(spec, dt):
    L = make_layer(spec)
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        for k in range(1, spec.M + 1):
            got = run_dequant(gl, k, dt)
            ref = oracle.dequant_canonical(L.codes, L.codebooks, L.scales, k, dt)
            assert np.array_equal(got.view(np.uint32) if dt == "f32" else got,
                                  ref.view(np.uint32) if dt == "f32" else ref), (spec.name, k, dt)


@pytest.mark.parametrize("name", ["tiny", "square", "mlp_up", "mlp_down", "b16"])
def test_dequant_workload_layers_bit_exact(name):
    spec = config(name)
    L = make_layer(spec)
    dts = ("bf16", "f16") if not name.startswith("mlp_") else ("bf16",)
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        for k in spec.ks:
            for dt in dts:
                got = run_dequant(gl, k, dt)
                ref = oracle.dequant_canonical(L.codes, L.codebooks, L.scales, k, dt)
                assert np.array_equal(got, ref), (name, k, dt)


def test_dequant_index_revealing():
    """C_0[c][t] = c + 256 t, s = 1: the dequantized matrix spells out plane 0's codes."""
    rng = np.random.default_rng(0)
    d_out, d_in = 515, 1048
    codes = rng.integers(0, 256, size=(2, d_out, d_in // 8)).astype(np.uint8)
    C = np.zeros((2, 256, 8)); C[0] = [[c + 256 * t for t in range(8)] for c in range(256)]; C[1] = 3.0
    cb = C.astype(np.float16).view(np.uint16)
    s = np.ones(d_out).astype(np.float16).view(np.uint16)
    with GpuLayer(codes, cb, s) as gl:
        W = run_dequant(gl, 1, "f32")
        j, t = np.divmod(np.arange(d_in), 8)
        assert np.array_equal(W.astype(np.float64), codes[0][:, j] + 256.0 * t[None, :])
        W2 = run_dequant(gl, 2, "f32")
        assert np.array_equal(W2.astype(np.float64), codes[0][:, j] + 256.0 * t[None, :] + 3.0)


def test_dequant_subnormal_and_tie_cases():
    """fp16 subnormal codebook entries and binary32 ties in the fold (the oracle's hand cases)."""
    codes = np.zeros((3, 4, 2), dtype=np.uint8)
    codes[:, 1] = 1
    C = np.zeros((3, 256, 8))
    C[0, 0], C[1, 0], C[2, 0] = 1.0, 2.0 ** -24, 2.0 ** -24
    C[0, 1], C[1, 1], C[2, 1] = 2.0 ** -24, 2.0 ** -23, -(2.0 ** -24)
    cb = C.astype(np.float16).view(np.uint16)
    s = np.array([1.0, 1.0, 0.5, 3.0]).astype(np.float16).view(np.uint16)
    with GpuLayer(codes, cb, s) as gl:
        for k in (1, 2, 3):
            for dt in ("f32", "f16", "bf16"):
                got = run_dequant(gl, k, dt)
                ref = oracle.dequant_canonical(codes, cb, s, k, dt)
                assert np.array_equal(got.view(np.uint32) if dt == "f32" else got,
                                      ref.view(np.uint32) if dt == "f32" else ref), (k, dt)


# ------------------------------------------------------------------------------------ GEMV

@pytest.mark.parametrize("spec,batches", [
    (LayerSpec("ragged", 1000, 1032, seed=31), (1, 2, 3, 4, 5, 8, 13, 16)),
    (LayerSpec("tiny", 1, 8, M=3, seed=32), (1, 4, 16)),
    (LayerSpec("M1", 700, 264, M=1, seed=33), (1, 2, 7)),
    (LayerSpec("M8", 520, 520, M=8, seed=34), (1, 4, 9)),
    (LayerSpec("b16", 1030, 328, M=2, B=16, seed=35), (1, 3, 16)),
], ids=lambda s: getattr(s, "name", str(s)))
@pytest.mark.parametrize("xdt", ["f16", "bf16"])
def test_gemv_small_shapes(spec, batches, xdt):
    L = make_layer(spec)
    C, s = _f64(L)
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        for b in batches:
            xbits = make_activations(L, b, xdt, heavy_tail=(b % 2 == 1))
            x = act_values(xbits, xdt)
            for k in range(1, spec.M + 1):
                ref = oracle.linear(x, L.codes, C, s, k)
                T = abs_terms(x, L.codes, C, s, k)
                for ydt in ("f32", "f16", "bf16"):
                    got = run_gemv(gl, k, xbits, xdt, ydt)
                    check_close(got, ref, ydt, f"{spec.name} b={b} k={k} {xdt}->{ydt}", terms=T, n_terms=k * spec.d_in)


@pytest.mark.parametrize("name", ["tiny", "square", "mlp_up", "mlp_down", "b16"])
def test_gemv_workloads(name):
    spec = config(name)
    L = make_layer(spec)
    C, s = _f64(L)
    ydt = spec.act_dtype
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        xs = {b: make_activations(L, b) for b in spec.batches}
        for k in spec.ks:
            W = oracle.reconstruct(L.codes, C, s, k)
            for b, xbits in xs.items():
                ref = act_values(xbits, spec.act_dtype) @ W.T
                got = run_gemv(gl, k, xbits, spec.act_dtype, ydt)
                check_close(got, ref, ydt, f"{name} b={b} k={k}")
            del W


@pytest.mark.parametrize("xdt", ["f16", "bf16"])
@pytest.mark.parametrize("d_in", [16384, 16392])
def test_gemv_wide_rows(d_in, xdt):
    """Rows of 2048 groups (the widest the direct-gather kernel keeps in registers) and of 2049
    groups (beyond it: the lookup-table kernel), batch 1, 2 and 4, every k. Rows of more than 512
    groups go to the matrix cores except at batch 1 with bf16 x and k < 4, which takes the
    direct-gather kernel (2048 groups) or the lookup-table kernel (2049)."""
    spec = LayerSpec(f"wide{d_in}", 130, d_in, M=4, seed=38, act_dtype=xdt)
    L = make_layer(spec)
    C, s = _f64(L)
    ydt = "f32" if xdt == "f16" else "bf16"
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        for b in (1, 2, 4):
            xbits = make_activations(L, b, xdt, heavy_tail=True)
            x = act_values(xbits, xdt)
            for k in range(1, 5):
                ref = oracle.linear(x, L.codes, C, s, k)
                got = run_gemv(gl, k, xbits, xdt, ydt)
                check_close(got, ref, ydt, f"d_in={d_in} b={b} k={k} {xdt}",
                            terms=abs_terms(x, L.codes, C, s, k), n_terms=k * d_in)


@pytest.mark.parametrize("xdt", ["f16", "bf16"])
def test_gemv_more_row_blocks_than_cus(xdt):
    """5000 rows = 313 blocks of 16 (the last one ragged): more than one block per compute unit,
    so each workgroup walks several blocks with the codebooks replicated once. Batch 1 (direct
    gathers) and 2, 3, 8, 16 (matrix cores; 65 groups = 5 runs of 16, so
    11 of the 16 waves run a dummy item per block), every k, against the oracle."""
    spec = LayerSpec("tall", 5000, 520, M=4, seed=39, act_dtype=xdt)
    L = make_layer(spec)
    C, s = _f64(L)
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        for b in (1, 2, 3, 8, 16):
            xbits = make_activations(L, b, xdt, heavy_tail=True)
            x = act_values(xbits, xdt)
            for k in range(1, 5):
                ref = oracle.linear(x, L.codes, C, s, k)
                T = abs_terms(x, L.codes, C, s, k)
                for ydt in ("f32", xdt):
                    got = run_gemv(gl, k, xbits, xdt, ydt)
                    check_close(got, ref, ydt, f"5000 rows {xdt} b={b} k={k} y={ydt}", terms=T, n_terms=k * 520)


@pytest.mark.parametrize("xdt", ["f16", "bf16"])
def test_gemv_tall_layer_long_rows(xdt):
    """4400 rows (275 blocks of 16) of 545 groups (35 runs of 16, the last with one group): the
    persistent matrix-core kernel with three items per wave and block, so x is loaded with every
    item rather than held across blocks; batch 1 (fp16 x: matrix cores on rows of more than 512
    groups; bf16 x: direct gathers), 8 and 16, every k, against the oracle with the fp32
    summation bound."""
    spec = LayerSpec("tall_long", 4400, 4360, M=4, seed=44, act_dtype=xdt)
    L = make_layer(spec)
    C, s = _f64(L)
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        for b in (1, 8, 16):
            xbits = make_activations(L, b, xdt, heavy_tail=True)
            x = act_values(xbits, xdt)
            for k in range(1, 5):
                ref = oracle.linear(x, L.codes, C, s, k)
                T = abs_terms(x, L.codes, C, s, k)
                for ydt in ("f32", xdt):
                    got = run_gemv(gl, k, xbits, xdt, ydt)
                    check_close(got, ref, ydt, f"4400 x 4360 {xdt} b={b} k={k} y={ydt}", terms=T, n_terms=k * 4360)


def test_gemv_plane_linearity():
    """gemv(k) - gemv(k-1) equals the GEMV of a one-codebook layer holding plane k-1 alone."""
    spec = LayerSpec("lin", 777, 1024, seed=36)
    L = make_layer(spec)
    xbits = make_activations(L, 2, "f16")
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        ys = [None] + [run_gemv(gl, k, xbits, "f16", "f32") for k in range(1, 5)]
    for k in range(2, 5):
        with GpuLayer(L.codes[k - 1:k].copy(), L.codebooks[k - 1:k].copy(), L.scales) as g1:
            y1 = run_gemv(g1, 1, xbits, "f16", "f32")
        check_close(ys[k] - ys[k - 1], y1, "f32", f"plane {k - 1}")


def test_gemv_repeated_calls_and_errors_write_nothing():
    """Counters re-arm: repeated calls agree; rejected calls leave y untouched."""
    spec = LayerSpec("rep", 600, 512, seed=37)
    L = make_layer(spec)
    xbits = make_activations(L, 3, "f16")
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        first = run_gemv(gl, 3, xbits, "f16", "f32")
        for _ in range(5):
            assert np.array_equal(run_gemv(gl, 3, xbits, "f16", "f32"), first)
        x = to_dev(xbits).view(torch.float16)
        y = torch.full((3, 600), 7.0, dtype=torch.float32, device="cuda")
        for k, b in ((0, 3), (5, 3), (1, 0), (1, 17)):
            with pytest.raises(A.AqmbError):
                A.gemv(gl.handle, k, x, A.DType.F16, b, y, A.DType.F32)
        torch.cuda.synchronize()
        assert torch.all(y == 7.0)


# ------------------------------------------------------------------------------------ GEMM

@pytest.mark.parametrize("shape", [(300, 200, 264, 4), (129, 130, 1032, 3), (1, 1, 8, 2), (17, 257, 520, 1)])
def test_gemm_small_shapes(shape):
    n, d_out, d_in, M = shape
    spec = LayerSpec("g", d_out, d_in, M=M, seed=41, act_dtype="bf16")
    L = make_layer(spec)
    Xbits = make_activations(L, n, "bf16", heavy_tail=True)
    X = act_values(Xbits, "bf16")
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        for k in range(1, M + 1):
            ref = oracle.gemm_reference(X, L.codes, L.codebooks, L.scales, k)
            for ydt in ("f32", "bf16"):
                got = run_gemm(gl, k, Xbits, ydt)
                check_close(got, ref, ydt, f"gemm {shape} k={k} {ydt}")


def test_gemm_subnormal_codebook_entries():
    """fp16 subnormal codebook entries enter the binary32 fold exactly in the GEMM's weight tile too."""
    spec = LayerSpec("gs", 130, 136, M=4, seed=43, act_dtype="bf16")
    L = make_layer(spec)
    cb = formats.f16_bits_to_f64(L.codebooks)
    rng = np.random.default_rng(1)
    mask = rng.random(cb.shape) < 0.3
    cb = np.where(mask, rng.integers(-1023, 1024, cb.shape) * 2.0 ** -24, cb)   # subnormal fp16 values
    cbits = cb.astype(np.float16).view(np.uint16)
    Xbits = make_activations(L, 70, "bf16")
    X = act_values(Xbits, "bf16")
    with GpuLayer(L.codes, cbits, L.scales) as gl:
        for k in range(1, 5):
            ref = oracle.gemm_reference(X, L.codes, cbits, L.scales, k)
            got = run_gemm(gl, k, Xbits, "f32")
            check_close(got, ref, "f32", f"subnormal k={k}")
            # tighter: fp32 accumulation of bf16 products only
            assert np.max(np.abs(got - ref)) <= 1e-5 * np.max(np.abs(ref)) + 1e-30


def test_gemm_workload_full_size():
    spec = config("prefill")
    L = make_layer(spec)
    Xbits = make_activations(L, spec.n_tokens, "bf16")
    X = act_values(Xbits, "bf16")
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        for k in spec.ks:
            ref = oracle.gemm_reference(X, L.codes, L.codebooks, L.scales, k)
            got = run_gemm(gl, k, Xbits, "bf16")
            check_close(got, ref, "bf16", f"c5 k={k}")


def test_gemm_matches_exact_layer_within_bf16_weight_rounding():
    """Against the exact fp64 layer the only extra error is the bf16 rounding of the weight tile."""
    spec = LayerSpec("gx", 256, 512, seed=42, act_dtype="bf16")
    L = make_layer(spec)
    C, s = _f64(L)
    Xbits = make_activations(L, 64, "bf16")
    X = act_values(Xbits, "bf16")
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        for k in range(1, 5):
            got = run_gemm(gl, k, Xbits, "f32")
            exact = oracle.linear(X, L.codes, C, s, k)
            W = oracle.reconstruct(L.codes, C, s, k)
            bound = (np.abs(X) @ np.abs(W).T) * (2.0 ** -8 + 2.0 ** -20)
            assert np.all(np.abs(got - exact) <= bound)
