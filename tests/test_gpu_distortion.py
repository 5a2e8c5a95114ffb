"""aqmb_prefix_distortion (GPU) against the oracle's prefix_distortions (fp64).

D^(k) = ||(W - W^(k)) X||_F^2 / (d_out n) for every k (section 5 with the weighted MSE of
section 2.2), computed by the GPU in one pass.

Two kinds of inputs:
- integer-valued (workloads.make_integer_layer / make_integer_rows): every fp32 product and
  partial sum the kernel forms is an exact integer or half-integer below 2^24, so the GPU value
  equals the oracle's up to the order of the final fp64 additions of N = d_out n non-negative
  terms: relative 2 N 2^-53. Any wrong index, dropped group or misplaced sample shows.
- the recipe's Gaussian fp16 draws: the difference is bounded element by element from the
  arithmetic the kernel performs (products exact, fp32 sums of d_in terms, one rounding of each
  s Q product and each difference), see _bound.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from oracle import formats
from oracle.search import encode_residual_kmeans
from workloads import (LayerSpec, make_layer, make_activations, make_weights, make_integer_layer,
                       make_integer_rows, float_to_f16_bits)

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU hosts too; every test here is marked gpu
    pytest.skip("no GPU", allow_module_level=True)

import paper_2606_12876_amd as A  # noqa: E402
from gpu_helpers import GpuLayer, to_dev  # noqa: E402

U32 = 2.0 ** -24
U64 = 2.0 ** -53


def _gpu(gl, Wbits, Xbits, n=None):
    M = gl.desc.num_codebooks
    n = Xbits.shape[0] if n is None else n
    W = to_dev(Wbits).view(torch.float16)
    X = to_dev(Xbits).view(torch.float16)
    D = torch.full((M,), -1.0, dtype=torch.float64, device="cuda")
    A.prefix_distortion(gl.handle, W, A.DType.F16, X, A.DType.F16, n, D)
    torch.cuda.synchronize()
    return D.cpu().numpy()


def _values(L):
    return formats.f16_bits_to_f64(L.codebooks), formats.f16_bits_to_f64(L.scales)


def _oracle(L, Wbits, Xbits):
    C, s = _values(L)
    return oracle.prefix_distortions(formats.f16_bits_to_f64(Wbits), L.codes, C, s, formats.f16_bits_to_f64(Xbits))


def _bound(L, Wbits, Xbits):
    """Per level, an upper bound on |D_gpu - D| from the kernel's arithmetic.

    Per output (sample t, row i): P = sum_t w x and Q_m = sum_t c_m x are fp32 sums of d_in exact
    products, each off by at most gamma * sum |products| with gamma = 2 d_in u (u = 2^-24, twice
    the classical (d_in - 1) u to leave room for any internal order of the matrix cores). Each
    update r -= s Q_m adds at most 2 u (|s Q_m| + |r|). With e the bound on the output's error
    and R its exact value, the square's error is at most 2 |R| e + e^2; the fp64 sums add a
    relative 2 N 2^-53.
    """
    C, s = _values(L)
    W = formats.f16_bits_to_f64(Wbits)
    X = formats.f16_bits_to_f64(Xbits)
    d_out, d_in = W.shape
    n = X.shape[0]
    gam = 2 * d_in * U32
    Xa = np.abs(X).T
    R = W @ X.T
    err = gam * (np.abs(W) @ Xa)
    out = []
    for m in range(L.codes.shape[0]):
        Cm = C[m][L.codes[m]].reshape(d_out, d_in)
        sQ = s[:, None] * (Cm @ X.T)
        R = R - sQ
        err = err + np.abs(s)[:, None] * gam * (np.abs(Cm) @ Xa) + 2 * U32 * (np.abs(sQ) + np.abs(R))
        D = float(np.sum(R * R)) / (d_out * n)
        out.append(float(np.sum(2 * np.abs(R) * err + err * err)) / (d_out * n) + 2 * d_out * n * U64 * D)
    return np.array(out)


def _check_exact(d_out, d_in, n, M, seed):
    L = make_integer_layer(LayerSpec(f"int{d_out}x{d_in}", d_out, d_in, M=M, seed=seed))
    Wb = make_integer_rows(L, d_out, 16)
    Xb = make_integer_rows(L, n, 4)
    ref = _oracle(L, Wb, Xb)
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        got = _gpu(gl, Wb, Xb)
    rtol = 2 * d_out * n * U64 + 1e-15
    assert np.all(ref > 0)
    np.testing.assert_allclose(got, ref, rtol=rtol, atol=0, err_msg=f"{d_out}x{d_in} n={n} M={M}")


@pytest.mark.parametrize("M", [1, 2, 3, 4, 5, 6, 7, 8])
def test_integer_exact_ragged(M):
    """200 rows (two row blocks, the second partial), d_in 520 (a last step with one group of four),
    77 samples (partial sample tiles), every M (both sample-tile widths, both replica counts)."""
    _check_exact(200, 520, 77, M, seed=100 + M)


@pytest.mark.parametrize("shape", [(1, 8, 1, 2), (130, 264, 65, 3), (256, 1024, 128, 4), (33, 40, 31, 6),
                                   (1100, 136, 2000, 5), (1100, 136, 2000, 8)])
def test_integer_exact_shapes(shape):
    """Degenerate sizes (one row, one group, one sample), whole tiles, and grids with more work
    items than workgroups (each workgroup loops over several items)."""
    d_out, d_in, n, M = shape
    _check_exact(d_out, d_in, n, M, seed=d_out + d_in + n + M)


def test_integer_exact_full_size():
    """The benchmarked workload: a 4096 x 4096 layer, M = 4, 4096 calibration inputs."""
    _check_exact(4096, 4096, 4096, 4, seed=7)


def _check_bound(L, Wb, Xb, what):
    ref = _oracle(L, Wb, Xb)
    bnd = _bound(L, Wb, Xb)
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        got = _gpu(gl, Wb, Xb)
    err = np.abs(got - ref)
    assert np.all(err <= bnd), f"{what}: |gpu - oracle| {err} above bound {bnd} (oracle {ref})"
    return ref, got


def test_gaussian_within_bound():
    for (d_out, d_in, n, M, seed) in [(300, 520, 100, 4, 11), (64, 4096, 96, 3, 12), (129, 72, 200, 8, 13)]:
        L = make_layer(LayerSpec("g", d_out, d_in, M=M, seed=seed))
        Wb = make_weights(L)
        Xb = make_activations(L, n, "f16")
        _check_bound(L, Wb, Xb, f"gaussian {d_out}x{d_in} n={n} M={M}")


def test_near_full_reconstruction_cancellation():
    """W = W^(M) + small noise: D^(M) is about 1e-5 of D^(1), so R_M is a small difference of
    large fp32 sums; the result must still be within the bound."""
    L = make_layer(LayerSpec("near", 257, 1032, M=4, seed=14))
    C, s = _values(L)
    W_hat = oracle.reconstruct(L.codes, C, s, 4)
    Wb = float_to_f16_bits(W_hat + L.rng.normal(0.0, 1e-4, size=W_hat.shape))
    Xb = make_activations(L, 150, "f16")
    ref, got = _check_bound(L, Wb, Xb, "near W^(M)")
    assert ref[-1] < 1e-3 * ref[0]
    np.testing.assert_allclose(got, ref, rtol=1e-3)


def test_residual_kmeans_encoded_layer():
    """A Gaussian W encoded by residual k-means (the initialisation of appendix C): the codes are
    no longer uniform and the distortion falls with every added codebook."""
    rng = np.random.Generator(np.random.PCG64(15))
    d_out, d_in, M = 96, 256, 3
    W = rng.normal(0.0, 0.02, size=(d_out, d_in))
    codes, C, s = encode_residual_kmeans(W, M=M, B=8, g=8, seed=15, iters=4)
    L = make_layer(LayerSpec("km", d_out, d_in, M=M, seed=15))
    L.codes = codes.astype(np.uint8)
    L.codebooks = float_to_f16_bits(C)
    L.scales = float_to_f16_bits(s)
    Wb = float_to_f16_bits(W)
    Xb = make_activations(L, 128, "f16")
    ref, got = _check_bound(L, Wb, Xb, "residual k-means")
    assert np.all(np.diff(got) < 0), f"distortion does not fall with k: {got}"


def test_identity_inputs_give_weight_mse():
    """X = I (n = d_in): the weighted MSE is the plain MSE of the weights (section 2.2)."""
    L = make_layer(LayerSpec("eye", 150, 264, M=3, seed=16))
    Wb = make_weights(L)
    Xb = float_to_f16_bits(np.eye(264))
    C, s = _values(L)
    W = formats.f16_bits_to_f64(Wb)
    mse = np.array([np.mean((W - oracle.reconstruct(L.codes, C, s, k)) ** 2) for k in (1, 2, 3)])
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        got = _gpu(gl, Wb, Xb)
    np.testing.assert_allclose(got, mse, rtol=1e-5)


def test_full_size_gaussian_within_bound():
    L = make_layer(LayerSpec("square", 4096, 4096, M=4, seed=2))
    Wb = make_weights(L)
    Xb = make_activations(L, 4096, "f16")
    _check_bound(L, Wb, Xb, "4096x4096 n=4096")


def test_reproducible_and_shares_workspace_with_gemv():
    """Two calls give the same bits; a gemv on the same layer before and after is unaffected."""
    L = make_layer(LayerSpec("ws", 512, 1024, M=4, seed=17))
    Wb = make_weights(L)
    Xb = make_activations(L, 300, "f16")
    xb = make_activations(L, 2, "f16")
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl:
        x = to_dev(xb).view(torch.float16)
        y0 = torch.empty((2, 512), dtype=torch.float32, device="cuda")
        y1 = torch.empty_like(y0)
        A.gemv(gl.handle, 3, x, A.DType.F16, 2, y0, A.DType.F32)
        d0 = _gpu(gl, Wb, Xb)
        A.gemv(gl.handle, 3, x, A.DType.F16, 2, y1, A.DType.F32)
        d1 = _gpu(gl, Wb, Xb)
        torch.cuda.synchronize()
        assert np.array_equal(d0, d1)
        assert torch.equal(y0, y1)


def test_rejections_write_nothing():
    L = make_layer(LayerSpec("rej", 64, 64, M=2, seed=18))
    L16 = make_layer(LayerSpec("rej16", 64, 64, M=2, B=16, seed=19))
    with GpuLayer(L.codes, L.codebooks, L.scales) as gl, GpuLayer(L16.codes, L16.codebooks, L16.scales) as g16:
        W = torch.zeros((64, 64), dtype=torch.float16, device="cuda")
        X = torch.zeros((8, 64 + 8), dtype=torch.float16, device="cuda")
        D = torch.full((2,), 5.0, dtype=torch.float64, device="cuda")
        f = A.lib.aqmb_prefix_distortion
        Xp, Wp, Dp = X.data_ptr(), W.data_ptr(), D.data_ptr()
        assert f(g16.handle, Wp, 0, Xp, 0, 8, Dp, None) == A.Status.EUNSUPPORTED      # B = 16
        assert f(gl.handle, Wp, 1, Xp, 0, 8, Dp, None) == A.Status.EUNSUPPORTED       # W bf16
        assert f(gl.handle, Wp, 0, Xp, 2, 8, Dp, None) == A.Status.EUNSUPPORTED       # X f32
        assert f(gl.handle, Wp, 0, Xp, 0, 0, Dp, None) == A.Status.EINVAL             # n = 0
        assert f(gl.handle, None, 0, Xp, 0, 8, Dp, None) == A.Status.EINVAL           # W null
        assert f(gl.handle, Wp, 0, None, 0, 8, Dp, None) == A.Status.EINVAL           # X null
        assert f(gl.handle, Wp, 0, Xp, 0, 8, None, None) == A.Status.EINVAL           # D null
        assert f(gl.handle, Wp, 0, Xp + 2, 0, 8, Dp, None) == A.Status.EINVAL         # X misaligned
        assert f(gl.handle, Wp + 8, 0, Xp, 0, 8, Dp, None) == A.Status.EINVAL         # W misaligned
        assert f(gl.handle, Wp, 0, Xp, 0, 8, Dp + 4, None) == A.Status.EINVAL         # D misaligned
        torch.cuda.synchronize()
        assert torch.all(D == 5.0)
