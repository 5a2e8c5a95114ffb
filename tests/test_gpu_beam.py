"""aqmb_beam_search (GPU) against the oracle's beam search with decisions in binary32.

The search (Appendix C, code optimisation) decides integer codes by comparing floating-point
errors, so both sides take every decision in binary32 in the same order (the order is stated in
include/aqmb.h and oracle.search.beam_search_codes_f32). The codes and the reported errors must
then be bit-identical. On integer-valued inputs every binary32 operation is exact, so the fp64
search (pinned against exhaustive search) gives the same codes as well.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from oracle import formats
from workloads import LayerSpec, make_layer, make_weights, make_integer_layer, make_integer_rows

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU hosts too; every test here is marked gpu
    pytest.skip("no GPU", allow_module_level=True)

import paper_2606_12876_amd as A  # noqa: E402
from gpu_helpers import GpuLayer, to_dev  # noqa: E402


def _gpu(L, Wbits, k, beam):
    spec = L.spec
    G = spec.d_in // 8
    desc = A.make_desc(spec.d_out, spec.d_in, spec.M, spec.B)
    codes = torch.full((k, spec.d_out, G), 0xAB, dtype=torch.uint8, device="cuda")
    errs = torch.full((spec.d_out, G), -1.0, dtype=torch.float32, device="cuda")
    A.beam_search(desc, k, beam, to_dev(Wbits).view(torch.float16), to_dev(L.codebooks), to_dev(L.scales),
                  codes, errs)
    torch.cuda.synchronize()
    return codes.cpu().numpy().astype(np.int64), errs.cpu().numpy()


def _oracle(L, Wbits, k, beam, groups=None):
    C = formats.f16_bits_to_f64(L.codebooks)
    s = formats.f16_bits_to_f64(L.scales)
    return oracle.beam_search_codes_f32(formats.f16_bits_to_f64(Wbits), C, s, k, beam, groups=groups)


def _check(L, Wbits, k, beam, what):
    c_gpu, e_gpu = _gpu(L, Wbits, k, beam)
    c_ref, e_ref = _oracle(L, Wbits, k, beam)
    bad = np.argwhere(np.any(c_gpu != c_ref, axis=0))
    assert len(bad) == 0, f"{what}: codes differ at {len(bad)} groups, first (row, group) {bad[:4].tolist()}"
    assert np.array_equal(e_gpu, e_ref), f"{what}: errors differ"
    return c_gpu, e_gpu


@pytest.mark.parametrize("k,beam", [(1, 1), (1, 8), (2, 1), (2, 5), (3, 8), (4, 2), (4, 16)])
def test_integer_inputs_exact(k, beam):
    """Integer-valued weights, codebooks and power-of-two scales: every binary32 operation is exact,
    so the codes are also those of the fp64 search."""
    L = make_integer_layer(LayerSpec("int", 7, 48, M=4, seed=200 + 10 * k + beam))
    Wb = make_integer_rows(L, 7, 16)
    codes, errs = _check(L, Wb, k, beam, f"integer k={k} beam={beam}")
    C = formats.f16_bits_to_f64(L.codebooks)
    s = formats.f16_bits_to_f64(L.scales)
    c64, t64 = oracle.beam_search_codes(formats.f16_bits_to_f64(Wb), C, s, k, beam)
    assert np.array_equal(codes, c64)
    assert float(errs.astype(np.float64).sum()) == t64


@pytest.mark.parametrize("k,beam", [(1, 4), (2, 8), (4, 8), (4, 3)])
def test_gaussian_bit_exact(k, beam):
    """The recipe's fp16 draws (codebooks N(0, 0.02/sqrt(M)), scales U(0.5, 1.5), weights
    N(0, 0.02)); 300 groups per row (a full and a partial 256-group chunk)."""
    L = make_layer(LayerSpec("g", 5, 2400, M=4, seed=210 + k + beam))
    Wb = make_weights(L)
    _check(L, Wb, k, beam, f"gaussian k={k} beam={beam}")


@pytest.mark.parametrize("k,beam", [(1, 3), (2, 4), (4, 16)])
def test_four_bit_codebooks(k, beam):
    """Codebooks of 16 codewords: integer inputs (codes of the fp64 search) and Gaussian ones."""
    L = make_integer_layer(LayerSpec("int4", 9, 64, M=4, B=4, seed=250 + k))
    Wb = make_integer_rows(L, 9, 16)
    codes, errs = _check(L, Wb, k, beam, f"4-bit integer k={k} beam={beam}")
    C = formats.f16_bits_to_f64(L.codebooks)
    s = formats.f16_bits_to_f64(L.scales)
    c64, t64 = oracle.beam_search_codes(formats.f16_bits_to_f64(Wb), C, s, k, beam)
    assert np.array_equal(codes, c64) and float(errs.astype(np.float64).sum()) == t64
    Lg = make_layer(LayerSpec("g4", 33, 2400, M=4, B=4, seed=260 + k))
    _check(Lg, make_weights(Lg), k, beam, f"4-bit gaussian k={k} beam={beam}")


def test_eight_codebooks_and_one_row():
    """k = 8 (code bytes 4..7 of a tuple), a single row with 9 groups."""
    L = make_layer(LayerSpec("m8", 1, 72, M=8, seed=220))
    Wb = make_weights(L)
    _check(L, Wb, 8, 4, "k=8")
    _check(L, Wb, 6, 2, "k=6 of 8")


def test_full_size_sampled_groups():
    """The benchmarked shape (4096 x 4096 weights, M = 4, k = 4, beam 8): the whole matrix on the
    GPU, against the oracle on 2000 groups spread over it, every group of the last row and the
    corners (about 7 s of oracle time)."""
    L = make_layer(LayerSpec("square", 4096, 4096, M=4, seed=2))
    Wb = make_weights(L)
    c_gpu, e_gpu = _gpu(L, Wb, 4, 8)
    rng = np.random.default_rng(5)
    groups = [(int(i), int(j)) for i, j in zip(rng.integers(0, 4096, 2000), rng.integers(0, 512, 2000))]
    groups += [(4095, j) for j in range(512)] + [(0, 0), (0, 511)]
    groups = sorted(set(groups))
    c_ref, e_ref = _oracle(L, Wb, 4, 8, groups=groups)
    for (i, j) in groups:
        assert np.array_equal(c_gpu[:, i, j], c_ref[:, i, j]), f"codes differ at ({i}, {j})"
        assert e_gpu[i, j] == e_ref[i, j], f"error differs at ({i}, {j})"
    assert np.all(np.isfinite(e_gpu)) and np.all(e_gpu >= 0)


def test_codes_feed_a_layer():
    """The codes come out in the layout aqmb_create takes: a layer built from them reconstructs
    the weights with the reported errors (binary32 rounding of the residual chain aside)."""
    L = make_layer(LayerSpec("feed", 64, 512, M=3, seed=230))
    Wb = make_weights(L)
    c_gpu, e_gpu = _gpu(L, Wb, 3, 4)
    with GpuLayer(c_gpu.astype(np.uint8), L.codebooks, L.scales) as gl:
        Wd = torch.empty((64, 512), dtype=torch.float32, device="cuda")
        A.dequant(gl.handle, 3, Wd, A.DType.F32)
        torch.cuda.synchronize()
        W_hat = Wd.cpu().numpy().astype(np.float64)
    W = formats.f16_bits_to_f64(Wb)
    e64 = ((W - W_hat).reshape(64, 64, 8) ** 2).sum(axis=2)
    np.testing.assert_allclose(e_gpu.astype(np.float64), e64, rtol=1e-4, atol=1e-12)


def test_rejections_write_nothing():
    L = make_layer(LayerSpec("rej", 4, 64, M=2, seed=240))
    W = to_dev(make_weights(L)).view(torch.float16)
    cb, sc = to_dev(L.codebooks), to_dev(L.scales)
    codes = torch.full((2, 4, 8), 7, dtype=torch.uint8, device="cuda")
    f = A.lib.aqmb_beam_search
    d = A.make_desc(4, 64, 2, 8)
    d16 = A.make_desc(4, 64, 2, 16)
    args = lambda **kw: [kw.get("desc", d), kw.get("k", 2), kw.get("beam", 4), kw.get("W", W.data_ptr()),
                         kw.get("cb", cb.data_ptr()), kw.get("sc", sc.data_ptr()), kw.get("codes", codes.data_ptr()),
                         None, None]
    import ctypes
    call = lambda **kw: f(ctypes.byref(args(**kw)[0]), *args(**kw)[1:])
    assert call(beam=0) == A.Status.EINVAL
    assert call(beam=17) == A.Status.EUNSUPPORTED
    assert call(k=3) == A.Status.EINVAL
    assert call(k=0) == A.Status.EINVAL
    assert call(desc=d16) == A.Status.EUNSUPPORTED
    assert call(W=None) == A.Status.EINVAL
    assert call(cb=None) == A.Status.EINVAL
    assert call(sc=None) == A.Status.EINVAL
    assert call(codes=None) == A.Status.EINVAL
    assert call(W=W.data_ptr() + 2) == A.Status.EINVAL
    assert call(cb=cb.data_ptr() + 8) == A.Status.EINVAL
    torch.cuda.synchronize()
    assert torch.all(codes == 7)
