"""aqmb_beam_search_weighted (GPU) against the oracle's data-aware beam search in binary32.

The objective of group (i, j) is d^T H_j d with H_j the group's 8 x 8 block of X X^T / n (§2.2,
Eq. wmse-task, restricted to the group; App. C's code optimisation minimises the error in the
layer's outputs). Both sides decide in binary32 in the order stated in include/aqmb.h and
oracle.search.beam_search_codes_weighted_f32, so codes and reported errors must be bit-identical.
On integer-valued inputs (integer weights, codewords and blocks, power-of-two scales) every
binary32 operation is exact and the fp64 weighted search (pinned against the WMSE and exhaustive
search) gives the same codes. The blocks H come from the oracle's group_hessian_blocks of seeded
calibration inputs, rounded to float32 (the kernel's input), and the oracle reads the same floats.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from oracle import formats
from workloads import (LayerSpec, make_layer, make_weights, make_integer_layer, make_integer_rows,
                       make_calibration_inputs)

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU hosts too; every test here is marked gpu
    pytest.skip("no GPU", allow_module_level=True)

import paper_2606_12876_amd as A  # noqa: E402
from gpu_helpers import to_dev  # noqa: E402


def _blocks(L, n=256):
    X = make_calibration_inputs(L, n)
    return oracle.group_hessian_blocks(X, 8).astype(np.float32)


def _gpu(L, Wbits, Hb, k, beam):
    spec = L.spec
    G = spec.d_in // 8
    desc = A.make_desc(spec.d_out, spec.d_in, spec.M, spec.B)
    codes = torch.full((k, spec.d_out, G), 0xAB, dtype=torch.uint8, device="cuda")
    errs = torch.full((spec.d_out, G), -1.0, dtype=torch.float32, device="cuda")
    A.beam_search_weighted(desc, k, beam, to_dev(Wbits).view(torch.float16), to_dev(L.codebooks), to_dev(L.scales),
                           torch.from_numpy(np.ascontiguousarray(Hb, dtype=np.float32)).cuda(), codes, errs)
    torch.cuda.synchronize()
    return codes.cpu().numpy().astype(np.int64), errs.cpu().numpy()


def _oracle(L, Wbits, Hb, k, beam, groups=None):
    C = formats.f16_bits_to_f64(L.codebooks)
    s = formats.f16_bits_to_f64(L.scales)
    return oracle.beam_search_codes_weighted_f32(formats.f16_bits_to_f64(Wbits), C, s, Hb.astype(np.float64),
                                                 k, beam, groups=groups)


def _check(L, Wbits, Hb, k, beam, what):
    c_gpu, e_gpu = _gpu(L, Wbits, Hb, k, beam)
    c_ref, e_ref = _oracle(L, Wbits, Hb, k, beam)
    bad = np.argwhere(np.any(c_gpu != c_ref, axis=0))
    assert len(bad) == 0, f"{what}: codes differ at {len(bad)} groups, first (row, group) {bad[:4].tolist()}"
    assert np.array_equal(e_gpu, e_ref), f"{what}: errors differ"
    return c_gpu, e_gpu


def _int_blocks(rng, G):
    Amat = rng.integers(-2, 3, size=(G, 8, 8)).astype(np.float64)
    return np.einsum("jut,juv->jtv", Amat, Amat).astype(np.float32)


@pytest.mark.parametrize("k,beam", [(1, 1), (1, 8), (2, 1), (2, 5), (3, 8), (4, 2), (4, 16)])
def test_integer_inputs_exact(k, beam):
    """Integer-valued inputs: the codes are also those of the fp64 weighted search."""
    L = make_integer_layer(LayerSpec("int", 7, 48, M=4, seed=300 + 10 * k + beam))
    Wb = make_integer_rows(L, 7, 16)
    Hb = _int_blocks(np.random.default_rng(k * 31 + beam), 6)
    codes, errs = _check(L, Wb, Hb, k, beam, f"integer k={k} beam={beam}")
    C = formats.f16_bits_to_f64(L.codebooks)
    s = formats.f16_bits_to_f64(L.scales)
    c64, t64 = oracle.beam_search_codes(formats.f16_bits_to_f64(Wb), C, s, k, beam, H_blocks=Hb.astype(np.float64))
    assert np.array_equal(codes, c64)
    assert float(errs.astype(np.float64).sum()) == t64


def test_identity_blocks_give_the_plain_search_on_integer_inputs():
    """X = I: the objective is the plain squared error, and on exact (integer) inputs the codes are
    those of aqmb_beam_search."""
    L = make_integer_layer(LayerSpec("eye", 5, 64, M=3, seed=330))
    Wb = make_integer_rows(L, 5, 16)
    eye = np.stack([np.eye(8, dtype=np.float32)] * 8)
    cw, ew = _gpu(L, Wb, eye, 3, 4)
    desc = A.make_desc(5, 64, 3, 8)
    codes = torch.zeros((3, 5, 8), dtype=torch.uint8, device="cuda")
    errs = torch.zeros((5, 8), dtype=torch.float32, device="cuda")
    A.beam_search(desc, 3, 4, to_dev(Wb).view(torch.float16), to_dev(L.codebooks), to_dev(L.scales), codes, errs)
    torch.cuda.synchronize()
    assert np.array_equal(cw, codes.cpu().numpy().astype(np.int64))
    assert np.array_equal(ew, errs.cpu().numpy())


@pytest.mark.parametrize("k,beam", [(1, 4), (2, 8), (4, 8), (4, 3)])
def test_gaussian_bit_exact(k, beam):
    """Gaussian fp16 weights and codebooks, blocks from seeded calibration inputs with outlier
    channels; 300 rows (a full and a ragged 256-row workgroup) of 24 groups."""
    L = make_layer(LayerSpec("g", 300, 192, M=4, seed=340 + k + beam))
    Wb = make_weights(L)
    _check(L, Wb, _blocks(L), k, beam, f"gaussian k={k} beam={beam}")


@pytest.mark.parametrize("k,beam", [(1, 3), (2, 4), (4, 16)])
def test_four_bit_codebooks(k, beam):
    L = make_integer_layer(LayerSpec("int4", 9, 64, M=4, B=4, seed=350 + k))
    Wb = make_integer_rows(L, 9, 16)
    Hb = _int_blocks(np.random.default_rng(351 + k), 8)
    codes, errs = _check(L, Wb, Hb, k, beam, f"4-bit integer k={k} beam={beam}")
    C = formats.f16_bits_to_f64(L.codebooks)
    s = formats.f16_bits_to_f64(L.scales)
    c64, t64 = oracle.beam_search_codes(formats.f16_bits_to_f64(Wb), C, s, k, beam, H_blocks=Hb.astype(np.float64))
    assert np.array_equal(codes, c64) and float(errs.astype(np.float64).sum()) == t64
    Lg = make_layer(LayerSpec("g4", 270, 96, M=4, B=4, seed=360 + k))
    _check(Lg, make_weights(Lg), _blocks(Lg), k, beam, f"4-bit gaussian k={k} beam={beam}")


def test_eight_codebooks():
    L = make_layer(LayerSpec("m8", 3, 72, M=8, seed=370))
    Wb = make_weights(L)
    Hb = _blocks(L)
    _check(L, Wb, Hb, 8, 4, "k=8")
    _check(L, Wb, Hb, 6, 2, "k=6 of 8")


def test_full_size_sampled_groups():
    """The benchmarked shape (4096 x 4096 weights, M = 4, k = 4, beam 8, blocks of 4096 seeded
    calibration inputs): the whole matrix on the GPU, against the oracle on 1000 groups spread over
    it, every group of the first row (each group has its own block of H) and a few fixed ones
    (about 7 s of oracle time)."""
    L = make_layer(LayerSpec("square", 4096, 4096, M=4, seed=2))
    Wb = make_weights(L)
    Hb = _blocks(L, 4096)
    c_gpu, e_gpu = _gpu(L, Wb, Hb, 4, 8)
    rng = np.random.default_rng(6)
    groups = [(int(i), int(j)) for i, j in zip(rng.integers(0, 4096, 1000), rng.integers(0, 512, 1000))]
    groups += [(0, j) for j in range(512)] + [(4095, 511), (4095, 0), (255, 3), (256, 3)]
    groups = sorted(set(groups))
    c_ref, e_ref = _oracle(L, Wb, Hb, 4, 8, groups=groups)
    for (i, j) in groups:
        assert np.array_equal(c_gpu[:, i, j], c_ref[:, i, j]), f"codes differ at ({i}, {j})"
        assert e_gpu[i, j] == e_ref[i, j], f"error differs at ({i}, {j})"
    assert np.all(np.isfinite(e_gpu))


def test_weighted_codes_lower_the_weighted_error():
    """On Gaussian data the weighted search's codes have a lower total weighted error d^T H d
    (evaluated in fp64 from the reconstruction) than the plain search's codes."""
    L = make_layer(LayerSpec("cmp", 64, 512, M=3, seed=380))
    Wb = make_weights(L)
    Hb = _blocks(L, 512)
    cw, _ = _gpu(L, Wb, Hb, 3, 4)
    desc = A.make_desc(64, 512, 3, 8)
    codes = torch.zeros((3, 64, 64), dtype=torch.uint8, device="cuda")
    A.beam_search(desc, 3, 4, to_dev(Wb).view(torch.float16), to_dev(L.codebooks), to_dev(L.scales), codes, None)
    torch.cuda.synchronize()
    cp = codes.cpu().numpy().astype(np.int64)
    W = formats.f16_bits_to_f64(Wb)
    C = formats.f16_bits_to_f64(L.codebooks)
    s = formats.f16_bits_to_f64(L.scales)
    H = Hb.astype(np.float64)

    def werr(c):
        R = (W - oracle.reconstruct(c, C[:3], s, 3)).reshape(64, 64, 8)
        return float(np.einsum("ijt,jtu,iju->", R, H, R))
    assert werr(cw) < werr(cp)


def test_rejections_write_nothing():
    L = make_layer(LayerSpec("rej", 4, 64, M=2, seed=390))
    W = to_dev(make_weights(L)).view(torch.float16)
    cb, sc = to_dev(L.codebooks), to_dev(L.scales)
    H = torch.from_numpy(np.stack([np.eye(8, dtype=np.float32)] * 8)).cuda()
    codes = torch.full((2, 4, 8), 7, dtype=torch.uint8, device="cuda")
    f = A.lib.aqmb_beam_search_weighted
    d = A.make_desc(4, 64, 2, 8)
    d16 = A.make_desc(4, 64, 2, 16)
    import ctypes
    base = dict(desc=ctypes.byref(d), k=2, beam=4, W=W.data_ptr(), cb=cb.data_ptr(), sc=sc.data_ptr(), H=H.data_ptr(),
                codes=codes.data_ptr(), errs=None, st=None)

    def call(**kw):
        a = dict(base, **kw)
        return f(a["desc"], a["k"], a["beam"], a["W"], a["cb"], a["sc"], a["H"], a["codes"], a["errs"], a["st"])
    assert call(H=None) == A.Status.EINVAL
    assert call(H=H.data_ptr() + 2) == A.Status.EINVAL
    assert call(k=3) == A.Status.EINVAL
    assert call(beam=0) == A.Status.EINVAL
    assert call(beam=17) == A.Status.EUNSUPPORTED
    assert call(desc=ctypes.byref(d16)) == A.Status.EUNSUPPORTED
    torch.cuda.synchronize()
    assert torch.all(codes == 7)
