"""The C-ABI library on the CPU: it loads, exports every symbol include/aqmb.h declares, and
its host-side validation, status strings and bits-per-weight formula behave as documented.
No test here launches anything on a GPU."""
import ctypes
import os
import re

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
A = pytest.importorskip("paper_2606_12876_amd", reason="libaqmb.so not built")


def declared_symbols():
    hdr = open(os.path.join(ROOT, "include", "aqmb.h")).read()
    hdr = re.sub(r"/\*.*?\*/", "", hdr, flags=re.S)
    return sorted(set(re.findall(r"\b(aqmb_[a-z_]+)\s*\(", hdr)))


def test_exports_every_declared_symbol():
    syms = declared_symbols()
    assert {"aqmb_create", "aqmb_gemv", "aqmb_gemm", "aqmb_dequant", "aqmb_destroy"} <= set(syms)
    lib = ctypes.CDLL(A.LIB_PATH)
    for s in syms:
        assert hasattr(lib, s), s


def test_strerror_and_last_error():
    for st in A.Status:
        assert A.strerror(st)
    assert A.strerror(99) == "unknown status"
    d = A.make_desc(64, 64, 4)
    assert A.validate(d, 0, 0, 1, A.DType.F16, A.DType.F16, 16, 32) == A.Status.EINVAL
    assert "k = 0" in A.last_error()
    assert A.validate(d, 0, 1, 1, A.DType.F16, A.DType.F16, 16, 32) == A.Status.OK
    assert A.last_error() == ""


@pytest.mark.parametrize("case,expect", [
    (dict(d_out=0), A.Status.EINVAL),
    (dict(d_in=12), A.Status.EINVAL),                     # not a multiple of g
    (dict(d_in=0), A.Status.EINVAL),
    (dict(group_size=4, d_in=64), A.Status.EUNSUPPORTED),
    (dict(code_bits=4), A.Status.OK),
    (dict(code_bits=12), A.Status.EUNSUPPORTED),
    (dict(code_bits=2), A.Status.EUNSUPPORTED),
    (dict(num_codebooks=0), A.Status.EINVAL),
    (dict(num_codebooks=9), A.Status.EUNSUPPORTED),
    (dict(d_out=1 << 18, d_in=1 << 13), A.Status.OK),
    (dict(d_out=1 << 19, d_in=1 << 13), A.Status.EINVAL),  # d_out * d_in >= 2^32
])
def test_descriptor_validation(case, expect):
    base = dict(d_out=64, d_in=64, group_size=8, num_codebooks=4, code_bits=8)
    base.update(case)
    d = A.Desc(base["d_out"], base["d_in"], base["group_size"], base["num_codebooks"], base["code_bits"])
    assert A.validate(d, 2, 1, 0, A.DType.F16, A.DType.F16, None, 16) == expect


@pytest.mark.parametrize("op,k,n,xdt,ydt,x,y,expect", [
    (0, 1, 1, 0, 0, 16, 32, A.Status.OK),
    (0, 4, 16, 1, 2, 16, 32, A.Status.OK),
    (0, 0, 1, 0, 0, 16, 32, A.Status.EINVAL),       # k < 1
    (0, 5, 1, 0, 0, 16, 32, A.Status.EINVAL),       # k > M
    (0, 1, 0, 0, 0, 16, 32, A.Status.EINVAL),       # batch < 1
    (0, 1, 17, 0, 0, 16, 32, A.Status.EUNSUPPORTED),  # batch > 16
    (0, 1, 1, 2, 0, 16, 32, A.Status.EUNSUPPORTED),  # x must be f16/bf16
    (0, 1, 1, 0, 7, 16, 32, A.Status.EUNSUPPORTED),  # bad y dtype
    (0, 1, 1, 0, 0, None, 32, A.Status.EINVAL),
    (0, 1, 1, 0, 0, 16, None, A.Status.EINVAL),
    (0, 1, 1, 0, 0, 18, 32, A.Status.EINVAL),       # misaligned
    (1, 2, 2048, 1, 1, 16, 32, A.Status.OK),
    (1, 2, 0, 1, 1, 16, 32, A.Status.EINVAL),
    (1, 2, 7, 1, 0, 16, 32, A.Status.EUNSUPPORTED),  # gemm output must be bf16/f32
    (2, 3, 0, 0, 2, None, 32, A.Status.OK),
    (2, 3, 0, 0, 2, None, None, A.Status.EINVAL),
    (5, 1, 1, 0, 0, 16, 32, A.Status.EINVAL),       # unknown op
    (4, 4, 8, 0, 0, 16, 32, A.Status.OK),           # beam search: n = beam
    (4, 4, 16, 0, 0, 16, 7, A.Status.OK),           # codes need no alignment
    (4, 5, 8, 0, 0, 16, 32, A.Status.EINVAL),       # k > M
    (4, 1, 0, 0, 0, 16, 32, A.Status.EINVAL),       # beam < 1
    (4, 1, 17, 0, 0, 16, 32, A.Status.EUNSUPPORTED),  # beam > 16
    (4, 1, 8, 0, 0, None, 32, A.Status.EINVAL),
    (4, 1, 8, 0, 0, 16, None, A.Status.EINVAL),
    (4, 1, 8, 0, 0, 24, 32, A.Status.EINVAL),       # W misaligned
    (3, 0, 4096, 0, 0, 16, 32, A.Status.OK),        # distortion: k is not checked
    (3, 9, 1, 0, 0, 16, 8, A.Status.OK),            # D needs 8-byte alignment only
    (3, 1, 0, 0, 0, 16, 32, A.Status.EINVAL),       # n < 1
    (3, 1, (1 << 30) + 1, 0, 0, 16, 32, A.Status.EUNSUPPORTED),
    (3, 1, 8, 1, 0, 16, 32, A.Status.EUNSUPPORTED),  # X must be f16
    (3, 1, 8, 0, 1, 16, 32, A.Status.EUNSUPPORTED),  # W must be f16
    (3, 1, 8, 0, 0, None, 32, A.Status.EINVAL),
    (3, 1, 8, 0, 0, 16, None, A.Status.EINVAL),
    (3, 1, 8, 0, 0, 24, 32, A.Status.EINVAL),       # X misaligned
    (3, 1, 8, 0, 0, 16, 36, A.Status.EINVAL),       # D misaligned
])
def test_call_validation(op, k, n, xdt, ydt, x, y, expect):
    d = A.make_desc(256, 512, 4)
    assert A.validate(d, op, k, n, xdt, ydt, x, y) == expect


def test_gemm_rejects_16bit_codes():
    d = A.make_desc(256, 512, 2, code_bits=16)
    assert A.validate(d, 1, 1, 8, A.DType.BF16, A.DType.BF16, 16, 32) == A.Status.EUNSUPPORTED
    assert A.validate(d, 0, 2, 8, A.DType.F16, A.DType.F16, 16, 32) == A.Status.OK
    assert A.validate(d, 3, 1, 8, A.DType.F16, A.DType.F16, 16, 32) == A.Status.EUNSUPPORTED
    assert A.validate(d, 4, 1, 8, A.DType.F16, A.DType.F16, 16, 32) == A.Status.EUNSUPPORTED


def test_bits_per_weight_matches_oracle():
    for (d_out, d_in, M, B) in [(28672, 8192, 2, 8), (4096, 4096, 4, 8), (11008, 4096, 4, 8), (14336, 4096, 2, 16)]:
        d = A.make_desc(d_out, d_in, M, B)
        for k in range(1, M + 1):
            assert A.bits_per_weight(d, k) == pytest.approx(oracle.bits_per_weight(d_out, d_in, 8, M, B, k), rel=1e-15)
    d = A.make_desc(64, 64, 4)
    assert A.bits_per_weight(d, 0) < 0 and A.bits_per_weight(d, 5) < 0


def test_bad_handles_rejected_without_gpu():
    assert A.lib.aqmb_destroy(None) == A.Status.OK
    bogus = ctypes.c_void_p(0x1000)
    assert A.lib.aqmb_destroy(bogus) == A.Status.EINVAL
    assert A.lib.aqmb_gemv(bogus, 1, 16, 0, 1, 32, 0, None) == A.Status.EINVAL
    assert A.lib.aqmb_gemm(bogus, 1, 16, 1, 32, 1, None) == A.Status.EINVAL
    assert A.lib.aqmb_dequant(bogus, 1, 32, 0, None) == A.Status.EINVAL
    assert A.lib.aqmb_gemv_select(bogus, 1, 16, 0, 1, 32, 0, 0, None) == A.Status.EINVAL
    assert A.lib.aqmb_gemm_select(bogus, 1, 16, 1, 32, 1, 0, None) == A.Status.EINVAL
    assert A.lib.aqmb_prefix_distortion(bogus, 16, 0, 32, 0, 8, 64, None) == A.Status.EINVAL
    assert "live" in A.last_error()
    assert A.lib.aqmb_beam_search(None, 1, 1, 16, 16, 16, 16, None, None) == A.Status.EINVAL   # null desc
    assert A.lib.aqmb_beam_search_weighted(None, 1, 1, 16, 16, 16, 16, 16, None, None) == A.Status.EINVAL
    dw = A.make_desc(4, 64, 2)
    assert A.lib.aqmb_beam_search_weighted(ctypes.byref(dw), 1, 1, 16, 16, 16, None, 16, None, None) == A.Status.EINVAL
    assert "H" in A.last_error()
    d = A.Desc()
    assert A.lib.aqmb_get_desc(bogus, ctypes.byref(d)) == A.Status.EINVAL
    h = ctypes.c_void_p(0x1234)
    desc = A.make_desc(64, 64, 4)
    assert A.lib.aqmb_create(ctypes.byref(h), ctypes.byref(desc), None, 16, 16, None) == A.Status.EINVAL
    assert h.value is None
    bad = A.make_desc(64, 60, 4)
    assert A.lib.aqmb_create(ctypes.byref(h), ctypes.byref(bad), 16, 16, 16, None) == A.Status.EINVAL


def test_gemv_multi_rejects_before_any_launch():
    vp = ctypes.c_void_p
    bogus = (vp * 2)(vp(0x1000), vp(0x2000))
    ys = (vp * 2)(vp(64), vp(128))
    f = A.lib.aqmb_gemv_multi
    assert f(None, 1, 1, 16, 0, 1, ys, 0, None) == A.Status.EINVAL                 # null layer array
    assert f(bogus, 1, 1, 16, 0, 1, None, 0, None) == A.Status.EINVAL              # null output array
    assert f(bogus, 0, 1, 16, 0, 1, ys, 0, None) == A.Status.EINVAL                # no layers
    many = (vp * 17)(*[vp(0x1000 + 64 * i) for i in range(17)])
    many_y = (vp * 17)(*[vp(64) for _ in range(17)])
    assert f(many, 17, 1, 16, 0, 1, many_y, 0, None) == A.Status.EUNSUPPORTED     # over AQMB_MAX_MULTI
    assert f(bogus, 2, 1, 16, 0, 1, ys, 0, None) == A.Status.EINVAL                # not live layers
    assert "live" in A.last_error()
    with pytest.raises(A.AqmbError):
        A.gemv_multi([0x1000], 1, 16, A.DType.F16, 1, [64, 128], A.DType.F16)    # one output per layer


def test_four_bit_codes_validation():
    """B = 4 (16-codeword codebooks) is accepted by every operation; B = 16 by the GEMV and the
    dequant only."""
    d = A.make_desc(256, 512, 4, code_bits=4)
    assert A.validate(d, 0, 4, 16, A.DType.BF16, A.DType.F32, 16, 32) == A.Status.OK
    assert A.validate(d, 2, 2, 0, A.DType.F16, A.DType.BF16, None, 16) == A.Status.OK
    assert A.validate(d, 1, 1, 8, A.DType.BF16, A.DType.BF16, 16, 32) == A.Status.OK
    assert A.validate(d, 3, 1, 8, A.DType.F16, A.DType.F16, 16, 32) == A.Status.OK
    assert A.validate(d, 4, 1, 8, A.DType.F16, A.DType.F16, 16, 32) == A.Status.OK
    d16 = A.make_desc(256, 512, 2, code_bits=16)
    for op in (1, 3, 4):
        assert A.validate(d16, op, 1, 8, A.DType.F16 if op != 1 else A.DType.BF16, A.DType.F16 if op != 1 else A.DType.BF16,
                          16, 32) == A.Status.EUNSUPPORTED
    assert A.validate(A.make_desc(256, 512, 4, code_bits=2), 0, 1, 1, 0, 0, 16, 32) == A.Status.EUNSUPPORTED


def test_ablation_budgets_are_two_bits():
    """The ablation on codebook precision against count compares 2 x 8-bit and 4 x 4-bit codebooks
    at about 2 bits per weight: both follow from Eq. avg_bits (codes term with the plane count)."""
    for (M, B) in [(2, 8), (4, 4)]:
        for (d_out, d_in) in [(2048, 2048), (16384, 2048)]:
            d = A.make_desc(d_out, d_in, M, code_bits=B)
            v = A.bits_per_weight(d, M)
            assert v == pytest.approx(oracle.bits_per_weight(d_out, d_in, 8, M, B, M), rel=1e-15)
            assert 2.0 < v < 2.1


def test_plane_calls_reject_without_gpu():
    bogus = ctypes.c_void_p(0x1000)
    r = ctypes.c_int32(-1)
    assert A.lib.aqmb_load_planes(bogus, 1, 16, None) == A.Status.EINVAL
    assert A.lib.aqmb_drop_planes(bogus, 1) == A.Status.EINVAL
    assert A.lib.aqmb_resident_planes(bogus, ctypes.byref(r)) == A.Status.EINVAL and r.value == -1
    h = ctypes.c_void_p(0x1234)
    d = A.make_desc(64, 64, 4)
    for resident in (0, 5):
        assert A.lib.aqmb_create_prefix(ctypes.byref(h), ctypes.byref(d), resident, 16, 16, 16, None) == A.Status.EINVAL
        assert h.value is None
