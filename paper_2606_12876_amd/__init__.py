"""aqmb: multi-bitwidth additive-codebook linear layers on MI355X (gfx950).

Thin ctypes binding over ``libaqmb.so`` (``include/aqmb.h``). The functions here have the
C names without the ``aqmb_`` prefix and only marshal arguments: every step of the
computation runs in the library's HIP kernels. PyTorch tensors are accepted for device
buffers and the current PyTorch stream is used when no stream is given; PyTorch is plumbing
(allocation and streams), not part of the computation.

If the library has not been built, importing this package fails loudly: there is no
fallback implementation.
"""
from __future__ import annotations

import ctypes
import enum
import os
from typing import Optional

__all__ = ["Status", "DType", "Desc", "AqmbError", "GemvKernel", "GemmTiling", "lib", "create", "destroy", "get_desc",
           "gemv", "gemv_select", "gemm", "gemm_select", "dequant", "bits_per_weight", "strerror", "last_error",
           "validate", "QuantLinear", "LIB_PATH"]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libaqmb.so")


class Status(enum.IntEnum):
    OK = 0
    EINVAL = 1
    EUNSUPPORTED = 2
    ENOMEM = 3
    EHIP = 4


class DType(enum.IntEnum):
    F16 = 0
    BF16 = 1
    F32 = 2


class GemvKernel(enum.IntEnum):
    """aqmb_gemv_kernel: which GEMV kernel aqmb_gemv_select runs."""
    AUTO = 0
    DIRECT = 1
    MMA = 2
    LUT = 3


class GemmTiling(enum.IntEnum):
    """aqmb_gemm_tiling: which tiling aqmb_gemm_select runs."""
    AUTO = 0
    ROWS16 = 1
    T256x128 = 2
    T128x128 = 3
    T128x64 = 4


class Desc(ctypes.Structure):
    _fields_ = [("d_out", ctypes.c_int32), ("d_in", ctypes.c_int32), ("group_size", ctypes.c_int32),
                ("num_codebooks", ctypes.c_int32), ("code_bits", ctypes.c_int32)]


class AqmbError(RuntimeError):
    def __init__(self, status: int, where: str, message: str):
        self.status = Status(status)
        super().__init__(f"{where}: {self.status.name}: {message}")


def _load() -> ctypes.CDLL:
    # One HIP runtime per process: PyTorch ships its own libamdhip64 (same SONAME). Importing
    # torch first makes the library bind to that runtime, so device pointers, streams and
    # devices are shared; loading the library first would start a second runtime.
    import torch  # noqa: F401
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it first (python -m paper_2606_12876_amd.build "
                          f"or __graft_entry__.build()); there is no fallback implementation")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, st = ctypes.c_void_p, ctypes.c_int, ctypes.c_int
    L.aqmb_create.argtypes = [ctypes.POINTER(vp), ctypes.POINTER(Desc), vp, vp, vp, vp]
    L.aqmb_destroy.argtypes = [vp]
    L.aqmb_create_prefix.argtypes = [ctypes.POINTER(vp), ctypes.POINTER(Desc), i32, vp, vp, vp, vp]
    L.aqmb_load_planes.argtypes = [vp, i32, vp, vp]
    L.aqmb_drop_planes.argtypes = [vp, i32]
    L.aqmb_resident_planes.argtypes = [vp, ctypes.POINTER(i32)]
    L.aqmb_get_desc.argtypes = [vp, ctypes.POINTER(Desc)]
    L.aqmb_gemv.argtypes = [vp, i32, vp, i32, i32, vp, i32, vp]
    L.aqmb_gemv_select.argtypes = [vp, i32, vp, i32, i32, vp, i32, i32, vp]
    L.aqmb_gemm_select.argtypes = [vp, i32, vp, i32, vp, i32, i32, vp]
    L.aqmb_gemv_multi.argtypes = [ctypes.POINTER(vp), i32, i32, vp, i32, i32, ctypes.POINTER(vp), i32, vp]
    L.aqmb_gemm.argtypes = [vp, i32, vp, i32, vp, i32, vp]
    L.aqmb_gemm_ws.argtypes = [vp, i32, vp, i32, vp, i32, vp, ctypes.c_size_t, vp]
    L.aqmb_gemm_workspace_bytes.argtypes = [vp, i32, i32, ctypes.POINTER(ctypes.c_size_t)]
    L.aqmb_dequant.argtypes = [vp, i32, vp, i32, vp]
    L.aqmb_prefix_distortion.argtypes = [vp, vp, i32, vp, i32, i32, vp, vp]
    L.aqmb_prefix_distortion_noalloc.argtypes = [vp, vp, i32, vp, i32, i32, vp, vp]
    L.aqmb_beam_search.argtypes = [ctypes.POINTER(Desc), i32, i32, vp, vp, vp, vp, vp, vp]
    L.aqmb_beam_search_weighted.argtypes = [ctypes.POINTER(Desc), i32, i32, vp, vp, vp, vp, vp, vp, vp]
    L.aqmb_validate.argtypes = [ctypes.POINTER(Desc), i32, i32, i32, i32, i32, vp, vp]
    L.aqmb_bits_per_weight.argtypes = [ctypes.POINTER(Desc), i32]
    L.aqmb_bits_per_weight.restype = ctypes.c_double
    L.aqmb_strerror.argtypes = [i32]
    L.aqmb_strerror.restype = ctypes.c_char_p
    L.aqmb_last_error.argtypes = []
    L.aqmb_last_error.restype = ctypes.c_char_p
    for f in ("aqmb_create", "aqmb_create_prefix", "aqmb_load_planes", "aqmb_drop_planes", "aqmb_resident_planes",
              "aqmb_destroy", "aqmb_get_desc", "aqmb_gemv", "aqmb_gemv_select", "aqmb_gemv_multi", "aqmb_gemm",
              "aqmb_gemm_select", "aqmb_gemm_ws", "aqmb_gemm_workspace_bytes",
              "aqmb_dequant", "aqmb_prefix_distortion", "aqmb_prefix_distortion_noalloc", "aqmb_beam_search",
              "aqmb_beam_search_weighted",
              "aqmb_validate"):
        getattr(L, f).restype = st
    return L


lib = _load()


def strerror(status: int) -> str:
    return lib.aqmb_strerror(int(status)).decode()


def last_error() -> str:
    return lib.aqmb_last_error().decode()


def _check(status: int, where: str):
    if status != Status.OK:
        raise AqmbError(status, where, last_error() or strerror(status))


def _ptr(t) -> Optional[int]:
    """Device address of a tensor (or an int address, or None)."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _dtype(t, default=None) -> DType:
    if isinstance(t, (DType, int)):
        return DType(t)
    import torch
    m = {torch.float16: DType.F16, torch.bfloat16: DType.BF16, torch.float32: DType.F32}
    if t.dtype not in m:
        raise TypeError(f"unsupported dtype {t.dtype}")
    return m[t.dtype]


def make_desc(d_out: int, d_in: int, num_codebooks: int, code_bits: int = 8, group_size: int = 8) -> Desc:
    return Desc(d_out, d_in, group_size, num_codebooks, code_bits)


def _nbytes(t) -> Optional[int]:
    if hasattr(t, "numel") and hasattr(t, "element_size"):
        return t.numel() * t.element_size()
    return None


def create(desc: Desc, codes, codebooks, scales, stream=None) -> int:
    """aqmb_create: codes [M][d_out][d_in/g] uint8|uint16, codebooks [M][2^B][g] fp16 bits,
    scales [d_out] fp16 bits, all device buffers. Returns the layer handle.

    The C library sees raw pointers; when tensors are passed their sizes are checked here so
    that a short buffer is rejected instead of read past its end."""
    g = desc.group_size if desc.group_size > 0 else 1
    need = {"codes": desc.num_codebooks * desc.d_out * (desc.d_in // g) * (1 if desc.code_bits <= 8 else 2),
            "codebooks": desc.num_codebooks * (1 << max(0, min(desc.code_bits, 16))) * desc.group_size * 2,
            "scales": desc.d_out * 2}
    for name, t in (("codes", codes), ("codebooks", codebooks), ("scales", scales)):
        n = _nbytes(t)
        if n is not None and n < need[name]:
            raise AqmbError(Status.EINVAL, "aqmb_create", f"{name} holds {n} bytes, the descriptor needs {need[name]}")
    h = ctypes.c_void_p()
    _check(lib.aqmb_create(ctypes.byref(h), ctypes.byref(desc), _ptr(codes), _ptr(codebooks), _ptr(scales),
                           _stream(stream)), "aqmb_create")
    return h.value


def _need_planes(desc: Desc, codes, n_planes: int, where: str):
    g = desc.group_size if desc.group_size > 0 else 1
    need = max(n_planes, 0) * desc.d_out * (desc.d_in // g) * (1 if desc.code_bits <= 8 else 2)
    n = _nbytes(codes)
    if n is not None and n < need:
        raise AqmbError(Status.EINVAL, where, f"codes holds {n} bytes, {n_planes} planes need {need}")


def create_prefix(desc: Desc, resident: int, codes, codebooks, scales, stream=None) -> int:
    """aqmb_create_prefix: a layer holding only code planes 0..resident-1 (codes [resident][d_out][d_in/g])."""
    _need_planes(desc, codes, resident, "aqmb_create_prefix")
    h = ctypes.c_void_p()
    _check(lib.aqmb_create_prefix(ctypes.byref(h), ctypes.byref(desc), resident, _ptr(codes), _ptr(codebooks),
                                  _ptr(scales), _stream(stream)), "aqmb_create_prefix")
    return h.value


def load_planes(layer: int, n_planes: int, codes, stream=None) -> None:
    """aqmb_load_planes: append the next n_planes code planes (codes [n_planes][d_out][d_in/g])."""
    _need_planes(get_desc(layer), codes, n_planes, "aqmb_load_planes")
    _check(lib.aqmb_load_planes(layer, n_planes, _ptr(codes), _stream(stream)), "aqmb_load_planes")


def drop_planes(layer: int, keep: int) -> None:
    """aqmb_drop_planes: keep code planes 0..keep-1 and free the others."""
    _check(lib.aqmb_drop_planes(layer, keep), "aqmb_drop_planes")


def resident_planes(layer: int) -> int:
    r = ctypes.c_int32()
    _check(lib.aqmb_resident_planes(layer, ctypes.byref(r)), "aqmb_resident_planes")
    return r.value


def destroy(layer: int) -> None:
    _check(lib.aqmb_destroy(layer), "aqmb_destroy")


def get_desc(layer: int) -> Desc:
    d = Desc()
    _check(lib.aqmb_get_desc(layer, ctypes.byref(d)), "aqmb_get_desc")
    return d


_ELEM = {0: 2, 1: 2, 2: 4}


def _need(t, n_elems: int, dtype, what: str, where: str):
    n = _nbytes(t)
    if n is not None and int(dtype) in _ELEM and n < n_elems * _ELEM[int(dtype)]:
        raise AqmbError(Status.EINVAL, where, f"{what} holds {n} bytes, needs {n_elems * _ELEM[int(dtype)]}")


def gemv(layer: int, k: int, x, x_dtype, batch: int, y, y_dtype, stream=None) -> None:
    d = get_desc(layer)
    if 1 <= batch <= 16:
        _need(x, batch * d.d_in, x_dtype, "x", "aqmb_gemv")
        _need(y, batch * d.d_out, y_dtype, "y", "aqmb_gemv")
    _check(lib.aqmb_gemv(layer, k, _ptr(x), int(x_dtype), batch, _ptr(y), int(y_dtype), _stream(stream)),
           "aqmb_gemv")


def gemv_select(layer: int, k: int, x, x_dtype, batch: int, y, y_dtype, kernel, stream=None) -> None:
    """aqmb_gemv_select: aqmb_gemv with the kernel named by ``kernel`` (a GemvKernel)."""
    d = get_desc(layer)
    if 1 <= batch <= 16:
        _need(x, batch * d.d_in, x_dtype, "x", "aqmb_gemv_select")
        _need(y, batch * d.d_out, y_dtype, "y", "aqmb_gemv_select")
    _check(lib.aqmb_gemv_select(layer, k, _ptr(x), int(x_dtype), batch, _ptr(y), int(y_dtype), int(kernel),
                                _stream(stream)), "aqmb_gemv_select")


MAX_MULTI = 16


def gemv_multi(layers, k: int, x, x_dtype, batch: int, ys, y_dtype, stream=None) -> None:
    """aqmb_gemv_multi: the GEMV of every layer in `layers` (same d_in) on the same x, one output each."""
    layers, ys = list(layers), list(ys)
    if len(layers) != len(ys):
        raise AqmbError(Status.EINVAL, "aqmb_gemv_multi", "one output per layer")
    if 1 <= batch <= 16 and 1 <= len(layers) <= MAX_MULTI:
        for layer, y in zip(layers, ys):
            d = get_desc(layer)
            _need(x, batch * d.d_in, x_dtype, "x", "aqmb_gemv_multi")
            _need(y, batch * d.d_out, y_dtype, "y", "aqmb_gemv_multi")
    n = len(layers)
    la = (ctypes.c_void_p * max(n, 1))(*[ctypes.c_void_p(h) for h in layers])
    ya = (ctypes.c_void_p * max(n, 1))(*[ctypes.c_void_p(_ptr(y)) for y in ys])
    _check(lib.aqmb_gemv_multi(la, n, k, _ptr(x), int(x_dtype), batch, ya, int(y_dtype), _stream(stream)),
           "aqmb_gemv_multi")


def gemm(layer: int, k: int, X, n_tokens: int, Y, y_dtype, stream=None) -> None:
    d = get_desc(layer)
    if n_tokens >= 1:
        _need(X, n_tokens * d.d_in, DType.BF16, "X", "aqmb_gemm")
        _need(Y, n_tokens * d.d_out, y_dtype, "Y", "aqmb_gemm")
    _check(lib.aqmb_gemm(layer, k, _ptr(X), n_tokens, _ptr(Y), int(y_dtype), _stream(stream)), "aqmb_gemm")


def gemm_select(layer: int, k: int, X, n_tokens: int, Y, y_dtype, tiling, stream=None) -> None:
    """aqmb_gemm_select: aqmb_gemm with the tiling named by ``tiling`` (a GemmTiling)."""
    d = get_desc(layer)
    if n_tokens >= 1:
        _need(X, n_tokens * d.d_in, DType.BF16, "X", "aqmb_gemm_select")
        _need(Y, n_tokens * d.d_out, y_dtype, "Y", "aqmb_gemm_select")
    _check(lib.aqmb_gemm_select(layer, k, _ptr(X), n_tokens, _ptr(Y), int(y_dtype), int(tiling), _stream(stream)),
           "aqmb_gemm_select")


def gemm_workspace_bytes(layer: int, k: int, n_tokens: int) -> int:
    """aqmb_gemm_workspace_bytes: the workspace gemm_ws needs for its two-pass path (0: not taken)."""
    n = ctypes.c_size_t(0)
    _check(lib.aqmb_gemm_workspace_bytes(layer, k, n_tokens, ctypes.byref(n)), "aqmb_gemm_workspace_bytes")
    return n.value


def gemm_ws(layer: int, k: int, X, n_tokens: int, Y, y_dtype, workspace, stream=None) -> None:
    """aqmb_gemm_ws: aqmb_gemm with a caller-owned device workspace (a tensor, or None)."""
    d = get_desc(layer)
    if n_tokens >= 1:
        _need(X, n_tokens * d.d_in, DType.BF16, "X", "aqmb_gemm_ws")
        _need(Y, n_tokens * d.d_out, y_dtype, "Y", "aqmb_gemm_ws")
    nb = _nbytes(workspace) if workspace is not None else 0
    _check(lib.aqmb_gemm_ws(layer, k, _ptr(X), n_tokens, _ptr(Y), int(y_dtype), _ptr(workspace), nb or 0,
                            _stream(stream)), "aqmb_gemm_ws")


def dequant(layer: int, k: int, W, w_dtype, stream=None) -> None:
    d = get_desc(layer)
    _need(W, d.d_out * d.d_in, w_dtype, "W", "aqmb_dequant")
    _check(lib.aqmb_dequant(layer, k, _ptr(W), int(w_dtype), _stream(stream)), "aqmb_dequant")


def prefix_distortion(layer: int, W, w_dtype, Xt, x_dtype, n: int, D, stream=None) -> None:
    """aqmb_prefix_distortion: D[k-1] = ||(W - W_k) X||_F^2 / (d_out n) for k = 1..M, with the n
    calibration inputs as the rows of Xt [n][d_in] (fp16) and W [d_out][d_in] fp16; D holds M
    float64 values in device memory."""
    d = get_desc(layer)
    _need(W, d.d_out * d.d_in, w_dtype, "W", "aqmb_prefix_distortion")
    if n >= 1:
        _need(Xt, n * d.d_in, x_dtype, "Xt", "aqmb_prefix_distortion")
    nd = _nbytes(D)
    need = 8 * resident_planes(layer)
    if nd is not None and nd < need:
        raise AqmbError(Status.EINVAL, "aqmb_prefix_distortion", f"D holds {nd} bytes, needs {need}")
    _check(lib.aqmb_prefix_distortion(layer, _ptr(W), int(w_dtype), _ptr(Xt), int(x_dtype), n, _ptr(D),
                                      _stream(stream)), "aqmb_prefix_distortion")


def prefix_distortion_noalloc(layer: int, W, w_dtype, Xt, x_dtype, n: int, D, stream=None) -> None:
    """aqmb_prefix_distortion_noalloc: prefix_distortion with the library's fixed scratch (no device
    allocation; calls that overlap on one device race)."""
    d = get_desc(layer)
    _need(W, d.d_out * d.d_in, w_dtype, "W", "aqmb_prefix_distortion_noalloc")
    if n >= 1:
        _need(Xt, n * d.d_in, x_dtype, "Xt", "aqmb_prefix_distortion_noalloc")
    nd = _nbytes(D)
    need = 8 * resident_planes(layer)
    if nd is not None and nd < need:
        raise AqmbError(Status.EINVAL, "aqmb_prefix_distortion_noalloc", f"D holds {nd} bytes, needs {need}")
    _check(lib.aqmb_prefix_distortion_noalloc(layer, _ptr(W), int(w_dtype), _ptr(Xt), int(x_dtype), n, _ptr(D),
                                              _stream(stream)), "aqmb_prefix_distortion_noalloc")


MAX_BEAM = 16


def beam_search(desc: Desc, k: int, beam: int, W, codebooks, scales, codes, errors=None, stream=None) -> None:
    """aqmb_beam_search: codes [k][d_out][d_in/8] uint8 (and errors [d_out][d_in/8] float32 if given)
    from a beam search over codebooks 0..k-1 for every group of W [d_out][d_in] fp16."""
    G = desc.d_in // max(desc.group_size, 1)
    _need(W, desc.d_out * desc.d_in, DType.F16, "W", "aqmb_beam_search")
    nc = _nbytes(codes)
    if nc is not None and 1 <= k and nc < k * desc.d_out * G:
        raise AqmbError(Status.EINVAL, "aqmb_beam_search", f"codes holds {nc} bytes, needs {k * desc.d_out * G}")
    ne = _nbytes(errors) if errors is not None else None
    if ne is not None and ne < 4 * desc.d_out * G:
        raise AqmbError(Status.EINVAL, "aqmb_beam_search", f"errors holds {ne} bytes, needs {4 * desc.d_out * G}")
    _check(lib.aqmb_beam_search(ctypes.byref(desc), k, beam, _ptr(W), _ptr(codebooks), _ptr(scales), _ptr(codes),
                                _ptr(errors) if errors is not None else None, _stream(stream)), "aqmb_beam_search")


def beam_search_weighted(desc: Desc, k: int, beam: int, W, codebooks, scales, H, codes, errors=None,
                         stream=None) -> None:
    """aqmb_beam_search_weighted: the code search with the data-aware error d^T H_j d; H is
    [d_in/8][8][8] float32 (the symmetric diagonal blocks of X X^T / n)."""
    G = desc.d_in // max(desc.group_size, 1)
    _need(W, desc.d_out * desc.d_in, DType.F16, "W", "aqmb_beam_search_weighted")
    _need(H, G * 64, DType.F32, "H", "aqmb_beam_search_weighted")
    nc = _nbytes(codes)
    if nc is not None and 1 <= k and nc < k * desc.d_out * G:
        raise AqmbError(Status.EINVAL, "aqmb_beam_search_weighted", f"codes holds {nc} bytes, needs {k * desc.d_out * G}")
    ne = _nbytes(errors) if errors is not None else None
    if ne is not None and ne < 4 * desc.d_out * G:
        raise AqmbError(Status.EINVAL, "aqmb_beam_search_weighted", f"errors holds {ne} bytes, needs {4 * desc.d_out * G}")
    _check(lib.aqmb_beam_search_weighted(ctypes.byref(desc), k, beam, _ptr(W), _ptr(codebooks), _ptr(scales), _ptr(H),
                                         _ptr(codes), _ptr(errors) if errors is not None else None, _stream(stream)),
           "aqmb_beam_search_weighted")


def bits_per_weight(desc: Desc, k: int) -> float:
    return float(lib.aqmb_bits_per_weight(ctypes.byref(desc), k))


def validate(desc: Desc, op: int, k: int, n: int, in_dtype, out_dtype, inp, out) -> Status:
    return Status(lib.aqmb_validate(ctypes.byref(desc), op, k, n, int(in_dtype), int(out_dtype), _ptr(inp), _ptr(out)))


class QuantLinear:
    """A quantized linear layer y = x . W_k^T served at any precision level k <= M.

    Holds the library's layer handle. ``forward`` allocates the output with PyTorch and calls the
    library on the current stream: up to 16 input rows go to aqmb_gemv (fp16 or bf16 x), more
    rows to aqmb_gemm, which takes bf16 x only (other dtypes are refused, not converted: the
    binding only marshals arguments). The code width B follows from the codebooks: 16, 256 or
    65536 codewords give 4-, 8- or 16-bit codes (4-bit codes are passed one per byte, 0..15).
    """

    _BITS = {16: 4, 256: 8, 65536: 16}

    def __init__(self, codes, codebooks, scales, group_size: int = 8):
        import torch
        M, d_out, n_groups = codes.shape
        n_cw = int(codebooks.shape[1])
        if n_cw not in self._BITS:
            raise AqmbError(Status.EUNSUPPORTED, "QuantLinear", f"codebooks of {n_cw} codewords (16, 256 or 65536)")
        code_bits = self._BITS[n_cw]
        want = torch.int16 if code_bits == 16 else torch.uint8
        if codes.dtype not in ((torch.int16, torch.uint16) if code_bits == 16 else (torch.uint8,)):
            raise AqmbError(Status.EINVAL, "QuantLinear", f"codes of dtype {codes.dtype} for {code_bits}-bit codes")
        self.desc = make_desc(d_out, n_groups * group_size, M, code_bits, group_size)
        self.handle = create(self.desc, codes.contiguous().view(want), codebooks.contiguous().view(torch.int16),
                             scales.contiguous().view(torch.int16))
        self.M, self.d_out, self.d_in, self.code_bits = M, d_out, n_groups * group_size, code_bits

    def forward(self, x, k: int, out_dtype=None):
        import torch
        out_dtype = out_dtype or x.dtype
        lead = x.shape[:-1]
        x2 = x.reshape(-1, self.d_in).contiguous()
        n = x2.shape[0]
        if n > 16 and x2.dtype != torch.bfloat16:
            raise AqmbError(Status.EUNSUPPORTED, "QuantLinear",
                            f"{n} rows go to aqmb_gemm, which takes bf16 x only (got {x2.dtype})")
        y = torch.empty((n, self.d_out), dtype=out_dtype, device=x.device)
        if n <= 16:
            gemv(self.handle, k, x2, _dtype(x2), n, y, _dtype(y))
        else:
            gemm(self.handle, k, x2, n, y, _dtype(y))
        return y.reshape(*lead, self.d_out)

    __call__ = forward

    def dequant(self, k: int, dtype=None):
        import torch
        W = torch.empty((self.d_out, self.d_in), dtype=dtype or torch.float16, device="cuda")
        dequant(self.handle, k, W, _dtype(W))
        return W

    def close(self):
        if self.handle:
            destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
