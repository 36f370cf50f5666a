"""Python binding of libspconv.so (C ABI declared in include/spconv.h).

Argument marshalling only: host arrays are numpy, device buffers are torch CUDA
(HIP) tensors, streams are torch streams. Every computation happens in the
library. Importing this module loads the library and raises ImportError if it
has not been built (``python -m paper_2005_04091_amd.build``).
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass
from pathlib import Path

import numpy as np

LIB_PATH = Path(__file__).resolve().parent / "libspconv.so"
if not LIB_PATH.exists():
    raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2005_04091_amd.build` first")

SPCONV_OK = 0
SPCONV_EINVAL = -1
SPCONV_ECAPACITY = -2
SPCONV_EHIP = -3
SPCONV_RELU = 1
SPCONV_MAXPOOL2X2 = 2
SPCONV_UNPADDED_INPUT = 4

EXPORTED = ("spconv_pack_csr", "spconv_pad_input", "spconv_resize_pad_input", "spconv_forward", "spconv_forward_ex", "spconv_plan",
            "spconv_output_shape", "spconv_strerror", "spconv_dense_size", "spconv_pack_dense",
            "spconv_forward_dense", "spconv_dense_plan", "spconv_select_path", "spconv_kernel_variants",
            "spconv_lowered_size", "spconv_pack_lowered")
SPCONV_KERNEL_STRIDE1 = 1
SPCONV_KERNEL_GENERIC = 2
SPCONV_KERNEL_DENSE = 3
SPCONV_KERNEL_STRIDE1_TILED = 4
SPCONV_PATH_SPARSE = 1
SPCONV_PATH_DENSE = 2


class spconv_csr(ctypes.Structure):
    """Mirror of ``struct spconv_csr``."""
    _fields_ = [("K", ctypes.c_int32), ("C", ctypes.c_int32), ("R", ctypes.c_int32), ("S", ctypes.c_int32),
                ("Hp", ctypes.c_int32), ("Wp", ctypes.c_int32), ("nnz", ctypes.c_int64),
                ("rowptr", ctypes.c_void_p), ("colidx", ctypes.c_void_p), ("offset", ctypes.c_void_p),
                ("vals", ctypes.c_void_p)]


class spconv_options(ctypes.Structure):
    """Mirror of ``struct spconv_options``."""
    _fields_ = [("out_pad", ctypes.c_int32), ("residual_pad", ctypes.c_int32), ("residual", ctypes.c_void_p),
                ("max_row_nnz", ctypes.c_int64), ("lowered", ctypes.c_void_p), ("lowered_words", ctypes.c_int64)]


class spconv_plan_info(ctypes.Structure):
    """Mirror of ``struct spconv_plan_info``."""
    _fields_ = [("kernel", ctypes.c_int32), ("pixels_per_lane", ctypes.c_int32), ("images_per_group", ctypes.c_int32),
                ("channels_per_wave", ctypes.c_int32), ("tile_rows", ctypes.c_int32),
                ("tiles_per_image", ctypes.c_int32), ("channels_per_chunk", ctypes.c_int32),
                ("chunks", ctypes.c_int32), ("workgroups", ctypes.c_int32), ("threads_per_workgroup", ctypes.c_int32),
                ("lds_bytes", ctypes.c_int64), ("lds_channel_floats", ctypes.c_int32), ("lds_row_pitch", ctypes.c_int32),
                ("lds_col_shift", ctypes.c_int32), ("launch_workgroups", ctypes.c_int32),
                ("tile_pixels", ctypes.c_int32)]


_c_int = ctypes.c_int
_vp = ctypes.c_void_p


def _bind(lib):
    """Declare the C signatures on a loaded libspconv.so and return it."""
    lib.spconv_pack_csr.restype = _c_int
    lib.spconv_pack_csr.argtypes = [_vp, _vp, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int, _vp, _vp, _vp, _vp,
                                    ctypes.c_int64, ctypes.POINTER(ctypes.c_int64)]
    lib.spconv_pad_input.restype = _c_int
    lib.spconv_pad_input.argtypes = [_vp, _c_int, _c_int, _c_int, _c_int, _c_int, _vp, _vp]
    lib.spconv_resize_pad_input.restype = _c_int
    lib.spconv_resize_pad_input.argtypes = [_vp] + [_c_int] * 7 + [_vp, _vp]
    lib.spconv_forward.restype = _c_int
    lib.spconv_forward.argtypes = [_vp, _c_int, _c_int, _c_int, _c_int, ctypes.POINTER(spconv_csr), _c_int, _c_int,
                                   _c_int, _c_int, _c_int, _vp, ctypes.c_uint32, _vp, _vp]
    lib.spconv_forward_ex.restype = _c_int
    lib.spconv_forward_ex.argtypes = [_vp, _c_int, _c_int, _c_int, _c_int, ctypes.POINTER(spconv_csr), _c_int,
                                      _c_int, _c_int, _c_int, _c_int, _vp, ctypes.c_uint32,
                                      ctypes.POINTER(spconv_options), _vp, _vp]
    lib.spconv_plan.restype = _c_int
    lib.spconv_plan.argtypes = [_c_int, _c_int, _c_int, _c_int, ctypes.POINTER(spconv_csr), _c_int, _c_int, _c_int,
                                _c_int, _c_int, ctypes.c_uint32, ctypes.POINTER(spconv_options),
                                ctypes.POINTER(spconv_plan_info)]
    lib.spconv_output_shape.restype = _c_int
    lib.spconv_output_shape.argtypes = [_c_int, _c_int, _c_int, _c_int, _c_int, _c_int, ctypes.c_uint32,
                                        ctypes.POINTER(_c_int), ctypes.POINTER(_c_int)]
    lib.spconv_strerror.restype = ctypes.c_char_p
    lib.spconv_strerror.argtypes = [_c_int]
    lib.spconv_dense_size.restype = _c_int
    lib.spconv_dense_size.argtypes = [_c_int] * 4 + [ctypes.POINTER(ctypes.c_int64)]
    lib.spconv_pack_dense.restype = _c_int
    lib.spconv_pack_dense.argtypes = [_vp, _vp] + [_c_int] * 4 + [_vp, ctypes.c_int64]
    lib.spconv_forward_dense.restype = _c_int
    lib.spconv_forward_dense.argtypes = [_vp] + [_c_int] * 4 + [_vp] + [_c_int] * 4 + [
        _vp, ctypes.c_uint32, ctypes.POINTER(spconv_options), _vp, _vp]
    lib.spconv_dense_plan.restype = _c_int
    lib.spconv_dense_plan.argtypes = [_c_int] * 8 + [ctypes.c_uint32, ctypes.POINTER(spconv_plan_info)]
    lib.spconv_select_path.restype = _c_int
    lib.spconv_select_path.argtypes = [_c_int] * 9 + [ctypes.c_int64, ctypes.c_uint32, ctypes.POINTER(_c_int)]
    lib.spconv_lowered_size.restype = _c_int
    lib.spconv_lowered_size.argtypes = [_c_int] * 4 + [ctypes.POINTER(spconv_csr)] + [_c_int] * 5 + [
        ctypes.c_uint32, ctypes.POINTER(spconv_options), ctypes.POINTER(ctypes.c_int64)]
    lib.spconv_pack_lowered.restype = _c_int
    lib.spconv_pack_lowered.argtypes = [_c_int] * 4 + [ctypes.POINTER(spconv_csr)] + [_c_int] * 5 + [
        ctypes.c_uint32, ctypes.POINTER(spconv_options), _vp, ctypes.c_int64]
    lib.spconv_kernel_variants.restype = _c_int
    lib.spconv_kernel_variants.argtypes = [ctypes.c_int32, _vp, ctypes.c_int32, ctypes.POINTER(ctypes.c_int32)]
    return lib


_lib = _bind(ctypes.CDLL(str(LIB_PATH)))


class SpconvError(RuntimeError):
    def __init__(self, code: int, what: str):
        self.code = code
        super().__init__(f"{what}: {spconv_strerror(code)} ({code})")


def _check(code: int, what: str):
    if code != SPCONV_OK:
        raise SpconvError(code, what)


def spconv_strerror(code: int) -> str:
    return _lib.spconv_strerror(int(code)).decode()


def spconv_output_shape(H, W, R, S, stride, pad, flags):
    ho, wo = _c_int(), _c_int()
    _check(_lib.spconv_output_shape(H, W, R, S, stride, pad, flags, ctypes.byref(ho), ctypes.byref(wo)),
           "spconv_output_shape")
    return ho.value, wo.value


@dataclass
class HostCSR:
    """CSR filter in host memory, as written by ``spconv_pack_csr``."""
    K: int
    C: int
    R: int
    S: int
    Hp: int
    Wp: int
    rowptr: np.ndarray
    colidx: np.ndarray
    offset: np.ndarray
    vals: np.ndarray

    @property
    def nnz(self) -> int:
        return int(self.colidx.size)


def _np_ptr(a):
    return None if a is None else a.ctypes.data


def spconv_pack_csr(w: np.ndarray, mask: np.ndarray | None, Hp: int, Wp: int) -> HostCSR:
    """Two-phase call of ``spconv_pack_csr`` (count, then fill) on host arrays."""
    w = np.ascontiguousarray(w, dtype=np.float32)
    if w.ndim != 4:
        raise ValueError("w must be [K, C, R, S]")
    K, C, R, S = (int(v) for v in w.shape)
    m = None
    if mask is not None:
        m = np.ascontiguousarray(mask, dtype=np.uint8)
        if m.shape != w.shape:
            raise ValueError("mask must have the weight's shape")
    nnz = ctypes.c_int64()
    rowptr = np.zeros(K + 1, np.int32)
    _check(_lib.spconv_pack_csr(_np_ptr(w), _np_ptr(m), K, C, R, S, Hp, Wp, _np_ptr(rowptr), None, None, None, 0,
                                ctypes.byref(nnz)), "spconv_pack_csr (count)")
    n = nnz.value
    colidx = np.zeros(max(n, 1), np.int32)
    offset = np.zeros(max(n, 1), np.int32)
    vals = np.zeros(max(n, 1), np.float32)
    _check(_lib.spconv_pack_csr(_np_ptr(w), _np_ptr(m), K, C, R, S, Hp, Wp, _np_ptr(rowptr), _np_ptr(colidx),
                                _np_ptr(offset), _np_ptr(vals), n, ctypes.byref(nnz)), "spconv_pack_csr")
    return HostCSR(K, C, R, S, Hp, Wp, rowptr, colidx[:n], offset[:n], vals[:n])


def host_csr_struct(host: HostCSR) -> spconv_csr:
    """A ``spconv_csr`` whose arrays are the host arrays of ``host`` (for the
    host-side calls: spconv_pack_lowered, and plans)."""
    return spconv_csr(host.K, host.C, host.R, host.S, host.Hp, host.Wp, host.nnz, host.rowptr.ctypes.data,
                      host.colidx.ctypes.data, host.offset.ctypes.data, host.vals.ctypes.data)


def spconv_pack_lowered(host: HostCSR, N: int, H: int, W: int, stride: int, pad: int, flags: int,
                        max_row_nnz: int = 0) -> np.ndarray:
    """The lowered entry stream (int32 host array) for a forward call with these
    arguments (see ``spconv_pack_lowered`` in include/spconv.h)."""
    st = host_csr_struct(host)
    opt = spconv_options(0, 0, None, max_row_nnz, None, 0)
    words = ctypes.c_int64()
    _check(_lib.spconv_lowered_size(N, host.C, H, W, ctypes.byref(st), host.K, host.R, host.S, stride, pad, flags,
                                    ctypes.byref(opt), ctypes.byref(words)), "spconv_lowered_size")
    out = np.empty(words.value, np.int32)
    _check(_lib.spconv_pack_lowered(N, host.C, H, W, ctypes.byref(st), host.K, host.R, host.S, stride, pad, flags,
                                    ctypes.byref(opt), out.ctypes.data, out.size), "spconv_pack_lowered")
    return out


def spconv_dense_size(K: int, C: int, R: int, S: int) -> int:
    n = ctypes.c_int64()
    _check(_lib.spconv_dense_size(K, C, R, S, ctypes.byref(n)), "spconv_dense_size")
    return n.value


def spconv_pack_dense(w: np.ndarray, mask: np.ndarray | None) -> np.ndarray:
    """The filter packed for ``spconv_forward_dense`` (host float32 array)."""
    w = np.ascontiguousarray(w, dtype=np.float32)
    if w.ndim != 4:
        raise ValueError("w must be [K, C, R, S]")
    K, C, R, S = (int(v) for v in w.shape)
    m = None
    if mask is not None:
        m = np.ascontiguousarray(mask, dtype=np.uint8)
        if m.shape != w.shape:
            raise ValueError("mask must have the weight's shape")
    packed = np.empty(spconv_dense_size(K, C, R, S), np.float32)
    _check(_lib.spconv_pack_dense(_np_ptr(w), _np_ptr(m), K, C, R, S, _np_ptr(packed), packed.size),
           "spconv_pack_dense")
    return packed


def spconv_select_path(N: int, C: int, H: int, W: int, K: int, R: int, S: int, stride: int, pad: int, nnz: int,
                       flags: int) -> int:
    """SPCONV_PATH_SPARSE or SPCONV_PATH_DENSE: the path predicted faster."""
    path = _c_int()
    _check(_lib.spconv_select_path(N, C, H, W, K, R, S, stride, pad, nnz, flags, ctypes.byref(path)),
           "spconv_select_path")
    return path.value


def spconv_dense_plan(N: int, C: int, H: int, W: int, K: int, R: int, S: int, pad: int, flags: int) -> dict:
    info = spconv_plan_info()
    _check(_lib.spconv_dense_plan(N, C, H, W, K, R, S, pad, flags, ctypes.byref(info)), "spconv_dense_plan")
    return {name: getattr(info, name) for name, _ in spconv_plan_info._fields_}


class DeviceCSR:
    """A HostCSR copied to device memory (torch tensors) plus its C struct."""

    def __init__(self, host: HostCSR, device="cuda"):
        import torch
        self.host = host
        self.rowptr = torch.from_numpy(host.rowptr).to(device)
        # Keep at least one element so the device pointers are valid even when nnz == 0.
        self.colidx = torch.from_numpy(np.concatenate([host.colidx, np.zeros(1, np.int32)])).to(device)
        self.offset = torch.from_numpy(np.concatenate([host.offset, np.zeros(1, np.int32)])).to(device)
        self.vals = torch.from_numpy(np.concatenate([host.vals, np.zeros(1, np.float32)])).to(device)
        # The largest row's entry count: the planner's hint for skewed filters
        # (passed in spconv_options; the planner never reads the device arrays).
        self.max_row_nnz = int(np.diff(host.rowptr).max()) if host.K > 0 else 0
        self.struct = spconv_csr(host.K, host.C, host.R, host.S, host.Hp, host.Wp, host.nnz,
                                 self.rowptr.data_ptr(), self.colidx.data_ptr(), self.offset.data_ptr(),
                                 self.vals.data_ptr())


def _dev_ptr(t, name):
    import torch
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise TypeError(f"{name} must be a device tensor")
    if t.dtype != torch.float32 or not t.is_contiguous():
        raise TypeError(f"{name} must be a contiguous float32 tensor")
    return t.data_ptr()


def _check_shape(t, shape, name):
    if tuple(int(v) for v in t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")


def _check_numel(t, n, name):
    """The kernels index raw pointers: a buffer must hold every element they touch."""
    if t is not None and t.numel() < n:
        raise ValueError(f"{name} holds {t.numel()} elements, the call needs {n}")


def _in_elems(N, C, H, W, pad, flags):
    """Elements of the forward input: padded, or the raw tensor with SPCONV_UNPADDED_INPUT."""
    p = 0 if flags & SPCONV_UNPADDED_INPUT else pad
    return N * C * (H + 2 * p) * (W + 2 * p)


def _stream_of(stream, device):
    import torch
    return stream if stream is not None else torch.cuda.current_stream(device)


def _empty(shape, device, stream):
    """A new float32 device tensor whose memory belongs to ``stream``: torch's
    caching allocator ties a block to the stream current at allocation, and
    reuses it on that stream once the tensor is freed, so allocating on the
    stream the kernels run on keeps a freed temporary from being handed out
    while those kernels still use it."""
    import torch
    with torch.cuda.stream(stream):
        return torch.empty(shape, dtype=torch.float32, device=device)


def spconv_pad_input(x, pad: int, out=None, stream=None):
    """Zero-padded copy of NCHW ``x`` (device), queued on ``stream``."""
    if x.dim() != 4:
        raise ValueError("x must be NCHW")
    N, C, H, W = (int(v) for v in x.shape)
    s = _stream_of(stream, x.device)
    if out is None:
        out = _empty((N, C, H + 2 * pad, W + 2 * pad), x.device, s)
    _check_shape(out, (N, C, H + 2 * pad, W + 2 * pad), "out")
    _check(_lib.spconv_pad_input(_dev_ptr(x, "x"), N, C, H, W, pad, _dev_ptr(out, "out"), s.cuda_stream),
           "spconv_pad_input")
    return out


def spconv_resize_pad_input(x, H: int, W: int, pad: int, out=None, stream=None):
    """Bilinear resize (pixel centres aligned) of NCHW ``x`` to H x W, written
    with a zero border of ``pad`` into ``out`` [N, C, H+2pad, W+2pad] (device),
    queued on ``stream``."""
    if x.dim() != 4:
        raise ValueError("x must be NCHW")
    N, C, Hin, Win = (int(v) for v in x.shape)
    shape = (N, C, H + 2 * pad, W + 2 * pad)
    s = _stream_of(stream, x.device)
    if out is None:
        out = _empty(shape, x.device, s)
    _check_shape(out, shape, "out")
    _check(_lib.spconv_resize_pad_input(_dev_ptr(x, "x"), N, C, Hin, Win, H, W, pad, _dev_ptr(out, "out"),
                                        s.cuda_stream), "spconv_resize_pad_input")
    return out


def spconv_forward(xp, N: int, C: int, H: int, W: int, csr: DeviceCSR, K: int, R: int, S: int, stride: int,
                   pad: int, bias=None, flags: int = SPCONV_RELU, out=None, stream=None):
    """Fused sparse conv + bias + ReLU (+ 2x2 max-pool) on the padded input
    ``xp``: the plain ``spconv_forward`` call (no options, so the planner does
    not see ``csr``'s row skew)."""
    Ho, Wo = spconv_output_shape(H, W, R, S, stride, pad, flags)
    s = _stream_of(stream, xp.device)
    if out is None:
        out = _empty((N, K, Ho, Wo), xp.device, s)
    _check_numel(xp, _in_elems(N, C, H, W, pad, flags), "xp")
    _check_numel(out, N * K * Ho * Wo, "out")
    _check_numel(bias, K, "bias")
    _check(_lib.spconv_forward(_dev_ptr(xp, "xp"), N, C, H, W, ctypes.byref(csr.struct), K, R, S, stride, pad,
                               _dev_ptr(bias, "bias"), flags, _dev_ptr(out, "out"), s.cuda_stream),
           "spconv_forward")
    return out


def spconv_forward_ex(xp, N: int, C: int, H: int, W: int, csr: DeviceCSR, K: int, R: int, S: int, stride: int,
                      pad: int, bias=None, flags: int = SPCONV_RELU, out_pad: int = 0, residual=None,
                      residual_pad: int = 0, out=None, stream=None, max_row_nnz: int | None = None, lowered=None):
    """``spconv_forward`` with options: the stored planes get a zero border of
    ``out_pad`` (the next layer's padded input), ``residual`` (on the
    convolution's grid, with a border of ``residual_pad``) is added before the
    activation, the planner gets ``max_row_nnz`` (default: the value measured
    on ``csr``'s host arrays; 0 = unknown), and ``lowered`` (a device int32
    tensor from ``spconv_pack_lowered`` for this call) feeds the stride-1
    kernel its entries ready-made."""
    Hs, Ws = spconv_output_shape(H, W, R, S, stride, pad, flags)
    s = _stream_of(stream, xp.device)
    if out is None:
        out = _empty((N, K, Hs + 2 * out_pad, Ws + 2 * out_pad), xp.device, s)
    Hc, Wc = spconv_output_shape(H, W, R, S, stride, pad, flags & ~SPCONV_MAXPOOL2X2)
    _check_numel(xp, _in_elems(N, C, H, W, pad, flags), "xp")
    _check_numel(out, N * K * (Hs + 2 * out_pad) * (Ws + 2 * out_pad), "out")
    _check_numel(bias, K, "bias")
    _check_numel(residual, N * K * (Hc + 2 * residual_pad) * (Wc + 2 * residual_pad), "residual")
    hint = csr.max_row_nnz if max_row_nnz is None else max_row_nnz
    lw = None
    if lowered is not None:
        import torch
        if not isinstance(lowered, torch.Tensor) or lowered.device.type != "cuda" or lowered.dtype != torch.int32 \
                or not lowered.is_contiguous():
            raise TypeError("lowered must be a contiguous int32 device tensor")
        lw = lowered.data_ptr()
    opt = spconv_options(out_pad, residual_pad, _dev_ptr(residual, "residual"), hint, lw,
                         0 if lowered is None else lowered.numel())
    _check(_lib.spconv_forward_ex(_dev_ptr(xp, "xp"), N, C, H, W, ctypes.byref(csr.struct), K, R, S, stride, pad,
                                  _dev_ptr(bias, "bias"), flags, ctypes.byref(opt), _dev_ptr(out, "out"),
                                  s.cuda_stream), "spconv_forward_ex")
    return out


def spconv_forward_dense(xp, N: int, C: int, H: int, W: int, packed, K: int, R: int, S: int, pad: int, bias=None,
                         flags: int = SPCONV_RELU, out_pad: int = 0, residual=None, residual_pad: int = 0, out=None,
                         stream=None):
    """The fused conv of ``spconv_forward_ex`` from the packed dense filter
    ``packed`` (device), stride 1."""
    Hs, Ws = spconv_output_shape(H, W, R, S, 1, pad, flags)
    s = _stream_of(stream, xp.device)
    if out is None:
        out = _empty((N, K, Hs + 2 * out_pad, Ws + 2 * out_pad), xp.device, s)
    Hc, Wc = spconv_output_shape(H, W, R, S, 1, pad, flags & ~SPCONV_MAXPOOL2X2)
    _check_numel(xp, _in_elems(N, C, H, W, pad, flags), "xp")
    _check_numel(packed, spconv_dense_size(K, C, R, S), "packed")
    _check_numel(out, N * K * (Hs + 2 * out_pad) * (Ws + 2 * out_pad), "out")
    _check_numel(bias, K, "bias")
    _check_numel(residual, N * K * (Hc + 2 * residual_pad) * (Wc + 2 * residual_pad), "residual")
    opt = spconv_options(out_pad, residual_pad, _dev_ptr(residual, "residual"), 0, None, 0)
    _check(_lib.spconv_forward_dense(_dev_ptr(xp, "xp"), N, C, H, W, _dev_ptr(packed, "packed"), K, R, S, pad,
                                     _dev_ptr(bias, "bias"), flags, ctypes.byref(opt), _dev_ptr(out, "out"),
                                     s.cuda_stream), "spconv_forward_dense")
    return out


def spconv_plan(N: int, C: int, H: int, W: int, csr, K: int, R: int, S: int, stride: int, pad: int,
                flags: int = SPCONV_RELU, max_row_nnz: int | None = None, lowered: bool = False) -> dict:
    """The launch plan ``spconv_forward_ex`` would use, as a dict of the
    ``spconv_plan_info`` fields. ``csr`` is a DeviceCSR (its arrays are not
    read; the hint defaults to its measured max_row_nnz) or a bare
    ``spconv_csr`` struct (hint default 0); ``lowered``: the call passes a
    lowered stream (only its presence matters to the plan)."""
    struct = csr.struct if isinstance(csr, DeviceCSR) else csr
    if max_row_nnz is None:
        max_row_nnz = csr.max_row_nnz if isinstance(csr, DeviceCSR) else 0
    opt = spconv_options(0, 0, None, max_row_nnz, 16 if lowered else None, 0)
    info = spconv_plan_info()
    _check(_lib.spconv_plan(N, C, H, W, ctypes.byref(struct), K, R, S, stride, pad, flags, ctypes.byref(opt),
                            ctypes.byref(info)), "spconv_plan")
    return {name: getattr(info, name) for name, _ in spconv_plan_info._fields_}


def spconv_kernel_variants(kernel: int) -> list:
    """The compiled instances of a kernel family, as 4-tuples (see
    ``spconv_kernel_variants`` in include/spconv.h)."""
    count = ctypes.c_int32()
    _check(_lib.spconv_kernel_variants(kernel, None, 0, ctypes.byref(count)), "spconv_kernel_variants (count)")
    buf = np.zeros(4 * max(count.value, 1), np.int32)
    _check(_lib.spconv_kernel_variants(kernel, _np_ptr(buf), count.value, ctypes.byref(count)),
           "spconv_kernel_variants")
    return [tuple(int(v) for v in buf[4 * i:4 * i + 4]) for i in range(count.value)]


def flags_of(relu: bool, pool: bool) -> int:
    return (SPCONV_RELU if relu else 0) | (SPCONV_MAXPOOL2X2 if pool else 0)


class SparseConvLayer:
    """One layer's device state: the packed CSR, bias and shape, ready to run.

    ``run(x)`` queues pad + fused forward on the current stream and returns the
    output tensor. ``path`` picks the kernel family: "sparse" (the CSR kernels),
    "dense" (the MFMA kernel on the packed dense filter) or "auto" (the one
    ``spconv_select_path`` predicts faster for this layer; needs the batch
    size ``N``). ``self.path`` is the resolved choice.
    """

    def __init__(self, w: np.ndarray, mask: np.ndarray | None, bias: np.ndarray | None, H: int, W: int,
                 stride: int = 1, pad: int = 1, relu: bool = True, pool: bool = False, device="cuda",
                 path: str = "sparse", N: int | None = None, lowered: bool = True):
        import torch
        # lowered: feed stride-1 sparse plans their entries as a lowered stream
        # (spconv_pack_lowered, packed once per batch size and flags); False
        # keeps the plain CSR walk.
        self.use_lowered = lowered
        self.device = device
        self._lowered_cache = {}
        self.K, self.C, self.R, self.S = (int(v) for v in w.shape)
        self.H, self.W, self.stride, self.pad = H, W, stride, pad
        self.flags = flags_of(relu, pool)
        self.host_csr = spconv_pack_csr(w, mask, H + 2 * pad, W + 2 * pad)
        if path == "auto":
            if N is None:
                raise ValueError('path="auto" needs the batch size N')
            sel = spconv_select_path(N, self.C, H, W, self.K, self.R, self.S, stride, pad, self.host_csr.nnz,
                                     self.flags)
            path = "dense" if sel == SPCONV_PATH_DENSE else "sparse"
        if path not in ("sparse", "dense"):
            raise ValueError(f"unknown path {path!r}")
        if path == "dense" and stride != 1:
            raise ValueError("the dense path is stride 1 only")
        self.path = path
        self.csr = DeviceCSR(self.host_csr, device)
        self.dense = torch.from_numpy(spconv_pack_dense(w, mask)).to(device) if path == "dense" else None
        self.bias = None if bias is None else torch.from_numpy(np.ascontiguousarray(bias, np.float32)).to(device)
        self.Ho, self.Wo = spconv_output_shape(H, W, self.R, self.S, stride, pad, self.flags)

    def pad_input(self, x, out=None, stream=None):
        return spconv_pad_input(x, self.pad, out=out, stream=stream)

    def resize_pad_input(self, x, out=None, stream=None):
        """Bilinear resize of ``x`` to this layer's H x W, written as its padded input."""
        return spconv_resize_pad_input(x, self.H, self.W, self.pad, out=out, stream=stream)

    def forward_padded(self, xp, out=None, stream=None, out_pad: int = 0, residual=None, residual_pad: int = 0,
                       _extra_flags: int = 0):
        """Fused forward on the padded input. With ``out_pad`` the output planes
        carry that zero border (ready as the next layer's padded input); with
        ``residual`` (border ``residual_pad``) the shortcut is added before the
        activation."""
        N = int(xp.shape[0])
        flags = self.flags | _extra_flags
        if self.path == "dense":
            return spconv_forward_dense(xp, N, self.C, self.H, self.W, self.dense, self.K, self.R, self.S, self.pad,
                                        self.bias, flags, out_pad=out_pad, residual=residual,
                                        residual_pad=residual_pad, out=out, stream=stream)
        # Through spconv_forward_ex, so that the planner sees the filter's row
        # skew (max_row_nnz) whatever the epilogue.
        return spconv_forward_ex(xp, N, self.C, self.H, self.W, self.csr, self.K, self.R, self.S, self.stride,
                                 self.pad, self.bias, flags, out_pad=out_pad, residual=residual,
                                 residual_pad=residual_pad, out=out, stream=stream, lowered=self.lowered(N, flags))

    def lowered(self, N: int, flags: int | None = None):
        """The device lowered entry stream for batch size ``N`` and ``flags``
        (cached), or None when this layer does not use one (dense path, an
        any-stride plan, or ``lowered=False``)."""
        flags = self.flags if flags is None else flags
        if self.path != "sparse" or not self.use_lowered:
            return None
        key = (N, flags)
        if key not in self._lowered_cache:
            import torch
            p = spconv_plan(N, self.C, self.H, self.W, self.csr, self.K, self.R, self.S, self.stride, self.pad, flags)
            t = None
            if p["kernel"] == SPCONV_KERNEL_STRIDE1:
                host = spconv_pack_lowered(self.host_csr, N, self.H, self.W, self.stride, self.pad, flags,
                                           self.csr.max_row_nnz)
                t = torch.from_numpy(host).to(self.device)
            self._lowered_cache[key] = t
        return self._lowered_cache[key]

    # The dense kernel stages an unpadded input one image row per LDS-DMA
    # instruction, and on MI355X such a copy costs about the same per
    # instruction up to 1 KiB; rows narrower than this many bytes make the
    # copies slower than a separate pad pass (measured: 224-byte rows 3.4x the
    # time of 1 KiB copies for the same bytes, 896-byte rows on par).
    MIN_ROW_BYTES_PAD_IN_KERNEL = 768
    # The stride-1 sparse kernel fills whole 1 KiB LDS blocks per instruction
    # whatever the row length, 16 bytes per lane when the rows are whole 16-byte
    # groups: then forming the border costs less than a pad pass (measured at
    # 16x16, 28x28, 56x56, 224x224). With 4 bytes per lane (W not a multiple
    # of 4) the two cost about the same (14x14), and the pad pass is kept.

    def can_pad_in_kernel(self, N: int) -> bool:
        """Whether this layer's kernel can form the zero border itself (the
        dense kernel and stride-1 sparse plans)."""
        cache = self.__dict__.setdefault("_can_pad_in_kernel", {})
        if N not in cache:
            cache[N] = self.path == "dense" or self.plan(N)["kernel"] == SPCONV_KERNEL_STRIDE1
        return cache[N]

    def pads_in_kernel(self, N: int) -> bool:
        """Whether ``forward`` forms the zero border in the kernel (it can, and
        that beats a pad pass: rows of whole 16-byte groups for the sparse
        stride-1 kernel, wide enough rows for the dense kernel)."""
        if not self.can_pad_in_kernel(N):
            return False
        if self.path == "dense":
            return 4 * self.W >= self.MIN_ROW_BYTES_PAD_IN_KERNEL
        return self.W % 4 == 0

    def forward(self, x, out=None, stream=None, out_pad: int = 0, residual=None, residual_pad: int = 0, xp=None,
                pad_in_kernel: bool | None = None):
        """Fused forward on the unpadded NCHW input ``x``: the kernel forms the
        zero border while staging the input (SPCONV_UNPADDED_INPUT), or a pad
        pass into ``xp`` comes first. ``pad_in_kernel`` None picks the faster
        (``pads_in_kernel``); True requires the kernel path."""
        N = int(x.shape[0])
        if pad_in_kernel is None:
            pad_in_kernel = self.pads_in_kernel(N)
        if pad_in_kernel and not self.can_pad_in_kernel(N):
            raise ValueError("this layer's kernel cannot pad its input (any-stride plan)")
        if pad_in_kernel:
            if x.dim() != 4 or tuple(int(v) for v in x.shape[1:]) != (self.C, self.H, self.W):
                raise ValueError("x must be [N, C, H, W] of this layer")
            return self.forward_padded(x, out=out, stream=stream, out_pad=out_pad, residual=residual,
                                       residual_pad=residual_pad, _extra_flags=SPCONV_UNPADDED_INPUT)
        xp = self.pad_input(x, out=xp, stream=stream)
        return self.forward_padded(xp, out=out, stream=stream, out_pad=out_pad, residual=residual,
                                   residual_pad=residual_pad)

    def plan(self, N: int, unpadded: bool = False) -> dict:
        """The launch plan of a forward of batch N: on the padded input, or with
        ``unpadded`` on the unpadded one (the kernel forming the border, as
        ``forward`` does when ``pads_in_kernel``), whose LDS row pitch may differ."""
        flags = self.flags | (SPCONV_UNPADDED_INPUT if unpadded else 0)
        if self.path == "dense":
            return spconv_dense_plan(N, self.C, self.H, self.W, self.K, self.R, self.S, self.pad, flags)
        lw = self.path == "sparse" and self.use_lowered and spconv_plan(
            N, self.C, self.H, self.W, self.csr, self.K, self.R, self.S, self.stride, self.pad,
            flags)["kernel"] == SPCONV_KERNEL_STRIDE1
        return spconv_plan(N, self.C, self.H, self.W, self.csr, self.K, self.R, self.S, self.stride, self.pad,
                           flags, lowered=lw)

    def run(self, x, xp=None, out=None, stream=None):
        xp = self.pad_input(x, out=xp, stream=stream)
        return self.forward_padded(xp, out=out, stream=stream)
