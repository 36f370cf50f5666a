"""CPU oracle for the fused sparse direct convolution.

TEST INFRASTRUCTURE ONLY: the tests, ``__graft_entry__.smoke()`` and the CPU-baseline
leg of ``bench.py`` are the only callers. The GPU library never imports this package
and this package never imports the GPU library.

The arithmetic lives in ``spconv_oracle.c`` (plain C, double accumulation, OpenMP over
output planes); this module compiles it with gcc and marshals numpy arrays. Padding
uses ``numpy.pad``, a library routine standing in for the zero border of the padded
input the paper's CSR loop reads ("Sparse Convolution with CSR").
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from pathlib import Path

import numpy as np

HERE = Path(__file__).resolve().parent
SOURCE = HERE / "spconv_oracle.c"
LIB_PATH = HERE / "liboracle.so"

_i32p = ctypes.POINTER(ctypes.c_int32)
_f32p = ctypes.POINTER(ctypes.c_float)
_f64p = ctypes.POINTER(ctypes.c_double)
_u8p = ctypes.POINTER(ctypes.c_uint8)


def build(source: Path | str = SOURCE, out: Path | str = LIB_PATH, extra_flags=()) -> Path:
    """Compile the oracle with gcc -O2 (no fast-math) into a shared library."""
    out = Path(out)
    tmp = out.with_name(out.name + f".tmp{os.getpid()}")
    cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", *extra_flags,
           str(source), "-o", str(tmp), "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


class Oracle:
    """ctypes view of one compiled oracle library (the real one, or a test mutant)."""

    def __init__(self, path: Path | str):
        self.path = Path(path)
        lib = ctypes.CDLL(str(self.path))
        lib.oracle_pack_csr.restype = ctypes.c_longlong
        lib.oracle_pack_csr.argtypes = [_f32p, _u8p, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                        ctypes.c_int, ctypes.c_int, _i32p, _i32p, _i32p, _f32p]
        lib.oracle_conv.restype = ctypes.c_int
        lib.oracle_conv.argtypes = [_f32p, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, _f32p, _u8p,
                                    ctypes.c_int, ctypes.c_int, ctypes.c_int, _f32p, ctypes.c_int, ctypes.c_int,
                                    ctypes.c_int, ctypes.c_int, _i32p, ctypes.c_int, _f64p, _f64p, ctypes.c_int]
        lib.oracle_conv_res.restype = ctypes.c_int
        lib.oracle_conv_res.argtypes = [_f32p, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, _f32p, _u8p,
                                        ctypes.c_int, ctypes.c_int, ctypes.c_int, _f32p, _f32p, ctypes.c_int,
                                        ctypes.c_int, ctypes.c_int, ctypes.c_int, _i32p, ctypes.c_int, _f64p, _f64p,
                                        ctypes.c_int]
        lib.oracle_resize_bilinear.restype = None
        lib.oracle_resize_bilinear.argtypes = [_f32p, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                               ctypes.c_int, ctypes.c_int, _f64p, _f64p]
        lib.oracle_max_threads.restype = ctypes.c_int
        lib.oracle_max_threads.argtypes = []
        self._lib = lib

    def max_threads(self) -> int:
        return int(self._lib.oracle_max_threads())

    def pack_csr(self, w: np.ndarray, mask: np.ndarray | None, Hp: int, Wp: int):
        """CSR of the (K, C*R*S) view of ``w`` (paper, "Sparse Convolution with CSR").

        Returns ``(rowptr, colidx, offset, vals)`` with int32 indices and fp32 values
        bit-copied from ``w``.
        """
        w = np.ascontiguousarray(w, dtype=np.float32)
        K, C, R, S = w.shape
        m = None if mask is None else np.ascontiguousarray(mask, dtype=np.uint8)
        if m is not None and m.shape != w.shape:
            raise ValueError("mask shape must equal weight shape")
        cap = max(1, w.size)
        rowptr = np.zeros(K + 1, np.int32)
        colidx = np.zeros(cap, np.int32)
        offset = np.zeros(cap, np.int32)
        vals = np.zeros(cap, np.float32)
        nnz = self._lib.oracle_pack_csr(_ptr(w, _f32p), _ptr(m, _u8p), K, C, R, S, Hp, Wp, _ptr(rowptr, _i32p),
                                        _ptr(colidx, _i32p), _ptr(offset, _i32p), _ptr(vals, _f32p))
        return rowptr, colidx[:nnz].copy(), offset[:nnz].copy(), vals[:nnz].copy()

    def conv(self, x: np.ndarray, w: np.ndarray, mask: np.ndarray | None = None, bias: np.ndarray | None = None,
             stride: int = 1, pad: int = 0, relu: bool = False, pool: bool = False, pairs=None,
             nthreads: int = 0, residual: np.ndarray | None = None):
        """Fused conv -> (bias) -> (+ residual) -> ReLU -> 2x2 max-pool, in double precision.

        ``residual`` (N, K, Ho, Wo), if given, is added to the pre-activation on
        the convolution's own grid (the shortcut of a ResNet basic block).
        Returns ``(out, absacc)``: float64 arrays of shape (N, K, Ho', Wo') or, when
        ``pairs`` (a sequence of (n, k)) is given, (len(pairs), Ho', Wo').
        """
        x = np.ascontiguousarray(x, dtype=np.float32)
        w = np.ascontiguousarray(w, dtype=np.float32)
        N, C, H, W = x.shape
        K, C2, R, S = w.shape
        if C2 != C:
            raise ValueError("weight input channels must equal input channels")
        m = None if mask is None else np.ascontiguousarray(mask, dtype=np.uint8)
        b = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
        Ho = (H + 2 * pad - R) // stride + 1
        Wo = (W + 2 * pad - S) // stride + 1
        if Ho < 1 or Wo < 1:
            raise ValueError("empty output")
        Hq, Wq = (Ho // 2, Wo // 2) if pool else (Ho, Wo)
        if pairs is None:
            pr = None
            shape = (N, K, Hq, Wq)
            npairs = 0
        else:
            pr = np.ascontiguousarray(np.asarray(pairs, dtype=np.int32).reshape(-1, 2))
            if pr.size and (pr[:, 0].min() < 0 or pr[:, 0].max() >= N or pr[:, 1].min() < 0 or pr[:, 1].max() >= K):
                raise ValueError("pair out of range")
            npairs = pr.shape[0]
            shape = (npairs, Hq, Wq)
        out = np.zeros(shape, np.float64)
        ab = np.zeros(shape, np.float64)
        if residual is None:
            rc = self._lib.oracle_conv(_ptr(x, _f32p), N, C, H, W, _ptr(w, _f32p), _ptr(m, _u8p), K, R, S,
                                       _ptr(b, _f32p), stride, pad, int(bool(relu)), int(bool(pool)),
                                       _ptr(pr, _i32p), npairs, _ptr(out, _f64p), _ptr(ab, _f64p), int(nthreads))
        else:
            res = np.ascontiguousarray(residual, dtype=np.float32)
            if res.shape != (N, K, Ho, Wo):
                raise ValueError(f"residual must have shape {(N, K, Ho, Wo)}")
            rc = self._lib.oracle_conv_res(_ptr(x, _f32p), N, C, H, W, _ptr(w, _f32p), _ptr(m, _u8p), K, R, S,
                                           _ptr(b, _f32p), _ptr(res, _f32p), stride, pad, int(bool(relu)),
                                           int(bool(pool)), _ptr(pr, _i32p), npairs, _ptr(out, _f64p),
                                           _ptr(ab, _f64p), int(nthreads))
        if rc != 0:
            raise ValueError("oracle_conv rejected the shapes")
        return out, ab

    def resize(self, x: np.ndarray, H: int, W: int):
        """Bilinear resize (half-pixel centres, clamped at the borders) of NCHW
        ``x`` to H x W, in double. Returns ``(out, absacc)``."""
        x = np.ascontiguousarray(x, dtype=np.float32)
        N, C, Hin, Win = x.shape
        if min(N, C, Hin, Win, H, W) < 1:
            raise ValueError("empty resize")
        out = np.zeros((N, C, H, W), np.float64)
        ab = np.zeros((N, C, H, W), np.float64)
        self._lib.oracle_resize_bilinear(_ptr(x, _f32p), N, C, Hin, Win, H, W, _ptr(out, _f64p), _ptr(ab, _f64p))
        return out, ab

    @staticmethod
    def pad(x: np.ndarray, pad: int) -> np.ndarray:
        """Zero-padded NCHW copy (the padded input the CSR offsets index)."""
        return np.pad(np.ascontiguousarray(x, dtype=np.float32), ((0, 0), (0, 0), (pad, pad), (pad, pad)))


def _ptr(a, ptype):
    if a is None:
        return ctypes.cast(None, ptype)
    return a.ctypes.data_as(ptype)


_default: Oracle | None = None


def get() -> Oracle:
    """The oracle built from ``spconv_oracle.c`` (compiled here only if no build exists)."""
    global _default
    if _default is None:
        if not LIB_PATH.exists():
            build()
        _default = Oracle(LIB_PATH)
    return _default


def pack_csr(*a, **k):
    return get().pack_csr(*a, **k)


def conv(*a, **k):
    return get().conv(*a, **k)


def pad(x, p):
    return Oracle.pad(x, p)


def resize(*a, **k):
    return get().resize(*a, **k)
