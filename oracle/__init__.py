"""Plain CPU oracle for the fp32 GEMM and the NHWC 2-D convolution forward.

TEST INFRASTRUCTURE ONLY: the product package never imports this module.  Only
``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` use it.  It shares no code with the HIP path.

The arithmetic lives in ``oracle.c`` (plain C, fp64 accumulation, one output
element at a time -- the GEMM definition of Section 3.1, the convolution of
Algorithm 1 with the centred window of Section 4.1, and the Winograd F(2x2, 3x3)
and F(4x4, 3x3) steps of Section 4.1.2 with their absolute-value error scale).  This module only builds
that file with gcc, marshals numpy arrays into it and applies the acceptance
rule ``|result - ref| <= rtol * scale`` where ``scale = sum_k |a_ik * b_kj|``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

# Acceptance bound on |result - ref| / sum_k |a*b| for fp32 results.
RTOL = 1e-5

_i64 = ctypes.c_int64
_f32 = ctypes.c_float
_p = ctypes.c_void_p


def build(force: bool = True) -> str:
    """Compile oracle.c into liboracle.so with gcc (OpenMP, -O2)."""
    if not force and os.path.exists(_LIB_PATH) and \
            os.path.getmtime(_LIB_PATH) >= os.path.getmtime(_SRC):
        return _LIB_PATH
    tmp = _LIB_PATH + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
           "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _bind(path):
    lib = ctypes.CDLL(path)
    lib.oracle_sgemm.argtypes = [ctypes.c_char, ctypes.c_char, _i64, _i64, _i64,
                                 _f32, _p, _i64, _p, _i64, _f32, _p, _i64, _p, _p]
    lib.oracle_sgemm_at.argtypes = [ctypes.c_char, ctypes.c_char, _i64, _i64, _i64,
                                    _f32, _p, _i64, _p, _i64, _f32, _p, _i64,
                                    _i64, _p, _p, _p, _p]
    lib.oracle_conv2d_out_dims.argtypes = [_i64] * 10 + [_p, _p]
    lib.oracle_same_pads.argtypes = [_i64] * 6 + [_p]
    conv_geom = [_p, _i64, _i64, _i64, _i64, _p, _i64, _i64, _i64,
                 _i64, _i64, _i64, _i64, _i64, _i64, _i64, _i64]
    lib.oracle_conv2d.argtypes = conv_geom + [_p, _p]
    lib.oracle_conv2d_at.argtypes = conv_geom + [_i64, _p, _p, _p]
    wino_geom = [_p, _i64, _i64, _i64, _i64, _p, _i64, _i64, _i64, _i64, _i64, _i64, _i64]
    for m in (2, 4):
        getattr(lib, "oracle_winograd_f%dx3" % m).argtypes = wino_geom + [_p, _p]
        getattr(lib, "oracle_winograd_f%dx3_at" % m).argtypes = wino_geom + [_i64, _p, _p, _p]
    lib.oracle_num_threads.restype = ctypes.c_int
    lib.oracle_set_threads.argtypes = [ctypes.c_int]
    return lib


def _ptr(a):
    if a is None:
        return None
    return a.ctypes.data


def _f32_buf(a):
    a = np.asarray(a)
    if a.dtype != np.float32:
        raise TypeError("oracle inputs are float32 arrays, got %s" % a.dtype)
    return np.ascontiguousarray(a).reshape(-1)


def _trans(t) -> bytes:
    if isinstance(t, bool):
        return b"T" if t else b"N"
    return str(t).encode()[:1]


def _check(status: int, what: str) -> None:
    if status != 0:
        raise ValueError("oracle: invalid arguments to %s" % what)


class Oracle:
    """The oracle's entry points over one compiled copy of oracle.c."""

    def __init__(self, path: str):
        self.path = path
        self._lib = _bind(path)

    def num_threads(self) -> int:
        return self._lib.oracle_num_threads()

    def set_threads(self, n: int) -> None:
        self._lib.oracle_set_threads(int(n))

    # -------------------------------------------------------------- GEMM

    def sgemm(self, trans_a, trans_b, M, N, K, alpha, A, lda, B, ldb, beta, C, ldc):
        """Whole product alpha op(A) op(B) + beta C.  Returns (ref, scale), M x N fp64."""
        A, B = _f32_buf(A), _f32_buf(B)
        Cb = _f32_buf(C) if C is not None else None
        ref = np.empty((M, N), dtype=np.float64)
        scale = np.empty((M, N), dtype=np.float64)
        st = self._lib.oracle_sgemm(_trans(trans_a), _trans(trans_b), M, N, K, alpha,
                                    _ptr(A), lda, _ptr(B), ldb, beta, _ptr(Cb), ldc,
                                    _ptr(ref), _ptr(scale))
        _check(st, "sgemm")
        return ref, scale

    def sgemm_at(self, trans_a, trans_b, M, N, K, alpha, A, lda, B, ldb, beta, C, ldc,
                 rows, cols):
        """Elements (rows[s], cols[s]) of alpha op(A) op(B) + beta C.  Returns (ref, scale)."""
        A, B = _f32_buf(A), _f32_buf(B)
        Cb = _f32_buf(C) if C is not None else None
        rows = np.ascontiguousarray(rows, dtype=np.int64)
        cols = np.ascontiguousarray(cols, dtype=np.int64)
        ref = np.empty(rows.shape, dtype=np.float64)
        scale = np.empty(rows.shape, dtype=np.float64)
        st = self._lib.oracle_sgemm_at(_trans(trans_a), _trans(trans_b), M, N, K, alpha,
                                       _ptr(A), lda, _ptr(B), ldb, beta, _ptr(Cb), ldc,
                                       rows.size, _ptr(rows), _ptr(cols),
                                       _ptr(ref), _ptr(scale))
        _check(st, "sgemm_at")
        return ref, scale

    # ------------------------------------------------------- convolution

    def conv2d_out_dims(self, H, W, KH, KW, sh, sw, pt, pl, pb, pr):
        ho = ctypes.c_int64()
        wo = ctypes.c_int64()
        st = self._lib.oracle_conv2d_out_dims(H, W, KH, KW, sh, sw, pt, pl, pb, pr,
                                              ctypes.addressof(ho), ctypes.addressof(wo))
        _check(st, "conv2d_out_dims")
        return ho.value, wo.value

    def same_pads(self, H, W, KH, KW, sh, sw):
        pads = (ctypes.c_int64 * 4)()
        st = self._lib.oracle_same_pads(H, W, KH, KW, sh, sw, ctypes.addressof(pads))
        _check(st, "same_pads")
        return tuple(pads)

    def _conv_args(self, x, f, stride, pads):
        x = np.asarray(x)
        f = np.asarray(f)
        if x.ndim != 4 or f.ndim != 4:
            raise ValueError("x is N x H x W x Cin, f is KH x KW x Cin x Cout")
        N, H, W, Cin = x.shape
        KH, KW, Cin2, Cout = f.shape
        if Cin2 != Cin:
            raise ValueError("channel mismatch")
        sh, sw = stride
        pt, pl, pb, pr = pads
        Ho, Wo = self.conv2d_out_dims(H, W, KH, KW, sh, sw, pt, pl, pb, pr)
        xb, fb = _f32_buf(x), _f32_buf(f)
        geom = [_ptr(xb), N, H, W, Cin, _ptr(fb), KH, KW, Cout, sh, sw, pt, pl, pb, pr, Ho, Wo]
        return geom, (N, Ho, Wo, Cout), (xb, fb)

    def conv2d(self, x, f, stride=(1, 1), pads=(0, 0, 0, 0)):
        """Whole NHWC output.  Returns (ref, scale), N x Ho x Wo x Cout fp64."""
        geom, shape, keep = self._conv_args(x, f, stride, pads)
        ref = np.empty(shape, dtype=np.float64)
        scale = np.empty(shape, dtype=np.float64)
        st = self._lib.oracle_conv2d(*geom, _ptr(ref), _ptr(scale))
        _check(st, "conv2d")
        del keep
        return ref, scale

    def conv2d_at(self, x, f, stride, pads, flat_idx):
        """Outputs at flat NHWC indices.  Returns (ref, scale) fp64."""
        geom, _shape, keep = self._conv_args(x, f, stride, pads)
        flat_idx = np.ascontiguousarray(flat_idx, dtype=np.int64)
        ref = np.empty(flat_idx.shape, dtype=np.float64)
        scale = np.empty(flat_idx.shape, dtype=np.float64)
        st = self._lib.oracle_conv2d_at(*geom, flat_idx.size, _ptr(flat_idx),
                                        _ptr(ref), _ptr(scale))
        _check(st, "conv2d_at")
        del keep
        return ref, scale

    # ------------------------------------ Winograd F(2x2, 3x3), F(4x4, 3x3)

    def _wino_args(self, x, f, pads):
        f = np.asarray(f)
        if f.ndim != 4 or f.shape[0] != 3 or f.shape[1] != 3:
            raise ValueError("Winograd F(m x m, 3x3) takes a 3 x 3 x Cin x Cout filter")
        geom, shape, keep = self._conv_args(x, f, (1, 1), pads)
        # drop KH, KW, sh, sw from the direct-convolution argument list
        wgeom = geom[:6] + [geom[8]] + geom[11:]
        return wgeom, shape, keep

    def winograd(self, m, x, f, pads=(1, 1, 1, 1)):
        """Whole NHWC output of the F(m x m, 3x3) computation (stride 1), m = 2 or 4.

        Returns (ref, scale) fp64: ref equals the convolution up to fp64
        rounding; scale is the absolute-value chain that bounds the rounding
        of the transformed computation."""
        if m not in (2, 4):
            raise ValueError("output tile m is 2 or 4")
        geom, shape, keep = self._wino_args(x, f, pads)
        ref = np.empty(shape, dtype=np.float64)
        scale = np.empty(shape, dtype=np.float64)
        st = getattr(self._lib, "oracle_winograd_f%dx3" % m)(*geom, _ptr(ref), _ptr(scale))
        _check(st, "winograd_f%dx3" % m)
        del keep
        return ref, scale

    def winograd_at(self, m, x, f, pads, flat_idx):
        """F(m x m, 3x3) outputs at flat NHWC indices.  Returns (ref, scale) fp64."""
        if m not in (2, 4):
            raise ValueError("output tile m is 2 or 4")
        geom, _shape, keep = self._wino_args(x, f, pads)
        flat_idx = np.ascontiguousarray(flat_idx, dtype=np.int64)
        ref = np.empty(flat_idx.shape, dtype=np.float64)
        scale = np.empty(flat_idx.shape, dtype=np.float64)
        st = getattr(self._lib, "oracle_winograd_f%dx3_at" % m)(*geom, flat_idx.size, _ptr(flat_idx),
                                                                _ptr(ref), _ptr(scale))
        _check(st, "winograd_f%dx3_at" % m)
        del keep
        return ref, scale

    def winograd_f2x3(self, x, f, pads=(1, 1, 1, 1)):
        return self.winograd(2, x, f, pads)

    def winograd_f2x3_at(self, x, f, pads, flat_idx):
        return self.winograd_at(2, x, f, pads, flat_idx)

    def winograd_f4x3(self, x, f, pads=(1, 1, 1, 1)):
        return self.winograd(4, x, f, pads)

    def winograd_f4x3_at(self, x, f, pads, flat_idx):
        return self.winograd_at(4, x, f, pads, flat_idx)


def compile_variant(src_text: str, out_path: str) -> "Oracle":
    """Compile a (test-modified) copy of the oracle source and bind it."""
    src = out_path + ".c"
    with open(src, "w") as fh:
        fh.write(src_text)
    subprocess.run(["gcc", "-O1", "-std=c11", "-fPIC", "-shared", "-fopenmp",
                    "-o", out_path, src, "-lm"], check=True)
    return Oracle(out_path)


def source() -> str:
    with open(_SRC) as fh:
        return fh.read()


def _default() -> Oracle:
    global _lib
    if _lib is None:
        build(force=False)
        _lib = Oracle(_LIB_PATH)
    return _lib


def num_threads() -> int:
    return _default().num_threads()


def set_threads(n: int) -> None:
    _default().set_threads(n)


def sgemm(*args, **kw):
    return _default().sgemm(*args, **kw)


def sgemm_at(*args, **kw):
    return _default().sgemm_at(*args, **kw)


def conv2d_out_dims(*args):
    return _default().conv2d_out_dims(*args)


def same_pads(*args):
    return _default().same_pads(*args)


def conv2d(*args, **kw):
    return _default().conv2d(*args, **kw)


def conv2d_at(*args, **kw):
    return _default().conv2d_at(*args, **kw)


def winograd_f2x3(*args, **kw):
    return _default().winograd_f2x3(*args, **kw)


def winograd_f2x3_at(*args, **kw):
    return _default().winograd_f2x3_at(*args, **kw)


def winograd_f4x3(*args, **kw):
    return _default().winograd_f4x3(*args, **kw)


def winograd_f4x3_at(*args, **kw):
    return _default().winograd_f4x3_at(*args, **kw)


def winograd(*args, **kw):
    return _default().winograd(*args, **kw)


def winograd_at(*args, **kw):
    return _default().winograd_at(*args, **kw)


# ------------------------------------------------------------ acceptance

def within_tolerance(result, ref, scale, rtol: float = RTOL, extra=None):
    """(ok, max_ratio, n_bad) for |result - ref| <= rtol * (scale + extra), per element.

    ``extra`` (default 0) widens the bound where the result also carries a
    term outside the sum of products, e.g. |beta * C| when the sum is empty.
    NaN or Inf in the result always fails; the max ratio is reported over
    the finite elements with a non-zero bound.
    """
    result = np.asarray(result, dtype=np.float64)
    bound = np.asarray(scale, dtype=np.float64)
    if extra is not None:
        bound = bound + np.asarray(extra, dtype=np.float64)
    finite = np.isfinite(result)
    diff = np.abs(result - ref)
    ok = finite & (diff <= rtol * bound)
    with np.errstate(divide="ignore", invalid="ignore"):
        ratio = np.where(diff == 0, 0.0, diff / bound)
    ratio = np.where(finite, ratio, np.inf)
    mx = float(np.max(ratio)) if ratio.size else 0.0
    n_bad = int(ratio.size - np.count_nonzero(ok))
    return n_bad == 0, mx, n_bad
