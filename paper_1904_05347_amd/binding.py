"""Python mirror of the C-ABI in include/pk.h (argument marshalling only).

Every call goes through libpk.so; there is no other compute path.  The
library must have been built (``python -m paper_1904_05347_amd.build``); a
missing library raises ``PkLibraryMissing`` instead of falling back to
anything.  torch is imported before the library is loaded so that both share
the one HIP runtime that torch brings.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("PK_LIBRARY") or os.path.join(HERE, "libpk.so")

PK_OK = 0
PK_ERR_INVALID_VALUE = 1
PK_ERR_NOT_SUPPORTED = 2
PK_ERR_WORKSPACE = 3
PK_ERR_LAUNCH = 4
PK_ERR_SCRATCH_LIMIT = 5
# bytes of the static device buffer pk_conv2d_fwd_noalloc works in (PK_NOALLOC_SCRATCH_BYTES)
NOALLOC_SCRATCH_BYTES = 80 << 20

_lib = None
_i64 = ctypes.c_int64
_p = ctypes.c_void_p


class PkLibraryMissing(RuntimeError):
    pass


class PkError(RuntimeError):
    def __init__(self, status: int, what: str, param: int = 0):
        self.status = status
        self.param = param
        msg = "%s: %s" % (what, _lib.pk_status_string(status).decode() if _lib else status)
        if status == PK_ERR_INVALID_VALUE:
            msg += " (argument %d)" % param
        super().__init__(msg)


class ConfigInfo(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char_p), ("kind", ctypes.c_int),
                ("bm", ctypes.c_int), ("bn", ctypes.c_int), ("bk", ctypes.c_int),
                ("waves_m", ctypes.c_int), ("waves_n", ctypes.c_int), ("threads", ctypes.c_int),
                ("trans_a", ctypes.c_int), ("trans_b", ctypes.c_int),
                ("vec_a", ctypes.c_int), ("vec_b", ctypes.c_int),
                ("stages", ctypes.c_int), ("lds_bytes", ctypes.c_int), ("occupancy", ctypes.c_int),
                ("persistent", ctypes.c_int), ("streamk", ctypes.c_int),
                ("bres", ctypes.c_int), ("kgroups", ctypes.c_int), ("dma", ctypes.c_int)]


class TuneResult(ctypes.Structure):
    _fields_ = [("config", ctypes.c_char * 64), ("splits", ctypes.c_int), ("ms", ctypes.c_float),
                ("candidates", ctypes.c_int)]


# Every symbol include/pk.h declares, with its ctypes signature.
SIGNATURES = {
    "pk_sgemm": (ctypes.c_int, [ctypes.c_char, ctypes.c_char, _i64, _i64, _i64, ctypes.c_float, _p, _i64,
                                _p, _i64, ctypes.c_float, _p, _i64, _p]),
    "pk_sgemm_workspace_bytes": (ctypes.c_size_t, [ctypes.c_char, ctypes.c_char, _i64, _i64, _i64]),
    "pk_sgemm_ws": (ctypes.c_int, [ctypes.c_char, ctypes.c_char, _i64, _i64, _i64, ctypes.c_float, _p, _i64,
                                   _p, _i64, ctypes.c_float, _p, _i64, _p, ctypes.c_size_t, _p]),
    "pk_conv2d_out_dims": (ctypes.c_int, [_i64] * 10 + [_p, _p]),
    "pk_conv2d_same_pads": (ctypes.c_int, [_i64] * 6 + [_p]),
    "pk_conv2d_workspace_bytes": (ctypes.c_size_t, [_i64] * 13),
    "pk_conv2d_fwd": (ctypes.c_int, [_p, _i64, _i64, _i64, _i64, _p, _i64, _i64, _i64,
                                     _i64, _i64, _i64, _i64, _i64, _i64, _p, _i64, _i64,
                                     _p, ctypes.c_size_t, _p]),
    "pk_conv2d_fwd_noalloc": (ctypes.c_int, [_p, _i64, _i64, _i64, _i64, _p, _i64, _i64, _i64,
                                             _i64, _i64, _i64, _i64, _i64, _i64, _p, _i64, _i64, _p]),
    "pk_conv2d_winograd_workspace_bytes": (ctypes.c_size_t, [_i64] * 9),
    "pk_conv2d_winograd_fwd": (ctypes.c_int, [_p, _i64, _i64, _i64, _i64, _p, _i64, _i64, _i64,
                                              _i64, _i64, _i64, _i64, _i64, _i64, _p, _i64, _i64,
                                              _p, ctypes.c_size_t, _p]),
    "pk_conv2d_winograd_tile_workspace_bytes": (ctypes.c_size_t, [_i64] * 10),
    "pk_conv2d_winograd_tile_fwd": (ctypes.c_int, [_p, _i64, _i64, _i64, _i64, _p, _i64, _i64, _i64,
                                                   _i64, _i64, _i64, _i64, _i64, _i64, _p, _i64, _i64, _i64,
                                                   _p, ctypes.c_size_t, _p]),
    "pk_tune_sgemm": (ctypes.c_int, [ctypes.c_char, ctypes.c_char, _i64, _i64, _i64, ctypes.c_float, _p, _i64,
                                     _p, _i64, ctypes.c_float, _p, _i64, _p, ctypes.c_size_t, ctypes.c_int, _p,
                                     ctypes.POINTER(TuneResult)]),
    "pk_tune_conv2d_fwd": (ctypes.c_int, [_p, _i64, _i64, _i64, _i64, _p, _i64, _i64, _i64,
                                          _i64, _i64, _i64, _i64, _i64, _i64, _p, _i64, _i64,
                                          _p, ctypes.c_size_t, ctypes.c_int, _p, ctypes.POINTER(TuneResult)]),
    "pk_tune_reset": (ctypes.c_int, []),
    "pk_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "pk_last_invalid_param": (ctypes.c_int, []),
    "pk_last_config_name": (ctypes.c_char_p, []),
    "pk_num_configs": (ctypes.c_int, []),
    "pk_get_config": (ctypes.c_int, [ctypes.c_int, ctypes.POINTER(ConfigInfo)]),
    "pk_force_config": (ctypes.c_int, [ctypes.c_char_p]),
    "pk_force_splits": (ctypes.c_int, [ctypes.c_int]),
    "pk_probe_mfma_peak": (ctypes.c_int, [ctypes.c_int, ctypes.c_int, _p, _p]),
    "pk_probe_mfma_data": (ctypes.c_int, [ctypes.c_int, ctypes.c_int, _p, _p, _p]),
    "pk_probe_copy": (ctypes.c_int, [_p, _p, _i64, _p]),
}


def load():
    """Load libpk.so (once).  Raises PkLibraryMissing when it was not built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise PkLibraryMissing("libpk.so is not built: run `python -m paper_1904_05347_amd.build`")
    try:
        import torch  # noqa: F401  (load torch's HIP runtime first: one runtime per process)
    except ImportError:
        pass
    lib = ctypes.CDLL(LIB_PATH)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(status: int, what: str) -> None:
    if status != PK_OK:
        raise PkError(status, what, _lib.pk_last_invalid_param())


def _trans(t) -> bytes:
    if isinstance(t, bool):
        return b"T" if t else b"N"
    return str(t).encode()[:1]


# ------------------------------------------------------------- raw entry points

def sgemm(trans_a, trans_b, M, N, K, alpha, A, lda, B, ldb, beta, C, ldc, stream=None) -> int:
    """pk_sgemm on raw device addresses; returns the status code."""
    return load().pk_sgemm(_trans(trans_a), _trans(trans_b), M, N, K, alpha, A, lda, B, ldb,
                           beta, C, ldc, stream)


def sgemm_ws(trans_a, trans_b, M, N, K, alpha, A, lda, B, ldb, beta, C, ldc, workspace=None,
             workspace_bytes=0, stream=None) -> int:
    """pk_sgemm_ws on raw device addresses; returns the status code."""
    return load().pk_sgemm_ws(_trans(trans_a), _trans(trans_b), M, N, K, alpha, A, lda, B, ldb,
                              beta, C, ldc, workspace, workspace_bytes, stream)


def sgemm_workspace_bytes(trans_a, trans_b, M, N, K) -> int:
    return load().pk_sgemm_workspace_bytes(_trans(trans_a), _trans(trans_b), M, N, K)


def conv2d_fwd_raw(x, N, H, W, Cin, f, KH, KW, Cout, sh, sw, pt, pl, pb, pr, y, Ho, Wo,
                   workspace=None, workspace_bytes=0, stream=None) -> int:
    """pk_conv2d_fwd on raw device addresses; returns the status code."""
    return load().pk_conv2d_fwd(x, N, H, W, Cin, f, KH, KW, Cout, sh, sw, pt, pl, pb, pr,
                                y, Ho, Wo, workspace, workspace_bytes, stream)


def conv2d_fwd_noalloc_raw(x, N, H, W, Cin, f, KH, KW, Cout, sh, sw, pt, pl, pb, pr, y, Ho, Wo,
                           stream=None) -> int:
    """pk_conv2d_fwd_noalloc on raw device addresses; returns the status code."""
    return load().pk_conv2d_fwd_noalloc(x, N, H, W, Cin, f, KH, KW, Cout, sh, sw, pt, pl, pb, pr,
                                        y, Ho, Wo, stream)


def conv2d_winograd_raw(x, N, H, W, Cin, f, KH, KW, Cout, sh, sw, pt, pl, pb, pr, y, Ho, Wo,
                        workspace, workspace_bytes, stream=None) -> int:
    """pk_conv2d_winograd_fwd on raw device addresses; returns the status code."""
    return load().pk_conv2d_winograd_fwd(x, N, H, W, Cin, f, KH, KW, Cout, sh, sw, pt, pl, pb, pr,
                                         y, Ho, Wo, workspace, workspace_bytes, stream)


def conv2d_winograd_workspace_bytes(N, H, W, Cin, Cout, pt, pl, pb, pr, tile=2) -> int:
    return load().pk_conv2d_winograd_tile_workspace_bytes(tile, N, H, W, Cin, Cout, pt, pl, pb, pr)


def conv2d_winograd_tile_raw(x, N, H, W, Cin, f, KH, KW, Cout, sh, sw, pt, pl, pb, pr, y, Ho, Wo, tile,
                             workspace, workspace_bytes, stream=None) -> int:
    """pk_conv2d_winograd_tile_fwd on raw device addresses; returns the status code."""
    return load().pk_conv2d_winograd_tile_fwd(x, N, H, W, Cin, f, KH, KW, Cout, sh, sw, pt, pl, pb, pr,
                                              y, Ho, Wo, tile, workspace, workspace_bytes, stream)


def conv2d_out_dims(H, W, KH, KW, sh, sw, pt, pl, pb, pr):
    ho, wo = ctypes.c_int64(), ctypes.c_int64()
    _check(load().pk_conv2d_out_dims(H, W, KH, KW, sh, sw, pt, pl, pb, pr,
                                     ctypes.addressof(ho), ctypes.addressof(wo)), "pk_conv2d_out_dims")
    return ho.value, wo.value


def conv2d_same_pads(H, W, KH, KW, sh, sw):
    pads = (ctypes.c_int64 * 4)()
    _check(load().pk_conv2d_same_pads(H, W, KH, KW, sh, sw, ctypes.addressof(pads)), "pk_conv2d_same_pads")
    return tuple(pads)


def conv2d_workspace_bytes(N, H, W, Cin, KH, KW, Cout, sh, sw, pt, pl, pb, pr) -> int:
    return load().pk_conv2d_workspace_bytes(N, H, W, Cin, KH, KW, Cout, sh, sw, pt, pl, pb, pr)


def last_config_name() -> str:
    return load().pk_last_config_name().decode()


def last_invalid_param() -> int:
    return load().pk_last_invalid_param()


def configs():
    lib = load()
    out = []
    for i in range(lib.pk_num_configs()):
        info = ConfigInfo()
        _check(lib.pk_get_config(i, ctypes.byref(info)), "pk_get_config")
        d = {k: getattr(info, k) for k, _ in ConfigInfo._fields_}
        d["name"] = d["name"].decode()
        out.append(d)
    return out


def force_config(name):
    _check(load().pk_force_config(name.encode() if name else None), "pk_force_config")


def force_splits(n: int):
    _check(load().pk_force_splits(int(n)), "pk_force_splits")


def probe_mfma_peak_tflops(blocks=2048, iters=2000):
    """Sustained fp32 MFMA rate (TFLOP/s) of back-to-back independent MFMAs."""
    import torch
    out = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")
    s = torch.cuda.current_stream()
    _check(load().pk_probe_mfma_peak(blocks, iters, out.data_ptr(), s.cuda_stream), "pk_probe_mfma_peak")
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(s)
    _check(load().pk_probe_mfma_peak(blocks, iters, out.data_ptr(), s.cuda_stream), "pk_probe_mfma_peak")
    e1.record(s)
    torch.cuda.synchronize()
    flops = blocks * 4 * iters * 4 * 4096
    return flops / (e0.elapsed_time(e1) * 1e-3) / 1e12


def probe_mfma_data_tflops(blocks=1024, iters=500):
    """As probe_mfma_peak_tflops, with random operands that change on every MFMA."""
    import torch
    src = torch.rand(1 << 20, dtype=torch.float32, device="cuda") * 2 - 1
    out = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")
    s = torch.cuda.current_stream()
    lib = load()
    _check(lib.pk_probe_mfma_data(blocks, iters, src.data_ptr(), out.data_ptr(), s.cuda_stream), "probe")
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(s)
    _check(lib.pk_probe_mfma_data(blocks, iters, src.data_ptr(), out.data_ptr(), s.cuda_stream), "probe")
    e1.record(s)
    torch.cuda.synchronize()
    flops = blocks * 4 * iters * 16 * 4096
    return flops / (e0.elapsed_time(e1) * 1e-3) / 1e12


def probe_copy_gbs(mib=2048, reps=5):
    """Sustained HBM bandwidth (GB/s, read + write) of a 16-byte streaming copy."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    s = torch.cuda.current_stream()
    _check(load().pk_probe_copy(src.data_ptr(), dst.data_ptr(), n, s.cuda_stream), "pk_probe_copy")
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(s)
    for _ in range(reps):
        _check(load().pk_probe_copy(src.data_ptr(), dst.data_ptr(), n, s.cuda_stream), "pk_probe_copy")
    e1.record(s)
    torch.cuda.synchronize()
    return reps * 8 * n / (e0.elapsed_time(e1) * 1e-3) / 1e9


# ------------------------------------------------------------ torch tensors

def _stream_handle(tensor):
    import torch
    return torch.cuda.current_stream(tensor.device).cuda_stream


def _check_f32_cuda(t, what):
    import torch
    if not isinstance(t, torch.Tensor) or t.dtype != torch.float32 or not t.is_cuda:
        raise TypeError("%s must be a float32 tensor on a HIP device" % what)


def _ld_2d(t, what):
    """Leading dimension of a row-major 2-D view (unit column stride)."""
    if t.dim() != 2:
        raise ValueError("%s must be 2-D" % what)
    if t.size(1) > 1 and t.stride(1) != 1:
        raise ValueError("%s must have unit column stride" % what)
    return max(t.stride(0), t.size(1), 1)


def gemm(a, b, c=None, alpha=1.0, beta=0.0, trans_a=False, trans_b=False, workspace=None):
    """C = alpha * op(a) @ op(b) + beta * c on the current stream.

    ``a`` is stored M x K (or K x M with trans_a), ``b`` K x N (or N x K with
    trans_b); both are row-major views with unit column stride.  Returns c
    (allocated when None; then beta must be 0).  workspace (a float32 device
    tensor) lets a product with few tiles split K across work-groups (see
    ``sgemm_workspace_bytes``); when None, one of the size the library asks
    for is allocated.
    """
    import torch
    _check_f32_cuda(a, "a")
    _check_f32_cuda(b, "b")
    lda, ldb = _ld_2d(a, "a"), _ld_2d(b, "b")
    M, K = (a.size(1), a.size(0)) if trans_a else (a.size(0), a.size(1))
    Kb, N = (b.size(1), b.size(0)) if trans_b else (b.size(0), b.size(1))
    if Kb != K:
        raise ValueError("inner dimensions differ: %d vs %d" % (K, Kb))
    if c is None:
        if beta != 0.0:
            raise ValueError("beta != 0 needs c")
        c = torch.empty((M, N), dtype=torch.float32, device=a.device)
    _check_f32_cuda(c, "c")
    if tuple(c.shape) != (M, N):
        raise ValueError("c must be %d x %d" % (M, N))
    ldc = _ld_2d(c, "c")
    if workspace is None:
        need = sgemm_workspace_bytes(bool(trans_a), bool(trans_b), M, N, K)
        if need:
            workspace = torch.empty((need + 3) // 4, dtype=torch.float32, device=a.device)
    ws_ptr, ws_bytes = None, 0
    if workspace is not None:
        _check_f32_cuda(workspace, "workspace")
        ws_ptr, ws_bytes = workspace.data_ptr(), workspace.numel() * 4
    st = sgemm_ws(bool(trans_a), bool(trans_b), M, N, K, float(alpha), a.data_ptr(), lda,
                  b.data_ptr(), ldb, float(beta), c.data_ptr(), ldc, ws_ptr, ws_bytes, _stream_handle(c))
    _check(st, "pk_sgemm_ws")
    return c


def resolve_padding(padding, H, W, KH, KW, sh, sw):
    if isinstance(padding, str):
        p = padding.upper()
        if p == "VALID":
            return (0, 0, 0, 0)
        if p == "SAME":
            return conv2d_same_pads(H, W, KH, KW, sh, sw)
        raise ValueError("padding must be 'SAME', 'VALID' or (top, left, bottom, right)")
    pads = tuple(int(v) for v in padding)
    if len(pads) != 4:
        raise ValueError("padding must be (top, left, bottom, right)")
    return pads


def conv2d_fwd(x, w, stride=(1, 1), padding="SAME", out=None, workspace=None):
    """NHWC x (N, H, W, Cin) convolved with HWIO w (KH, KW, Cin, Cout).

    ``padding`` is 'SAME', 'VALID' or (top, left, bottom, right).  The
    workspace (a float32 device tensor) lets the reduction be split across
    work-groups (split-K or stream-K, see ``conv2d_workspace_bytes``); when
    None, one of the size the chosen configuration needs is allocated.
    """
    import torch
    _check_f32_cuda(x, "x")
    _check_f32_cuda(w, "w")
    if x.dim() != 4 or w.dim() != 4:
        raise ValueError("x is N x H x W x Cin, w is KH x KW x Cin x Cout")
    if not x.is_contiguous() or not w.is_contiguous():
        raise ValueError("x and w must be contiguous (NHWC / HWIO)")
    N, H, W, Cin = x.shape
    KH, KW, Cin2, Cout = w.shape
    if Cin2 != Cin:
        raise ValueError("input channels differ: %d vs %d" % (Cin, Cin2))
    sh, sw = (stride, stride) if isinstance(stride, int) else tuple(stride)
    pt, pl, pb, pr = resolve_padding(padding, H, W, KH, KW, sh, sw)
    Ho, Wo = conv2d_out_dims(H, W, KH, KW, sh, sw, pt, pl, pb, pr)
    if out is None:
        out = torch.empty((N, Ho, Wo, Cout), dtype=torch.float32, device=x.device)
    _check_f32_cuda(out, "out")
    if tuple(out.shape) != (N, Ho, Wo, Cout) or not out.is_contiguous():
        raise ValueError("out must be a contiguous %s tensor" % ((N, Ho, Wo, Cout),))
    ws_ptr, ws_bytes = None, 0
    if workspace is None:
        need = conv2d_workspace_bytes(N, H, W, Cin, KH, KW, Cout, sh, sw, pt, pl, pb, pr)
        if need:
            workspace = torch.empty((need + 3) // 4, dtype=torch.float32, device=x.device)
    if workspace is not None:
        _check_f32_cuda(workspace, "workspace")
        ws_ptr, ws_bytes = workspace.data_ptr(), workspace.numel() * 4
    st = conv2d_fwd_raw(x.data_ptr(), N, H, W, Cin, w.data_ptr(), KH, KW, Cout, sh, sw,
                        pt, pl, pb, pr, out.data_ptr(), Ho, Wo, ws_ptr, ws_bytes, _stream_handle(out))
    _check(st, "pk_conv2d_fwd")
    return out


def conv2d_winograd(x, w, padding="SAME", out=None, workspace=None, tile=2):
    """Winograd F(tile x tile, 3x3) convolution of NHWC x with a 3 x 3 HWIO w,
    stride 1; tile (the output-tile size m) is 2 or 4.

    Same result as ``conv2d_fwd`` up to fp32 rounding of the transforms.  The
    workspace (float32 device tensor of at least
    ``conv2d_winograd_workspace_bytes(..., tile)`` bytes) is allocated when None.
    """
    import torch
    _check_f32_cuda(x, "x")
    _check_f32_cuda(w, "w")
    if x.dim() != 4 or w.dim() != 4:
        raise ValueError("x is N x H x W x Cin, w is KH x KW x Cin x Cout")
    if not x.is_contiguous() or not w.is_contiguous():
        raise ValueError("x and w must be contiguous (NHWC / HWIO)")
    N, H, W, Cin = x.shape
    KH, KW, Cin2, Cout = w.shape
    if Cin2 != Cin:
        raise ValueError("input channels differ: %d vs %d" % (Cin, Cin2))
    pt, pl, pb, pr = resolve_padding(padding, H, W, KH, KW, 1, 1)
    Ho, Wo = conv2d_out_dims(H, W, KH, KW, 1, 1, pt, pl, pb, pr)
    if out is None:
        out = torch.empty((N, Ho, Wo, Cout), dtype=torch.float32, device=x.device)
    _check_f32_cuda(out, "out")
    if tuple(out.shape) != (N, Ho, Wo, Cout) or not out.is_contiguous():
        raise ValueError("out must be a contiguous %s tensor" % ((N, Ho, Wo, Cout),))
    if workspace is None:
        need = conv2d_winograd_workspace_bytes(N, H, W, Cin, Cout, pt, pl, pb, pr, tile)
        workspace = torch.empty(max(need // 4, 1), dtype=torch.float32, device=x.device)
    _check_f32_cuda(workspace, "workspace")
    st = conv2d_winograd_tile_raw(x.data_ptr(), N, H, W, Cin, w.data_ptr(), KH, KW, Cout, 1, 1,
                                  pt, pl, pb, pr, out.data_ptr(), Ho, Wo, int(tile), workspace.data_ptr(),
                                  workspace.numel() * 4, _stream_handle(out))
    _check(st, "pk_conv2d_winograd_tile_fwd")
    return out


def _tune_dict(r):
    return {"config": r.config.decode(), "splits": r.splits, "ms": r.ms, "candidates": r.candidates}


def tune_gemm(a, b, c, alpha=1.0, beta=0.0, trans_a=False, trans_b=False, iters=5, workspace=None):
    """Time every compiled configuration (and reduction split the workspace
    allows) on these operands and record the fastest for this shape (see
    pk_tune_sgemm).  c is overwritten.  Without a workspace, one that holds
    16 splits (at least 256 MiB, for the stream-K plans; at most 1 GiB) is
    allocated."""
    import torch
    _check_f32_cuda(a, "a")
    _check_f32_cuda(b, "b")
    _check_f32_cuda(c, "c")
    lda, ldb, ldc = _ld_2d(a, "a"), _ld_2d(b, "b"), _ld_2d(c, "c")
    M, K = (a.size(1), a.size(0)) if trans_a else (a.size(0), a.size(1))
    Kb, N = (b.size(1), b.size(0)) if trans_b else (b.size(0), b.size(1))
    if Kb != K or tuple(c.shape) != (M, N):
        raise ValueError("operand shapes do not match")
    if workspace is None:
        need = min(max(16 * M * N * 4, 256 << 20), 1 << 30)
        workspace = torch.empty(need // 4, dtype=torch.float32, device=a.device)
    _check_f32_cuda(workspace, "workspace")
    r = TuneResult()
    st = load().pk_tune_sgemm(b"T" if trans_a else b"N", b"T" if trans_b else b"N", M, N, K, float(alpha),
                              a.data_ptr(), lda, b.data_ptr(), ldb, float(beta), c.data_ptr(), ldc,
                              workspace.data_ptr(), workspace.numel() * 4, int(iters),
                              _stream_handle(c), ctypes.byref(r))
    _check(st, "pk_tune_sgemm")
    return _tune_dict(r)


def tune_conv2d(x, w, stride=(1, 1), padding="SAME", out=None, workspace=None, iters=5):
    """Time every compiled configuration (and reduction split the workspace
    allows) on this convolution and record the fastest (see pk_tune_conv2d_fwd)."""
    import torch
    _check_f32_cuda(x, "x")
    _check_f32_cuda(w, "w")
    N, H, W, Cin = x.shape
    KH, KW, _, Cout = w.shape
    sh, sw = (stride, stride) if isinstance(stride, int) else tuple(stride)
    pt, pl, pb, pr = resolve_padding(padding, H, W, KH, KW, sh, sw)
    Ho, Wo = conv2d_out_dims(H, W, KH, KW, sh, sw, pt, pl, pb, pr)
    if out is None:
        out = torch.empty((N, Ho, Wo, Cout), dtype=torch.float32, device=x.device)
    ws_ptr, ws_bytes = None, 0
    if workspace is None:
        need = conv2d_workspace_bytes(N, H, W, Cin, KH, KW, Cout, sh, sw, pt, pl, pb, pr)
        if need:
            workspace = torch.empty((need + 3) // 4, dtype=torch.float32, device=x.device)
    if workspace is not None:
        _check_f32_cuda(workspace, "workspace")
        ws_ptr, ws_bytes = workspace.data_ptr(), workspace.numel() * 4
    r = TuneResult()
    st = load().pk_tune_conv2d_fwd(x.data_ptr(), N, H, W, Cin, w.data_ptr(), KH, KW, Cout, sh, sw, pt, pl, pb, pr,
                                   out.data_ptr(), Ho, Wo, ws_ptr, ws_bytes, int(iters), _stream_handle(out),
                                   ctypes.byref(r))
    _check(st, "pk_tune_conv2d_fwd")
    return _tune_dict(r)


def tune_reset():
    _check(load().pk_tune_reset(), "pk_tune_reset")
