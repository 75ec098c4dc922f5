"""MI355X (gfx950) integer-only quantized linear layer of MobileQuant
(arXiv 2408.13933), behind a C ABI (include/mq.h, libmq.so).

This module is the thin Python binding: each ``mq_*`` function has the
name of the C entry point it calls and only marshals arguments (torch
device tensors -> pointers, the current HIP stream -> ``void*``).  All
arithmetic runs in the HIP kernels of libmq.so; there is no fallback.  If
the library is missing, loading fails loudly.
"""
from __future__ import annotations

import ctypes
import os

__all__ = [
    "MQError", "lib", "lib_path", "mq_version", "mq_act_params", "mq_fold_weights",
    "mq_fold_acts", "mq_quantize_act", "mq_pack_weights", "mq_qlinear", "mq_dequant",
    "mq_pack_weights_asym", "mq_act_rowsum", "mq_quantize_act_rowsum", "mq_qlinear_asym",
    "mq_qlinear_a16", "mq_smooth_scales", "mq_arl_forward", "mq_arl_backward", "ARL_PARTIALS",
    "mq_add_requant", "mq_lut_build", "mq_lut_apply", "mq_rmsnorm", "mq_softmax", "LUT_SILU",
    "mq_qlinear_workspace_bytes", "mq_qlinear_noalloc", "NOALLOC_SCRATCH_BYTES",
    "PATH_AUTO", "PATH_DECODE", "PATH_PREFILL", "PATH_GENERIC", "MAX_K",
    "PATH_PREFILL_TILE0", "PREFILL_TILES", "prefill_tile_path", "mq_probe_read",
    "mq_qlinear_group", "MAX_GROUP", "QLinearOut", "mq_qlinear_dequant",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
lib_path = os.path.join(_HERE, "libmq.so")

MQ_OK, MQ_ERR_INVALID_ARG, MQ_ERR_UNSUPPORTED, MQ_ERR_HIP = 0, 1, 2, 3
PATH_AUTO, PATH_DECODE, PATH_PREFILL, PATH_GENERIC = 0, 1, 2, 3
# the prefill kernel with one explicit output tile (tests and measurements)
PATH_PREFILL_TILE0, PREFILL_TILES = 16, 6
PREFILL_TILE_SHAPES = ((256, 128), (128, 128), (192, 256), (64, 64), (256, 256), (128, 64))


def prefill_tile_path(tile: int) -> int:
    """Path value that runs the prefill kernel on output tile ``tile``."""
    if not 0 <= tile < PREFILL_TILES:
        raise ValueError(f"tile {tile} outside 0..{PREFILL_TILES - 1}")
    return PATH_PREFILL_TILE0 + tile
MAX_K = 65536
NOALLOC_SCRATCH_BYTES = 32 << 20
ARL_PARTIALS = 1024
LUT_SILU = 1

_lib = None


class MQError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {_status_string(status)}")


def _status_string(status: int) -> str:
    try:
        return lib().mq_status_string(status).decode()
    except Exception:
        return f"status {status}"


MAX_GROUP = 4  # MQ_MAX_GROUP


class QLinearOut(ctypes.Structure):
    """mq_qlinear_out of mq.h: one linear of an mq_qlinear_group call."""
    _fields_ = [("w_q", ctypes.c_void_p), ("w_scale", ctypes.c_void_p),
                ("w_zp", ctypes.c_void_p), ("w_colsum", ctypes.c_void_p),
                ("bias", ctypes.c_void_p), ("N", ctypes.c_int64), ("out_scale", ctypes.c_float),
                ("out_zp", ctypes.c_int32), ("y_q", ctypes.c_void_p)]


def lib():
    """The loaded libmq.so (ctypes), with argument types declared."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(lib_path):
        raise ImportError(f"{lib_path} is missing: build it with "
                          "`python -c 'import __graft_entry__ as g; g.build()'`")
    L = ctypes.CDLL(lib_path)
    c_i64, c_i32, c_f, c_p = ctypes.c_int64, ctypes.c_int32, ctypes.c_float, ctypes.c_void_p
    L.mq_status_string.argtypes = [ctypes.c_int]
    L.mq_status_string.restype = ctypes.c_char_p
    L.mq_version.argtypes = []
    L.mq_version.restype = c_i32
    L.mq_act_params.argtypes = [c_f, c_f, c_i32, ctypes.POINTER(c_f), ctypes.POINTER(c_i32)]
    L.mq_fold_weights.argtypes = [c_p, c_p, c_i64, c_i64, c_p, c_p]
    L.mq_fold_acts.argtypes = [c_p, c_p, c_i64, c_i64, c_p, c_p]
    L.mq_quantize_act.argtypes = [c_p, c_i64, c_f, c_i32, c_i32, c_p, c_p]
    L.mq_pack_weights.argtypes = [c_p, c_i64, c_i64, c_i32, c_p, c_p, c_p, c_p]
    L.mq_qlinear.argtypes = [c_p, c_i64, c_i64, c_i64, c_p, c_i32, c_p, c_p, c_f, c_i32, c_f,
                             c_i32, c_i32, c_p, c_p, c_p]
    L.mq_qlinear_ex.argtypes = [c_p, c_i64, c_i64, c_i64, c_p, c_i32, c_p, c_p, c_f, c_i32,
                                c_f, c_i32, c_i32, c_p, c_p, c_i32, c_p]
    L.mq_qlinear_ws.argtypes = [c_p, c_i64, c_i64, c_i64, c_p, c_i32, c_p, c_p, c_f, c_i32,
                                c_f, c_i32, c_i32, c_p, c_p, c_p, c_i64, c_i32, c_p]
    L.mq_qlinear_noalloc.argtypes = [c_p, c_i64, c_i64, c_i64, c_p, c_i32, c_p, c_p, c_f, c_i32,
                                     c_f, c_i32, c_i32, c_p, c_p, c_p]
    L.mq_qlinear_workspace_bytes.argtypes = [c_i64, c_i64, c_i64, c_i32, c_i32]
    L.mq_qlinear_workspace_bytes.restype = c_i64
    L.mq_dequant.argtypes = [c_p, c_i32, c_i64, c_f, c_i32, c_p, c_p]
    L.mq_pack_weights_asym.argtypes = [c_p, c_i64, c_i64, c_i32, c_i32, c_p, c_p, c_p, c_p,
                                       c_p]
    L.mq_act_rowsum.argtypes = [c_p, c_i64, c_i64, c_p, c_p]
    L.mq_quantize_act_rowsum.argtypes = [c_p, c_i64, c_i64, c_f, c_i32, c_p, c_p, c_p]
    L.mq_add_requant.argtypes = [c_p, c_f, c_i32, c_p, c_f, c_i32, c_i64, c_f, c_i32, c_i32, c_p,
                                 c_p]
    L.mq_lut_build.argtypes = [c_i32, c_f, c_i32, c_f, c_i32, c_i32, c_p, c_p]
    L.mq_lut_apply.argtypes = [c_p, c_i64, c_p, c_i32, c_p, c_p]
    L.mq_rmsnorm.argtypes = [c_p, c_i64, c_i64, c_f, c_i32, c_p, c_f, c_f, c_i32, c_i32, c_p, c_p]
    L.mq_softmax.argtypes = [c_p, c_i64, c_i64, c_f, c_i32, c_f, c_i32, c_i32, c_p, c_p]
    L.mq_mul_requant.argtypes = [c_p, c_f, c_i32, c_p, c_f, c_i32, c_i64, c_f, c_i32, c_i32, c_p,
                                 c_p]
    L.mq_rope.argtypes = [c_p, c_i64, c_i64, c_i64, c_f, c_i32, ctypes.c_double, c_i64, c_f, c_i32,
                          c_i32, c_p, c_p, c_p]
    L.mq_add_rmsnorm.argtypes = [c_p, c_f, c_i32, c_p, c_f, c_i32, c_i64, c_i64, c_f, c_i32, c_p,
                                 c_p, c_f, c_f, c_i32, c_i32, c_p, c_p]
    L.mq_lut_mul.argtypes = [c_p, c_p, c_i32, c_f, c_i32, c_p, c_f, c_i32, c_i64, c_f, c_i32,
                             c_i32, c_p, c_p]
    L.mq_rope_table.argtypes = [c_i64, c_i64, ctypes.c_double, c_i64, c_p, c_p]
    L.mq_rope_apply.argtypes = [c_p, c_i64, c_i64, c_i64, c_f, c_i32, c_p, c_f, c_i32, c_i32, c_p,
                                c_p]
    L.mq_softmax_causal.argtypes = [c_p, c_i64, c_i64, c_f, c_i32, c_f, c_i32, c_i32, c_i64,
                                    c_i64, c_p, c_p]
    L.mq_smooth_scales.argtypes = [c_p, c_i64, c_i64, c_p, c_i64, c_f, c_p, c_p, c_p, c_p]
    L.mq_arl_forward.argtypes = [c_p, c_i64, c_f, c_f, c_i32, c_p, c_p]
    L.mq_arl_backward.argtypes = [c_p, c_p, c_i64, c_f, c_f, c_i32, c_p, c_p, c_p]
    L.mq_qlinear_a16.argtypes = [c_p, c_i64, c_i64, c_i64, c_p, c_i32, c_p, c_p, c_f, c_i32,
                                 c_f, c_i32, c_i32, c_p, c_p, c_i32, c_p]
    L.mq_qlinear_asym.argtypes = [c_p, c_p, c_i64, c_i64, c_i64, c_p, c_i32, c_p, c_p, c_p,
                                  c_f, c_i32, c_f, c_i32, c_i32, c_p, c_p, c_p, c_i64, c_i32,
                                  c_p]
    L.mq_attn_matmul_workspace_bytes.argtypes = [c_i32, c_i32, c_i64, c_i64]
    L.mq_attn_matmul_workspace_bytes.restype = ctypes.c_int64
    L.mq_attn_matmul.argtypes = [c_p, c_i64, c_i64, c_i32, c_p, c_i64, c_i64, c_i32, c_i64, c_i64,
                                 c_i64, c_f, c_i32, c_f, c_i32, c_f, c_i32, c_i32, c_p, c_i64,
                                 c_i64, c_i64, c_i64, c_p, c_i64, c_i32, c_p]
    L.mq_transpose_i8.argtypes = [c_p, c_i64, c_i64, c_i64, c_p, c_p]
    L.mq_probe_read.argtypes = [c_p, c_i64, c_i32, c_i32, c_i32, c_p, c_p]
    L.mq_qlinear_dequant.argtypes = [c_p, c_p, c_i64, c_i64, c_i64, c_p, c_i32, c_p, c_p, c_p,
                                     c_f, c_i32, c_f, c_i32, c_i32, c_p, c_p, c_p, c_p, c_i64,
                                     c_i32, c_p]
    L.mq_qlinear_group.argtypes = [c_p, c_p, c_i64, c_i64, c_i32, c_f, c_i32, c_i32,
                                   ctypes.POINTER(QLinearOut), c_i32, c_i32, c_p]
    for name in ("mq_qlinear_dequant", "mq_qlinear_group", "mq_probe_read", "mq_attn_matmul", "mq_transpose_i8", "mq_act_params", "mq_fold_weights", "mq_fold_acts", "mq_quantize_act",
                 "mq_pack_weights", "mq_qlinear", "mq_qlinear_ex", "mq_qlinear_ws", "mq_dequant",
                 "mq_qlinear_noalloc",
                 "mq_pack_weights_asym", "mq_act_rowsum", "mq_quantize_act_rowsum",
                 "mq_qlinear_asym", "mq_qlinear_a16", "mq_smooth_scales", "mq_arl_forward",
                 "mq_arl_backward", "mq_add_requant", "mq_lut_build", "mq_lut_apply",
                 "mq_rmsnorm", "mq_softmax", "mq_softmax_causal", "mq_mul_requant",
                 "mq_rope", "mq_rope_table", "mq_rope_apply", "mq_lut_mul",
                 "mq_add_rmsnorm"):
        getattr(L, name).restype = ctypes.c_int
    _lib = L
    return L


def _check(status: int, where: str):
    if status != MQ_OK:
        raise MQError(status, where)


# --------------------------------------------------------------------------
# marshalling helpers (torch is only device memory and streams here)
def _torch():
    import torch
    return torch


def _dev_ptr(t, dtype, name, shape=None):
    torch = _torch()
    if t is None:
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    return ctypes.c_void_p(t.data_ptr())


def _stream_ptr(stream):
    torch = _torch()
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _act_dtype(bits):
    torch = _torch()
    if bits == 8:
        return torch.int8
    if bits == 16:
        return torch.int16
    raise ValueError("activation bits must be 8 or 16")


def _bits_of(t):
    torch = _torch()
    return {torch.int8: 8, torch.int16: 16}.get(t.dtype)


# --------------------------------------------------------------------------
def mq_version() -> int:
    return int(lib().mq_version())


def mq_act_params(f_min: float, f_max: float, bits: int):
    """(alpha, zp) of a static per-tensor range (Section 4.2, Eq.(2)-(3))."""
    a = ctypes.c_float()
    z = ctypes.c_int32()
    _check(lib().mq_act_params(float(f_min), float(f_max), int(bits), ctypes.byref(a),
                               ctypes.byref(z)), "mq_act_params")
    return float(a.value), int(z.value)


def mq_fold_weights(w, s, out=None, stream=None):
    """S W of Eq.(1): out[n][k] = w[n][k] * s[k] (fp32, on the GPU)."""
    torch = _torch()
    N, K = w.shape
    out = torch.empty_like(w) if out is None else out
    _check(lib().mq_fold_weights(_dev_ptr(w, torch.float32, "w"),
                                 _dev_ptr(s, torch.float32, "s", (K,)), N, K,
                                 _dev_ptr(out, torch.float32, "out", (N, K)),
                                 _stream_ptr(stream)), "mq_fold_weights")
    return out


def mq_fold_acts(x, s, out=None, stream=None):
    """X S^-1 of Eq.(1): out[m][k] = x[m][k] / s[k] (fp32, on the GPU)."""
    torch = _torch()
    M, K = x.shape
    out = torch.empty_like(x) if out is None else out
    _check(lib().mq_fold_acts(_dev_ptr(x, torch.float32, "x"),
                              _dev_ptr(s, torch.float32, "s", (K,)), M, K,
                              _dev_ptr(out, torch.float32, "out", (M, K)),
                              _stream_ptr(stream)), "mq_fold_acts")
    return out


def mq_quantize_act(x, alpha: float, zp: int, bits: int = 8, out=None, stream=None):
    """Static per-tensor quantizer (Section 4.2, Eq.(4)), signed storage."""
    torch = _torch()
    out = torch.empty(x.shape, dtype=_act_dtype(bits), device=x.device) if out is None else out
    _check(lib().mq_quantize_act(_dev_ptr(x, torch.float32, "x"), x.numel(), float(alpha),
                                 int(zp), int(bits),
                                 _dev_ptr(out, _act_dtype(bits), "out", x.shape),
                                 _stream_ptr(stream)), "mq_quantize_act")
    return out


def mq_pack_weights(w, bits: int = 8, w_q=None, w_scale=None, w_colsum=None, stream=None):
    """Per-output-channel symmetric weight codes, scales and column sums."""
    torch = _torch()
    N, K = w.shape
    dev = w.device
    w_q, wq_dtype, wq_shape = _packed_weights(N, K, bits, dev, w_q)
    w_scale = torch.empty(N, dtype=torch.float32, device=dev) if w_scale is None else w_scale
    w_colsum = torch.empty(N, dtype=torch.int32, device=dev) if w_colsum is None else w_colsum
    _check(lib().mq_pack_weights(_dev_ptr(w, torch.float32, "w"), N, K, int(bits),
                                 _dev_ptr(w_q, wq_dtype, "w_q", wq_shape),
                                 _dev_ptr(w_scale, torch.float32, "w_scale", (N,)),
                                 _dev_ptr(w_colsum, torch.int32, "w_colsum", (N,)),
                                 _stream_ptr(stream)), "mq_pack_weights")
    return w_q, w_scale, w_colsum


def _packed_weights(N, K, bits, dev, w_q):
    torch = _torch()
    if bits == 8:
        w_q = torch.empty((N, K), dtype=torch.int8, device=dev) if w_q is None else w_q
        return w_q, torch.int8, (N, K)
    if bits == 4:
        w_q = torch.empty((N, K // 2), dtype=torch.uint8, device=dev) if w_q is None else w_q
        return w_q, torch.uint8, (N, K // 2)
    raise ValueError("bits must be 8 or 4")


def mq_pack_weights_asym(w, bits: int = 8, per_tensor: bool = False, w_q=None, w_scale=None,
                         w_zp=None, w_colsum=None, stream=None):
    """Asymmetric weight codes, per-row scales, zero-points and code sums
    (Section 5.1); one range per output channel or per tensor."""
    torch = _torch()
    N, K = w.shape
    dev = w.device
    w_q, wq_dtype, wq_shape = _packed_weights(N, K, bits, dev, w_q)
    w_scale = torch.empty(N, dtype=torch.float32, device=dev) if w_scale is None else w_scale
    w_zp = torch.empty(N, dtype=torch.int32, device=dev) if w_zp is None else w_zp
    w_colsum = torch.empty(N, dtype=torch.int32, device=dev) if w_colsum is None else w_colsum
    _check(lib().mq_pack_weights_asym(_dev_ptr(w, torch.float32, "w"), N, K, int(bits),
                                      int(bool(per_tensor)),
                                      _dev_ptr(w_q, wq_dtype, "w_q", wq_shape),
                                      _dev_ptr(w_scale, torch.float32, "w_scale", (N,)),
                                      _dev_ptr(w_zp, torch.int32, "w_zp", (N,)),
                                      _dev_ptr(w_colsum, torch.int32, "w_colsum", (N,)),
                                      _stream_ptr(stream)), "mq_pack_weights_asym")
    return w_q, w_scale, w_zp, w_colsum


def mq_act_rowsum(a_q, out=None, stream=None):
    """sum_k a_q[m][k] as int32 [M]."""
    torch = _torch()
    M, K = a_q.shape
    out = torch.empty(M, dtype=torch.int32, device=a_q.device) if out is None else out
    _check(lib().mq_act_rowsum(_dev_ptr(a_q, torch.int8, "a_q"), M, K,
                               _dev_ptr(out, torch.int32, "out", (M,)), _stream_ptr(stream)),
           "mq_act_rowsum")
    return out


def mq_quantize_act_rowsum(x, alpha: float, zp: int, out=None, rowsum=None, stream=None):
    """8-bit Eq.(4) quantizer on x [M][K] and the row sums of its codes, in
    one pass: returns (x_q, rowsum)."""
    torch = _torch()
    M, K = x.shape
    out = torch.empty((M, K), dtype=torch.int8, device=x.device) if out is None else out
    rowsum = torch.empty(M, dtype=torch.int32, device=x.device) if rowsum is None else rowsum
    _check(lib().mq_quantize_act_rowsum(_dev_ptr(x, torch.float32, "x"), M, K, float(alpha),
                                        int(zp), _dev_ptr(out, torch.int8, "out", (M, K)),
                                        _dev_ptr(rowsum, torch.int32, "rowsum", (M,)),
                                        _stream_ptr(stream)), "mq_quantize_act_rowsum")
    return out, rowsum


def _workspace_args(workspace):
    torch = _torch()
    if workspace is None:
        return None, 0
    if workspace.dtype != torch.uint8 or workspace.device.type != "cuda" or \
            not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous uint8 device tensor")
    return ctypes.c_void_p(workspace.data_ptr()), int(workspace.numel())


def mq_qlinear_asym(a_q, a_rowsum, w_q, w_bits: int, w_scale, w_zp, w_colsum, a_scale: float,
                    a_zp: int, out_scale: float, out_zp: int, out_bits: int = 8, bias=None,
                    out=None, path: int = PATH_AUTO, stream=None, workspace=None):
    """Integer-only linear layer with asymmetric per-channel weights."""
    torch = _torch()
    M, K = a_q.shape
    N = w_q.shape[0]
    wq_dtype, wq_shape = (torch.int8, (N, K)) if w_bits == 8 else (torch.uint8, (N, K // 2))
    out = (torch.empty((M, N), dtype=_act_dtype(out_bits), device=a_q.device)
           if out is None else out)
    bptr = None if bias is None else _dev_ptr(bias, torch.float32, "bias", (N,))
    ws, ws_bytes = _workspace_args(workspace)
    _check(lib().mq_qlinear_asym(
        _dev_ptr(a_q, torch.int8, "a_q"), _dev_ptr(a_rowsum, torch.int32, "a_rowsum", (M,)),
        M, K, N, _dev_ptr(w_q, wq_dtype, "w_q", wq_shape), int(w_bits),
        _dev_ptr(w_scale, torch.float32, "w_scale", (N,)),
        _dev_ptr(w_zp, torch.int32, "w_zp", (N,)),
        _dev_ptr(w_colsum, torch.int32, "w_colsum", (N,)),
        float(a_scale), int(a_zp), float(out_scale), int(out_zp), int(out_bits), bptr,
        _dev_ptr(out, _act_dtype(out_bits), "out", (M, N)), ws, ws_bytes, int(path),
        _stream_ptr(stream)), "mq_qlinear_asym")
    return out


def mq_qlinear_dequant(a_q, w_q, w_bits: int, w_scale, w_colsum, a_scale: float, a_zp: int,
                       out_scale: float, out_zp: int, out_bits: int = 8, bias=None, out=None,
                       codes=None, w_zp=None, a_rowsum=None, path: int = PATH_AUTO,
                       stream=None, workspace=None):
    """Integer-only linear layer whose epilogue writes the dequantized
    outputs (fp32 ``out``, mq_dequant of the codes bit for bit) and the
    codes only into ``codes`` when given."""
    torch = _torch()
    M, K = a_q.shape
    N = w_q.shape[0]
    wq_dtype, wq_shape = (torch.int8, (N, K)) if w_bits == 8 else (torch.uint8, (N, K // 2))
    out = torch.empty((M, N), dtype=torch.float32, device=a_q.device) if out is None else out
    bptr = None if bias is None else _dev_ptr(bias, torch.float32, "bias", (N,))
    cptr = None if codes is None else _dev_ptr(codes, _act_dtype(out_bits), "codes", (M, N))
    zptr = None if w_zp is None else _dev_ptr(w_zp, torch.int32, "w_zp", (N,))
    rptr = None if a_rowsum is None else _dev_ptr(a_rowsum, torch.int32, "a_rowsum", (M,))
    ws, ws_bytes = _workspace_args(workspace)
    _check(lib().mq_qlinear_dequant(
        _dev_ptr(a_q, torch.int8, "a_q"), rptr, M, K, N, _dev_ptr(w_q, wq_dtype, "w_q", wq_shape),
        int(w_bits), _dev_ptr(w_scale, torch.float32, "w_scale", (N,)), zptr,
        _dev_ptr(w_colsum, torch.int32, "w_colsum", (N,)), float(a_scale), int(a_zp),
        float(out_scale), int(out_zp), int(out_bits), bptr, cptr,
        _dev_ptr(out, torch.float32, "out", (M, N)), ws, ws_bytes, int(path),
        _stream_ptr(stream)), "mq_qlinear_dequant")
    return out


def mq_qlinear_group(a_q, linears, w_bits: int, a_scale: float, a_zp: int, out_bits: int = 8,
                     a_rowsum=None, path: int = PATH_AUTO, stream=None):
    """Linears that read one activation input, in one call (one launch on the
    prefill path).  ``linears``: up to MAX_GROUP dicts with w_q, w_scale,
    w_colsum, out_scale, out_zp and optionally w_zp (all or none), bias and
    out.  Returns the outputs, each as mq_qlinear / mq_qlinear_asym would."""
    torch = _torch()
    M, K = a_q.shape
    n = len(linears)
    if n < 1 or n > MAX_GROUP:
        raise MQError(f"mq_qlinear_group: {n} linears (1..{MAX_GROUP})")
    arr = (QLinearOut * n)()
    outs = []
    for i, d in enumerate(linears):
        N = d["w_q"].shape[0]
        wq_dtype, wq_shape = (torch.int8, (N, K)) if w_bits == 8 else (torch.uint8, (N, K // 2))
        out = d.get("out")
        if out is None:
            out = torch.empty((M, N), dtype=_act_dtype(out_bits), device=a_q.device)
        outs.append(out)
        zp, bias = d.get("w_zp"), d.get("bias")
        arr[i] = QLinearOut(
            _dev_ptr(d["w_q"], wq_dtype, "w_q", wq_shape),
            _dev_ptr(d["w_scale"], torch.float32, "w_scale", (N,)),
            None if zp is None else _dev_ptr(zp, torch.int32, "w_zp", (N,)),
            _dev_ptr(d["w_colsum"], torch.int32, "w_colsum", (N,)),
            None if bias is None else _dev_ptr(bias, torch.float32, "bias", (N,)),
            N, float(d["out_scale"]), int(d["out_zp"]),
            _dev_ptr(out, _act_dtype(out_bits), "out", (M, N)))
    rs = None if a_rowsum is None else _dev_ptr(a_rowsum, torch.int32, "a_rowsum", (M,))
    _check(lib().mq_qlinear_group(_dev_ptr(a_q, torch.int8, "a_q"), rs, M, K, int(w_bits),
                                  float(a_scale), int(a_zp), int(out_bits), arr, n, int(path),
                                  _stream_ptr(stream)), "mq_qlinear_group")
    return outs


def mq_add_requant(x1, a1: float, z1: int, x2, a2: float, z2: int, ay: float, zy: int,
                   out_bits: int = 16, out=None, stream=None):
    """Residual add of two int16 code tensors, requantized."""
    torch = _torch()
    out = torch.empty(x1.shape, dtype=_act_dtype(out_bits), device=x1.device) if out is None else out
    _check(lib().mq_add_requant(_dev_ptr(x1, torch.int16, "x1"), float(a1), int(z1),
                                _dev_ptr(x2, torch.int16, "x2", x1.shape), float(a2), int(z2),
                                x1.numel(), float(ay), int(zy), int(out_bits),
                                _dev_ptr(out, _act_dtype(out_bits), "out", x1.shape),
                                _stream_ptr(stream)), "mq_add_requant")
    return out


def mq_lut_build(op: int, ax: float, zx: int, ay: float, zy: int, out_bits: int = 8, lut=None,
                 stream=None):
    """65536-entry table of an elementwise op on int16 codes."""
    torch = _torch()
    lut = torch.empty(65536, dtype=_act_dtype(out_bits), device="cuda") if lut is None else lut
    _check(lib().mq_lut_build(int(op), float(ax), int(zx), float(ay), int(zy), int(out_bits),
                              _dev_ptr(lut, _act_dtype(out_bits), "lut", (65536,)),
                              _stream_ptr(stream)), "mq_lut_build")
    return lut


def mq_lut_apply(x, lut, out=None, stream=None):
    """y = lut[x + 32768] elementwise."""
    torch = _torch()
    bits = _bits_of(lut)
    out = torch.empty(x.shape, dtype=lut.dtype, device=x.device) if out is None else out
    _check(lib().mq_lut_apply(_dev_ptr(x, torch.int16, "x"), x.numel(),
                              _dev_ptr(lut, lut.dtype, "lut", (65536,)), int(bits),
                              _dev_ptr(out, lut.dtype, "out", x.shape), _stream_ptr(stream)),
           "mq_lut_apply")
    return out


def mq_rmsnorm(x, ax: float, zx: int, gamma, eps: float, ay: float, zy: int, out_bits: int = 8,
               out=None, stream=None):
    """RMSNorm over rows of int16 codes, requantized."""
    torch = _torch()
    M, K = x.shape
    out = torch.empty((M, K), dtype=_act_dtype(out_bits), device=x.device) if out is None else out
    gptr = None if gamma is None else _dev_ptr(gamma, torch.float32, "gamma", (K,))
    _check(lib().mq_rmsnorm(_dev_ptr(x, torch.int16, "x"), M, K, float(ax), int(zx), gptr,
                            float(eps), float(ay), int(zy), int(out_bits),
                            _dev_ptr(out, _act_dtype(out_bits), "out", (M, K)),
                            _stream_ptr(stream)), "mq_rmsnorm")
    return out


def mq_softmax(x, ax: float, zx: int, ay: float, zy: int, out_bits: int = 16, out=None,
               stream=None):
    """Softmax over rows of int16 score codes, requantized."""
    torch = _torch()
    M, K = x.shape
    out = torch.empty((M, K), dtype=_act_dtype(out_bits), device=x.device) if out is None else out
    _check(lib().mq_softmax(_dev_ptr(x, torch.int16, "x"), M, K, float(ax), int(zx), float(ay),
                            int(zy), int(out_bits),
                            _dev_ptr(out, _act_dtype(out_bits), "out", (M, K)),
                            _stream_ptr(stream)), "mq_softmax")
    return out


def mq_mul_requant(x1, a1: float, z1: int, x2, a2: float, z2: int, ay: float, zy: int,
                   out_bits: int = 8, out=None, stream=None):
    """Product of two int16 code tensors, requantized."""
    torch = _torch()
    if tuple(x1.shape) != tuple(x2.shape):
        raise ValueError("x1 and x2 must have the same shape")
    out = torch.empty(x1.shape, dtype=_act_dtype(out_bits), device=x1.device) if out is None else out
    _check(lib().mq_mul_requant(_dev_ptr(x1, torch.int16, "x1"), float(a1), int(z1),
                                _dev_ptr(x2, torch.int16, "x2"), float(a2), int(z2), x1.numel(),
                                float(ay), int(zy), int(out_bits),
                                _dev_ptr(out, _act_dtype(out_bits), "out", tuple(x1.shape)),
                                _stream_ptr(stream)), "mq_mul_requant")
    return out


def mq_add_rmsnorm(x1, a1: float, z1: int, x2, a2: float, z2: int, ah: float, zh: int, gamma,
                   eps: float, ay: float, zy: int, out_bits: int = 8, h=None, out=None,
                   stream=None):
    """Residual add (int16 codes h, format ah, zh) and RMSNorm of h in one
    pass; returns (h, y)."""
    torch = _torch()
    M, K = x1.shape
    if tuple(x2.shape) != (M, K):
        raise ValueError("x1 and x2 must have the same shape")
    h = torch.empty((M, K), dtype=torch.int16, device=x1.device) if h is None else h
    out = torch.empty((M, K), dtype=_act_dtype(out_bits), device=x1.device) if out is None else out
    g = None if gamma is None else _dev_ptr(gamma, torch.float32, "gamma", (K,))
    _check(lib().mq_add_rmsnorm(_dev_ptr(x1, torch.int16, "x1"), float(a1), int(z1),
                                _dev_ptr(x2, torch.int16, "x2"), float(a2), int(z2), M, K,
                                float(ah), int(zh), _dev_ptr(h, torch.int16, "h", (M, K)), g,
                                float(eps), float(ay), int(zy), int(out_bits),
                                _dev_ptr(out, _act_dtype(out_bits), "out", (M, K)),
                                _stream_ptr(stream)), "mq_add_rmsnorm")
    return h, out


def mq_lut_mul(x1, lut, a1: float, z1: int, x2, a2: float, z2: int, ay: float, zy: int,
               out_bits: int = 8, out=None, stream=None):
    """lut[x1 + 32768] (format a1, z1) times the codes x2, requantized: the
    gated unit in one pass (mq_lut_apply then mq_mul_requant)."""
    torch = _torch()
    if tuple(x1.shape) != tuple(x2.shape):
        raise ValueError("x1 and x2 must have the same shape")
    bits = _bits_of(lut)
    out = torch.empty(x1.shape, dtype=_act_dtype(out_bits), device=x1.device) if out is None else out
    _check(lib().mq_lut_mul(_dev_ptr(x1, torch.int16, "x1"),
                            _dev_ptr(lut, lut.dtype, "lut", (65536,)), int(bits), float(a1),
                            int(z1), _dev_ptr(x2, torch.int16, "x2"), float(a2), int(z2),
                            x1.numel(), float(ay), int(zy), int(out_bits),
                            _dev_ptr(out, _act_dtype(out_bits), "out", tuple(x1.shape)),
                            _stream_ptr(stream)), "mq_lut_mul")
    return out


def mq_rope_table(T: int, D: int, base: float = 10000.0, pos0: int = 0, out=None, device=None,
                  stream=None):
    """cos/sin table of the rotary angles, fp64 [T * D] (mq_rope's first step)."""
    torch = _torch()
    if out is None:
        out = torch.empty(max(T * D, 1), dtype=torch.float64, device=device or "cuda")
    if out.numel() < T * D:
        raise ValueError("table needs T * D fp64 values")
    _check(lib().mq_rope_table(int(T), int(D), float(base), int(pos0),
                               _dev_ptr(out, torch.float64, "table"), _stream_ptr(stream)),
           "mq_rope_table")
    return out


def mq_rope_apply(x, heads: int, ax: float, zx: int, ay: float, zy: int, table,
                  out_bits: int = 16, out=None, stream=None):
    """Rotary position embedding with a table from mq_rope_table."""
    torch = _torch()
    T, HD = x.shape
    D = HD // int(heads)
    if D * int(heads) != HD:
        raise ValueError("x's row length must be heads * D")
    if table.numel() < T * D:
        raise ValueError("table needs T * D fp64 values")
    out = torch.empty((T, HD), dtype=_act_dtype(out_bits), device=x.device) if out is None else out
    _check(lib().mq_rope_apply(_dev_ptr(x, torch.int16, "x"), T, int(heads), D, float(ax),
                               int(zx), _dev_ptr(table, torch.float64, "table"), float(ay),
                               int(zy), int(out_bits),
                               _dev_ptr(out, _act_dtype(out_bits), "out", (T, HD)),
                               _stream_ptr(stream)), "mq_rope_apply")
    return out


def mq_rope(x, heads: int, ax: float, zx: int, ay: float, zy: int, out_bits: int = 16,
            base: float = 10000.0, pos0: int = 0, out=None, table=None, stream=None):
    """Rotary position embedding on int16 codes [T][heads * D]."""
    torch = _torch()
    T, HD = x.shape
    D = HD // int(heads)
    if D * int(heads) != HD:
        raise ValueError("x's row length must be heads * D")
    out = torch.empty((T, HD), dtype=_act_dtype(out_bits), device=x.device) if out is None else out
    if table is None:
        table = torch.empty(max(T * D, 1), dtype=torch.float64, device=x.device)
    if table.numel() < T * D:
        raise ValueError("table needs T * D fp64 values")
    _check(lib().mq_rope(_dev_ptr(x, torch.int16, "x"), T, int(heads), D, float(ax), int(zx),
                         float(base), int(pos0), float(ay), int(zy), int(out_bits),
                         _dev_ptr(table, torch.float64, "table"),
                         _dev_ptr(out, _act_dtype(out_bits), "out", (T, HD)),
                         _stream_ptr(stream)), "mq_rope")
    return out


def mq_softmax_causal(x, ax: float, zx: int, ay: float, zy: int, period: int, offset: int = 0,
                      out_bits: int = 16, out=None, stream=None):
    """Causal softmax: row m covers keys k <= (m % period) + offset."""
    torch = _torch()
    M, K = x.shape
    out = torch.empty((M, K), dtype=_act_dtype(out_bits), device=x.device) if out is None else out
    _check(lib().mq_softmax_causal(_dev_ptr(x, torch.int16, "x"), M, K, float(ax), int(zx),
                                   float(ay), int(zy), int(out_bits), int(period), int(offset),
                                   _dev_ptr(out, _act_dtype(out_bits), "out", (M, K)),
                                   _stream_ptr(stream)), "mq_softmax_causal")
    return out


def mq_smooth_scales(x, w, a: float, s=None, x_absmax=None, w_absmax=None, stream=None):
    """SmoothQuant's closed-form scales (Section 3.2): (s, x_absmax, w_absmax)."""
    torch = _torch()
    M, K = x.shape
    N, K2 = w.shape
    if K2 != K:
        raise ValueError("x and w must have the same number of columns")
    dev = x.device
    s = torch.empty(K, dtype=torch.float32, device=dev) if s is None else s
    x_absmax = torch.empty(K, dtype=torch.float32, device=dev) if x_absmax is None else x_absmax
    w_absmax = torch.empty(K, dtype=torch.float32, device=dev) if w_absmax is None else w_absmax
    _check(lib().mq_smooth_scales(_dev_ptr(x, torch.float32, "x"), M, K,
                                  _dev_ptr(w, torch.float32, "w"), N, float(a),
                                  _dev_ptr(x_absmax, torch.float32, "x_absmax", (K,)),
                                  _dev_ptr(w_absmax, torch.float32, "w_absmax", (K,)),
                                  _dev_ptr(s, torch.float32, "s", (K,)), _stream_ptr(stream)),
           "mq_smooth_scales")
    return s, x_absmax, w_absmax


def mq_arl_forward(x, alpha: float, beta: float, bits: int, out=None, stream=None):
    """Fake-quantized alpha * (X_int + beta) of Eq.(2)-(4) (training form)."""
    torch = _torch()
    out = torch.empty_like(x) if out is None else out
    _check(lib().mq_arl_forward(_dev_ptr(x, torch.float32, "x"), x.numel(), float(alpha),
                                float(beta), int(bits),
                                _dev_ptr(out, torch.float32, "out", x.shape),
                                _stream_ptr(stream)), "mq_arl_forward")
    return out


def mq_arl_backward(x, g, alpha: float, beta: float, bits: int, gx=None, grads=None,
                    stream=None):
    """Straight-through gradients: (gx, grads) with grads[0] = dL/dalpha and
    grads[1] = dL/dbeta on the device (fp64; the rest is scratch)."""
    torch = _torch()
    gx = torch.empty_like(x) if gx is None else gx
    grads = (torch.empty(2 + 2 * ARL_PARTIALS, dtype=torch.float64, device=x.device)
             if grads is None else grads)
    _check(lib().mq_arl_backward(_dev_ptr(x, torch.float32, "x"),
                                 _dev_ptr(g, torch.float32, "g", x.shape), x.numel(),
                                 float(alpha), float(beta), int(bits),
                                 _dev_ptr(gx, torch.float32, "gx", x.shape),
                                 _dev_ptr(grads, torch.float64, "grads", (2 + 2 * ARL_PARTIALS,)),
                                 _stream_ptr(stream)), "mq_arl_backward")
    return gx, grads


def mq_qlinear_a16(a_q, w_q, w_bits: int, w_scale, w_colsum, a_scale: float, a_zp: int,
                   out_scale: float, out_zp: int, out_bits: int = 8, bias=None, out=None,
                   path: int = PATH_AUTO, stream=None):
    """Integer-only linear layer on 16-bit activation codes (W8A16)."""
    torch = _torch()
    M, K = a_q.shape
    N = w_q.shape[0]
    wq_dtype, wq_shape = (torch.int8, (N, K)) if w_bits == 8 else (torch.uint8, (N, K // 2))
    out = (torch.empty((M, N), dtype=_act_dtype(out_bits), device=a_q.device)
           if out is None else out)
    bptr = None if bias is None else _dev_ptr(bias, torch.float32, "bias", (N,))
    _check(lib().mq_qlinear_a16(
        _dev_ptr(a_q, torch.int16, "a_q"), M, K, N, _dev_ptr(w_q, wq_dtype, "w_q", wq_shape),
        int(w_bits), _dev_ptr(w_scale, torch.float32, "w_scale", (N,)),
        _dev_ptr(w_colsum, torch.int32, "w_colsum", (N,)), float(a_scale), int(a_zp),
        float(out_scale), int(out_zp), int(out_bits), bptr,
        _dev_ptr(out, _act_dtype(out_bits), "out", (M, N)), int(path), _stream_ptr(stream)),
        "mq_qlinear_a16")
    return out


def _strided3(t, dtype, name, shape=None):
    """Pointer and (batch, row) element strides of a [batch][rows][cols] view
    whose last dimension is contiguous."""
    torch = _torch()
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if t.dim() != 3 or (t.shape[2] > 1 and t.stride(2) != 1):
        raise ValueError(f"{name} must be a 3-d view with a contiguous last dimension")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    bs, rs = t.stride(0), t.stride(1)
    if t.shape[1] <= 1:
        rs = max(rs, t.shape[2])
    return ctypes.c_void_p(t.data_ptr()), int(bs), int(rs)


def mq_attn_matmul_workspace_bytes(H: int, G: int, M: int, N: int) -> int:
    n = lib().mq_attn_matmul_workspace_bytes(int(H), int(G), int(M), int(N))
    if n < 0:
        raise ValueError(f"mq_attn_matmul_workspace_bytes: invalid shape {(H, G, M, N)}")
    return n


def mq_attn_matmul(a, b, a_scale: float, a_zp: int, b_scale: float, b_zp: int,
                   out_scale: float, out_zp: int, out_bits: int = 16, out=None, workspace=None,
                   path: int = PATH_AUTO, stream=None, out_causal: int = -1, in_causal: int = -1):
    """Batched attention matmul between 16-bit codes a [H][M][K] and 8-bit
    codes b [G][N][K] (views with a contiguous last dimension; head h uses
    b[h // (H // G)]) -> y [H][M][N].  out_causal >= 0: outputs with
    n > m + out_causal may be left unwritten; in_causal >= 0: promise that
    a[h][m][k] == a_zp for k > m + in_causal."""
    torch = _torch()
    H, M, K = a.shape
    G, N, Kb = b.shape
    if Kb != K:
        raise ValueError("a and b must share K")
    pa, a_hs, lda = _strided3(a, torch.int16, "a")
    pb, b_hs, ldb = _strided3(b, torch.int8, "b")
    if out is None:
        out = torch.empty((H, M, N), dtype=_act_dtype(out_bits), device=a.device)
    py, y_hs, ldy = _strided3(out, _act_dtype(out_bits), "out", (H, M, N))
    if workspace is None:
        workspace = torch.empty(mq_attn_matmul_workspace_bytes(H, G, M, N), dtype=torch.uint8,
                                device=a.device)
    _check(lib().mq_attn_matmul(
        pa, lda, a_hs, int(H), pb, ldb, b_hs, int(G), int(M), int(N), int(K), float(a_scale),
        int(a_zp), float(b_scale), int(b_zp), float(out_scale), int(out_zp), int(out_bits), py,
        ldy, y_hs, int(out_causal), int(in_causal),
        _dev_ptr(workspace, torch.uint8, "workspace"), int(workspace.numel()),
        int(path), _stream_ptr(stream)), "mq_attn_matmul")
    return out


def mq_transpose_i8(x, out=None, stream=None):
    """y[c][r] = x[r][c] for an int8 [rows][cols] view with contiguous rows."""
    torch = _torch()
    rows, cols = x.shape
    if not isinstance(x, torch.Tensor) or not x.is_cuda or x.dtype != torch.int8:
        raise ValueError("x must be an int8 GPU tensor")
    if cols > 1 and x.stride(1) != 1:
        raise ValueError("x must have contiguous rows")
    ldx = max(int(x.stride(0)), cols)
    out = torch.empty((cols, rows), dtype=torch.int8, device=x.device) if out is None else out
    _check(lib().mq_transpose_i8(ctypes.c_void_p(x.data_ptr()), rows, cols, ldx,
                                 _dev_ptr(out, torch.int8, "out", (cols, rows)),
                                 _stream_ptr(stream)), "mq_transpose_i8")
    return out


def mq_qlinear_workspace_bytes(M: int, K: int, N: int, w_bits: int = 8, out_bits: int = 8) -> int:
    """Workspace bytes mq_qlinear can use to split K for this shape (0: none)."""
    n = lib().mq_qlinear_workspace_bytes(int(M), int(K), int(N), int(w_bits), int(out_bits))
    if n < 0:
        raise ValueError(f"mq_qlinear_workspace_bytes: invalid shape {(M, K, N, w_bits, out_bits)}")
    return n


def mq_qlinear(a_q, w_q, w_bits: int, w_scale, w_colsum, a_scale: float, a_zp: int,
               out_scale: float, out_zp: int, out_bits: int = 8, bias=None, out=None,
               path: int = PATH_AUTO, stream=None, workspace=None):
    """Integer-only linear layer: int8 A_q [M][K] x W_q -> Y_q [M][N].

    `workspace`: an optional zero-filled uint8 device tensor of at least
    mq_qlinear_workspace_bytes(...) bytes, kept by the caller across calls
    (the K split leaves it zero-filled again)."""
    torch = _torch()
    M, K = a_q.shape
    N = w_q.shape[0]
    wq_dtype, wq_shape = (torch.int8, (N, K)) if w_bits == 8 else (torch.uint8, (N, K // 2))
    out = (torch.empty((M, N), dtype=_act_dtype(out_bits), device=a_q.device)
           if out is None else out)
    bptr = None if bias is None else _dev_ptr(bias, torch.float32, "bias", (N,))
    args = (_dev_ptr(a_q, torch.int8, "a_q"), M, K, N,
            _dev_ptr(w_q, wq_dtype, "w_q", wq_shape), int(w_bits),
            _dev_ptr(w_scale, torch.float32, "w_scale", (N,)),
            _dev_ptr(w_colsum, torch.int32, "w_colsum", (N,)),
            float(a_scale), int(a_zp), float(out_scale), int(out_zp), int(out_bits), bptr,
            _dev_ptr(out, _act_dtype(out_bits), "out", (M, N)))
    if workspace is not None:
        ws, ws_bytes = _workspace_args(workspace)
        st = lib().mq_qlinear_ws(*args, ws, ws_bytes, int(path), _stream_ptr(stream))
    elif path == PATH_AUTO:
        st = lib().mq_qlinear(*args, _stream_ptr(stream))
    else:
        st = lib().mq_qlinear_ex(*args, int(path), _stream_ptr(stream))
    _check(st, "mq_qlinear")
    return out


def mq_qlinear_noalloc(a_q, w_q, w_bits: int, w_scale, w_colsum, a_scale: float, a_zp: int,
                       out_scale: float, out_zp: int, out_bits: int = 8, bias=None, out=None,
                       stream=None):
    """mq_qlinear whose K split uses the library's static per-GPU array
    instead of any allocation (pass `out` to allocate nothing here either)."""
    torch = _torch()
    M, K = a_q.shape
    N = w_q.shape[0]
    wq_dtype, wq_shape = (torch.int8, (N, K)) if w_bits == 8 else (torch.uint8, (N, K // 2))
    out = (torch.empty((M, N), dtype=_act_dtype(out_bits), device=a_q.device)
           if out is None else out)
    bptr = None if bias is None else _dev_ptr(bias, torch.float32, "bias", (N,))
    _check(lib().mq_qlinear_noalloc(
        _dev_ptr(a_q, torch.int8, "a_q"), M, K, N, _dev_ptr(w_q, wq_dtype, "w_q", wq_shape),
        int(w_bits), _dev_ptr(w_scale, torch.float32, "w_scale", (N,)),
        _dev_ptr(w_colsum, torch.int32, "w_colsum", (N,)), float(a_scale), int(a_zp),
        float(out_scale), int(out_zp), int(out_bits), bptr,
        _dev_ptr(out, _act_dtype(out_bits), "out", (M, N)), _stream_ptr(stream)),
        "mq_qlinear_noalloc")
    return out


def mq_probe_read(buf, blocks: int, waves: int, unroll: int = 8, sink=None, stream=None):
    """Measurement helper: stream every byte of the device tensor `buf`
    through a grid of `blocks` x `waves` wavefronts (the read floor of a
    kernel with that grid); returns the int32 sink [blocks * waves]."""
    torch = _torch()
    if not buf.is_cuda or not buf.is_contiguous():
        raise ValueError("buf must be a contiguous GPU tensor")
    sink = (torch.empty(blocks * waves, dtype=torch.int32, device=buf.device)
            if sink is None else sink)
    _check(lib().mq_probe_read(ctypes.c_void_p(buf.data_ptr()),
                               buf.numel() * buf.element_size(), int(blocks), int(waves),
                               int(unroll), _dev_ptr(sink, torch.int32, "sink",
                                                     (blocks * waves,)),
                               _stream_ptr(stream)), "mq_probe_read")
    return sink


def mq_dequant(q, alpha: float, zp: int, out=None, stream=None):
    """alpha * (q - zp) in fp32 (inverse of Eq.(4))."""
    torch = _torch()
    bits = _bits_of(q)
    if bits is None:
        raise ValueError("q must be int8 or int16")
    out = torch.empty(q.shape, dtype=torch.float32, device=q.device) if out is None else out
    _check(lib().mq_dequant(_dev_ptr(q, q.dtype, "q"), bits, q.numel(), float(alpha), int(zp),
                            _dev_ptr(out, torch.float32, "out", q.shape), _stream_ptr(stream)),
           "mq_dequant")
    return out
