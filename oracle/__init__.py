"""CPU oracle of MobileQuant's integer-only quantized linear layer.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU
baseline leg of the benchmark may import this package; the product path
never does.  It shares no code with the HIP library: the arithmetic lives
in ``mq_oracle.c`` (plain C loops, int64 accumulation, IEEE fp32/fp64) and
this module only marshals numpy arrays into it.

Functions and the passages they follow (arXiv 2408.13933):

* ``act_params``      -- Section 4.2, Eq.(2)-(3) (alpha, beta from a range)
* ``quantize_act``    -- Section 4.2, Eq.(4) (static per-tensor quantizer)
* ``dequant``         -- inverse of Eq.(4)
* ``fold_weights`` / ``fold_acts`` -- Section 3.2, Eq.(1) (S W and X S^-1)
* ``smooth_scales``   -- Section 3.2: SmoothQuant's closed-form S
* ``add_requant``, ``lut_build``, ``rmsnorm``, ``softmax`` -- decoder-block
  glue on 16-bit integer activations (Section 4.1, Section 5.1)
* ``arl_forward`` / ``arl_backward`` -- Section 4.2, Eq.(2)-(4) in its
  training form (learnable alpha, beta; straight-through rounding)
* ``pack_weights``    -- Section 5.1 / appendix: symmetric per-channel W8, W4
* ``pack_weights_asym`` -- Section 5.1: asymmetric W8, W4 (the quantizer of
  Eq.(2)-(4) over each output row's range, or the whole matrix's)
* ``act_rowsum``      -- sum_k A_q[m][k] (the zero-point cross term)
* ``requant_params`` / ``requant_value`` -- fixed-point rescale to the next
  layer's integer format (Section 1, Section 3.1: integer-only arithmetic)
* ``qlinear``         -- the integer-only linear layer end to end, with
  optional per-channel weight zero-points
* ``int_matmul``      -- the raw integer product, for pinning the accumulate

Parity status: every function is pinned by ``tests/test_oracle_pins.py``
(closed forms, invariants, library routines, exact rational brute force).
Nothing here is pinned to a printed number of the paper: the paper prints
no worked numeric example of its quantizer or of a linear layer.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libmq_oracle.so")
_lib = None

_f32p = np.ctypeslib.ndpointer(dtype=np.float32, flags="C_CONTIGUOUS")
_i32p = np.ctypeslib.ndpointer(dtype=np.int32, flags="C_CONTIGUOUS")
_i64p = np.ctypeslib.ndpointer(dtype=np.int64, flags="C_CONTIGUOUS")
_i8p = np.ctypeslib.ndpointer(dtype=np.int8, flags="C_CONTIGUOUS")
_vp = ctypes.c_void_p


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _b
        _b.build()
    lib = ctypes.CDLL(_LIB_PATH)
    lib.oracle_act_params.argtypes = [ctypes.c_float, ctypes.c_float, ctypes.c_int,
                                      ctypes.POINTER(ctypes.c_float),
                                      ctypes.POINTER(ctypes.c_int32)]
    lib.oracle_act_params.restype = ctypes.c_int
    lib.oracle_quantize_act.argtypes = [_f32p, ctypes.c_int64, ctypes.c_float,
                                        ctypes.c_int32, ctypes.c_int, _vp]
    lib.oracle_quantize_act.restype = None
    lib.oracle_dequant.argtypes = [_vp, ctypes.c_int, ctypes.c_int64, ctypes.c_float,
                                   ctypes.c_int32, _f32p]
    lib.oracle_dequant.restype = None
    lib.oracle_fold_weights.argtypes = [_f32p, _f32p, ctypes.c_int64, ctypes.c_int64, _f32p]
    lib.oracle_fold_weights.restype = None
    lib.oracle_fold_acts.argtypes = [_f32p, _f32p, ctypes.c_int64, ctypes.c_int64, _f32p]
    lib.oracle_fold_acts.restype = None
    _i16p = np.ctypeslib.ndpointer(dtype=np.int16, flags="C_CONTIGUOUS")
    lib.oracle_add_requant.argtypes = [_i16p, ctypes.c_float, ctypes.c_int32, _i16p,
                                       ctypes.c_float, ctypes.c_int32, ctypes.c_int64,
                                       ctypes.c_float, ctypes.c_int32, ctypes.c_int, _vp]
    lib.oracle_add_requant.restype = None
    lib.oracle_lut_build.argtypes = [ctypes.c_int, ctypes.c_float, ctypes.c_int32,
                                     ctypes.c_float, ctypes.c_int32, ctypes.c_int, _vp]
    lib.oracle_lut_build.restype = None
    lib.oracle_rmsnorm.argtypes = [_i16p, ctypes.c_int64, ctypes.c_int64, ctypes.c_float,
                                   ctypes.c_int32, _vp, ctypes.c_float, ctypes.c_float,
                                   ctypes.c_int32, ctypes.c_int, _vp]
    lib.oracle_rmsnorm.restype = None
    lib.oracle_softmax.argtypes = [_i16p, ctypes.c_int64, ctypes.c_int64, ctypes.c_float,
                                   ctypes.c_int32, ctypes.c_float, ctypes.c_int32, ctypes.c_int,
                                   _vp]
    lib.oracle_softmax.restype = None
    lib.oracle_softmax_causal.argtypes = [_i16p, ctypes.c_int64, ctypes.c_int64, ctypes.c_float,
                                          ctypes.c_int32, ctypes.c_float, ctypes.c_int32,
                                          ctypes.c_int, ctypes.c_int64, ctypes.c_int64,
                                          ctypes.c_void_p]
    lib.oracle_softmax_causal.restype = None
    lib.oracle_mul_requant.argtypes = [_i16p, ctypes.c_float, ctypes.c_int32, _i16p, ctypes.c_float,
                                       ctypes.c_int32, ctypes.c_int64, ctypes.c_float,
                                       ctypes.c_int32, ctypes.c_int, ctypes.c_void_p]
    lib.oracle_mul_requant.restype = None
    lib.oracle_rope.argtypes = [_i16p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                                ctypes.c_float, ctypes.c_int32, ctypes.c_double, ctypes.c_int64,
                                ctypes.c_float, ctypes.c_int32, ctypes.c_int, ctypes.c_void_p]
    lib.oracle_rope.restype = None
    lib.oracle_smooth_scales.argtypes = [_f32p, ctypes.c_int64, ctypes.c_int64, _f32p,
                                         ctypes.c_int64, ctypes.c_float, _f32p, _f32p, _f32p]
    lib.oracle_smooth_scales.restype = None
    lib.oracle_arl_forward.argtypes = [_f32p, ctypes.c_int64, ctypes.c_float, ctypes.c_float,
                                       ctypes.c_int, _f32p]
    lib.oracle_arl_forward.restype = None
    lib.oracle_arl_backward.argtypes = [_f32p, _f32p, ctypes.c_int64, ctypes.c_float,
                                        ctypes.c_float, ctypes.c_int, _f32p,
                                        ctypes.POINTER(ctypes.c_double),
                                        ctypes.POINTER(ctypes.c_double)]
    lib.oracle_arl_backward.restype = None
    lib.oracle_pack_weights.argtypes = [_f32p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int,
                                        _vp, _f32p, _i32p]
    lib.oracle_pack_weights.restype = None
    lib.oracle_pack_weights_asym.argtypes = [_f32p, ctypes.c_int64, ctypes.c_int64,
                                             ctypes.c_int, ctypes.c_int, _vp, _f32p, _i32p,
                                             _i32p]
    lib.oracle_pack_weights_asym.restype = None
    lib.oracle_act_rowsum.argtypes = [_i8p, ctypes.c_int64, ctypes.c_int64, _i32p]
    lib.oracle_act_rowsum.restype = None
    lib.oracle_requant_params.argtypes = [ctypes.c_float, ctypes.c_float, ctypes.c_float,
                                          ctypes.POINTER(ctypes.c_float),
                                          ctypes.POINTER(ctypes.c_int64),
                                          ctypes.POINTER(ctypes.c_int32),
                                          ctypes.POINTER(ctypes.c_int64)]
    lib.oracle_requant_params.restype = None
    lib.oracle_requant_value.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                                         ctypes.c_int32, ctypes.c_int]
    lib.oracle_requant_value.restype = ctypes.c_int64
    lib.oracle_requant_round.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int32]
    lib.oracle_requant_round.restype = ctypes.c_int64
    lib.oracle_qlinear.argtypes = [_i8p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                                   _vp, ctypes.c_int, _f32p, ctypes.c_float, ctypes.c_int32,
                                   ctypes.c_float, ctypes.c_int32, ctypes.c_int, _vp, _vp,
                                   ctypes.c_int]
    lib.oracle_qlinear.restype = None
    lib.oracle_qlinear_asym.argtypes = [_i8p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                                        _vp, ctypes.c_int, _f32p, _vp, ctypes.c_float,
                                        ctypes.c_int32, ctypes.c_float, ctypes.c_int32,
                                        ctypes.c_int, _vp, _vp, ctypes.c_int]
    lib.oracle_qlinear_asym.restype = None
    lib.oracle_qlinear_gen.argtypes = [_vp, ctypes.c_int, ctypes.c_int64, ctypes.c_int64,
                                       ctypes.c_int64, _vp, ctypes.c_int, _f32p, _vp,
                                       ctypes.c_float, ctypes.c_int32, ctypes.c_float,
                                       ctypes.c_int32, ctypes.c_int, _vp, _vp, ctypes.c_int]
    lib.oracle_qlinear_gen.restype = None
    lib.oracle_int_matmul.argtypes = [_i8p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                                      _vp, ctypes.c_int, _i64p]
    lib.oracle_int_matmul.restype = None
    _lib = lib
    return lib


def _act_dtype(bits: int):
    if bits == 8:
        return np.int8
    if bits == 16:
        return np.int16
    raise ValueError(f"activation bits must be 8 or 16, got {bits}")


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def default_threads() -> int:
    return max(1, len(os.sched_getaffinity(0)))


# --------------------------------------------------------------------------
def act_params(f_min: float, f_max: float, bits: int):
    """(alpha, zp) for a static per-tensor range, Section 4.2 Eq.(2)-(3)."""
    a = ctypes.c_float()
    z = ctypes.c_int32()
    rc = _load().oracle_act_params(float(f_min), float(f_max), int(bits),
                                   ctypes.byref(a), ctypes.byref(z))
    if rc != 0:
        raise ValueError("invalid activation range")
    return float(a.value), int(z.value)


def quantize_act(x: np.ndarray, alpha: float, zp: int, bits: int) -> np.ndarray:
    """Static per-tensor quantizer, Section 4.2 Eq.(4), signed storage."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    q = np.empty(x.shape, dtype=_act_dtype(bits))
    _load().oracle_quantize_act(x.reshape(-1), x.size, alpha, zp, bits, _ptr(q))
    return q


def dequant(q: np.ndarray, alpha: float, zp: int) -> np.ndarray:
    """alpha * (q - zp) in fp32 (inverse of Eq.(4))."""
    q = np.ascontiguousarray(q)
    bits = {np.dtype(np.int8): 8, np.dtype(np.int16): 16}[q.dtype]
    y = np.empty(q.shape, dtype=np.float32)
    _load().oracle_dequant(_ptr(q), bits, q.size, alpha, zp, y.reshape(-1))
    return y


def fold_weights(w: np.ndarray, s: np.ndarray) -> np.ndarray:
    """S W of Eq.(1): W_hat[n][k] = W[n][k] * s[k]."""
    w = np.ascontiguousarray(w, dtype=np.float32)
    s = np.ascontiguousarray(s, dtype=np.float32)
    N, K = w.shape
    assert s.shape == (K,)
    out = np.empty_like(w)
    _load().oracle_fold_weights(w, s, N, K, out)
    return out


def fold_acts(x: np.ndarray, s: np.ndarray) -> np.ndarray:
    """X S^-1 of Eq.(1): X_hat[m][k] = X[m][k] / s[k]."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    s = np.ascontiguousarray(s, dtype=np.float32)
    M, K = x.shape
    assert s.shape == (K,)
    out = np.empty_like(x)
    _load().oracle_fold_acts(x, s, M, K, out)
    return out


def pack_weights(w: np.ndarray, bits: int):
    """Symmetric per-output-channel quantizer and packer.

    Returns (w_q, w_scale, colsum); w_q is int8 [N][K] for bits=8 and
    uint8 [N][K/2] (low nibble = even k) for bits=4.
    """
    w = np.ascontiguousarray(w, dtype=np.float32)
    N, K = w.shape
    if bits == 8:
        wq = np.empty((N, K), dtype=np.int8)
    elif bits == 4:
        if K % 2:
            raise ValueError("int4 packing needs an even K")
        wq = np.empty((N, K // 2), dtype=np.uint8)
    else:
        raise ValueError("bits must be 8 or 4")
    scale = np.empty(N, dtype=np.float32)
    colsum = np.empty(N, dtype=np.int32)
    _load().oracle_pack_weights(w, N, K, bits, _ptr(wq), scale, colsum)
    return wq, scale, colsum


LUT_SILU = 1


def add_requant(x1, a1, z1, x2, a2, z2, ay, zy, bits_y):
    """Residual add of two int16 code tensors, requantized."""
    x1 = np.ascontiguousarray(x1, dtype=np.int16)
    x2 = np.ascontiguousarray(x2, dtype=np.int16)
    assert x1.shape == x2.shape
    y = np.empty(x1.shape, dtype=_act_dtype(bits_y))
    _load().oracle_add_requant(x1.reshape(-1), a1, z1, x2.reshape(-1), a2, z2, x1.size, ay, zy,
                               bits_y, _ptr(y))
    return y


def mul_requant(x1, a1, z1, x2, a2, z2, ay, zy, bits_y):
    """Elementwise product of two int16 code tensors, requantized."""
    x1 = np.ascontiguousarray(x1, dtype=np.int16)
    x2 = np.ascontiguousarray(x2, dtype=np.int16)
    assert x1.shape == x2.shape
    y = np.empty(x1.shape, dtype=_act_dtype(bits_y))
    _load().oracle_mul_requant(x1, a1, z1, x2, a2, z2, x1.size, ay, zy, bits_y, _ptr(y))
    return y


def rope(x, heads, ax, zx, ay, zy, bits_y, base=10000.0, pos0=0):
    """Rotary position embedding on int16 codes [T][heads * D], pairs
    (i, i + D/2) of every head, requantized."""
    x = np.ascontiguousarray(x, dtype=np.int16)
    T, HD = x.shape
    D = HD // heads
    assert D * heads == HD and D % 2 == 0
    y = np.empty(x.shape, dtype=_act_dtype(bits_y))
    _load().oracle_rope(x, T, heads, D, ax, zx, float(base), int(pos0), ay, zy, bits_y, _ptr(y))
    return y


def lut_build(op, ax, zx, ay, zy, bits_y):
    """65536-entry table of a non-linear op on int16 codes (entry i + 32768)."""
    lut = np.empty(65536, dtype=_act_dtype(bits_y))
    _load().oracle_lut_build(int(op), ax, zx, ay, zy, bits_y, _ptr(lut))
    return lut


def rmsnorm(x, ax, zx, gamma, eps, ay, zy, bits_y):
    """RMSNorm over rows of int16 codes, requantized."""
    x = np.ascontiguousarray(x, dtype=np.int16)
    M, K = x.shape
    g = None
    if gamma is not None:
        gamma = np.ascontiguousarray(gamma, dtype=np.float32)
        g = _ptr(gamma)
    y = np.empty((M, K), dtype=_act_dtype(bits_y))
    _load().oracle_rmsnorm(x, M, K, ax, zx, g, eps, ay, zy, bits_y, _ptr(y))
    return y


def softmax(x, ax, zx, ay, zy, bits_y, causal_period: int = 0, causal_offset: int = 0):
    """Softmax over rows of int16 score codes, requantized.  causal_period
    > 0: row m sees only keys k <= (m mod causal_period) + causal_offset
    (the others get probability 0)."""
    x = np.ascontiguousarray(x, dtype=np.int16)
    M, K = x.shape
    y = np.empty((M, K), dtype=_act_dtype(bits_y))
    _load().oracle_softmax_causal(x, M, K, ax, zx, ay, zy, bits_y, int(causal_period),
                                  int(causal_offset), _ptr(y))
    return y


def smooth_scales(x: np.ndarray, w: np.ndarray, a: float):
    """SmoothQuant's s_k = max|X_k|^a / max|W_k|^(1-a): (s, x_absmax, w_absmax)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    w = np.ascontiguousarray(w, dtype=np.float32)
    M, K = x.shape
    N, K2 = w.shape
    assert K == K2
    s = np.empty(K, np.float32)
    mx = np.empty(K, np.float32)
    mw = np.empty(K, np.float32)
    _load().oracle_smooth_scales(x, M, K, w, N, float(a), mx, mw, s)
    return s, mx, mw


def arl_forward(x: np.ndarray, alpha: float, beta: float, bits: int) -> np.ndarray:
    """Fake-quantized X_hat = alpha (X_int + beta) of Eq.(2)-(4)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    y = np.empty_like(x)
    _load().oracle_arl_forward(x.reshape(-1), x.size, float(alpha), float(beta), int(bits),
                               y.reshape(-1))
    return y


def arl_backward(x: np.ndarray, g: np.ndarray, alpha: float, beta: float, bits: int):
    """Straight-through gradients: (dL/dX, dL/dalpha, dL/dbeta)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    g = np.ascontiguousarray(g, dtype=np.float32)
    assert g.shape == x.shape
    gx = np.empty_like(x)
    ga, gb = ctypes.c_double(), ctypes.c_double()
    _load().oracle_arl_backward(x.reshape(-1), g.reshape(-1), x.size, float(alpha), float(beta),
                                int(bits), gx.reshape(-1), ctypes.byref(ga), ctypes.byref(gb))
    return gx, float(ga.value), float(gb.value)


def _packed_weight_buffer(N: int, K: int, bits: int) -> np.ndarray:
    if bits == 8:
        return np.empty((N, K), dtype=np.int8)
    if bits == 4:
        if K % 2:
            raise ValueError("int4 packing needs an even K")
        return np.empty((N, K // 2), dtype=np.uint8)
    raise ValueError("bits must be 8 or 4")


def pack_weights_asym(w: np.ndarray, bits: int, per_tensor: bool = False):
    """Asymmetric weight quantizer and packer (Section 5.1), one range per
    output channel or (per_tensor) one for the whole matrix.

    Returns (w_q, w_scale, w_zp, colsum), all per output row; codes are
    signed (the unsigned Eq.(4) code minus 2^(bits-1)), w_zp is the signed
    zero-point, colsum the row sum of the stored codes.
    """
    w = np.ascontiguousarray(w, dtype=np.float32)
    N, K = w.shape
    wq = _packed_weight_buffer(N, K, bits)
    scale = np.empty(N, dtype=np.float32)
    zp = np.empty(N, dtype=np.int32)
    colsum = np.empty(N, dtype=np.int32)
    _load().oracle_pack_weights_asym(w, N, K, bits, int(bool(per_tensor)), _ptr(wq), scale, zp,
                                     colsum)
    return wq, scale, zp, colsum


def act_rowsum(a_q: np.ndarray) -> np.ndarray:
    """sum_k A_q[m][k] as int32 [M]."""
    a_q = np.ascontiguousarray(a_q, dtype=np.int8)
    M, K = a_q.shape
    out = np.empty(M, dtype=np.int32)
    _load().oracle_act_rowsum(a_q, M, K, out)
    return out


def requant_params(alpha_a: float, w_scale: float, alpha_y: float, bias=None):
    """(M0, sh, bias_q) for one output channel."""
    M0 = ctypes.c_int64()
    sh = ctypes.c_int32()
    bq = ctypes.c_int64()
    b = None if bias is None else ctypes.byref(ctypes.c_float(float(bias)))
    _load().oracle_requant_params(alpha_a, w_scale, alpha_y, b, ctypes.byref(M0),
                                  ctypes.byref(sh), ctypes.byref(bq))
    return int(M0.value), int(sh.value), int(bq.value)


def requant_round(c: int, M0: int, sh: int) -> int:
    """r = floor((c*M0 + 2^(sh-1)) / 2^sh) for one corrected accumulator."""
    return int(_load().oracle_requant_round(int(c), int(M0), int(sh)))


def requant_value(c: int, M0: int, sh: int, zp_y: int, bits_y: int) -> int:
    """Requantize one corrected int32 accumulator value."""
    return int(_load().oracle_requant_value(int(c), int(M0), int(sh), int(zp_y), int(bits_y)))


def qlinear(a_q: np.ndarray, w_q: np.ndarray, bits: int, w_scale: np.ndarray,
            alpha_a: float, zp_a: int, alpha_y: float, zp_y: int, bits_y: int,
            bias=None, nthreads: int | None = None, w_zp=None) -> np.ndarray:
    """Integer-only linear layer: Y_q[m][n] from A_q[M][K] and W_q.

    ``a_q`` is int8, or int16 for 16-bit activations (W8A16).  ``w_zp``
    (int32 [N]) gives per-channel weight zero-points; None means symmetric
    weights.
    """
    a_q = np.ascontiguousarray(a_q)
    if a_q.dtype not in (np.int8, np.int16):
        raise ValueError("a_q must be int8 or int16")
    a_bits = 8 if a_q.dtype == np.int8 else 16
    M, K = a_q.shape
    w_q = np.ascontiguousarray(w_q)
    N = w_q.shape[0]
    if bits == 8:
        assert w_q.dtype == np.int8 and w_q.shape == (N, K)
    elif bits == 4:
        assert w_q.dtype == np.uint8 and w_q.shape == (N, K // 2) and K % 2 == 0
    else:
        raise ValueError("bits must be 8 or 4")
    w_scale = np.ascontiguousarray(w_scale, dtype=np.float32)
    assert w_scale.shape == (N,)
    bptr = None
    if bias is not None:
        bias = np.ascontiguousarray(bias, dtype=np.float32)
        assert bias.shape == (N,)
        bptr = _ptr(bias)
    zptr = None
    if w_zp is not None:
        w_zp = np.ascontiguousarray(w_zp, dtype=np.int32)
        assert w_zp.shape == (N,)
        zptr = _ptr(w_zp)
    y = np.empty((M, N), dtype=_act_dtype(bits_y))
    if M == 0 or N == 0:
        return y
    _load().oracle_qlinear_gen(_ptr(a_q), a_bits, M, K, N, _ptr(w_q), bits, w_scale, zptr,
                               alpha_a, zp_a, alpha_y, zp_y, bits_y, bptr, _ptr(y),
                               nthreads or default_threads())
    return y


def attn_matmul(a: np.ndarray, b: np.ndarray, a_scale: float, a_zp: int, b_scale: float,
                b_zp: int, out_scale: float, out_zp: int, bits_y: int,
                nthreads: int | None = None) -> np.ndarray:
    """Batched matmul of self-attention between 16-bit and 8-bit activation
    codes (Section 5.6: the W8A16 setting multiplies 8-bit by 16-bit
    activations in the attention products), both per-tensor quantized
    (Eq.(2)-(4)) with their own zero-points.  For head h, with the G groups
    of b shared by H / G consecutive heads:
        Y[h] = requant( (A[h] - a_zp) (B[h // (H / G)] - b_zp)^T )
    with the rescale a_scale * b_scale / out_scale and no bias: the integer
    linear layer of `qlinear`, with b as per-tensor asymmetric "weights".
    a: int16 [H][M][K], b: int8 [G][N][K] -> [H][M][N]."""
    a = np.asarray(a)
    b = np.asarray(b)
    assert a.dtype == np.int16 and b.dtype == np.int8 and a.ndim == 3 and b.ndim == 3
    H, M, K = a.shape
    G, N, Kb = b.shape
    assert Kb == K and G >= 1 and H % G == 0
    y = np.empty((H, M, N), dtype=_act_dtype(bits_y))
    w_scale = np.full(N, b_scale, dtype=np.float32)
    w_zp = np.full(N, b_zp, dtype=np.int32)
    for h in range(H):
        y[h] = qlinear(a[h], b[h // (H // G)], 8, w_scale, a_scale, a_zp, out_scale, out_zp,
                       bits_y, nthreads=nthreads, w_zp=w_zp)
    return y


def int_matmul(a_q: np.ndarray, w_q: np.ndarray, bits: int) -> np.ndarray:
    """sum_k A_q[m][k] * W_q[n][k], exact, int64 [M][N]."""
    a_q = np.ascontiguousarray(a_q, dtype=np.int8)
    M, K = a_q.shape
    w_q = np.ascontiguousarray(w_q)
    N = w_q.shape[0]
    acc = np.empty((M, N), dtype=np.int64)
    _load().oracle_int_matmul(a_q, M, K, N, _ptr(w_q), bits, acc)
    return acc
