"""CPU-side checks of the C ABI: the library loads, exports every entry point
declared in include/mq.h, and rejects invalid arguments before touching a
device.  The Eq.(2)-(3) host arithmetic is compared with the oracle here too.
"""
import ctypes
import math
import os
import re

import numpy as np
import pytest

import oracle
import paper_2408_13933_amd as mq

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mq.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(mq_[a-z0-9_]+)\s*\(", src)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("mq_quantize_act", "mq_pack_weights", "mq_qlinear", "mq_dequant",
                     "mq_act_params", "mq_fold_weights", "mq_fold_acts"):
        assert required in names


def test_library_exports_every_declared_symbol():
    L = mq.lib()
    for name in declared_functions():
        assert hasattr(L, name), f"{name} declared in mq.h but not exported"


def test_status_strings_and_version():
    L = mq.lib()
    assert L.mq_status_string(0) == b"MQ_OK"
    for s in (1, 2, 3):
        assert L.mq_status_string(s).startswith(b"MQ_ERR_")
    assert mq.mq_version() == 1


P = ctypes.c_void_p
NZ = P(16)  # never dereferenced: every call below fails validation first


def qlin(**kw):
    a = dict(a_q=NZ, M=4, K=64, N=8, w_q=NZ, w_bits=8, w_scale=NZ, w_colsum=NZ, a_scale=0.1,
             a_zp=0, out_scale=0.1, out_zp=0, out_bits=8, bias=None, y_q=NZ, path=0,
             stream=None)
    a.update(kw)
    return mq.lib().mq_qlinear_ex(a["a_q"], a["M"], a["K"], a["N"], a["w_q"], a["w_bits"],
                                  a["w_scale"], a["w_colsum"], a["a_scale"], a["a_zp"],
                                  a["out_scale"], a["out_zp"], a["out_bits"], a["bias"],
                                  a["y_q"], a["path"], a["stream"])


@pytest.mark.parametrize("kw", [
    dict(a_q=None), dict(w_q=None), dict(w_scale=None), dict(w_colsum=None), dict(y_q=None),
    dict(M=-1), dict(N=-1), dict(K=0), dict(K=-5), dict(K=65537),
    dict(w_bits=2), dict(w_bits=16), dict(w_bits=4, K=63), dict(out_bits=4), dict(out_bits=32),
    dict(a_scale=0.0), dict(a_scale=-1.0), dict(a_scale=float("nan")), dict(a_scale=float("inf")),
    dict(out_scale=0.0), dict(out_scale=float("nan")),
    dict(a_zp=128), dict(a_zp=-129), dict(out_zp=128), dict(out_bits=16, out_zp=40000),
    dict(path=7), dict(path=-1), dict(path=1, M=17), dict(path=15), dict(path=16 + mq.PREFILL_TILES),
    dict(path=16, a_q=None),
])
def test_qlinear_rejects_invalid_arguments(kw):
    assert qlin(**kw) == 1


def qlin_group(parts=None, n=None, **kw):
    """mq_qlinear_group with fake pointers; ``parts``: per-linear overrides."""
    a = dict(a_q=NZ, a_rowsum=None, M=4, K=64, w_bits=8, a_scale=0.1, a_zp=0, out_bits=8,
             path=0, stream=None)
    a.update(kw)
    parts = [{}, {}] if parts is None else parts
    arr = (mq.QLinearOut * max(1, len(parts)))()
    for i, over in enumerate(parts):
        d = dict(w_q=NZ, w_scale=NZ, w_zp=None, w_colsum=NZ, bias=None, N=8, out_scale=0.1,
                 out_zp=0, y_q=NZ)
        d.update(over)
        arr[i] = mq.QLinearOut(d["w_q"], d["w_scale"], d["w_zp"], d["w_colsum"], d["bias"],
                               d["N"], d["out_scale"], d["out_zp"], d["y_q"])
    return mq.lib().mq_qlinear_group(a["a_q"], a["a_rowsum"], a["M"], a["K"], a["w_bits"],
                                     a["a_scale"], a["a_zp"], a["out_bits"],
                                     arr if parts else None, len(parts) if n is None else n,
                                     a["path"], a["stream"])


def test_qlinear_out_layout():
    # the C struct: five pointers, int64 N, float, int32, pointer (64 bytes)
    assert ctypes.sizeof(mq.QLinearOut) == 64
    assert mq.QLinearOut.N.offset == 40 and mq.QLinearOut.y_q.offset == 56
    text = open(HEADER).read()
    assert re.search(r"#define MQ_MAX_GROUP (\d+)", text).group(1) == str(mq.MAX_GROUP)


@pytest.mark.parametrize("case", [
    dict(parts=[]), dict(n=0), dict(n=-1), dict(parts=[{}] * 5),
    dict(parts=[{}, {"w_zp": NZ}]),                              # asymmetric mixed with symmetric
    dict(parts=[{"w_zp": NZ}, {"w_zp": NZ}]),                    # asymmetric without row sums
    dict(parts=[{}, {}], a_rowsum=NZ),                            # row sums without zero-points
    dict(parts=[{}, {"out_scale": 0.0}]), dict(parts=[{"y_q": None}, {}]),
    dict(parts=[{}, {"N": -1}]), dict(parts=[{}, {"out_zp": 200}]),
    dict(K=0), dict(M=-1), dict(w_bits=2), dict(out_bits=4), dict(a_scale=float("nan")),
    dict(path=1, M=17), dict(path=16 + mq.PREFILL_TILES), dict(a_q=None),
], ids=str)
def test_qlinear_group_rejects_invalid_arguments(case):
    assert qlin_group(**case) == 1


def test_qlinear_group_nothing_to_do():
    # no linear with work: nothing enqueued, no device touched
    assert qlin_group(M=0) == 0
    assert qlin_group(parts=[{"N": 0}, {"N": 0}]) == 0
    assert qlin_group(parts=[{"N": 0}], M=0, a_q=None) == 0


def qlin_deq(**kw):
    a = dict(a_q=NZ, a_rowsum=None, M=4, K=64, N=8, w_q=NZ, w_bits=8, w_scale=NZ, w_zp=None,
             w_colsum=NZ, a_scale=0.1, a_zp=0, out_scale=0.1, out_zp=0, out_bits=8, bias=None,
             y_q=None, y=NZ, ws=None, ws_bytes=0, path=0, stream=None)
    a.update(kw)
    return mq.lib().mq_qlinear_dequant(a["a_q"], a["a_rowsum"], a["M"], a["K"], a["N"],
                                       a["w_q"], a["w_bits"], a["w_scale"], a["w_zp"],
                                       a["w_colsum"], a["a_scale"], a["a_zp"], a["out_scale"],
                                       a["out_zp"], a["out_bits"], a["bias"], a["y_q"], a["y"],
                                       a["ws"], a["ws_bytes"], a["path"], a["stream"])


@pytest.mark.parametrize("kw", [
    dict(y=None), dict(y=None, y_q=NZ), dict(a_q=None), dict(w_q=None), dict(K=0),
    dict(w_bits=2), dict(out_bits=4), dict(out_scale=0.0), dict(a_zp=128),
    dict(w_zp=NZ), dict(a_rowsum=NZ), dict(path=7), dict(path=16 + mq.PREFILL_TILES),
    dict(ws=P(256 + 16), ws_bytes=4096),
], ids=str)
def test_qlinear_dequant_rejects_invalid_arguments(kw):
    assert qlin_deq(**kw) == 1


def test_qlinear_dequant_nothing_to_do():
    assert qlin_deq(M=0, y=None) == 0 and qlin_deq(N=0, y=None) == 0


def qlin_noalloc(**kw):
    a = dict(a_q=NZ, M=4, K=64, N=8, w_q=NZ, w_bits=8, w_scale=NZ, w_colsum=NZ, a_scale=0.1,
             a_zp=0, out_scale=0.1, out_zp=0, out_bits=8, bias=None, y_q=NZ, stream=None)
    a.update(kw)
    return mq.lib().mq_qlinear_noalloc(a["a_q"], a["M"], a["K"], a["N"], a["w_q"], a["w_bits"],
                                       a["w_scale"], a["w_colsum"], a["a_scale"], a["a_zp"],
                                       a["out_scale"], a["out_zp"], a["out_bits"], a["bias"],
                                       a["y_q"], a["stream"])


@pytest.mark.parametrize("kw", [
    dict(a_q=None), dict(w_q=None), dict(y_q=None), dict(M=-1), dict(K=0), dict(K=65537),
    dict(w_bits=2), dict(w_bits=4, K=63), dict(out_bits=32), dict(a_scale=0.0),
    dict(out_scale=float("nan")), dict(a_zp=128), dict(out_bits=16, out_zp=40000),
])
def test_qlinear_noalloc_rejects_invalid_arguments(kw):
    assert qlin_noalloc(**kw) == 1


def test_qlinear_noalloc_rejects_split_beyond_its_array():
    # the K split of this shape needs more than MQ_NOALLOC_SCRATCH_BYTES:
    # refused on the host before any device work
    need = mq.mq_qlinear_workspace_bytes(1024, 65536, 2048, 8, 16)
    assert need > mq.NOALLOC_SCRATCH_BYTES
    assert qlin_noalloc(M=1024, K=65536, N=2048, out_bits=16) == 2
    # nothing to do: no device work either
    assert qlin_noalloc(M=0) == 0 and qlin_noalloc(N=0) == 0


def test_noalloc_scratch_size_matches_header():
    text = open(HEADER).read()
    m = re.search(r"#define MQ_NOALLOC_SCRATCH_BYTES \((\d+) << (\d+)\)", text)
    assert m and (int(m.group(1)) << int(m.group(2))) == mq.NOALLOC_SCRATCH_BYTES


def qlin_ws(workspace, workspace_bytes, **kw):
    a = dict(a_q=NZ, M=64, K=4096, N=64, w_q=NZ, w_bits=8, w_scale=NZ, w_colsum=NZ, a_scale=0.1,
             a_zp=0, out_scale=0.1, out_zp=0, out_bits=8, bias=None, y_q=NZ, path=0,
             stream=None)
    a.update(kw)
    return mq.lib().mq_qlinear_ws(a["a_q"], a["M"], a["K"], a["N"], a["w_q"], a["w_bits"],
                                  a["w_scale"], a["w_colsum"], a["a_scale"], a["a_zp"],
                                  a["out_scale"], a["out_zp"], a["out_bits"], a["bias"],
                                  a["y_q"], workspace, workspace_bytes, a["path"], a["stream"])


def test_qlinear_ws_rejects_invalid_workspace():
    assert qlin_ws(P(256), -1) == 1            # negative size
    assert qlin_ws(P(256 + 16), 4096) == 1     # not 256-byte aligned
    assert qlin_ws(P(256), 4096, K=0) == 1     # the usual validation applies too
    assert qlin_ws(P(256), 4096, M=0) == 0     # empty: nothing enqueued
    assert qlin_ws(None, 0, M=0) == 0


def test_workspace_bytes_query():
    f = mq.lib().mq_qlinear_workspace_bytes
    assert f(-1, 64, 64, 8, 8) == -1
    assert f(64, 0, 64, 8, 8) == -1
    assert f(64, 65537, 64, 8, 8) == -1
    assert f(64, 64, 64, 3, 8) == -1
    assert f(64, 64, 64, 8, 12) == -1
    assert f(16, 65536, 64, 8, 8) == 0      # decode-shaped: never split
    assert f(2048, 2048, 5632, 8, 8) == 0   # enough output tiles
    # few output tiles, long K: split, and the size covers one int32 tile per
    # slice (at least two slices of a 128x128 tile) plus the counters
    n = f(512, 16384, 2048, 8, 16)
    assert n >= 2 * 128 * 128 * 4 * ((512 // 128) * (2048 // 128))
    assert n % 256 == 0
    assert mq.mq_qlinear_workspace_bytes(512, 16384, 2048, 8, 16) == n


def qlin_asym(**kw):
    a = dict(a_q=NZ, a_rowsum=NZ, M=4, K=64, N=8, w_q=NZ, w_bits=8, w_scale=NZ, w_zp=NZ,
             w_colsum=NZ, a_scale=0.1, a_zp=0, out_scale=0.1, out_zp=0, out_bits=8, bias=None,
             y_q=NZ, workspace=None, workspace_bytes=0, path=0, stream=None)
    a.update(kw)
    return mq.lib().mq_qlinear_asym(a["a_q"], a["a_rowsum"], a["M"], a["K"], a["N"], a["w_q"],
                                    a["w_bits"], a["w_scale"], a["w_zp"], a["w_colsum"],
                                    a["a_scale"], a["a_zp"], a["out_scale"], a["out_zp"],
                                    a["out_bits"], a["bias"], a["y_q"], a["workspace"],
                                    a["workspace_bytes"], a["path"], a["stream"])


@pytest.mark.parametrize("kw", [
    dict(a_rowsum=None), dict(w_zp=None), dict(a_q=None), dict(w_colsum=None), dict(K=0),
    dict(K=65537), dict(w_bits=4, K=63), dict(out_bits=12), dict(a_zp=200), dict(path=1, M=17),
    dict(workspace=P(256 + 16), workspace_bytes=4096), dict(workspace_bytes=-1),
])
def test_qlinear_asym_rejects_invalid_arguments(kw):
    assert qlin_asym(**kw) == 1


def qlin_a16(**kw):
    a = dict(a_q=NZ, M=4, K=64, N=8, w_q=NZ, w_bits=8, w_scale=NZ, w_colsum=NZ, a_scale=0.1,
             a_zp=0, out_scale=0.1, out_zp=0, out_bits=8, bias=None, y_q=NZ, path=0,
             stream=None)
    a.update(kw)
    return mq.lib().mq_qlinear_a16(a["a_q"], a["M"], a["K"], a["N"], a["w_q"], a["w_bits"],
                                   a["w_scale"], a["w_colsum"], a["a_scale"], a["a_zp"],
                                   a["out_scale"], a["out_zp"], a["out_bits"], a["bias"],
                                   a["y_q"], a["path"], a["stream"])


@pytest.mark.parametrize("kw", [
    dict(a_q=None), dict(K=0), dict(K=65537), dict(w_bits=4, K=63), dict(out_bits=12),
    dict(a_zp=32768), dict(a_zp=-32769), dict(a_scale=0.0), dict(path=1, M=17), dict(path=9),
])
def test_qlinear_a16_rejects_invalid_arguments(kw):
    assert qlin_a16(**kw) == 1


def test_qlinear_a16_accepts_int16_zero_points():
    # a zero-point outside int8 but inside int16 passes validation (M = 0:
    # nothing is launched)
    assert qlin_a16(M=0, a_zp=-30000) == 0
    assert qlin(M=0, a_zp=-30000) == 1   # the 8-bit entry point still rejects it


def test_qlinear_asym_empty_shapes_are_noops():
    assert qlin_asym(M=0, a_rowsum=None, a_q=None) == 0
    assert qlin_asym(N=0, w_zp=None) == 0


def test_qlinear_empty_shapes_are_noops():
    # M = 0 or N = 0: nothing to compute, no device touched
    assert qlin(M=0) == 0
    assert qlin(N=0) == 0
    assert qlin(M=0, a_q=None, y_q=None) == 0


@pytest.mark.parametrize("call", [
    lambda L: L.mq_quantize_act(NZ, 10, 0.0, 0, 8, NZ, None),
    lambda L: L.mq_quantize_act(NZ, 10, 0.1, 200, 8, NZ, None),
    lambda L: L.mq_quantize_act(NZ, 10, 0.1, 0, 12, NZ, None),
    lambda L: L.mq_quantize_act(None, 10, 0.1, 0, 8, NZ, None),
    lambda L: L.mq_quantize_act(NZ, -1, 0.1, 0, 8, NZ, None),
    lambda L: L.mq_dequant(NZ, 8, 10, float("inf"), 0, NZ, None),
    lambda L: L.mq_dequant(NZ, 16, 10, 1.0, 40000, NZ, None),
    lambda L: L.mq_dequant(None, 8, 10, 1.0, 0, NZ, None),
    lambda L: L.mq_pack_weights(NZ, 4, 63, 4, NZ, NZ, NZ, None),
    lambda L: L.mq_pack_weights(NZ, 4, 0, 8, NZ, NZ, NZ, None),
    lambda L: L.mq_pack_weights(NZ, 4, 65537, 8, NZ, NZ, NZ, None),
    lambda L: L.mq_pack_weights(NZ, 4, 64, 3, NZ, NZ, NZ, None),
    lambda L: L.mq_pack_weights(NZ, 4, 64, 8, NZ, None, NZ, None),
    lambda L: L.mq_pack_weights_asym(NZ, 4, 63, 4, 0, NZ, NZ, NZ, NZ, None),
    lambda L: L.mq_pack_weights_asym(NZ, 4, 0, 8, 0, NZ, NZ, NZ, NZ, None),
    lambda L: L.mq_pack_weights_asym(NZ, 4, 64, 2, 0, NZ, NZ, NZ, NZ, None),
    lambda L: L.mq_pack_weights_asym(NZ, 4, 64, 8, 0, NZ, NZ, None, NZ, None),
    lambda L: L.mq_pack_weights_asym(NZ, -1, 64, 8, 0, NZ, NZ, NZ, NZ, None),
    lambda L: L.mq_pack_weights_asym(NZ, 4, 64, 8, 2, NZ, NZ, NZ, NZ, None),
    lambda L: L.mq_quantize_act_rowsum(NZ, 4, 0, 0.1, 0, NZ, NZ, None),
    lambda L: L.mq_quantize_act_rowsum(NZ, -1, 8, 0.1, 0, NZ, NZ, None),
    lambda L: L.mq_quantize_act_rowsum(NZ, 4, 8, 0.0, 0, NZ, NZ, None),
    lambda L: L.mq_quantize_act_rowsum(NZ, 4, 8, float("nan"), 0, NZ, NZ, None),
    lambda L: L.mq_quantize_act_rowsum(NZ, 4, 8, 0.1, 128, NZ, NZ, None),
    lambda L: L.mq_quantize_act_rowsum(NZ, 4, 8, 0.1, 0, NZ, None, None),
    lambda L: L.mq_quantize_act_rowsum(None, 4, 8, 0.1, 0, NZ, NZ, None),
    lambda L: L.mq_act_rowsum(NZ, 4, 0, NZ, None),
    lambda L: L.mq_act_rowsum(NZ, -1, 4, NZ, None),
    lambda L: L.mq_act_rowsum(NZ, 4, 65537, NZ, None),
    lambda L: L.mq_act_rowsum(None, 4, 4, NZ, None),
    lambda L: L.mq_act_rowsum(NZ, 4, 4, None, None),
    lambda L: L.mq_fold_weights(NZ, None, 4, 4, NZ, None),
    lambda L: L.mq_fold_acts(NZ, NZ, -1, 4, NZ, None),
])
def test_other_entry_points_reject_invalid_arguments(call):
    assert call(mq.lib()) == 1


def test_zero_sized_elementwise_calls_are_noops():
    L = mq.lib()
    assert L.mq_quantize_act(None, 0, 0.1, 0, 8, None, None) == 0
    assert L.mq_dequant(None, 16, 0, 0.1, 0, None, None) == 0
    assert L.mq_pack_weights(None, 0, 64, 8, None, None, None, None) == 0
    assert L.mq_fold_weights(None, None, 0, 7, None, None) == 0
    assert L.mq_pack_weights_asym(None, 0, 64, 4, 1, None, None, None, None, None) == 0
    assert L.mq_act_rowsum(None, 0, 64, None, None) == 0
    assert L.mq_quantize_act_rowsum(None, 0, 64, 0.1, 0, None, None, None) == 0


def test_act_params_matches_oracle():
    rng = np.random.default_rng(21)
    cases = [(-64.0, 191.0), (-10.0, 117.5), (5.0, 255.0), (-7.0, -1.0), (0.0, 0.0),
             (-1e-30, 1e-30), (-3e38, 3e38), (-1.0, 0.0)]
    for _ in range(2000):
        lo, hi = sorted(rng.standard_normal(2) * 10 ** rng.uniform(-6, 6, 2))
        cases.append((float(np.float32(lo)), float(np.float32(hi))))
    for lo, hi in cases:
        for bits in (8, 16):
            assert mq.mq_act_params(lo, hi, bits) == oracle.act_params(lo, hi, bits), (lo, hi)


@pytest.mark.parametrize("lo,hi,bits", [(1.0, 0.0, 8), (float("nan"), 1.0, 8),
                                        (0.0, float("inf"), 8), (0.0, 1.0, 4)])
def test_act_params_rejects(lo, hi, bits):
    with pytest.raises(mq.MQError):
        mq.mq_act_params(lo, hi, bits)


@pytest.mark.parametrize("call", [
    lambda L: L.mq_smooth_scales(NZ, 4, 8, NZ, 4, 1.5, NZ, NZ, NZ, None),
    lambda L: L.mq_smooth_scales(NZ, 4, 8, NZ, 4, -0.1, NZ, NZ, NZ, None),
    lambda L: L.mq_smooth_scales(NZ, 4, 8, NZ, 4, float("nan"), NZ, NZ, NZ, None),
    lambda L: L.mq_smooth_scales(NZ, -1, 8, NZ, 4, 0.5, NZ, NZ, NZ, None),
    lambda L: L.mq_smooth_scales(None, 4, 8, NZ, 4, 0.5, NZ, NZ, NZ, None),
    lambda L: L.mq_smooth_scales(NZ, 4, 8, NZ, 4, 0.5, NZ, NZ, None, None),
    lambda L: L.mq_arl_forward(NZ, 10, 0.0, 1.0, 8, NZ, None),
    lambda L: L.mq_arl_forward(NZ, 10, 0.1, float("inf"), 8, NZ, None),
    lambda L: L.mq_arl_forward(NZ, 10, 0.1, 1.0, 1, NZ, None),
    lambda L: L.mq_arl_forward(NZ, 10, 0.1, 1.0, 17, NZ, None),
    lambda L: L.mq_arl_forward(None, 10, 0.1, 1.0, 8, NZ, None),
    lambda L: L.mq_arl_backward(NZ, NZ, 10, 0.1, 1.0, 8, NZ, None, None),
    lambda L: L.mq_arl_backward(NZ, None, 10, 0.1, 1.0, 8, NZ, NZ, None),
    lambda L: L.mq_arl_backward(NZ, NZ, 10, float("nan"), 1.0, 8, NZ, NZ, None),
])
def test_calibration_entry_points_reject_invalid_arguments(call):
    assert call(mq.lib()) == 1


def test_calibration_empty_calls():
    L = mq.lib()
    assert L.mq_smooth_scales(None, 0, 0, None, 0, 0.5, None, None, None, None) == 0
    assert L.mq_arl_forward(None, 0, 0.1, 1.0, 8, None, None) == 0


@pytest.mark.parametrize("call", [
    lambda L: L.mq_add_requant(NZ, 0.0, 0, NZ, 1.0, 0, 10, 1.0, 0, 16, NZ, None),
    lambda L: L.mq_add_requant(NZ, 1.0, 40000, NZ, 1.0, 0, 10, 1.0, 0, 16, NZ, None),
    lambda L: L.mq_add_requant(NZ, 1.0, 0, NZ, 1.0, 0, 10, 1.0, 200, 8, NZ, None),
    lambda L: L.mq_add_requant(NZ, 1.0, 0, None, 1.0, 0, 10, 1.0, 0, 16, NZ, None),
    lambda L: L.mq_lut_build(2, 1.0, 0, 1.0, 0, 8, NZ, None),
    lambda L: L.mq_lut_build(1, 1.0, 0, 1.0, 0, 8, None, None),
    lambda L: L.mq_lut_build(1, float("nan"), 0, 1.0, 0, 8, NZ, None),
    lambda L: L.mq_lut_apply(NZ, 10, None, 8, NZ, None),
    lambda L: L.mq_lut_apply(NZ, 10, NZ, 4, NZ, None),
    lambda L: L.mq_rmsnorm(NZ, 4, 0, 1.0, 0, None, 0.0, 1.0, 0, 8, NZ, None),
    lambda L: L.mq_rmsnorm(NZ, 4, 8, 1.0, 0, None, -1.0, 1.0, 0, 8, NZ, None),
    lambda L: L.mq_rmsnorm(NZ, 4, 8, 1.0, 0, None, 0.0, 0.0, 0, 8, NZ, None),
    lambda L: L.mq_softmax(NZ, 4, 0, 1.0, 0, 1.0, 0, 16, NZ, None),
    lambda L: L.mq_softmax(NZ, 4, 8, 1.0, 0, 1.0, 0, 16, None, None),
    lambda L: L.mq_softmax(NZ, -1, 8, 1.0, 0, 1.0, 0, 16, NZ, None),
])
def test_glue_entry_points_reject_invalid_arguments(call):
    assert call(mq.lib()) == 1


def attn(**kw):
    a = dict(a=NZ, lda=64, a_hs=64 * 16, H=4, b=NZ, ldb=64, b_hs=64 * 16, G=2, M=16, N=16, K=64,
             a_scale=0.1, a_zp=0, b_scale=0.1, b_zp=0, out_scale=0.1, out_zp=0, out_bits=16,
             y=NZ, ldy=16, y_hs=256, oc=-1, ic=-1, ws=P(256), ws_bytes=1 << 20, path=0,
             stream=None)
    a.update(kw)
    return mq.lib().mq_attn_matmul(a["a"], a["lda"], a["a_hs"], a["H"], a["b"], a["ldb"],
                                   a["b_hs"], a["G"], a["M"], a["N"], a["K"], a["a_scale"],
                                   a["a_zp"], a["b_scale"], a["b_zp"], a["out_scale"],
                                   a["out_zp"], a["out_bits"], a["y"], a["ldy"], a["y_hs"],
                                   a["oc"], a["ic"], a["ws"], a["ws_bytes"], a["path"],
                                   a["stream"])


@pytest.mark.parametrize("kw", [
    dict(H=0), dict(G=0), dict(H=4, G=3), dict(M=-1), dict(K=0), dict(K=65537),
    dict(lda=63), dict(ldb=32), dict(ldy=15), dict(a_hs=-1), dict(out_bits=4),
    dict(a_scale=0.0), dict(b_scale=float("inf")), dict(out_scale=-1.0),
    dict(a_zp=40000), dict(b_zp=128), dict(out_zp=200, out_bits=8), dict(path=1),
    dict(a=None), dict(b=None), dict(y=None), dict(ws=None), dict(ws_bytes=16),
    dict(ws=P(264)), dict(oc=-2), dict(ic=-2), dict(ic=1 << 41),
])
def test_attn_matmul_rejects_invalid_arguments(kw):
    assert attn(**kw) == 1


def test_attn_matmul_sizes_and_empty_calls():
    L = mq.lib()
    n = L.mq_attn_matmul_workspace_bytes(32, 4, 1024, 1024)
    assert n >= 32 * 1024 * 8 + 4 * 1024 * 4 and n % 256 == 0
    assert L.mq_attn_matmul_workspace_bytes(4, 3, 8, 8) == -1
    assert L.mq_attn_matmul_workspace_bytes(0, 1, 8, 8) == -1
    assert attn(M=0, a=None, b=None, y=None, ws=None) == 0
    assert attn(N=0, a=None, b=None, y=None, ws=None, ldy=0) == 0
    assert L.mq_transpose_i8(None, 0, 5, 5, None, None) == 0
    assert L.mq_transpose_i8(NZ, 4, 5, 4, NZ, None) == 1
    assert L.mq_transpose_i8(None, 4, 5, 5, NZ, None) == 1
    assert L.mq_transpose_i8(NZ, -1, 5, 5, NZ, None) == 1


@pytest.mark.parametrize("call", [
    lambda L: L.mq_softmax_causal(NZ, 4, 8, 1.0, 0, 1.0, 0, 16, 0, 0, NZ, None),
    lambda L: L.mq_softmax_causal(NZ, 4, 8, 1.0, 0, 1.0, 0, 16, 4, -1, NZ, None),
    lambda L: L.mq_softmax_causal(NZ, 4, 0, 1.0, 0, 1.0, 0, 16, 4, 0, NZ, None),
    lambda L: L.mq_softmax_causal(None, 4, 8, 1.0, 0, 1.0, 0, 16, 4, 0, NZ, None),
    lambda L: L.mq_softmax_causal(NZ, 4, 8, 0.0, 0, 1.0, 0, 16, 4, 0, NZ, None),
])
def test_softmax_causal_rejects_invalid_arguments(call):
    assert call(mq.lib()) == 1


@pytest.mark.parametrize("call", [
    lambda L: L.mq_mul_requant(NZ, 0.0, 0, NZ, 1.0, 0, 10, 1.0, 0, 16, NZ, None),
    lambda L: L.mq_mul_requant(NZ, 1.0, 0, NZ, 1.0, 0, 10, 1.0, 200, 8, NZ, None),
    lambda L: L.mq_mul_requant(NZ, 1.0, 0, None, 1.0, 0, 10, 1.0, 0, 16, NZ, None),
    lambda L: L.mq_rope(NZ, 4, 2, 3, 1.0, 0, 10000.0, 0, 1.0, 0, 16, NZ, NZ, None),
    lambda L: L.mq_rope(NZ, 4, 0, 8, 1.0, 0, 10000.0, 0, 1.0, 0, 16, NZ, NZ, None),
    lambda L: L.mq_rope(NZ, 4, 2, 8, 1.0, 0, 1.0, 0, 1.0, 0, 16, NZ, NZ, None),
    lambda L: L.mq_rope(NZ, 4, 2, 8, 1.0, 0, 10000.0, -1, 1.0, 0, 16, NZ, NZ, None),
    lambda L: L.mq_rope(NZ, 4, 2, 8, 1.0, 0, 10000.0, 0, 1.0, 0, 16, None, NZ, None),
    lambda L: L.mq_rope(NZ, 4, 2, 8, 1.0, 0, float("nan"), 0, 1.0, 0, 16, NZ, NZ, None),
    lambda L: L.mq_add_rmsnorm(NZ, 1.0, 0, NZ, 1.0, 0, 4, 0, 1.0, 0, NZ, None, 1e-5, 1.0, 0, 8, NZ, None),
    lambda L: L.mq_add_rmsnorm(NZ, 1.0, 0, NZ, 1.0, 0, 4, 8, 0.0, 0, NZ, None, 1e-5, 1.0, 0, 8, NZ, None),
    lambda L: L.mq_add_rmsnorm(NZ, 1.0, 0, NZ, 1.0, 0, 4, 8, 1.0, 0, NZ, None, -1.0, 1.0, 0, 8, NZ, None),
    lambda L: L.mq_add_rmsnorm(NZ, 1.0, 0, NZ, 1.0, 0, 4, 8, 1.0, 0, None, None, 1e-5, 1.0, 0, 8, NZ, None),
    lambda L: L.mq_add_rmsnorm(NZ, 1.0, 0, NZ, 1.0, 0, 4, 8, 1.0, 0, NZ, None, 1e-5, 1.0, 300, 8, NZ, None),
    lambda L: L.mq_lut_mul(NZ, NZ, 12, 1.0, 0, NZ, 1.0, 0, 10, 1.0, 0, 8, NZ, None),
    lambda L: L.mq_lut_mul(NZ, NZ, 8, 1.0, 200, NZ, 1.0, 0, 10, 1.0, 0, 8, NZ, None),
    lambda L: L.mq_lut_mul(NZ, NZ, 16, 0.0, 0, NZ, 1.0, 0, 10, 1.0, 0, 8, NZ, None),
    lambda L: L.mq_lut_mul(NZ, None, 16, 1.0, 0, NZ, 1.0, 0, 10, 1.0, 0, 8, NZ, None),
    lambda L: L.mq_lut_mul(NZ, NZ, 16, 1.0, 0, NZ, 1.0, 0, -1, 1.0, 0, 8, NZ, None),
    lambda L: L.mq_rope_table(4, 3, 10000.0, 0, NZ, None),
    lambda L: L.mq_rope_table(4, 8, 0.5, 0, NZ, None),
    lambda L: L.mq_rope_table(4, 8, 10000.0, -1, NZ, None),
    lambda L: L.mq_rope_table(4, 8, 10000.0, 0, None, None),
    lambda L: L.mq_rope_table(-1, 8, 10000.0, 0, NZ, None),
    lambda L: L.mq_rope_apply(NZ, 4, 2, 3, 1.0, 0, NZ, 1.0, 0, 16, NZ, None),
    lambda L: L.mq_rope_apply(NZ, 4, 0, 8, 1.0, 0, NZ, 1.0, 0, 16, NZ, None),
    lambda L: L.mq_rope_apply(NZ, 4, 2, 8, 0.0, 0, NZ, 1.0, 0, 16, NZ, None),
    lambda L: L.mq_rope_apply(NZ, 4, 2, 8, 1.0, 0, None, 1.0, 0, 16, NZ, None),
    lambda L: L.mq_rope_apply(NZ, 4, 2, 8, 1.0, 0, NZ, 1.0, 300, 8, NZ, None),
    lambda L: L.mq_rope_apply(NZ, 4, 2, 8, 1.0, 0, NZ, 1.0, 0, 12, NZ, None),
])
def test_mul_and_rope_reject_invalid_arguments(call):
    assert call(mq.lib()) == 1


def test_probe_read_validation():
    L = mq.lib()
    ok = dict(src=NZ, bytes=4096, blocks=4, waves=4, unroll=8, sink=NZ)

    def call(**kw):
        a = dict(ok)
        a.update(kw)
        return L.mq_probe_read(a["src"], a["bytes"], a["blocks"], a["waves"], a["unroll"],
                               a["sink"], None)

    for bad in (dict(bytes=-1), dict(blocks=0), dict(waves=0), dict(waves=17), dict(unroll=3),
                dict(unroll=32), dict(sink=None), dict(src=None)):
        assert call(**bad) == mq.MQ_ERR_INVALID_ARG, bad
    assert call(bytes=1 << 40, blocks=1) == mq.MQ_ERR_UNSUPPORTED
