"""GPU parity of mq_qlinear_dequant (the epilogue writes the dequantized
outputs, and the codes only when asked) against the oracle's qlinear
followed by the oracle's dequantization: every fp32 value bit for bit, on
every path (prefill tiles, K split, decode, one-token GEMV, generic),
symmetric and asymmetric weights, int8 and int16 codes, with and without
the codes stored.
"""
import numpy as np
import pytest

import oracle

pytestmark = pytest.mark.gpu


def _mq():
    import paper_2408_13933_amd as mq
    return mq


def _torch():
    import torch
    return torch


def _pack_int4(codes):
    """Two's-complement nibbles, the even k in the low nibble (the packed
    int4 layout), written out independently of both pipelines."""
    lo = codes[:, 0::2].astype(np.int64) & 0xF
    hi = codes[:, 1::2].astype(np.int64) & 0xF
    return (lo | (hi << 4)).astype(np.uint8)


def _case(seed, M, K, N, w_bits, asym, bias):
    rng = np.random.default_rng(seed)
    qw = 128 if w_bits == 8 else 8
    a = rng.integers(-128, 128, (M, K)).astype(np.int8)
    codes = rng.integers(-qw, qw, (N, K))
    return dict(a=a, wq=codes.astype(np.int8) if w_bits == 8 else _pack_int4(codes),
                cs=codes.sum(axis=1).astype(np.int32),
                ws=(10.0 ** rng.uniform(-5, -2, N)).astype(np.float32),
                zw=rng.integers(-qw, qw, N).astype(np.int32) if asym else None,
                bias=(rng.standard_normal(N) * 0.5).astype(np.float32) if bias else None)


def _check(c, w_bits, out_bits, out_scale, out_zp, path, with_codes, workspace=None):
    mq, torch = _mq(), _torch()
    dev = torch.device("cuda", 0)
    a_scale, a_zp = 0.03, -3
    M, N = c["a"].shape[0], c["wq"].shape[0]
    g = {k: (None if v is None else torch.from_numpy(v).to(dev)) for k, v in c.items()}
    rs = mq.mq_act_rowsum(g["a"]) if c["zw"] is not None else None
    codes = (torch.empty((M, N), dtype=torch.int8 if out_bits == 8 else torch.int16, device=dev)
             if with_codes else None)
    y = mq.mq_qlinear_dequant(g["a"], g["wq"], w_bits, g["ws"], g["cs"], a_scale, a_zp,
                              out_scale, out_zp, out_bits, bias=g["bias"], codes=codes,
                              w_zp=g["zw"], a_rowsum=rs, path=path, workspace=workspace)
    ref_q = oracle.qlinear(c["a"], c["wq"], w_bits, c["ws"], a_scale, a_zp, out_scale, out_zp,
                           out_bits, bias=c["bias"], w_zp=c["zw"])
    ref = oracle.dequant(ref_q, out_scale, out_zp)
    got = y.cpu().numpy()
    assert got.dtype == np.float32 and np.array_equal(got, ref), int((got != ref).sum())
    if with_codes:
        assert np.array_equal(codes.cpu().numpy(), ref_q)


@pytest.mark.parametrize("with_codes", [False, True])
@pytest.mark.parametrize("case", [
    # M, K, N, w_bits, out_bits, asym, bias, out_scale, out_zp
    (300, 512, 520, 8, 16, False, True, 0.002, 1234),   # the pre-shift form (int16 codes)
    (257, 1024, 388, 8, 8, False, False, 0.05, -7),
    (130, 640, 260, 4, 16, True, True, 30.0, -3),
    (96, 768, 132, 4, 8, True, False, 0.05, 5),
    (64, 256, 258, 8, 8, False, True, 0.05, 0),          # N % 4 != 0: the generic kernel
], ids=lambda c: "x".join(map(str, c[:5])) + ("a" if c[5] else ""))
def test_dequant_output_prefill_and_generic(case, with_codes):
    M, K, N, w_bits, out_bits, asym, bias, out_scale, out_zp = case
    c = _case(M * 31 + N, M, K, N, w_bits, asym, bias)
    _check(c, w_bits, out_bits, out_scale, out_zp, _mq().PATH_AUTO, with_codes)


@pytest.mark.parametrize("tile", list(range(6)))
def test_dequant_output_every_tile(tile):
    c = _case(tile, 264, 1024, 520, 8, False, True)
    _check(c, 8, 16, 0.002, 77, _mq().prefill_tile_path(tile), False)


def test_dequant_output_with_k_split():
    mq, torch = _mq(), _torch()
    M, K, N = 130, 8192, 300
    nbytes = mq.mq_qlinear_workspace_bytes(M, K, N, 8, 16)
    assert nbytes > 0, "the shape is expected to split"
    ws = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")
    c = _case(11, M, K, N, 8, False, True)
    for _ in range(2):
        _check(c, 8, 16, 0.01, -40, mq.PATH_AUTO, False, workspace=ws)


@pytest.mark.parametrize("M,K,N,w_bits,asym", [(8, 512, 136, 8, False), (16, 2048, 200, 4, False),
                                              (1, 1024, 264, 8, True), (1, 2048, 3000, 4, False),
                                              (5, 272, 37, 8, False)],
                         ids=["decode", "decode-int4", "gemv-asym", "gemv-int4", "decode-ragged"])
@pytest.mark.parametrize("with_codes", [False, True])
def test_dequant_output_decode_paths(M, K, N, w_bits, asym, with_codes):
    c = _case(M * 7 + N, M, K, N, w_bits, asym, True)
    _check(c, w_bits, 16, 0.004, 12, _mq().PATH_AUTO, with_codes)


def test_dequant_output_full_size_lm_head():
    """The Gemma-2B LM head at M = 512 (the bench step's last launch), full
    size: every fused fp32 logit equals mq_dequant of mq_qlinear's codes
    (which the full-size parity test compares with the oracle)."""
    mq, torch = _mq(), _torch()
    from paper_2408_13933_amd import workloads as wl
    dev = torch.device("cuda", 0)
    layer = next(l for l in wl.WORKLOADS["gemma2b_w8a8"].layers if l.name == "lm_head_m512")
    ld = wl.make_layer("gemma2b_w8a8", layer)
    a_scale, a_zp = mq.mq_act_params(*ld.act_range, 8)
    o_scale, o_zp = mq.mq_act_params(*ld.out_range, layer.out_bits)
    a_q = mq.mq_quantize_act(torch.from_numpy(ld.x).to(dev), a_scale, a_zp, 8)
    wq, ws, cs = mq.mq_pack_weights(torch.from_numpy(ld.w).to(dev), layer.w_bits)
    codes = mq.mq_qlinear(a_q, wq, layer.w_bits, ws, cs, a_scale, a_zp, o_scale, o_zp,
                          layer.out_bits)
    ref = mq.mq_dequant(codes, o_scale, o_zp)
    del codes
    y = mq.mq_qlinear_dequant(a_q, wq, layer.w_bits, ws, cs, a_scale, a_zp, o_scale, o_zp,
                              layer.out_bits)
    assert torch.equal(y, ref)
