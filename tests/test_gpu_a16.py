"""GPU parity of the 16-bit-activation linear layer (the W8A16 setting of
Section 5.6) against the CPU oracle: bit-exact integer outputs on every
kernel path.
"""
import numpy as np
import pytest

import oracle
from paper_2408_13933_amd import workloads as wl
from tests.pipelines import assert_same, gpu_layer, oracle_layer

pytestmark = pytest.mark.gpu


def _mq():
    import paper_2408_13933_amd as mq
    return mq


def _torch():
    import torch
    return torch


A16_CASES = [
    # M, K, N, w_bits, out_bits, bias -- several tiles, ragged tails
    (1, 2048, 520, 8, 8, True),        # decode
    (5, 272, 37, 8, 16, True),         # decode, K not a multiple of 64
    (16, 5632, 300, 4, 16, False),     # decode, int4, several load rounds
    (300, 2048, 520, 8, 8, True),      # prefill, ragged M and N
    (129, 640, 257, 8, 16, False),
    (261, 1088, 384, 8, 16, True),
    (200, 1024, 300, 4, 16, False),    # int4 weights above 16 tokens: generic kernel
    (300, 64, 257, 8, 16, True),       # short K: the two-stage tile
    (129, 128, 200, 8, 8, False),
    (300, 1024, 48, 8, 16, True),      # at most 64 channels: the 64x64 tile, ragged N
    (129, 2048, 64, 8, 8, False),
]


@pytest.mark.parametrize("case", A16_CASES, ids=lambda c: "x".join(map(str, c[:5])))
def test_a16_layer_parity(case):
    M, K, N, wb, ob, has_bias = case
    layer = wl.Layer("x", M, K, N, w_bits=wb, out_bits=ob, bias=has_bias, a_bits=16)
    ld = wl.make_layer("a16", layer)
    assert_same(gpu_layer(ld), oracle_layer(ld))


@pytest.mark.parametrize("w_bits,out_bits", [(8, 8), (8, 16), (4, 16)])
@pytest.mark.parametrize("M", [1, 7, 16])
def test_a16_paths_agree(w_bits, out_bits, M):
    mq = _mq()
    layer = wl.Layer("x", M, 1024, 200, w_bits=w_bits, out_bits=out_bits, a_bits=16)
    ld = wl.make_layer("a16_paths", layer)
    outs = [gpu_layer(ld, path=p).y_q for p in (mq.PATH_DECODE, mq.PATH_PREFILL, mq.PATH_GENERIC)]
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])
    assert np.array_equal(outs[0], oracle_layer(ld).y_q)


@pytest.mark.parametrize("K,has_bias", [(65536, True), (4096, True), (64, True), (128, False)])
def test_a16_extreme_codes(K, has_bias):
    """Activation codes and zero-points at the int16 ends, weights at the
    int8 ends: sums far beyond int32 (the accumulator saturates), an offset
    beyond int32, and sums that stay inside it, on every kernel path (K =
    128 without bias: the int32 epilogue at its largest sums)."""
    mq, torch = _mq(), _torch()
    dev = torch.device("cuda", 0)
    rng = np.random.default_rng(K)
    N = 96
    codes = np.where(rng.random((N, K)) < 0.5, -127, 127).astype(np.int8)
    codes[0] = 127
    codes[1] = -127
    cs = codes.astype(np.int64).sum(axis=1).astype(np.int32)
    ws = rng.uniform(1e-4, 1e-3, N).astype(np.float32)
    bias = (rng.standard_normal(N) * 50.0).astype(np.float32)
    g_w, g_ws, g_cs, g_b = (torch.from_numpy(v).to(dev) for v in (codes, ws, cs, bias))
    if not has_bias:
        bias, g_b = None, None
    for M, path in ((16, mq.PATH_DECODE), (300, mq.PATH_PREFILL), (16, mq.PATH_GENERIC)):
        a = np.where(rng.random((M, K)) < 0.5, -32768, 32767).astype(np.int16)
        a[0] = 32767
        a[1] = -32768
        a[2] = rng.integers(-300, 300, K)   # small codes: sums well inside int32
        g_a = torch.from_numpy(a).to(dev)
        for a_zp, a_scale, out_scale, out_bits in ((-32768, 1e-4, 1e-3, 16),
                                                   (32767, 1e-5, 0.5, 8), (0, 3e-6, 2e-5, 16)):
            y = mq.mq_qlinear_a16(g_a, g_w, 8, g_ws, g_cs, a_scale, a_zp, out_scale, 5, out_bits,
                                  bias=g_b, path=path)
            ref = oracle.qlinear(a, codes, 8, ws, a_scale, a_zp, out_scale, 5, out_bits,
                                 bias=bias)
            got = y.cpu().numpy()
            if not np.array_equal(got, ref):
                bad = np.argwhere(got != ref)
                m, n = bad[0]
                raise AssertionError(f"path {path} a_zp {a_zp}: {len(bad)} differ, first "
                                     f"({m},{n}) gpu {got[m, n]} oracle {ref[m, n]}")


def test_a16_int8_range_codes_equal_the_int8_layer():
    # int8-range codes stored as int16 give the int8 layer's outputs
    mq, torch = _mq(), _torch()
    ld = wl.make_layer("a16_vs_a8", wl.Layer("x", 130, 1024, 256, out_bits=16))
    g, d = gpu_layer(ld, keep_device=True)
    for path in (mq.PATH_PREFILL, mq.PATH_GENERIC):
        y = mq.mq_qlinear_a16(d["a_q"].to(torch.int16), d["w_q"], 8, d["w_scale"], d["w_colsum"],
                              d["a_scale"], d["a_zp"], d["out_scale"], d["out_zp"], 16,
                              bias=d["bias"], path=path)
        assert np.array_equal(y.cpu().numpy(), g.y_q)
    y = mq.mq_qlinear_a16(d["a_q"][:16].to(torch.int16), d["w_q"], 8, d["w_scale"],
                          d["w_colsum"], d["a_scale"], d["a_zp"], d["out_scale"], d["out_zp"], 16,
                          bias=d["bias"], path=mq.PATH_DECODE)
    assert np.array_equal(y.cpu().numpy(), g.y_q[:16])
