"""GPU parity of asymmetric weights (Section 5.1): the packer, the
activation row sums and the layer with weight zero-points, against the
CPU oracle.  Integer results bit-exact, scales identical.
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


def _weights(N, K, seed):
    rng = np.random.default_rng(seed)
    w = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
    w += (rng.uniform(-2, 2, N) * 0.02).astype(np.float32)[:, None]
    if N > 8:
        w[1] = 0.0                                   # zero-width range
        w[2] = np.abs(w[2]) + 0.01                   # all positive
        w[3] = -np.abs(w[3]) - 0.01                  # all negative
        w[4] = 0.37                                  # constant
        w[5, :3] = [np.inf, np.nan, -np.inf]         # ignored by the range
        w[6, :] = np.linspace(-1e-3, 9e-3, K)        # ties at both ends
    return w


@pytest.mark.parametrize("per_tensor", [False, True])
@pytest.mark.parametrize("bits", [8, 4])
@pytest.mark.parametrize("N,K", [(37, 96), (300, 2048), (9, 1000), (3, 2)])
def test_pack_weights_asym_parity(N, K, bits, per_tensor):
    mq, torch = _mq(), _torch()
    if bits == 4 and K % 2:
        pytest.skip("int4 needs an even K")
    w = _weights(N, K, N * K + bits)
    if per_tensor and N > 8:
        w[0, 0], w[-1, -1] = -0.3, 0.5               # the extremes in the first and last row
    gq, gs, gz, gc = mq.mq_pack_weights_asym(torch.from_numpy(w).cuda(), bits,
                                             per_tensor=per_tensor)
    oq, os_, oz, oc = oracle.pack_weights_asym(w, bits, per_tensor=per_tensor)
    assert np.array_equal(gs.cpu().numpy().view(np.uint32), os_.view(np.uint32))
    assert np.array_equal(gz.cpu().numpy(), oz)
    assert np.array_equal(gq.cpu().numpy(), oq)
    assert np.array_equal(gc.cpu().numpy(), oc)


@pytest.mark.parametrize("M,K,offset", [(1, 1, 0), (3, 7, 0), (17, 300, 1), (64, 2048, 0),
                                        (5, 65536, 0), (2048, 2048, 0), (33, 4112, 3)])
def test_act_rowsum_parity(M, K, offset):
    mq, torch = _mq(), _torch()
    rng = np.random.default_rng(M + K)
    a = rng.integers(-128, 128, (M, K)).astype(np.int8)
    a[0] = -128
    buf = torch.empty(M * K + offset, dtype=torch.int8, device="cuda")
    ga = buf[offset:].view(M, K)
    ga.copy_(torch.from_numpy(a))
    rs = mq.mq_act_rowsum(ga)
    assert np.array_equal(rs.cpu().numpy(), oracle.act_rowsum(a))


@pytest.mark.parametrize("M,K,offset", [(1, 2048, 0), (7, 5632, 0), (33, 1001, 0), (64, 2048, 1),
                                        (3, 65536, 0), (1024, 2048, 0), (5, 6, 2)])
def test_quantize_act_rowsum_parity(M, K, offset):
    """The fused quantizer + row sum: codes equal the oracle's Eq.(4) codes
    and the plain quantizer's, row sums the oracle's sums of those codes.
    offset > 0 puts x off its 16-byte alignment (the scalar path)."""
    mq, torch = _mq(), _torch()
    rng = np.random.default_rng(M * 7 + K)
    x = rng.standard_normal((M, K)).astype(np.float32) * 3
    x[:, : min(K, 4)] *= 30.0
    x.reshape(-1)[:3] = [np.nan, np.inf, -np.inf]
    alpha, zp = mq.mq_act_params(-10.0, 14.0, 8)
    # values on and next to the rounding ties of the grid
    ties = ((np.arange(K) % 40 - 20) + 0.5).astype(np.float32) * np.float32(alpha)
    x[-1] = np.where(np.arange(K) % 2 == 0, ties, np.nextafter(ties, np.float32(np.inf)))
    buf = torch.empty(M * K + offset, dtype=torch.float32, device="cuda")
    gx = buf[offset:].view(M, K)
    gx.copy_(torch.from_numpy(x))
    q, rs = mq.mq_quantize_act_rowsum(gx, alpha, zp)
    ref = oracle.quantize_act(x, alpha, zp, 8)
    assert np.array_equal(q.cpu().numpy(), ref)
    assert np.array_equal(rs.cpu().numpy(), oracle.act_rowsum(ref))
    assert np.array_equal(mq.mq_quantize_act(gx, alpha, zp, 8).cpu().numpy(), ref)


ASYM_CASES = [
    # M, K, N, w_bits, out_bits, bias, per_tensor -- several tiles, ragged tails
    (1, 2048, 520, 8, 8, True, False),       # decode
    (5, 272, 37, 8, 16, True, True),         # decode, K not a multiple of 64
    (16, 5632, 300, 4, 16, False, False),    # decode, int4, several rounds
    (300, 2048, 520, 8, 8, True, True),      # prefill, ragged M and N
    (129, 640, 257, 8, 16, False, False),
    (200, 5632, 300, 4, 16, False, False),   # prefill, int4
    (261, 1088, 389, 4, 8, True, False),
    (96, 2048, 384, 8, 16, False, True),
]


@pytest.mark.parametrize("case", ASYM_CASES, ids=lambda c: "x".join(map(str, c[:5])) +
                         ("-tensor" if c[6] else "-channel"))
def test_asym_layer_parity(case):
    M, K, N, wb, ob, has_bias, per_tensor = case
    layer = wl.Layer("x", M, K, N, w_bits=wb, out_bits=ob, bias=has_bias, asym=True,
                     per_tensor=per_tensor)
    ld = wl.make_layer("asym", layer)
    assert_same(gpu_layer(ld), oracle_layer(ld))


@pytest.mark.parametrize("w_bits,out_bits", [(8, 8), (8, 16), (4, 8), (4, 16)])
@pytest.mark.parametrize("M", [1, 7, 16])
def test_asym_paths_agree(w_bits, out_bits, M):
    mq = _mq()
    layer = wl.Layer("x", M, 1024, 200, w_bits=w_bits, out_bits=out_bits, asym=True)
    ld = wl.make_layer("asym_paths", layer)
    outs = [gpu_layer(ld, path=p).y_q for p in (mq.PATH_DECODE, mq.PATH_PREFILL, mq.PATH_GENERIC)]
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])
    assert np.array_equal(outs[0], oracle_layer(ld).y_q)


@pytest.mark.parametrize("w_bits", [8, 4])
def test_asym_prefill_equals_generic_ragged(w_bits):
    mq = _mq()
    layer = wl.Layer("x", 261, 1088, 389, w_bits=w_bits, out_bits=16, asym=True)
    ld = wl.make_layer("asym_ragged", layer)
    a = gpu_layer(ld, path=mq.PATH_PREFILL).y_q
    b = gpu_layer(ld, path=mq.PATH_GENERIC).y_q
    assert np.array_equal(a, b)


@pytest.mark.parametrize("case", [(130, 8192, 300, 8, 8), (200, 5632, 300, 4, 16)],
                         ids=lambda c: "x".join(map(str, c)))
def test_asym_split_k_parity(case):
    """K split through a workspace: the zero-point term joins in the last
    slice's epilogue; twice in a row on one workspace."""
    mq, torch = _mq(), _torch()
    M, K, N, wb, ob = case
    nbytes = mq.mq_qlinear_workspace_bytes(M, K, N, wb, ob)
    assert nbytes > 0
    ws = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")
    layer = wl.Layer("x", M, K, N, w_bits=wb, out_bits=ob, asym=True)
    ld = wl.make_layer("asym_splitk", layer)
    o = oracle_layer(ld)
    for _ in range(2):
        assert_same(gpu_layer(ld, workspace=ws), o)
    assert int(ws[:256].count_nonzero()) == 0


def _pack_codes(codes, w_bits):
    if w_bits == 8:
        return codes.astype(np.int8)
    c = codes.astype(np.int64)
    return ((c[:, 0::2] & 0xF) | ((c[:, 1::2] & 0xF) << 4)).astype(np.uint8)


@pytest.mark.parametrize("w_bits", [8, 4])
@pytest.mark.parametrize("K", [65536, 32768, 4096])
def test_asym_extreme_zero_points(w_bits, K):
    """Weight codes and zero-points at the grid ends, activations at the
    int8 ends, a large bias: the largest zero-point terms the format allows.
    K = 65536 leaves the tiled kernels' 24-bit fast form for the exact int64
    one; K = 32768 with a large bias mixes both forms across tiles."""
    mq, torch = _mq(), _torch()
    dev = torch.device("cuda", 0)
    rng = np.random.default_rng(K + w_bits)
    qlo, qhi = (-128, 127) if w_bits == 8 else (-8, 7)
    N = 96
    codes = np.where(rng.random((N, K)) < 0.5, qlo, qhi).astype(np.int64)
    codes[0::3] = qlo
    codes[1::3] = qhi
    zw = np.where(np.arange(N) % 2 == 0, qlo, qhi).astype(np.int32)
    zw[5::7] = 0
    wq = _pack_codes(codes, w_bits)
    colsum = codes.sum(axis=1).astype(np.int32)
    ws = rng.uniform(1e-4, 1e-3, N).astype(np.float32)
    bias = (rng.standard_normal(N) * 200.0).astype(np.float32)
    g_wq, g_ws, g_zw, g_cs, g_b = (torch.from_numpy(v).to(dev) for v in (wq, ws, zw, colsum, bias))
    for M, path in ((16, mq.PATH_DECODE), (300, mq.PATH_PREFILL), (16, mq.PATH_GENERIC)):
        a = np.where(rng.random((M, K)) < 0.5, -128, 127).astype(np.int8)
        a[0] = -128
        a[1] = 127
        g_a = torch.from_numpy(a).to(dev)
        rs = mq.mq_act_rowsum(g_a)
        for a_zp, out_scale, out_bits in ((127, 50.0, 16), (-128, 2.0, 8), (0, 1e3, 16)):
            y = mq.mq_qlinear_asym(g_a, rs, g_wq, w_bits, g_ws, g_zw, g_cs, 0.05, a_zp,
                                   out_scale, 3, out_bits, bias=g_b, path=path)
            ref = oracle.qlinear(a, wq, w_bits, ws, 0.05, a_zp, out_scale, 3, out_bits,
                                 bias=bias, w_zp=zw)
            got = y.cpu().numpy()
            if not np.array_equal(got, ref):
                bad = np.argwhere(got != ref)
                m, n = bad[0]
                raise AssertionError(f"path {path} a_zp {a_zp}: {len(bad)} differ, first "
                                     f"({m},{n}) gpu {got[m, n]} oracle {ref[m, n]}")


def test_asym_zero_points_of_zero_equal_symmetric():
    # the asymmetric entry point with w_zp = 0 is the symmetric layer
    mq, torch = _mq(), _torch()
    ld = wl.make_layer("asym_zero", wl.Layer("x", 130, 1024, 200, out_bits=16))
    for path in (mq.PATH_PREFILL, mq.PATH_GENERIC):
        g, d = gpu_layer(ld, keep_device=True, path=path)
        rs = mq.mq_act_rowsum(d["a_q"])
        zero = torch.zeros(200, dtype=torch.int32, device="cuda")
        y = mq.mq_qlinear_asym(d["a_q"], rs, d["w_q"], 8, d["w_scale"], zero, d["w_colsum"],
                               d["a_scale"], d["a_zp"], d["out_scale"], d["out_zp"], 16,
                               bias=d["bias"], path=path)
        assert np.array_equal(y.cpu().numpy(), g.y_q)
