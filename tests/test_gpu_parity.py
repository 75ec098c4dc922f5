"""GPU parity: the HIP path (libmq.so via its C ABI) against the CPU oracle.

Integer results must be bit-exact, scales identical, dequantized values
within 1e-6 relative.  Oracle-sized cases span several tiles with ragged
tails; full-size workload cases compare every GPU intermediate and every
output in full.
"""
import functools

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


@functools.lru_cache(maxsize=4)
def _full_layer(workload, name):
    layer = next(l for l in wl.WORKLOADS[workload].layers if l.name == name)
    return wl.make_layer(workload, layer)


def _scaled(workload, name, M=None, K=None, N=None):
    layer = next(l for l in wl.WORKLOADS[workload].layers if l.name == name)
    small = wl.scaled_layer(layer, M=M, K=K, N=N)
    return wl.make_layer(workload + "/scaled", small)


# ---------------------------------------------------------------------------
# oracle-sized cases (full oracle comparison)
# ---------------------------------------------------------------------------
SMALL_CASES = [
    # workload, layer, M, K, N   -- several tiles plus ragged tails
    ("decode_w8a8_m16", "linear", None, None, None),           # the whole config, M=16
    ("decode_w8a8_m16", "linear", 5, 272, 37),                 # K not a multiple of 64
    ("prefill_w8a8_tinyllama_m2048", "gate_proj", 300, 2048, 520),
    ("prefill_w8a8_tinyllama_m2048", "o_proj", 129, 640, 257),
    ("w4a8_down_tinyllama", "down_proj_m1", None, None, None),  # whole decode layer, int4
    ("w4a8_down_tinyllama", "down_proj_m1024", 200, 5632, 300),
    ("block_w8a8_tinyllama_s1024", "q_proj", 96, 2048, 384),
    ("block_w8a8_tinyllama_s1024", "k_proj", 96, 2048, 256),
    ("block_w8a8_tinyllama_s1024", "o_proj", 70, 2048, 200),
    ("block_w8a8_tinyllama_s1024", "down_proj", 40, 5632, 136),
    ("gemma2b_w8a8", "gate_proj", 64, 2048, 700),
    ("gemma2b_w8a8", "down_proj", 33, 16384, 160),
    ("gemma2b_w8a8", "lm_head_m1", 1, 2048, 3000),
]


@pytest.mark.parametrize("case", SMALL_CASES, ids=lambda c: f"{c[0]}-{c[1]}-{c[2]}x{c[3]}x{c[4]}")
def test_small_layer_parity(case):
    workload, name, M, K, N = case
    ld = _scaled(workload, name, M, K, N) if M else _full_layer(workload, name)
    g = gpu_layer(ld)
    o = oracle_layer(ld)
    assert_same(g, o)


@pytest.mark.parametrize("w_bits,out_bits", [(8, 8), (8, 16), (4, 8), (4, 16)])
@pytest.mark.parametrize("M", [1, 7, 16])
def test_decode_prefill_generic_agree(w_bits, out_bits, M):
    mq = _mq()
    layer = wl.Layer("x", M, 1024, 200, w_bits=w_bits, out_bits=out_bits)
    ld = wl.make_layer("paths", layer)
    outs = [gpu_layer(ld, path=p).y_q for p in (mq.PATH_DECODE, mq.PATH_PREFILL, mq.PATH_GENERIC)]
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])
    assert np.array_equal(outs[0], oracle_layer(ld).y_q)


@pytest.mark.parametrize("w_bits,out_bits", [(8, 8), (4, 16)])
@pytest.mark.parametrize("M,K,N", [(1, 5632, 48), (16, 4096, 40), (3, 16384, 33), (2, 1088, 20)])
def test_decode_multi_round_k(w_bits, out_bits, M, K, N):
    """Decode waves that stream several load rounds each (long K, few
    channel groups), against the generic path and the oracle."""
    mq = _mq()
    layer = wl.Layer("x", M, K, N, w_bits=w_bits, out_bits=out_bits)
    ld = wl.make_layer("decode_rounds", layer)
    d = gpu_layer(ld, path=mq.PATH_DECODE).y_q
    g = gpu_layer(ld, path=mq.PATH_GENERIC).y_q
    assert np.array_equal(g, oracle_layer(ld).y_q)
    assert np.array_equal(d, g)


@pytest.mark.parametrize("w_bits,out_bits", [(8, 8), (8, 16), (4, 8), (4, 16)])
@pytest.mark.parametrize("K,N", [(2048, 2048), (5632, 7), (272, 9), (16384, 33), (64, 1),
                                 (1056, 4099)])
@pytest.mark.parametrize("asym", [False, True])
def test_one_token_gemv(w_bits, out_bits, K, N, asym):
    """The one-token path (M = 1, the vector-ALU GEMV): ragged N (blocks of
    8 channels), K that is not a multiple of one wave load's 128 row bytes,
    several load rounds per wave (K = 16384), asymmetric weights and a bias,
    against the oracle and the generic kernel.  int4 rows need K % 32 == 0
    (K = 272 takes the MFMA decode kernel)."""
    mq = _mq()
    layer = wl.Layer("x", 1, K, N, w_bits=w_bits, out_bits=out_bits, bias=True, asym=asym)
    ld = wl.make_layer("gemv", layer)
    o = oracle_layer(ld)
    g = gpu_layer(ld, path=mq.PATH_DECODE)
    assert_same(g, o)
    assert np.array_equal(gpu_layer(ld, path=mq.PATH_GENERIC).y_q, o.y_q)


SPLIT_CASES = [
    # M, K, N, w_bits, out_bits, bias: few output tiles, long K (N a whole
    # number of 4-channel output groups: the tuned kernel's store rule)
    (130, 8192, 300, 8, 8, True),
    (200, 5632, 300, 4, 16, False),
    (64, 16384, 160, 8, 16, False),
    (257, 4128, 132, 8, 8, True),   # ragged M and N, K tail, uneven last slice
    (257, 4128, 132, 4, 8, False),
]


def split_workspace_bound(M, N, tile):
    """Workspace bytes a K split on prefill tile ``tile`` can use at most
    (the bound stated with the tile paths in mq.h) and its counter bytes."""
    tm, tn = _mq().PREFILL_TILE_SHAPES[tile]
    tiles = -(-M // tm) * -(-N // tn)
    counters = 256 * -(-tiles // 64)
    return counters + 8 * tiles * tm * tn * 4, counters


@pytest.mark.parametrize("tile", [1, 3, 4])
@pytest.mark.parametrize("case", SPLIT_CASES, ids=lambda c: "x".join(map(str, c[:5])))
def test_split_k_parity(case, tile):
    """K split across work-groups (workspace path) on the 128x128, the 64x64
    and the eight-wave 256x256 tile, whose cost model splits these shapes:
    bit-identical to the oracle, twice in a row on one workspace, whose
    counters end at zero."""
    mq, torch = _mq(), _torch()
    M, K, N, wb, ob, has_bias = case
    nbytes, counters = split_workspace_bound(M, N, tile)
    ws = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")
    layer = wl.Layer("x", M, K, N, w_bits=wb, out_bits=ob, bias=has_bias)
    ld = wl.make_layer("splitk", layer)
    o = oracle_layer(ld)
    path = mq.prefill_tile_path(tile)
    for _ in range(2):
        assert_same(gpu_layer(ld, workspace=ws, path=path), o)
    assert int(ws[:counters].count_nonzero()) == 0, "arrival counters not returned to zero"
    assert int(ws[counters:].count_nonzero()) > 0, "the layer did not split"
    # without a workspace the same call does not split and gives the same bits
    assert np.array_equal(gpu_layer(ld, path=path).y_q, o.y_q)


MANY_TILE_CASES = [
    # M, K, N, w_bits, out_bits, bias, asym: more 256x256 output tiles than
    # the chip has CUs (two to three rounds of work-groups), ragged M and N
    # (the last tile column takes the unstaged epilogue), K of one to five
    # stages
    (300, 128, 40004, 8, 16, True, False),
    (520, 256, 33024, 8, 8, False, False),
    (768, 384, 22016, 4, 16, True, False),
    (300, 256, 40004, 8, 8, True, True),
    (257, 640, 65536, 4, 8, False, True),
    (1024, 128, 49152, 8, 16, True, False),
]


@pytest.mark.parametrize("case", MANY_TILE_CASES, ids=lambda c: "x".join(map(str, c)))
def test_eight_wave_tile_many_rounds(case):
    """The eight-wave 256x256 tile (the LM head's) without a K split on
    layers of several rounds of tiles: bit-identical to the oracle, twice in
    a row."""
    mq = _mq()
    M, K, N, wb, ob, has_bias, asym = case
    layer = wl.Layer("x", M, K, N, w_bits=wb, out_bits=ob, bias=has_bias, asym=asym)
    ld = wl.make_layer("rounds", layer)
    o = oracle_layer(ld)
    for _ in range(2):
        assert_same(gpu_layer(ld, path=mq.prefill_tile_path(4)), o)


@pytest.mark.parametrize("w_bits", [8, 4])
def test_prefill_equals_generic_ragged(w_bits):
    mq = _mq()
    layer = wl.Layer("x", 261, 1088, 389, w_bits=w_bits, out_bits=16)
    ld = wl.make_layer("ragged", layer)
    a = gpu_layer(ld, path=mq.PATH_PREFILL).y_q
    b = gpu_layer(ld, path=mq.PATH_GENERIC).y_q
    assert np.array_equal(a, b)
    assert np.array_equal(a, oracle_layer(ld).y_q)


@pytest.mark.parametrize("K,w_bits", [(100, 8), (50, 4), (8, 8), (2, 4)])
def test_odd_k_takes_generic_path(K, w_bits):
    layer = wl.Layer("x", 37, K, 45, w_bits=w_bits, out_bits=8)
    ld = wl.make_layer("oddk", layer)
    assert_same(gpu_layer(ld), oracle_layer(ld))


def test_unaligned_buffers():
    mq, torch = _mq(), _torch()
    layer = wl.Layer("x", 20, 256, 64)
    ld = wl.make_layer("unaligned", layer)
    o = oracle_layer(ld)
    dev = torch.device("cuda", 0)
    # place every integer buffer one byte past an aligned address
    a_buf = torch.empty(20 * 256 + 1, dtype=torch.int8, device=dev)
    a_q = a_buf[1:].view(20, 256)
    a_q.copy_(torch.from_numpy(o.a_q))
    w_buf = torch.empty(64 * 256 + 1, dtype=torch.int8, device=dev)
    w_q = w_buf[1:].view(64, 256)
    w_q.copy_(torch.from_numpy(o.w_q))
    y_buf = torch.empty(20 * 64 + 1, dtype=torch.int8, device=dev)
    y = y_buf[1:].view(20, 64)
    ws = torch.from_numpy(o.w_scale).to(dev)
    cs = torch.from_numpy(o.w_colsum).to(dev)
    bias = torch.from_numpy(ld.bias).to(dev)
    for path in (mq.PATH_AUTO, mq.PATH_PREFILL):
        mq.mq_qlinear(a_q, w_q, 8, ws, cs, o.a_scale, o.a_zp, o.out_scale, o.out_zp, 8,
                      bias=bias, out=y, path=path)
        torch.cuda.synchronize()
        assert np.array_equal(y.cpu().numpy(), o.y_q)
    y16 = y_buf[1:1 + 16 * 64].view(16, 64)
    mq.mq_qlinear(a_buf[1:1 + 16 * 256].view(16, 256), w_q, 8, ws, cs, o.a_scale, o.a_zp,
                  o.out_scale, o.out_zp, 8, bias=bias, out=y16, path=mq.PATH_DECODE)
    torch.cuda.synchronize()
    assert np.array_equal(y16.cpu().numpy(), o.y_q[:16])


def test_m1_rows_equal_batched_rows():
    # rows are independent: the decode kernel on row m equals row m of prefill
    mq, torch = _mq(), _torch()
    ld = _full_layer("w4a8_down_tinyllama", "down_proj_m1024")
    g, d = gpu_layer(ld, keep_device=True)
    for m in (0, 1, 511, 1023):
        y1 = mq.mq_qlinear(d["a_q"][m:m + 1].contiguous(), d["w_q"], 4, d["w_scale"],
                           d["w_colsum"], d["a_scale"], d["a_zp"], d["out_scale"], d["out_zp"],
                           16, bias=d["bias"])
        assert np.array_equal(y1.cpu().numpy()[0], g.y_q[m])


def test_deterministic_and_guard_bytes():
    mq, torch = _mq(), _torch()
    ld = wl.make_layer("guard", wl.Layer("x", 130, 512, 140, out_bits=16))
    g, d = gpu_layer(ld, keep_device=True)
    M, N = 130, 140
    for path in (mq.PATH_PREFILL, mq.PATH_GENERIC):
        buf = torch.full((M * N + 2 * 4096,), 0x5A5A, dtype=torch.int16, device="cuda")
        y = buf[4096:4096 + M * N].view(M, N)
        for _ in range(3):
            mq.mq_qlinear(d["a_q"], d["w_q"], 8, d["w_scale"], d["w_colsum"], d["a_scale"],
                          d["a_zp"], d["out_scale"], d["out_zp"], 16, bias=d["bias"], out=y,
                          path=path)
            torch.cuda.synchronize()
            assert np.array_equal(y.cpu().numpy(), g.y_q)
        host = buf.cpu().numpy()
        assert np.all(host[:4096] == 0x5A5A) and np.all(host[4096 + M * N:] == 0x5A5A)
    for Mdec in (1, 16):
        buf = torch.full((Mdec * N + 2 * 4096,), 0x5A5A, dtype=torch.int16, device="cuda")
        y = buf[4096:4096 + Mdec * N].view(Mdec, N)
        mq.mq_qlinear(d["a_q"][:Mdec].contiguous(), d["w_q"], 8, d["w_scale"], d["w_colsum"],
                      d["a_scale"], d["a_zp"], d["out_scale"], d["out_zp"], 16, bias=d["bias"],
                      out=y, path=mq.PATH_DECODE)
        torch.cuda.synchronize()
        assert np.array_equal(y.cpu().numpy(), g.y_q[:Mdec])
        host = buf.cpu().numpy()
        assert np.all(host[:4096] == 0x5A5A) and np.all(host[4096 + Mdec * N:] == 0x5A5A)


def test_zero_input_and_saturation():
    mq, torch = _mq(), _torch()
    dev = torch.device("cuda", 0)
    rng = np.random.default_rng(31)
    M, K, N = 40, 256, 96
    w = torch.from_numpy((rng.standard_normal((N, K)) * 0.02).astype(np.float32)).to(dev)
    for w_bits in (8, 4):
        wq, ws, cs = mq.mq_pack_weights(w, w_bits)
        a_scale, a_zp = mq.mq_act_params(-3.0, 5.0, 8)
        a_q = mq.mq_quantize_act(torch.zeros((M, K), device=dev), a_scale, a_zp, 8)
        assert bool((a_q == a_zp).all())
        for out_bits, zp in ((8, -37), (16, 1234)):
            for path in (mq.PATH_PREFILL, mq.PATH_GENERIC, mq.PATH_DECODE):
                a_use = a_q[:16].contiguous() if path == mq.PATH_DECODE else a_q
                y = mq.mq_qlinear(a_use, wq, w_bits, ws, cs, a_scale, a_zp, 0.01, zp, out_bits,
                                  path=path)
                assert bool((y == zp).all())
        # vanishing output scale: outputs are the grid ends by the sign of c
        a_q = torch.from_numpy(rng.integers(-128, 128, (M, K)).astype(np.int8)).to(dev)
        y = mq.mq_qlinear(a_q, wq, w_bits, ws, cs, 0.1, 3, 1e-30, 5, 16).cpu().numpy()
        wi = (wq.cpu().numpy() if w_bits == 8 else
              oracle.int_matmul(np.eye(K, dtype=np.int8), wq.cpu().numpy(), 4).T)
        c = (a_q.cpu().numpy().astype(np.int64) - 3) @ np.asarray(wi, np.int64).T
        assert np.array_equal(y.astype(np.int64), np.where(c > 0, 32767, np.where(c < 0, -32768, 5)))


@pytest.mark.parametrize("w_bits", [8, 4])
def test_extreme_accumulators_at_max_k(w_bits):
    # K = 65536 with A = -128 everywhere and weights at the grid ends: the
    # largest accumulators the format allows
    mq, torch = _mq(), _torch()
    dev = torch.device("cuda", 0)
    K, N = 65536, 32
    Q = 127 if w_bits == 8 else 7
    wf = np.full((N, K), 0.01, np.float32)
    wf[1::2] = -0.01
    w = torch.from_numpy(wf).to(dev)
    wq, ws, cs = mq.mq_pack_weights(w, w_bits)
    o_wq, o_ws, o_cs = oracle.pack_weights(wf, w_bits)
    assert np.array_equal(wq.cpu().numpy(), o_wq) and np.array_equal(cs.cpu().numpy(), o_cs)
    for M, path in ((3, mq.PATH_DECODE), (1, mq.PATH_DECODE), (20, mq.PATH_PREFILL),
                    (3, mq.PATH_GENERIC)):
        a = np.full((M, K), -128, np.int8)
        a[M // 2] = 127 if M > 1 else -128
        a_q = torch.from_numpy(a).to(dev)
        for a_zp, out_scale in ((0, 10.0), (-128, 1e-4), (127, 1.0)):
            y = mq.mq_qlinear(a_q, wq, w_bits, ws, cs, 0.5, a_zp, out_scale, 0, 16, path=path)
            ref = oracle.qlinear(a, o_wq, w_bits, o_ws, 0.5, a_zp, out_scale, 0, 16)
            assert np.array_equal(y.cpu().numpy(), ref), (M, path, a_zp)


def _pack_int4(codes):
    """Two's-complement nibbles, the even k in the low nibble (the packed
    int4 layout), written out independently of both pipelines."""
    lo = codes[:, 0::2].astype(np.int64) & 0xF
    hi = codes[:, 1::2].astype(np.int64) & 0xF
    return (lo | (hi << 4)).astype(np.uint8)


@pytest.mark.parametrize("tile", list(range(6)))
@pytest.mark.parametrize("asym", [False, True])
@pytest.mark.parametrize("w_bits", [8, 4])
def test_prefill_epilogue_forms(tile, asym, w_bits):
    """Every epilogue form of every prefill tile: per-column rescale factors
    spread over 8 decades (shifts from 0 to 64 over the output scales, so
    one tile mixes columns with and without the pre-shift), int8 and int16
    outputs, N giving staged stores (256) and a ragged last tile (260); N %
    4 != 0 (258) takes the generic kernel, whose results must agree too."""
    mq, torch = _mq(), _torch()
    dev = torch.device("cuda", 0)
    rng = np.random.default_rng(int(tile) * 4 + asym * 2 + (w_bits == 4))
    path = mq.prefill_tile_path(tile)
    qw = 128 if w_bits == 8 else 8
    M, K = 300, 512
    a = rng.integers(-128, 128, (M, K)).astype(np.int8)
    g_a = torch.from_numpy(a).to(dev)
    rs = mq.mq_act_rowsum(g_a)
    for N in (256, 260, 258):
        codes = rng.integers(-qw, qw, (N, K))
        wq = codes.astype(np.int8) if w_bits == 8 else _pack_int4(codes)
        cs = codes.sum(axis=1).astype(np.int32)
        zw = rng.integers(-qw, qw, N).astype(np.int32) if asym else None
        ws = (10.0 ** rng.uniform(-7, 1, N)).astype(np.float32)
        bias = (rng.standard_normal(N) * 0.5).astype(np.float32)
        g = [torch.from_numpy(v).to(dev) for v in (wq, ws, cs, bias)]
        for out_bits, out_scale, zp in ((8, 0.05, -7), (16, 0.002, 1234), (16, 30.0, -3),
                                        (16, 1e-10, 0)):
            if asym:
                y = mq.mq_qlinear_asym(g_a, rs, g[0], w_bits, g[1], torch.from_numpy(zw).to(dev),
                                       g[2], 0.02, 5, out_scale, zp, out_bits, bias=g[3],
                                       path=path)
            else:
                y = mq.mq_qlinear(g_a, g[0], w_bits, g[1], g[2], 0.02, 5, out_scale, zp,
                                  out_bits, bias=g[3], path=path)
            ref = oracle.qlinear(a, wq, w_bits, ws, 0.02, 5, out_scale, zp, out_bits, bias=bias,
                                 w_zp=zw)
            got = y.cpu().numpy()
            assert np.array_equal(got, ref), (N, out_bits, out_scale, int((got != ref).sum()))


def test_empty_shapes():
    mq, torch = _mq(), _torch()
    dev = torch.device("cuda", 0)
    a = torch.zeros((0, 64), dtype=torch.int8, device=dev)
    wq = torch.zeros((8, 64), dtype=torch.int8, device=dev)
    ws = torch.ones(8, device=dev)
    cs = torch.zeros(8, dtype=torch.int32, device=dev)
    y = mq.mq_qlinear(a, wq, 8, ws, cs, 0.1, 0, 0.1, 0, 8)
    assert tuple(y.shape) == (0, 8)
    q = mq.mq_quantize_act(torch.zeros(0, device=dev), 0.1, 0, 8)
    assert q.numel() == 0


@pytest.mark.parametrize("n", [1, 7, 8, 9, 1000, 4099])
@pytest.mark.parametrize("bits", [8, 16])
def test_quantize_dequant_ragged(n, bits):
    mq, torch = _mq(), _torch()
    rng = np.random.default_rng(n)
    x = (rng.standard_normal(n) * 7).astype(np.float32)
    x[: min(n, 3)] = [np.nan, np.inf, -np.inf][: min(n, 3)]
    alpha, zp = mq.mq_act_params(-20.0, 15.0, bits)
    xt = torch.from_numpy(x).cuda()
    q = mq.mq_quantize_act(xt, alpha, zp, bits).cpu().numpy()
    assert np.array_equal(q, oracle.quantize_act(x, alpha, zp, bits))
    y = mq.mq_dequant(torch.from_numpy(q).cuda(), alpha, zp).cpu().numpy()
    assert np.array_equal(y.view(np.uint32), oracle.dequant(q, alpha, zp).view(np.uint32))
    # unaligned views take the scalar kernels
    xb = torch.from_numpy(np.concatenate([[0.0], x]).astype(np.float32)).cuda()[1:]
    q2 = mq.mq_quantize_act(xb, alpha, zp, bits).cpu().numpy()
    assert np.array_equal(q2, q)


@pytest.mark.parametrize("bits", [8, 16])
@pytest.mark.parametrize("alpha", [0.1, 0.0373, 0.5, 3.0e-3, 1.7e-30, 2.5e37])
def test_quantize_near_rounding_ties(bits, alpha):
    """Inputs within a few ulp of (n + 1/2) * alpha, where the quotient's
    rounding decides the code: every lane must match the correctly rounded
    division, including the lanes that fall back to it, and an alpha whose
    reciprocal would be subnormal."""
    mq, torch = _mq(), _torch()
    alpha = np.float32(alpha)
    qmax = (1 << (bits - 1)) - 1
    n = np.arange(-qmax - 3, qmax + 3, max(1, (2 * qmax) // 509), dtype=np.float64)
    with np.errstate(over="ignore"):  # the largest alpha overflows to +-inf at the ends
        centers = ((n + 0.5) * np.float64(alpha)).astype(np.float32)
    xs = [centers]
    for direction in (np.inf, -np.inf):
        cur = centers
        for _ in range(8):
            cur = np.nextafter(cur, np.float32(direction))
            xs.append(cur)
    x = np.concatenate(xs).astype(np.float32)
    zp = 3
    got = mq.mq_quantize_act(torch.from_numpy(x).cuda(), float(alpha), zp, bits).cpu().numpy()
    assert np.array_equal(got, oracle.quantize_act(x, float(alpha), zp, bits))


def test_fold_acts_matches_oracle():
    mq, torch = _mq(), _torch()
    rng = np.random.default_rng(41)
    x = rng.standard_normal((33, 300)).astype(np.float32)
    s = np.exp(rng.uniform(np.log(0.5), np.log(2), 300)).astype(np.float32)
    got = mq.mq_fold_acts(torch.from_numpy(x).cuda(), torch.from_numpy(s).cuda()).cpu().numpy()
    assert np.array_equal(got.view(np.uint32), oracle.fold_acts(x, s).view(np.uint32))


# ---------------------------------------------------------------------------
# full-size workloads: every intermediate and every output in full
# ---------------------------------------------------------------------------
FULL = [(w.name, l.name) for w in wl.WORKLOADS.values() for l in w.layers]


@pytest.mark.parametrize("case", FULL, ids=lambda c: f"{c[0]}-{c[1]}")
def test_full_size_parity(case):
    workload, name = case
    ld = wl.make_layer(workload, next(l for l in wl.WORKLOADS[workload].layers
                                      if l.name == name))
    L = ld.layer
    ws = None
    nbytes = _mq().mq_qlinear_workspace_bytes(L.M, L.K, L.N, L.w_bits, L.out_bits)
    if nbytes:  # the layer splits K when given a workspace: take that path
        ws = _torch().zeros(nbytes, dtype=_torch().uint8, device="cuda")
    print(f"full-size {workload}/{name} M={L.M} K={L.K} N={L.N} split_ws={nbytes}", flush=True)
    g = gpu_layer(ld, workspace=ws)
    o = oracle_layer(ld)
    assert_same(g, o)
