"""GPU parity of mq_qlinear_group (linears that read one activation input,
one launch on the prefill path) against the oracle, one linear at a time,
and against separate mq_qlinear calls: bit-exact on every tile, ragged and
empty linears, int4 and asymmetric weights, and the per-linear fallback
paths (decode-sized M, shapes the tuned kernels do not take).
"""
import numpy as np
import pytest

import oracle
from paper_2408_13933_amd import workloads as wl

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


def _make_group(seed, M, K, Ns, w_bits, asym, biases):
    """Random codes and constants for a group of linears on one input."""
    rng = np.random.default_rng(seed)
    qw = 128 if w_bits == 8 else 8
    a = rng.integers(-128, 128, (M, K)).astype(np.int8)
    parts = []
    for i, N in enumerate(Ns):
        codes = rng.integers(-qw, qw, (N, K))
        wq = codes.astype(np.int8) if w_bits == 8 else _pack_int4(codes)
        parts.append(dict(
            wq=wq, cs=codes.sum(axis=1).astype(np.int32),
            ws=(10.0 ** rng.uniform(-5, -2, N)).astype(np.float32),
            zw=rng.integers(-qw, qw, N).astype(np.int32) if asym else None,
            bias=(rng.standard_normal(N) * 0.5).astype(np.float32) if biases[i] else None,
            out_scale=float(10.0 ** rng.uniform(-3, -1)), out_zp=int(rng.integers(-20, 20))))
    return a, parts


def _run(a, parts, w_bits, out_bits, a_scale, a_zp, path):
    mq, torch = _mq(), _torch()
    dev = torch.device("cuda", 0)
    g_a = torch.from_numpy(a).to(dev)
    asym = parts[0]["zw"] is not None
    rs = mq.mq_act_rowsum(g_a) if asym else None
    lin = []
    for p in parts:
        d = dict(w_q=torch.from_numpy(p["wq"]).to(dev), w_scale=torch.from_numpy(p["ws"]).to(dev),
                 w_colsum=torch.from_numpy(p["cs"]).to(dev), out_scale=p["out_scale"],
                 out_zp=p["out_zp"])
        if p["zw"] is not None:
            d["w_zp"] = torch.from_numpy(p["zw"]).to(dev)
        if p["bias"] is not None:
            d["bias"] = torch.from_numpy(p["bias"]).to(dev)
        lin.append(d)
    ys = mq.mq_qlinear_group(g_a, lin, w_bits, a_scale, a_zp, out_bits, a_rowsum=rs, path=path)
    # the same linears one call at a time
    single = []
    for d in lin:
        if asym:
            y = mq.mq_qlinear_asym(g_a, rs, d["w_q"], w_bits, d["w_scale"], d["w_zp"],
                                   d["w_colsum"], a_scale, a_zp, d["out_scale"], d["out_zp"],
                                   out_bits, bias=d.get("bias"))
        else:
            y = mq.mq_qlinear(g_a, d["w_q"], w_bits, d["w_scale"], d["w_colsum"], a_scale, a_zp,
                              d["out_scale"], d["out_zp"], out_bits, bias=d.get("bias"))
        single.append(y.cpu().numpy())
    return [y.cpu().numpy() for y in ys], single


GROUP_CASES = [
    # M, K, Ns, w_bits, out_bits, asym, biases
    (300, 512, (2048, 256, 256), 8, 16, False, (True, False, True)),  # q/k/v-shaped, ragged M
    (257, 1024, (1100, 1028), 8, 8, False, (False, True)),             # gate/up-shaped, ragged N
    (130, 640, (384, 260, 4, 132), 4, 16, False, (True, True, False, True)),
    (200, 768, (520, 264), 8, 16, True, (True, False)),
    (96, 1024, (300, 40), 4, 8, True, (False, False)),
]


@pytest.mark.parametrize("case", GROUP_CASES, ids=lambda c: f"{c[0]}x{c[1]}x{'+'.join(map(str, c[2]))}-w{c[3]}o{c[4]}{'a' if c[5] else ''}")
def test_group_matches_oracle(case):
    M, K, Ns, w_bits, out_bits, asym, biases = case
    a, parts = _make_group(hash(case) % 2**32, M, K, Ns, w_bits, asym, biases)
    a_scale, a_zp = 0.03, -3
    got, single = _run(a, parts, w_bits, out_bits, a_scale, a_zp, _mq().PATH_AUTO)
    for i, p in enumerate(parts):
        ref = oracle.qlinear(a, p["wq"], w_bits, p["ws"], a_scale, a_zp, p["out_scale"],
                             p["out_zp"], out_bits, bias=p["bias"], w_zp=p["zw"])
        assert np.array_equal(got[i], ref), (i, int((got[i] != ref).sum()))
        assert np.array_equal(single[i], ref), i


@pytest.mark.parametrize("tile", list(range(6)))
def test_group_every_tile(tile):
    """One launch on each prefill tile (forced): the same bits as the
    separate calls."""
    mq = _mq()
    a, parts = _make_group(tile, 264, 1024, (520, 132, 260), 8, False, (True, False, True))
    got, single = _run(a, parts, 8, 16, 0.02, 5, mq.prefill_tile_path(tile))
    for g, s in zip(got, single):
        assert np.array_equal(g, s)


@pytest.mark.parametrize("M,K,path", [(8, 512, 0), (1, 1024, 0), (40, 100, 0), (64, 512, 3)],
                         ids=["decode-M8", "gemv-M1", "K100-generic", "path-generic"])
def test_group_per_linear_paths(M, K, path):
    """Shapes the grouped launch does not take run linear by linear on the
    path mq_qlinear would take: same bits."""
    a, parts = _make_group(M * 7 + K, M, K, (136, 40, 264), 8, False, (True, True, False))
    got, single = _run(a, parts, 8, 8, 0.05, 1, path)
    for i, p in enumerate(parts):
        ref = oracle.qlinear(a, p["wq"], 8, p["ws"], 0.05, 1, p["out_scale"], p["out_zp"], 8,
                             bias=p["bias"])
        assert np.array_equal(got[i], ref) and np.array_equal(single[i], ref), i


def test_group_with_an_empty_linear():
    """A linear with N = 0 has nothing to do; the others are computed."""
    mq, torch = _mq(), _torch()
    a, parts = _make_group(5, 200, 512, (260, 1, 132), 8, False, (True, False, True))
    parts[1] = dict(parts[1], wq=parts[1]["wq"][:0], cs=parts[1]["cs"][:0],
                    ws=parts[1]["ws"][:0], bias=None)
    got, single = _run(a, parts, 8, 8, 0.05, 0, mq.PATH_AUTO)
    assert got[1].shape == (200, 0)
    for i in (0, 2):
        assert np.array_equal(got[i], single[i])


@pytest.mark.parametrize("workload,names", [
    ("gemma2b_w8a8", ("gate_proj", "up_proj")),
    ("block_w8a8_tinyllama_s1024", ("q_proj", "k_proj", "v_proj")),
])
def test_group_full_size_layers(workload, names):
    """The workloads' linears that share an input, at full size, grouped:
    every output equal to that of the separate calls (which the full-size
    parity tests compare with the oracle)."""
    mq, torch = _mq(), _torch()
    dev = torch.device("cuda", 0)
    layers = [next(l for l in wl.WORKLOADS[workload].layers if l.name == n) for n in names]
    lds = [wl.make_layer(workload, l) for l in layers]
    # the linears of one group read one input: the first layer's codes
    a_scale, a_zp = mq.mq_act_params(*lds[0].act_range, 8)
    g_a = mq.mq_quantize_act(torch.from_numpy(lds[0].x).to(dev), a_scale, a_zp, 8)
    lin, single = [], []
    for l, ld in zip(layers, lds):
        wq, ws, cs = mq.mq_pack_weights(torch.from_numpy(ld.w).to(dev), l.w_bits)
        o_scale, o_zp = mq.mq_act_params(*ld.out_range, l.out_bits)
        bias = torch.from_numpy(ld.bias).to(dev) if ld.bias is not None else None
        d = dict(w_q=wq, w_scale=ws, w_colsum=cs, out_scale=o_scale, out_zp=o_zp)
        if bias is not None:
            d["bias"] = bias
        lin.append(d)
        single.append(mq.mq_qlinear(g_a, wq, l.w_bits, ws, cs, a_scale, a_zp, o_scale, o_zp,
                                     l.out_bits, bias=bias))
    got = mq.mq_qlinear_group(g_a, lin, layers[0].w_bits, a_scale, a_zp, layers[0].out_bits)
    for g, s in zip(got, single):
        assert torch.equal(g, s)
