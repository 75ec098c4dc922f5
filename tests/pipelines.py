"""The two pipelines the parity tests compare, step for step.

``gpu_layer`` drives libmq.so through its Python binding (every step a HIP
kernel); ``oracle_layer`` drives the CPU oracle.  Both start from the same
seeded fp32 tensors and static float ranges (paper_2408_13933_amd.workloads)
and derive every scale, zero-point and integer on their own side.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

import oracle
from paper_2408_13933_amd.workloads import LayerData


@dataclasses.dataclass
class LayerResult:
    a_scale: float
    a_zp: int
    out_scale: float
    out_zp: int
    a_q: np.ndarray
    w_q: np.ndarray
    w_scale: np.ndarray
    w_colsum: np.ndarray
    w_hat: Optional[np.ndarray]
    y_q: np.ndarray
    y: np.ndarray
    w_zp: Optional[np.ndarray] = None      # asymmetric weights only
    a_rowsum: Optional[np.ndarray] = None  # asymmetric weights only


def oracle_layer(ld: LayerData, rows=None, nthreads=None) -> LayerResult:
    L = ld.layer
    w_hat = oracle.fold_weights(ld.w, ld.s) if ld.s is not None else None
    w_in = w_hat if w_hat is not None else ld.w
    zw = None
    if L.asym:
        wq, ws, zw, cs = oracle.pack_weights_asym(w_in, L.w_bits, per_tensor=L.per_tensor)
    else:
        wq, ws, cs = oracle.pack_weights(w_in, L.w_bits)
    a_scale, a_zp = oracle.act_params(*ld.act_range, L.a_bits)
    out_scale, out_zp = oracle.act_params(*ld.out_range, L.out_bits)
    x = ld.x if rows is None else ld.x[rows]
    a_q = oracle.quantize_act(x, a_scale, a_zp, L.a_bits)
    y_q = oracle.qlinear(a_q, wq, L.w_bits, ws, a_scale, a_zp, out_scale, out_zp, L.out_bits,
                         bias=ld.bias, nthreads=nthreads, w_zp=zw)
    y = oracle.dequant(y_q, out_scale, out_zp)
    rs = oracle.act_rowsum(a_q) if L.asym else None
    return LayerResult(a_scale, a_zp, out_scale, out_zp, a_q, wq, ws, cs, w_hat, y_q, y, zw, rs)


def gpu_layer(ld: LayerData, path: int = 0, keep_device=False, workspace=None):
    import torch
    import paper_2408_13933_amd as mq

    L = ld.layer
    dev = torch.device("cuda", 0)
    x = torch.from_numpy(ld.x).to(dev)
    w = torch.from_numpy(ld.w).to(dev)
    w_hat = None
    if ld.s is not None:
        s = torch.from_numpy(ld.s).to(dev)
        w_hat = mq.mq_fold_weights(w, s)
    bias = torch.from_numpy(ld.bias).to(dev) if ld.bias is not None else None
    a_scale, a_zp = mq.mq_act_params(*ld.act_range, L.a_bits)
    out_scale, out_zp = mq.mq_act_params(*ld.out_range, L.out_bits)
    a_q = mq.mq_quantize_act(x, a_scale, a_zp, L.a_bits)
    w_in = w_hat if w_hat is not None else w
    zw = rs = None
    if L.asym:
        wq, ws, zw, cs = mq.mq_pack_weights_asym(w_in, L.w_bits, per_tensor=L.per_tensor)
        rs = mq.mq_act_rowsum(a_q)
        y_q = mq.mq_qlinear_asym(a_q, rs, wq, L.w_bits, ws, zw, cs, a_scale, a_zp, out_scale,
                                 out_zp, L.out_bits, bias=bias, path=path, workspace=workspace)
    elif L.a_bits == 16:
        wq, ws, cs = mq.mq_pack_weights(w_in, L.w_bits)
        y_q = mq.mq_qlinear_a16(a_q, wq, L.w_bits, ws, cs, a_scale, a_zp, out_scale, out_zp,
                                L.out_bits, bias=bias, path=path)
    else:
        wq, ws, cs = mq.mq_pack_weights(w_in, L.w_bits)
        y_q = mq.mq_qlinear(a_q, wq, L.w_bits, ws, cs, a_scale, a_zp, out_scale, out_zp,
                            L.out_bits, bias=bias, path=path, workspace=workspace)
    y = mq.mq_dequant(y_q, out_scale, out_zp)
    torch.cuda.synchronize()
    res = LayerResult(a_scale, a_zp, out_scale, out_zp, a_q.cpu().numpy(), wq.cpu().numpy(),
                      ws.cpu().numpy(), cs.cpu().numpy(),
                      None if w_hat is None else w_hat.cpu().numpy(), y_q.cpu().numpy(),
                      y.cpu().numpy(), None if zw is None else zw.cpu().numpy(),
                      None if rs is None else rs.cpu().numpy())
    if keep_device:
        return res, dict(a_q=a_q, w_q=wq, w_scale=ws, w_colsum=cs, bias=bias, a_scale=a_scale,
                         a_zp=a_zp, out_scale=out_scale, out_zp=out_zp, w_zp=zw, a_rowsum=rs)
    return res


def assert_same(g: LayerResult, o: LayerResult, rows=None, check_weights=True):
    """Bit-exact integer parity, exact scales; dequant within 1e-6 relative."""
    assert (g.a_scale, g.a_zp) == (o.a_scale, o.a_zp), "activation format differs"
    assert (g.out_scale, g.out_zp) == (o.out_scale, o.out_zp), "output format differs"
    if check_weights:
        if o.w_hat is not None:
            assert np.array_equal(g.w_hat.view(np.uint32), o.w_hat.view(np.uint32)), "fold differs"
        assert np.array_equal(g.w_scale.view(np.uint32), o.w_scale.view(np.uint32)), "w_scale"
        assert np.array_equal(g.w_q, o.w_q), "packed weights differ"
        assert np.array_equal(g.w_colsum, o.w_colsum), "column sums differ"
        if o.w_zp is not None:
            assert np.array_equal(g.w_zp, o.w_zp), "weight zero-points differ"
    ga = g.a_q if rows is None else g.a_q[rows]
    assert np.array_equal(ga, o.a_q), "quantized activations differ"
    if o.a_rowsum is not None:
        gr = g.a_rowsum if rows is None else g.a_rowsum[rows]
        assert np.array_equal(gr, o.a_rowsum), "activation row sums differ"
    gy = g.y_q if rows is None else g.y_q[rows]
    if not np.array_equal(gy, o.y_q):
        bad = np.argwhere(gy != o.y_q)
        m, n = bad[0]
        raise AssertionError(f"{len(bad)} outputs differ; first at ({m},{n}): "
                             f"gpu {gy[m, n]} oracle {o.y_q[m, n]}")
    gf = g.y if rows is None else g.y[rows]
    denom = np.maximum(np.abs(o.y), np.float32(1e-30))
    assert np.all(np.abs(gf - o.y) <= 1e-6 * denom), "dequantized outputs differ"


# ---------------------------------------------------------------------------
# the decoder block through the oracle (the same stages as
# paper_2408_13933_amd.block, each computed by the oracle's own functions
# from the same float inputs and static ranges)

def block_oracle(data, nthreads=None):
    from paper_2408_13933_amd import block as blk
    from paper_2408_13933_amd import workloads as wl

    d = wl.BLOCK_DIMS
    T, H, G, D = data.T, d["heads"], d["kv_heads"], d["head_dim"]
    f = blk.formats(data.ranges, oracle.act_params)
    out = {"h0": oracle.quantize_act(data.h0, *f["h0"], 16)}
    packed = {n: oracle.pack_weights(w, 8) for n, w in data.w.items()}

    def linear(stage):
        name, src = blk.LINEARS[stage]
        wq, ws, _ = packed[name]
        out[stage] = oracle.qlinear(out[src], wq, 8, ws, *f[src], *f[stage],
                                    blk.STAGE_BITS[stage], nthreads=nthreads)

    out["x1"] = oracle.rmsnorm(out["h0"], *f["h0"], data.gamma1, d["eps"], *f["x1"], 8)
    for s in ("q", "k", "v"):
        linear(s)
    out["qr"] = oracle.rope(out["q"], H, *f["q"], *f["qr"], 16, base=d["rope_base"])
    out["kr"] = oracle.rope(out["k"], G, *f["k"], *f["kr"], 8, base=d["rope_base"])
    qh = np.ascontiguousarray(out["qr"].reshape(T, H, D).transpose(1, 0, 2))
    kh = np.ascontiguousarray(out["kr"].reshape(T, G, D).transpose(1, 0, 2))
    out["scores"] = oracle.attn_matmul(qh, kh, *f["qr"], *f["kr"], *f["scores"], 16,
                                       nthreads=nthreads)
    sa, sz = f["scores"]
    out["probs"] = oracle.softmax(out["scores"].reshape(H * T, T), sa / D ** 0.5, sz,
                                  *f["probs"], 16, causal_period=T).reshape(H, T, T)
    vt = np.ascontiguousarray(out["v"].T).reshape(G, D, T)
    ctx = oracle.attn_matmul(out["probs"], vt, *f["probs"], *f["v"], *f["ctx"], 8,
                             nthreads=nthreads)
    out["ctx"] = np.ascontiguousarray(ctx.transpose(1, 0, 2).reshape(T, H * D))
    linear("o")
    out["h1"] = oracle.add_requant(out["h0"], *f["h0"], out["o"], *f["o"], *f["h1"], 16)
    out["x2"] = oracle.rmsnorm(out["h1"], *f["h1"], data.gamma2, d["eps"], *f["x2"], 8)
    linear("gate")
    linear("up")
    lut = oracle.lut_build(oracle.LUT_SILU, *f["gate"], *f["silu"], 16)
    out["silu"] = lut[out["gate"].astype(np.int64) + 32768]
    out["mul"] = oracle.mul_requant(out["silu"], *f["silu"], out["up"], *f["up"], *f["mul"], 8)
    linear("down")
    out["h2"] = oracle.add_requant(out["h1"], *f["h1"], out["down"], *f["down"], *f["h2"], 16)
    return out, f
