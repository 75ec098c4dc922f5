"""A whole decoder block on the GPU (paper_2408_13933_amd.block) against the
oracle.

test_block_each_stage_from_the_gpu_inputs: every stage recomputed by the
oracle from the GPU's own inputs to that stage.  Stages built from integer
arithmetic and correctly rounded fp64 operations (the linears, the
attention products, the residual adds, RMSNorm, the gated product) must be
bit-exact; the stages through exp, cos and sin (RoPE, softmax, the SiLU
table) may differ by one step only where their fp64 value lies on a
rounding tie (Section 4.1 keeps these operators in higher precision and
fixes no arithmetic inside them).

test_block_chain_drift: the GPU block against the oracle's block run from
the same float inputs; after the first stage that differs at a tie, the
difference can move codes downstream: bounded and reported."""
import numpy as np
import pytest

import oracle

pytestmark = pytest.mark.gpu

TIE_STAGES = ("qr", "kr", "probs", "mul")  # "mul": through the SiLU table


def _equal_but_ties(got, ref, pre, what, max_frac=1e-3):
    """Codes equal except one step where the fp64 value `pre` (in output
    steps, before the zero-point) lies within 1e-9 of a half-integer."""
    got = got.astype(np.int64)
    ref = ref.astype(np.int64)
    f = pre - np.floor(pre)
    tie = np.abs(f - 0.5) < 1e-9
    bad = (got != ref) & ~(tie & (np.abs(got - ref) <= 1))
    assert not np.any(bad), (what, int(bad.sum()), np.argwhere(bad)[:5])
    assert np.mean(got != ref) <= max_frac, (what, float(np.mean(got != ref)))
    return int(np.count_nonzero(got != ref))


def _f32(v):
    return np.float64(np.float32(v))


def _rope_pre(x, heads, ax, zx, ay, base):
    T, HD = x.shape
    D = HD // heads
    xh = (_f32(ax) * (x.astype(np.float64) - zx)).reshape(T, heads, D)
    inv = base ** (-np.arange(0, D, 2, dtype=np.float64) / D)
    ang = np.arange(T, dtype=np.float64)[:, None] * inv[None, :]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    u, w = xh[..., :D // 2], xh[..., D // 2:]
    return np.concatenate([u * c - w * s, w * c + u * s], axis=-1).reshape(T, HD) / _f32(ay)


def _softmax_causal_pre(x, ax, zx, ay, period):
    import torch
    M, K = x.shape
    n = np.minimum(np.arange(M) % period + 1, K)
    mask = np.arange(K)[None, :] < n[:, None]
    xr = np.where(mask, _f32(ax) * (x.astype(np.float64) - zx), -np.inf)
    return torch.softmax(torch.tensor(xr), dim=1).numpy() / _f32(ay)


@pytest.mark.parametrize("T", [128, 200, 1024])
def test_block_each_stage_from_the_gpu_inputs(T):
    import torch

    from paper_2408_13933_amd import block as blk
    from paper_2408_13933_amd import workloads as wl

    data = wl.make_block(T)
    g = blk.BlockGPU(data)
    g.run()
    torch.cuda.synchronize()
    o = {s: t.cpu().numpy() for s, t in g.out.items()}
    f = g.fmt
    assert f == blk.formats(data.ranges, oracle.act_params)
    d = wl.BLOCK_DIMS
    H, G, D = d["heads"], d["kv_heads"], d["head_dim"]
    ties = {}

    packed = {}
    for name, w in data.w.items():
        ref = oracle.pack_weights(w, 8)
        for got, exp in zip(g.w[name], ref):
            assert np.array_equal(got.cpu().numpy(), exp), name
        packed[name] = ref

    def exact(stage, ref):
        assert o[stage].shape == ref.shape and o[stage].dtype == ref.dtype, stage
        n_bad = int(np.count_nonzero(o[stage] != ref))
        assert n_bad == 0, (stage, n_bad)

    def linear(stage):
        name, src = blk.LINEARS[stage]
        wq, ws, _ = packed[name]
        exact(stage, oracle.qlinear(o[src], wq, 8, ws, *f[src], *f[stage],
                                    blk.STAGE_BITS[stage]))

    exact("h0", oracle.quantize_act(data.h0, *f["h0"], 16))
    exact("x1", oracle.rmsnorm(o["h0"], *f["h0"], data.gamma1, d["eps"], *f["x1"], 8))
    for s in ("q", "k", "v"):
        linear(s)
    for s, src, heads, bits in (("qr", "q", H, 16), ("kr", "k", G, 8)):
        ref = oracle.rope(o[src], heads, *f[src], *f[s], bits, base=d["rope_base"])
        pre = _rope_pre(o[src], heads, f[src][0], f[src][1], f[s][0], d["rope_base"])
        ties[s] = _equal_but_ties(o[s], ref, pre, s)
    qh = np.ascontiguousarray(o["qr"].reshape(T, H, D).transpose(1, 0, 2))
    kh = np.ascontiguousarray(o["kr"].reshape(T, G, D).transpose(1, 0, 2))
    ref = oracle.attn_matmul(qh, kh, *f["qr"], *f["kr"], *f["scores"], 16)
    low = np.tril(np.ones((T, T), dtype=bool))  # only the causal triangle is computed
    assert np.array_equal(o["scores"][:, low], ref[:, low]), "scores"
    sa, sz = f["scores"]
    scores = o["scores"].reshape(H * T, T)
    ref = oracle.softmax(scores, sa / D ** 0.5, sz, *f["probs"], 16, causal_period=T)
    pre = _softmax_causal_pre(scores, sa / D ** 0.5, sz, f["probs"][0], T)
    ties["probs"] = _equal_but_ties(o["probs"].reshape(H * T, T), ref, pre, "probs")
    vt = np.ascontiguousarray(o["v"].T).reshape(G, D, T)
    ctx = oracle.attn_matmul(o["probs"], vt, *f["probs"], *f["v"], *f["ctx"], 8)
    exact("ctx", np.ascontiguousarray(ctx.transpose(1, 0, 2).reshape(T, H * D)))
    linear("o")
    exact("h1", oracle.add_requant(o["h0"], *f["h0"], o["o"], *f["o"], *f["h1"], 16))
    exact("x2", oracle.rmsnorm(o["h1"], *f["h1"], data.gamma2, d["eps"], *f["x2"], 8))
    linear("gate")
    linear("up")
    # the SiLU table (built once on the GPU) against the oracle's, then the
    # fused lookup and gated product on the GPU's table
    glut = g.lut.cpu().numpy()
    rlut = oracle.lut_build(oracle.LUT_SILU, *f["gate"], *f["silu"], 16)
    i = np.arange(-32768, 32768)
    v = _f32(f["gate"][0]) * (i - f["gate"][1])
    with np.errstate(over="ignore"):
        pre = v / (1.0 + np.exp(-v)) / _f32(f["silu"][0])
    ties["silu_table"] = _equal_but_ties(glut, rlut, pre, "silu_table")
    silu = glut[o["gate"].astype(np.int64) + 32768]
    exact("mul", oracle.mul_requant(silu, *f["silu"], o["up"], *f["up"], *f["mul"], 8))
    linear("down")
    exact("h2", oracle.add_requant(o["h1"], *f["h1"], o["down"], *f["down"], *f["h2"], 16))
    print(f"T={T}: codes at rounding ties that differ: {ties}")


@pytest.mark.parametrize("T", [128, 200, 1024])
def test_block_chain_drift(T):
    from paper_2408_13933_amd import block as blk
    from paper_2408_13933_amd import workloads as wl
    from tests.pipelines import block_oracle

    data = wl.make_block(T)
    g = blk.BlockGPU(data)
    g.run()
    ref, fmt = block_oracle(data)
    assert fmt == g.fmt
    diverged = None
    drift = {}
    for stage in blk.STAGE_BITS:
        if stage in blk.NOT_STORED:  # fused into the next step
            continue
        got = g.out[stage].cpu().numpy()
        exp = ref[stage]
        if stage == "scores":  # only the causal lower triangle is computed
            low = np.tril(np.ones((T, T), dtype=bool))
            got, exp = got[:, low], exp[:, low]
        assert got.shape == exp.shape and got.dtype == exp.dtype, stage
        diff = got.astype(np.int64) - exp.astype(np.int64)
        n_bad = int(np.count_nonzero(diff))
        if diverged is None:
            if n_bad == 0:
                continue
            # the first difference comes from a tie stage, one step, rare
            assert stage in TIE_STAGES, (stage, n_bad)
            assert np.abs(diff).max() == 1 and n_bad <= max(1, got.size // 100000), (stage, n_bad)
            diverged = stage
        else:
            # downstream of a tie a one-step input change moves a few codes
            # by at most two steps (the stagewise test pins every stage)
            assert n_bad <= got.size // 1000 and np.abs(diff).max() <= 2, (stage, diverged, n_bad)
        drift[stage] = n_bad
    print(f"T={T}: first stage that differs: {diverged}; codes that differ: {drift}")
