"""Seeded synthetic workloads for the integer-only linear layer.

This module only draws random numbers and describes shapes.  It holds none
of the quantization arithmetic: it hands both the HIP library and the CPU
oracle the same fp32 tensors and the same static float ranges, and each
side derives scales, zero-points and integer codes on its own.

Recipe (stand-in for the paper's calibration and evaluation data, which
are not used): layer shapes are those of the small Llama-style and
Gemma-2B-style models the paper deploys; activations carry a few
large-magnitude channels, the property that makes per-tensor activation
quantization hard (Section 3.2).

* activations X_hat [M][K] fp32: N(0, 1) with 4 outlier channels scaled by
  20 (TinyLlama-shaped layers), or N(0, 1) with max(4, round(0.01 K))
  channels drawn from Student-t(3) instead (Gemma-shaped layers).  These
  are the activations as they reach the layer, i.e. already in the
  smoothed domain of Eq.(1).
* weights W [N][K] fp32: N(0, 0.02^2), before folding.
* smoothing vector s [K] (only where a layer folds one): exp(U(ln 0.5,
  ln 2)); the fold W_hat = W diag(s) is done by the code under test.
* asymmetric-weight layers (Section 5.1 quantizes weights asymmetrically
  per channel): each weight row gets its own mean, W[n] += mu_n with mu_n
  ~ U(-2, 2) * 0.02, so row ranges are off-centre and the zero-points
  spread over the grid instead of sitting near 0.
* bias [N] fp32: N(0, 0.01^2) where the layer has one.
* static activation range: min and max of X_hat (a plain data statistic).
* static output range: the layer output has standard deviation
  sigma_y = 0.02 * rms_m sqrt(sum_k (X_hat[m,k] s[k])^2) under this recipe;
  the range is [-4.5 sigma_y - 3 sigma_b, 5.5 sigma_y + 3 sigma_b], skewed
  so the output zero-point is not zero and a few outputs saturate.  With
  row means mu_n, sigma_y^2 adds mean_n(mu_n^2) * mean_m((sum_k X_hat s)^2).
"""
from __future__ import annotations

import dataclasses
import zlib
from typing import Optional

import numpy as np

W_STD = 0.02
B_STD = 0.01


@dataclasses.dataclass(frozen=True)
class Layer:
    name: str
    M: int
    K: int
    N: int
    w_bits: int = 8          # 8 or 4
    out_bits: int = 8        # 8 or 16
    bias: bool = True
    act: str = "outlier"     # "outlier" | "student_t"
    smooth: Optional[str] = None   # name of the smoothing vector folded in
    smooth_len: int = 0            # length of that vector
    asym: bool = False             # asymmetric weights
    per_tensor: bool = False       # one weight range per tensor (asym only)
    a_bits: int = 8                # activation codes: 8, or 16 (W8A16)

    @property
    def ops(self) -> int:
        return 2 * self.M * self.N * self.K

    def alg_bytes(self) -> int:
        """Minimum bytes one qlinear call moves: A, W, Y and per-column params."""
        w = self.N * self.K * self.w_bits // 8
        a = self.M * self.K * self.a_bits // 8
        y = self.M * self.N * self.out_bits // 8
        params = self.N * (8 + (4 if self.bias else 0))
        if self.asym:  # weight zero-points and activation row sums
            params += self.N * 4 + self.M * 4
        return w + a + y + params


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    description: str
    layers: tuple


def _tinyllama_block(M: int, asym: bool = False, a_bits: int = 8):
    L = dict(out_bits=16, bias=False, asym=asym, a_bits=a_bits)
    # asymmetric (Section 5.1 W8A8): one weight range per tensor except the
    # MLP down projection, which keeps one per output channel
    T = dict(per_tensor=asym)
    return (
        Layer("q_proj", M, 2048, 2048, smooth="attn_norm", smooth_len=2048, **L, **T),
        Layer("k_proj", M, 2048, 256, smooth="attn_norm", smooth_len=2048, **L, **T),
        Layer("v_proj", M, 2048, 256, smooth="attn_norm", smooth_len=2048, **L, **T),
        Layer("o_proj", M, 2048, 2048, smooth="v_to_o", smooth_len=256, **L, **T),
        Layer("gate_proj", M, 2048, 5632, smooth="mlp_norm", smooth_len=2048, **L, **T),
        Layer("up_proj", M, 2048, 5632, smooth="mlp_norm", smooth_len=2048, **L, **T),
        Layer("down_proj", M, 5632, 2048, smooth="up_to_down", smooth_len=5632, **L),
    )


def _tinyllama_block_fused(M: int):
    # q/k/v as one 2560-channel GEMM and gate/up as one 11264-channel GEMM,
    # each with one joint output range (the fused layers share a per-tensor
    # output format)
    L = dict(out_bits=16, bias=False)
    return (
        Layer("qkv_proj", M, 2048, 2560, smooth="attn_norm", smooth_len=2048, **L),
        Layer("o_proj", M, 2048, 2048, smooth="v_to_o", smooth_len=256, **L),
        Layer("gate_up_proj", M, 2048, 11264, smooth="mlp_norm", smooth_len=2048, **L),
        Layer("down_proj", M, 5632, 2048, smooth="up_to_down", smooth_len=5632, **L),
    )


WORKLOADS = {
    "decode_w8a8_m16": Workload(
        "decode_w8a8_m16",
        "single W8A8 qlinear, M=16, K=2048, N=2048, int8 out, bias",
        (Layer("linear", 16, 2048, 2048),)),
    "prefill_w8a8_tinyllama_m2048": Workload(
        "prefill_w8a8_tinyllama_m2048",
        "TinyLlama-shaped MLP gate/up (M=2048, K=2048, N=5632) and attention "
        "o-proj (M=2048, K=2048, N=2048), W8A8, int8 out, bias",
        (Layer("gate_proj", 2048, 2048, 5632),
         Layer("up_proj", 2048, 2048, 5632),
         Layer("o_proj", 2048, 2048, 2048))),
    "w4a8_down_tinyllama": Workload(
        "w4a8_down_tinyllama",
        "W4A8 down-proj K=5632, N=2048, symmetric per-channel int4, int16 out, "
        "at M=1 (decode) and M=1024 (prefill)",
        (Layer("down_proj_m1", 1, 5632, 2048, w_bits=4, out_bits=16),
         Layer("down_proj_m1024", 1024, 5632, 2048, w_bits=4, out_bits=16))),
    "block_w8a8_tinyllama_s1024": Workload(
        "block_w8a8_tinyllama_s1024",
        "the seven linears of one hidden-2048, 32-head, 4-KV-head, "
        "intermediate-5632 decoder block at batch 1, seq 1024, W8A8 with "
        "folded smoothing vectors, int8 in, int16 out",
        _tinyllama_block(1024)),
    "block_w8a8_fused_tinyllama_s1024": Workload(
        "block_w8a8_fused_tinyllama_s1024",
        "the same decoder block with q/k/v fused into one N=2560 GEMM and gate/up "
        "into one N=11264 GEMM (one output range each)",
        _tinyllama_block_fused(1024)),
    "block_w8a8_asym_tinyllama_s1024": Workload(
        "block_w8a8_asym_tinyllama_s1024",
        "the same decoder block in the paper's main W8A8 setting: asymmetric "
        "weights, one range per tensor except per-channel down_proj",
        _tinyllama_block(1024, asym=True)),
    "block_w8a16_tinyllama_s1024": Workload(
        "block_w8a16_tinyllama_s1024",
        "the same decoder block in the W8A16 comparison setting (Section 5.6): "
        "16-bit activation codes into the seven linears, int8 weights",
        _tinyllama_block(1024, a_bits=16)),
    "w4a8_asym_down_tinyllama": Workload(
        "w4a8_asym_down_tinyllama",
        "the paper's main W4A8 setting on the down-proj K=5632, N=2048: "
        "asymmetric per-channel int4, int16 out, at M=1 and M=1024",
        (Layer("down_proj_m1", 1, 5632, 2048, w_bits=4, out_bits=16, asym=True),
         Layer("down_proj_m1024", 1024, 5632, 2048, w_bits=4, out_bits=16, asym=True))),
    "gemma2b_w8a8": Workload(
        "gemma2b_w8a8",
        "Gemma-2B-shaped W8A8 layers: MLP gate/up K=2048 N=16384 and down "
        "K=16384 N=2048 at M=512, LM head K=2048 N=256000 at M=1 and M=512, "
        "int16 out, heavy-tailed activation channels",
        (Layer("gate_proj", 512, 2048, 16384, out_bits=16, bias=False, act="student_t"),
         Layer("up_proj", 512, 2048, 16384, out_bits=16, bias=False, act="student_t"),
         Layer("down_proj", 512, 16384, 2048, out_bits=16, bias=False, act="student_t"),
         Layer("lm_head_m1", 1, 2048, 256000, out_bits=16, bias=False, act="student_t"),
         Layer("lm_head_m512", 512, 2048, 256000, out_bits=16, bias=False,
               act="student_t"))),
}


def _rng(*keys) -> np.random.Generator:
    seed = [zlib.crc32(str(k).encode()) for k in keys]
    return np.random.default_rng(seed)


def gen_activations(M: int, K: int, act: str, seed_key) -> np.ndarray:
    rng = _rng("act", *seed_key)
    x = rng.standard_normal((M, K), dtype=np.float32)
    if act == "outlier":
        ch = rng.choice(K, min(4, K), replace=False)
        x[:, ch] *= np.float32(20.0)
    elif act == "student_t":
        n_ch = min(K, max(4, int(round(0.01 * K))))
        ch = rng.choice(K, n_ch, replace=False)
        x[:, ch] = rng.standard_t(3.0, size=(M, n_ch)).astype(np.float32)
    else:
        raise ValueError(act)
    return x


def gen_weights(N: int, K: int, seed_key) -> np.ndarray:
    rng = _rng("w", *seed_key)
    w = rng.standard_normal((N, K), dtype=np.float32)
    w *= np.float32(W_STD)
    return w


def gen_row_means(N: int, seed_key) -> np.ndarray:
    rng = _rng("mu", *seed_key)
    return (rng.uniform(-2.0, 2.0, size=N) * W_STD).astype(np.float32)


def gen_bias(N: int, seed_key) -> np.ndarray:
    rng = _rng("b", *seed_key)
    return (rng.standard_normal(N, dtype=np.float32) * np.float32(B_STD)).astype(np.float32)


def gen_smoothing(length: int, seed_key) -> np.ndarray:
    rng = _rng("s", *seed_key)
    return np.exp(rng.uniform(np.log(0.5), np.log(2.0), size=length)).astype(np.float32)


def smoothing_for(layer: Layer, workload: str) -> Optional[np.ndarray]:
    """The per-input-channel smoothing vector folded into this layer, or None.

    The v->o vector has one entry per value channel (4 KV heads x 64); each
    KV head's entries are shared by the 8 query heads of its group, so it is
    repeated along o_proj's 2048 inputs (32 heads x 64).
    """
    if layer.smooth is None:
        return None
    if layer.smooth == "v_to_o" and layer.K == 2048:
        s = gen_smoothing(256, (workload, layer.smooth))
        kv_heads, head_dim, q_heads = 4, 64, 32
        s = s.reshape(kv_heads, 1, head_dim)
        s = np.broadcast_to(s, (kv_heads, q_heads // kv_heads, head_dim)).reshape(-1)
        return np.ascontiguousarray(s, dtype=np.float32)
    return gen_smoothing(layer.K, (workload, layer.smooth))


@dataclasses.dataclass
class LayerData:
    layer: Layer
    x: np.ndarray                  # fp32 [M][K], smoothed-domain activations
    w: np.ndarray                  # fp32 [N][K], before folding
    s: Optional[np.ndarray]        # fp32 [K] or None
    bias: Optional[np.ndarray]     # fp32 [N] or None
    act_range: tuple               # (f_min, f_max) of x
    out_range: tuple               # static output range


def _output_range(x: np.ndarray, s: Optional[np.ndarray], has_bias: bool,
                  mu: Optional[np.ndarray] = None):
    xs = x.astype(np.float64)
    if s is not None:
        xs = xs * s.astype(np.float64)[None, :]
    row_ss = np.einsum("mk,mk->m", xs, xs)
    var_y = W_STD ** 2 * float(np.mean(row_ss))
    if mu is not None:
        var_y += float(np.mean(mu.astype(np.float64) ** 2)) * float(np.mean(xs.sum(axis=1) ** 2))
    sigma_y = float(np.sqrt(var_y))
    sb = 3.0 * B_STD if has_bias else 0.0
    return (float(np.float32(-4.5 * sigma_y - sb)), float(np.float32(5.5 * sigma_y + sb)))


def make_layer(workload: str, layer: Layer, rows: Optional[slice] = None,
               shared_x: Optional[np.ndarray] = None) -> LayerData:
    """Draw one layer's tensors.

    Layers that read the same activation in the model (q/k/v, gate/up) share
    one draw; the M=1 decode variants take row 0 of their prefill partner.
    """
    key_x = _x_key(workload, layer)
    if shared_x is not None:
        x = shared_x
    else:
        x = gen_activations(_x_rows(workload, layer), layer.K, layer.act, key_x)
    x = np.ascontiguousarray(x[: layer.M])
    w = gen_weights(layer.N, layer.K, (workload, _w_name(layer)))
    mu = None
    if layer.asym:
        mu = gen_row_means(layer.N, (workload, _w_name(layer)))
        w += mu[:, None]
    s = smoothing_for(layer, workload)
    bias = gen_bias(layer.N, (workload, _w_name(layer))) if layer.bias else None
    act_range = (float(x.min()), float(x.max()))
    out_range = _output_range(x, s, layer.bias, mu)
    if rows is not None:
        x = np.ascontiguousarray(x[rows])
    return LayerData(layer, x, w, s, bias, act_range, out_range)


def _w_name(layer: Layer) -> str:
    # decode and prefill variants of one layer share the weight matrix
    for suf in ("_m1024", "_m512", "_m1"):
        if layer.name.endswith(suf):
            return layer.name[: -len(suf)]
    return layer.name


def _x_key(workload: str, layer: Layer):
    name = _w_name(layer)
    if name in ("q_proj", "k_proj", "v_proj", "qkv_proj"):
        name = "qkv_in"
    if name in ("gate_proj", "up_proj", "gate_up_proj"):
        name = "mlp_in"
    return (workload, name)


def _x_rows(workload: str, layer: Layer) -> int:
    """Rows to draw so that an M=1 variant reuses row 0 of its prefill twin."""
    wl = WORKLOADS.get(workload)
    if wl is None:
        return layer.M
    base = _w_name(layer)
    return max([l.M for l in wl.layers if _w_name(l) == base] + [layer.M])


def scaled_layer(layer: Layer, M=None, K=None, N=None, name=None) -> Layer:
    """A copy of ``layer`` at another shape (for oracle-sized parity cases)."""
    K2 = layer.K if K is None else K
    return dataclasses.replace(layer, M=layer.M if M is None else M, K=K2,
                               N=layer.N if N is None else N,
                               name=layer.name if name is None else name,
                               smooth_len=K2 if layer.smooth else 0)


# ---------------------------------------------------------------------------
# One whole decoder block (TinyLlama-shaped: hidden 2048, 32 query heads, 4
# key/value heads of 64, feed-forward 5632) on integer codes.  The inputs
# are the block's residual stream, the seven projection matrices and the two
# RMSNorm gains, drawn as above; the static float range of every
# intermediate comes from an fp64 float forward pass of the same block (the
# paper calibrates its static activation ranges on a float model, Section
# 4.2).  The float pass (fp32 products, fp64 elsewhere) is a statistic of
# the synthetic data, like the layer output ranges above: no quantization
# arithmetic happens here.

BLOCK_DIMS = dict(hidden=2048, heads=32, kv_heads=4, head_dim=64, ffn=5632, eps=1e-5,
                  rope_base=10000.0)
BLOCK_LINEARS = (("q_proj", "hidden", "hidden"), ("k_proj", "kv", "hidden"),
                 ("v_proj", "kv", "hidden"), ("o_proj", "hidden", "hidden"),
                 ("gate_proj", "ffn", "hidden"), ("up_proj", "ffn", "hidden"),
                 ("down_proj", "hidden", "ffn"))


@dataclasses.dataclass
class BlockData:
    T: int
    h0: np.ndarray                 # fp32 [T][hidden], residual stream entering the block
    w: dict                        # name -> fp32 [N][K]
    gamma1: np.ndarray             # fp32 [hidden]
    gamma2: np.ndarray
    ranges: dict                   # stage -> (f_min, f_max), static ranges
    floats: Optional[dict] = None  # stage -> float values of the float pass (keep_floats)


def _block_dim(name: str) -> int:
    d = BLOCK_DIMS
    return {"hidden": d["hidden"], "kv": d["kv_heads"] * d["head_dim"], "ffn": d["ffn"]}[name]


def _rope_f64(x: np.ndarray, heads: int, base: float) -> np.ndarray:
    T, HD = x.shape
    D = HD // heads
    xh = x.reshape(T, heads, D)
    inv = base ** (-np.arange(0, D, 2, dtype=np.float64) / D)
    ang = np.arange(T, dtype=np.float64)[:, None] * inv[None, :]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    u, w = xh[..., :D // 2], xh[..., D // 2:]
    return np.concatenate([u * c - w * s, w * c + u * s], axis=-1).reshape(T, HD)


def _rmsnorm_f64(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    return x / np.sqrt(np.mean(x * x, axis=1, keepdims=True) + eps) * g[None, :]


def _range(v: np.ndarray, pad: float = 1.05) -> tuple:
    lo, hi = float(v.min()), float(v.max())
    return (float(np.float32(min(lo, 0.0) * pad)), float(np.float32(max(hi, 0.0) * pad)))


def make_block(T: int, seed: str = "block_tinyllama", keep_floats: bool = False) -> BlockData:
    d = BLOCK_DIMS
    H, G, D, F = d["heads"], d["kv_heads"], d["head_dim"], d["ffn"]
    hid = d["hidden"]
    h0 = gen_activations(T, hid, "outlier", (seed, "h0"))
    w = {n: gen_weights(_block_dim(a), _block_dim(b), (seed, n)) for n, a, b in BLOCK_LINEARS}
    rng = _rng("gamma", seed)
    g1 = rng.uniform(0.5, 1.5, hid).astype(np.float32)
    g2 = rng.uniform(0.5, 1.5, hid).astype(np.float32)
    # float pass: fp32 products (ranges need no more), the rest in fp64
    def mm(x, name):
        return (x.astype(np.float32) @ w[name].T).astype(np.float64)

    r = {}
    h = h0.astype(np.float64)
    r["h0"] = _range(h)
    x1 = _rmsnorm_f64(h, g1.astype(np.float64), d["eps"])
    r["x1"] = _range(x1)
    q, k, v = mm(x1, "q_proj"), mm(x1, "k_proj"), mm(x1, "v_proj")
    r["q"], r["k"], r["v"] = _range(q), _range(k), _range(v)
    qr, kr = _rope_f64(q, H, d["rope_base"]), _rope_f64(k, G, d["rope_base"])
    r["qr"], r["kr"] = _range(qr), _range(kr)
    qh = qr.reshape(T, H, D).transpose(1, 0, 2)
    kh = kr.reshape(T, G, D).transpose(1, 0, 2)
    vh = v.reshape(T, G, D).transpose(1, 0, 2)
    scores = np.stack([qh[h_] @ kh[h_ // (H // G)].T for h_ in range(H)])
    r["scores"] = _range(scores)
    z = scores / np.sqrt(D)
    mask = np.triu(np.ones((T, T), dtype=bool), 1)
    z = np.where(mask[None], -np.inf, z)
    z = z - z.max(axis=2, keepdims=True)
    p = np.exp(z)
    p /= p.sum(axis=2, keepdims=True)
    r["probs"] = (0.0, 1.0)
    ctx = np.stack([p[h_] @ vh[h_ // (H // G)] for h_ in range(H)])  # [H][T][D]
    ctx = ctx.transpose(1, 0, 2).reshape(T, H * D)
    r["ctx"] = _range(ctx)
    o = mm(ctx, "o_proj")
    r["o"] = _range(o)
    h1 = h + o
    r["h1"] = _range(h1)
    x2 = _rmsnorm_f64(h1, g2.astype(np.float64), d["eps"])
    r["x2"] = _range(x2)
    gt, up = mm(x2, "gate_proj"), mm(x2, "up_proj")
    r["gate"], r["up"] = _range(gt), _range(up)
    sg = gt / (1.0 + np.exp(-gt))
    r["silu"] = _range(sg)
    m = sg * up
    r["mul"] = _range(m)
    dn = mm(m, "down_proj")
    r["down"] = _range(dn)
    h2 = h1 + dn
    r["h2"] = _range(h2)
    del F
    floats = None
    if keep_floats:
        floats = dict(h0=h, x1=x1, q=q, k=k, v=v, qr=qr, kr=kr, scores=scores, probs=p, ctx=ctx,
                      o=o, h1=h1, x2=x2, gate=gt, up=up, silu=sg, mul=m, down=dn, h2=h2)
    return BlockData(T, h0, w, g1, g2, r, floats)
