"""One decoder block of a Llama-family model on integer codes, every step on
the GPU through the library's entry points (Section 4.1: 8-bit inputs to the
linears, 16-bit activations around the non-linear operators; Section 5.6:
attention products between 16-bit and 8-bit activations).

    x1 = RMSNorm(h0)                  int16 -> int8
    q, k, v = x1 Wq^T, x1 Wk^T, x1 Wv^T    -> int16, int16, int8 (q, k: one launch)
    q, k = RoPE(q), RoPE(k)                -> int16, int8
    s = q k^T per head (grouped keys)      -> int16 scores
    p = causal softmax(s / sqrt(64))       -> int16 probabilities
    c = p v per head                       -> int8 context
    h1 = h0 + c Wo^T                       -> int16
    x2 = RMSNorm(h1)                       -> int8
    g, u = x2 Wg^T, x2 Wu^T                -> int16 (one launch)
    m = SiLU(g) * u                        -> int16 table lookup, int8 product
    h2 = h1 + m Wd^T                       -> int16

Static formats: every intermediate's (alpha, zero-point) comes from its
float range through mq_act_params; the weights are packed on the device
(symmetric per output channel, int8).  `run()` only enqueues kernels on the
current stream (no allocation, no host synchronisation), so it can be
captured in a HIP graph.
"""
from __future__ import annotations

from . import workloads as wl

# stage -> output bit width
STAGE_BITS = dict(h0=16, x1=8, q=16, k=16, v=8, qr=16, kr=8, scores=16, probs=16, ctx=8, o=16,
                  h1=16, x2=8, gate=16, up=16, silu=16, mul=8, down=16, h2=16)
# stages whose codes the GPU block keeps out of memory (fused into the next step)
NOT_STORED = ("silu",)
# stage -> (weight, input stage) of the linears
LINEARS = dict(q=("q_proj", "x1"), k=("k_proj", "x1"), v=("v_proj", "x1"), o=("o_proj", "ctx"),
               gate=("gate_proj", "x2"), up=("up_proj", "x2"), down=("down_proj", "mul"))


def formats(ranges: dict, act_params) -> dict:
    """(alpha, zp) per stage from the static float ranges."""
    return {s: act_params(ranges[s][0], ranges[s][1], STAGE_BITS[s]) for s in STAGE_BITS}


class BlockGPU:
    def __init__(self, data: wl.BlockData, device=None):
        import torch

        import paper_2408_13933_amd as mq

        self.mq, self.torch = mq, torch
        dev = device or torch.device("cuda", 0)
        d = wl.BLOCK_DIMS
        self.T, self.H, self.G, self.D = data.T, d["heads"], d["kv_heads"], d["head_dim"]
        self.eps, self.base = d["eps"], d["rope_base"]
        self.fmt = formats(data.ranges, mq.mq_act_params)
        T, H, G, D = self.T, self.H, self.G, self.D
        hid, ffn = d["hidden"], d["ffn"]
        self.gamma1 = torch.from_numpy(data.gamma1).to(dev)
        self.gamma2 = torch.from_numpy(data.gamma2).to(dev)
        self.w = {}
        for name, w in data.w.items():
            self.w[name] = mq.mq_pack_weights(torch.from_numpy(w).to(dev), 8)
        a, z = self.fmt["h0"]
        self.h0 = mq.mq_quantize_act(torch.from_numpy(data.h0).to(dev), a, z, 16)
        i8, i16 = torch.int8, torch.int16
        shapes = dict(x1=(T, hid), q=(T, H * D), k=(T, G * D), v=(T, G * D), qr=(T, H * D),
                      kr=(T, G * D), scores=(H, T, T), probs=(H, T, T), ctx=(T, H * D),
                      o=(T, hid), h1=(T, hid), x2=(T, hid), gate=(T, ffn), up=(T, ffn),
                      silu=(T, ffn), mul=(T, ffn), down=(T, hid), h2=(T, hid))
        self.out = {s: torch.empty(shp, dtype=i8 if STAGE_BITS[s] == 8 else i16, device=dev)
                    for s, shp in shapes.items() if s not in NOT_STORED}
        self.out["h0"] = self.h0
        self.vt = torch.empty((G * D, T), dtype=i8, device=dev)
        # the rotary angles depend only on T, D and the base: one table for
        # the queries and the keys, built once
        self.rope_table = mq.mq_rope_table(T, D, base=self.base, device=dev)
        # the SiLU table depends only on the static formats: built once
        self.lut = mq.mq_lut_build(mq.LUT_SILU, *self.fmt["gate"], *self.fmt["silu"], 16)
        ws = max(mq.mq_qlinear_workspace_bytes(T, K, N, 8, STAGE_BITS[s])
                 for s, (name, _) in LINEARS.items()
                 for (N, K) in [tuple(data.w[name].shape)])
        self.ws = torch.zeros(max(ws, 256), dtype=torch.uint8, device=dev)
        self.attn_ws = torch.empty(max(mq.mq_attn_matmul_workspace_bytes(H, G, T, T),
                                       mq.mq_attn_matmul_workspace_bytes(H, G, T, D)),
                                   dtype=torch.uint8, device=dev)

    def _linear(self, stage):
        name, src = LINEARS[stage]
        wq, ws, cs = self.w[name]
        a, z = self.fmt[src]
        oa, oz = self.fmt[stage]
        self.mq.mq_qlinear(self.out[src], wq, 8, ws, cs, a, z, oa, oz, STAGE_BITS[stage],
                           out=self.out[stage], workspace=self.ws)

    def _group(self, stages):
        """Linears that read one input (and write one code width) in one
        call: one launch on the prefill path, each output as _linear's."""
        src = LINEARS[stages[0]][1]
        a, z = self.fmt[src]
        lin = []
        for st in stages:
            wq, ws, cs = self.w[LINEARS[st][0]]
            oa, oz = self.fmt[st]
            lin.append(dict(w_q=wq, w_scale=ws, w_colsum=cs, out_scale=oa, out_zp=oz,
                            out=self.out[st]))
        self.mq.mq_qlinear_group(self.out[src], lin, 8, a, z, STAGE_BITS[stages[0]])

    def stages(self):
        """(name, callable) per step of the block, in order; each callable
        only enqueues kernels on the current stream."""
        mq, f, o = self.mq, self.fmt, self.out
        T, H, G, D = self.T, self.H, self.G, self.D
        qv = o["qr"].view(T, H, D).permute(1, 0, 2)
        kv = o["kr"].view(T, G, D).permute(1, 0, 2)
        cv = o["ctx"].view(T, H, D).permute(1, 0, 2)
        sa, sz = f["scores"]
        return [
            ("rmsnorm1", lambda: mq.mq_rmsnorm(o["h0"], *f["h0"], self.gamma1, self.eps, *f["x1"],
                                               8, out=o["x1"])),
            # q and k (16-bit outputs) in one launch; v writes 8-bit codes
            ("qk_proj", lambda: self._group(("q", "k"))),
            ("v_proj", lambda: self._linear("v")),
            ("rope_q", lambda: mq.mq_rope_apply(o["q"], H, *f["q"], *f["qr"], self.rope_table,
                                                16, out=o["qr"])),
            ("rope_k", lambda: mq.mq_rope_apply(o["k"], G, *f["k"], *f["kr"], self.rope_table, 8,
                                                out=o["kr"])),
            # causal: scores past the diagonal are never read
            ("qk_scores", lambda: mq.mq_attn_matmul(qv, kv, *f["qr"], *f["kr"], *f["scores"], 16,
                                                    out=o["scores"], workspace=self.attn_ws,
                                                    out_causal=0)),
            # the 1/sqrt(head dim) of the attention logits joins the score
            # scale (a power of two here, so exact in fp32)
            ("softmax", lambda: mq.mq_softmax_causal(o["scores"].view(H * T, T), sa / D ** 0.5,
                                                     sz, *f["probs"], T, 0, 16,
                                                     out=o["probs"].view(H * T, T))),
            ("v_transpose", lambda: mq.mq_transpose_i8(o["v"], out=self.vt)),
            # the hidden keys hold the probability-0 code
            ("pv_context", lambda: mq.mq_attn_matmul(o["probs"], self.vt.view(G, D, T),
                                                     *f["probs"], *f["v"], *f["ctx"], 8, out=cv,
                                                     workspace=self.attn_ws, in_causal=0)),
            ("o_proj", lambda: self._linear("o")),
            # the residual add and the RMSNorm of its sum in one pass (both
            # outputs written)
            ("residual1_rmsnorm2", lambda: mq.mq_add_rmsnorm(o["h0"], *f["h0"], o["o"], *f["o"],
                                                             *f["h1"], self.gamma2, self.eps,
                                                             *f["x2"], 8, h=o["h1"],
                                                             out=o["x2"])),
            ("gate_up_proj", lambda: self._group(("gate", "up"))),
            # SiLU table and gated product in one pass: the SiLU codes stay
            # in registers (the "silu" buffer is not written)
            ("silu_gated", lambda: mq.mq_lut_mul(o["gate"], self.lut, *f["silu"], o["up"],
                                                 *f["up"], *f["mul"], 8, out=o["mul"])),
            ("down_proj", lambda: self._linear("down")),
            ("residual2", lambda: mq.mq_add_requant(o["h1"], *f["h1"], o["down"], *f["down"],
                                                    *f["h2"], 16, out=o["h2"])),
        ]

    def run(self):
        for _, fn in self.stages():
            fn()
        return self.out["h2"]

    def ops(self) -> int:
        """Integer multiply-adds x 2 of the block's products (linears and
        attention; the causal half of the attention products included)."""
        d = wl.BLOCK_DIMS
        T, H, D = self.T, self.H, self.D
        hid, kv, ffn = d["hidden"], d["kv_heads"] * D, d["ffn"]
        lin = T * hid * (hid + 2 * kv + hid) + 3 * T * hid * ffn
        att = 2 * H * T * T * D
        return 2 * (lin + att)
