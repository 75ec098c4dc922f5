"""Throughput of the integer-only quantized linear layer on one MI355X.

One step = one pass of the hot path over one batch of the TinyLlama-shaped
prefill workload (synthetic, seeded): quantize the two layer inputs
(Section 4.2, Eq.(4)), run the three int8 qlinears -- MLP gate and up
(M=2048, K=2048, N=5632) and attention o-proj (M=2048, K=2048, N=2048) --
with their fused fixed-point requant epilogues, and dequantize the o-proj
output.  Weights are folded/packed once before timing (offline steps).

`value` is whole-step int8 TOPS = sum(2*M*N*K) / step time, inputs already
in HBM.  The JSON line also carries the roofline of the dominant kernel (the
gate/up-shaped prefill GEMM, timed with HIP events on the launch stream) and
the CPU oracle's rate on a bounded sample of the same workload.

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--workload NAME]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "qlinear int8 TOPS (prefill, % MFMA peak) + decode GB/s (% HBM peak), bit-exact"
PEAK_INT8_TOPS = 5000.0      # MI355X dense int8 MFMA, 5.0 POP/s
PEAK_HBM_GBS = 8000.0        # MI355X HBM3E, 8 TB/s
DEFAULT_WORKLOAD = "prefill_w8a8_tinyllama_m2048"


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--graph", action="store_true",
                    help="also time the step replayed from a captured HIP graph")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target CPU time of the oracle sample")
    return ap.parse_args()


class Prepared:
    """Device-resident inputs and packed weights of one workload."""

    def __init__(self, workload_name):
        import torch

        import paper_2408_13933_amd as mq
        from paper_2408_13933_amd import workloads as wl

        self.mq = mq
        self.wl = wl.WORKLOADS[workload_name]
        self.layers = []
        dev = torch.device("cuda", 0)
        xs = {}
        for layer in self.wl.layers:
            key = wl._x_key(workload_name, layer)
            ld = wl.make_layer(workload_name, layer, shared_x=xs.get(key))
            xs.setdefault(key, ld.x)
            w = torch.from_numpy(ld.w).to(dev)
            if ld.s is not None:
                w = mq.mq_fold_weights(w, torch.from_numpy(ld.s).to(dev))
            w_q, w_scale, w_colsum = mq.mq_pack_weights(w, layer.w_bits)
            del w
            a_scale, a_zp = mq.mq_act_params(*ld.act_range, 8)
            out_scale, out_zp = mq.mq_act_params(*ld.out_range, layer.out_bits)
            entry = dict(layer=layer, data=ld, key=key, w_q=w_q, w_scale=w_scale,
                         w_colsum=w_colsum, a_scale=a_scale, a_zp=a_zp, out_scale=out_scale,
                         out_zp=out_zp,
                         bias=None if ld.bias is None else torch.from_numpy(ld.bias).to(dev))
            self.layers.append(entry)
        # one fp32 input and one int8 buffer per distinct activation; the
        # layers that read the same activation share its quantization
        self.inputs = {}
        for e in self.layers:
            if e["key"] not in self.inputs:
                x = torch.from_numpy(e["data"].x).to(dev)
                self.inputs[e["key"]] = dict(x=x, q=torch.empty(x.shape, dtype=torch.int8,
                                                                device=dev),
                                             scale=e["a_scale"], zp=e["a_zp"])
        for e in self.layers:
            L = e["layer"]
            e["y"] = torch.empty((L.M, L.N), dtype=torch.int8 if L.out_bits == 8 else torch.int16,
                                 device=dev)
        last = self.layers[-1]
        self.deq = torch.empty(last["y"].shape, dtype=torch.float32, device=dev)
        torch.cuda.synchronize()

    def step(self, events=None, dom=()):
        """One pass of the hot path.  `events` = (start, end) recorded around
        the consecutive run of dominant-kernel launches listed in `dom`."""
        mq = self.mq
        for inp in self.inputs.values():
            mq.mq_quantize_act(inp["x"], inp["scale"], inp["zp"], 8, out=inp["q"])
        for i, e in enumerate(self.layers):
            L = e["layer"]
            a = self.inputs[e["key"]]["q"]
            if events is not None and dom and i == dom[0]:
                events[0].record()
            mq.mq_qlinear(a, e["w_q"], L.w_bits, e["w_scale"], e["w_colsum"], e["a_scale"],
                          e["a_zp"], e["out_scale"], e["out_zp"], L.out_bits, bias=e["bias"],
                          out=e["y"])
            if events is not None and dom and i == dom[-1]:
                events[1].record()
        last = self.layers[-1]
        mq.mq_dequant(last["y"], last["out_scale"], last["out_zp"], out=self.deq)


def cpu_baseline(prep: Prepared, target_s: float):
    """The oracle, as it stands, on a bounded row sample of the same step."""
    import oracle

    nthreads = oracle.default_threads()
    w_host = []
    for e in prep.layers:
        w_host.append((e["w_q"].cpu().numpy(), e["w_scale"].cpu().numpy(),
                       None if e["bias"] is None else e["bias"].cpu().numpy()))

    def run(rows):
        ops = 0
        t0 = time.perf_counter()
        for e, (wq, ws, b) in zip(prep.layers, w_host):
            L = e["layer"]
            x = e["data"].x[:rows]
            a = oracle.quantize_act(x, e["a_scale"], e["a_zp"], 8)
            oracle.qlinear(a, wq, L.w_bits, ws, e["a_scale"], e["a_zp"], e["out_scale"],
                           e["out_zp"], L.out_bits, bias=b, nthreads=nthreads)
            ops += 2 * rows * L.N * L.K
        return ops, time.perf_counter() - t0

    max_rows = min(e["layer"].M for e in prep.layers)
    probe_rows = max(1, min(nthreads, max_rows))
    ops, dt = run(probe_rows)
    rows = int(probe_rows * max(1.0, target_s / max(dt, 1e-3)))
    rows = max(probe_rows, min(rows, max_rows))
    rows = (rows // nthreads) * nthreads or probe_rows
    total_ops, total_dt, reps = 0, 0.0, 0
    while total_dt < target_s and reps < 50:
        ops, dt = run(rows)
        total_ops += ops
        total_dt += dt
        reps += 1
    return {"value": total_ops / total_dt / 1e12, "unit": "TOPS", "cores": nthreads,
            "kind": "oracle",
            "sample": f"first {rows} token rows of each layer of the step (quantize + integer "
                      f"GEMM + requant), {reps} pass(es), {total_dt:.1f} s on {nthreads} host "
                      f"threads"}


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build measures one GPU only; run with --gpus 1"}))
        sys.exit(2)
    import torch

    prep = Prepared(args.workload)
    layers = [e["layer"] for e in prep.layers]
    ops_step = sum(L.ops for L in layers)

    # dominant kernel: the layers with the largest op count (launched back
    # to back in the step, so one event pair brackets them all)
    big = max(L.ops for L in layers)
    dom = [i for i, L in enumerate(layers) if L.ops == big]
    assert dom == list(range(dom[0], dom[-1] + 1)), "dominant launches must be consecutive"

    for _ in range(args.warmup):
        prep.step()
    torch.cuda.synchronize()

    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    start.record()
    for s in range(args.steps):
        prep.step(events=evs[s], dom=dom)
    end.record()
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    ms = start.elapsed_time(end) / args.steps
    k_avg_ms = float(np.mean([a.elapsed_time(b) for a, b in evs])) / len(dom)

    graph_ms = None
    if args.graph:
        # the same step captured once into a HIP graph and replayed: no
        # host launch gaps between the kernels
        g = torch.cuda.CUDAGraph()
        s_cap = torch.cuda.Stream()
        s_cap.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s_cap):
            with torch.cuda.graph(g, stream=s_cap):
                prep.step()
        torch.cuda.current_stream().wait_stream(s_cap)
        for _ in range(3):
            g.replay()
        torch.cuda.synchronize()
        gs, ge = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        gs.record()
        for _ in range(args.steps):
            g.replay()
        ge.record()
        torch.cuda.synchronize()
        graph_ms = gs.elapsed_time(ge) / args.steps
    L = layers[dom[0]]
    if L.M <= 16:
        achieved = L.alg_bytes() / (k_avg_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": achieved / PEAK_HBM_GBS, "traffic": None}
    else:
        achieved = L.ops / (k_avg_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": achieved, "peak": PEAK_INT8_TOPS, "unit": "TOP/s",
                "frac": achieved / PEAK_INT8_TOPS, "traffic": None}
    roof.update({"kernel": f"qlinear_prefill {L.name} M={L.M} K={L.K} N={L.N} "
                           f"w{L.w_bits}/o{L.out_bits}" if L.M > 16 else
                           f"qlinear_decode {L.name} M={L.M} K={L.K} N={L.N}",
                 "kernel_us": k_avg_ms * 1e3})

    value = ops_step / (ms * 1e-3) / 1e12
    line = {
        "metric": METRIC,
        "value": value,
        "unit": "TOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "i8",
        "data": "synthetic (seeded; layer shapes of the paper's models, outlier channels)",
        "config": {"workload": args.workload,
                   "layers": [f"{l.name} M={l.M} K={l.K} N={l.N} w{l.w_bits} o{l.out_bits}"
                              for l in layers],
                   "step": "quantize inputs + qlinear x%d + dequant of last output" % len(layers),
                   "ops_per_step": ops_step},
        "roofline": roof,
        "wall_s_timed": t_wall,
    }
    if graph_ms is not None:
        line["graph_ms_per_step"] = graph_ms
        line["graph_value"] = ops_step / (graph_ms * 1e-3) / 1e12
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(prep, args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
