"""Throughput of the integer-only quantized linear layer on one MI355X.

One step = one pass of the hot path over one batch of a workload's
synthetic, seeded inputs: quantize each distinct layer input (Section 4.2,
Eq.(4)), run every qlinear of the workload with its fused fixed-point
requant epilogue, and dequantize the last layer's output (written by that
layer's own epilogue through mq_qlinear_dequant when it has several rounds
of output tiles, as the LM head; else, or with --no-fuse-dequant, a pass of
its own over the stored codes).  The layers that read one input and
write one code width (gate and up) go out as one mq_qlinear_group launch
(--no-group: one launch per layer).  Weights are
folded/packed once before timing (offline steps).

The default workload is the Gemma-2B-shaped one (the largest of the layer
sets that fit one GPU): MLP gate and up (M=512, K=2048, N=16384), down
(M=512, K=16384, N=2048), and the LM head K=2048 -> N=256000 at M=1 (a
decode step) and M=512 (a prompt), all int8 weights and activations with
int16 outputs; the dequantized step output is the 512 x 256000 logits.

`value` is whole-step int8 TOPS = sum(2*M*N*K) / step time, inputs already
in HBM.  The JSON line also carries
* `roofline`: the dominant prefill kernel (the launch with the most
  operations), int8 TOP/s against the MFMA peak, timed with HIP events on
  the launch stream inside the timed steps;
* `decode`: the decode-shaped layers (M <= 16) with cold weights, GB/s of
  algorithmic bytes against the HBM peak -- the workload's own and those of
  the single-layer W8A8 (16 x 2048 x 2048) and W4A8 (1 x 5632 x 2048)
  workloads;
* `layers`: every launch's average kernel time in the timed steps;
* `cpu_baseline`: the CPU oracle's rate on a bounded sample of the step.

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--workload NAME]
"""
from __future__ import annotations

import argparse
import csv
import gc
import hashlib
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
DEFAULT_WORKLOAD = "gemma2b_w8a8"
# HBM traffic of the dominant prefill kernel (and of the decode kernel),
# from two rocprofv3 --pmc passes (FETCH_SIZE, WRITE_SIZE) summarised by
# --pmc-summary; valid only while the kernel sources hash to the value
# recorded with it
TRAFFIC_FILES = {
    "gemma2b_w8a8": os.path.join(ROOT, "profiles", "qlinear_lm_head_gemma2b_hbm_traffic.txt"),
    "prefill_w8a8_tinyllama_m2048": os.path.join(
        ROOT, "profiles", "qlinear_prefill_gate_up_tinyllama_m2048_hbm_traffic.txt"),
}
KERNEL_SOURCES = ("paper_2408_13933_amd/csrc/qlinear_prefill.hip",
                  "paper_2408_13933_amd/csrc/qlinear_decode.hip",
                  "paper_2408_13933_amd/csrc/qlinear_gemv.hip",
                  "paper_2408_13933_amd/csrc/requant.h",
                  "paper_2408_13933_amd/csrc/mq_internal.h")
# decode-shaped layers of the other workloads timed cold beside the
# workload's own: the single W8A8 layer and the W4A8 down projection at M=1
EXTRA_DECODE = (("decode_w8a8_m16", "linear"), ("w4a8_down_tinyllama", "down_proj_m1"))


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-fuse-dequant", action="store_true",
                    help="dequantize the last layer's codes in a pass of their own (by default "
                         "the last launch, mq_qlinear_dequant, writes the fp32 output itself)")
    ap.add_argument("--no-group", action="store_true",
                    help="launch every layer on its own (by default the layers that read one "
                         "quantized input and write one code width go out as one "
                         "mq_qlinear_group launch)")
    ap.add_argument("--graph", action="store_true",
                    help="also time the step replayed from a captured HIP graph, and the "
                         "dominant layer's launches replayed back to back")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target CPU time of the oracle sample")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="after timing, stream this many MiB through a plain elementwise kernel "
                         "three times (one read and one write of that size: the calibration "
                         "kernel of the HBM byte counters)")
    ap.add_argument("--calib-sweep", action="store_true",
                    help="time the calibration-side kernels (range learning, SmoothQuant "
                         "scales) instead of the step")
    ap.add_argument("--block-sweep", action="store_true",
                    help="time one whole TinyLlama decoder block on integer codes (1024 tokens) "
                         "and each of its steps, and exit")
    ap.add_argument("--attn-sweep", action="store_true",
                    help="time the attention matmuls (Q K^T, P V) and the value transpose "
                         "at the TinyLlama shape, seq 1024, and exit")
    ap.add_argument("--glue-sweep", action="store_true",
                    help="time the decoder-block glue kernels (residual add, SiLU lookup, "
                         "RMSNorm, softmax) instead of the step")
    ap.add_argument("--decode-sweep", action="store_true",
                    help="time the decode-shaped layers (M <= 16) cold: each launch reads a "
                         "different copy of the weights, >= 512 MB per sweep; prints one JSON "
                         "line per layer (run under rocprofv3 --kernel-trace for kernel-only "
                         "durations) and exits")
    ap.add_argument("--trace-summary", metavar="KERNEL_TRACE_CSV",
                    help="summarise a rocprofv3 --kernel-trace -f csv kernel_trace.csv: per "
                         "(kernel, grid, work-group) the dispatch count and the mean, median and "
                         "minimum duration, and exit")
    ap.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="summarise two rocprofv3 --pmc counter_collection.csv files (FETCH_SIZE "
                         "and WRITE_SIZE passes over a run with --calib-copy-mib) and exit")
    ap.add_argument("--sq-summary", nargs=2, metavar=("PASS_A_CSV", "PASS_B_CSV"),
                    help="summarise two rocprofv3 --pmc counter_collection.csv files of shader "
                         "counters (pass A: " + " ".join(SQ_PASS_A) + "; pass B: "
                         + " ".join(SQ_PASS_B) + ") per prefill kernel and exit")
    return ap.parse_args()


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def _pmc_rows(path, counter):
    """(kernel name, grid size, value) per dispatch of one counter."""
    out = []
    with open(path, newline="") as f:
        for row in csv.DictReader(f):
            if row["Counter_Name"] == counter:
                out.append((row["Kernel_Name"], int(row["Grid_Size"]), float(row["Counter_Value"])))
    return out


def _decode_layers(workload):
    """(workload, layer) of every decode-shaped layer the bench times cold:
    the workload's own, then the extra single-layer ones."""
    from paper_2408_13933_amd import workloads as wl

    own = [(workload, l) for l in wl.WORKLOADS[workload].layers if l.M <= 16]
    extra = [(w, next(l for l in wl.WORKLOADS[w].layers if l.name == n))
             for w, n in EXTRA_DECODE if w != workload]
    return own + extra


def launch_groups(workload, layers, group=True, max_group=4):
    """The layers (indices) of each launch of a step: consecutive
    prefill-shaped layers with 8-bit inputs that read one input (same
    activation and token count) and write one code width, up to max_group,
    form one mq_qlinear_group launch; every other layer is a launch of its
    own."""
    from paper_2408_13933_amd import workloads as wl

    out = []
    for i, L in enumerate(layers):
        if out and group:
            F = layers[out[-1][0]]
            if ((wl._x_key(workload, L), L.M) == (wl._x_key(workload, F), F.M) and L.M > 16 and
                    L.a_bits == 8 and (L.w_bits, L.out_bits, L.asym) ==
                    (F.w_bits, F.out_bits, F.asym) and len(out[-1]) < max_group):
                out[-1].append(i)
                continue
        out.append([i])
    return out


def launch_alg_bytes(layers, idx, f32_out=False):
    """Minimum bytes one launch moves: its shared input (and row sums) once,
    each layer's weights, outputs and per-channel parameters; f32_out: the
    output written as fp32 values instead of codes (fused dequantization)."""
    Ls = [layers[i] for i in idx]
    F = Ls[0]
    shared = F.M * F.K * F.a_bits // 8 + (F.M * 4 if F.asym else 0)
    b = sum(L.alg_bytes() for L in Ls) - (len(Ls) - 1) * shared
    if f32_out:
        b += sum(L.M * L.N * (4 - L.out_bits // 8) for L in Ls)
    return b


def launch_label(layers, idx):
    Ls = [layers[i] for i in idx]
    return (f"{'+'.join(L.name for L in Ls)} M={Ls[0].M} K={Ls[0].K} "
            f"N={'+'.join(str(L.N) for L in Ls)}")


def pmc_summary(fetch_csv, write_csv, copy_mib, workload, group=True, fuse_dequant=True):
    """HBM bytes per launch of the dominant prefill kernel and of each
    decode-shaped layer, each counter scaled by what it reads for the plain
    copy of known size in the same run."""
    import re

    from paper_2408_13933_amd import workloads as wl

    layers = wl.WORKLOADS[workload].layers
    launches = launch_groups(workload, layers, group)
    dom = max(launches, key=lambda idx: sum(layers[i].ops for i in idx))
    L = layers[dom[0]]
    # the step's last launch writes fp32 outputs when the dequantization is fused
    f32 = (fuse_dequant and dom is launches[-1] and len(dom) == 1 and L.a_bits == 8 and
           -(-L.M // 256) * -(-L.N // 256) > 256)
    per = {}
    for key, path, counter in (("fetch", fetch_csv, "FETCH_SIZE"), ("write", write_csv, "WRITE_SIZE")):
        rows = _pmc_rows(path, counter)
        c = [v for n, g, v in rows if "bitwise_not" in n]
        if not c:
            raise SystemExit(f"{counter}: no copy dispatches")
        factor = copy_mib * 1024.0 / (sum(c) / len(c))  # the copy reads and writes copy_mib
        groups = {}
        for n, g, v in rows:
            if ("qlinear_prefill" in n or "qlinear_decode_kernel" in n or
                    "qlinear_gemv_kernel" in n):
                groups.setdefault((n, g), []).append(v)
        per[key] = (groups, factor, sum(c) / len(c))

    def entry(kname, grid, alg):
        out = {"kernel": kname, "grid": grid, "alg_bytes_per_launch": alg}
        total = 0.0
        for key in ("fetch", "write"):
            groups, factor, copy_kib = per[key]
            v = groups.get((kname, grid), [])
            if not v:
                raise SystemExit(f"{key}: no dispatches of {kname} grid {grid}")
            kib = sum(v) / len(v)
            out[key] = {"kib_per_launch": kib, "launches": len(v), "copy_kib": copy_kib,
                        "factor": factor, "bytes_per_launch": kib * 1024.0 * factor}
            total += kib * 1024.0 * factor
        out["hbm_bytes_per_launch"] = total
        out["hbm_over_alg"] = total / alg
        return out

    # the dominant prefill launches: the prefill (kernel, grid) that fetches
    # the most bytes per dispatch (the launch with the most operations)
    pre = {k: v for k, v in per["fetch"][0].items() if "qlinear_prefill" in k[0]}
    (kname, grid), _ = max(pre.items(), key=lambda kv: sum(kv[1]) / len(kv[1]))
    res = {"workload": workload, "source_hash": kernel_source_hash(), "copy_mib": copy_mib,
           "prefill": dict(layer=f"{launch_label(layers, dom)} w{L.w_bits}/o{L.out_bits}"
                                 + (" fp32 out" if f32 else ""),
                           **entry(kname, grid, launch_alg_bytes(layers, dom, f32))),
           "decode": []}
    # decode layers: the decode (kernel, grid) with their weight and output
    # widths (template arguments), the most dispatched group of each
    dec = {k: v for k, v in per["fetch"][0].items()
           if "qlinear_decode_kernel" in k[0] or "qlinear_gemv_kernel" in k[0]}
    for wname, D in _decode_layers(workload):
        # one token of 8-bit codes runs the GEMV, more tokens the MFMA kernel
        kern = "qlinear_gemv_kernel" if D.M == 1 and D.a_bits == 8 else "qlinear_decode_kernel"
        pat = re.compile(rf"{kern}<{D.w_bits}, {D.out_bits},")
        cand = [(k, v) for k, v in dec.items() if pat.search(k[0])]
        if not cand:
            continue
        (kname, grid), _ = max(cand, key=lambda kv: len(kv[1]))
        res["decode"].append(dict(layer=f"{wname}/{D.name} M={D.M} K={D.K} N={D.N} "
                                        f"w{D.w_bits}/o{D.out_bits}",
                                  **entry(kname, grid, D.alg_bytes())))
    return res


# Shader counters of the prefill kernels, two rocprofv3 --pmc passes (at most
# 8 SQ counters per pass) over the same bench command.
SQ_PASS_A = ("SQ_WAVES", "SQ_BUSY_CU_CYCLES", "SQ_VALU_MFMA_BUSY_CYCLES", "SQ_INSTS_VALU",
             "SQ_INSTS_MFMA", "SQ_INSTS_LDS", "SQ_INSTS_SALU", "SQ_WAVE_CYCLES", "GRBM_GUI_ACTIVE")
SQ_PASS_B = ("SQ_LDS_BANK_CONFLICT", "SQ_LDS_IDX_ACTIVE", "SQ_WAIT_INST_LDS", "SQ_WAIT_INST_ANY",
             "SQ_ACTIVE_INST_VALU", "SQ_ACTIVE_INST_LDS", "SQ_ACTIVE_INST_ANY", "GRBM_GUI_ACTIVE")
XCDS, SIMDS = 8, 1024


def sq_summary(a_csv, b_csv):
    """Per prefill (kernel, grid) of the two shader-counter passes, averaged
    over dispatches: cycles (GRBM_GUI_ACTIVE is reported summed over the 8
    XCDs), the MFMA-busy fraction of the SIMD-cycles, instructions per wave,
    the LDS bank-conflict fraction of the LDS-active cycles, and the
    fractions of wave time spent waiting to issue and issuing VALU / LDS."""
    import re

    groups = {}
    for path in (a_csv, b_csv):
        per = {}
        with open(path, newline="") as f:
            for r in csv.DictReader(f):
                if "qlinear_prefill" not in r["Kernel_Name"]:
                    continue
                name = re.sub(r"\(anonymous namespace\)::|mq::", "", r["Kernel_Name"])
                name = re.sub(r"^void ", "", name).split("(QLinearArgs")[0]
                key = (name, int(r["Grid_Size"]))
                d = per.setdefault(int(r["Dispatch_Id"]), (key, {}))[1]
                d[r["Counter_Name"]] = d.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
        for key, d in per.values():
            g = groups.setdefault(key, {})
            for c, v in d.items():
                g.setdefault(c, []).append(v)
    rows = []
    for (name, grid), g in groups.items():
        m = {c: sum(v) / len(v) for c, v in g.items()}
        waves, cyc = m["SQ_WAVES"], m["GRBM_GUI_ACTIVE"] / XCDS
        rows.append({
            "kernel": name, "grid": grid, "dispatches": len(g["SQ_WAVES"]),
            "cycles": round(cyc),
            "mfma_busy": round(m["SQ_VALU_MFMA_BUSY_CYCLES"] / (cyc * SIMDS), 3),
            "per_wave": {k: round(m["SQ_INSTS_" + k.upper()] / waves, 1)
                         for k in ("valu", "mfma", "lds", "salu")},
            "lds_bank_conflict": round(m["SQ_LDS_BANK_CONFLICT"] / max(1.0, m["SQ_LDS_IDX_ACTIVE"]), 3),
            "wait_issue": round(m["SQ_WAIT_INST_ANY"] / max(1.0, m["SQ_WAVE_CYCLES"]), 3),
            "active_valu": round(m["SQ_ACTIVE_INST_VALU"] / max(1.0, m["SQ_ACTIVE_INST_ANY"]), 3),
            "active_lds": round(m["SQ_ACTIVE_INST_LDS"] / max(1.0, m["SQ_ACTIVE_INST_ANY"]), 3),
        })
    rows.sort(key=lambda r: -r["cycles"] * r["dispatches"])
    return "\n".join(json.dumps(r) for r in rows)


def trace_summary(path):
    """Per (kernel, grid, work-group size) of a rocprofv3 kernel trace:
    dispatches and durations (us), largest total time first."""
    import re

    groups = {}
    with open(path, newline="") as f:
        for r in csv.DictReader(f):
            name = r["Kernel_Name"]
            # namespaces and the argument list off; template arguments kept
            short = re.sub(r"\(anonymous namespace\)::|mq::|at::native::", "", name)
            short = re.sub(r"^void ", "", short)
            depth, cut = 0, len(short)
            for i, ch in enumerate(short):
                if ch == "<":
                    depth += 1
                elif ch == ">":
                    depth -= 1
                elif ch == "(" and depth == 0:
                    cut = i
                    break
            short = short[:cut]
            grid = int(r["Grid_Size_X"]) * int(r["Grid_Size_Y"]) * int(r["Grid_Size_Z"])
            wg = int(r["Workgroup_Size_X"]) * int(r["Workgroup_Size_Y"]) * int(r["Workgroup_Size_Z"])
            us = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
            groups.setdefault((short, grid, wg), []).append(us)
    rows = sorted(groups.items(), key=lambda kv: -sum(kv[1]))
    out = [f"{'kernel':<78} {'grid':>9} {'wg':>5} {'n':>6} {'avg_us':>9} {'med_us':>9} "
           f"{'min_us':>9}"]
    for (k, grid, wg), v in rows:
        v = sorted(v)
        out.append(f"{k[:78]:<78} {grid:>9} {wg:>5} {len(v):>6} {sum(v) / len(v):>9.2f} "
                   f"{v[len(v) // 2]:>9.2f} {v[0]:>9.2f}")
    return "\n".join(out)


def read_traffic(workload):
    """Calibrated HBM bytes per launch, or None when absent or stale."""
    path = TRAFFIC_FILES.get(workload)
    if path is None:
        return None
    try:
        with open(path) as f:
            line = [l for l in f if l.startswith("{")][-1]
        rec = json.loads(line)
    except (OSError, IndexError, ValueError):
        return None
    if rec.get("source_hash") != kernel_source_hash() or rec.get("workload") != workload:
        return None
    return rec


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


class TimingEvent:
    """A HIP event for timing only, created with hipEventDisableSystemFence:
    recording it does not release to system scope, which on MI355X writes
    back and invalidates the L2s and left a ~5.6 us gap before the next
    kernel (measured: a Gemma-2B step 0.658-0.690 ms with one default event
    per layer, 0.641-0.646 ms with none).  Recorded on torch's current
    stream, through the HIP runtime torch has loaded."""

    _hip = None
    DISABLE_SYSTEM_FENCE = 0x20000000

    @classmethod
    def _lib(cls):
        if cls._hip is None:
            import ctypes

            import torch

            torch.cuda.init()
            path = None
            with open("/proc/self/maps") as f:
                for line in f:
                    if "libamdhip64.so" in line:
                        path = line.split()[-1]
                        break
            if path is None:
                raise RuntimeError("the HIP runtime is not loaded")
            L = ctypes.CDLL(path)
            L.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
            L.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
            L.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                              ctypes.c_void_p]
            L.hipEventDestroy.argtypes = [ctypes.c_void_p]
            cls._hip = L
        return cls._hip

    def __init__(self):
        import ctypes

        self._c = ctypes
        self.ev = ctypes.c_void_p()
        st = self._lib().hipEventCreateWithFlags(ctypes.byref(self.ev), self.DISABLE_SYSTEM_FENCE)
        if st != 0:
            raise RuntimeError(f"hipEventCreateWithFlags: {st}")

    def record(self, stream=None):
        import torch

        s = (stream or torch.cuda.current_stream()).cuda_stream
        st = self._lib().hipEventRecord(self.ev, self._c.c_void_p(s))
        if st != 0:
            raise RuntimeError(f"hipEventRecord: {st}")

    def elapsed_time(self, other) -> float:
        """Milliseconds from this event to `other` (both complete)."""
        ms = self._c.c_float()
        st = self._lib().hipEventElapsedTime(self._c.byref(ms), self.ev, other.ev)
        if st != 0:
            raise RuntimeError(f"hipEventElapsedTime: {st}")
        return ms.value

    def __del__(self):
        if self._hip is not None and self.ev:
            self._hip.hipEventDestroy(self.ev)


class Prepared:
    """Device-resident inputs and packed weights of one workload."""

    def __init__(self, workload_name, group=True, fuse_dequant=True):
        import torch

        import paper_2408_13933_amd as mq
        from paper_2408_13933_amd import workloads as wl

        self.mq = mq
        self.wl = wl.WORKLOADS[workload_name]
        self.layers = []
        dev = torch.device("cuda", 0)
        xs = {}
        for layer in self.wl.layers:
            # layers reading the same activation at the same token count share
            # its draw and its quantization (q/k/v, gate/up)
            key = (wl._x_key(workload_name, layer), layer.M)
            ld = wl.make_layer(workload_name, layer, shared_x=xs.get(key))
            xs.setdefault(key, ld.x)
            w = torch.from_numpy(ld.w).to(dev)
            ld.w = None  # the host copy is not needed after the upload
            if ld.s is not None:
                w = mq.mq_fold_weights(w, torch.from_numpy(ld.s).to(dev))
            w_zp = None
            if layer.asym:
                w_q, w_scale, w_zp, w_colsum = mq.mq_pack_weights_asym(
                    w, layer.w_bits, per_tensor=layer.per_tensor)
            else:
                w_q, w_scale, w_colsum = mq.mq_pack_weights(w, layer.w_bits)
            del w
            a_scale, a_zp = mq.mq_act_params(*ld.act_range, layer.a_bits)
            out_scale, out_zp = mq.mq_act_params(*ld.out_range, layer.out_bits)
            entry = dict(layer=layer, data=ld, key=key, w_q=w_q, w_scale=w_scale, w_zp=w_zp,
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
                a_bits = e["layer"].a_bits
                qdt = torch.int8 if a_bits == 8 else torch.int16
                self.inputs[e["key"]] = dict(x=x, q=torch.empty(x.shape, dtype=qdt, device=dev),
                                             scale=e["a_scale"], zp=e["a_zp"], rs=None,
                                             bits=a_bits)
            if e["layer"].asym and self.inputs[e["key"]]["rs"] is None:
                # asymmetric weights read the row sums of their quantized input
                self.inputs[e["key"]]["rs"] = torch.empty(e["layer"].M, dtype=torch.int32,
                                                          device=dev)
        for e in self.layers:
            L = e["layer"]
            e["y"] = torch.empty((L.M, L.N), dtype=torch.int8 if L.out_bits == 8 else torch.int16,
                                 device=dev)
        # one zero-filled workspace shared by the (sequential) qlinear calls:
        # layers with few output tiles and a long K split K through it
        ws_bytes = max(mq.mq_qlinear_workspace_bytes(e["layer"].M, e["layer"].K, e["layer"].N,
                                                     e["layer"].w_bits, e["layer"].out_bits)
                       for e in self.layers)
        self.workspace = (torch.zeros(ws_bytes, dtype=torch.uint8, device=dev) if ws_bytes
                          else None)
        last = self.layers[-1]
        self.deq = torch.empty(last["y"].shape, dtype=torch.float32, device=dev)
        # launches: gate/up (q/k/v) as one mq_qlinear_group call each
        self.launches = launch_groups(workload_name, [e["layer"] for e in self.layers], group,
                                      mq.MAX_GROUP)
        # the last launch writes the step's dequantized output itself (its
        # codes feed nothing else) when the layer has several rounds of
        # output tiles (more 256x256 tiles than CUs): then one tile's fp32
        # stores overlap the other tiles' products.  In one round they all
        # come at the end (2048 x 2048 o-proj: 21.8 us fused against 14.5 +
        # 5.8 us for the codes and a pass of its own).
        L = last["layer"]
        rounds = -(-L.M // 256) * -(-L.N // 256) > 256
        self.fuse_dequant = (fuse_dequant and rounds and len(self.launches[-1]) == 1 and
                             L.a_bits == 8)
        torch.cuda.synchronize()

    def qlinear(self, e, w_q=None, workspace=None):
        """One qlinear launch of layer entry e on its already quantized input
        (and, for asymmetric weights, its row sums)."""
        L = e["layer"]
        inp = self.inputs[e["key"]]
        w_q = e["w_q"] if w_q is None else w_q
        if L.asym:
            self.mq.mq_qlinear_asym(inp["q"], inp["rs"], w_q, L.w_bits, e["w_scale"], e["w_zp"],
                                    e["w_colsum"], e["a_scale"], e["a_zp"], e["out_scale"],
                                    e["out_zp"], L.out_bits, bias=e["bias"], out=e["y"],
                                    workspace=workspace)
        elif L.a_bits == 16:
            self.mq.mq_qlinear_a16(inp["q"], w_q, L.w_bits, e["w_scale"], e["w_colsum"],
                                   e["a_scale"], e["a_zp"], e["out_scale"], e["out_zp"],
                                   L.out_bits, bias=e["bias"], out=e["y"])
        else:
            self.mq.mq_qlinear(inp["q"], w_q, L.w_bits, e["w_scale"], e["w_colsum"],
                               e["a_scale"], e["a_zp"], e["out_scale"], e["out_zp"], L.out_bits,
                               bias=e["bias"], out=e["y"], workspace=workspace)

    def launch(self, j):
        """Launch j (one layer, or a group of layers on one input) on its
        already quantized input."""
        idx = self.launches[j]
        if j == len(self.launches) - 1 and self.fuse_dequant:
            e = self.layers[idx[0]]
            L = e["layer"]
            inp = self.inputs[e["key"]]
            self.mq.mq_qlinear_dequant(inp["q"], e["w_q"], L.w_bits, e["w_scale"], e["w_colsum"],
                                       e["a_scale"], e["a_zp"], e["out_scale"], e["out_zp"],
                                       L.out_bits, bias=e["bias"], out=self.deq, w_zp=e["w_zp"],
                                       a_rowsum=inp["rs"] if L.asym else None,
                                       workspace=self.workspace)
            return
        if len(idx) == 1:
            self.qlinear(self.layers[idx[0]], workspace=self.workspace)
            return
        es = [self.layers[i] for i in idx]
        L = es[0]["layer"]
        inp = self.inputs[es[0]["key"]]
        lin = [dict(w_q=e["w_q"], w_scale=e["w_scale"], w_zp=e["w_zp"], w_colsum=e["w_colsum"],
                    bias=e["bias"], out_scale=e["out_scale"], out_zp=e["out_zp"], out=e["y"])
               for e in es]
        self.mq.mq_qlinear_group(inp["q"], lin, L.w_bits, es[0]["a_scale"], es[0]["a_zp"],
                                 L.out_bits, a_rowsum=inp["rs"] if L.asym else None)

    def launch_name(self, j):
        return launch_label([e["layer"] for e in self.layers], self.launches[j])

    def step(self, events=None):
        """One pass of the hot path.  `events`: len(launches) + 1 events, the
        first recorded before the first qlinear launch and event j + 1 after
        launch j (all on the launch stream)."""
        mq = self.mq
        for inp in self.inputs.values():
            if inp["rs"] is not None:  # codes and their row sums in one pass
                mq.mq_quantize_act_rowsum(inp["x"], inp["scale"], inp["zp"], out=inp["q"],
                                          rowsum=inp["rs"])
            else:
                mq.mq_quantize_act(inp["x"], inp["scale"], inp["zp"], inp["bits"], out=inp["q"])
        if events is not None:
            events[0].record()
        for j in range(len(self.launches)):
            self.launch(j)
            if events is not None:
                events[j + 1].record()
        if not self.fuse_dequant:
            last = self.layers[-1]
            mq.mq_dequant(last["y"], last["out_scale"], last["out_zp"], out=self.deq)


def cold_graph_us(prep: Prepared, i: int, min_bytes: int = 512 * 10**6, replays: int = 5):
    """Per-launch time of layer i with its weights cold: copies of the packed
    weights (>= min_bytes in total) used in turn by launches captured into
    one HIP graph, replayed back to back.  For decode-shaped layers, whose
    kernels are shorter than a host launch, eager event timing measures the
    host instead."""
    import torch

    e = prep.layers[i]
    L = e["layer"]
    wbytes = e["w_q"].numel()
    copies = max(2, -(-min_bytes // wbytes))
    ws = [e["w_q"]] + [e["w_q"].clone() for _ in range(copies - 1)]

    def launch(w):
        prep.qlinear(e, w_q=w)

    for w in ws:
        launch(w)
    g = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cap):
        with torch.cuda.graph(g, stream=cap):
            for w in ws:
                launch(w)
    torch.cuda.current_stream().wait_stream(cap)
    g.replay()
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(replays):
        g.replay()
    t1.record()
    torch.cuda.synchronize()
    us = t0.elapsed_time(t1) * 1e3 / (replays * copies)
    del g, ws
    torch.cuda.empty_cache()
    return us, copies


def cpu_baseline(prep: Prepared, target_s: float):
    """The oracle, as it stands, on a bounded sample of the same step: the
    first R token rows of every prefill-shaped layer (R sized to about
    target_s of CPU time) and every decode-shaped layer (M <= 16) whole."""
    import oracle

    nthreads = oracle.default_threads()
    w_host = []
    for e in prep.layers:
        w_host.append((e["w_q"].cpu().numpy(), e["w_scale"].cpu().numpy(),
                       None if e["bias"] is None else e["bias"].cpu().numpy(),
                       None if e["w_zp"] is None else e["w_zp"].cpu().numpy()))

    def run(rows):
        ops = 0
        t0 = time.perf_counter()
        for e, (wq, ws, b, zw) in zip(prep.layers, w_host):
            L = e["layer"]
            r = L.M if L.M <= 16 else min(rows, L.M)
            x = e["data"].x[:r]
            a = oracle.quantize_act(x, e["a_scale"], e["a_zp"], L.a_bits)
            oracle.qlinear(a, wq, L.w_bits, ws, e["a_scale"], e["a_zp"], e["out_scale"],
                           e["out_zp"], L.out_bits, bias=b, nthreads=nthreads, w_zp=zw)
            ops += 2 * r * L.N * L.K
        return ops, time.perf_counter() - t0

    max_rows = max(e["layer"].M for e in prep.layers)
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
    dec = [e["layer"].name for e in prep.layers if e["layer"].M <= 16]
    model = cpu_model()
    single = cpu_single_thread()
    return {"value": total_ops / total_dt / 1e12, "unit": "TOPS", "cores": nthreads,
            "kind": "oracle",
            "sample": f"first {rows} token rows of each prefill-shaped layer"
                      + (f" and the whole decode layer(s) {', '.join(dec)} (one token row: "
                         f"one thread)" if dec else "")
                      + f" (quantize + integer GEMM + requant), {reps} pass(es), "
                        f"{total_dt:.1f} s on {nthreads} host threads of {model}",
            "cpu_model": model, "single_thread": single}


def cpu_single_thread(min_s: float = 1.0):
    """The oracle on one host thread over the whole single W8A8 layer
    (16 x 2048 x 2048 with bias): quantize + integer GEMM + requant."""
    import oracle
    from paper_2408_13933_amd import workloads as wl

    L = next(l for l in wl.WORKLOADS["decode_w8a8_m16"].layers if l.name == "linear")
    ld = wl.make_layer("decode_w8a8_m16", L)
    wq, ws, _ = oracle.pack_weights(ld.w, L.w_bits)
    a_scale, a_zp = oracle.act_params(*ld.act_range, L.a_bits)
    o_scale, o_zp = oracle.act_params(*ld.out_range, L.out_bits)
    reps, dt = 0, 0.0
    t0 = time.perf_counter()
    while dt < min_s:
        a = oracle.quantize_act(ld.x, a_scale, a_zp, L.a_bits)
        oracle.qlinear(a, wq, L.w_bits, ws, a_scale, a_zp, o_scale, o_zp, L.out_bits,
                       bias=ld.bias, nthreads=1)
        reps += 1
        dt = time.perf_counter() - t0
    return {"value": reps * L.ops / dt / 1e12, "unit": "TOPS", "cores": 1, "kind": "oracle",
            "sample": f"decode_w8a8_m16/linear 16x2048x2048 whole, {reps} pass(es), "
                      f"{dt:.2f} s on one host thread",
            "ms_per_layer": dt / reps * 1e3}


DECODE_LAYERS = (("decode_w8a8_m16", "linear"), ("w4a8_down_tinyllama", "down_proj_m1"),
                 ("gemma2b_w8a8", "lm_head_m1"))


def decode_grid(L):
    """(work-groups, waves per work-group) of the decode kernel the library
    launches for layer L: the launch rules of qlinear_gemv.hip (one token)
    and qlinear_decode.hip (2..16 tokens), restated for the floor probe."""
    if L.M == 1 and L.a_bits == 8 and L.K % (16 if L.w_bits == 8 else 32) == 0:
        wrow = L.K * L.w_bits // 8
        steps = -(-wrow // 128)
        nw = 1
        while nw < 8 and nw * 4 < steps:
            nw *= 2
        return -(-L.N // 8), nw
    R = 8 if -(-L.N // 16) < 256 else 16
    blocks = -(-L.N // R)
    steps = -(-L.K // 64)
    nw, nwmax = 1, 8 if L.a_bits == 16 else 16
    while nw < nwmax and nw * 8 < steps:
        nw *= 2
    if blocks < 2048:
        while nw < 4 and nw < steps:
            nw *= 2
    return blocks, nw


def decode_sweep(launches_per_layer=400):
    """Cold decode launches.  Weight codes are random (the kernel's time does
    not depend on their values); shapes, formats and bias follow the
    workload's layer.  Two timings per layer: HIP events around the launch
    loop (bounded below by host launch overhead for kernels of a few us) and
    one captured sweep replayed as a HIP graph."""
    import torch

    import paper_2408_13933_amd as mq
    from paper_2408_13933_amd import workloads as wl

    dev = torch.device("cuda", 0)
    g = torch.Generator(device=dev)
    g.manual_seed(0)
    for wname, lname in DECODE_LAYERS:
        L = next(l for l in wl.WORKLOADS[wname].layers if l.name == lname)
        kb = L.K * L.w_bits // 8
        wbytes = L.N * kb
        copies = max(2, -(-512 * 10**6 // wbytes))
        ws = [torch.randint(0, 256, (L.N, kb), dtype=torch.uint8, device=dev, generator=g)
              for _ in range(copies)]
        if L.w_bits == 8:
            ws = [w.view(torch.int8) for w in ws]
        scale = torch.rand(L.N, device=dev, generator=g) * 1e-3 + 1e-4
        cs = torch.randint(-50000, 50000, (L.N,), dtype=torch.int32, device=dev, generator=g)
        bias = torch.randn(L.N, device=dev, generator=g) * 0.01 if L.bias else None
        a = torch.randint(-128, 128, (L.M, L.K), dtype=torch.int8, device=dev, generator=g)
        y = torch.empty((L.M, L.N), dtype=torch.int8 if L.out_bits == 8 else torch.int16,
                        device=dev)

        def launch(w):
            mq.mq_qlinear(a, w, L.w_bits, scale, cs, 0.05, 3, 0.02, -2, L.out_bits, bias=bias,
                          out=y)

        for w in ws:
            launch(w)
        torch.cuda.synchronize()
        reps = max(1, launches_per_layer // copies)
        s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s0.record()
        for _ in range(reps):
            for w in ws:
                launch(w)
        s1.record()
        torch.cuda.synchronize()
        event_us = s0.elapsed_time(s1) * 1e3 / (reps * copies)
        graph = torch.cuda.CUDAGraph()
        cap = torch.cuda.Stream()
        cap.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(cap):
            with torch.cuda.graph(graph, stream=cap):
                for w in ws:
                    launch(w)
        torch.cuda.current_stream().wait_stream(cap)
        graph.replay()
        torch.cuda.synchronize()
        s0.record()
        for _ in range(reps):
            graph.replay()
        s1.record()
        torch.cuda.synchronize()
        graph_us = s0.elapsed_time(s1) * 1e3 / (reps * copies)
        # the floor: a plain streaming read of the same weight copies with the
        # kernel's grid (mq_probe_read), replayed the same way
        blocks, waves = decode_grid(L)
        per_wave_kib = -(-wbytes // (blocks * waves * 1024))
        unroll = 1
        while unroll < 8 and unroll < per_wave_kib:
            unroll *= 2
        sink = torch.empty(blocks * waves, dtype=torch.int32, device=dev)
        fgraph = torch.cuda.CUDAGraph()
        with torch.cuda.stream(cap):
            with torch.cuda.graph(fgraph, stream=cap):
                for w in ws:
                    mq.mq_probe_read(w, blocks, waves, unroll, sink=sink)
        torch.cuda.current_stream().wait_stream(cap)
        fgraph.replay()
        torch.cuda.synchronize()
        s0.record()
        for _ in range(reps):
            fgraph.replay()
        s1.record()
        torch.cuda.synchronize()
        floor_us = s0.elapsed_time(s1) * 1e3 / (reps * copies)
        alg = L.alg_bytes()
        print(json.dumps({"layer": f"{wname}/{lname}", "M": L.M, "K": L.K, "N": L.N,
                          "w_bits": L.w_bits, "out_bits": L.out_bits, "weight_copies": copies,
                          "launches": 2 * reps * copies + copies, "alg_bytes": alg,
                          "event_us_per_launch": event_us, "graph_us_per_launch": graph_us,
                          "graph_GBps": alg / (graph_us * 1e-6) / 1e9,
                          "graph_frac_hbm": alg / (graph_us * 1e-6) / 1e9 / PEAK_HBM_GBS,
                          "floor": {"grid": [blocks, waves], "unroll": unroll,
                                    "bytes": wbytes, "graph_us_per_launch": floor_us,
                                    "kernel_over_floor": graph_us / floor_us}}),
              flush=True)
        del ws, graph, fgraph
        torch.cuda.empty_cache()


def calib_sweep(reps=5, per_graph=10):
    """Calibration-side kernels on TinyLlama-sized tensors: activation range
    learning forward/backward on a 2048x2048 fp32 activation and SmoothQuant
    scales over X 2048x2048 and W 5632x2048.  Each op is captured
    `per_graph` times into a HIP graph and replayed; algorithmic bytes per
    launch / time against the 8 TB/s HBM peak."""
    import torch

    import paper_2408_13933_amd as mq

    dev = torch.device("cuda", 0)
    g = torch.Generator(device=dev)
    g.manual_seed(0)
    M, K, N = 2048, 2048, 5632
    x = torch.randn((M, K), device=dev, generator=g) * 3
    gr = torch.randn((M, K), device=dev, generator=g)
    w = torch.randn((N, K), device=dev, generator=g) * 0.02
    y = torch.empty_like(x)
    gx = torch.empty_like(x)
    grads = torch.empty(2 + 2 * mq.ARL_PARTIALS, dtype=torch.float64, device=dev)
    s = torch.empty(K, device=dev)
    mx = torch.empty(K, device=dev)
    mw = torch.empty(K, device=dev)
    ops = {
        "arl_forward": (lambda: mq.mq_arl_forward(x, 0.05, -128.0, 8, out=y), 8 * M * K),
        "arl_backward": (lambda: mq.mq_arl_backward(x, gr, 0.05, -128.0, 8, gx=gx, grads=grads),
                         12 * M * K),
        "smooth_scales": (lambda: mq.mq_smooth_scales(x, w, 0.5, s=s, x_absmax=mx, w_absmax=mw),
                          4 * (M + N) * K + 12 * K),
    }
    for name, (fn, nbytes) in ops.items():
        fn()
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        cap = torch.cuda.Stream()
        cap.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(cap):
            with torch.cuda.graph(graph, stream=cap):
                for _ in range(per_graph):
                    fn()
        torch.cuda.current_stream().wait_stream(cap)
        graph.replay()
        torch.cuda.synchronize()
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0.record()
        for _ in range(reps):
            graph.replay()
        t1.record()
        torch.cuda.synchronize()
        us = t0.elapsed_time(t1) * 1e3 / (reps * per_graph)
        gbs = nbytes / us / 1e3
        print(json.dumps({"op": name, "shape": [M, K] if name != "smooth_scales" else [M, N, K],
                          "us_graph_replay": round(us, 2), "alg_bytes": nbytes,
                          "GB/s": round(gbs, 1), "frac_hbm": round(gbs / 8000.0, 3)}), flush=True)


def _time_graph(fn, reps=5, per_graph=10):
    """Per-launch time of fn from a HIP graph of `per_graph` launches."""
    import torch

    fn()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cap):
        with torch.cuda.graph(graph, stream=cap):
            for _ in range(per_graph):
                fn()
    torch.cuda.current_stream().wait_stream(cap)
    graph.replay()
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(reps):
        graph.replay()
    t1.record()
    torch.cuda.synchronize()
    return t0.elapsed_time(t1) * 1e3 / (reps * per_graph)


def glue_sweep():
    """The decoder-block glue at TinyLlama shapes, seq 1024: residual add on
    the 1024x2048 hidden state (int16 + int16 -> int16), SiLU lookup on the
    1024x5632 gate output (int16 -> int8), RMSNorm 1024x2048 (int16 -> int8),
    softmax over 32 heads x 1024 x 1024 scores (int16 -> int16).  Codes are
    uniform random int16 from torch's seeded generator."""
    import torch

    import paper_2408_13933_amd as mq

    dev = torch.device("cuda", 0)
    g = torch.Generator(device=dev)
    g.manual_seed(0)

    def codes(*shape):
        return torch.randint(-32768, 32768, shape, dtype=torch.int32, device=dev,
                             generator=g).to(torch.int16)

    h1, h2 = codes(1024, 2048), codes(1024, 2048)
    gate = codes(1024, 5632)
    scores = codes(32 * 1024, 1024)
    lut = mq.mq_lut_build(mq.LUT_SILU, 1e-3, 0, 0.05, 0, 8)
    gamma = torch.ones(2048, device=dev)
    out16 = torch.empty_like(h1)
    out8 = torch.empty((1024, 2048), dtype=torch.int8, device=dev)
    g8 = torch.empty((1024, 5632), dtype=torch.int8, device=dev)
    p16 = torch.empty_like(scores)
    ops = {
        "add_requant": (lambda: mq.mq_add_requant(h1, 3e-4, 0, h2, 5e-4, 0, 6e-4, 0, 16,
                                                  out=out16), 6 * h1.numel(), [1024, 2048]),
        "silu_lookup": (lambda: mq.mq_lut_apply(gate, lut, out=g8), 3 * gate.numel(),
                        [1024, 5632]),
        "rmsnorm": (lambda: mq.mq_rmsnorm(h1, 3e-4, 0, gamma, 1e-5, 0.02, 0, 8, out=out8),
                    3 * h1.numel() + 4 * 2048, [1024, 2048]),
        "softmax": (lambda: mq.mq_softmax(scores, 1e-3, 0, 1.0 / 65535, -32768, 16, out=p16),
                    4 * scores.numel(), [32 * 1024, 1024]),
    }
    for name, (fn, nbytes, shape) in ops.items():
        us = _time_graph(fn)
        gbs = nbytes / us / 1e3
        print(json.dumps({"op": name, "shape": shape, "us_graph_replay": round(us, 2),
                          "alg_bytes": nbytes, "GB/s": round(gbs, 1),
                          "frac_hbm": round(gbs / 8000.0, 3)}), flush=True)


def attn_sweep():
    """The self-attention matmuls of the W8A16 setting at TinyLlama shapes,
    seq 1024: 32 query heads, 4 key/value heads, head dimension 64.  Q K^T:
    int16 query codes (head views of the [1024][2048] projection output) x
    int8 key codes ([1024][256] views) -> int16 scores [32][1024][1024]; P V:
    int16 probability codes x the transposed int8 value codes -> int16
    context written into the [1024][2048] layout; the value transpose.  Ops
    count 2 per multiply-add of the 16 x 8-bit products (each runs as two
    int8 MFMAs).  Codes are uniform random from torch's seeded generator."""
    import torch

    import paper_2408_13933_amd as mq

    dev = torch.device("cuda", 0)
    g = torch.Generator(device=dev)
    g.manual_seed(0)
    T, D, H, G = 1024, 64, 32, 4

    def codes(lo, hi, shape, dt):
        return torch.randint(lo, hi, shape, dtype=torch.int32, device=dev, generator=g).to(dt)

    q = codes(-32768, 32768, (T, H * D), torch.int16)
    k = codes(-128, 128, (T, G * D), torch.int8)
    v = codes(-128, 128, (T, G * D), torch.int8)
    p = codes(-32768, 32768, (H, T, T), torch.int16)
    scores = torch.empty((H, T, T), dtype=torch.int16, device=dev)
    ctx = torch.empty((T, H * D), dtype=torch.int16, device=dev)
    vt = torch.empty((G * D, T), dtype=torch.int8, device=dev)
    ws1 = torch.empty(mq.mq_attn_matmul_workspace_bytes(H, G, T, T), dtype=torch.uint8, device=dev)
    ws2 = torch.empty(mq.mq_attn_matmul_workspace_bytes(H, G, T, D), dtype=torch.uint8, device=dev)
    qa, kb = q.view(T, H, D).permute(1, 0, 2), k.view(T, G, D).permute(1, 0, 2)
    cview = ctx.view(T, H, D).permute(1, 0, 2)
    macs = H * T * T * D
    ops = {
        "qk_scores": (lambda: mq.mq_attn_matmul(qa, kb, 2e-5, 0, 0.03, 0, 1e-3, 0, 16, out=scores,
                                                workspace=ws1),
                      2 * macs, 2 * T * H * D + T * G * D + 2 * H * T * T),
        "pv_context": (lambda: mq.mq_attn_matmul(p, vt.view(G, D, T), 1.0 / 65535, -32768, 0.03,
                                                 0, 1e-3, 0, 16, out=cview, workspace=ws2),
                       2 * macs, 2 * H * T * T + T * G * D + 2 * T * H * D),
        "v_transpose": (lambda: mq.mq_transpose_i8(v, out=vt), 0, 2 * T * G * D),
    }
    for name, (fn, nops, nbytes) in ops.items():
        us = _time_graph(fn)
        rec = {"op": name, "heads": H, "kv_heads": G, "seq": T, "head_dim": D,
               "us_graph_replay": round(us, 2), "alg_bytes": nbytes,
               "GB/s": round(nbytes / us / 1e3, 1)}
        if nops:
            rec["TOPS"] = round(nops / us / 1e6, 1)
        print(json.dumps(rec), flush=True)


def block_sweep(T=1024):
    """One TinyLlama decoder block on integer codes, every step on the GPU
    (paper_2408_13933_amd.block): RMSNorm, q/k/v projections, RoPE, Q K^T,
    causal softmax, P V, o projection, residual add fused with the RMSNorm, gate/up, SiLU
    table fused with the gated product, down projection, residual add.  Inputs: seeded
    synthetic residual stream and weights (workloads.make_block), static
    formats from the float pass.  Prints the graph-replayed time of each
    step and of the whole block."""
    import torch

    from paper_2408_13933_amd import block as blk
    from paper_2408_13933_amd import workloads as wl

    g = blk.BlockGPU(wl.make_block(T))
    g.run()
    torch.cuda.synchronize()
    total = 0.0
    for name, fn in g.stages():
        us = _time_graph(fn)
        total += us
        print(json.dumps({"step": name, "tokens": T, "us_graph_replay": round(us, 2)}), flush=True)
    us = _time_graph(g.run, reps=5, per_graph=2)
    print(json.dumps({"block": "tinyllama_w8a8_attn_a16", "tokens": T,
                      "us_graph_replay": round(us, 2), "sum_of_steps_us": round(total, 2),
                      "ops": g.ops(), "TOPS": round(g.ops() / us / 1e6, 1)}), flush=True)


def main():
    args = parse()
    if args.block_sweep:
        block_sweep()
        return
    if args.attn_sweep:
        attn_sweep()
        return
    if args.calib_sweep:
        calib_sweep()
        return
    if args.glue_sweep:
        glue_sweep()
        return
    if args.decode_sweep:
        decode_sweep()
        return
    if args.trace_summary:
        print(trace_summary(args.trace_summary))
        return
    if args.sq_summary:
        print(sq_summary(*args.sq_summary))
        return
    if args.pmc_summary:
        if args.calib_copy_mib <= 0:
            raise SystemExit("--pmc-summary needs the --calib-copy-mib size of the profiled run")
        print(json.dumps(pmc_summary(args.pmc_summary[0], args.pmc_summary[1],
                                     args.calib_copy_mib, args.workload,
                                     group=not args.no_group,
                                     fuse_dequant=not args.no_fuse_dequant)))
        return
    if args.gpus != 1:
        print(json.dumps({"error": "the qlinear path is measured on one GPU only (its multi-GPU "
                                   "sharding is a design, not a run); use --gpus 1"}))
        sys.exit(2)
    import torch

    prep = Prepared(args.workload, group=not args.no_group,
                    fuse_dequant=not args.no_fuse_dequant)
    layers = [e["layer"] for e in prep.layers]
    ops_step = sum(L.ops for L in layers)
    # operations of each launch (a layer, or a group of layers on one input)
    launch_ops = [sum(layers[i].ops for i in idx) for idx in prep.launches]
    launch_m = [layers[idx[0]].M for idx in prep.launches]
    # dominant kernel: the prefill-shaped launch with the most operations
    dom = max((j for j in range(len(prep.launches)) if launch_m[j] > 16),
              key=lambda j: launch_ops[j], default=None)

    for _ in range(args.warmup):
        prep.step()
    torch.cuda.synchronize()

    # per-layer events inside the timed steps: timing-only (no system fence)
    evs = [[TimingEvent() for _ in range(len(prep.launches) + 1)] for _ in range(args.steps)]
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    # no garbage-collection pause of the launching thread inside the timed
    # steps (the events time the stream, so a stalled host shows up as GPU
    # idle time)
    gc.collect()
    gc.disable()
    t_wall = time.perf_counter()
    start.record()
    for s in range(args.steps):
        prep.step(events=evs[s])
    end.record()
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    gc.enable()
    ms = start.elapsed_time(end) / args.steps
    # average duration of each launch inside the timed steps
    launch_us = [float(np.mean([ev[j].elapsed_time(ev[j + 1]) for ev in evs])) * 1e3
                 for j in range(len(prep.launches))]

    line = {
        "metric": METRIC,
        "value": ops_step / (ms * 1e-3) / 1e12,
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
                   "step": "quantize inputs + %d qlinear launches (%s) + dequant of last output%s"
                           % (len(prep.launches),
                              ", ".join(prep.launch_name(j).split(" ")[0]
                                        for j in range(len(prep.launches))),
                              " (written by the last launch's epilogue)" if prep.fuse_dequant
                              else " (its own pass)"),
                   "ops_per_step": ops_step},
    }
    tr = read_traffic(args.workload)

    if dom is not None:
        L = layers[prep.launches[dom][0]]
        k_us = launch_us[dom]
        k_graph_us = None
        if args.graph:
            # Cross-check of the dominant kernel's duration, outside the
            # timed region: its launches replayed back to back from a HIP
            # graph (no host launch gaps; sustained, so the chip runs hotter
            # and clocks lower than within the step)
            reps = 10
            gk = torch.cuda.CUDAGraph()
            s_k = torch.cuda.Stream()
            s_k.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(s_k):
                with torch.cuda.graph(gk, stream=s_k):
                    for _ in range(reps):
                        prep.launch(dom)
            torch.cuda.current_stream().wait_stream(s_k)
            gk.replay()
            torch.cuda.synchronize()
            k0, k1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            n_replay = 5
            k0.record()
            for _ in range(n_replay):
                gk.replay()
            k1.record()
            torch.cuda.synchronize()
            k_graph_us = k0.elapsed_time(k1) * 1e3 / (n_replay * reps)
            del gk
        achieved = launch_ops[dom] / (k_us * 1e-6) / 1e12
        roof = {"bound": "mfma", "achieved": achieved, "peak": PEAK_INT8_TOPS, "unit": "TOP/s",
                "frac": achieved / PEAK_INT8_TOPS, "traffic": None}
        f32 = prep.fuse_dequant and dom == len(prep.launches) - 1
        if (tr is not None and tr["prefill"]["layer"].startswith(prep.launch_name(dom) + " ") and
                tr["prefill"]["layer"].endswith(" fp32 out") == f32):
            t = tr["prefill"]
            roof["traffic"] = t["hbm_bytes_per_launch"]
            roof["traffic_detail"] = {"unit": "bytes per launch",
                                      "fetch": t["fetch"]["bytes_per_launch"],
                                      "write": t["write"]["bytes_per_launch"],
                                      "algorithmic": t["alg_bytes_per_launch"]}
        roof.update({"kernel": f"qlinear_prefill {prep.launch_name(dom)} "
                               f"w{L.w_bits}/o{L.out_bits}" + (" fp32 out" if f32 else ""),
                     "ops_per_launch": launch_ops[dom], "kernel_us": k_us})
        if k_graph_us is not None:
            roof["kernel_us_graph_replay"] = k_graph_us
        line["roofline"] = roof

    # decode half of the metric: cold weights (each launch reads another copy
    # of the packed weights, >= 512 MB per sweep), graph replay
    dec = []
    extra = {w: Prepared(w) for w, _ in EXTRA_DECODE if w != args.workload}
    for wname, D in _decode_layers(args.workload):
        pp = prep if wname == args.workload else extra[wname]
        i = next(j for j, e in enumerate(pp.layers) if e["layer"] is D)
        cold_us, copies = cold_graph_us(pp, i)
        gbs = D.alg_bytes() / (cold_us * 1e-6) / 1e9
        d = {"bound": "hbm", "achieved": gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s",
             "frac": gbs / PEAK_HBM_GBS, "traffic": None,
             "kernel": f"qlinear_decode {wname}/{D.name} M={D.M} K={D.K} N={D.N} "
                       f"w{D.w_bits}/o{D.out_bits}",
             "alg_bytes_per_launch": D.alg_bytes(), "kernel_us": cold_us,
             "timing": f"cold weights ({copies} copies), graph replay"}
        if tr is not None:
            t = [x for x in tr["decode"] if x["layer"].startswith(f"{wname}/{D.name} ")]
            if t:
                d["traffic"] = t[0]["hbm_bytes_per_launch"]
        dec.append(d)
    del extra
    if dec:
        line["decode"] = dec[0]
        line["decode_layers"] = dec
    line["layers"] = [{"layer": prep.launch_name(j), "kernel_us": u,
                       ("TOP/s" if launch_m[j] > 16 else "GB/s"):
                           (launch_ops[j] / (u * 1e-6) / 1e12 if launch_m[j] > 16
                            else launch_alg_bytes(layers, prep.launches[j]) / (u * 1e-6) / 1e9)}
                      for j, u in enumerate(launch_us)]
    line["wall_s_timed"] = t_wall

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
        line["graph_ms_per_step"] = graph_ms
        line["graph_value"] = ops_step / (graph_ms * 1e-3) / 1e12
        del g
    if args.calib_copy_mib > 0:
        n = args.calib_copy_mib * (1 << 20)
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.bitwise_not(src, out=dst)  # one streaming read and write of n bytes
        torch.cuda.synchronize()
        del src, dst
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(prep, args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
