"""CPU tests of bench.py's measurement helpers: the launch grouping of a
step, the algorithmic bytes per launch, the traffic record's staleness rule
and the summaries of rocprofv3 output (kernel trace, shader counters) on
small hand-written CSV files whose expected figures are worked out here.
"""
import csv
import json

import pytest

import bench
from paper_2408_13933_amd import workloads as wl


def _layers(name):
    return list(wl.WORKLOADS[name].layers)


def test_launch_groups_gemma_step():
    """gate and up read one input and write int16 codes: one launch; down,
    the one-token LM head and the 512-token LM head each launch alone."""
    ls = _layers("gemma2b_w8a8")
    names = [[ls[i].name for i in g] for g in bench.launch_groups("gemma2b_w8a8", ls)]
    assert names == [["gate_proj", "up_proj"], ["down_proj"], ["lm_head_m1"], ["lm_head_m512"]]
    # without grouping every layer is a launch of its own
    assert bench.launch_groups("gemma2b_w8a8", ls, group=False) == [[i] for i in range(len(ls))]


def test_launch_groups_block_caps_and_code_width():
    """q/k/v share an input; grouping stops at the group limit."""
    ls = _layers("block_w8a8_tinyllama_s1024")
    groups = bench.launch_groups("block_w8a8_tinyllama_s1024", ls)
    names = [[ls[i].name for i in g] for g in groups]
    assert names[0] == ["q_proj", "k_proj", "v_proj"]
    assert ["gate_proj", "up_proj"] in names
    two = bench.launch_groups("block_w8a8_tinyllama_s1024", ls, max_group=2)
    assert [[ls[i].name for i in g] for g in two][0] == ["q_proj", "k_proj"]


def test_launch_alg_bytes_counts_the_shared_input_once():
    ls = _layers("gemma2b_w8a8")
    gate, up = ls[0], ls[1]
    both = bench.launch_alg_bytes(ls, [0, 1])
    shared = gate.M * gate.K  # int8 activations
    assert both == gate.alg_bytes() + up.alg_bytes() - shared
    # fp32 outputs add 2 bytes per int16 output
    lm = len(ls) - 1
    L = ls[lm]
    assert bench.launch_alg_bytes(ls, [lm], f32_out=True) == L.alg_bytes() + 2 * L.M * L.N


def test_traffic_record_needs_the_current_source_hash(tmp_path, monkeypatch):
    rec = {"workload": "gemma2b_w8a8", "source_hash": bench.kernel_source_hash(),
           "prefill": {"hbm_bytes_per_launch": 123}}
    p = tmp_path / "t.txt"
    p.write_text("header\n" + json.dumps(rec) + "\n")
    monkeypatch.setitem(bench.TRAFFIC_FILES, "gemma2b_w8a8", str(p))
    assert bench.read_traffic("gemma2b_w8a8") is not None
    rec["source_hash"] = "0" * 16
    p.write_text(json.dumps(rec) + "\n")
    assert bench.read_traffic("gemma2b_w8a8") is None


def _write_csv(path, fields, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=fields)
        w.writeheader()
        for r in rows:
            w.writerow(r)


def test_trace_summary_mean_median_min(tmp_path):
    fields = ["Kernel_Name", "Grid_Size_X", "Grid_Size_Y", "Grid_Size_Z", "Workgroup_Size_X",
              "Workgroup_Size_Y", "Workgroup_Size_Z", "Start_Timestamp", "End_Timestamp"]
    name = "void mq::(anonymous namespace)::k<1, 2>(mq::QLinearArgs, int)"
    rows = [dict(Kernel_Name=name, Grid_Size_X=512, Grid_Size_Y=2, Grid_Size_Z=1,
                 Workgroup_Size_X=256, Workgroup_Size_Y=1, Workgroup_Size_Z=1,
                 Start_Timestamp=1000, End_Timestamp=1000 + ns) for ns in (3000, 1000, 2000)]
    p = tmp_path / "trace.csv"
    _write_csv(p, fields, rows)
    out = bench.trace_summary(str(p)).splitlines()
    assert len(out) == 2
    cols = out[1].split()
    # namespaces and the argument list dropped, template arguments kept
    assert cols[0] == "k<1," and cols[1] == "2>"
    assert cols[2:] == ["1024", "256", "3", "2.00", "2.00", "1.00"]


def test_sq_summary_fields(tmp_path):
    """One prefill kernel, two dispatches per pass; the counters are chosen
    so each derived field is a round number."""
    fields = ["Dispatch_Id", "Grid_Size", "Kernel_Name", "Counter_Name", "Counter_Value"]
    name = "void mq::(anonymous namespace)::qlinear_prefill_kernel<Cfg<8>, false>(mq::QLinearArgs, int)"
    a = {"SQ_WAVES": 100, "SQ_BUSY_CU_CYCLES": 1, "SQ_VALU_MFMA_BUSY_CYCLES": 1024 * 500,
         "SQ_INSTS_VALU": 1500, "SQ_INSTS_MFMA": 300, "SQ_INSTS_LDS": 200, "SQ_INSTS_SALU": 100,
         "SQ_WAVE_CYCLES": 4000, "GRBM_GUI_ACTIVE": 8 * 1000}
    b = {"SQ_LDS_BANK_CONFLICT": 25, "SQ_LDS_IDX_ACTIVE": 100, "SQ_WAIT_INST_LDS": 10,
         "SQ_WAIT_INST_ANY": 1000, "SQ_ACTIVE_INST_VALU": 60, "SQ_ACTIVE_INST_LDS": 20,
         "SQ_ACTIVE_INST_ANY": 200, "GRBM_GUI_ACTIVE": 8 * 1000}
    for tag, cs in (("A", a), ("B", b)):
        rows = []
        for disp in (1, 2):
            for c, v in cs.items():
                rows.append(dict(Dispatch_Id=disp, Grid_Size=4096, Kernel_Name=name,
                                 Counter_Name=c, Counter_Value=v))
        # another kernel's rows are ignored
        rows.append(dict(Dispatch_Id=3, Grid_Size=64, Kernel_Name="void other()",
                         Counter_Name="SQ_WAVES", Counter_Value=1))
        _write_csv(tmp_path / f"{tag}.csv", fields, rows)
    out = bench.sq_summary(str(tmp_path / "A.csv"), str(tmp_path / "B.csv")).splitlines()
    assert len(out) == 1
    r = json.loads(out[0])
    assert r["kernel"] == "qlinear_prefill_kernel<Cfg<8>, false>"
    assert r["grid"] == 4096 and r["dispatches"] == 2
    assert r["cycles"] == 1000           # GRBM_GUI_ACTIVE summed over 8 XCDs
    assert r["mfma_busy"] == 0.5         # 1024*500 busy SIMD-cycles / (1000 * 1024)
    assert r["per_wave"] == {"valu": 15.0, "mfma": 3.0, "lds": 2.0, "salu": 1.0}
    assert r["lds_bank_conflict"] == 0.25
    assert r["wait_issue"] == 0.25
    assert r["active_valu"] == 0.3 and r["active_lds"] == 0.1


@pytest.mark.parametrize("workload", sorted(bench.TRAFFIC_FILES))
def test_committed_traffic_records_parse(workload):
    """The committed traffic profiles end with a JSON record for their
    workload (stale or current)."""
    with open(bench.TRAFFIC_FILES[workload]) as f:
        rec = json.loads([l for l in f if l.startswith("{")][-1])
    assert rec["workload"] == workload
    assert rec["prefill"]["hbm_bytes_per_launch"] > rec["prefill"]["alg_bytes_per_launch"] * 0.9
