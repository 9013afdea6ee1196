"""Host logic of bench.py (no GPU): the one-GPU guard and the algorithmic flop
accounting of the prefill stages, with and without a shared system prefix."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_stage_flops_closed_forms():
    d, ffn = 4096, 11008
    lens = [643] * 6 + [355] * 18 + [211] * 25 + [131] * 51
    T = sum(lens)
    fl = bench.stage_flops(T, d, ffn, lens)
    assert fl["qkv_rope"] == 2 * T * d * 3 * d and fl["out_proj"] == 2 * T * d * d
    assert fl["gate_up_swiglu"] == 2 * T * d * 2 * ffn and fl["down_proj"] == 2 * T * ffn * d
    assert fl["attention"] == sum(2 * d * L * (L + 1) for L in lens)


@pytest.mark.parametrize("P", [1, 35])
def test_stage_flops_with_a_shared_prefix(P):
    """Sharing removes (n - 1) copies of the prefix rows from every GEMM and
    (n - 1) copies of the prefix's causal triangle from the attention."""
    d, ffn = 4096, 11008
    lens = [643] * 6 + [355] * 18 + [211] * 25 + [131] * 51
    n = len(lens)
    T = sum(lens)
    Ts = T - (n - 1) * P
    a = bench.stage_flops(T, d, ffn, lens)
    b = bench.stage_flops(Ts, d, ffn, lens, P)
    for k in ("qkv_rope", "out_proj", "gate_up_swiglu", "down_proj"):
        assert a[k] * Ts == b[k] * T
    assert a["attention"] - b["attention"] == (n - 1) * 2 * d * P * (P + 1)


def test_cpu_baseline_uses_the_affinity_cores_and_reports_stages():
    """The CPU baseline on the small f32 scene: the core count is the
    affinity set (capped at one GPU's host share of 16), every stage has a
    time, and the rate is retained tokens over their sum."""
    import synth
    w = synth.get("tiny")
    sc = synth.make_scene(w)
    lens = [w.n_sys + 64 + w.n_qry] * 2
    cb = bench.cpu_baseline(w, sc, [(lens[0], 2)], 1)
    assert cb["cores"] == min(len(os.sched_getaffinity(0)), 16)
    assert set(cb["stage_s"]) == {"stage1_s", "select_s", "compact_s", "prefill_s"}
    assert cb["kind"] == "oracle" and cb["value"] > 0


def test_counter_report_derives_clock_busy_and_bytes(tmp_path):
    """The rocprofv3 CSV summary: clock = GRBM_GUI_ACTIVE / 8 over the
    duration, MFMA busy over 1,024 SIMDs, bytes scaled by the calibration
    copy's readings."""
    hdr = ('"Correlation_Id","Dispatch_Id","Agent_Id","Queue_Id","Process_Id","Thread_Id","Grid_Size",'
           '"Kernel_Id","Kernel_Name","Workgroup_Size","LDS_Block_Size","Scratch_Size","VGPR_Count",'
           '"Accum_VGPR_Count","SGPR_Count","Counter_Name","Counter_Value","Start_Timestamp","End_Timestamp"')

    def row(i, name, c, v, t0, t1):
        return f'{i},{i},"Agent 1",1,1,1,256,1,"{name}",256,0,0,8,0,32,"{c}",{v},{t0},{t1}'
    # 1 ms kernel at 2 GHz: 8 x 2e6 GUI cycles; MFMA busy half of 1,024 SIMDs
    rows = [row(1, "void rift::gemm_x<2>(int)", "GRBM_GUI_ACTIVE", 8 * 2e6, 0, 1_000_000),
            row(1, "void rift::gemm_x<2>(int)", "SQ_VALU_MFMA_BUSY_CYCLES", 0.5 * 2e6 * 1024, 0, 1_000_000),
            row(1, "void rift::gemm_x<2>(int)", "FETCH_SIZE", 1e6 / 1024 / 2, 0, 1_000_000),
            row(2, "void at::neg_kernel(float)", "FETCH_SIZE", (1 << 30) / 1024 / 2, 0, 10)]
    f = tmp_path / "p_counter_collection.csv"
    f.write_text("\n".join([hdr] + rows) + "\n")
    rep = bench.counter_report([str(tmp_path)])
    line = [l for l in rep.splitlines() if "gemm_x<2>" in l][0]
    cells = [c.strip() for c in line.split("|")]
    assert cells[3] == "1000.0" and cells[4] == "2.000" and cells[5] == "50.0%"
    assert cells[7] == "0.0010"   # 1e6 bytes after the x2 calibration
