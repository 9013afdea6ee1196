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
