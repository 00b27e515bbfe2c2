"""Host-only checks of the measurement arithmetic in bench.py (no GPU)."""
import math
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def _row(name, a, b, stream):
    return (f'"KERNEL_DISPATCH","Agent 1",1,{stream},1,1,1,"void erase::{name}<unsigned short, 64, 64>'
            f'(erase::GemmDesc, erase::EpiParams)",1,{a},{b}')


def test_trace_overlap_by_kernel_name(tmp_path):
    """Backward kernel [5, 25] against forward kernels [0, 10] and [20, 30]:
    half of it runs beside forward work; a second backward kernel [40, 50]
    runs alone; two prologues 100 ns apart give the step time."""
    head = ('"Kind","Agent_Id","Queue_Id","Stream_Id","Thread_Id","Dispatch_Id","Kernel_Id","Kernel_Name",'
            '"Correlation_Id","Start_Timestamp","End_Timestamp"')
    rows = [_row("erase_prologue", 0, 1, 0), _row("erase_fwd_gemm", 0, 10, 0), _row("erase_fwd_head_gemm", 20, 30, 0),
            _row("erase_bwd_gemm", 5, 25, 1), _row("erase_wgrad_adam_kg2", 40, 50, 2), _row("erase_prologue", 100, 101, 0),
            _row("other_kernel", 0, 200, 0)]
    p = tmp_path / "kernel_trace.csv"
    p.write_text("\n".join([head] + rows) + "\n")
    r = bench.analyze_trace(str(p))
    assert r["bwd_kernels"] == 2 and r["fwd_kernels"] == 4
    assert math.isclose(r["overlap_fraction"], 10 / 30)
    assert r["steps"] == 2 and math.isclose(r["median_step_ms"], 100 / 1e6)
    assert r["bwd_streams"] == ["1", "2"]


def test_library_overlap_counts_every_backward_stream():
    recs = [{"stream": 0, "start_ms": 0.0, "end_ms": 10.0}, {"stream": 1, "start_ms": 5.0, "end_ms": 15.0},
            {"stream": 2, "start_ms": 0.0, "end_ms": 10.0}]
    assert math.isclose(bench.overlap_fraction(recs), 15 / 20)


def test_normalized_entropy_of_the_base_rate_predictor():
    """A head that predicts the base rate p everywhere has NE 1; a perfect
    head 0."""
    y = np.array([1.0] * 3 + [0.0] * 97)
    p = 0.03
    bce = -(p * np.log(p) + (1 - p) * np.log(1 - p))
    r = bench.normalized_entropy([bce, 0.0], y)
    assert math.isclose(r["per_block"][0], 1.0) and r["per_block"][1] == 0.0
    assert math.isclose(r["label_rate"], 0.03)
