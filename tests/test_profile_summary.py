"""Host logic of the profile summaries (no GPU): counter calibration against
the run's 1 GiB copy, the step window of the decoder-stack counters, and the
source hashes the bench compares the committed counters against."""
import csv
import json
import os
import subprocess
import sys

import pytest

from paper_2609_26638_amd import rocprof_summary as rs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GIB = 1 << 30


def _write_counters(d, counter, dispatches):
    """dispatches: [(kernel name, [instance values in KiB])] in dispatch order."""
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "run_counter_collection.csv"), "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value",
                    "Start_Timestamp", "End_Timestamp"])
        for i, (name, vals) in enumerate(dispatches, start=1):
            for v in vals:
                w.writerow([i, name, counter, v, 1000 * i, 1000 * i + 500])


def _stack_run(fetch_scale_kib):
    """Two warmup steps and three measured steps of three kernels, a fill of
    the calibration buffer and a small runtime copy (a host read) before
    them, a kernel and another small copy after the calibration copy."""
    step = [("embed_rows_kernel", [1.0]), ("gemm_ws_kernel", [10.0, 10.0]),
            ("attn_bf16_kernel", [4.0])]
    return ([("fill_kernel", [999.0])] + step * 2 + [("__amd_rocclr_copyBuffer", [0.5])] +
            step * 3 + [("__amd_rocclr_copyBuffer", [fetch_scale_kib]), ("reduce_kernel", [7.0]),
                        ("__amd_rocclr_copyBuffer", [0.5])])


def test_traffic_calibrates_against_the_copy(tmp_path):
    # FETCH_SIZE reading half the copy's bytes: scale 2
    _write_counters(tmp_path / "f", "FETCH_SIZE",
                    [("attn_bf16_pc_kernel", [100.0, 100.0]), ("attn_bf16_pc_kernel", [300.0]),
                     ("__amd_rocclr_copyBuffer", [GIB / 2048.0])])
    _write_counters(tmp_path / "w", "WRITE_SIZE",
                    [("attn_bf16_pc_kernel", [8.0]), ("attn_bf16_pc_kernel", [8.0]),
                     ("__amd_rocclr_copyBuffer", [GIB / 1024.0])])
    tr = rs.traffic(str(tmp_path / "f"), str(tmp_path / "w"), "attn_bf16", GIB)
    assert tr["FETCH_SIZE"]["scale"] == pytest.approx(2.0)
    assert tr["WRITE_SIZE"]["scale"] == pytest.approx(1.0)
    # instances of one dispatch are summed, dispatches averaged
    assert tr["FETCH_SIZE"]["bytes_per_dispatch"] == pytest.approx((200.0 + 300.0) / 2 * 1024 * 2.0)
    assert tr["WRITE_SIZE"]["bytes_per_dispatch"] == pytest.approx(8.0 * 1024)


def test_steps_window_and_calibration(tmp_path):
    _write_counters(tmp_path / "f", "FETCH_SIZE", _stack_run(GIB / 2048.0))
    _write_counters(tmp_path / "w", "WRITE_SIZE", _stack_run(GIB / 1024.0))
    out = rs.steps(str(tmp_path / "f"), str(tmp_path / "w"), "embed_rows", 3, GIB)
    fs, fa = out["FETCH_SIZE"]
    assert fs == pytest.approx(2.0)
    # the last three steps only: the fill before them and the kernel after
    # the copy are outside the window
    assert list(fa) == ["embed_rows_kernel", "gemm_ws_kernel", "attn_bf16_kernel"]
    assert fa["gemm_ws_kernel"][0] == 3
    assert fa["gemm_ws_kernel"][1] == pytest.approx(3 * 20.0 * 1024 * 2.0)
    with pytest.raises(ValueError):
        rs.steps(str(tmp_path / "f"), str(tmp_path / "w"), "embed_rows", 6, GIB)


def test_steps_command_writes_json_and_table(tmp_path):
    _write_counters(tmp_path / "f", "FETCH_SIZE", _stack_run(GIB / 2048.0))
    _write_counters(tmp_path / "w", "WRITE_SIZE", _stack_run(GIB / 1024.0))
    meta = {"profile_stack": "ar", "steps": 3, "marker": "embed_rows_kernel",
            "step_algorithmic_bytes": 50000, "copy_bytes": GIB, "src_hash": "abc"}
    (tmp_path / "meta.json").write_text("log line\n" + json.dumps(meta) + "\n")
    js, md = tmp_path / "c.json", tmp_path / "c.md"
    subprocess.run([sys.executable, os.path.join(ROOT, "paper_2609_26638_amd", "rocprof_summary.py"),
                    "steps", "--fetch", str(tmp_path / "f"), "--write", str(tmp_path / "w"),
                    "--meta", str(tmp_path / "meta.json"), "--title", "t", "--command", "cmd",
                    "--out-json", str(js), "--out-md", str(md)], check=True, capture_output=True)
    res = json.loads(js.read_text())
    # per step: fetch (1 + 20 + 4) KiB x 2, write (1 + 20 + 4) KiB x 1
    per_step = 25 * 1024 * 2.0 + 25 * 1024 * 1.0
    assert res["bytes_per_step"] == pytest.approx(per_step)
    assert res["traffic_over_algorithmic"] == pytest.approx(per_step / 50000)
    assert res["src_hash"] == "abc"
    assert [k["kernel"] for k in res["kernels"]][0] == "gemm_ws_kernel"
    assert "| `gemm_ws_kernel` | 1.0 |" in md.read_text()


def test_step_times_window(tmp_path):
    d = tmp_path / "t"
    os.makedirs(d)
    # (kernel, start us, duration us): warmup step, copy for a host read,
    # two measured steps, the calibration copy, a later small copy
    seq = [("embed_rows_kernel", 0, 1), ("gemm_ws_kernel", 2, 5),
           ("__amd_rocclr_copyBuffer", 10, 1),
           ("embed_rows_kernel", 20, 1), ("gemm_ws_kernel", 22, 5),
           ("embed_rows_kernel", 30, 1), ("gemm_ws_kernel", 32, 7),
           ("__amd_rocclr_copyBuffer", 50, 400), ("__amd_rocclr_copyBuffer", 460, 2)]
    with open(d / "run_kernel_trace.csv", "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        for name, t, dt in seq:
            w.writerow([name, t * 1000, (t + dt) * 1000])
    span, ks = rs.step_times(str(d), "embed_rows", 2)
    assert span == pytest.approx(19.0)                 # 20 us .. 39 us
    assert ks[0] == ("gemm_ws_kernel", 2, pytest.approx(12.0))
    assert [k for k, _, _ in ks] == ["gemm_ws_kernel", "embed_rows_kernel"]


def test_source_hashes_ignore_comments():
    sys.path.insert(0, ROOT)
    import bench
    src = "int a; // note\n/* block\n comment */ int  b;\n"
    assert bench._code_only(src) == bench._code_only("int a;\nint b;")
    assert bench._code_only(src) != bench._code_only("int a; int c;")
    h1, h2 = bench.attn_source_hash(), bench.stack_source_hash()
    assert len(h1) == 16 and len(h2) == 16 and h1 != h2
