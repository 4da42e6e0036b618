"""Host-side checks of bench.py: the algorithmic byte count the roofline is
priced on, the one-GPU contract, and the profile summary's steady-state
table (on a synthetic kernel trace)."""
import csv
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_scan_bytes_of_the_32k_workload():
    # 64 MiB of 16-bit keys + 32 heads x 32768 fp32 logits + 32 x 128 (max, sum) pairs
    assert bench.scan_kernel_bytes(1, 32, 8, 128, 32768) == 67108864 + 4194304 + 32768 == 71335936
    # odd unit counts round the pairs per head up to an even number
    assert bench.scan_kernel_bytes(1, 4, 4, 128, 300) == 4 * 300 * 256 + 4 * 300 * 4 + 4 * 2 * 8
    # RAW: keys plus one fp32 sum per token read and written
    assert bench.scan_kernel_bytes(2, 8, 2, 128, 1000, mode="raw") == 2 * 2 * 1000 * 256 + 2 * 1000 * 8


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, cwd=ROOT, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def _trace(path, names_durations):
    fields = ["Kind", "Kernel_Name", "Start_Timestamp", "End_Timestamp"]
    t = 1000
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=fields)
        w.writeheader()
        for name, d in names_durations:
            w.writerow({"Kind": "KERNEL_DISPATCH", "Kernel_Name": name, "Start_Timestamp": t, "End_Timestamp": t + d})
            t += d + 500


def test_steady_state_table(tmp_path):
    scan = "void hill::(anonymous namespace)::score_tiles_kernel<4, 0, hill::(anonymous namespace)::KeysF16<1, 4> >(hill::ScoreArgs)"
    upd = "hill::(anonymous namespace)::update_attn_kernel(hill::UpdateArgs)"
    emit = "void hill::(anonymous namespace)::topk_emit_kernel<1, 4, true, true, true>(hill::RefineArgs, hill::AttnArgs)"
    merge = "hill::(anonymous namespace)::merge_write_kernel(hill::RefineArgs, hill::AttnArgs, int*)"
    other = "void at::native::fill(float)"
    seq = [(other, 9000)]
    for i in range(9):   # the first third runs slower (no bound yet)
        slow = 3 if i < 3 else 1
        seq += [(scan, 16000), (upd, 8000), (emit, 9000 * slow), (merge, 4000)]
    _trace(tmp_path / "x_kernel_trace.csv", seq)
    lines = bench._steady_state(str(tmp_path / "x_kernel_trace.csv"), str(tmp_path))
    text = "\n".join(lines)
    assert "9 layer-steps in the trace, the last 6 used" in text
    assert "| hill::topk_emit_kernel<1, 4, true, true, true> | 9.00 |" in text
    assert "| hill::update_attn_kernel | 8.00 |" in text
