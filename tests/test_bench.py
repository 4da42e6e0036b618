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


def test_sweep_summary_maps_launches_to_cells(tmp_path):
    """--summarize-sweep walks the trace in sweep order, one step per scan
    launch: per cell its warm-up steps (replicas) are skipped and the medians
    of the timed steps are kept; a softmax_stats launch counts where a step has
    one; a cell's scan GB/s are its algorithmic bytes over that median."""
    from paper_2602_18750_amd import workloads as W
    names = {"scan": "void hill::score_tiles_kernel<4, 0, hill::KeysF16<1, 4> >(hill::ScoreArgs)",
             "stats": "hill::softmax_stats_kernel(float2 const*, float2*, int, int)",
             "update": "hill::update_attn_kernel(hill::UpdateArgs)",
             "refine": "hill::topk_refine_kernel(hill::RefineArgs)",
             "select": "void hill::topk_emit_kernel<1, 4, true, false, true, false>(hill::RefineArgs, hill::AttnArgs)",
             "merge": "hill::merge_write_kernel(hill::RefineArgs, hill::AttnArgs, int*)"}
    seq = []
    for ci, w in enumerate(W.sweep_workloads()):
        kv = 2 * w.batch * w.n_kv_heads * w.n_tokens * w.head_dim * 2
        reps = max(1, min(16, -(-(1 << 30) // kv)))
        for i in range(reps + max(20, reps)):
            warm = i < reps
            # warm-up steps take 10x longer: they must not reach the medians
            seq += [(names["scan"], (1000 + ci) * (10 if warm else 1))]
            if w.n_tokens > 32768:   # some steps reduce the partials in a launch of their own
                seq += [(names["stats"], 700)]
            seq += [(names["update"], 2000), (names["refine"], 3000), (names["select"], 4000 + ci),
                    (names["merge"], 5000)]
    _trace(tmp_path / "s_kernel_trace.csv", seq)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--summarize-sweep", str(tmp_path)],
                       capture_output=True, text=True, cwd=ROOT, timeout=120)
    assert r.returncode == 0, r.stderr
    rows = [l for l in r.stdout.splitlines() if l.startswith("| ") and "K," in l]
    assert len(rows) == 27
    first = [c.strip() for c in rows[0].split("|")[1:-1]]
    assert first[0] == "1, 8K, 5%" and first[2] == "1.00" and first[5] == "0.00" and first[6] == "2.00"
    assert first[8] == "4.00" and first[10] == "%.2f" % (1.0 + 2.0 + 3.0 + 4.0 + 5.0)
    nbytes = bench.scan_kernel_bytes(1, 32, 8, 128, 8192)
    assert first[3] == "%.0f" % (nbytes / 1e-6 / 1e9)
    last = [c.strip() for c in rows[-1].split("|")[1:-1]]
    assert last[0] == "32, 64K, 20%" and last[2] == "%.2f" % ((1000 + 26) * 1e-3) and last[8] == "%.2f" % ((4000 + 26) * 1e-3)
    assert last[5] == "0.70" and last[6] == "2.00"
