"""bench.py's host logic, on the CPU (no GPU, no library calls):

- a run asked for more than one GPU exits with status 2 and says why, before
  it touches the GPU;
- --trace-summary takes the contract steps as the last `steps` launch
  triples (append, video, merge) of the first unbroken run of them, so the
  settle and warm-up steps before them, and the later passes (steps with a
  separate audio kernel, the breakdown's separate calls, other workloads),
  never enter the contract medians.
"""
import csv
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


KERNEL_NAMES = {
    "append": "kv_append_kernel(ws::AppendArgs)",
    "video": "unit_attn_kernel(ws::AttnArgs)",
    "audio": "audio_attn_kernel(ws::AttnArgs)",
    "step_merge": "step_combine_kernel(ws::CombineArgs, ws::CombineArgs, int)",
    "video_merge": "video_combine_kernel(ws::CombineArgs)",
    "merge": "combine_kernel(ws::CombineArgs)",
}
GRIDS = {"append": 1024, "video": 256, "audio": 480, "step_merge": 2310, "video_merge": 2300, "merge": 10}


def write_trace(path, launches):
    """launches: (kind, duration in us); 256-thread workgroups, 1 us apart."""
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Kernel_Name", "Start_Timestamp", "End_Timestamp", "Grid_Size_X", "Workgroup_Size_X",
                    "Grid_Size_Y", "Workgroup_Size_Y"])
        t = 10_000
        for kind, us in launches:
            ns = int(round(us * 1000))
            w.writerow([KERNEL_NAMES[kind], t, t + ns, GRIDS[kind] * 256, 256, 1, 1])
            t += ns + 1000


def test_trace_summary_takes_the_contract_steps(tmp_path, capsys):
    launches = []
    # settle and warm-up steps: slower while the clocks rise
    for i in range(30):
        launches += [("append", 25.0), ("video", 190.0 - i), ("step_merge", 9.0)]
    # the contract steps
    for i in range(20):
        launches += [("append", 19.0), ("video", 150.0 + (i % 3)), ("step_merge", 8.0)]
    # steps with the separate audio kernel: a triple never forms
    for _ in range(5):
        launches += [("append", 19.0), ("video", 152.0), ("audio", 28.0), ("step_merge", 8.0)]
    # the breakdown pass: separate calls
    for _ in range(4):
        launches += [("append", 19.0), ("video", 147.0), ("video_merge", 7.0), ("audio", 46.0), ("merge", 4.0)]
    # a later workload issuing the step again (a second run of triples)
    for _ in range(6):
        launches += [("append", 17.0), ("video", 140.0), ("step_merge", 12.0)]
    path = tmp_path / "kernel_trace.csv"
    write_trace(path, launches)
    bench.trace_summary(str(path), steps=20)
    out = capsys.readouterr().out
    assert "Contract steps (20 after 30 settle and warm-up steps, medians): append 19.00 us, " \
           "video 151.00 us, merge 8.00 us: 178.0 us of kernel time per step." in out
    assert "Breakdown pass (separate video calls): 4 unit_attn_kernel launches, average 147.00 us" in out
    # the table groups the video launches by workload (all of them 8536-key steps here)
    row = [ln for ln in out.splitlines() if ln.startswith("| unit_attn_kernel | 256 | v0.2 unit, 8536 keys |")]
    assert len(row) == 1 and f"| {30 + 20 + 5 + 4 + 6} |" in row[0]


def test_video_flop_counts_both_products():
    # S = Q K^T and O = P V: 2 * lq * lk * D multiply-adds per head, 2 FLOP each
    lq, lk = 920, 8536
    assert bench.video_flop(lq, lk) == 2 * 2 * bench.H * lq * lk * bench.D
    assert bench.video_flop(920, 8536) == 160831897600.0
