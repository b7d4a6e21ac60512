"""bench.py's command line on the CPU: it runs the p logical ranks on one GPU
and refuses more GPUs with a message and exit status 2, before touching any
device."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "ONE GPU" in r.stderr and r.stdout == ""


def test_launched_as_a_second_rank_is_refused():
    env = dict(os.environ, WORLD_SIZE="2")
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py")], capture_output=True,
                       text=True, timeout=120, env=env)
    assert r.returncode == 2


def test_trace_summary_splits_dispatches_by_workload(tmp_path):
    """--trace-summary attributes the executor's dispatches of a kernel trace
    to the workloads in the line's dispatch order (no GPU involved)."""
    import json
    line = {"metric": "m", "config": {"workload": "a"},
            "roofline": {"algorithmic_bytes": 8000, "kernel_ms": 0.001},
            "configs": {"b": {"roofline": {"algorithmic_bytes": 4000, "kernel_ms": 0.002}}},
            "dispatch_order": [["a", 2], ["b", 3]]}
    lp = tmp_path / "line.txt"
    lp.write_text("some log line\n" + json.dumps(line) + "\n")
    hdr = '"Kind","Dispatch_Id","Kernel_Name","Start_Timestamp","End_Timestamp"\n'
    rows = [(1, "optcc_exec_kernel<A>", 0, 1000), (2, "copyBuffer", 0, 5),
            (3, "optcc_exec_kernel<A>", 0, 3000), (4, "optcc_exec_kernel<B>", 0, 2000),
            (5, "optcc_exec_kernel<B>", 0, 2000), (6, "optcc_exec_kernel<B>", 0, 2000)]
    cp = tmp_path / "trace.csv"
    cp.write_text(hdr + "".join(f'"K",{d},"{k}",{a},{b}\n' for d, k, a, b in rows))
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--trace-summary",
                        str(cp), "--line", str(lp)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    out = r.stdout.splitlines()
    a = next(l for l in out if l.startswith("| a |"))
    b = next(l for l in out if l.startswith("| b |"))
    assert "| 2 | 2,000 | 1,000 | 3,000 |" in a and "| 4.0 |" in a   # 8000 B / 2000 ns
    assert "| 3 | 2,000 | 2,000 | 2,000 |" in b and "| 2.0 |" in b
