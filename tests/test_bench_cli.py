"""bench.py paths that need no GPU: the multi-GPU guard and the host-only
selector bench keep the one-JSON-line contract."""
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], cwd=ROOT,
                          capture_output=True, text=True, timeout=300)


def test_more_than_one_gpu_is_refused_with_a_message():
    r = _run("--gpus", "2")
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_selector_bench_prints_one_json_line():
    r = _run("--select")
    assert r.returncode == 0, r.stderr
    lines = [l for l in r.stdout.splitlines() if l.strip()]
    assert len(lines) == 1
    rec = json.loads(lines[0])["select"]
    assert rec["candidates"] > 0 and rec["us_per_call"] > 0 and rec["admitted"] >= 0


def test_percentiles_follow_the_nearest_rank_definition():
    """p_q is the observation at rank ceil(q N / 100) of the sorted values
    (the paper's evaluation, Section 5.1), not an interpolation."""
    sys.path.insert(0, ROOT)
    import bench
    v = list(range(20, 0, -1))               # 20 .. 1, unsorted
    assert bench.nearest_rank(v, 50) == 10   # rank 10 of 20
    assert bench.nearest_rank(v, 95) == 19   # rank 19
    assert bench.nearest_rank(v, 5) == 1     # rank 1
    w = [float(x) for x in range(1, 31)]
    assert bench.nearest_rank(w, 5) == 2.0   # ceil(1.5) = 2
    assert bench.nearest_rank(w, 95) == 29.0  # ceil(28.5) = 29
    assert bench.nearest_rank([7.0], 50) == 7.0
    d = bench.dist([3.0, 1.0, 2.0, 4.0])
    assert d["p50"] == 2.0 and d["p5"] == 1.0 and d["p95"] == 4.0 and d["mean"] == 2.5
