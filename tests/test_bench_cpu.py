"""Host-side pieces of bench.py: the op model behind roofline.achieved, the
traffic table's tie to the kernel source, and the refusals that need no GPU."""
import json
import os
import subprocess
import sys

import numpy as np

import bench
from paper_2010_13972_amd import gts, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_op_model_per_path():
    """F = 10q^2 + 8q per (row, path); interactions add q(q-1)(10q+4)."""
    q = np.array([0, 1, 2, 7])
    assert bench.modelled_flops(q, False) == 0 + 18 + 56 + 546
    assert bench.modelled_flops(q, True) == 620 + 0 + 0 + 48 + 3108


def test_path_features_count_the_extracted_elements():
    w = synth.workload("tiny")
    q = bench.path_features(gts, w.ensemble)
    el, num_paths, _ = gts.extract_paths(w.ensemble)
    assert len(q) == num_paths == 80
    assert int((q + 1).sum()) == len(el)
    assert q.min() >= 1 and q.max() <= 3   # depth-3 trees, repeats merged


def test_traffic_is_tied_to_the_kernel_code(tmp_path, monkeypatch):
    src = tmp_path / "k.hip"
    src.write_text("int a;  // one\n\n// two\nint b;\n")
    monkeypatch.setattr(bench, "KERNEL_SOURCE", str(src))
    h = bench.kernel_source_hash()
    src.write_text("int a;\n// edited comment\nint b;   // another\n")
    assert bench.kernel_source_hash() == h          # comments and blank lines do not count
    key = ("covtype_med", "f32", False)
    monkeypatch.setattr(bench, "TRAFFIC", {key: {"fetch_bytes": 3, "write_bytes": 4, "source": h}})
    assert bench.traffic_for(key) == 7
    assert bench.traffic_for(("wide", "f32", False)) is None
    src.write_text("int a;\nint c;\n")              # code changed: the counters no longer apply
    assert bench.traffic_for(key) is None


def run_bench(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args],
                          capture_output=True, text=True, timeout=120, cwd=ROOT)


def test_more_than_one_gpu_is_refused():
    r = run_bench("--gpus", "2")
    assert r.returncode == 2
    line = json.loads(r.stdout.strip().splitlines()[-1])
    assert line["n_gpus"] == 2 and "one GPU" in line["error"]


def test_empty_step_counts_are_refused():
    for args in (("--steps", "0"), ("--streams", "0"), ("--warmup", "-1")):
        r = run_bench(*args)
        assert r.returncode == 2 and "at least" in r.stderr
