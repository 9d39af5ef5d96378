"""Host-side pieces of bench.py: the op model behind roofline.achieved, the
traffic table's tie to the kernel source, and the refusals that need no GPU."""
import json
import os
import subprocess
import sys

import numpy as np
import pytest

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


def test_counters_are_tied_to_the_kernel_code(tmp_path, monkeypatch):
    src = tmp_path / "k.hip"
    src.write_text("int a;  // one\n\n// two\nint b;\n")
    monkeypatch.setattr(bench, "KERNEL_SOURCES", [str(src)])
    h = bench.kernel_source_hash()
    src.write_text("int a;\n// edited comment\nint b;   // another\n")
    assert bench.kernel_source_hash() == h          # comments and blank lines do not count
    key = ("covtype_med", "f32", False)
    monkeypatch.setattr(bench, "COUNTERS", {key: {
        "fetch_bytes": 3e6, "write_bytes": 4e6, "valu_insts": 1024 * 2.4e6 * 0.2,
        "salu_insts": 1, "lds_insts": 2, "source": h}})
    assert bench.traffic_for(key) == 7e6
    ex = bench.executed(key, 1.0)                   # 1 ms
    assert abs(ex["hbm_gbps"] - 7.0) < 1e-9
    assert abs(ex["valu_issue_per_simd_cycle"] - 0.2) < 1e-12
    assert abs(ex["valu_issue_frac_of_ceiling"] - 0.2 / bench.VALU_ISSUE_CEILING) < 1e-12
    assert bench.traffic_for(("wide", "f32", False)) is None
    src.write_text("int a;\nint c;\n")              # code changed: the counters no longer apply
    assert bench.traffic_for(key) is None and bench.executed(key, 1.0) is None


def test_kernel_sources_exist():
    for path in bench.KERNEL_SOURCES:
        assert os.path.exists(path), path


@pytest.mark.parametrize("name,dtype", [("tiny", "f64"), ("covtype_med", "f32")])
def test_live_pairs_match_a_direct_count(name, dtype):
    """The roofline's live (row, path) pairs, counted with torch on the CPU,
    against a direct per-path loop: a pair is dead when some element with
    zero fraction 0 has a range that misses the row."""
    import torch
    w = synth.workload(name, rows=200)
    X = w.X
    q, lr, lt = bench.live_pairs(torch, gts, w.ensemble, X, dtype, tile=64, dev="cpu")
    el, _, _ = gts.extract_paths(w.ensemble)
    roots = np.flatnonzero(el["feature_idx"] == -1)
    ends = np.append(roots[1:], len(el))
    ft = np.float32 if dtype == "f32" else np.float64
    for p, (a, e) in enumerate(zip(roots, ends)):
        seg = el[a + 1:e]
        z0 = seg[seg["zero_fraction"].astype(ft) == 0]
        ok = np.ones(len(X), bool)
        for f, lo, hi in zip(z0["feature_idx"], z0["lower"], z0["upper"]):
            ok &= (lo <= X[:, f]) & (X[:, f] < hi)
        assert q[p] == e - a - 1
        assert lr[p] == ok.sum(), p
        assert lt[p] == sum(ok[t:t + 64].any() for t in range(0, len(X), 64)), p
    assert (lr < len(X)).any()      # these models do have dead pairs


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
