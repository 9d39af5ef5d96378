"""The host half of libgts under sanitizers, on the CPU.

tests/native/host_check.cpp is compiled with gts_host.cpp by g++ with
AddressSanitizer + UndefinedBehaviorSanitizer, and separately with
ThreadSanitizer (the worker pool, the parallel walks, the parallel sort and
the parallel blob writers, preparations from three threads at once).  It
prepares models of seeded ensembles for every packing heuristic and compares
them with the three-call route, and compares concurrent preparations with
one-at-a-time ones.  Any sanitizer report or mismatch fails the test.
"""
import os
import shutil
import subprocess

import numpy as np
import pytest

from paper_2010_13972_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = [os.path.join(ROOT, "tests", "native", "host_check.cpp"),
       os.path.join(ROOT, "paper_2010_13972_amd", "csrc", "gts_host.cpp")]
INC = ["-I", os.path.join(ROOT, "include"), "-I",
       os.path.join(ROOT, "paper_2010_13972_amd", "csrc")]

pytestmark = pytest.mark.slow


def _write_ensemble(e, d):
    np.array([e.num_features, e.num_groups, len(e.tree_group), len(e.left)],
             np.int64).tofile(os.path.join(d, "hdr.bin"))
    for name, arr, dt in (("off", e.tree_node_offsets, np.int64), ("grp", e.tree_group, np.int32),
                          ("left", e.left, np.int32), ("right", e.right, np.int32),
                          ("feat", e.feature, np.int32), ("thr", e.threshold, np.float32),
                          ("cov", e.cover, np.float64), ("val", e.value, np.float64)):
        np.asarray(arr, dt).tofile(os.path.join(d, name + ".bin"))


def _build(tmp, flags, name):
    if shutil.which("g++") is None:
        pytest.skip("g++ not available")
    exe = os.path.join(tmp, name)
    cmd = ["g++", "-O1", "-g", "-std=c++17", "-ffp-contract=off", *flags, *INC, *SRC, "-o", exe,
           "-lpthread"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        pytest.skip(f"sanitizer build unavailable: {res.stderr[-300:]}")
    return exe


def _cases():
    yield "covtype_med", synth.workload("covtype_med").ensemble
    yield "wide", synth.workload("wide").ensemble
    for s in range(3):
        yield f"random{s}", synth.random_workload(s, num_trees=12, max_depth=7, M=5,
                                                  num_groups=3, n_bg=40, rows=4).ensemble


@pytest.mark.parametrize("kind,flags", [
    ("asan", ["-fsanitize=address,undefined", "-fno-omit-frame-pointer",
              "-fno-sanitize-recover=undefined"]),
    ("tsan", ["-fsanitize=thread"]),
])
def test_host_library_under_sanitizers(tmp_path, kind, flags):
    exe = _build(str(tmp_path), flags, "host_check_" + kind)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
               TSAN_OPTIONS="halt_on_error=1")
    for name, ens in _cases():
        d = tmp_path / name
        d.mkdir()
        _write_ensemble(ens, str(d))
        res = subprocess.run([exe], cwd=str(d), capture_output=True, text=True, env=env,
                             timeout=600)
        report = res.stdout + res.stderr
        assert res.returncode == 0, f"{kind} {name}:\n{report[-3000:]}"
        assert "runtime error" not in report and "WARNING: ThreadSanitizer" not in report, report
        assert report.count("same") >= 8, report
        assert report.count("concurrent") == 2 and "DIFFERENT" not in report, report
