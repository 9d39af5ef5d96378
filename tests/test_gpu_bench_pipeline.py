"""The benchmark's pipelined step loop (bench.time_pipeline): every timed
step's output equals gts.shap's on the same model, in the loop's shapes --
the blob built on the device from a host plan or prepared on the host, one
or two compute streams, two or three preparations in flight -- so buffer
reuse, uploads of whichever step is ready and alternating streams never give
a kernel another step's model or output buffer."""
import os
import sys

import pytest

from paper_2010_13972_amd import gts, synth
from test_gpu_shap import say

pytestmark = pytest.mark.gpu

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402


@pytest.fixture(scope="module")
def torch():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    return torch


# (where the blob is built, compute streams (0: builds and prunings on one
# stream, kernels on another), preparations in flight)
CASES = [("device", 2, 3), ("device", 1, 2), ("host", 2, 3), ("device", 0, 3), ("host", 0, 2)]


@pytest.mark.parametrize("build,streams,preps", CASES,
                         ids=[f"{b}-{s or 'split'}streams-{p}preps" for b, s, p in CASES])
def test_every_step_matches_the_binding(torch, build, streams, preps):
    w = synth.random_workload(11, num_trees=80, max_depth=10, M=8, num_groups=2, n_bg=200,
                              rows=3000)
    Xd = torch.from_numpy(w.X).cuda()
    say("pipeline", build, streams, preps)
    steps = 12
    res = bench.time_pipeline(torch, gts, w.ensemble, Xd, "f32", steps, 2, False, max(1, streams),
                              preps, True, build == "device", None, keep_outputs=True,
                              split=streams == 0)
    kept, model = res[-1], res[5]
    ref = gts.shap(model, Xd)
    torch.cuda.synchronize()
    scale = float(ref.abs().max())
    assert len(kept) == steps and all(o is not None for o in kept)
    for k, out in enumerate(kept):
        err = float((out - ref).abs().max())
        assert err <= 1e-5 * scale, f"step {k}: max |difference| {err:.3g} (|phi| up to {scale:.3g})"
