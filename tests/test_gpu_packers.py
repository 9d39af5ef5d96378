"""The kernels on models packed by every heuristic of Section 3.3 / Table 1
(BFD, FFD, NF, one path per bin) and at several bin capacities: packing only
decides which paths a wave takes together, so every packing must give the
oracle's values."""
import numpy as np
import pytest

from paper_2010_13972_amd import gts, synth
from parity import assert_parity
from test_gpu_shap import sample_rows, say

pytestmark = pytest.mark.gpu

ALGS = ["bfd", "ffd", "nf", "none"]


@pytest.fixture(scope="module")
def torch():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    return torch


@pytest.mark.parametrize("alg", ALGS)
@pytest.mark.parametrize("cap", [64, 32, 17])
def test_random_ensembles_any_packing(torch, orc, alg, cap):
    w = synth.random_workload(3, num_trees=14, max_depth=6, M=7, num_groups=3, n_bg=40, rows=77)
    say("packing", alg, cap)
    Xd = torch.from_numpy(w.X).cuda()
    want = orc.treeshap(w.ensemble, w.X)
    want_i = orc.interactions(w.ensemble, w.X)
    for dtype in ("f64", "f32"):
        model = gts.prepare(w.ensemble, dtype, bin_capacity=cap, alg=alg)
        phi = gts.shap(model, Xd)
        inter = gts.shap_interactions(model, Xd)
        torch.cuda.synchronize()
        assert_parity(phi.cpu().numpy(), want, dtype, what=f"{alg} B={cap} {dtype}")
        assert_parity(inter.cpu().numpy(), want_i, dtype, 2, what=f"{alg} B={cap} {dtype} inter")


@pytest.mark.parametrize("alg", ["ffd", "nf", "none"])
@pytest.mark.parametrize("name", ["covtype_med", "wide"])
def test_full_size_models_other_packings(torch, orc, alg, name):
    """The full models (all their paths) on a few hundred rows."""
    w = synth.workload(name, rows=300)
    say("packing full model", name, alg)
    Xd = torch.from_numpy(w.X).cuda()
    model = gts.prepare(w.ensemble, "f32", alg=alg)
    phi = gts.shap(model, Xd)
    torch.cuda.synchronize()
    rows = sample_rows(w.X.shape[0], k=12)
    assert_parity(phi.cpu().numpy()[rows], orc.treeshap(w.ensemble, w.X[rows]), "f32",
                  what=f"{name} {alg}")
