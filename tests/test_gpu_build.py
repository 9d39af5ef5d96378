"""gts_plan_model + gts_build_model_device: the model blob written on the GPU
from the host's plan equals gts_prepare_model's blob byte for byte
(extraction and merging of Sections 3.1-3.2 on the device, the packing of
Section 3.3 on the host), and SHAP values on it match the oracle."""
import ctypes

import numpy as np
import pytest

from paper_2010_13972_amd import gts, synth
from parity import assert_parity
from test_gpu_shap import empty_ensemble, sample_rows, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    return torch


def device_blob(torch, ens, dtype):
    desc, plan, hp = gts.plan_model(ens, dtype)
    dens = gts.DeviceEnsemble(ens)
    d_plan = torch.from_numpy(np.ascontiguousarray(hp)).cuda()
    model = gts.build_model_device(dens, desc, plan, d_plan, dtype)
    torch.cuda.synchronize()
    return model, model.blob.cpu().numpy()


def chain(depth, M):
    nodes, cover = [], 1000.0
    for d in range(depth):
        b = len(nodes)
        nodes.append((b + 2, b + 1, d % M, np.float32(0.5 + 0.001 * d), cover, 0.0))
        nodes.append((-1, -1, -1, 0.0, 0.0 if d % 3 == 0 else 1.0, 0.25 * d))
        cover -= 0.0 if d % 3 == 0 else 1.0
    nodes.append((-1, -1, -1, 0.0, cover, 1.0))
    return nodes


def stumps(n):
    """n small trees: single leaves, one-split stumps and two-split trees, so a
    wave of 64 paths spans up to 64 trees and the tree search takes two rounds
    of probes."""
    trees = []
    for k in range(n):
        c = 100.0 + k
        if k % 3 == 0:
            trees.append([(-1, -1, -1, 0.0, c, 0.01 * k)])
        elif k % 3 == 1:
            trees.append([(1, 2, k % 5, np.float32(0.1 * (k % 7)), c, 0.0),
                          (-1, -1, -1, 0.0, c - 1.0 - (k % 4), -0.5),
                          (-1, -1, -1, 0.0, 1.0 + (k % 4), 0.5 + 0.001 * k)])
        else:
            trees.append([(1, 2, k % 5, np.float32(0.2), c, 0.0),
                          (3, 4, (k + 1) % 5, np.float32(-0.3), c - 10.0, 0.0),
                          (-1, -1, -1, 0.0, 10.0, 1.0),
                          (-1, -1, -1, 0.0, 0.0, 2.0 - 0.01 * k),
                          (-1, -1, -1, 0.0, c - 10.0, -1.0)])
    return synth.ensemble_from_lists(trees, M=5, num_groups=2)


# random<s>: M = 5 + 3 s (fp64 plans need M <= 11)
CASES = [("tiny", "f64"), ("deep", "f32"), ("deep", "f64"), ("random0", "f32"), ("random1", "f64"),
         ("random2", "f64"), ("random3", "f32"), ("chain64", "f32"), ("chain64", "f64"),
         ("stumps", "f32"), ("stumps", "f64"), ("empty", "f32")]


def case(name):
    if name.startswith("random"):
        s = int(name[6:])
        return synth.random_workload(40 + s, num_trees=16, max_depth=8, M=5 + 3 * s,
                                     num_groups=3, n_bg=30, rows=50).ensemble
    if name == "chain64":
        return synth.ensemble_from_lists([chain(64, 7), chain(30, 7)], M=7, num_groups=2,
                                         tree_group=[1, 0])
    if name == "stumps":
        return stumps(300)
    if name == "empty":
        return empty_ensemble(4, 2)
    return synth.workload(name).ensemble


@pytest.mark.parametrize("name,dtype", CASES, ids=[f"{n}-{d}" for n, d in CASES])
def test_device_blob_equals_host_blob(torch, name, dtype):
    ens = case(name)
    say("device build", name, dtype)
    _, got = device_blob(torch, ens, dtype)
    desc, want, _ = gts.prepare_blob(ens, dtype)
    assert got.nbytes == want.nbytes == desc.bytes
    if got.tobytes() != want.tobytes():
        bad = np.flatnonzero(got != want)
        raise AssertionError(f"{name}: {len(bad)} bytes differ, first at {bad[:8]} "
                             f"(array offsets {list(desc.off[:7])})")


@pytest.mark.parametrize("dtype", ["f32", "f64"])
def test_shap_on_a_device_built_model(torch, orc, dtype):
    w = synth.random_workload(7, num_trees=12, max_depth=7, M=6, num_groups=2, n_bg=40, rows=45)
    model, _ = device_blob(torch, w.ensemble, dtype)
    # the bias lives in the blob; the binding's copy is the host's
    Xd = torch.from_numpy(w.X).cuda()
    got = gts.shap(model, Xd)
    torch.cuda.synchronize()
    assert_parity(got.cpu().numpy(), orc.treeshap(w.ensemble, w.X), dtype, what="device-built")


def test_plan_and_ensemble_must_match(torch):
    a = synth.random_workload(1, num_trees=4, max_depth=5, M=5, rows=4).ensemble
    b = synth.random_workload(2, num_trees=5, max_depth=5, M=5, rows=4).ensemble
    desc, plan, hp = gts.plan_model(a, "f32")
    dens = gts.DeviceEnsemble(b)
    d_plan = torch.from_numpy(hp).cuda()
    with pytest.raises(gts.GtsError) as e:
        gts.build_model_device(dens, desc, plan, d_plan, "f32")
    assert e.value.status == gts.GTS_EINVAL and "belong together" in str(e.value)
    dens = gts.DeviceEnsemble(a)
    out = torch.empty(desc.bytes, dtype=torch.uint8, device="cuda")
    ws = torch.empty(gts.build_workspace_bytes(plan), dtype=torch.uint8, device="cuda")
    st = gts.lib().gts_build_model_device(ctypes.byref(dens.struct), ctypes.byref(desc),
                                          ctypes.byref(plan), ctypes.c_void_p(d_plan.data_ptr()),
                                          ctypes.c_void_p(out.data_ptr()),
                                          ctypes.c_void_p(ws.data_ptr()), ws.numel() - 8, None)
    assert st == gts.GTS_EBUFSIZE
    torch.cuda.synchronize()
