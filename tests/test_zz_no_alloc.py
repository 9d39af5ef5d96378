"""gts_extract_paths_device_noalloc (the allocation-free variant of the
device path extraction, Sections 3.1-3.2) against gts_extract_paths_device
with a caller workspace: the same elements and bias, byte for byte, on two
calls in a row, the second on a smaller ensemble, and the size limit."""
import numpy as np
import pytest

from paper_2010_13972_amd import gts, synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    return torch


def both(torch, ens):
    dens = gts.DeviceEnsemble(ens)
    raw, npaths, bias = gts.extract_paths_device(dens)
    raw2, npaths2, bias2 = gts.extract_paths_device_noalloc(dens)
    torch.cuda.synchronize()
    return (raw.cpu().numpy().tobytes(), npaths, bias.cpu().numpy().tobytes(),
            raw2.cpu().numpy().tobytes(), npaths2, bias2.cpu().numpy().tobytes())


def test_two_calls_in_a_row_second_smaller(torch):
    for name in ("deep", "covtype_med"):   # 646k nodes, then 18k
        print("noalloc extraction", name, flush=True)
        w = synth.workload(name, rows=1)
        a, pa, ba, b, pb, bb = both(torch, w.ensemble)
        assert pa == pb and a == b and ba == bb, name
        # and the host extraction, itself bit-exact to the oracle's
        el, npaths, bias = gts.extract_paths(w.ensemble)
        assert npaths == pb and el.tobytes() == b and bias.tobytes() == bb


def test_errors_and_limit(torch):
    # a malformed ensemble: the same status as the caller-workspace call
    good = [(1, 2, 0, 0.5, 10.0, 0.0), (-1, -1, -1, 0, 4.0, 1.0), (-1, -1, -1, 0, 6.0, 2.0)]
    bad = [(1, 5, 0, 0.5, 10.0, 0.0)] + good[1:]
    dens = gts.DeviceEnsemble(synth.ensemble_from_lists([good, bad], M=2))
    with pytest.raises(gts.GtsError) as err:
        gts.extract_paths_device_noalloc(dens)
    assert err.value.status == gts.GTS_EINVAL
    # an ensemble whose workspace exceeds the fixed array: refused before any
    # device work
    n = 700_000
    stump = synth.ensemble_from_lists([good], M=2)
    big = synth.Ensemble(
        num_features=2, num_groups=1,
        tree_node_offsets=np.arange(n + 1, dtype=np.int64) * 3,
        tree_group=np.zeros(n, np.int32), left=np.tile(stump.left, n),
        right=np.tile(stump.right, n), feature=np.tile(stump.feature, n),
        threshold=np.tile(stump.threshold, n), cover=np.tile(stump.cover, n),
        value=np.tile(stump.value, n))
    dens = gts.DeviceEnsemble(big)
    with pytest.raises(gts.GtsError) as err:
        gts.extract_paths_device_noalloc(dens)
    assert err.value.status == gts.GTS_EINVAL and "workspace" in str(err.value)
    # a small model still works afterwards
    w = synth.workload("tiny", rows=1)
    a, pa, ba, b, pb, bb = both(torch, w.ensemble)
    assert pa == pb and a == b and ba == bb
