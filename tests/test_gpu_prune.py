"""gts_prune_model on the GPU: the model without the paths no row of a batch
reaches (a zero-fraction element whose range holds no row's value; such a
path contributes exactly nothing, the zero-cover pruning of Algorithm 1).

- SHAP values and interaction values on the pruned model against the fp64
  oracle (and against the unpruned model), on random edge-case ensembles, the
  tiny and covtype-shaped models and the deep model in the benchmark's launch
  configuration;
- the kept paths themselves: read back from the device and compared byte for
  byte with the paths a plain numpy evaluation of the same predicate keeps
  from the host blob, and the bins' structure (one path length per bin,
  64 / length paths per bin, groups in order, longest paths first);
- batches larger than one sorted chunk of keys, batches that reach no
  zero-cover path at all or every path, models without trees, and the error
  statuses.
"""
import ctypes

import numpy as np
import pytest

from paper_2010_13972_amd import gts, synth
from parity import assert_parity
from test_gpu_shap import empty_ensemble, sample_rows, say

pytestmark = pytest.mark.gpu

F32, F64 = "f32", "f64"


@pytest.fixture(scope="module")
def torch():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    return torch


def device_X(torch, X):
    return torch.from_numpy(np.ascontiguousarray(X, np.float32)).cuda()


def pruned_shap(torch, ens, X, dtype, interactions=False):
    model = gts.prepare(ens, dtype)
    Xd = device_X(torch, X)
    pm = gts.prune(model, Xd)
    fn = gts.shap_interactions if interactions else gts.shap
    got = fn(pm, Xd)
    full = fn(model, Xd)
    torch.cuda.synchronize()
    return got.cpu().numpy().astype(np.float64), full.cpu().numpy().astype(np.float64)


# --------------------------------------------------------------------------
# blob parsing (host side, independent of the pruning code)
# --------------------------------------------------------------------------

def blob_arrays(desc, blob: np.ndarray, dtype, num_elements, num_bins):
    zt = np.float64 if dtype == F64 else np.float32
    G = desc.num_groups

    def arr(k, t, n):
        o = desc.off[k]
        return np.frombuffer(blob[o:o + n * np.dtype(t).itemsize].tobytes(), t)

    return dict(feat=arr(0, np.int32, num_elements), lower=arr(1, np.float32, num_elements),
                upper=arr(2, np.float32, num_elements), zero=arr(3, zt, num_elements),
                bin_start=arr(4, np.int32, num_bins + 1), group_bins=arr(5, np.int32, G + 1),
                bias=arr(6, zt, G))


def path_table(a, G):
    """Per path (blob order): its first element, its length, its group and
    its bin; every path starts at a root (feat < 0) and ends at the next."""
    E = int(a["bin_start"][-1])
    feat = a["feat"][:E]
    starts = np.flatnonzero(feat < 0)
    ends = np.append(starts[1:], E)
    bins = np.searchsorted(a["bin_start"], starts, "right") - 1
    groups = np.searchsorted(a["group_bins"], bins, "right") - 1
    return starts, ends - starts, groups, bins


def blob_paths(a, G):
    """[(group, bytes of the path's elements)] in blob order, and the paths of
    every bin as (group, [lengths])."""
    starts, lens, groups, bins = path_table(a, G)
    paths = []
    for s, n, g in zip(starts.tolist(), lens.tolist(), groups.tolist()):
        sl = slice(s, s + n)
        paths.append((g, a["feat"][sl].tobytes() + a["lower"][sl].tobytes() +
                      a["upper"][sl].tobytes() + a["zero"][sl].tobytes()))
    nb = len(a["bin_start"]) - 1
    counts = np.bincount(bins, minlength=nb)
    bin_group = np.searchsorted(a["group_bins"], np.arange(nb), "right") - 1
    per_bin = [(int(g), l.tolist())
               for g, l in zip(bin_group, np.split(lens, np.cumsum(counts)[:-1]))]
    return paths, per_bin


def kept_by_numpy(a, G, X):
    """The paths a plain evaluation keeps: none of its zero-fraction elements
    (the first -1 - feat after the root) has a [lower, upper) that holds no
    row's value.  Per feature, the rows' sorted values and one search per
    element."""
    starts, lens, groups, _ = path_table(a, G)
    feat = a["feat"]
    n0 = -1 - feat[starts]
    pid = np.repeat(np.arange(len(starts)), lens)
    pos = np.arange(int(lens.sum())) - np.repeat(starts, lens)
    idx = np.flatnonzero((pos >= 1) & (pos <= n0[pid]))
    hit = np.zeros(len(idx), bool)
    for f in np.unique(feat[idx]):
        m = feat[idx] == f
        S = np.sort(X[:, f])
        k = np.searchsorted(S, a["lower"][idx[m]], "left")
        hit[m] = (k < len(S)) & (S[np.minimum(k, len(S) - 1)] < a["upper"][idx[m]])
    dead = np.zeros(len(starts), bool)
    dead[pid[idx[~hit]]] = True
    paths, _ = blob_paths(a, G)
    return [p for p, d in zip(paths, dead) if not d]


def read_pruned(torch, pm):
    host = pm.blob.cpu().numpy()
    G = pm.num_groups
    gb = np.frombuffer(host[pm.desc.off[5]:pm.desc.off[5] + 4 * (G + 1)].tobytes(), np.int32)
    nb = int(gb[G])
    bs = np.frombuffer(host[pm.desc.off[4]:pm.desc.off[4] + 4 * (nb + 1)].tobytes(), np.int32)
    return blob_arrays(pm.desc, host, pm.dtype, int(bs[nb]), nb)


# --------------------------------------------------------------------------
# values against the oracle
# --------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("dtype", [F64, F32])
def test_random_edge_case_ensembles(torch, orc, seed, dtype):
    """Repeated features, ties, zero-cover nodes, three output groups: values
    on the pruned model against Algorithm 1 and the unpruned model."""
    w = synth.random_workload(seed, num_trees=14, max_depth=8, M=6, num_groups=3, n_bg=30,
                              rows=41 + 23 * seed)
    say("prune random", seed, dtype)
    got, full = pruned_shap(torch, w.ensemble, w.X, dtype)
    want = orc.treeshap(w.ensemble, w.X)
    assert_parity(got, want, dtype, what=f"pruned random{seed}")
    assert_parity(full, want, dtype, what=f"unpruned random{seed}")


@pytest.mark.parametrize("dtype", [F64, F32])
def test_interactions_on_pruned_models(torch, orc, dtype):
    for seed in range(3):
        w = synth.random_workload(40 + seed, num_trees=8, max_depth=7, M=6, num_groups=2,
                                  n_bg=30, rows=33)
        say("prune interactions", seed, dtype)
        got, _ = pruned_shap(torch, w.ensemble, w.X, dtype, interactions=True)
        assert_parity(got, orc.interactions(w.ensemble, w.X), dtype, 2, f"pruned inter{seed}")


@pytest.mark.parametrize("name,dtype", [("tiny", F64), ("covtype_med", F32)])
def test_workload_models(torch, orc, name, dtype):
    w = synth.workload(name)
    rows = sample_rows(w.X.shape[0], k=40, seed=3)
    say("prune workload", name, dtype)
    got, full = pruned_shap(torch, w.ensemble, w.X, dtype)
    assert_parity(got[rows], orc.treeshap(w.ensemble, w.X[rows]), dtype, what=name)
    assert_parity(got, full, dtype, what=f"{name} pruned vs unpruned")


@pytest.mark.parametrize("dtype", [F32, F64])
def test_deep_model_full_batch(torch, orc, dtype):
    """The deep model (1000 trees, 10k rows, the benchmark's launch): about 90 %
    of its paths are dropped; every row against the unpruned model (itself
    checked against the oracle on every row in test_gpu_shap) and 40 rows
    against the oracle."""
    w = synth.workload("deep")
    say("prune deep", dtype)
    got, full = pruned_shap(torch, w.ensemble, w.X, dtype)
    assert_parity(got, full, dtype, what="deep pruned vs unpruned")
    rows = sample_rows(w.X.shape[0], k=32, seed=9)
    assert_parity(got[rows], orc.treeshap(w.ensemble, w.X[rows]), dtype, what="deep vs oracle")


@pytest.mark.parametrize("name", ["wide", "interactions"])
def test_full_size_wide_and_interaction_batches(torch, orc, name):
    """The wide model (784 features, 10 groups, 10k rows; the multi-path
    launch) and the 1000-row interaction batch: every row against the
    unpruned model (itself checked against the oracle in test_gpu_shap and
    test_gpu_interactions), and sampled rows against the oracle."""
    w = synth.workload(name)
    inter = name == "interactions"
    say("prune full size", name)
    got, full = pruned_shap(torch, w.ensemble, w.X, F32, interactions=inter)
    blocks = 2 if inter else 1
    assert_parity(got, full, F32, blocks, f"{name} pruned vs unpruned")
    rows = sample_rows(w.X.shape[0], k=6 if inter else 8, seed=11)
    want = (orc.interactions if inter else orc.treeshap)(w.ensemble, w.X[rows])
    assert_parity(got[rows], want, F32, blocks, f"{name} vs oracle")


# --------------------------------------------------------------------------
# the kept paths and the bins
# --------------------------------------------------------------------------

CASES = [("random", 0, F32), ("random", 1, F64), ("random", 2, F32), ("groups20", 0, F32),
         ("covtype_med", 0, F32), ("deep", 0, F32), ("wide", 0, F32)]


@pytest.mark.parametrize("name,seed,dtype", CASES, ids=[f"{n}{s}-{d}" for n, s, d in CASES])
def test_kept_paths_bit_exact(torch, name, seed, dtype):
    if name == "random":
        w = synth.random_workload(50 + seed, num_trees=20, max_depth=8, M=5, num_groups=3,
                                  n_bg=25, rows=60)
    elif name == "groups20":
        # 20 output groups: 1280 (group, length) classes, more than one block
        # of the planning scan
        w = synth.random_workload(60, num_trees=60, max_depth=7, M=5, num_groups=20, n_bg=25,
                                  rows=45)
    else:
        w = synth.workload(name)
    ens = w.ensemble
    desc, blob, bias = gts.prepare_blob(ens, dtype)
    orig = blob_arrays(desc, blob, dtype, desc.num_elements, desc.num_bins)
    want = kept_by_numpy(orig, ens.num_groups, w.X.astype(np.float32))
    model = gts.upload(desc, blob, ens.num_features, ens.num_groups, dtype, bias)
    pm = gts.prune(model, device_X(torch, w.X))
    torch.cuda.synchronize()
    assert pm.desc.flags & 2 and pm.desc.flags & 1
    got_a = read_pruned(torch, pm)
    got, bins = blob_paths(got_a, ens.num_groups)
    say("kept paths", name, seed, dtype, len(want), "of", desc.num_paths)
    # the same multiset of (group, path) records
    assert sorted(got) == sorted(want)
    # groups in order, every bin one length, 64 // length paths per bin except
    # a length's last bin, lengths non-increasing within a group
    for g in range(ens.num_groups):
        gl = [lens for gg, lens in bins if gg == g]
        flat = [l for lens in gl for l in lens]
        assert flat == sorted(flat, reverse=True)
        for i, lens in enumerate(gl):
            assert len(set(lens)) == 1 and len(lens) <= 64 // lens[0]
            last = i + 1 == len(gl) or gl[i + 1][0] != lens[0]
            assert last or len(lens) == 64 // lens[0]
    assert np.array_equal(got_a["bias"], orig["bias"])


def test_batches_beyond_one_sorted_chunk(torch, orc):
    """40 000 rows: more than one sorted chunk of keys per feature (16 384 at
    most); a path is kept when any chunk has a row in range."""
    w = synth.random_workload(77, num_trees=12, max_depth=8, M=5, num_groups=2, n_bg=30,
                              rows=40000)
    X = w.X.astype(np.float32)
    say("prune chunks", X.shape)
    got, full = pruned_shap(torch, w.ensemble, X, F32)
    assert_parity(got, full, F32, what="40000 rows pruned vs unpruned")
    rows = sample_rows(X.shape[0], k=24, seed=4)
    assert_parity(got[rows], orc.treeshap(w.ensemble, X[rows]), F32, what="40000 rows")
    # the kept paths equal the numpy evaluation on the whole batch
    desc, blob, bias = gts.prepare_blob(w.ensemble, F32)
    orig = blob_arrays(desc, blob, F32, desc.num_elements, desc.num_bins)
    want = kept_by_numpy(orig, w.ensemble.num_groups, X)
    model = gts.upload(desc, blob, w.ensemble.num_features, w.ensemble.num_groups, F32, bias)
    pm = gts.prune(model, device_X(torch, X))
    torch.cuda.synchronize()
    got_paths, _ = blob_paths(read_pruned(torch, pm), w.ensemble.num_groups)
    assert sorted(got_paths) == sorted(want)


def test_nothing_and_everything_dropped(torch, orc):
    """Stumps whose right child has zero cover: rows all left of the split
    reach none of the right paths (dropped: those paths contribute nothing,
    the values still match); a batch with no zero-cover path in reach keeps
    every path; a model without trees prunes to no bins."""
    rng = np.random.default_rng(5)
    trees = []
    for t in range(10):
        f = t % 3
        trees.append([(1, 2, f, 0.5, 10.0, 0.0), (-1, -1, -1, 0, 10.0, float(rng.normal())),
                      (-1, -1, -1, 0, 0.0, float(rng.normal()))])
    ens = synth.ensemble_from_lists(trees, M=3)
    for lo, hi, kept in ((0.0, 0.4, 10), (0.0, 1.0, 20)):
        X = rng.uniform(lo, hi, size=(50, 3)).astype(np.float32)
        for dtype in (F64, F32):
            model = gts.prepare(ens, dtype)
            Xd = device_X(torch, X)
            pm = gts.prune(model, Xd)
            got = gts.shap(pm, Xd)
            torch.cuda.synchronize()
            paths, _ = blob_paths(read_pruned(torch, pm), 1)
            say("prune stumps", lo, hi, dtype, len(paths))
            assert len(paths) == kept
            assert_parity(got.cpu().numpy(), orc.treeshap(ens, X), dtype, what=f"stumps {hi}")
    X = rng.uniform(0, 1, size=(20, 3)).astype(np.float32)
    model = gts.prepare(empty_ensemble(3, 2), F32)
    Xd = device_X(torch, X)
    pm = gts.prune(model, Xd)
    got = gts.shap(pm, Xd)
    torch.cuda.synchronize()
    assert np.all(got.cpu().numpy() == 0.0)
    assert read_pruned(torch, pm)["group_bins"].tolist() == [0, 0, 0]


def test_errors(torch):
    w = synth.random_workload(3, num_trees=3, max_depth=4, M=4, rows=10)
    model = gts.prepare(w.ensemble, F32)
    Xd = device_X(torch, w.X)
    pm = gts.prune(model, Xd)
    with pytest.raises(gts.GtsError) as e:
        gts.prune(pm, Xd)
    assert e.value.status == gts.GTS_EINVAL and "already pruned" in str(e.value)
    L = gts.lib()
    need = gts.prune_workspace_bytes(model, 10)
    ws = torch.empty(need + 512, dtype=torch.uint8, device="cuda")
    out = gts.ModelDesc()
    ptr = ctypes.c_void_p()
    args = (ctypes.byref(model.desc), ctypes.c_void_p(model.blob.data_ptr()),
            ctypes.c_void_p(Xd.data_ptr()), 10, Xd.stride(0))
    st = L.gts_prune_model(*args, ctypes.c_void_p(ws.data_ptr()), need - 1, ctypes.byref(out),
                           ctypes.byref(ptr), None)
    assert st == gts.GTS_EBUFSIZE
    st = L.gts_prune_model(*args, ctypes.c_void_p(ws.data_ptr() + 16), need, ctypes.byref(out),
                           ctypes.byref(ptr), None)
    assert st == gts.GTS_EINVAL and "aligned" in gts.last_error()
    st = L.gts_prune_model(*args, ctypes.c_void_p(ws.data_ptr()), need, None, ctypes.byref(ptr),
                           None)
    assert st == gts.GTS_EINVAL
    torch.cuda.synchronize()
