"""libgts host calls against the oracle, on the CPU.

Extraction (Sections 3.1-3.2), the bias and Best-Fit-Decreasing packing
(Section 3.3) must match the oracle's independent implementations bit for
bit.  Also: every symbol of include/gts.h is exported, and malformed input
is rejected with the documented status.
"""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2010_13972_amd import gts, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_library_exports_every_declared_symbol():
    header = open(os.path.join(ROOT, "include", "gts.h")).read()
    names = set(re.findall(r"^\S.*?\b(gts_\w+)\(", header, flags=re.M))
    assert {"gts_extract_paths", "gts_pack_paths", "gts_model_layout", "gts_shap",
            "gts_shap_interactions", "gts_last_error", "gts_version"} <= names
    L = gts.lib()
    for n in sorted(names):
        assert hasattr(L, n), f"libgts.so does not export {n}"
    assert "gfx950" in gts.version()


def _as_oracle_fields(el):
    return (el["path_idx"], el["feature_idx"], el["group"], el["lower"], el["upper"],
            el["zero_fraction"], el["v"])


def _assert_bitwise(a, b):
    a = np.asarray(a)
    b = np.asarray(b)
    assert a.shape == b.shape
    assert a.tobytes() == b.tobytes()


EXTRACT_CASES = ["tiny", "covtype_med", "wide", "random0", "random1", "random2", "random3"]


def _workload(name):
    if name.startswith("random"):
        s = int(name[6:])
        return synth.random_workload(s, num_trees=6, max_depth=7, M=5, num_groups=3,
                                     n_bg=40, rows=4)
    return synth.workload(name)


@pytest.mark.parametrize("name", EXTRACT_CASES)
def test_extract_paths_bitwise_equal_to_oracle(orc, name):
    w = _workload(name)
    el, npaths, bias = gts.extract_paths(w.ensemble)
    oel, onpaths, obias = orc.extract_paths(w.ensemble)
    assert npaths == onpaths
    for a, b in zip(_as_oracle_fields(el), _as_oracle_fields(oel)):
        _assert_bitwise(a, b)
    _assert_bitwise(bias, obias)


@pytest.mark.slow
def test_extract_and_pack_deep_ensemble(orc):
    w = synth.workload("deep")
    el, npaths, bias = gts.extract_paths(w.ensemble)
    oel, onpaths, obias = orc.extract_paths(w.ensemble)
    for a, b in zip(_as_oracle_fields(el), _as_oracle_fields(oel)):
        _assert_bitwise(a, b)
    _assert_bitwise(bias, obias)
    _check_pack_against_oracle(orc, el, 64)


def _paths_of(el):
    roots = np.flatnonzero(el["feature_idx"] == -1)
    sizes = np.diff(np.append(roots, len(el)))
    return roots, sizes, el["group"][roots]


def _check_pack_against_oracle(orc, el, cap, alg="bfd"):
    packed, offs = gts.pack_paths(el, cap, alg)
    roots, sizes, groups = _paths_of(el)
    bin_of, lane_of, k = orc.pack(sizes, groups, cap, alg)
    assert len(offs) == k + 1
    # rebuild the oracle's packed element order and compare raw bytes
    order = np.lexsort((lane_of, bin_of))
    want_idx = np.concatenate([np.arange(roots[p], roots[p] + sizes[p]) for p in order])
    _assert_bitwise(packed, el[want_idx])
    fill = np.bincount(bin_of, weights=sizes, minlength=k).astype(np.int64)
    _assert_bitwise(offs, np.concatenate([[0], np.cumsum(fill)]))


@pytest.mark.parametrize("name", EXTRACT_CASES)
@pytest.mark.parametrize("cap", [64, 32, 17])
@pytest.mark.parametrize("alg", ["bfd", "ffd", "nf", "none"])
def test_pack_paths_bitwise_equal_to_oracle(orc, name, cap, alg):
    w = _workload(name)
    el, _, _ = gts.extract_paths(w.ensemble)
    if int(np.max(_paths_of(el)[1])) > cap:
        with pytest.raises(gts.GtsError) as e:
            gts.pack_paths(el, cap, alg)
        assert e.value.status == gts.GTS_EPATHLEN
        return
    _check_pack_against_oracle(orc, el, cap, alg)


@pytest.mark.parametrize("alg", ["bfd", "ffd", "nf", "none"])
def test_pack_shuffled_groups_bitwise_equal_to_oracle(orc, alg):
    """Trees of several output groups interleaved in input order."""
    rng = np.random.default_rng(8)
    sizes = rng.integers(1, 65, size=700)
    groups = rng.integers(0, 5, size=700)
    el = _synthetic_elements(sizes, groups)
    _check_pack_against_oracle(orc, el, 64, alg)


def test_pack_golden_instances(orc):
    """The hand-worked packing instances (BFD, FFD, NF, none), run through the
    library."""
    import json
    fx = json.load(open(os.path.join(ROOT, "tests", "golden", "bin_packing.json")))
    cases = [dict(c, alg="bfd") for c in fx["cases"]] + fx["other_algorithms"]["cases"]
    for case in cases:
        el = _synthetic_elements(case["sizes"], case["groups"])
        packed, offs = gts.pack_paths(el, case["capacity"], case["alg"])
        assert len(offs) - 1 == case["num_bins"]
        roots = np.flatnonzero(el["feature_idx"] == -1)
        for p, (b, lane) in enumerate(zip(case["bin_of"], case["lane_of"])):
            pos = offs[b] + lane
            assert packed["path_idx"][pos] == p and packed["feature_idx"][pos] == -1
            assert roots[p] >= 0


def _synthetic_elements(sizes, groups):
    rows = []
    for p, (s, g) in enumerate(zip(sizes, groups)):
        rows.append((p, -1, g, -np.inf, np.inf, 1.0, 0.5))
        for k in range(s - 1):
            rows.append((p, k, g, 0.0, 1.0, 0.5, 0.5))
    return np.array(rows, dtype=gts.PATH_ELEMENT)


@pytest.mark.parametrize("alg", ["bfd", "ffd", "nf", "none"])
def test_pack_invariants_all_algorithms(alg):
    rng = np.random.default_rng(5)
    sizes = rng.integers(1, 65, size=500)
    groups = np.sort(rng.integers(0, 3, size=500))
    el = _synthetic_elements(sizes, groups)
    packed, offs = gts.pack_paths(el, 64, alg)
    assert offs[0] == 0 and offs[-1] == len(el)
    fills = np.diff(offs)
    assert np.all((fills >= 1) & (fills <= 64))
    assert sorted(packed["path_idx"].tolist()) == sorted(el["path_idx"].tolist())
    for b in range(len(offs) - 1):
        seg = packed[offs[b]:offs[b + 1]]
        assert seg["feature_idx"][0] == -1
        assert len(set(seg["group"].tolist())) == 1
    k = len(offs) - 1
    assert k >= int(np.ceil(sizes.sum() / 64))
    if alg == "none":
        assert k == len(sizes)


def test_model_layout_roundtrip():
    """The blob holds the packed elements in bin order (roots carry the leaf
    value in their zero-fraction slot), bin offsets and per-group bin ranges.
    Inside a path, the elements whose zero fraction is 0 (in the blob's
    precision) come first in feature order and their count is in the root's
    feature slot (-1 - count); the other elements follow as a cyclic rotation
    of their feature order."""
    w = synth.workload("wide")
    el, npaths, bias = gts.extract_paths(w.ensemble)
    packed, offs = gts.pack_paths(el, 64, "bfd")
    roots = packed["feature_idx"] == -1
    for dtype, ft in (("f32", np.float32), ("f64", np.float64)):
        desc, blob = gts.model_layout(packed, offs, 784, 10, bias, dtype)
        assert desc.num_paths == npaths and desc.num_bins == len(offs) - 1
        assert desc.bytes == len(blob) and all(o % 256 == 0 for o in desc.off[:7])
        assert desc.max_path_len == 9
        n = len(packed)
        feat = np.frombuffer(blob, np.int32, n, desc.off[0])
        lo = np.frombuffer(blob, np.float32, n, desc.off[1])
        hi = np.frombuffer(blob, np.float32, n, desc.off[2])
        z = np.frombuffer(blob, ft, n, desc.off[3])
        zsrc = np.where(roots, packed["v"], packed["zero_fraction"]).astype(ft)
        coll_sorted = coll_stored = 0
        paths_with_zero = 0
        for b in range(len(offs) - 1):
            r = np.flatnonzero(roots[offs[b]:offs[b + 1]]) + offs[b]
            ends = np.append(r[1:], offs[b + 1])
            seen_sorted, seen_stored = set(), set()
            for a, e in zip(r, ends):
                src = np.arange(a + 1, e)
                zero = zsrc[src] == 0
                n0 = int(zero.sum())
                paths_with_zero += n0 > 0
                assert feat[a] == -1 - n0 and z[a] == zsrc[a]
                rest = src[~zero]
                if len(rest):
                    rho = int(np.flatnonzero(packed["feature_idx"][rest] == feat[a + 1 + n0])[0])
                    rest = rest[(np.arange(len(rest)) + rho) % len(rest)]
                want = np.concatenate([src[zero], rest]).astype(np.int64)
                assert np.array_equal(feat[a + 1:e], packed["feature_idx"][want])
                assert np.array_equal(lo[a + 1:e], packed["lower"][want])
                assert np.array_equal(hi[a + 1:e], packed["upper"][want])
                assert np.array_equal(z[a + 1:e], zsrc[want])
                sf = packed["feature_idx"][src]
                for k in range(e - a - 1):
                    coll_sorted += (k, sf[k]) in seen_sorted
                    coll_stored += (k, feat[a + 1 + k]) in seen_stored
                    seen_sorted.add((k, sf[k]))
                    seen_stored.add((k, feat[a + 1 + k]))
        assert paths_with_zero > 0
        assert coll_stored * 4 < coll_sorted, (coll_stored, coll_sorted)
        bstart = np.frombuffer(blob, np.int32, len(offs), desc.off[4])
        assert np.array_equal(bstart, offs)
        gb = np.frombuffer(blob, np.int32, 11, desc.off[5])
        assert gb[0] == 0 and gb[-1] == len(offs) - 1
        for g in range(10):
            seg = packed[offs[gb[g]]:offs[gb[g + 1]]]
            assert np.all(seg["group"] == g)
        assert np.array_equal(np.frombuffer(blob, ft, 10, desc.off[6]), bias.astype(ft))


# ----------------------------------------------------------------------------
# error paths (forced from the host)
# ----------------------------------------------------------------------------

def _bad(ens_mod, **kw):
    import copy
    e = copy.deepcopy(ens_mod)
    for k, v in kw.items():
        setattr(e, k, v)
    return e


def test_extract_rejects_malformed_ensembles():
    base = synth.workload("tiny").ensemble
    left = base.left.copy()
    left[0] = 99                                        # child out of range
    cases = [_bad(base, left=left)]
    left2 = base.left.copy()
    left2[1] = 0                                        # cycle back to the root
    cases.append(_bad(base, left=left2))
    feat = base.feature.copy()
    feat[0] = 8                                         # feature >= M
    cases.append(_bad(base, feature=feat))
    grp = base.tree_group.copy()
    grp[3] = 1                                          # group >= G
    cases.append(_bad(base, tree_group=grp))
    cov = base.cover.copy()
    cov[2] = -1.0                                       # negative cover
    cases.append(_bad(base, cover=cov))
    thr = base.threshold.copy()
    thr[0] = np.nan
    cases.append(_bad(base, threshold=thr))
    for e in cases:
        with pytest.raises(gts.GtsError) as exc:
            gts.extract_paths(e)
        assert exc.value.status == gts.GTS_EINVAL


def test_extract_capacity_and_null_arguments():
    w = synth.workload("tiny")
    s, keep = gts._ensemble_struct(w.ensemble)
    n = ctypes.c_int64(0)
    npaths = ctypes.c_int64(0)
    L = gts.lib()
    assert L.gts_extract_paths(ctypes.byref(s), None, 0, ctypes.byref(n), ctypes.byref(npaths),
                               None) == gts.GTS_OK
    small = np.zeros(5, gts.PATH_ELEMENT)
    st = L.gts_extract_paths(ctypes.byref(s), small.ctypes.data_as(ctypes.c_void_p), 5,
                             ctypes.byref(n), ctypes.byref(npaths), None)
    assert st == gts.GTS_EBUFSIZE and n.value == 284 and npaths.value == 80
    assert L.gts_extract_paths(None, None, 0, ctypes.byref(n), ctypes.byref(npaths),
                               None) == gts.GTS_EINVAL
    assert L.gts_extract_paths(ctypes.byref(s), None, 0, None, None, None) == gts.GTS_EINVAL


def test_pack_errors():
    el = _synthetic_elements([3, 65 - 1, 2], [0, 0, 0])
    with pytest.raises(gts.GtsError) as e:
        gts.pack_paths(el, 32, "bfd")
    assert e.value.status == gts.GTS_EPATHLEN
    with pytest.raises(gts.GtsError) as e:
        gts.pack_paths(el, 65, "bfd")
    assert e.value.status == gts.GTS_EINVAL
    bad = el.copy()
    bad["feature_idx"][0] = 2                           # does not start at a root
    with pytest.raises(gts.GtsError) as e:
        gts.pack_paths(bad, 64, "bfd")
    assert e.value.status == gts.GTS_EINVAL
    L = gts.lib()
    k = ctypes.c_int64(0)
    offs = np.zeros(1, np.int64)
    packed = np.zeros(len(el), gts.PATH_ELEMENT)
    st = L.gts_pack_paths(el.ctypes.data_as(ctypes.c_void_p), len(el), 64, 0,
                          packed.ctypes.data_as(ctypes.c_void_p),
                          offs.ctypes.data_as(ctypes.c_void_p), 1, ctypes.byref(k))
    assert st == gts.GTS_EBUFSIZE and k.value == 2
    assert L.gts_pack_paths(el.ctypes.data_as(ctypes.c_void_p), len(el), 64, 9, None, None, 0,
                            ctypes.byref(k)) == gts.GTS_EINVAL


def test_layout_errors():
    w = synth.workload("tiny")
    el, _, bias = gts.extract_paths(w.ensemble)
    packed, offs = gts.pack_paths(el, 64, "bfd")
    with pytest.raises(gts.GtsError):
        gts.model_layout(packed, offs, 4, 1, bias, "f32")       # feature >= M
    bad = offs.copy()
    bad[1] += 1                                                 # bin not on a root
    with pytest.raises(gts.GtsError):
        gts.model_layout(packed, bad, 8, 1, bias, "f32")
    with pytest.raises(KeyError):
        gts.model_layout(packed, offs, 8, 1, bias, "f16")


def test_device_calls_reject_bad_arguments_without_touching_the_gpu():
    """Argument checks happen before any HIP call."""
    w = synth.workload("tiny")
    el, _, bias = gts.extract_paths(w.ensemble)
    packed, offs = gts.pack_paths(el, 64, "bfd")
    desc, blob = gts.model_layout(packed, offs, 8, 1, bias, "f64")
    L = gts.lib()
    vp = ctypes.c_void_p
    for fn in (L.gts_shap, L.gts_shap_interactions):
        assert fn(None, vp(1), vp(1), 4, 8, vp(1), None) == gts.GTS_EINVAL
        assert fn(ctypes.byref(desc), vp(1), vp(1), -1, 8, vp(1), None) == gts.GTS_EINVAL
        assert fn(ctypes.byref(desc), vp(1), vp(1), 4, 7, vp(1), None) == gts.GTS_EINVAL
        assert fn(ctypes.byref(desc), None, vp(1), 4, 8, vp(1), None) == gts.GTS_EINVAL
        assert fn(ctypes.byref(desc), vp(1), vp(1), 0, 8, vp(1), None) == gts.GTS_OK  # no-op
        forged = gts.ModelDesc.from_buffer_copy(desc)
        forged.magic = 0
        assert fn(ctypes.byref(forged), vp(1), vp(1), 4, 8, vp(1), None) == gts.GTS_EINVAL
    info = gts.LaunchInfo()
    assert L.gts_launch_config(ctypes.byref(desc), 10, 0, None) == gts.GTS_EINVAL
    assert L.gts_launch_config(None, 10, 0, ctypes.byref(info)) == gts.GTS_EINVAL
    assert L.gts_launch_config(ctypes.byref(desc), -1, 1, ctypes.byref(info)) == gts.GTS_EINVAL


@pytest.mark.parametrize("name", ["tiny", "covtype_med", "wide", "random0", "random2"])
@pytest.mark.parametrize("dtype", ["f32", "f64"])
@pytest.mark.parametrize("alg", ["bfd", "ffd", "nf", "none"])
def test_prepare_model_equals_the_three_step_route(name, dtype, alg):
    """gts_prepare_model writes byte for byte the blob and descriptor of
    gts_model_layout(gts_pack_paths(gts_extract_paths(.)))."""
    w = _workload(name)
    el, npaths, bias = gts.extract_paths(w.ensemble)
    packed, offs = gts.pack_paths(el, 64, alg)
    d1, b1 = gts.model_layout(packed, offs, w.ensemble.num_features, w.ensemble.num_groups,
                              bias, dtype)
    for _ in range(2):  # second call takes the cached-size fast path
        d2, b2, bias2 = gts.prepare_blob(w.ensemble, dtype, 64, alg)
        assert bytes(d1) == bytes(d2)
        assert b1.tobytes() == b2.tobytes()
        assert bias.tobytes() == bias2.tobytes()


def test_prepare_model_from_concurrent_threads():
    """Preparations from several threads at once (ctypes releases the GIL;
    up to four callers run on their own teams of the worker pool, the others
    alone, each in its own scratch, with per-thread caps on the thread count)
    give the blobs of one-at-a-time calls, also when one thread alternates
    between models of different sizes."""
    import threading
    names = ["covtype_med", "wide", "random0", "tiny"]
    ens = {n: _workload(n).ensemble for n in names}
    want = {}
    for n in names:
        d, b, bias = gts.prepare_blob(ens[n], "f32")
        want[n] = (bytes(d), b.tobytes(), bias.tobytes())
    errors = []

    caps = [0, 1, 2, 3, 8, 16]

    def work(k):
        try:
            gts.set_host_threads(caps[k])
            for r in range(6):
                n = names[(k + r) % len(names)]
                d, b, bias = gts.prepare_blob(ens[n], "f32")
                if (bytes(d), b.tobytes(), bias.tobytes()) != want[n]:
                    errors.append((k, r, n))
        except Exception as e:  # pragma: no cover - reported below
            errors.append((k, repr(e)))

    threads = [threading.Thread(target=work, args=(k,)) for k in range(6)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert errors == []


def test_host_thread_cap():
    """gts_set_host_threads: results do not depend on the cap; a negative cap
    is an error; the cap belongs to the calling thread."""
    import threading
    w = _workload("covtype_med")
    want = gts.prepare_blob(w.ensemble, "f64")
    try:
        for cap in (1, 2, 5, 0):
            gts.set_host_threads(cap)
            d, b, bias = gts.prepare_blob(w.ensemble, "f64")
            assert bytes(d) == bytes(want[0]) and b.tobytes() == want[1].tobytes()
            assert bias.tobytes() == want[2].tobytes()
        with pytest.raises(gts.GtsError) as e:
            gts.set_host_threads(-1)
        assert e.value.status == gts.GTS_EINVAL
        gts.set_host_threads(1)
        seen = []
        t = threading.Thread(target=lambda: seen.append(gts.prepare_blob(w.ensemble, "f64")))
        t.start()
        t.join()
        assert seen[0][1].tobytes() == want[1].tobytes()
    finally:
        gts.set_host_threads(0)


def test_prepare_model_errors():
    w = synth.workload("deep")
    with pytest.raises(gts.GtsError) as e:           # depth-16 paths do not fit 8 lanes
        gts.prepare_blob(w.ensemble, "f32", 8, "bfd")
    assert e.value.status == gts.GTS_EPATHLEN
    base = synth.workload("tiny").ensemble
    import copy
    bad = copy.deepcopy(base)
    bad.feature = bad.feature.copy()
    bad.feature[0] = 99
    with pytest.raises(gts.GtsError) as e:
        gts.prepare_blob(bad, "f32")
    assert e.value.status == gts.GTS_EINVAL


def test_extract_workspace_and_device_argument_checks():
    """Sizing and the argument checks of the device extraction run before any
    HIP call."""
    L = gts.lib()
    b = ctypes.c_int64(0)
    assert L.gts_extract_workspace_bytes(10, 1000, ctypes.byref(b)) == gts.GTS_OK
    small = b.value
    assert L.gts_extract_workspace_bytes(10, 100000, ctypes.byref(b)) == gts.GTS_OK
    assert b.value > small >= 1000 * 40
    assert L.gts_extract_workspace_bytes(-1, 10, ctypes.byref(b)) == gts.GTS_EINVAL
    assert L.gts_extract_workspace_bytes(1, 10, None) == gts.GTS_EINVAL
    n, p = ctypes.c_int64(0), ctypes.c_int64(0)
    w = synth.workload("tiny")
    s, keep = gts._ensemble_struct(w.ensemble)
    vp = ctypes.c_void_p
    f = L.gts_extract_paths_device
    assert f(None, None, 0, ctypes.byref(n), ctypes.byref(p), None, None, 0, None) == gts.GTS_EINVAL
    assert f(ctypes.byref(s), None, -1, ctypes.byref(n), ctypes.byref(p), None, None, 0,
             None) == gts.GTS_EINVAL
    assert f(ctypes.byref(s), None, 5, ctypes.byref(n), ctypes.byref(p), None, None, 0,
             None) == gts.GTS_EINVAL
    assert f(ctypes.byref(s), None, 0, ctypes.byref(n), ctypes.byref(p), None, None, 0,
             None) == gts.GTS_EBUFSIZE


def test_feature_count_beyond_the_lds_is_rejected():
    """A phi row of M + 1 entries that cannot fit a 4-row tile in a
    workgroup's LDS is refused with GTS_EINVAL before any launch."""
    ens = synth.ensemble_from_lists([[(1, 2, 3, 0.5, 10.0, 0.0), (-1, -1, -1, 0, 4.0, 1.0),
                                      (-1, -1, -1, 0, 6.0, 2.0)]], M=200000)
    desc, blob, bias = gts.prepare_blob(ens, "f32")
    L = gts.lib()
    vp = ctypes.c_void_p
    for fn in (L.gts_shap, L.gts_shap_interactions):
        assert fn(ctypes.byref(desc), vp(1), vp(1), 4, 200000, vp(1), None) == gts.GTS_EINVAL
        assert "LDS" in gts.last_error() or "too large" in gts.last_error()


@pytest.mark.parametrize("alg", ["bfd", "ffd", "nf", "none"])
def test_sorted_bins_flag(alg):
    """GTS_MODEL_SORTED_BINS is set exactly when every bin's paths never grow
    in length (always for the decreasing heuristics)."""
    for name in ("covtype_med", "random3"):
        w = _workload(name)
        el, _, bias = gts.extract_paths(w.ensemble)
        packed, offs = gts.pack_paths(el, 64, alg)
        roots = np.flatnonzero(packed["feature_idx"] == -1)
        ends = np.append(roots[1:], len(packed))
        sorted_ = True
        for b in range(len(offs) - 1):
            sizes = [e - a for a, e in zip(roots, ends) if offs[b] <= a < offs[b + 1]]
            sorted_ &= all(x >= y for x, y in zip(sizes, sizes[1:]))
        desc, blob = gts.model_layout(packed, offs, w.ensemble.num_features,
                                      w.ensemble.num_groups, bias, "f32")
        assert bool(desc.flags & 1) == sorted_, (name, alg)
        if alg in ("bfd", "ffd", "none"):
            assert sorted_
        assert gts.prepare_blob(w.ensemble, "f32", alg=alg)[0].flags == desc.flags


# --------------------------------------------------------------------------
# gts_plan_model: the host half of a model built on the device
# --------------------------------------------------------------------------

def _plan_arrays(plan, hp):
    P, T, K = plan.num_paths, plan.num_trees, plan.num_bins

    def arr(k, t, n):
        o = plan.off[k]
        return np.frombuffer(hp[o:o + n * np.dtype(t).itemsize].tobytes(), t)

    return (arr(0, np.uint64, P), arr(1, np.int32, P), arr(2, np.int32, T + 1),
            arr(3, np.int32, K + 1))


@pytest.mark.parametrize("name,dtype", [("tiny", "f64"), ("random0", "f32"), ("random2", "f64"),
                                        ("random3", "f32")])
def test_plan_walks_to_the_blob_paths(name, dtype):
    """Every path's turns, followed from its tree's root, end at a leaf whose
    value is the root slot of the blob at the path's place, and pass exactly
    the features the blob holds for the path; the plan's bins are the blob's."""
    ens = _workload(name).ensemble
    desc, plan, hp = gts.plan_model(ens, dtype)
    pdesc, blob, _ = gts.prepare_blob(ens, dtype)
    assert bytes(desc) == bytes(pdesc)
    dirs, dest, tree_paths, bins = _plan_arrays(plan, hp)
    zt = np.float64 if dtype == "f64" else np.float32

    def barr(k, t, n):
        o = desc.off[k]
        return np.frombuffer(blob[o:o + n * np.dtype(t).itemsize].tobytes(), t)

    feat = barr(0, np.int32, desc.num_elements)
    zero = barr(3, zt, desc.num_elements)
    assert np.array_equal(bins, barr(4, np.int32, desc.num_bins + 1))
    off = ens.tree_node_offsets
    assert tree_paths[0] == 0 and tree_paths[-1] == desc.num_paths
    for t in range(ens.num_trees):
        base = off[t]
        for p in range(tree_paths[t], tree_paths[t + 1]):
            node, feats = 0, set()
            for d in range(64):
                a, b = ens.left[base + node], ens.right[base + node]
                if a < 0 and b < 0:
                    break
                feats.add(int(ens.feature[base + node]))
                node = b if (int(dirs[p]) >> d) & 1 else a
            e = dest[p]
            n0 = -1 - feat[e]
            assert n0 >= 0 and zero[e] == zt(ens.value[base + node])
            q = len(feats)
            assert set(feat[e + 1:e + 1 + q].tolist()) == feats
            assert e + 1 + q == len(feat) or feat[e + 1 + q] < 0


def test_plan_refusals():
    """Plans only for models whose launches run one path per wave, with
    paths of at most 64 splits; the two-call idiom's capacity check."""
    w = synth.random_workload(5, num_trees=3, max_depth=4, M=18, rows=4)
    with pytest.raises(gts.GtsError) as e:
        gts.plan_model(w.ensemble, "f32")
    assert e.value.status == gts.GTS_EINVAL
    w = synth.random_workload(5, num_trees=3, max_depth=4, M=12, rows=4)
    with pytest.raises(gts.GtsError):
        gts.plan_model(w.ensemble, "f64")      # M <= 11 in fp64
    desc, plan, hp = gts.plan_model(w.ensemble, "f32")
    s, keep = gts._ensemble_struct(w.ensemble)
    small = np.empty(plan.bytes - 1, np.uint8)
    st = gts.lib().gts_plan_model(ctypes.byref(s), 64, 0, 0, ctypes.byref(gts.ModelDesc()),
                                  ctypes.byref(gts.PlanDesc()),
                                  small.ctypes.data_as(ctypes.c_void_p), small.nbytes)
    assert st == gts.GTS_EBUFSIZE

    def chain(depth):
        nodes, cover = [], 1000.0
        for d in range(depth):
            b = len(nodes)
            nodes.append((b + 2, b + 1, d % 5, 0.5 + 0.001 * d, cover, 0.0))
            nodes.append((-1, -1, -1, 0.0, 1.0, 0.5))
            cover -= 1.0
        nodes.append((-1, -1, -1, 0.0, cover, 1.0))
        return nodes

    gts.plan_model(synth.ensemble_from_lists([chain(64)], M=5), "f32")
    with pytest.raises(gts.GtsError) as e:
        gts.plan_model(synth.ensemble_from_lists([chain(65)], M=5), "f32")
    assert "64 splits" in str(e.value)
