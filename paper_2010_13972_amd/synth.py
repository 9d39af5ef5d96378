"""Seeded synthetic tree ensembles and feature matrices.

This module only *makes inputs*: tree structure, split features, thresholds,
node covers, leaf values and the rows to explain.  It contains none of the
SHAP arithmetic, so both the CPU oracle and the GPU library can be fed from
it without sharing any part of the method.

The ensembles stand in for the XGBoost models of the paper's evaluation
(Section 4, Tables 2 and 3), whose datasets and trained weights are not
available.  Each named workload copies the shape of one of those models:

* ``tiny``        10 full depth-3 trees, M=8, X ~ U[0,1), 1000 background rows,
                  256 explained rows (cal_housing-small shape).
* ``covtype_med`` 100 trees, depth <= 8, split probability 0.85, M=54
                  (10 columns N(0,1), 44 columns Bernoulli(0.2)), 10k/10k rows.
* ``deep``        1000 trees, depth <= 16, split probability 0.7, at most 1024
                  leaves per tree, M=8, X ~ N(0,1), 20k background / 10k rows.
* ``wide``        10 classes x 100 rounds = 1000 trees, depth <= 8, p=0.85,
                  M=784 with half the entries exactly 0 (else U[0,1)),
                  tree t -> output group t mod 10, 10k/10k rows.
* ``interactions`` the ``covtype_med`` model, first 1000 explained rows.

Construction rules (shared by every workload):

* RNG: ``PCG64(SeedSequence(201013972, spawn_key=(workload_id, stream)))``,
  streams 0 = structure/features/thresholds, 1 = leaf values,
  2 = background rows, 3 = explained rows, 4 = extra rows for row-count
  sweeps (``sweep_rows``).
* Trees grow breadth first; a node at depth d < max_depth splits with
  probability p; under a leaf cap a split that would exceed it is not taken.
  Node storage is BFS order per tree, root at local index 0.
* Split feature uniform over M.  Threshold = the value of that feature in a
  uniformly drawn background row, redrawn while it equals the column minimum
  (so the left side ``x < t`` is never globally empty).
* Cover = number of background rows reaching the node under ``x < t -> left``.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

SEED = 201013972

WORKLOADS = ("tiny", "covtype_med", "deep", "wide", "interactions")
_WORKLOAD_ID = {"tiny": 0, "covtype_med": 1, "deep": 2, "wide": 3, "interactions": 4}


def rng_for(workload_id: int, stream: int) -> np.random.Generator:
    return np.random.Generator(
        np.random.PCG64(np.random.SeedSequence(SEED, spawn_key=(workload_id, stream))))


@dataclasses.dataclass
class Ensemble:
    """Flattened tree ensemble; field meaning follows the tree lists
    {v, a, b, t, r, d} of Section 2.1 (leaf value, left child, right child,
    threshold, cover, feature), plus the tree -> output group map."""
    num_features: int
    num_groups: int
    tree_node_offsets: np.ndarray  # int64 [T+1]
    tree_group: np.ndarray         # int32 [T]
    left: np.ndarray               # int32 [N], tree-local, -1 = leaf
    right: np.ndarray              # int32 [N]
    feature: np.ndarray            # int32 [N], -1 on leaves
    threshold: np.ndarray          # float32 [N], go left iff x < threshold
    cover: np.ndarray              # float64 [N]
    value: np.ndarray              # float64 [N], leaf value (0 on internal nodes)

    @property
    def num_trees(self) -> int:
        return int(self.tree_group.shape[0])

    @property
    def num_nodes(self) -> int:
        return int(self.left.shape[0])

    def max_depth(self) -> int:
        best = 0
        for t in range(self.num_trees):
            a = int(self.tree_node_offsets[t])
            b = int(self.tree_node_offsets[t + 1])
            depth = np.zeros(b - a, dtype=np.int64)
            for n in range(b - a):  # BFS order: parents precede children
                for c in (self.left[a + n], self.right[a + n]):
                    if c >= 0:
                        depth[c] = depth[n] + 1
            best = max(best, int(depth.max()))
        return best


@dataclasses.dataclass
class Workload:
    name: str
    ensemble: Ensemble
    X_background: np.ndarray  # float32 [n_bg, M]
    X: np.ndarray             # float32 [rows, M]
    dtype: str                # "f32" or "f64": accumulation type the workload is quoted in


# ----------------------------------------------------------------------------
# feature distributions
# ----------------------------------------------------------------------------

def _features(kind: str, rng: np.random.Generator, n: int, M: int) -> np.ndarray:
    if kind == "uniform":
        x = rng.random((n, M))
    elif kind == "normal":
        x = rng.standard_normal((n, M))
    elif kind == "covtype":  # 10 continuous N(0,1) + 44 binary Bernoulli(0.2)
        x = np.empty((n, M))
        x[:, :10] = rng.standard_normal((n, 10))
        x[:, 10:] = (rng.random((n, M - 10)) < 0.2).astype(np.float64)
    elif kind == "sparse_image":  # exact 0 w.p. 0.5, else U[0,1)
        u = rng.random((n, M))
        keep = rng.random((n, M)) >= 0.5
        x = np.where(keep, u, 0.0)
    elif kind == "discrete4":  # small integer grid: many exact ties x == t
        x = rng.integers(0, 4, size=(n, M)).astype(np.float64)
    else:
        raise ValueError(f"unknown feature distribution {kind!r}")
    return np.ascontiguousarray(x, dtype=np.float32)


# ----------------------------------------------------------------------------
# tree growth
# ----------------------------------------------------------------------------

def _grow_tree(rng: np.random.Generator, Xbg: np.ndarray, colmin: np.ndarray,
               max_depth: int, p_split: float, max_leaves: Optional[int]):
    """Grow one tree breadth first.  Returns (left, right, feature, threshold)."""
    n_bg, M = Xbg.shape
    left, right, feat, thr = [-1], [-1], [-1], [0.0]
    level = [0]
    leaves = 1
    depth = 0
    while level and depth < max_depth:
        n = len(level)
        want = rng.random(n) < p_split if p_split < 1.0 else np.ones(n, dtype=bool)
        if max_leaves is not None:
            want &= (leaves + np.cumsum(want)) <= max_leaves
        n_acc = int(want.sum())
        if n_acc == 0:
            break
        f = rng.integers(0, M, size=n_acc)
        idx = rng.integers(0, n_bg, size=n_acc)
        t = Xbg[idx, f]
        bad = t == colmin[f]
        while bad.any():
            k = int(bad.sum())
            idx[bad] = rng.integers(0, n_bg, size=k)
            t[bad] = Xbg[idx[bad], f[bad]]
            bad = t == colmin[f]
        nxt = []
        j = 0
        for i, node in enumerate(level):
            if not want[i]:
                continue
            feat[node] = int(f[j])
            thr[node] = float(t[j])
            j += 1
            a = len(left)
            for _ in range(2):
                left.append(-1)
                right.append(-1)
                feat.append(-1)
                thr.append(0.0)
            left[node] = a
            right[node] = a + 1
            nxt.extend((a, a + 1))
        leaves += n_acc
        level = nxt
        depth += 1
    return (np.asarray(left, np.int32), np.asarray(right, np.int32),
            np.asarray(feat, np.int32), np.asarray(thr, np.float32))


def _covers(left, right, feat, thr, Xbg) -> np.ndarray:
    """Count background rows reaching each node (x < t goes left)."""
    n = left.shape[0]
    cover = np.zeros(n, dtype=np.float64)
    cover[0] = Xbg.shape[0]
    cur = np.zeros(Xbg.shape[0], dtype=np.int64)
    alive = np.arange(Xbg.shape[0])
    while alive.size:
        nd = cur[alive]
        internal = left[nd] >= 0
        alive = alive[internal]
        nd = nd[internal]
        if not alive.size:
            break
        go_left = Xbg[alive, feat[nd]] < thr[nd]
        cur[alive] = np.where(go_left, left[nd], right[nd])
        cover += np.bincount(cur[alive], minlength=n)
    return cover


def make_ensemble(*, num_trees: int, max_depth: int, p_split: float, M: int,
                  num_groups: int, leaf_std: float, Xbg: np.ndarray,
                  rng_struct: np.random.Generator, rng_leaf: np.random.Generator,
                  max_leaves: Optional[int] = None,
                  tree_group: Optional[np.ndarray] = None) -> Ensemble:
    colmin = Xbg.min(axis=0)
    colmax = Xbg.max(axis=0)
    if np.any(colmin == colmax):
        raise ValueError("a background column is constant; no threshold can split it")
    lefts, rights, feats, thrs, covs, vals, offs = [], [], [], [], [], [], [0]
    for _ in range(num_trees):
        l, r, f, t = _grow_tree(rng_struct, Xbg, colmin, max_depth, p_split, max_leaves)
        c = _covers(l, r, f, t, Xbg)
        v = np.zeros(l.shape[0], dtype=np.float64)
        leaf = l < 0
        v[leaf] = rng_leaf.normal(0.0, leaf_std, size=int(leaf.sum()))
        lefts.append(l), rights.append(r), feats.append(f), thrs.append(t)
        covs.append(c), vals.append(v)
        offs.append(offs[-1] + l.shape[0])
    if tree_group is None:
        tree_group = np.arange(num_trees) % num_groups
    return Ensemble(
        num_features=M, num_groups=num_groups,
        tree_node_offsets=np.asarray(offs, np.int64),
        tree_group=np.asarray(tree_group, np.int32),
        left=np.concatenate(lefts), right=np.concatenate(rights),
        feature=np.concatenate(feats), threshold=np.concatenate(thrs),
        cover=np.concatenate(covs), value=np.concatenate(vals))


# ----------------------------------------------------------------------------
# named workloads
# ----------------------------------------------------------------------------

_SPECS = {
    #             trees depth  p     leaves M    G   leaf_std dist            n_bg   rows   dtype
    "tiny":        (10,   3,  1.00, None,  8,   1,  1.0, "uniform",      1000,   256, "f64"),
    "covtype_med": (100,  8,  0.85, None,  54,  1,  0.1, "covtype",      10000, 10000, "f32"),
    "deep":        (1000, 16, 0.70, 1024,  8,   1,  1.0, "normal",       20000, 10000, "f32"),
    "wide":        (1000, 8,  0.85, None,  784, 10, 0.1, "sparse_image", 10000, 10000, "f32"),
}

_CACHE: dict = {}


def workload(name: str, rows: Optional[int] = None) -> Workload:
    """Build (and memoise) a named workload.  ``rows`` truncates the explained
    rows to a prefix (the prefix of the same seeded stream)."""
    if name == "interactions":
        base = workload("covtype_med")
        n = 1000 if rows is None else rows
        return Workload("interactions", base.ensemble, base.X_background,
                        base.X[:n], "f32")
    if name not in _SPECS:
        raise KeyError(f"unknown workload {name!r}; choose from {WORKLOADS}")
    if name not in _CACHE:
        T, D, p, cap, M, G, lstd, dist, n_bg, n_rows, dt = _SPECS[name]
        wid = _WORKLOAD_ID[name]
        Xbg = _features(dist, rng_for(wid, 2), n_bg, M)
        X = _features(dist, rng_for(wid, 3), n_rows, M)
        ens = make_ensemble(num_trees=T, max_depth=D, p_split=p, M=M, num_groups=G,
                            leaf_std=lstd, Xbg=Xbg, rng_struct=rng_for(wid, 0),
                            rng_leaf=rng_for(wid, 1), max_leaves=cap)
        _CACHE[name] = Workload(name, ens, Xbg, X, dt)
    w = _CACHE[name]
    if rows is not None:
        return Workload(w.name, w.ensemble, w.X_background, w.X[:rows], w.dtype)
    return w


def sweep_rows(name: str, n: int) -> np.ndarray:
    """``n`` rows from the feature distribution of a named workload, drawn from
    a stream of their own (for sweeps over the number of explained rows)."""
    if name == "interactions":
        name = "covtype_med"
    _, _, _, _, M, _, _, dist, _, _, _ = _SPECS[name]
    return _features(dist, rng_for(_WORKLOAD_ID[name], 4), n, M)


def random_workload(seed: int, *, num_trees: int = 3, max_depth: int = 4,
                    p_split: float = 0.8, M: int = 5, num_groups: int = 1,
                    dist: str = "discrete4", n_bg: int = 50, rows: int = 16,
                    leaf_std: float = 1.0, max_leaves: Optional[int] = None) -> Workload:
    """Small random ensemble for property tests.  With the default ``discrete4``
    features, few columns and a small background set it produces repeated
    features on a path, exact ties ``x == t`` and zero-cover nodes."""
    base = 1000 + seed
    Xbg = _features(dist, rng_for(base, 2), n_bg, M)
    X = _features(dist, rng_for(base, 3), rows, M)
    ens = make_ensemble(num_trees=num_trees, max_depth=max_depth, p_split=p_split, M=M,
                        num_groups=num_groups, leaf_std=leaf_std, Xbg=Xbg,
                        rng_struct=rng_for(base, 0), rng_leaf=rng_for(base, 1),
                        max_leaves=max_leaves)
    return Workload(f"random{seed}", ens, Xbg, X, "f64")


def ensemble_from_lists(trees, M: int, num_groups: int = 1, tree_group=None) -> Ensemble:
    """Build an Ensemble from explicit per-tree node lists.  Each tree is a list
    of nodes ``(left, right, feature, threshold, cover, value)`` in storage
    order with the root first; leaves have left = right = -1."""
    lefts, rights, feats, thrs, covs, vals, offs = [], [], [], [], [], [], [0]
    for nodes in trees:
        for (l, r, f, t, c, v) in nodes:
            lefts.append(l), rights.append(r), feats.append(f)
            thrs.append(t), covs.append(c), vals.append(v)
        offs.append(offs[-1] + len(nodes))
    if tree_group is None:
        tree_group = np.arange(len(trees)) % num_groups
    return Ensemble(
        num_features=M, num_groups=num_groups,
        tree_node_offsets=np.asarray(offs, np.int64),
        tree_group=np.asarray(tree_group, np.int32),
        left=np.asarray(lefts, np.int32), right=np.asarray(rights, np.int32),
        feature=np.asarray(feats, np.int32), threshold=np.asarray(thrs, np.float32),
        cover=np.asarray(covs, np.float64), value=np.asarray(vals, np.float64))
