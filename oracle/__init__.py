"""ctypes front end of the plain CPU oracle (``oracle.c``).

TEST INFRASTRUCTURE ONLY: the tests, the package smoke check and the
benchmark's CPU-baseline leg are the only callers.  The product library never
imports, links or calls anything here.

All results are fp64 numpy arrays.  See ``oracle.c`` for what each route
computes and which passage of the paper it follows.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile oracle.c with gcc (fp64, OpenMP, no FP contraction)."""
    if force or not os.path.exists(_LIB_PATH):
        build_to(_SRC, _LIB_PATH)
    return _LIB_PATH


def build_to(src: str, out: str) -> str:
    """Compile an oracle source file to a shared library at ``out``."""
    tmp = out + ".tmp"
    cmd = ["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fPIC", "-shared",
           "-std=c11", "-Wall", "-Wno-unused-function", src, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def default() -> "Oracle":
    """The oracle built from oracle.c (built on first use if missing)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=True)
        _lib = Oracle(_LIB_PATH)
    return _lib


def _p(a: Optional[np.ndarray]):
    if a is None:
        return None
    return a.ctypes.data_as(ctypes.c_void_p)


def _ens_args(ens):
    """Contiguous arrays in the dtypes oracle.c expects (kept alive by caller)."""
    arrs = dict(
        off=np.ascontiguousarray(ens.tree_node_offsets, np.int64),
        group=np.ascontiguousarray(ens.tree_group, np.int32),
        left=np.ascontiguousarray(ens.left, np.int32),
        right=np.ascontiguousarray(ens.right, np.int32),
        feat=np.ascontiguousarray(ens.feature, np.int32),
        thr=np.ascontiguousarray(ens.threshold, np.float32),
        cover=np.ascontiguousarray(ens.cover, np.float64),
        value=np.ascontiguousarray(ens.value, np.float64),
    )
    head = (ctypes.c_int32(ens.num_features), ctypes.c_int32(ens.num_groups),
            ctypes.c_int64(len(arrs["group"])))
    ptrs = tuple(_p(arrs[k]) for k in ("off", "group", "left", "right", "feat",
                                       "thr", "cover", "value"))
    return arrs, head + ptrs


def _X(X: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(X, np.float32)


PATH_DTYPE = np.dtype([("path_idx", np.int64), ("feature_idx", np.int32),
                       ("group", np.int32), ("lower", np.float32),
                       ("upper", np.float32), ("zero_fraction", np.float64),
                       ("v", np.float64)])


class Oracle:
    """One loaded build of oracle.c."""

    def __init__(self, path: str):
        self.path = path
        self._lib = ctypes.CDLL(path)

    def predict(self, ens, X) -> np.ndarray:
        arrs, ea = _ens_args(ens)
        X = _X(X)
        out = np.zeros((X.shape[0], ens.num_groups), np.float64)
        self._lib.or_predict(*ea, _p(X), ctypes.c_int64(X.shape[0]), ctypes.c_int64(X.shape[1]),
                         _p(out))
        return out

    def expected_value(self, ens) -> np.ndarray:
        arrs, ea = _ens_args(ens)
        out = np.zeros(ens.num_groups, np.float64)
        self._lib.or_expected_value(*ea, _p(out))
        return out

    def brute_shap(self, ens, X) -> np.ndarray:
        arrs, ea = _ens_args(ens)
        X = _X(X)
        M, G = ens.num_features, ens.num_groups
        out = np.zeros((X.shape[0], G, M + 1), np.float64)
        rc = self._lib.or_brute_shap(*ea, _p(X), ctypes.c_int64(X.shape[0]),
                                 ctypes.c_int64(X.shape[1]), _p(out))
        if rc != 0:
            raise ValueError("brute force supports M <= 20")
        return out

    def brute_interactions(self, ens, X) -> np.ndarray:
        arrs, ea = _ens_args(ens)
        X = _X(X)
        M, G = ens.num_features, ens.num_groups
        out = np.zeros((X.shape[0], G, M + 1, M + 1), np.float64)
        rc = self._lib.or_brute_interactions(*ea, _p(X), ctypes.c_int64(X.shape[0]),
                                         ctypes.c_int64(X.shape[1]), _p(out))
        if rc != 0:
            raise ValueError("brute-force interactions support 2 <= M <= 16")
        return out

    def treeshap(self, ens, X, nthreads: int = 0) -> np.ndarray:
        arrs, ea = _ens_args(ens)
        X = _X(X)
        M, G = ens.num_features, ens.num_groups
        out = np.zeros((X.shape[0], G, M + 1), np.float64)
        self._lib.or_treeshap(*ea, _p(X), ctypes.c_int64(X.shape[0]), ctypes.c_int64(X.shape[1]),
                          _p(out), ctypes.c_int32(nthreads))
        return out

    def interactions(self, ens, X, nthreads: int = 0) -> np.ndarray:
        arrs, ea = _ens_args(ens)
        X = _X(X)
        M, G = ens.num_features, ens.num_groups
        out = np.zeros((X.shape[0], G, M + 1, M + 1), np.float64)
        self._lib.or_interactions(*ea, _p(X), ctypes.c_int64(X.shape[0]),
                              ctypes.c_int64(X.shape[1]), _p(out), ctypes.c_int32(nthreads))
        return out

    def path_brute(self, feature, lower, upper, zero_fraction, v, x, interactions: bool = False):
        """Eq. (2) (and Eq. (3)-(6)) of one merged path's own game for one row.
        Arrays exclude the root element.  Returns phi[q] (and inter[q, q])."""
        feature = np.ascontiguousarray(feature, np.int32)
        lower = np.ascontiguousarray(lower, np.float32)
        upper = np.ascontiguousarray(upper, np.float32)
        zero_fraction = np.ascontiguousarray(zero_fraction, np.float64)
        x = np.ascontiguousarray(x, np.float32)
        q = feature.shape[0]
        phi = np.zeros(q, np.float64)
        inter = np.zeros((q, q), np.float64) if interactions else None
        rc = self._lib.or_path_brute(ctypes.c_int32(q), _p(feature), _p(lower), _p(upper),
                                 _p(zero_fraction), ctypes.c_double(v), _p(x), _p(phi),
                                 _p(inter))
        if rc != 0:
            raise ValueError("path enumeration supports q <= 20")
        return (phi, inter) if interactions else phi

    def extract_paths(self, ens):
        """Merged unique paths in canonical order.  Returns (elements, num_paths,
        bias) with elements a structured array of PATH_DTYPE."""
        arrs, ea = _ens_args(ens)
        n_paths = ctypes.c_int64(0)
        f = self._lib.or_extract_paths
        f.restype = ctypes.c_int64
        n = f(*ea, ctypes.c_int64(0), None, None, None, None, None, None, None,
              ctypes.byref(n_paths), None)
        cols = dict(path_idx=np.zeros(n, np.int64), feature=np.zeros(n, np.int32),
                    group=np.zeros(n, np.int32), lower=np.zeros(n, np.float32),
                    upper=np.zeros(n, np.float32), zero=np.zeros(n, np.float64),
                    v=np.zeros(n, np.float64))
        bias = np.zeros(ens.num_groups, np.float64)
        n2 = f(*ea, ctypes.c_int64(n), _p(cols["path_idx"]), _p(cols["feature"]),
               _p(cols["group"]), _p(cols["lower"]), _p(cols["upper"]), _p(cols["zero"]),
               _p(cols["v"]), ctypes.byref(n_paths), _p(bias))
        assert n2 == n
        el = np.zeros(n, PATH_DTYPE)
        el["path_idx"], el["feature_idx"], el["group"] = cols["path_idx"], cols["feature"], cols["group"]
        el["lower"], el["upper"] = cols["lower"], cols["upper"]
        el["zero_fraction"], el["v"] = cols["zero"], cols["v"]
        return el, int(n_paths.value), bias

    def pack(self, sizes, groups, capacity: int = 64, alg: str = "bfd"):
        """Bin packing of Section 3.3 per group with alg in {"bfd", "ffd", "nf",
        "none"}.  Returns (bin_of[p], lane_of[p], num_bins)."""
        if alg not in ("bfd", "ffd", "nf", "none"):
            raise ValueError(f"unknown packing algorithm {alg!r}")
        sizes = np.ascontiguousarray(sizes, np.int32)
        groups = np.ascontiguousarray(groups, np.int32)
        n = sizes.shape[0]
        bin_of = np.zeros(n, np.int64)
        lane_of = np.zeros(n, np.int32)
        f = getattr(self._lib, "or_pack_" + alg)
        f.restype = ctypes.c_int64
        k = f(ctypes.c_int64(n), _p(sizes), _p(groups), ctypes.c_int32(capacity),
              _p(bin_of), _p(lane_of))
        if k < 0:
            raise ValueError("an item is larger than the bin capacity")
        return bin_of, lane_of, int(k)

    def pack_bfd(self, sizes, groups, capacity: int = 64):
        """Best-Fit-Decreasing per group.  Returns (bin_of[p], lane_of[p], num_bins)."""
        return self.pack(sizes, groups, capacity, "bfd")


def __getattr__(name):
    # module-level access (oracle.treeshap, ...) goes to the default build
    if name.startswith("_"):
        raise AttributeError(name)
    return getattr(default(), name)
