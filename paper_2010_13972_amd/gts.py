"""ctypes binding of libgts (``include/gts.h``).

Argument marshalling only: extraction, packing and layout run in the
library's host code, SHAP values in its gfx950 kernels.  PyTorch supplies
device memory and the stream.  There is no fallback: if ``libgts.so`` is
missing or fails to load, every call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgts.so")

GTS_OK, GTS_EINVAL, GTS_EPATHLEN, GTS_EBUFSIZE, GTS_ENOMEM, GTS_EDEVICE = range(6)
STATUS_NAMES = {0: "GTS_OK", 1: "GTS_EINVAL", 2: "GTS_EPATHLEN", 3: "GTS_EBUFSIZE",
                4: "GTS_ENOMEM", 5: "GTS_EDEVICE"}
DTYPES = {"f32": 0, "f64": 1}
PACK_ALGS = {"bfd": 0, "ffd": 1, "nf": 2, "none": 3}

# gts_path_element, 40 bytes
PATH_ELEMENT = np.dtype([("path_idx", np.int64), ("feature_idx", np.int32),
                         ("group", np.int32), ("lower", np.float32),
                         ("upper", np.float32), ("zero_fraction", np.float64),
                         ("v", np.float64)])
assert PATH_ELEMENT.itemsize == 40


class GtsError(RuntimeError):
    def __init__(self, status: int, func: str, message: str):
        self.status = status
        super().__init__(f"{func}: {STATUS_NAMES.get(status, status)}: {message}")


class _Ensemble(ctypes.Structure):
    _fields_ = [("num_features", ctypes.c_int32), ("num_groups", ctypes.c_int32),
                ("num_trees", ctypes.c_int64), ("num_nodes", ctypes.c_int64),
                ("tree_node_offsets", ctypes.c_void_p), ("tree_group", ctypes.c_void_p),
                ("left", ctypes.c_void_p), ("right", ctypes.c_void_p),
                ("feature", ctypes.c_void_p), ("threshold", ctypes.c_void_p),
                ("cover", ctypes.c_void_p), ("value", ctypes.c_void_p)]


class ModelDesc(ctypes.Structure):
    """gts_model"""
    _fields_ = [("magic", ctypes.c_uint32), ("dtype", ctypes.c_int32),
                ("num_features", ctypes.c_int32), ("num_groups", ctypes.c_int32),
                ("max_path_len", ctypes.c_int32), ("flags", ctypes.c_int32),
                ("num_elements", ctypes.c_int64), ("num_paths", ctypes.c_int64),
                ("num_bins", ctypes.c_int64), ("bytes", ctypes.c_int64),
                ("off", ctypes.c_int64 * 16)]


_lib = None


class PlanDesc(ctypes.Structure):
    """gts_plan"""
    _fields_ = [("num_paths", ctypes.c_int64), ("num_trees", ctypes.c_int64),
                ("num_bins", ctypes.c_int64), ("num_nodes", ctypes.c_int64),
                ("bytes", ctypes.c_int64), ("off", ctypes.c_int64 * 5)]


class LaunchInfo(ctypes.Structure):
    """gts_launch (include/gts.h)."""
    _fields_ = [("rows_per_tile", ctypes.c_int32), ("waves", ctypes.c_int32),
                ("private_tiles", ctypes.c_int32), ("slices", ctypes.c_int32),
                ("workgroups", ctypes.c_int64), ("lds_bytes", ctypes.c_int64)]


def lib() -> ctypes.CDLL:
    """The loaded libgts.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                              "or python -m paper_2010_13972_amd.build")
        # torch carries its own copy of the HIP runtime.  Loaded first, it is
        # the copy libgts binds to; loaded after libgts had brought in the
        # system one, the process held two runtimes and torch found no device.
        try:
            import torch  # noqa: F401
        except ImportError:
            pass
        L = ctypes.CDLL(LIB_PATH)
        st = ctypes.c_int
        vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        L.gts_extract_paths.argtypes = [ctypes.POINTER(_Ensemble), vp, i64, vp, vp, vp]
        L.gts_extract_paths.restype = st
        L.gts_pack_paths.argtypes = [vp, i64, i32, i32, vp, vp, i64, vp]
        L.gts_pack_paths.restype = st
        L.gts_model_layout.argtypes = [vp, i64, vp, i64, i32, i32, vp, i32,
                                       ctypes.POINTER(ModelDesc), vp, i64]
        L.gts_model_layout.restype = st
        L.gts_prepare_model.argtypes = [ctypes.POINTER(_Ensemble), i32, i32, i32,
                                        ctypes.POINTER(ModelDesc), vp, i64, vp]
        L.gts_prepare_model.restype = st
        L.gts_extract_workspace_bytes.argtypes = [i64, i64, vp]
        L.gts_extract_workspace_bytes.restype = st
        L.gts_extract_paths_device.argtypes = [ctypes.POINTER(_Ensemble), vp, i64, vp, vp, vp,
                                               vp, i64, vp]
        L.gts_extract_paths_device.restype = st
        L.gts_extract_paths_device_noalloc.argtypes = [ctypes.POINTER(_Ensemble), vp, i64, vp,
                                                       vp, vp, vp]
        L.gts_extract_paths_device_noalloc.restype = st
        for name in ("gts_shap", "gts_shap_interactions"):
            f = getattr(L, name)
            f.argtypes = [ctypes.POINTER(ModelDesc), vp, vp, i64, i64, vp, vp]
            f.restype = st
        L.gts_launch_config.argtypes = [ctypes.POINTER(ModelDesc), i64, i32,
                                        ctypes.POINTER(LaunchInfo)]
        L.gts_launch_config.restype = st
        L.gts_plan_model.argtypes = [ctypes.POINTER(_Ensemble), i32, i32, i32,
                                     ctypes.POINTER(ModelDesc), ctypes.POINTER(PlanDesc), vp,
                                     i64]
        L.gts_plan_model.restype = st
        L.gts_build_workspace_bytes.argtypes = [ctypes.POINTER(PlanDesc), vp]
        L.gts_build_workspace_bytes.restype = st
        L.gts_build_model_device.argtypes = [ctypes.POINTER(_Ensemble), ctypes.POINTER(ModelDesc),
                                             ctypes.POINTER(PlanDesc), vp, vp, vp, i64, vp]
        L.gts_build_model_device.restype = st
        L.gts_prune_workspace_bytes.argtypes = [ctypes.POINTER(ModelDesc), i64, vp]
        L.gts_prune_workspace_bytes.restype = st
        L.gts_prune_model.argtypes = [ctypes.POINTER(ModelDesc), vp, vp, i64, i64, vp, i64,
                                      ctypes.POINTER(ModelDesc), ctypes.POINTER(vp), vp]
        L.gts_prune_model.restype = st
        L.gts_set_host_threads.argtypes = [i32]
        L.gts_set_host_threads.restype = st
        L.gts_last_error.restype = ctypes.c_char_p
        L.gts_version.restype = ctypes.c_char_p
        _lib = L
    return _lib


def last_error() -> str:
    return lib().gts_last_error().decode()


def set_host_threads(n: int):
    """gts_set_host_threads: cap the host threads of the calling thread's
    library calls (0: every core, up to 16)."""
    _check(lib().gts_set_host_threads(int(n)), "gts_set_host_threads")


def version() -> str:
    return lib().gts_version().decode()


def _check(status: int, func: str):
    if status != GTS_OK:
        raise GtsError(status, func, last_error())


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


# ----------------------------------------------------------------------------
# host calls
# ----------------------------------------------------------------------------

def _ensemble_struct(ens):
    arrs = dict(
        off=np.ascontiguousarray(ens.tree_node_offsets, np.int64),
        group=np.ascontiguousarray(ens.tree_group, np.int32),
        left=np.ascontiguousarray(ens.left, np.int32),
        right=np.ascontiguousarray(ens.right, np.int32),
        feat=np.ascontiguousarray(ens.feature, np.int32),
        thr=np.ascontiguousarray(ens.threshold, np.float32),
        cover=np.ascontiguousarray(ens.cover, np.float64),
        value=np.ascontiguousarray(ens.value, np.float64))
    s = _Ensemble(ens.num_features, ens.num_groups, len(arrs["group"]), len(arrs["left"]),
                  arrs["off"].ctypes.data, arrs["group"].ctypes.data, arrs["left"].ctypes.data,
                  arrs["right"].ctypes.data, arrs["feat"].ctypes.data, arrs["thr"].ctypes.data,
                  arrs["cover"].ctypes.data, arrs["value"].ctypes.data)
    return s, arrs


def extract_paths(ens) -> Tuple[np.ndarray, int, np.ndarray]:
    """gts_extract_paths: (elements[PATH_ELEMENT], num_paths, bias[G])."""
    s, keep = _ensemble_struct(ens)
    n = ctypes.c_int64(0)
    npaths = ctypes.c_int64(0)
    _check(lib().gts_extract_paths(ctypes.byref(s), None, 0, ctypes.byref(n),
                                   ctypes.byref(npaths), None), "gts_extract_paths")
    out = np.zeros(n.value, PATH_ELEMENT)
    bias = np.zeros(ens.num_groups, np.float64)
    _check(lib().gts_extract_paths(ctypes.byref(s), _ptr(out), n.value, ctypes.byref(n),
                                   ctypes.byref(npaths), _ptr(bias)), "gts_extract_paths")
    return out, int(npaths.value), bias


class DeviceEnsemble:
    """An ensemble's node arrays in device memory (torch tensors), with the
    gts_ensemble struct that points at them."""

    def __init__(self, ens, device="cuda"):
        import torch
        _, arrs = _ensemble_struct(ens)
        self.tensors = {k: torch.from_numpy(v).to(device) for k, v in arrs.items()}
        t = self.tensors
        self.num_trees = len(arrs["group"])
        self.num_nodes = len(arrs["left"])
        self.num_groups = ens.num_groups
        self.struct = _Ensemble(ens.num_features, ens.num_groups, self.num_trees,
                                self.num_nodes, t["off"].data_ptr(), t["group"].data_ptr(),
                                t["left"].data_ptr(), t["right"].data_ptr(),
                                t["feat"].data_ptr(), t["thr"].data_ptr(),
                                t["cover"].data_ptr(), t["value"].data_ptr())


def extract_paths_device(dens: DeviceEnsemble, stream=None, workspace=None):
    """gts_extract_paths_device: (elements as a device uint8 tensor of
    num_elements * 40 bytes, num_paths, bias as a device float64 tensor)."""
    import torch
    dev = dens.tensors["left"].device
    ws_bytes = ctypes.c_int64(0)
    _check(lib().gts_extract_workspace_bytes(dens.num_trees, dens.num_nodes,
                                             ctypes.byref(ws_bytes)),
           "gts_extract_workspace_bytes")
    if workspace is None or workspace.numel() < ws_bytes.value:
        workspace = torch.empty(ws_bytes.value, dtype=torch.uint8, device=dev)
    n = ctypes.c_int64(0)
    npaths = ctypes.c_int64(0)
    h = _stream_handle(stream)
    _check(lib().gts_extract_paths_device(ctypes.byref(dens.struct), None, 0, ctypes.byref(n),
                                          ctypes.byref(npaths), None,
                                          ctypes.c_void_p(workspace.data_ptr()),
                                          workspace.numel(), h), "gts_extract_paths_device")
    out = torch.empty(max(1, n.value) * PATH_ELEMENT.itemsize, dtype=torch.uint8, device=dev)
    bias = torch.empty(dens.num_groups, dtype=torch.float64, device=dev)
    _check(lib().gts_extract_paths_device(ctypes.byref(dens.struct),
                                          ctypes.c_void_p(out.data_ptr()), n.value,
                                          ctypes.byref(n), ctypes.byref(npaths),
                                          ctypes.c_void_p(bias.data_ptr()),
                                          ctypes.c_void_p(workspace.data_ptr()),
                                          workspace.numel(), h), "gts_extract_paths_device")
    return out[:n.value * PATH_ELEMENT.itemsize], int(npaths.value), bias


def extract_paths_device_noalloc(dens: DeviceEnsemble, stream=None):
    """gts_extract_paths_device_noalloc: as extract_paths_device, with the
    library's fixed device workspace instead of a caller's."""
    import torch
    dev = dens.tensors["left"].device
    n = ctypes.c_int64(0)
    npaths = ctypes.c_int64(0)
    h = _stream_handle(stream)
    _check(lib().gts_extract_paths_device_noalloc(ctypes.byref(dens.struct), None, 0,
                                                  ctypes.byref(n), ctypes.byref(npaths), None, h),
           "gts_extract_paths_device_noalloc")
    out = torch.empty(max(1, n.value) * PATH_ELEMENT.itemsize, dtype=torch.uint8, device=dev)
    bias = torch.empty(dens.num_groups, dtype=torch.float64, device=dev)
    _check(lib().gts_extract_paths_device_noalloc(ctypes.byref(dens.struct),
                                                  ctypes.c_void_p(out.data_ptr()), n.value,
                                                  ctypes.byref(n), ctypes.byref(npaths),
                                                  ctypes.c_void_p(bias.data_ptr()), h),
           "gts_extract_paths_device_noalloc")
    return out[:n.value * PATH_ELEMENT.itemsize], int(npaths.value), bias


def elements_from_device(raw) -> np.ndarray:
    """A device byte tensor of gts_path_element records as a host array."""
    return np.frombuffer(raw.cpu().numpy().tobytes(), dtype=PATH_ELEMENT).copy()


def pack_paths(elements: np.ndarray, bin_capacity: int = 64,
               alg: str = "bfd") -> Tuple[np.ndarray, np.ndarray]:
    """gts_pack_paths: (packed elements, bin_offsets[num_bins+1])."""
    elements = np.ascontiguousarray(elements, PATH_ELEMENT)
    k = ctypes.c_int64(0)
    a = PACK_ALGS[alg]
    # one call: there are never more bins than paths
    num_paths = int(np.count_nonzero(elements["feature_idx"] == -1))
    packed = np.empty(len(elements), PATH_ELEMENT)
    offs = np.empty(num_paths + 1, np.int64)
    _check(lib().gts_pack_paths(_ptr(elements), len(elements), bin_capacity, a, _ptr(packed),
                                _ptr(offs), len(offs), ctypes.byref(k)), "gts_pack_paths")
    return packed, offs[:k.value + 1].copy()


def model_layout(packed: np.ndarray, bin_offsets: np.ndarray, num_features: int,
                 num_groups: int, bias: np.ndarray, dtype: str = "f32"):
    """gts_model_layout: (ModelDesc, host blob as uint8 array)."""
    packed = np.ascontiguousarray(packed, PATH_ELEMENT)
    bin_offsets = np.ascontiguousarray(bin_offsets, np.int64)
    bias = np.ascontiguousarray(bias, np.float64)
    desc = ModelDesc()
    args = (_ptr(packed), len(packed), _ptr(bin_offsets), len(bin_offsets) - 1, num_features,
            num_groups, _ptr(bias), DTYPES[dtype])
    _check(lib().gts_model_layout(*args, ctypes.byref(desc), None, 0), "gts_model_layout")
    blob = np.empty(desc.bytes, np.uint8)
    _check(lib().gts_model_layout(*args, ctypes.byref(desc), _ptr(blob), len(blob)),
           "gts_model_layout")
    return desc, blob


# ----------------------------------------------------------------------------
# device calls
# ----------------------------------------------------------------------------

class DeviceModel:
    """A packed model resident in device memory (torch uint8 tensor)."""

    def __init__(self, desc: ModelDesc, blob, num_features: int, num_groups: int, dtype: str,
                 num_paths: int, num_bins: int, bias: np.ndarray):
        self.desc = desc
        self.blob = blob
        self.num_features = num_features
        self.num_groups = num_groups
        self.dtype = dtype
        self.num_paths = num_paths
        self.num_bins = num_bins
        self.bias = bias

    @property
    def torch_dtype(self):
        import torch
        return torch.float64 if self.dtype == "f64" else torch.float32


def upload(desc: ModelDesc, blob: np.ndarray, num_features: int, num_groups: int, dtype: str,
           bias: np.ndarray, device="cuda") -> DeviceModel:
    import torch
    t = torch.from_numpy(blob).to(device, non_blocking=False)
    return DeviceModel(desc, t, num_features, num_groups, dtype, desc.num_paths, desc.num_bins,
                       bias)


def prepare_blob(ens, dtype: str = "f32", bin_capacity: int = 64, alg: str = "bfd",
                 out: Optional[np.ndarray] = None, _cache={}):
    """gts_prepare_model: (ModelDesc, host blob, bias) straight from the
    ensemble.  The blob is written into ``out`` (a uint8 array, e.g. a view of
    pinned memory) when it is large enough, else into a new array.  The blob
    size of the last model with the same node count is tried first, so
    repeated preparation of one ensemble is a single call."""
    s, keep = _ensemble_struct(ens)
    desc = ModelDesc()
    bias = np.zeros(ens.num_groups, np.float64)
    key = (ens.num_nodes, ens.num_trees, dtype, bin_capacity, alg)
    size = _cache.get(key, 0)
    if size and out is not None and out.nbytes >= size:
        blob = out
    else:
        blob = np.empty(size, np.uint8) if size else None
    cap = blob.nbytes if blob is not None else 0
    st = lib().gts_prepare_model(ctypes.byref(s), bin_capacity, PACK_ALGS[alg], DTYPES[dtype],
                                 ctypes.byref(desc), _ptr(blob), cap, _ptr(bias))
    if st == GTS_OK and blob is not None and desc.bytes <= cap:
        _cache[key] = int(desc.bytes)
        return desc, blob[:desc.bytes], bias
    if st not in (GTS_OK, GTS_EBUFSIZE):
        _check(st, "gts_prepare_model")
    if out is not None and out.nbytes >= desc.bytes:
        blob = out
    else:
        blob = np.empty(desc.bytes, np.uint8)
    _check(lib().gts_prepare_model(ctypes.byref(s), bin_capacity, PACK_ALGS[alg], DTYPES[dtype],
                                   ctypes.byref(desc), _ptr(blob), blob.nbytes, _ptr(bias)),
           "gts_prepare_model")
    _cache[key] = int(desc.bytes)
    return desc, blob[:desc.bytes], bias


def plan_model(ens, dtype: str = "f32", bin_capacity: int = 64, alg: str = "bfd",
               out: Optional[np.ndarray] = None):
    """gts_plan_model: (ModelDesc of the blob to build, PlanDesc, host plan blob
    as a uint8 array; written into ``out`` when it is large enough)."""
    s, keep = _ensemble_struct(ens)
    desc, plan = ModelDesc(), PlanDesc()
    _check(lib().gts_plan_model(ctypes.byref(s), bin_capacity, PACK_ALGS[alg], DTYPES[dtype],
                                ctypes.byref(desc), ctypes.byref(plan), None, 0),
           "gts_plan_model")
    buf = out if out is not None and out.nbytes >= plan.bytes else np.empty(plan.bytes, np.uint8)
    _check(lib().gts_plan_model(ctypes.byref(s), bin_capacity, PACK_ALGS[alg], DTYPES[dtype],
                                ctypes.byref(desc), ctypes.byref(plan), _ptr(buf), buf.nbytes),
           "gts_plan_model")
    return desc, plan, buf[:plan.bytes]


def build_workspace_bytes(plan: PlanDesc) -> int:
    n = ctypes.c_int64(0)
    _check(lib().gts_build_workspace_bytes(ctypes.byref(plan), ctypes.byref(n)),
           "gts_build_workspace_bytes")
    return int(n.value)


def build_model_device(dens: "DeviceEnsemble", desc: ModelDesc, plan: PlanDesc, d_plan,
                       dtype: str, out=None, workspace=None, stream=None) -> DeviceModel:
    """gts_build_model_device: the model blob of a plan, written on the GPU
    into ``out`` (a device uint8 tensor of desc.bytes; allocated when None)."""
    import torch
    dev = dens.tensors["left"].device
    if out is None or out.numel() < desc.bytes:
        out = torch.empty(desc.bytes, dtype=torch.uint8, device=dev)
    need = build_workspace_bytes(plan)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    _check(lib().gts_build_model_device(ctypes.byref(dens.struct), ctypes.byref(desc),
                                        ctypes.byref(plan), ctypes.c_void_p(d_plan.data_ptr()),
                                        ctypes.c_void_p(out.data_ptr()),
                                        ctypes.c_void_p(workspace.data_ptr()), workspace.numel(),
                                        _stream_handle(stream)), "gts_build_model_device")
    return DeviceModel(desc, out[:desc.bytes], desc.num_features, desc.num_groups, dtype,
                       desc.num_paths, desc.num_bins, None)


def prepare(ens, dtype: str = "f32", device="cuda", bin_capacity: int = 64,
            alg: str = "bfd") -> DeviceModel:
    """Extract, pack, lay out and upload an ensemble (Section 3, steps 1-3)."""
    desc, blob, bias = prepare_blob(ens, dtype, bin_capacity, alg)
    return upload(desc, blob, ens.num_features, ens.num_groups, dtype, bias, device)


def prepare_stepwise(ens, dtype: str = "f32", device="cuda", bin_capacity: int = 64,
                     alg: str = "bfd") -> DeviceModel:
    """The same as prepare() through the three separate host calls."""
    elements, _, bias = extract_paths(ens)
    packed, offs = pack_paths(elements, bin_capacity, alg)
    desc, blob = model_layout(packed, offs, ens.num_features, ens.num_groups, bias, dtype)
    return upload(desc, blob, ens.num_features, ens.num_groups, dtype, bias, device)


def _stream_handle(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _check_X(model: DeviceModel, X):
    import torch
    if not isinstance(X, torch.Tensor) or X.device.type != "cuda":
        raise TypeError("X must be a CUDA (HIP) torch tensor")
    if X.dtype != torch.float32 or X.dim() != 2 or X.stride(1) != 1:
        raise TypeError("X must be a 2-D float32 tensor with unit column stride")
    if X.shape[1] < model.num_features:
        raise ValueError(f"X has {X.shape[1]} columns, the model needs {model.num_features}")
    ld = X.stride(0) if X.shape[0] > 1 else max(X.shape[1], model.num_features)
    return X.shape[0], ld


def shap(model: DeviceModel, X, out=None, stream=None):
    """gts_shap: phi[rows, G, M+1] (bias in the last column)."""
    import torch
    rows, ld = _check_X(model, X)
    shape = (rows, model.num_groups, model.num_features + 1)
    if out is None:
        out = torch.empty(shape, dtype=model.torch_dtype, device=X.device)
    elif tuple(out.shape) != shape or out.dtype != model.torch_dtype or not out.is_contiguous():
        raise ValueError(f"out must be a contiguous {model.torch_dtype} tensor of shape {shape}")
    _check(lib().gts_shap(ctypes.byref(model.desc), ctypes.c_void_p(model.blob.data_ptr()),
                          ctypes.c_void_p(X.data_ptr()), rows, ld,
                          ctypes.c_void_p(out.data_ptr()), _stream_handle(stream)), "gts_shap")
    return out


def shap_interactions(model: DeviceModel, X, out=None, stream=None):
    """gts_shap_interactions: phi[rows, G, M+1, M+1] (bias at [M, M])."""
    import torch
    rows, ld = _check_X(model, X)
    W = model.num_features + 1
    shape = (rows, model.num_groups, W, W)
    if out is None:
        out = torch.empty(shape, dtype=model.torch_dtype, device=X.device)
    elif tuple(out.shape) != shape or out.dtype != model.torch_dtype or not out.is_contiguous():
        raise ValueError(f"out must be a contiguous {model.torch_dtype} tensor of shape {shape}")
    _check(lib().gts_shap_interactions(ctypes.byref(model.desc),
                                       ctypes.c_void_p(model.blob.data_ptr()),
                                       ctypes.c_void_p(X.data_ptr()), rows, ld,
                                       ctypes.c_void_p(out.data_ptr()), _stream_handle(stream)),
           "gts_shap_interactions")
    return out


def prune_workspace_bytes(model: DeviceModel, rows: int) -> int:
    """gts_prune_workspace_bytes for this model and row count."""
    n = ctypes.c_int64(0)
    _check(lib().gts_prune_workspace_bytes(ctypes.byref(model.desc), int(rows), ctypes.byref(n)),
           "gts_prune_workspace_bytes")
    return int(n.value)


def prune(model: DeviceModel, X, workspace=None, stream=None) -> DeviceModel:
    """gts_prune_model: the model without the paths that no row of X reaches,
    for shap / shap_interactions on the same X.  The pruned blob lives in
    ``workspace`` (a device uint8 tensor; allocated when None or too small),
    which must stay alive and unchanged while the returned model is used."""
    import torch
    rows, ld = _check_X(model, X)
    need = prune_workspace_bytes(model, rows)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=X.device)
    desc = ModelDesc()
    ptr = ctypes.c_void_p()
    _check(lib().gts_prune_model(ctypes.byref(model.desc), ctypes.c_void_p(model.blob.data_ptr()),
                                 ctypes.c_void_p(X.data_ptr()), rows, ld,
                                 ctypes.c_void_p(workspace.data_ptr()), workspace.numel(),
                                 ctypes.byref(desc), ctypes.byref(ptr), _stream_handle(stream)),
           "gts_prune_model")
    off = (ptr.value or workspace.data_ptr()) - workspace.data_ptr()
    blob = workspace[off:off + desc.bytes]
    return DeviceModel(desc, blob, model.num_features, model.num_groups, model.dtype,
                       model.num_paths, model.num_bins, model.bias)


def launch_config(model: DeviceModel, rows: int, interactions: bool = False) -> dict:
    """gts_launch_config: the launch shape gts_shap (or gts_shap_interactions)
    uses for this model and row count on the current device."""
    info = LaunchInfo()
    _check(lib().gts_launch_config(ctypes.byref(model.desc), int(rows), 1 if interactions else 0,
                                   ctypes.byref(info)), "gts_launch_config")
    return {name: int(getattr(info, name)) for name, _ in LaunchInfo._fields_}
