"""Benchmark: exact TreeShap rows/s on one MI355X.

One step is one pass of the whole path over one batch of rows of the deep
regression workload (1000 trees, depth <= 16, split probability 0.7, at most
1024 leaves per tree, M = 8, 10 000 rows, fp32): path extraction with
duplicate merging and the bias, Best-Fit-Decreasing packing into 64-element
bins and the device layout of the model, then on the device the model pruned
for the batch (the paths none of its rows reaches dropped, gts_prune_model;
--no-prune leaves this out) and the SHAP kernel over the batch.  By default
(--build auto) the host runs the validating walk that counts the paths, the
packing and each path's place (gts_plan_model), the plan is uploaded, and
the GPU extracts, merges and lays out the paths and sums the bias
(gts_build_model_device); --build host prepares the whole blob on the host
(gts_prepare_model) and uploads it.  Three steps' host work runs at once on
the library's worker pool, which serves the oldest first.  The inputs, the
rows X and the ensemble's node arrays, are resident in HBM (the ensemble also
in host memory, for the plans) before timing starts.  `value` is rows explained per second over the timed
steps.

The same JSON line carries:
  roofline      the SHAP kernel against the MI355X FP32 vector peak.  Its
                algorithmic flops are the op model (10 q^2 + 8 q per
                (row, path) with q path features; interactions add
                q (q-1)(10 q + 4)) summed over the live (row, path) pairs --
                a pair with a zero-cover element whose range misses the row
                contributes exactly nothing and is not work the method needs
                -- counted exactly on the device; its duration is the mean
                of HIP events around its launches inside the timed steps, on
                the launch stream.  HBM traffic and executed VALU
                instructions come from rocprofv3 counters of the same kernel
                code (null when the kernel sources differ from the ones the
                counters were taken on);
  kernel        kernel-only rows/s over back-to-back launches;
  configs       every workload of the suite (tiny, covtype-shaped, deep fp32
                and fp64, wide multiclass, interactions): host preparation,
                device extraction, the plan and the device build where the
                model admits a plan, kernel time and rows/s, live pairs,
                modelled rate and fraction, the pruning pass and the kernel on
                the pruned model, and the CPU oracle's rate on a row prefix;
  cpu_baseline  the fp64 CPU oracle (Algorithm 1, OpenMP over rows) on a row
                prefix of the headline batch, on the host's cores, and on one
                thread.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_FP32_TFLOPS = 157.3   # MI355X FP32 vector, vendor figure
PEAK_FP64_TFLOPS = 78.6    # MI355X FP64 vector
PEAK_HBM_GBPS = 8000.0     # MI355X HBM3E
# Non-packed FP32 wave64 VALU instructions issued per SIMD per cycle, measured
# with standalone FMA streams on this chip (about 129 TFLOP/s of FMAs over 1024
# SIMDs at 2.4 GHz): the ceiling for code built without packed FP32.
VALU_ISSUE_CEILING = 0.41
SIMDS = 256 * 4
CLOCK_HZ = 2.4e9
METRIC = "rows/sec for SHAP values and SHAP interaction values; % FP32 VALU peak"
CSRC = os.path.join(ROOT, "paper_2010_13972_amd", "csrc")
KERNEL_SOURCES = [os.path.join(CSRC, f) for f in (
    "gts_shap_kernel.h", "gts_launch.h", "gts_kernels.hip", "gts_shap_f32.hip",
    "gts_shap_f64.hip", "gts_inter_f32.hip", "gts_inter_f64.hip", "gts_prune.hip")]

WORKLOAD_TEXT = {
    "tiny": "tiny: 10 full depth-3 trees, M=8, X~U[0,1), 256 rows",
    "covtype_med": "covtype-shaped: 100 trees, depth<=8, p_split=0.85, M=54 "
                   "(10 N(0,1) + 44 Bernoulli(0.2)), 10k rows",
    "deep": "deep: 1000 trees, depth<=16, p_split=0.7, <=1024 leaves, M=8, N(0,1), 10k rows",
    "wide": "wide: 10 classes x 100 rounds, depth<=8, p_split=0.85, M=784, 50% zeros, 10k rows",
    "interactions": "covtype-shaped model, 1000 rows, SHAP interaction values",
}

# The suite: (name, workload, dtype, interactions)
SUITE = [
    ("tiny_f64", "tiny", "f64", False),
    ("covtype_med_f32", "covtype_med", "f32", False),
    ("deep_f32", "deep", "f32", False),
    ("deep_f64", "deep", "f64", False),
    ("wide_f32", "wide", "f32", False),
    ("interactions_f32", "interactions", "f32", True),
]

# rocprofv3 counters of the SHAP kernel per launch, keyed by (workload, dtype,
# interactions), with a fourth entry "pruned" for the kernel on the model
# pruned for the batch; `source` is kernel_source_hash() of the kernel sources the
# counters were taken on.  fetch_bytes / write_bytes: FETCH_SIZE and
# WRITE_SIZE, each scaled by the ratio of a plain 256 MiB copy's true bytes to
# the counter's reading of it.  valu_insts / salu_insts / lds_insts:
# SQ_INSTS_VALU / SQ_INSTS_SALU / SQ_INSTS_LDS (wave instructions).  The
# summaries and the commands that made them are in profiles/.
COUNTERS = {
    ('deep', 'f32', False): {"fetch_bytes": 63853273, "write_bytes": 46080000, "valu_insts": 1788702723, "salu_insts": 347312558, "lds_insts": 276472423, "source": "350d1b7705dfaf9f090c31ecde4176169ea0ea396c0774d3335996c7356ca8be"},
    ('deep', 'f32', False, 'pruned'): {"fetch_bytes": 8800363, "write_bytes": 8640000, "valu_insts": 809664337, "salu_insts": 160894055, "lds_insts": 137874440, "source": "350d1b7705dfaf9f090c31ecde4176169ea0ea396c0774d3335996c7356ca8be"},
    ('deep', 'f64', False): {"fetch_bytes": 73801557, "write_bytes": 92160000, "valu_insts": 1879096606, "salu_insts": 322527272, "lds_insts": 292643883, "source": "350d1b7705dfaf9f090c31ecde4176169ea0ea396c0774d3335996c7356ca8be"},
    ('deep', 'f64', False, 'pruned'): {"fetch_bytes": 9788162, "write_bytes": 17280000, "valu_insts": 880342252, "salu_insts": 134735606, "lds_insts": 152810820, "source": "350d1b7705dfaf9f090c31ecde4176169ea0ea396c0774d3335996c7356ca8be"},
    ('covtype_med', 'f32', False): {"fetch_bytes": 19339592, "write_bytes": 35200000, "valu_insts": 288902461, "salu_insts": 73822658, "lds_insts": 41738121, "source": "350d1b7705dfaf9f090c31ecde4176169ea0ea396c0774d3335996c7356ca8be"},
    ('covtype_med', 'f32', False, 'pruned'): {"fetch_bytes": 19017006, "write_bytes": 35200000, "valu_insts": 280929231, "salu_insts": 67801742, "lds_insts": 41065418, "source": "350d1b7705dfaf9f090c31ecde4176169ea0ea396c0774d3335996c7356ca8be"},
    ('wide', 'f32', False): {"fetch_bytes": 415594796, "write_bytes": 316800000, "valu_insts": 5550767852, "salu_insts": 1076499619, "lds_insts": 765583007, "source": "350d1b7705dfaf9f090c31ecde4176169ea0ea396c0774d3335996c7356ca8be"},
    ('wide', 'f32', False, 'pruned'): {"fetch_bytes": 414847272, "write_bytes": 316800000, "valu_insts": 5506767273, "salu_insts": 1055679113, "lds_insts": 754426459, "source": "350d1b7705dfaf9f090c31ecde4176169ea0ea396c0774d3335996c7356ca8be"},
    ('interactions', 'f32', True): {"fetch_bytes": 11157364, "write_bytes": 48400000, "valu_insts": 181893001, "salu_insts": 31405970, "lds_insts": 16051232, "source": "350d1b7705dfaf9f090c31ecde4176169ea0ea396c0774d3335996c7356ca8be"},
    ('interactions', 'f32', True, 'pruned'): {"fetch_bytes": 9414571, "write_bytes": 48400000, "valu_insts": 156394351, "salu_insts": 27377190, "lds_insts": 13662430, "source": "350d1b7705dfaf9f090c31ecde4176169ea0ea396c0774d3335996c7356ca8be"},
}


def kernel_source_hash() -> str:
    """SHA-256 of the kernel sources' code: line comments and blank lines are
    dropped, so editing a comment keeps the measured counters."""
    code = []
    for path in KERNEL_SOURCES:
        with open(path) as f:
            for line in f:
                c = line.split("//", 1)[0].rstrip()
                if c.strip():
                    code.append(c)
    return hashlib.sha256("\n".join(code).encode()).hexdigest()


def counters_for(key):
    c = COUNTERS.get(key)
    if c is None or c["source"] != kernel_source_hash():
        return None
    return c


def traffic_for(key):
    c = counters_for(key)
    return None if c is None else c["fetch_bytes"] + c["write_bytes"]


def executed(key, kernel_ms: float):
    """Counter-derived rates of the kernel: HBM GB/s from FETCH_SIZE +
    WRITE_SIZE, VALU lane operations (instructions x 64) and the VALU issue
    rate per SIMD-cycle, also as a fraction of the measured non-packed
    ceiling."""
    c = counters_for(key)
    if c is None:
        return None
    s = kernel_ms * 1e-3
    issue = c["valu_insts"] / (s * SIMDS * CLOCK_HZ)
    return {"hbm_gbps": (c["fetch_bytes"] + c["write_bytes"]) / s / 1e9,
            "hbm_frac": (c["fetch_bytes"] + c["write_bytes"]) / s / 1e9 / PEAK_HBM_GBPS,
            "valu_lane_ops_per_launch": 64 * c["valu_insts"],
            "valu_issue_per_simd_cycle": issue,
            "valu_issue_frac_of_ceiling": issue / VALU_ISSUE_CEILING,
            "salu_insts_per_launch": c["salu_insts"], "lds_insts_per_launch": c["lds_insts"],
            "counters_source": c["source"][:16]}


def op_model(q: np.ndarray, interactions: bool) -> np.ndarray:
    """Flops per (row, path) for paths of q features."""
    q = q.astype(np.float64)
    f = 10 * q * q + 8 * q
    if interactions:
        f = f + q * (q - 1) * (10 * q + 4)
    return f


def modelled_flops(q: np.ndarray, interactions: bool) -> float:
    """Per row: the op model summed over the extracted paths."""
    return float(op_model(q, interactions).sum())


def path_features(gts, ens) -> np.ndarray:
    el, _, _ = gts.extract_paths(ens)
    roots = np.flatnonzero(el["feature_idx"] == -1)
    return np.diff(np.append(roots, len(el))) - 1


def live_pairs(torch, gts, ens, X: np.ndarray, dtype: str, tile: int = 64, dev: str = "cuda"):
    """Exact count of the live (row, path) pairs: a pair is dead when the path
    has an element whose zero fraction is 0 (in the model's precision) and
    whose range [lower, upper) misses the row -- its weight polynomial has a
    factor z + o t = 0 and it contributes exactly nothing.  Counted on the
    device (torch), per path: live rows, and live tiles of `tile` rows.
    Returns (q per path, live rows per path, live tiles per path)."""
    el, _, _ = gts.extract_paths(ens)
    roots = np.flatnonzero(el["feature_idx"] == -1)
    P = len(roots)
    q = np.diff(np.append(roots, len(el))) - 1
    rows = X.shape[0]
    ntiles = (rows + tile - 1) // tile
    live_rows = np.full(P, rows, np.int64)
    live_tiles = np.full(P, ntiles, np.int64)
    z = el["zero_fraction"].astype(np.float32 if dtype == "f32" else np.float64)
    zero = (z == 0) & (el["feature_idx"] >= 0)
    if not zero.any() or rows == 0:
        return q, live_rows, live_tiles
    path_of = np.cumsum(el["feature_idx"] == -1) - 1
    zi = np.flatnonzero(zero)
    zp = path_of[zi]
    counts = np.bincount(zp, minlength=P)
    K = int(counts.max())
    # [P, K] padded with an always-true element
    rank = np.arange(len(zi)) - np.searchsorted(zp, zp)   # zi is sorted by path
    F = np.zeros((P, K), np.int64)
    Lo = np.full((P, K), -np.inf, np.float32)
    Hi = np.full((P, K), np.inf, np.float32)
    F[zp, rank] = el["feature_idx"][zi]
    Lo[zp, rank] = el["lower"][zi]
    Hi[zp, rank] = el["upper"][zi]
    has = np.flatnonzero(counts > 0)
    Xt = torch.from_numpy(np.ascontiguousarray(X.T, np.float32)).to(dev)   # [M, rows]
    pad = ntiles * tile - rows
    chunk = max(1, (1 << 28) // max(1, K * rows))
    for a in range(0, len(has), chunk):
        idx = has[a:a + chunk]
        f = torch.from_numpy(F[idx]).to(dev)
        lo = torch.from_numpy(Lo[idx]).to(dev)[..., None]
        hi = torch.from_numpy(Hi[idx]).to(dev)[..., None]
        vals = Xt[f]                                              # [C, K, rows]
        ok = ((lo <= vals) & (vals < hi)).all(dim=1)              # [C, rows]
        live_rows[idx] = ok.sum(dim=1).cpu().numpy()
        if pad:
            ok = torch.nn.functional.pad(ok, (0, pad))
        live_tiles[idx] = ok.view(len(idx), ntiles, tile).any(dim=2).sum(dim=1).cpu().numpy()
    return q, live_rows, live_tiles


def work_model(torch, gts, ens, X, dtype, interactions):
    """Algorithmic flops of one launch over X: the op model over the live
    (row, path) pairs, and over all pairs (dense equivalent)."""
    q, lr, lt = live_pairs(torch, gts, ens, X, dtype)
    f = op_model(q, interactions)
    rows = X.shape[0]
    return {"flops_live": float((f * lr).sum()), "flops_dense": float(f.sum() * rows),
            "pairs": int(len(q)) * rows, "live_pairs": int(lr.sum()),
            "tile_pairs": int(len(q)) * int(-(-rows // 64)), "live_tile_pairs": int(lt.sum()),
            "paths": int(len(q)), "path_elements": int((q + 1).sum())}


def kernel_fn(gts, interactions):
    return gts.shap_interactions if interactions else gts.shap


def time_pipeline(torch, gts, ens, Xd, dtype, steps, warmup, interactions, nstreams=1,
                  preps=2, prune=True, device_build=False, prep_threads=None,
                  keep_outputs=False, split=False):
    """Whole-path steps, pipelined.  `preps` host threads prepare the models
    of consecutive steps at the same time: step k runs gts_prepare_model on
    thread k mod preps, into pinned buffer k mod NB (NB = preps + nstreams +
    3: a step's buffers are reused once the kernel of the step NB before it
    is done, so the host can run that far ahead).  The
    preparations share the library's worker pool, which serves the one that
    started first; each may use every core unless `prep_threads` caps it
    (through gts_set_host_threads).  The main
    thread uploads step k's model on a copy stream into device buffer k mod NB
    once it is prepared and launches the kernel of step k as soon as that
    upload has finished, on compute stream k mod nstreams; the compute
    streams hold only kernels, with no cross-stream waits.  The host orders buffer reuse: a preparation waits until the kernel
    that last used its buffers has been launched and its upload has finished,
    an upload for the kernel that last read its device buffer.  The loop
    calls the C ABI with arguments marshalled once.  With `prune`, each step
    first prunes its model for the batch (gts_prune_model, on the compute
    stream, into that stream's workspace) and runs the kernel on the pruned
    model.  With `device_build`, a preparation is gts_plan_model (the host
    half: the counting walk, the packing, each path's place) into a pinned
    plan buffer, the plan goes up once it is made (the ensemble, an input
    like X, is resident in HBM and in host memory), and the compute stream
    runs
    gts_build_model_device (extraction and merging into the blob on the GPU)
    before the pruning and the kernel.  Timed on the host clock; the build,
    the pruning and the kernel are bracketed by HIP events on their stream,
    each preparation by the host clock of its thread.  With `split`, every
    step's build and pruning run on one stream and every SHAP kernel on
    another (the kernel stream waits, on the GPU, for the step's pruned
    model; the pruning waits for the kernel that last read its workspace,
    two alternate), so the build and pruning of a step overlap the kernel
    of the one before while the kernels run back to back; `nstreams` is
    then unused.  With `keep_outputs`
    (for tests, not for timing) every timed step's output is copied on its
    stream after its kernel, and the copies are returned last."""
    import collections
    import ctypes
    import gc
    import queue
    import threading
    L = gts.lib()
    launch = L.gts_shap_interactions if interactions else L.gts_shap
    NB = preps + nstreams + 3
    if split:
        nstreams = 2   # workspaces and output buffers, alternating by step
    computes = [torch.cuda.current_stream()] + [torch.cuda.Stream()
                                                for _ in range(nstreams - 1)]
    # split: builds and prunings on pstream, kernels on kstream
    kstream = computes[0]
    pstream = torch.cuda.Stream() if split else None
    build_streams = [pstream if split else computes[j] for j in range(nstreams)]
    kernel_streams = [kstream if split else computes[j] for j in range(nstreams)]
    pruned_ev = [torch.cuda.Event() for _ in range(nstreams)]   # step's model ready
    shap_done = [torch.cuda.Event() for _ in range(nstreams)]   # kernel read workspace j
    copy = torch.cuda.Stream()
    desc0 = gts.prepare_blob(ens, dtype)[0]
    nbytes = int(desc0.bytes)
    dev = [torch.empty(nbytes, dtype=torch.uint8, device="cuda") for _ in range(NB)]
    if device_build:
        # the ensemble as the host walks it (pinned, so its upload is a DMA),
        # one device copy per buffer, the plan buffers and the build workspace
        plan0 = gts.plan_model(ens, dtype)[1]
        _, arrs = gts._ensemble_struct(ens)
        # the node arrays in one buffer (each 256-byte aligned), so a step's
        # ensemble upload is one copy
        names = ("off", "group", "left", "right", "feat", "thr", "cover", "value")
        offs, total = {}, 0
        for k in names:
            offs[k] = total
            total += (arrs[k].nbytes + 255) // 256 * 256
        ens_host = torch.empty(total, dtype=torch.uint8)
        for k in names:
            ens_host[offs[k]:offs[k] + arrs[k].nbytes].copy_(
                torch.from_numpy(arrs[k].view(np.uint8)))
        # the ensemble is an input of the path like X: resident in HBM (and
        # in host memory for the plans) before timing starts, read by every
        # step's build
        ens_dev = ens_host.cuda()

        def ens_struct(t):
            base = t.data_ptr()
            return gts._Ensemble(ens.num_features, ens.num_groups, len(arrs["group"]),
                                 len(arrs["left"]), *(base + offs[k] for k in names))

        host_ens = ens_struct(ens_host)
        dev_ens = ens_struct(ens_dev)
        pinned = [torch.empty(int(plan0.bytes), dtype=torch.uint8).pin_memory()
                  for _ in range(NB)]
        dev_plan = [torch.empty(int(plan0.bytes), dtype=torch.uint8, device="cuda")
                    for _ in range(NB)]
        plans = [gts.PlanDesc() for _ in range(NB)]
        build_ws_bytes = gts.build_workspace_bytes(plan0)
        build_ws = [torch.empty(build_ws_bytes, dtype=torch.uint8, device="cuda")
                    for _ in range(nstreams)]
    else:
        pinned = [torch.empty(nbytes, dtype=torch.uint8).pin_memory() for _ in range(NB)]
    copied = [torch.cuda.Event() for _ in range(NB)]    # upload from pinned[i] done
    consumed = [torch.cuda.Event() for _ in range(NB)]  # kernel reading dev[i] done
    ev = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(4)) for _ in range(steps)]
    evp = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]   # pruning done
    kept = [None] * steps
    ens_struct, keep = gts._ensemble_struct(ens)   # keep: the arrays ens_struct points at
    descs = [gts.ModelDesc() for _ in range(NB)]
    biases = [np.zeros(ens.num_groups, np.float64) for _ in range(NB)]
    rows, M, G = Xd.shape[0], ens.num_features, ens.num_groups
    shape = (rows, G, M + 1, M + 1) if interactions else (rows, G, M + 1)
    outs = [torch.empty(shape, dtype=torch.float64 if dtype == "f64" else torch.float32,
                        device="cuda") for _ in range(nstreams)]
    if device_build:
        prep = L.gts_plan_model
        prep_args = [(ctypes.byref(host_ens), 64, gts.PACK_ALGS["bfd"], gts.DTYPES[dtype],
                      ctypes.byref(descs[i]), ctypes.byref(plans[i]),
                      ctypes.c_void_p(pinned[i].data_ptr()), pinned[i].numel())
                     for i in range(NB)]
        build_args = [[(ctypes.byref(dev_ens), ctypes.byref(descs[i]), ctypes.byref(plans[i]),
                        ctypes.c_void_p(dev_plan[i].data_ptr()),
                        ctypes.c_void_p(dev[i].data_ptr()),
                        ctypes.c_void_p(build_ws[j].data_ptr()), build_ws_bytes,
                        ctypes.c_void_p(build_streams[j].cuda_stream))
                       for j in range(nstreams)] for i in range(NB)]
    else:
        prep = L.gts_prepare_model
        prep_args = [(ctypes.byref(ens_struct), 64, gts.PACK_ALGS["bfd"], gts.DTYPES[dtype],
                      ctypes.byref(descs[i]), ctypes.c_void_p(pinned[i].data_ptr()), nbytes,
                      biases[i].ctypes.data_as(ctypes.c_void_p)) for i in range(NB)]
    run_args = [[(ctypes.byref(descs[i]), ctypes.c_void_p(dev[i].data_ptr()),
                  ctypes.c_void_p(Xd.data_ptr()), rows, Xd.stride(0),
                  ctypes.c_void_p(outs[j].data_ptr()),
                  ctypes.c_void_p(kernel_streams[j].cuda_stream))
                 for j in range(nstreams)] for i in range(NB)]
    # batch pruning: per compute stream a workspace (the pruned blob stays in
    # it until that stream's kernel has read it) and the pruned descriptor
    ws_bytes = ctypes.c_int64(0)
    if prune:
        gts._check(L.gts_prune_workspace_bytes(ctypes.byref(desc0), rows, ctypes.byref(ws_bytes)),
                   "gts_prune_workspace_bytes")
    wss = [torch.empty(max(1, ws_bytes.value), dtype=torch.uint8, device="cuda")
           for _ in range(nstreams if prune else 0)]
    pdescs = [gts.ModelDesc() for _ in range(nstreams)]
    pptrs = [ctypes.c_void_p() for _ in range(nstreams)]
    prune_args = [[(ctypes.byref(descs[i]), ctypes.c_void_p(dev[i].data_ptr()),
                    ctypes.c_void_p(Xd.data_ptr()), rows, Xd.stride(0),
                    ctypes.c_void_p(wss[j].data_ptr()), ws_bytes.value, ctypes.byref(pdescs[j]),
                    ctypes.byref(pptrs[j]), ctypes.c_void_p(build_streams[j].cuda_stream))
                   for j in range(nstreams)] for i in range(NB)] if prune else None
    pruned_args = [(ctypes.byref(pdescs[j]), pptrs[j], ctypes.c_void_p(Xd.data_ptr()), rows,
                    Xd.stride(0), ctypes.c_void_p(outs[j].data_ptr()),
                    ctypes.c_void_p(kernel_streams[j].cuda_stream)) for j in range(nstreams)]
    share = 0 if prep_threads is None else prep_threads

    # persistent preparation threads (their per-thread working memory stays
    # warm between runs), each running the tasks of its queue in order
    tasks = [queue.Queue() for _ in range(preps)]

    def worker(h):
        L.gts_set_host_threads(share)
        while True:
            task = tasks[h].get()
            if task is None:
                return
            task()

    threads = [threading.Thread(target=worker, args=(h,), daemon=True) for h in range(preps)]
    for t in threads:
        t.start()

    def wait_for(event):
        # poll and sleep: a wait inside the runtime keeps a core busy, which
        # the preparations need
        while not event.query():
            time.sleep(2e-5)

    def run_steps(n, timed):
        if n == 0:
            return []
        prepared = [threading.Event() for _ in range(n)]
        launched = [threading.Event() for _ in range(n)]
        ready = collections.deque()   # prepared steps, in the order they finish
        host_ms = [0.0] * n
        errors = []

        def prepare(k):
            try:
                i = k % NB
                if k >= NB:
                    launched[k - NB].wait()   # step k-NB's kernel launch has read descs[i]
                    wait_for(copied[i])       # and its upload has read pinned[i]
                h0 = time.perf_counter()
                st = prep(*prep_args[i])
                host_ms[k] = 1e3 * (time.perf_counter() - h0)
                if st != gts.GTS_OK:
                    raise RuntimeError(f"model preparation: {L.gts_last_error().decode()}")
            except BaseException as e:  # reported by the main thread
                errors.append(e)
            ready.append(k)
            prepared[k].set()

        for k in range(n):
            tasks[k % preps].put(lambda k=k: prepare(k))
        try:
            # the main thread uploads every prepared step (in the order the
            # preparations finish) once its device buffer is free, and
            # launches each uploaded step once its upload has finished; it
            # polls and sleeps instead of blocking in the runtime.  (A step's
            # device buffer is free once the kernel of step k - NB is done:
            # that kernel was launched before step k's preparation began.)
            uploaded = collections.deque()
            done = 0

            while done < n:
                busy = False
                if errors:
                    raise errors[0]
                # any prepared step whose buffers are free, not only the
                # oldest: a step prepared early must not wait behind one
                # whose buffers a late kernel still holds
                for k in [k for k in list(ready) if consumed[k % NB].query()]:
                    ready.remove(k)
                    i = k % NB
                    with torch.cuda.stream(copy):
                        if device_build:
                            dev_plan[i].copy_(pinned[i], non_blocking=True)
                        else:
                            dev[i].copy_(pinned[i], non_blocking=True)
                        copied[i].record(copy)
                    uploaded.append(k)
                    busy = True
                while uploaded and copied[uploaded[0] % NB].query():
                    k = uploaded.popleft()
                    i, j = k % NB, k % nstreams
                    bstream, stream = build_streams[j], kernel_streams[j]
                    if timed:
                        ev[k][0].record(bstream)
                    if device_build:
                        st = L.gts_build_model_device(*build_args[i][j])
                        if st != gts.GTS_OK:
                            raise RuntimeError(f"gts_build_model_device: "
                                               f"{L.gts_last_error().decode()}")
                    if timed:
                        ev[k][1].record(bstream)
                    if prune:
                        if split:
                            # workspace j: free once the kernel two steps back has read it
                            pstream.wait_event(shap_done[j])
                        st = L.gts_prune_model(*prune_args[i][j])
                        if st != gts.GTS_OK:
                            raise RuntimeError(f"gts_prune_model: {L.gts_last_error().decode()}")
                    if split:
                        pruned_ev[j].record(pstream)
                        if timed:
                            evp[k].record(pstream)
                        kstream.wait_event(pruned_ev[j])
                    if timed:
                        ev[k][2].record(stream)
                    st = launch(*(pruned_args[j] if prune else run_args[i][j]))
                    if st != gts.GTS_OK:
                        raise RuntimeError(f"kernel launch: {L.gts_last_error().decode()}")
                    if timed:
                        ev[k][3].record(stream)
                        if keep_outputs:
                            with torch.cuda.stream(stream):
                                kept[k] = outs[j].clone()
                    if split:
                        shap_done[j].record(kstream)
                    consumed[i].record(stream)
                    launched[k].set()
                    done += 1
                    busy = True
                if not busy:
                    time.sleep(2e-5)
        finally:
            for e in launched:   # no preparation waits forever after an error
                e.set()
            for k in range(n):
                prepared[k].wait()
        return host_ms

    # no garbage collection while steps run: a collection holds the
    # interpreter lock for tens of milliseconds, which stalls the threads
    # that return from the library
    gc_was_on = gc.isenabled()
    gc.collect()
    gc.disable()
    try:
        # untimed: back-to-back launches, then pipelined steps for at least
        # 0.5 s (host threads, copies and GPU clocks in the state of the timed
        # steps), before the warm-up steps
        ref_model = gts.prepare(ens, dtype)
        fn = kernel_fn(gts, interactions)
        for _ in range(5):
            fn(ref_model, Xd, out=outs[0])
        torch.cuda.synchronize()
        t_end = time.perf_counter() + 0.5
        while True:
            run_steps(2 * NB, False)
            if time.perf_counter() >= t_end:
                break
        torch.cuda.synchronize()
        run_steps(warmup, False)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        host_ms = run_steps(steps, True)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
    finally:
        if gc_was_on:
            gc.enable()
        for q in tasks:
            q.put(None)
        for t in threads:
            t.join()
    build_ms = np.array([a.elapsed_time(b) for a, b, c, d in ev])
    prune_ms = (np.array([b.elapsed_time(e) for (a, b, c, d), e in zip(ev, evp)]) if split
                else np.array([b.elapsed_time(c) for a, b, c, d in ev]))
    kern = np.array([c.elapsed_time(d) for a, b, c, d in ev])
    result = (wall, kern, prune_ms, build_ms, outs[(steps - 1) % nstreams], ref_model,
              np.array(host_ms))
    return result + (kept,) if keep_outputs else result


def time_kernel(torch, gts, model, Xd, reps, interactions):
    """Kernel-only: each launch bracketed by HIP events on the launch stream."""
    fn = kernel_fn(gts, interactions)
    stream = torch.cuda.current_stream()
    out = fn(model, Xd)
    for _ in range(4):
        out = fn(model, Xd, out=out)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(reps)]
    for a, b in ev:
        a.record(stream)
        fn(model, Xd, out=out)
        b.record(stream)
    torch.cuda.synchronize()
    return np.array([a.elapsed_time(b) for a, b in ev])


def time_prune(torch, gts, model, Xd, reps, interactions):
    """gts_prune_model for the batch (HIP events around each call), then the
    kernel on the pruned model as time_kernel times it: (prune ms per call,
    kernel ms per launch, pruned model)."""
    ws = torch.empty(gts.prune_workspace_bytes(model, Xd.shape[0]), dtype=torch.uint8,
                     device="cuda")
    stream = torch.cuda.current_stream()
    pm = gts.prune(model, Xd, workspace=ws)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(reps)]
    for a, b in ev:
        a.record(stream)
        pm = gts.prune(model, Xd, workspace=ws)
        b.record(stream)
    torch.cuda.synchronize()
    p = np.array([a.elapsed_time(b) for a, b in ev])
    k = time_kernel(torch, gts, pm, Xd, reps, interactions)
    return p, k, pm


def pruned_counts(gts, pm):
    """(bins, paths, elements) of a pruned model, read back from the device."""
    host = pm.blob.cpu().numpy()
    G = pm.num_groups
    o5, o4, o0 = pm.desc.off[5], pm.desc.off[4], pm.desc.off[0]
    gb = np.frombuffer(host[o5:o5 + 4 * (G + 1)].tobytes(), np.int32)
    nb = int(gb[G])
    bs = np.frombuffer(host[o4:o4 + 4 * (nb + 1)].tobytes(), np.int32)
    ne = int(bs[nb])
    feat = np.frombuffer(host[o0:o0 + 4 * ne].tobytes(), np.int32)
    return nb, int(np.count_nonzero(feat < 0)), ne


def warm_host(fn, seconds=0.2):
    """Calls fn back to back for a while: host cores that have idled (the
    suite's other parts, model generation) take a while to wake and clock up,
    and a few timed calls right after would catch that instead of the
    preparation itself."""
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        fn()


def time_prepare(gts, ens, dtype, reps=20):
    """Host preparation (one gts_prepare_model call) into pinned memory, and
    the upload from there into a device buffer, as the step loop does them."""
    import ctypes
    import torch
    desc, blob, _ = gts.prepare_blob(ens, dtype)
    pinned = torch.empty(len(blob), dtype=torch.uint8).pin_memory()
    dev = torch.empty(len(blob), dtype=torch.uint8, device="cuda")
    L = gts.lib()
    s, keep = gts._ensemble_struct(ens)
    bias = np.zeros(ens.num_groups, np.float64)
    args = (ctypes.byref(s), 64, gts.PACK_ALGS["bfd"], gts.DTYPES[dtype], ctypes.byref(desc),
            ctypes.c_void_p(pinned.data_ptr()), pinned.numel(),
            bias.ctypes.data_as(ctypes.c_void_p))
    warm_host(lambda: L.gts_prepare_model(*args))
    host, up = [], []
    for _ in range(reps):
        t0 = time.perf_counter()
        if L.gts_prepare_model(*args) != gts.GTS_OK:
            raise RuntimeError(f"gts_prepare_model: {L.gts_last_error().decode()}")
        t1 = time.perf_counter()
        dev.copy_(pinned, non_blocking=True)
        torch.cuda.synchronize()
        t2 = time.perf_counter()
        host.append(t1 - t0)
        up.append(t2 - t1)
    return 1e3 * float(np.median(host)), 1e3 * float(np.median(up)), int(len(blob))


def time_device_extract(torch, gts, ens, reps=10):
    """gts_extract_paths_device (paths and bias on the GPU from device-resident
    node arrays), wall clock per call including its two count read-backs;
    gts_extract_paths on the host for comparison."""
    dens = gts.DeviceEnsemble(ens)
    gts.extract_paths_device(dens)
    torch.cuda.synchronize()
    warm_host(lambda: gts.extract_paths(ens))
    dev, host = [], []
    for _ in range(reps):
        t0 = time.perf_counter()
        gts.extract_paths_device(dens)
        torch.cuda.synchronize()
        dev.append(time.perf_counter() - t0)
        t0 = time.perf_counter()
        gts.extract_paths(ens)
        host.append(time.perf_counter() - t0)
    return 1e3 * float(np.median(dev)), 1e3 * float(np.median(host))


def time_device_build(torch, gts, ens, dtype, reps=10):
    """A device build as the step loop runs it: gts_plan_model on the host
    into pinned memory (wall clock), the plan's upload, and
    gts_build_model_device on the GPU (HIP events around it on the current
    stream); None when the model admits no plan."""
    import ctypes
    try:
        desc, plan, _ = gts.plan_model(ens, dtype)
    except gts.GtsError:
        return None
    L = gts.lib()
    s, keep = gts._ensemble_struct(ens)
    pinned = torch.empty(int(plan.bytes), dtype=torch.uint8).pin_memory()
    d_plan = torch.empty(int(plan.bytes), dtype=torch.uint8, device="cuda")
    dens = gts.DeviceEnsemble(ens)
    out = torch.empty(int(desc.bytes), dtype=torch.uint8, device="cuda")
    ws = torch.empty(max(1, gts.build_workspace_bytes(plan)), dtype=torch.uint8, device="cuda")
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    warm_host(lambda: L.gts_plan_model(ctypes.byref(s), 64, gts.PACK_ALGS["bfd"],
                                       gts.DTYPES[dtype], ctypes.byref(desc), ctypes.byref(plan),
                                       ctypes.c_void_p(pinned.data_ptr()), pinned.numel()))
    host, up, dev = [], [], []
    for _ in range(reps):
        t0 = time.perf_counter()
        st = L.gts_plan_model(ctypes.byref(s), 64, gts.PACK_ALGS["bfd"], gts.DTYPES[dtype],
                              ctypes.byref(desc), ctypes.byref(plan),
                              ctypes.c_void_p(pinned.data_ptr()), pinned.numel())
        t1 = time.perf_counter()
        if st != gts.GTS_OK:
            raise RuntimeError(f"gts_plan_model: {L.gts_last_error().decode()}")
        d_plan.copy_(pinned, non_blocking=True)
        torch.cuda.synchronize()
        t2 = time.perf_counter()
        e0.record()
        gts.build_model_device(dens, desc, plan, d_plan, dtype, out=out, workspace=ws)
        e1.record()
        torch.cuda.synchronize()
        host.append(t1 - t0)
        up.append(t2 - t1)
        dev.append(e0.elapsed_time(e1))
    return {"plan_ms_host": 1e3 * float(np.median(host)),
            "plan_upload_ms": 1e3 * float(np.median(up)),
            "build_ms_device": float(np.median(dev)), "plan_bytes": int(plan.bytes)}


def cpu_threads() -> int:
    threads = len(os.sched_getaffinity(0))
    env = os.environ.get("OMP_NUM_THREADS")
    if env and env.isdigit():
        threads = min(threads, int(env))
    return threads


def oracle_rate(oracle, ens, X, budget_s: float, interactions: bool, nthreads: int):
    """The oracle on a row prefix grown until one call takes about budget_s,
    or the whole batch repeated until that much time has passed: (rows per
    second, rows in the prefix, passes, seconds)."""
    fn = oracle.interactions if interactions else oracle.treeshap
    n = 4 if interactions else 16
    while True:
        n = min(n, X.shape[0])
        t0 = time.perf_counter()
        fn(ens, X[:n], nthreads=nthreads)
        dt = time.perf_counter() - t0
        if dt >= budget_s or n == X.shape[0]:
            break
        n = min(X.shape[0], max(n + 1, int(n * 1.05 * budget_s / max(dt, 1e-3))))
    passes = 1
    if dt < budget_s:
        passes = max(1, int(np.ceil(budget_s / max(dt, 1e-3))))
        t0 = time.perf_counter()
        for _ in range(passes):
            fn(ens, X[:n], nthreads=nthreads)
        dt = time.perf_counter() - t0
    return n * passes / dt, n, passes, dt


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return ""


def suite_entry(torch, gts, synth, oracle, workload, dtype, interactions, reps, oracle_s):
    w = synth.workload(workload)
    ens = w.ensemble
    rows = w.X.shape[0]
    Xd = torch.from_numpy(w.X).cuda()
    host_ms, upload_ms, blob_bytes = time_prepare(gts, ens, dtype)
    dev_extract_ms, host_extract_ms = time_device_extract(torch, gts, ens)
    model = gts.prepare(ens, dtype)
    k = time_kernel(torch, gts, model, Xd, reps, interactions)
    med = float(np.median(k))
    wm = work_model(torch, gts, ens, w.X, dtype, interactions)
    peak = PEAK_FP64_TFLOPS if dtype == "f64" else PEAK_FP32_TFLOPS
    achieved = wm["flops_live"] / (med * 1e-3) / 1e12
    dense = wm["flops_dense"] / (med * 1e-3) / 1e12
    entry = {
        "workload": WORKLOAD_TEXT[workload], "dtype": dtype, "rows": rows,
        "output": (f"phi[{rows}, {ens.num_groups}, {ens.num_features + 1}"
                   + (f", {ens.num_features + 1}]" if interactions else "]")),
        "paths": wm["paths"], "path_elements": wm["path_elements"],
        "bins": int(model.num_bins),
        "live_pair_fraction": wm["live_pairs"] / max(1, wm["pairs"]),
        "live_tile_fraction": wm["live_tile_pairs"] / max(1, wm["tile_pairs"]),
        "launch": gts.launch_config(model, rows, interactions),
        "host_prepare_ms": host_ms, "upload_ms": upload_ms, "model_bytes": blob_bytes,
        "extract_ms_device": dev_extract_ms, "extract_ms_host": host_extract_ms,
        "device_build": time_device_build(torch, gts, ens, dtype),
        "kernel_ms_median": med, "kernel_ms_mean": float(k.mean()),
        "kernel_ms_std": float(k.std()), "kernel_runs": len(k),
        "kernel_rows_per_s": rows / (med * 1e-3),
        "end_to_end_rows_per_s": rows / ((host_ms + upload_ms + med) * 1e-3),
        "modelled_tflops": achieved, "peak_tflops": peak, "frac": achieved / peak,
        "dense_equivalent_tflops": dense,
        "traffic_bytes": traffic_for((workload, dtype, interactions)),
        "executed": executed((workload, dtype, interactions), med),
    }
    p, kp, pm = time_prune(torch, gts, model, Xd, reps, interactions)
    pmed, kpmed = float(np.median(p)), float(np.median(kp))
    nb, npaths, nel = pruned_counts(gts, pm)
    entry["pruned"] = {
        "prune_ms_median": pmed, "kernel_ms_median": kpmed,
        "kernel_rows_per_s": rows / (kpmed * 1e-3),
        "prune_and_kernel_rows_per_s": rows / ((pmed + kpmed) * 1e-3),
        "paths": npaths, "path_elements": nel, "bins": nb,
        "modelled_tflops": wm["flops_live"] / (kpmed * 1e-3) / 1e12,
        "frac": wm["flops_live"] / (kpmed * 1e-3) / 1e12 / peak,
        "traffic_bytes": traffic_for((workload, dtype, interactions, "pruned")),
        "executed": executed((workload, dtype, interactions, "pruned"), kpmed),
    }
    if oracle is not None and oracle_s > 0:
        threads = cpu_threads()
        rate, n, passes, dt = oracle_rate(oracle, ens, w.X, oracle_s, interactions, threads)
        entry["oracle_rows_per_s"] = rate
        entry["oracle"] = {"cores": threads, "sample": f"first {n} of {rows} rows x {passes} "
                           f"pass(es) in {dt:.2f} s, fp64, OpenMP over rows"}
    return entry


def cpu_baseline(oracle, ens, X, budget_s: float, interactions: bool):
    """The oracle as it stands, on all usable cores, on a bounded sample of
    the batch (about budget_s / 2), then on one thread (about budget_s / 4)."""
    threads = cpu_threads()
    rate, n, passes, dt = oracle_rate(oracle, ens, X, budget_s / 2, interactions, threads)
    rate1, n1, passes1, dt1 = oracle_rate(oracle, ens, X, budget_s / 4, interactions, 1)
    what = "conditioning interactions" if interactions else "Algorithm 1"
    return {"value": rate, "unit": "rows/s", "cores": threads, "kind": "oracle",
            "sample": f"first {n} of {X.shape[0]} rows x {passes} pass(es) in {dt:.2f} s, fp64 "
                      f"{what}, OpenMP over rows",
            "one_thread_value": rate1,
            "one_thread_sample": f"first {n1} rows x {passes1} pass(es) in {dt1:.2f} s",
            "cpu": cpu_model()}


def copy_probe(torch):
    """A plain device copy of 256 MiB (read 256 MiB, write 256 MiB) whose
    FETCH_SIZE / WRITE_SIZE readings calibrate the kernel's."""
    n = 64 << 20
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    torch.neg(src, out=dst)
    torch.cuda.synchronize()
    return n * 4


def profile_launches(torch, gts, synth, workload, dtype, launches, pruned=False):
    """Only the kernel of one workload, `launches` times back to back (for
    rocprofv3 counter and trace runs); with `pruned`, on the model pruned for
    the batch once beforehand."""
    w = synth.workload(workload)
    inter = workload == "interactions"
    model = gts.prepare(w.ensemble, dtype)
    Xd = torch.from_numpy(w.X).cuda()
    if pruned:
        model = gts.prune(model, Xd)
    fn = kernel_fn(gts, inter)
    out = fn(model, Xd)
    for _ in range(launches - 1):
        fn(model, Xd, out=out)
    torch.cuda.synchronize()
    print(json.dumps({"profiled": workload, "dtype": dtype, "launches": launches,
                      "pruned": pruned}), flush=True)


def profile_extract(torch, gts, synth, workload, calls):
    """Only gts_extract_paths_device on one workload's model, `calls` times
    (for rocprofv3 kernel traces); one workspace for all calls."""
    w = synth.workload(workload)
    dens = gts.DeviceEnsemble(w.ensemble)
    ws = None
    for _ in range(calls):
        raw, npaths, _ = gts.extract_paths_device(dens, workspace=ws)
    torch.cuda.synchronize()
    print(json.dumps({"profiled_extract": workload, "calls": calls, "paths": npaths}), flush=True)


# ---------------------------------------------------------------------------
# experiments (each prints one JSON line of its own instead of the bench line)
# ---------------------------------------------------------------------------

PACK_WORKLOADS = [("tiny", "f64", False), ("covtype_med", "f32", False), ("deep", "f32", False),
                  ("wide", "f32", False), ("interactions", "f32", True)]


def experiment_packers(torch, gts, synth, reps):
    """Section 4.1 / Table 5 on the synthetic models: for each heuristic and
    bin capacity, the bin count K, the utilisation sum(L) / (B K), the host
    packing time (gts_pack_paths on the extracted paths, median of 3), and
    the kernel time on the model packed that way."""
    table = []
    for wl, dtype, inter in PACK_WORKLOADS:
        w = synth.workload(wl)
        ens = w.ensemble
        el, _, _ = gts.extract_paths(ens)
        roots = np.flatnonzero(el["feature_idx"] == -1)
        sizes = np.diff(np.append(roots, len(el)))
        Xd = torch.from_numpy(w.X).cuda()
        rows = w.X.shape[0]
        for cap in (32, 64):
            for alg in ("none", "nf", "ffd", "bfd"):
                rec = {"workload": wl, "dtype": dtype, "interactions": inter, "B": cap,
                       "alg": alg, "paths": int(len(sizes)), "elements": int(sizes.sum())}
                if int(sizes.max()) > cap:
                    rec["skipped"] = f"longest path {int(sizes.max())} > B"
                    table.append(rec)
                    continue
                t = []
                for _ in range(3):
                    t0 = time.perf_counter()
                    packed, offs = gts.pack_paths(el, cap, alg)
                    t.append(time.perf_counter() - t0)
                K = len(offs) - 1
                model = gts.prepare(ens, dtype, bin_capacity=cap, alg=alg)
                assert model.num_bins == K
                k = time_kernel(torch, gts, model, Xd, reps, inter)
                rec.update({"bins": K, "utilisation": float(sizes.sum()) / (cap * K),
                            "pack_ms": 1e3 * float(np.median(t)),
                            "kernel_ms": float(np.median(k)),
                            "kernel_rows_per_s": rows / (float(np.median(k)) * 1e-3)})
                table.append(rec)
                print(json.dumps(rec), file=sys.stderr, flush=True)
    return {"experiment": "packers", "table": table}


def experiment_rows(torch, gts, synth, oracle, workloads, cpu_limit_s):
    """The paper's latency sweep (Fig. 4): time to explain n rows for n from
    1 to 2^20 with the model prepared once.  GPU: the kernel alone on
    device-resident rows (HIP events), and host to host (upload of X from
    pinned memory, kernel, download of phi), median of several calls.  CPU: the
    oracle on all cores while one call stays under cpu_limit_s."""
    threads = cpu_threads()
    out = {"experiment": "rows", "cpu_threads": threads, "sweeps": []}
    for wl in workloads:
        w = synth.workload(wl)
        ens = w.ensemble
        dtype = w.dtype
        inter = wl == "interactions"
        fn = kernel_fn(gts, inter)
        host_ms, upload_ms, _ = time_prepare(gts, ens, dtype)
        model = gts.prepare(ens, dtype)
        nmax = 1 << (16 if inter else 20)
        Xall = synth.sweep_rows(wl, nmax)
        Xpin = torch.from_numpy(Xall).pin_memory()
        Xdev = torch.empty_like(Xpin, device="cuda")
        Xdev.copy_(Xpin)
        width = ens.num_groups * (ens.num_features + 1) * ((ens.num_features + 1) if inter else 1)
        phi_host = torch.empty(nmax * width, dtype=model.torch_dtype).pin_memory()
        stream = torch.cuda.current_stream()
        cpu_fn = oracle.interactions if inter else oracle.treeshap
        cpu_open = True
        points = []
        n = 1
        while n <= nmax:
            reps = 20 if n <= 4096 else 5
            # device-resident rows
            k = time_kernel(torch, gts, model, Xdev[:n], reps, inter)
            # host to host
            phi_dev = fn(model, Xdev[:n])
            torch.cuda.synchronize()
            hh = []
            for _ in range(reps):
                t0 = time.perf_counter()
                Xdev[:n].copy_(Xpin[:n], non_blocking=True)
                fn(model, Xdev[:n], out=phi_dev)
                phi_host[:n * width].copy_(phi_dev.reshape(-1), non_blocking=True)
                stream.synchronize()
                hh.append(time.perf_counter() - t0)
            rec = {"rows": n, "gpu_kernel_ms": float(np.median(k)),
                   "gpu_host_to_host_ms": 1e3 * float(np.median(hh))}
            if cpu_open:
                t0 = time.perf_counter()
                cpu_fn(ens, Xall[:n], nthreads=threads)
                dt = time.perf_counter() - t0
                rec["cpu_ms"] = 1e3 * dt
                if dt > cpu_limit_s:
                    cpu_open = False
            points.append(rec)
            print(json.dumps(dict(rec, workload=wl)), file=sys.stderr, flush=True)
            n *= 4
        cross = [p["rows"] for p in points
                 if "cpu_ms" in p and p["gpu_host_to_host_ms"] < p["cpu_ms"]]
        out["sweeps"].append({"workload": wl, "dtype": dtype, "interactions": inter,
                              "host_prepare_ms": host_ms, "upload_ms": upload_ms,
                              "gpu_faster_from_rows": min(cross) if cross else None,
                              "points": points})
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="deep",
                    choices=["tiny", "covtype_med", "deep", "wide", "interactions"],
                    help="the batch one step explains (interactions: the interaction kernel "
                         "on the covtype-shaped model)")
    ap.add_argument("--dtype", default=None, choices=["f32", "f64"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-suite", action="store_true",
                    help="skip the per-workload suite (kernel and preparation of every workload)")
    ap.add_argument("--suite-reps", type=int, default=10)
    ap.add_argument("--suite-oracle-s", type=float, default=2.0,
                    help="seconds of oracle time per suite workload (0: none)")
    ap.add_argument("--cpu-budget", type=float, default=16.0,
                    help="seconds of oracle time for the CPU baseline (about half on all "
                         "cores, a quarter on one thread)")
    ap.add_argument("--experiment", default=None, choices=["packers", "rows"],
                    help="instead of the bench line, print one JSON line of an experiment: "
                         "the packing heuristics (Table 5 with kernel times) or the rows "
                         "sweep (Fig. 4)")
    ap.add_argument("--sweep-workloads", default="covtype_med,deep,interactions")
    ap.add_argument("--cpu-limit", type=float, default=4.0)
    ap.add_argument("--streams", type=int, default=2,
                    help="compute streams the pipelined steps alternate between (default "
                         "two: a step's build and pruning overlap the previous step's "
                         "SHAP kernel)")
    ap.add_argument("--split-streams", action="store_true",
                    help="builds and prunings on one stream, every SHAP kernel on another "
                         "(instead of whole steps alternating between compute streams)")
    ap.add_argument("--prep-threads", type=int, default=0,
                    help="host threads each preparation in flight may use (0: every core)")
    ap.add_argument("--preps", type=int, default=0,
                    help="model preparations in flight at once in the pipelined steps "
                         "(0: three for models of 128 k nodes or more, else one)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="run a plain 256 MiB device copy first (counter calibration)")
    ap.add_argument("--profile-launches", type=int, default=0,
                    help="only launch the kernel of --workload this many times (rocprofv3)")
    ap.add_argument("--profile-extract", type=int, default=0,
                    help="only run gts_extract_paths_device on --workload's model this many "
                         "times (rocprofv3)")
    ap.add_argument("--profile-pruned", action="store_true",
                    help="with --profile-launches: on the model pruned for the batch")
    ap.add_argument("--build", default="auto", choices=["auto", "host", "device"],
                    help="host: each step prepares the whole blob on the host "
                         "(gts_prepare_model); device: the host plans it (gts_plan_model) "
                         "and the GPU writes it (gts_build_model_device); auto: device "
                         "where a plan can be made (one path per wave, paths of at most 64 "
                         "splits), else host")
    ap.add_argument("--no-prune", action="store_true",
                    help="the steps run the kernel on the whole model, without pruning it "
                         "for the batch first")
    args = ap.parse_args()
    if (args.steps < 1 or args.warmup < 0 or args.streams < 1 or args.preps < 0 or
            args.prep_threads < 0):
        ap.error("--steps and --streams must be at least 1, --warmup, --preps and "
                 "--prep-threads at least 0")

    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; the row-sharded "
                                   "multi-GPU design is documented but not built",
                          "n_gpus": args.gpus}), flush=True)
        sys.exit(2)

    import torch
    from paper_2010_13972_amd import gts, synth

    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a HIP device")
    gts.lib()  # fails loudly if libgts.so is missing

    if args.copy_probe:
        copy_probe(torch)
    if args.profile_extract:
        profile_extract(torch, gts, synth, args.workload, args.profile_extract)
        return
    if args.profile_launches:
        profile_launches(torch, gts, synth, args.workload,
                         args.dtype or synth.workload(args.workload).dtype, args.profile_launches,
                         args.profile_pruned)
        return

    if args.experiment == "packers":
        print(json.dumps(experiment_packers(torch, gts, synth, args.suite_reps)), flush=True)
        return
    if args.experiment == "rows":
        import oracle
        print(json.dumps(experiment_rows(torch, gts, synth, oracle,
                                         args.sweep_workloads.split(","), args.cpu_limit)),
              flush=True)
        return

    w = synth.workload(args.workload)
    inter = args.workload == "interactions"
    dtype = args.dtype or w.dtype
    ens = w.ensemble
    rows = w.X.shape[0]
    Xd = torch.from_numpy(w.X).cuda()

    prune = not args.no_prune
    device_build = args.build == "device"
    if args.build == "auto":
        try:
            gts.plan_model(ens, dtype)
            device_build = True
        except gts.GtsError:
            device_build = False
    # a large model's host work does not use 16 cores fully: three steps' in
    # flight at once finish more of them per second (the worker pool gives
    # every free core to the one that started first); a small one's does
    preps = args.preps or (3 if ens.num_nodes >= (1 << 17) else 1)
    wall, kern, prune_ms, build_ms, out, model, step_host = time_pipeline(
        torch, gts, ens, Xd, dtype, args.steps, args.warmup, inter, args.streams, preps, prune,
        device_build, args.prep_threads, split=args.split_streams)
    # the steps' last output against the Python binding's call on the same
    # model (up to the order of the tile additions)
    ref = kernel_fn(gts, inter)(model, Xd)
    torch.cuda.synchronize()
    rel = float((out - ref).abs().max() / (ref.abs().max() + 1e-30))
    if not rel < 1e-4:
        raise SystemExit(f"pipelined steps disagree with gts.shap: relative difference {rel:.3g}")
    # roofline: the kernel's launches inside the timed steps (events on its
    # stream); back-to-back launches in a timed region of their own as well
    kern_ms = float(kern.mean())
    nrep = max(5, min(args.steps, 50))
    if prune:
        _, k_only, kmodel = time_prune(torch, gts, model, Xd, nrep, inter)
        pbins, ppaths, pelems = pruned_counts(gts, kmodel)
    else:
        k_only = time_kernel(torch, gts, model, Xd, nrep, inter)
    wm = work_model(torch, gts, ens, w.X, dtype, inter)
    peak = PEAK_FP64_TFLOPS if dtype == "f64" else PEAK_FP32_TFLOPS
    achieved = wm["flops_live"] / (kern_ms * 1e-3) / 1e12
    key = (args.workload, dtype, inter) + (("pruned",) if prune else ())
    line = {
        "metric": METRIC,
        "value": rows * args.steps / wall, "unit": "rows/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": 1e3 * wall / args.steps,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": dtype,
        "data": "synthetic (seeded ensembles and rows shaped like the paper's models)",
        "config": {"workload": WORKLOAD_TEXT[args.workload], "rows": rows,
                   "trees": int(ens.num_trees), "paths": wm["paths"],
                   "path_elements": wm["path_elements"], "bins": int(model.num_bins),
                   "output": (f"phi[{rows}, {ens.num_groups}, {ens.num_features + 1}"
                              + (f", {ens.num_features + 1}]" if inter else "]")),
                   "step": ("validating walk with path counts + BFD pack (B=64) + each "
                            "path's place (host) + upload of the plan + "
                            "extract + merge + bias + layout (device) "
                            if device_build else
                            "extract + merge + bias + BFD pack (B=64) + layout (host) + upload ")
                           + ("+ batch pruning (device) " if prune else "")
                           + ("+ interaction kernel" if inter else "+ SHAP kernel")
                           + f"; {preps} steps' host work in flight at once on a shared "
                           + "worker pool that serves the oldest first; uploads and host "
                           + "work overlap the kernels of earlier steps",
                   "compute_streams": args.streams, "preparations_in_flight": preps,
                   "blob_built_on": "device" if device_build else "host",
                   "pruned_for_the_batch": ({"paths": ppaths, "path_elements": pelems,
                                             "bins": pbins} if prune else None)},
        "roofline": {"bound": "alu", "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                     "frac": achieved / peak,
                     "traffic": traffic_for(key),
                     "kernel": "shap_kernel" + (" (interactions)" if inter else "")
                               + (" on the model pruned for the batch" if prune else ""),
                     "kernel_ms": kern_ms,
                     "prune_ms_in_steps": float(prune_ms.mean()) if prune else None,
                     "device_build_ms_in_steps": float(build_ms.mean()) if device_build else None,
                     "kernel_launches": int(len(kern)),
                     "kernel_ms_back_to_back": float(k_only.mean()),
                     "modelled_gflop_per_launch": wm["flops_live"] / 1e9,
                     "live_pair_fraction": wm["live_pairs"] / max(1, wm["pairs"]),
                     "live_tile_fraction": wm["live_tile_pairs"] / max(1, wm["tile_pairs"]),
                     "dense_equivalent_tflops": wm["flops_dense"] / (kern_ms * 1e-3) / 1e12,
                     "executed": executed(key, kern_ms),
                     "host_prepare_ms_in_steps": float(np.median(step_host)),
                     "host_prepare_ms_in_steps_mean": float(step_host.mean()),
                     "host_prepare_ms_in_steps_p90": float(np.percentile(step_host, 90)),
                     "note": "achieved: op model over the live (row, path) pairs (a pair "
                             "whose zero-cover element misses the row contributes exactly "
                             "0; pruning drops only paths without live pairs) / mean "
                             "in-step launch time of the kernel (with two compute "
                             "streams it shares the GPU with the next step's build and "
                             "pruning, so its span is longer than alone: "
                             "kernel_ms_back_to_back); peak is the packed-FP32 "
                             "vendor figure (non-packed FP32 FMAs measured about 129 "
                             "TFLOP/s); dense_equivalent_tflops counts every pair"},
        "launch": gts.launch_config(model, rows, inter),
        "kernel": {"rows_per_s": rows / (float(np.median(k_only)) * 1e-3),
                   "ms_median": float(np.median(k_only)), "ms_mean": float(k_only.mean()),
                   "ms_std": float(k_only.std()), "runs": len(k_only)},
    }
    orc = None
    if not args.no_cpu_baseline or args.suite_oracle_s > 0:
        import oracle
        orc = oracle
    if not args.no_suite:
        line["configs"] = {name: suite_entry(torch, gts, synth, orc, wl, dt, it,
                                             args.suite_reps, args.suite_oracle_s)
                           for name, wl, dt, it in SUITE}
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(orc, ens, w.X, args.cpu_budget, inter)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
