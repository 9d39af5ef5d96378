"""The compiler's resource report of the SHAP and interaction kernels
(written by the build into _build/kernel_resources.txt): the variants built
for paths of at most 8, 12 or 16 features hold no runtime-length path code and
no per-lane path arrays; only the long-path variants do."""
import os
import re

import pytest

REPORT = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                      "paper_2010_13972_amd", "_build", "kernel_resources.txt")
# shap_kernel<T, RW, INTER, WAVES, PRIV, QMAX> in the mangled name
KERNEL = re.compile(r"shap_kernelI([fd])Li(\d+)ELb(\d)ELi(\d+)ELb(\d)ELi(\d+)E")


def variants():
    if not os.path.exists(REPORT):
        pytest.skip("library not built (the report comes from the build)")
    out = []
    with open(REPORT) as f:
        for line in f:
            d = dict(kv.split("=", 1) for kv in line.rstrip("\n").split("\t"))
            m = KERNEL.search(d["name"])
            if m:
                t, rw, inter, waves, priv, qmax = m.groups()
                out.append(dict(dtype=t, rw=int(rw), inter=inter == "1", waves=int(waves),
                                priv=priv == "1", qmax=int(qmax),
                                scratch=int(d["ScratchSize [bytes/lane]"]),
                                vgprs=int(d["VGPRs"])))
    return out


def test_every_variant_is_built():
    v = variants()
    # 12 launch shapes x (4 SHAP + 2 interaction variants) x 2 dtypes
    assert len(v) == 12 * 6 * 2
    assert {x["qmax"] for x in v if not x["inter"]} == {8, 12, 16, 64}
    assert {x["qmax"] for x in v if x["inter"]} == {8, 64}


# registers per lane a wave may hold when a workgroup of `waves` waves must
# fit on a CU (4 SIMDs, 512 registers per SIMD lane, granule 8)
VGPR_CAP = {4: 256, 8: 256, 12: 168, 16: 128}


def test_short_path_variants_hold_no_path_arrays():
    for x in variants():
        if x["qmax"] == 64:
            # the runtime-length code keeps 64-entry arrays per lane
            assert x["scratch"] >= 64 * 8, x
        elif x["scratch"]:
            # only register spills of a variant at its launch bound's cap
            assert x["vgprs"] == VGPR_CAP[x["waves"]] and x["scratch"] < 1024, x
            # fp32 SHAP spills only in the 16-feature variant (fp64 arithmetic)
            assert x["inter"] or x["dtype"] == "d" or x["qmax"] == 16, x


def test_fp32_shap_short_variants_use_no_scratch():
    for x in variants():
        if x["dtype"] == "f" and not x["inter"] and x["qmax"] <= 12:
            assert x["scratch"] == 0, x


def test_fp32_extended_variants_spill_little():
    """The 16-feature fp32 SHAP variant computes in fp64: it spills only at
    16 waves per workgroup (128 registers), and only a few words per lane."""
    for x in variants():
        if x["dtype"] == "f" and not x["inter"] and x["qmax"] == 16:
            assert x["scratch"] == 0 or (x["waves"] == 16 and x["scratch"] <= 64), x


def test_headline_variants_fit_their_occupancy():
    """The fp32 SHAP kernels for paths of at most 8 features with 64-row
    tiles: the shared-tile variant (covtype-shaped workload) stays within 64
    registers (8 waves per SIMD); the private-tile variant (deep and tiny
    workloads), whose rank tables hold a workgroup to 24 KB of LDS and so a
    CU to 6 workgroups of 4 waves, within 80 (6 waves per SIMD)."""
    seen = 0
    for x in variants():
        if x["dtype"] == "f" and not x["inter"] and x["qmax"] == 8 and x["rw"] == 64:
            cap = 80 if x["priv"] else 64
            assert x["vgprs"] <= cap and x["scratch"] == 0, x
            seen += 1
    assert seen == 2


def test_prune_kernels_use_no_private_memory():
    """The batch-pruning kernels (key sort, search, plan, copy) keep their
    arrays in registers and LDS: no scratch."""
    if not os.path.exists(REPORT):
        pytest.skip("library not built (the report comes from the build)")
    names = ("sort_keys", "mark_paths", "plan_pruned", "copy_paths")
    seen = set()
    with open(REPORT) as f:
        for line in f:
            d = dict(kv.split("=", 1) for kv in line.rstrip("\n").split("\t"))
            for n in names:
                if n in d["name"]:
                    seen.add(n)
                    assert d["ScratchSize [bytes/lane]"] == "0", d
    assert seen == set(names)


def test_device_build_kernels_use_no_private_memory():
    """The kernels that write a model blob from a host plan keep every path's
    merged feature ranges and fractions in registers: no scratch."""
    if not os.path.exists(REPORT):
        pytest.skip("library not built (the report comes from the build)")
    names = ("k_build_paths", "k_plan_tree_sums", "k_plan_bias", "k_plan_bins", "k_zero_gaps")
    seen = set()
    with open(REPORT) as f:
        for line in f:
            d = dict(kv.split("=", 1) for kv in line.rstrip("\n").split("\t"))
            for n in names:
                if n in d["name"]:
                    seen.add(n)
                    assert d["ScratchSize [bytes/lane]"] == "0", d
    assert seen == set(names)
