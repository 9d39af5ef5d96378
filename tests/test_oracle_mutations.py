"""Planted mistakes in the CPU oracle must be caught by the pins.

Each case copies ``oracle/oracle.c``, makes one plausible error (a wrong
tie rule, an off-by-one weight, a dropped factor, a swapped bound, first fit
instead of best fit, ...), builds it into a temporary library and runs every
check of ``oracle_checks``: at least one must fail.  Everything runs on the
CPU.
"""
import os

import pytest

import oracle
import oracle_checks as oc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "oracle.c")

# (name, text to replace, replacement, expected number of occurrences)
MUTATIONS = [
    ("tie_goes_left_on_equal", "x[d] < e->thr[b + n]", "x[d] <= e->thr[b + n]", 2),
    ("alg1_tie_rule", "c->x[d] < e->thr[b + j]", "c->x[d] <= e->thr[b + j]", 1),
    ("extend_left_weight_off_by_one", "m[a].w * (double)(a + 1) / (double)(l + 1)",
     "m[a].w * (double)(a) / (double)(l + 1)", 1),
    ("extend_self_weight", "pz * m[a].w * (double)(l - a) / (double)(l + 1)",
     "pz * m[a].w * (double)(l - a + 1) / (double)(l + 1)", 1),
    ("unwind_wrong_factor", "n = t - mj->w * z * (double)(l - j) / (double)l;",
     "n = t - mj->w * (double)(l - j) / (double)l;", 1),
    ("unwind_zero_branch", "mj->w = (mj->w * (double)l) / (z * (double)(l - j));",
     "mj->w = (mj->w * (double)l) / (z * (double)(l - j + 1));", 1),
    ("leaf_sign", "F * w * (m[i].o - m[i].z) * v", "F * w * (m[i].z - m[i].o) * v", 1),
    ("no_zero_cover_guard", "if (!(zh == 0.0 && io == 0.0)) recurse",
     "if (1) recurse", 1),
    ("findfirst_ignored", "if (m[a2].d == d) { k = a2; break; }", "if (0) { k = a2; break; }", 1),
    ("cold_child_one_fraction", "recurse(c, cold, level + 1, l, zc, 0.0, d, F);",
     "recurse(c, cold, level + 1, l, zc, io, d, F);", 1),
    ("zero_cover_ratio_one", "return parent > 0.0 ? child / parent : 0.0;",
     "return parent > 0.0 ? child / parent : 1.0;", 1),
    ("interaction_not_halved", "out[i * W + j] = (on[i] - offv[i]) / 2.0;",
     "out[i * W + j] = (on[i] - offv[i]);", 1),
    ("interaction_off_not_cover_weighted",
     "double Fh = F * ratio(e->cover[b + h], rj);", "double Fh = F;", 1),
    ("interaction_diag_sign", "if (j != i) s -= out[i * W + j];",
     "if (j != i) s += out[i * W + j];", 1),
    ("brute_interaction_diag_sign", "if (j != i) s -= out[i * n + j];",
     "if (j != i) s += out[i * n + j];", 1),
    ("shapley_weight", "double w = factorial(k) * factorial(n - k - 1) / nf;",
     "double w = factorial(k) * factorial(n - k) / nf;", 1),
    ("interaction_weight", "double w = factorial(k) * factorial(n - k - 2) / denom;",
     "double w = factorial(k) * factorial(n - k - 1) / denom;", 1),
    ("brute_bias_dropped", "out[M] = v[0];", "out[M] = 0.0;", 1),
    ("merge_lower_uses_min", "if (s[i].lo > m[nm - 1].lo)", "if (s[i].lo < m[nm - 1].lo)", 1),
    ("merge_drops_zero_fraction", "m[nm - 1].z = m[nm - 1].z * s[i].z;",
     "m[nm - 1].z = m[nm - 1].z;", 1),
    ("right_turn_sets_upper", "splits[ns].lo = th;\n  splits[ns].hi = INFINITY;",
     "splits[ns].lo = -INFINITY;\n  splits[ns].hi = th;", 1),
    ("path_game_absent_uses_one", "p *= ((S >> k) & 1u) ? o[k] : zero_fraction[k];",
     "p *= ((S >> k) & 1u) ? o[k] : 1.0;", 1),
    ("bfd_is_first_fit", "if (best < 0 || resid[b] < resid[best]) best = b;",
     "if (best < 0) best = b;", 1),
    ("bfd_ties_by_descending_index", "return (x->idx > y->idx) - (x->idx < y->idx);",
     "return (x->idx < y->idx) - (x->idx > y->idx);", 1),
    ("bfd_mixes_groups", "group_first_bin = nbins;\n", "\n", 2),
    ("ffd_takes_last_fit", "if (resid[b] >= s) { first = b; break; }",
     "if (resid[b] >= s) { first = b; }", 1),
    ("ffd_lane_after_placement", "lane_of[it[k].idx] = capacity - resid[first];\n    resid[first] -= s;",
     "resid[first] -= s;\n    lane_of[it[k].idx] = capacity - resid[first];", 1),
    ("nf_closes_exactly_fitting_bin", "if (resid < size[p]) {", "if (resid <= size[p]) {", 1),
    ("nf_keeps_bin_across_groups", "int32_t resid = -1; /* no open bin in this group yet */",
     "static int32_t resid = -1;", 1),
    ("none_bins_in_path_order_only", "      if (group[p] != g) continue;\n      bin_of[p] = nbins++;",
     "      if (group[p] != g) continue;\n      bin_of[p] = p;\n      nbins++;", 1),
]


@pytest.fixture(scope="module")
def source():
    with open(SRC) as f:
        return f.read()


@pytest.mark.parametrize("name,old,new,count", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_planted_mistake_is_caught(tmp_path, source, name, old, new, count):
    assert source.count(old) == count, f"mutation {name} no longer matches oracle.c"
    mutated = source.replace(old, new)
    src = tmp_path / "oracle_mut.c"
    src.write_text(mutated)
    lib = oracle.build_to(str(src), str(tmp_path / "liboracle_mut.so"))
    orc = oracle.Oracle(lib)
    failed = []
    for check in oc.ALL_CHECKS:
        try:
            check(orc)
        except AssertionError:
            failed.append(check.__name__)
        except (ValueError, FloatingPointError, ZeroDivisionError, OverflowError):
            failed.append(check.__name__)
    assert failed, f"no pin catches the planted mistake {name}"
