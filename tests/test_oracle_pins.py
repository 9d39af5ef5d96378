"""The CPU oracle against facts outside itself (hand-worked fixtures, closed
forms, Shapley axioms, invariants of the path form, bin-packing bounds)."""
import pytest

import oracle_checks as oc


@pytest.mark.parametrize("check", oc.ALL_CHECKS, ids=lambda c: c.__name__)
def test_oracle_pin(orc, check):
    check(orc)
