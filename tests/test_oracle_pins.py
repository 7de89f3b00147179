"""The CPU reference against hand-derived fixtures, brute force, library
routines, closed forms and sequential greedy decoding (CPU only)."""

import pytest

import oracle_checks as oc
from oracle import tree_verify as ov


@pytest.mark.parametrize("check", oc.ALL_CHECKS, ids=lambda c: c.__name__)
def test_reference_pin(check):
    check(ov)
