"""The decoding-rounds reference (asynchronous hint at the candidate boundary,
Eq. 3; verify and commit, Section 4.5) against sequential greedy decoding,
brute-force slicing of a planted hint and the readiness cases; planted
mistakes in copies of it must each fail one of those pins (CPU only)."""

import os
import sys
import types

import pytest

import decode_checks as dc
from oracle import decode_loop as dl


@pytest.mark.parametrize("check", dc.ALL_CHECKS, ids=lambda c: c.__name__)
def test_decode_reference_pin(check):
    check(dl)


SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle", "decode_loop.py")

# (name, original text, mutated text)
MUTATIONS = [
    ("checks_outside_retrieval_rounds", "if views is not None and retrieval(r, committed) and done(r):",
     "if views is not None and done(r):"),
    ("ignores_readiness", "if views is not None and retrieval(r, committed) and done(r):",
     "if views is not None and retrieval(r, committed):"),
    ("native_lanes_first", "lanes = tv.merge_lanes(hints, nat, n_lanes) if ready else nat[:n_lanes]",
     "lanes = tv.merge_lanes(nat, hints, n_lanes) if ready else nat[:n_lanes]"),
    ("suffix_of_first_root", "found = tv.hint_continuations(bank, eos, committed, max_suffix, max_depth)",
     "found = tv.hint_continuations(bank, eos, committed[:1], max_suffix, max_depth)"),
    ("stale_root", "step = tm.verify_step(committed[-1], lanes,", "step = tm.verify_step(committed[0], lanes,"),
    ("prefix_without_bonus", "        P += int(step[\"L\"]) + 1", "        P += int(step[\"L\"])"),
    ("bank_without_eos", "        bank += [int(t) for t in v] + [int(eos)]", "        bank += [int(t) for t in v]"),
]


def _mutant(name, old, new):
    with open(SRC) as f:
        text = f.read()
    assert text.count(old) == 1, f"mutation {name}: anchor text not found exactly once"
    mod = types.ModuleType(f"mutant_decode_{name}")
    sys.modules[mod.__name__] = mod
    exec(compile(text.replace(old, new), f"<{mod.__name__}>", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_planted_mistake_fails_a_pin(name, old, new):
    mod = _mutant(name, old, new)
    failed = []
    for check in dc.ALL_CHECKS:
        try:
            check(mod)
        except AssertionError:
            failed.append(check.__name__)
    assert failed, f"mutation {name} passed every pin"
