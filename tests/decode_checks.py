"""Checks that pin the decoding-rounds reference (``oracle/decode_loop.py``)
to things other than itself.

Each ``check_*`` takes the reference module and raises AssertionError on a
mismatch, so the same checks run against the committed reference (they must
pass) and against copies with a planted mistake (some check must fail).
What each check leans on:

* sequential greedy decoding with a dense causal forward written with
  library routines (``model_checks.dense_forward``): whatever the candidates
  and the hint hold, the rounds commit exactly the greedy tokens (Section 3,
  target authority), and a correct hint makes them commit more per round;
* brute-force slicing of a planted hint view: a hint that becomes ready late
  proposes the part of the view after the committed position (Section 4.4,
  suffix matching), not what is already committed;
* the readiness cases of Eq. 3, read off the records: pending rounds use the
  native candidates unchanged, a hint that completes after the last round
  changes nothing, and rounds that are not retrieval rounds do not check.
"""

from __future__ import annotations

import numpy as np

import model_checks as mc
from oracle import target_model as tm

N_LANES, MAX_NODES, MAX_DEPTH, MAX_SUFFIX = 6, 16, 6, 7


def _setup(seed, n_prefix=5, cap=160):
    model = mc.tiny_model(seed, om=tm)
    rs = np.random.default_rng(seed + 100)
    V = model["V"]
    prefix = [int(t) for t in rs.integers(0, V, size=n_prefix)]
    root = int(rs.integers(0, V))
    return model, prefix, root, cap


def _native(seed, V):
    """Two short random lanes per round (a stand-in for the schema chain and a
    retrieved call; they are rarely right)."""
    def fn(r, committed):
        g = np.random.default_rng([seed, r, 7])
        return [[int(t) for t in g.integers(0, V, size=3)], [int(t) for t in g.integers(0, V, size=2)]]
    return fn


def _run(dl, model, prefix, root, cap, n_rounds, native, views=None, done=lambda r: True,
         retrieval=lambda r, y: True, eos=None):
    kcs, vcs = mc._prefix_caches(model, prefix, cap)
    return dl.run_rounds(n_rounds, len(prefix), root, native, views, done, retrieval,
                         model["V"] - 1 if eos is None else eos, N_LANES, MAX_SUFFIX, MAX_NODES, MAX_DEPTH,
                         model["emb"], model["layers"], model["final"], model["lm"], model["shp"], kcs, vcs)


def _greedy(model, prefix, root, n):
    toks, margin = mc._dense_greedy(model, prefix + [root], n)
    assert margin > 1e-6, "near tie in the dense greedy run"
    return toks


def check_rounds_commit_greedy_tokens(dl):
    """With native candidates only, with a wrong hint and with a correct one,
    the committed tokens are the dense forward's greedy tokens; the correct
    hint commits them in fewer rounds."""
    seed = 31
    model, prefix, root, cap = _setup(seed)
    V = model["V"]
    native = _native(seed, V)
    greedy = _greedy(model, prefix, root, 40)
    plain = _run(dl, model, prefix, root, cap, 6, native)
    got = plain["committed"][1:]
    assert got == greedy[:len(got)] and len(got) >= 6
    rs = np.random.default_rng(seed)
    wrong = [[int(t) for t in rs.integers(0, V - 1, size=30)] for _ in range(3)]
    noisy = _run(dl, model, prefix, root, cap, 6, native, views=wrong)
    got = noisy["committed"][1:]
    assert got == greedy[:len(got)]
    right = [wrong[0], [root] + greedy[:30]]
    hinted = _run(dl, model, prefix, root, cap, 4, native, views=right)
    got = hinted["committed"][1:]
    assert got == greedy[:len(got)]
    assert len(got) >= 4 * (MAX_DEPTH + 1) - 2, "a correct hint should be accepted to the depth cap"
    # the prefix advances by what each round commits
    for rec in hinted["records"]:
        assert rec["L"] == len(rec["committed"]) - 1
    P = len(prefix)
    for rec in hinted["records"]:
        assert rec["prefix_len"] == P
        P += len(rec["committed"])
    assert hinted["prefix_len"] == P


def check_late_hint_proposes_uncommitted_part(dl):
    """A correct hint ready from round 3 on: at round 3 one hint lane is the
    view's continuation after the committed position (brute-force slicing),
    the round accepts it, and earlier rounds saw no hint."""
    seed = 32
    model, prefix, root, cap = _setup(seed)
    V = model["V"]
    eos = V - 1
    native = _native(seed, V)
    greedy = _greedy(model, prefix, root, 40)
    view = [root] + greedy[:36]
    out = _run(dl, model, prefix, root, cap, 5, native, views=[view], done=lambda r: r >= 3, eos=eos)
    recs = out["records"]
    for rec in recs[:3]:
        assert not rec["hint_ready"] and rec["n_hint"] == 0
        assert rec["lanes"] == native(rec["round"], None)[:N_LANES]
    k = sum(len(rec["committed"]) for rec in recs[:3])  # greedy tokens committed before round 3
    want = []
    for t in view[k + 1:]:
        if t == eos or len(want) == MAX_DEPTH:
            break
        want.append(t)
    assert want, "the planted view ends before round 3"
    rec = recs[3]
    assert rec["hint_ready"] and rec["n_hint"] >= 1
    assert want in rec["lanes"][:rec["n_hint"]]
    assert rec["committed"][:len(want)] == want
    assert rec["suffix_len"] == min(MAX_SUFFIX, k + 1)


def check_readiness_cases(dl):
    """A hint that completes after the last round changes nothing; a round
    that is not a retrieval round does not check; pending rounds keep the
    native candidates unchanged."""
    seed = 33
    model, prefix, root, cap = _setup(seed)
    V = model["V"]
    native = _native(seed, V)
    greedy = _greedy(model, prefix, root, 40)
    view = [root] + greedy[:30]
    base = _run(dl, model, prefix, root, cap, 4, native)
    late = _run(dl, model, prefix, root, cap, 4, native, views=[view], done=lambda r: False)
    for a, b in zip(base["records"], late["records"]):
        assert a["lanes"] == b["lanes"] and a["committed"] == b["committed"] and not b["hint_ready"]
    odd = _run(dl, model, prefix, root, cap, 4, native, views=[view], retrieval=lambda r, y: r % 2 == 1)
    for rec in odd["records"]:
        if rec["round"] % 2 == 0:
            assert not rec["hint_ready"] and rec["lanes"] == native(rec["round"], None)[:N_LANES]
        else:
            assert rec["hint_ready"] and rec["n_hint"] >= 1
    got = odd["committed"][1:]
    assert got == greedy[:len(got)]


def check_proposals_stop_at_view_end(dl):
    """Views are separated by EOS in the bank: a correct view shorter than
    the depth cap is proposed exactly (brute force: the view itself), not run
    on into the next view, and committing it still gives the greedy tokens."""
    seed = 34
    model, prefix, root, cap = _setup(seed)
    V = model["V"]
    eos = V - 1
    native = _native(seed, V)
    greedy = _greedy(model, prefix, root, 20)
    assert eos not in greedy[:4]
    decoy = [t for t in range(V - 1) if t != root][:12]
    out = _run(dl, model, prefix, root, cap, 2, native, views=[[root] + greedy[:4], decoy], eos=eos)
    rec = out["records"][0]
    hints = rec["lanes"][:rec["n_hint"]]
    assert greedy[:4] in hints
    assert all(h[:4] != greedy[:4] or len(h) == 4 for h in hints)
    got = out["committed"][1:]
    assert got == greedy[:len(got)] and rec["L"] >= 4


ALL_CHECKS = [
    check_rounds_commit_greedy_tokens,
    check_late_hint_proposes_uncommitted_part,
    check_readiness_cases,
    check_proposals_stop_at_view_end,
]
