"""ooo_hint_merge (Section 4.4, Suffix matching; Eq. 3) on the CPU: the C ABI
against the CPU reference's hint continuations and lane filling, on the
hand-derived fixtures, on random banks, on a long bank, and into the trie."""

import json
import os

import numpy as np
import pytest

from oracle import tree_verify as ov
from paper_2608_00814_amd import ooo

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "hint_cases.json")


def _csr(cands):
    offs = np.zeros(len(cands) + 1, np.int32)
    for i, c in enumerate(cands):
        offs[i + 1] = offs[i] + len(c)
    return np.array([t for c in cands for t in c], dtype=np.int32), offs


def _lanes(r):
    return [r["tokens"][r["offsets"][i]:r["offsets"][i + 1]].tolist() for i in range(r["n_out"])]


def _reference(bank, eos, committed, native, n_lanes, max_suffix, max_len):
    h = ov.hint_continuations(bank, eos, committed, max_suffix, max_len)
    return h, ov.merge_lanes(h["continuations"], native, n_lanes)


def test_hint_merge_golden():
    g = json.load(open(GOLDEN))
    for c in g["hint_cases"]:
        r = ooo.hint_merge(np.array(c["bank"]), 0, np.array(c["committed"]), np.zeros(0), np.zeros(1), 8,
                           c["max_suffix"], c["max_len"])
        assert r["suffix_len"] == c["n"], c["name"]
        assert _lanes(r) == c["continuations"], c["name"]
        assert r["n_hint"] == len(c["continuations"])
    for c in g["lane_cases"]:
        # the hints come from a bank built to propose exactly them
        bank, committed = [], [77]
        for h in c["hints"]:
            bank += [77] + h + [0]
        toks, offs = _csr(c["native"])
        r = ooo.hint_merge(np.array(bank), 0, np.array(committed), toks, offs, c["n_lanes"], 7, 16)
        assert _lanes(r) == c["lanes"]


@pytest.mark.parametrize("seed", range(4))
def test_hint_merge_matches_reference_on_random_banks(seed):
    rs = np.random.default_rng(100 + seed)
    for trial in range(250):
        vocab = int(rs.integers(2, 7))
        eos = 0
        bank = [int(t) for t in rs.integers(0, vocab + 1, size=int(rs.integers(0, 120)))]
        committed = [int(t) for t in rs.integers(1, vocab + 1, size=int(rs.integers(0, 12)))]
        native = [[int(t) for t in rs.integers(1, 50, size=int(rs.integers(0, 6)))]
                  for _ in range(int(rs.integers(0, 5)))]
        n_lanes = int(rs.integers(0, 6))
        max_suffix = int(rs.integers(1, 9))
        max_len = int(rs.integers(1, 8))
        toks, offs = _csr(native)
        r = ooo.hint_merge(np.array(bank, dtype=np.int32), eos, np.array(committed, dtype=np.int32), toks, offs,
                           n_lanes, max_suffix, max_len)
        h, lanes = _reference(bank, eos, committed, native, n_lanes, max_suffix, max_len)
        assert _lanes(r) == lanes, (seed, trial)
        assert r["suffix_len"] == h["n"], (seed, trial)
        assert r["n_hint"] == min(len(h["continuations"]), n_lanes), (seed, trial)


def test_hint_merge_long_bank_and_trie():
    """A 200k-token bank with planted views; the merged lanes give the same
    trie through ooo_pack_tree as the reference's lanes through its packer."""
    rs = np.random.default_rng(5)
    eos = 2
    bank = rs.integers(3, 30000, size=200_000).astype(np.int32)
    suffix = [11, 12, 13, 14, 15, 16, 17]
    for at, cont in ((1_000, [101, 102, 103]), (90_000, [201, 202]), (150_000, [101, 102, 103])):
        bank[at:at + 7] = suffix
        bank[at + 7:at + 7 + len(cont)] = cont
        bank[at + 7 + len(cont)] = eos
    committed = np.array([5, 6] + suffix, dtype=np.int32)
    native = [[7, 8, 9], [7, 10], [11]]
    toks, offs = _csr(native)
    r = ooo.hint_merge(bank, eos, committed, toks, offs, 4, 7, 40)
    h, lanes = _reference(bank.tolist(), eos, committed.tolist(), native, 4, 7, 40)
    assert r["suffix_len"] == 7 and h["n"] == 7
    assert _lanes(r) == lanes == [[101, 102, 103], [201, 202], [7, 8, 9], [7, 10]]
    root = int(committed[-1])
    got = ooo.pack_tree(root, r["tokens"], r["offsets"], 16, 8)
    ref = ov.pack_tree(root, lanes, 16, 8)
    assert np.array_equal(got["token"], ref["token"]) and np.array_equal(got["parent"], ref["parent"])


def test_hint_merge_rejects_bad_arguments():
    e = np.zeros(0, np.int32)
    one = np.zeros(1, np.int32)
    with pytest.raises(ooo.OooError):  # max_suffix < 1
        ooo.hint_merge(np.array([1, 2, 3]), 0, np.array([1]), e, one, 2, max_suffix=0)
    with pytest.raises(ooo.OooError):  # max_len < 1
        ooo.hint_merge(np.array([1, 2, 3]), 0, np.array([1]), e, one, 2, max_len=0)
    with pytest.raises(ooo.OooError):  # non-monotone native offsets
        ooo.hint_merge(np.array([1, 2]), 0, np.array([1]), np.array([4, 5]), np.array([0, 2, 1]), 2)
    with pytest.raises(ooo.OooError):  # negative native token
        ooo.hint_merge(np.array([1, 2]), 0, np.array([1]), np.array([-4]), np.array([0, 1]), 2)
    st = ooo.lib().ooo_hint_merge(None, 5, 0, None, 0, 7, 4, None, one.ctypes.data_as(ooo._c_i32p), 0, 1,
                                  None, 0, one.ctypes.data_as(ooo._c_i32p), None, None, None)
    assert st == ooo.ERR_INVALID  # bank_len > 0 with a null bank


def test_hint_merge_capacity():
    import ctypes
    bank = np.array([1, 5, 6, 7, 0], dtype=np.int32)
    committed = np.array([1], dtype=np.int32)
    one = np.zeros(1, np.int32)
    out = np.zeros(2, np.int32)
    offs = np.zeros(3, np.int32)
    n_out, n_hint, slen = ctypes.c_int32(9), ctypes.c_int32(9), ctypes.c_int32(9)
    P = ooo._c_i32p
    st = ooo.lib().ooo_hint_merge(bank.ctypes.data_as(P), 5, 0, committed.ctypes.data_as(P), 1, 7, 8, None,
                                  one.ctypes.data_as(P), 0, 2, out.ctypes.data_as(P), 2, offs.ctypes.data_as(P),
                                  ctypes.byref(n_out), ctypes.byref(n_hint), ctypes.byref(slen))
    assert st == ooo.ERR_CAPACITY and n_out.value == 0  # three tokens do not fit in two


@pytest.mark.parametrize("name", ["qwen3-8b", "qwen3-0.6b"])
def test_hint_bank_reproduces_the_candidate_lanes(name):
    """The synthetic bank proposes the step's first candidate (the hint lane)
    for the committed suffix; with the other candidates as native lanes, the
    merged lanes are the step's candidate list, and the reference agrees."""
    from paper_2608_00814_amd import workload as wl
    cfg = wl.CONFIGS[name]
    for seed in range(3):
        cand = wl.candidates_for(cfg, seed, 0)
        hb = wl.hint_bank_for(cfg, seed, cand)
        toks, offs = _csr(cand.seqs[1:])
        n_lanes = len(cand.seqs)
        r = ooo.hint_merge(hb.bank, hb.eos, hb.committed, toks, offs, n_lanes, 7, cfg.max_depth)
        h, lanes = _reference(hb.bank.tolist(), hb.eos, hb.committed.tolist(), cand.seqs[1:], n_lanes, 7,
                              cfg.max_depth)
        hint = cand.seqs[0][:cfg.max_depth]
        assert r["suffix_len"] == 7 and r["n_hint"] >= 1
        assert _lanes(r)[0] == hint and lanes[0] == hint
        assert _lanes(r) == lanes


# ----------------------------------------------------------------------------
# the sidecar's future at the candidate boundary (Eq. 3): never blocks, bank
# built once, a failed sidecar is never ready


class _Fut:
    def __init__(self, views=None, ready_after=0, exc=None):
        self.views, self.ready_after, self.exc = views, ready_after, exc
        self.done_calls = self.result_calls = 0

    def done(self):
        self.done_calls += 1
        return self.done_calls > self.ready_after

    def result(self):
        self.result_calls += 1
        if self.exc is not None:
            raise self.exc
        return self.views


def test_sidecar_hint_pending_then_ready_once():
    from paper_2608_00814_amd.decode import SidecarHint
    f = _Fut(views=[[5, 6, 7], [], [8]], ready_after=2)
    h = SidecarHint(f, eos_token=99)
    assert h.poll(0) is None and h.poll(1) is None
    b = h.poll(2)
    assert b.tolist() == [5, 6, 7, 99, 99, 8, 99] and h.first_ready_round == 2
    assert h.poll(3) is b and h.poll(4) is b and f.result_calls == 1


def test_sidecar_hint_failure_is_never_ready():
    from paper_2608_00814_amd.decode import SidecarHint
    h = SidecarHint(_Fut(exc=RuntimeError("sidecar crashed")), eos_token=99)
    assert all(h.poll(r) is None for r in range(4)) and isinstance(h.failed, RuntimeError)
    h2 = SidecarHint(_Fut(views=[[1, -3]]), eos_token=99)
    assert h2.poll(0) is None and h2.failed is not None and h2.poll(1) is None
    assert SidecarHint(None, eos_token=99).poll(0) is None
