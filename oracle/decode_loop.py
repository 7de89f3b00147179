"""Plain CPU reference for decoding rounds with an asynchronous hint.

TEST INFRASTRUCTURE ONLY.  Like ``tree_verify`` and ``target_model``, this
module is the slow, obviously-correct definition the native library is
checked against; only the test suite, the smoke check and the benchmark's
CPU-baseline leg may import it, the product path never does, and it shares
no code with the native library.

What a round computes, in the paper's order:

* Section 4.4, candidate boundary (Eq. 3): at a retrieval-candidate round the
  runtime checks, without blocking, whether the sidecar has finished.  If it
  has not, the round's candidates C_r are the native ones C^TS_r.  If it has,
  C_r = Merge_B(hint continuations, C^TS_r): the bank's continuations of the
  current committed suffix (n = 7 down to 1) take the first lanes, the
  native candidates the rest, and the budget B is kept.  A completion that
  falls just after one check is first seen at the next retrieval round.
* Section 4.4, tokenizer and hint bank: the rendered views are joined into
  one bank, each followed by the EOS token, once, when the hint is first
  seen; later rounds reuse it.
* Section 4.5, verify and commit: the target scores the trie of C_r in one
  forward pass (``target_model.verify_step``), commits the accepted path and
  its own next token, and only those states enter the cache.
* Recovery: a hint that completes after the last round is never used.

The sidecar's completion time is an input here: ``done(r)`` says whether the
future has completed when round r checks (monotone in r).

Parity pins: none from the paper (it prints no decoding trace).  The test
suite pins the loop by sequential greedy decoding with a dense causal
forward (committed tokens must equal it whatever the hint holds), by
brute-force slicing of a planted hint (the continuation proposed at a late
round is the part of the hint after the committed position), and by the
readiness cases (pending, ready at round s, ready after the last round, no
check outside retrieval rounds).
"""

from __future__ import annotations

from typing import Callable, Dict, List, Optional, Sequence

import numpy as np

from oracle import target_model as tm
from oracle import tree_verify as tv


def build_bank(views: Sequence[Sequence[int]], eos: int) -> List[int]:
    """The request-level bank: every view followed by the EOS token."""
    bank: List[int] = []
    for v in views:
        bank += [int(t) for t in v] + [int(eos)]
    return bank


def run_rounds(n_rounds: int, prefix_len: int, root_token: int,
               native: Callable[[int, Sequence[int]], Sequence[Sequence[int]]],
               views: Optional[Sequence[Sequence[int]]], done: Callable[[int], bool],
               retrieval: Callable[[int, Sequence[int]], bool], eos: int, n_lanes: int, max_suffix: int,
               max_nodes: int, max_depth: int, emb, layers: Sequence[tm.LayerWeights], final_norm, lm_head,
               shp: tm.ModelShape, k_caches: Sequence[np.ndarray], v_caches: Sequence[np.ndarray]) -> Dict:
    """``n_rounds`` rounds from committed length ``prefix_len`` (the caches'
    rows [0, P) hold the prefix; modified in place).  Returns the per-round
    records and the committed tokens (the first root first)."""
    committed = [int(root_token)]
    P = int(prefix_len)
    bank: Optional[List[int]] = None
    records = []
    for r in range(n_rounds):
        nat = [[int(t) for t in c] for c in native(r, committed)]
        ready = False
        hints: List[List[int]] = []
        slen = 0
        if views is not None and retrieval(r, committed) and done(r):
            if bank is None:
                bank = build_bank(views, eos)
            ready = True
            found = tv.hint_continuations(bank, eos, committed, max_suffix, max_depth)
            hints, slen = found["continuations"], found["n"]
        lanes = tv.merge_lanes(hints, nat, n_lanes) if ready else nat[:n_lanes]
        n_hint = min(len(hints), n_lanes) if ready else 0
        step = tm.verify_step(committed[-1], lanes, max_nodes, max_depth, P, emb, layers, final_norm, lm_head,
                              shp, k_caches, v_caches)
        toks = [int(t) for t in step["committed"]]
        records.append({"round": r, "prefix_len": P, "lanes": lanes, "hint_ready": ready, "n_hint": n_hint,
                        "suffix_len": slen if ready else 0, "n_nodes": int(step["tree"]["n_nodes"]),
                        "L": int(step["L"]), "bonus": int(step["bonus"]), "path": np.asarray(step["path"]),
                        "committed": toks, "margin": np.asarray(step["margin"])})
        committed += toks
        P += int(step["L"]) + 1
    return {"records": records, "committed": committed, "prefix_len": P}
