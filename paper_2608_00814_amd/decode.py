"""Multi-step decoding around the verification step.

Section 3 (the ToolSpec decoding loop): every round builds candidates,
verifies them with the target and commits the longest agreeing prefix.
Section 4.4 (candidate boundary, Eq. 3): at a retrieval-candidate round the
runtime checks, without blocking, whether the sidecar's hint is ready.  While
it is pending the round uses the native candidates alone; once ready, the
hint bank's suffix-aligned continuations fill the first lanes and the native
candidates the rest (``ooo_hint_merge``).  A hint that completes just after
one check is first seen at the next retrieval round; nothing is rolled back,
and a hint that completes after the last round is never used.
Section 4.5 (verify and commit): the target scores the trie in one forward
pass, commits the accepted path plus its own next token, and the next round's
root is that token.

Device side: one HIP graph per trie size, captured the first time that size
occurs and replayed afterwards.  The trie arrays and the prefix length travel
in one host-to-device copy from pinned staging at the start of the graph, the
kernels read the prefix length from device memory (so the same graph serves
every round while the prefix grows), and (L, bonus, path) come back in one
device-to-host copy at its end.  The host waits for that copy only: it needs
the committed tokens to build the next round's candidates.
"""

from __future__ import annotations

import time
from dataclasses import dataclass, field
from typing import Callable, Dict, List, Optional, Sequence

import numpy as np
import torch

from . import ooo
from .model import ModelRunner


class SidecarHint:
    """The sidecar's result as the target sees it (Section 4.4, tokenizer and
    hint bank).

    ``future`` is any object with ``done()`` and ``result()`` (for example a
    ``concurrent.futures.Future``) whose result is the rendered views of the
    hint, each already tokenized by the target's tokenizer.  ``poll()`` never
    blocks: it returns None while the future is pending; the first poll that
    finds it done joins the views into one bank, each view followed by the
    EOS token, and every later poll returns that same array (encoded once).
    A sidecar that failed (``result()`` raised, or views that are not token
    sequences) is treated as never ready: the target does not depend on it.
    """

    def __init__(self, future, eos_token: int):
        self.future = future
        self.eos = int(eos_token)
        self.bank: Optional[np.ndarray] = None
        self.first_ready_round: Optional[int] = None
        self.failed: Optional[BaseException] = None

    def poll(self, round_index: int) -> Optional[np.ndarray]:
        if self.bank is None and self.failed is None and self.future is not None and self.future.done():
            try:
                parts: List[int] = []
                for v in self.future.result():
                    parts.extend(int(t) for t in v)
                    parts.append(self.eos)
                bank = np.asarray(parts, dtype=np.int32)
                if (bank < 0).any():
                    raise ValueError("negative token in the hint")
            except Exception as e:  # a failed sidecar never delays or stops the target
                self.failed = e
                return None
            self.bank = bank
            self.first_ready_round = round_index
        return self.bank


@dataclass
class RoundRecord:
    round: int
    prefix_len: int            # P before the round (the root's row)
    n_nodes: int
    n_truncated: int
    hint_ready: bool           # the readiness check of this round found the bank
    n_hint: int                # lanes the bank filled
    suffix_len: int            # suffix length whose occurrences proposed them
    L: int                     # accepted draft tokens
    bonus: int                 # the target's own next token
    committed: List[int] = field(default_factory=list)  # the L + 1 tokens of this round
    host_us: float = 0.0       # candidates, readiness check, merge and packing
    device_us: float = 0.0     # graph launch to the result in host memory


class DecodeLoop:
    """Greedy batch-one decoding of ``model`` with tree verification.

    k_cache, v_cache   [n_layers][Hkv][cap][D] bf16; rows [0, prefix_len)
                       hold the committed prefix
    root_token         the first round's root (the target's next token after
                       the prefix; its K/V are computed in that round)
    native(r, y)       the round's native candidates (priority order) given the
                       round index and the committed tokens y (oldest first,
                       ending with the current root)
    hint               a SidecarHint, or None
    retrieval_round(r, y)  whether round r is a retrieval-candidate round
                       (readiness is checked only there); default: every round
    n_lanes, max_suffix    Merge_B's lane count and the longest suffix tried
    graphs             replay captured graphs (False: launch every call)
    """

    def __init__(self, model: ModelRunner, k_cache: torch.Tensor, v_cache: torch.Tensor, prefix_len: int,
                 root_token: int, native: Callable[[int, Sequence[int]], Sequence[Sequence[int]]],
                 hint: Optional[SidecarHint] = None,
                 retrieval_round: Optional[Callable[[int, Sequence[int]], bool]] = None,
                 n_lanes: int = 8, max_suffix: int = 7, graphs: bool = True, stream=None):
        cfg = model.cfg
        if k_cache.shape != (cfg.n_layers, cfg.n_kv_heads, cfg.cap, cfg.head_dim) or v_cache.shape != k_cache.shape:
            raise ValueError("k_cache / v_cache must be [n_layers][n_kv_heads][cap][head_dim]")
        self.model, self.k, self.v = model, k_cache, v_cache
        self.native, self.hint = native, hint
        self.retrieval_round = retrieval_round or (lambda r, y: True)
        self.n_lanes, self.max_suffix = int(n_lanes), int(max_suffix)
        self.P = int(prefix_len)
        self.committed: List[int] = [int(root_token)]
        self.rounds = 0
        self.use_graphs = graphs
        self.stream = stream if stream is not None else torch.cuda.Stream(device=model.device)
        # the prefix bound every launch is planned and validated for
        self.bound = cfg.cap - cfg.max_nodes
        # A captured graph keeps the workspace addresses it was captured with,
        # so the attention workspace is sized for every trie size now and is
        # never reallocated afterwards.
        vr = model.vr
        for n in range(1, cfg.max_nodes + 1):
            vr.ensure_workspace(self.bound, n)
        self._ws_ptr = vr.attn_ws.data_ptr()
        self._graphs: Dict[int, torch.cuda.CUDAGraph] = {}
        self._done = torch.cuda.Event()

    # ---------------------------------------------------------------------
    def can_continue(self) -> bool:
        return self.P <= self.bound

    def _candidates(self, r: int):
        y = self.committed
        native = [list(map(int, c)) for c in self.native(r, y)]
        bank = self.hint.poll(r) if self.hint is not None and self.retrieval_round(r, y) else None
        if bank is None:
            lanes = native[:self.n_lanes]
            flat = np.array([t for c in lanes for t in c], np.int32)
            offs = np.zeros(len(lanes) + 1, np.int32)
            offs[1:] = np.cumsum([len(c) for c in lanes])
            return flat, offs, False, 0, 0
        nt = np.array([t for c in native for t in c], np.int32)
        no = np.zeros(len(native) + 1, np.int32)
        no[1:] = np.cumsum([len(c) for c in native])
        m = ooo.hint_merge(bank, self.hint.eos, np.asarray(y, np.int32), nt, no, self.n_lanes,
                           max_suffix=self.max_suffix, max_len=self.model.cfg.max_depth)
        return m["tokens"], m["offsets"], True, m["n_hint"], m["suffix_len"]

    def _launch(self, N: int) -> None:
        vr = self.model.vr
        if not self.use_graphs:
            with torch.cuda.stream(self.stream):
                self.model.device_step(self.k, self.v, self.bound, prefix_dev=vr.prefix_dev)
            return
        if vr.attn_ws.data_ptr() != self._ws_ptr:
            raise RuntimeError("attention workspace was reallocated after graphs were captured")
        g = self._graphs.get(N)
        if g is None:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=self.stream):
                self.model.device_step(self.k, self.v, self.bound, prefix_dev=vr.prefix_dev)
            self._graphs[N] = g
        g.replay()

    def round(self) -> RoundRecord:
        """One candidate boundary and one verify step; returns its record."""
        if not self.can_continue():
            raise RuntimeError(f"cache full: prefix {self.P} + {self.model.cfg.max_nodes} nodes exceed the capacity")
        r = self.rounds
        vr = self.model.vr
        t0 = time.perf_counter()
        flat, offs, ready, n_hint, slen = self._candidates(r)
        root = self.committed[-1]
        vr.pack(root, flat, offs, keep=False)
        vr.set_prefix(self.P)
        N = vr.n_nodes
        t1 = time.perf_counter()
        with torch.cuda.stream(self.stream):
            self._launch(N)
            self._done.record(self.stream)
        self._done.synchronize()
        t2 = time.perf_counter()
        res = vr.result()
        toks = [int(vr._h_token[i]) for i in res.path[1:]] + [res.bonus]
        rec = RoundRecord(r, self.P, N, vr.n_truncated, ready, n_hint, slen, res.L, res.bonus, toks,
                          (t1 - t0) * 1e6, (t2 - t1) * 1e6)
        self.committed.extend(toks)
        self.P += res.L + 1
        self.rounds += 1
        return rec

    def run(self, max_rounds: int, max_new_tokens: Optional[int] = None) -> List[RoundRecord]:
        """Rounds until ``max_rounds``, ``max_new_tokens`` committed tokens or
        a full cache, whichever comes first."""
        out: List[RoundRecord] = []
        made = 0
        while len(out) < max_rounds and self.can_continue():
            if max_new_tokens is not None and made >= max_new_tokens:
                break
            rec = self.round()
            made += len(rec.committed)
            out.append(rec)
        return out
