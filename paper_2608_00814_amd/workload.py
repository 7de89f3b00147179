"""Seeded synthetic inputs for the tree-verification step.

This module only *draws* inputs: candidate token sequences, K/V rows, node
queries, LM-head weights and the hidden rows that feed the LM head.  It holds
none of the verification arithmetic (no attention, no logits, no argmax, no
trie packing, no acceptance walk); both the native library's tests and the
plain CPU reference consume what it produces.

Shapes follow the target models the paper evaluates (Section 5.1): Qwen3,
Qwen2.5 and Llama families at batch one.  The trie recipes mimic the three
candidate sources the method merges before one target verification pass
(Section 4.4: schema-FSM chain, retrieved earlier calls and the sidecar's
re-tokenised hint, hint lanes first).  The paper's datasets (API-Bank,
ToolAlpaca, BFCL) are not used; seeded draws of the same shapes stand in.

Every tensor comes from ``numpy.random.Generator(PCG64(SeedSequence(key)))``
with ``key = [cfg_id, seed, step, stream, *extra]``, drawn in float32 and, for
bf16 workloads, rounded to bfloat16 by round-to-nearest-even.  bf16 data is
held as ``uint16`` bit patterns (the device layout); ``bf16_to_f64`` widens
them exactly.

Acceptance is planted by construction: each node ``i`` gets a designated
token ``tau[i]`` and its hidden row is ``z + beta * W[tau]/|W[tau]|`` with
``z ~ N(0, 1)``.  The boost makes ``tau[i]`` the LM head's greedy token by a
wide margin without this module computing any logit; tests confirm the margin
and the planted depth against the CPU reference.  Along the plant branch,
``tau`` of the node at depth ``k < d`` is the branch's token at depth
``k + 1``, so exactly ``d`` draft tokens are accepted.
"""

from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

# stream ids inside the seed key
S_TRIE = 0
S_QUERY = 1
S_KPRE = 2
S_VPRE = 3
S_KTREE = 4
S_VTREE = 5
S_LMW = 6
S_HIDDEN = 7
S_TAU = 8
S_PLANT = 9
S_BANK = 10

# boost applied to the designated token's weight direction in a hidden row
HIDDEN_BOOST = 12.0


@dataclasses.dataclass(frozen=True)
class VerifyConfig:
    """One verification workload.  Sizes are per step; ``cap`` is the number
    of cache rows per (layer, KV head)."""

    name: str
    cfg_id: int
    dtype: str  # "f32" or "bf16"
    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    prefix_len: int
    cap: int
    hidden: int
    vocab: int
    max_nodes: int
    max_depth: int
    steps: int = 1
    description: str = ""

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def mask_words(self) -> int:
        return (self.max_nodes + 63) // 64

    @property
    def elt_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2


CONFIGS: Dict[str, VerifyConfig] = {
    c.name: c
    for c in [
        VerifyConfig(
            "tiny-fp32", 0, "f32", n_layers=1, n_q_heads=4, n_kv_heads=1, head_dim=64,
            prefix_len=128, cap=153, hidden=256, vocab=1024, max_nodes=25, max_depth=8,
            description="single-layer fp32 step, 3 candidates of 8 tokens under one root",
        ),
        VerifyConfig(
            "qwen3-0.6b", 1, "bf16", n_layers=28, n_q_heads=16, n_kv_heads=8, head_dim=128,
            prefix_len=1024, cap=1056, hidden=1024, vocab=151936, max_nodes=32, max_depth=12,
            description="Qwen3-0.6B shape, 32-node trie, depth cap 12, 1k prefix",
        ),
        VerifyConfig(
            "qwen3-8b", 2, "bf16", n_layers=36, n_q_heads=32, n_kv_heads=8, head_dim=128,
            prefix_len=4096, cap=4160, hidden=4096, vocab=151936, max_nodes=64, max_depth=40,
            description="Qwen3-8B shape, 64-node trie (hint + FSM chain + 2 retrieved calls), 4k prefix",
        ),
        VerifyConfig(
            "qwen2.5-32b", 3, "bf16", n_layers=64, n_q_heads=40, n_kv_heads=8, head_dim=128,
            prefix_len=8192, cap=8320, hidden=5120, vocab=152064, max_nodes=128, max_depth=48,
            description="Qwen2.5-32B shape, 128-node trie with branching 6 at argument values, 8k prefix",
        ),
        VerifyConfig(
            "llama3.1-8b-decode", 4, "bf16", n_layers=32, n_q_heads=32, n_kv_heads=8, head_dim=128,
            prefix_len=32768, cap=46080, hidden=4096, vocab=128256, max_nodes=256, max_depth=64,
            steps=200,
            description="Llama-3.1-8B shape, 200 verify steps with compaction from a 32k prefix, "
            "256-node trie, hint branch from step 30",
        ),
    ]
}


# ----------------------------------------------------------------------------
# number formats


def _bf16_round(x: np.ndarray) -> np.ndarray:
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> 16) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def _chunked(n: int, fn) -> None:
    """Run fn(a, b) over [0, n) in chunks on a thread pool."""
    step = 1 << 22
    spans = [(a, min(n, a + step)) for a in range(0, n, step)]
    if len(spans) <= 1:
        for a, b in spans:
            fn(a, b)
        return
    with ThreadPoolExecutor(_THREADS) as ex:
        list(ex.map(lambda ab: fn(*ab), spans))


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), round to nearest even."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, dtype=np.uint16)
    xf, of = x.reshape(-1), out.reshape(-1)

    def fn(a, b):
        of[a:b] = _bf16_round(xf[a:b])

    _chunked(xf.size, fn)
    return out


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    out = np.empty(bits.shape, dtype=np.float32)
    bf, of = bits.reshape(-1), out.reshape(-1)

    def fn(a, b):
        of[a:b] = (bf[a:b].astype(np.uint32) << np.uint32(16)).view(np.float32)

    _chunked(bf.size, fn)
    return out


def to_f32(arr: np.ndarray, dtype: str) -> np.ndarray:
    """Stored values as float32 (exact for bf16 and float32 storage)."""
    return bf16_to_f32(arr) if dtype == "bf16" else np.asarray(arr, dtype=np.float32)


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    out = np.empty(bits.shape, dtype=np.float64)
    bf, of = bits.reshape(-1), out.reshape(-1)

    def fn(a, b):
        of[a:b] = (bf[a:b].astype(np.uint32) << np.uint32(16)).view(np.float32)

    _chunked(bf.size, fn)
    return out


def to_f64(arr: np.ndarray, dtype: str) -> np.ndarray:
    """Widen stored values (uint16 bf16 bits or float32) to float64 exactly."""
    if dtype == "bf16":
        return bf16_to_f64(arr)
    return np.asarray(arr, dtype=np.float64)


def store(x: np.ndarray, dtype: str) -> np.ndarray:
    """float32 draw -> stored representation of ``dtype``."""
    return to_bf16_bits(x) if dtype == "bf16" else np.ascontiguousarray(x, dtype=np.float32)


# ----------------------------------------------------------------------------
# random streams


def rng(cfg: VerifyConfig, seed: int, step: int, stream: int, *extra: int) -> np.random.Generator:
    key = [cfg.cfg_id, seed, step, stream, *extra]
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(key)))


_THREADS = max(1, min(16, len(os.sched_getaffinity(0))))


def normal(cfg: VerifyConfig, seed: int, step: int, stream: int, shape: Tuple[int, ...],
           std: float = 1.0, extra: Sequence[int] = (), stored: Optional[str] = None) -> np.ndarray:
    """N(0, std^2) draw in float32, generated in independent chunks along
    axis 0 on several threads (values do not depend on the thread count).
    With ``stored="bf16"`` each chunk is rounded to bf16 bits as it is drawn,
    so the float32 array is never materialised."""
    shape = tuple(int(s) for s in shape)
    out = np.empty(shape, dtype=np.uint16 if stored == "bf16" else np.float32)
    if out.size == 0:
        return out
    lead = shape[0]
    per_row = out.size // lead
    rows_per_chunk = max(1, (1 << 22) // max(per_row, 1))
    chunks = [(i, min(lead, i + rows_per_chunk)) for i in range(0, lead, rows_per_chunk)]

    def fill(ci: int) -> None:
        a, b = chunks[ci]
        g = rng(cfg, seed, step, stream, *extra, ci)
        x = g.standard_normal((b - a,) + shape[1:], dtype=np.float32)
        if std != 1.0:
            x *= np.float32(std)
        out[a:b] = _bf16_round(x) if stored == "bf16" else x

    if len(chunks) == 1:
        fill(0)
    else:
        with ThreadPoolExecutor(_THREADS) as ex:
            list(ex.map(fill, range(len(chunks))))
    return out


def draw(cfg: VerifyConfig, seed: int, step: int, stream: int, shape, std: float = 1.0,
         extra: Sequence[int] = ()) -> np.ndarray:
    """N(0, std^2) in the workload's stored representation."""
    return normal(cfg, seed, step, stream, shape, std, extra, stored=cfg.dtype if cfg.dtype == "bf16" else None)


# ----------------------------------------------------------------------------
# candidate tries


@dataclasses.dataclass
class Candidates:
    """Priority-ordered draft continuations after the root token (CSR)."""

    root_token: int
    seqs: List[List[int]]
    plant_index: int  # which candidate carries the planted acceptance
    plant_depth: int  # number of its leading tokens the target will accept
    max_nodes: int
    max_depth: int

    def csr(self) -> Tuple[np.ndarray, np.ndarray]:
        offs = np.zeros(len(self.seqs) + 1, dtype=np.int32)
        for i, s in enumerate(self.seqs):
            offs[i + 1] = offs[i] + len(s)
        toks = np.array([t for s in self.seqs for t in s], dtype=np.int32)
        return toks, offs


def _fresh(g: np.random.Generator, vocab: int, avoid: Sequence[int] = ()) -> int:
    avoid = set(int(a) for a in avoid)
    while True:
        t = int(g.integers(0, vocab))
        if t not in avoid:
            return t


def _fresh_seq(g: np.random.Generator, vocab: int, n: int, first_avoid: Sequence[int] = ()) -> List[int]:
    if n <= 0:
        return []
    return [_fresh(g, vocab, first_avoid)] + [int(t) for t in g.integers(0, vocab, size=n - 1)]


@dataclasses.dataclass
class HintBank:
    """A request-level hint bank (Section 4.4, Tokenizer and hint bank):
    tokenized views joined by ``eos``, plus the committed tokens (oldest
    first, ending with the root) whose suffix the bank continues."""

    bank: np.ndarray
    eos: int
    committed: np.ndarray
    hint_lanes: int  # leading candidates that the bank holds


def hint_bank_for(cfg: VerifyConfig, seed: int, cand: Candidates, step: int = 0, n_views: int = 8,
                  view_len: int = 512, history: int = 16) -> HintBank:
    """Random views of ``view_len`` tokens separated by EOS (token vocab-1);
    one view holds the last seven committed tokens followed by the step's
    first candidate (the hint lane) and then EOS, so the bank proposes that
    candidate for this position.  The other candidates are the native lanes.
    Only the first candidate is planted: recipes whose first candidate is not
    a hint still get a bank, and the finder then proposes it as well."""
    g = rng(cfg, seed, step, S_BANK)
    eos = cfg.vocab - 1
    committed = [int(t) for t in g.integers(0, eos, size=history - 1)] + [int(cand.root_token)]
    views = [[int(t) for t in g.integers(0, eos, size=view_len)] for _ in range(n_views)]
    hint = list(cand.seqs[0]) if cand.seqs else []
    at = int(g.integers(0, n_views))
    plant = committed[-7:] + hint
    pos = int(g.integers(0, max(1, view_len - len(plant))))
    views[at] = views[at][:pos] + plant + [eos]
    bank = []
    for v in views:
        bank += v + [eos]
    return HintBank(np.array(bank, dtype=np.int32), eos, np.array(committed, dtype=np.int32), 1 if hint else 0)


def candidates_for(cfg: VerifyConfig, seed: int, step: int = 0, root_token: Optional[int] = None) -> Candidates:
    """Build the priority-ordered candidate set for one step of ``cfg``."""
    g = rng(cfg, seed, step, S_TRIE)
    V = cfg.vocab
    root = int(g.integers(0, V)) if root_token is None else int(root_token)
    gp = rng(cfg, seed, step, S_PLANT)

    if cfg.name == "tiny-fp32":
        seqs = [[int(t) for t in g.integers(0, V, size=8)] for _ in range(3)]
        return Candidates(root, seqs, 0, 5, cfg.max_nodes, cfg.max_depth)

    if cfg.name == "qwen3-0.6b":
        chain = _fresh_seq(g, V, 20)  # schema chain, cut to 12 by the depth cap
        a = chain[:3] + _fresh_seq(g, V, 9, first_avoid=[chain[3]])
        b = chain[:2] + _fresh_seq(g, V, 10, first_avoid=[chain[2]])
        d = int(gp.integers(0, 13))
        return Candidates(root, [chain, a, b], 0, d, cfg.max_nodes, cfg.max_depth)

    if cfg.name == "qwen3-8b":
        hint = _fresh_seq(g, V, 40)  # sidecar hint, first priority
        fsm = hint[:4] + _fresh_seq(g, V, 8, first_avoid=[hint[4]])
        ra = fsm[:6] + _fresh_seq(g, V, 8, first_avoid=[fsm[6]])
        rb = fsm[:5] + _fresh_seq(g, V, 7, first_avoid=[fsm[5]])
        d = int(gp.integers(4, 41))
        return Candidates(root, [hint, fsm, ra, rb], 0, d, cfg.max_nodes, cfg.max_depth)

    if cfg.name == "qwen2.5-32b":
        spine = _fresh_seq(g, V, 48)
        seqs = [spine]
        for bi, b in enumerate((10, 20, 30, 40)):
            used = [spine[b]]
            for ai in range(5):
                n_new = 3 if (bi == 3 and ai == 4) else 4
                alt = _fresh_seq(g, V, n_new, first_avoid=used)
                used.append(alt[0])
                seqs.append(spine[:b] + alt)
        d = int(gp.integers(8, 49))
        return Candidates(root, seqs, 0, d, cfg.max_nodes, cfg.max_depth)

    if cfg.name == "llama3.1-8b-decode":
        spine = _fresh_seq(g, V, 64)
        seqs: List[List[int]] = []
        divergent: Dict[Tuple[int, int], List[int]] = {}  # (source, depth) -> tokens used there
        sources: List[List[int]] = []
        if step >= 30:
            hint = spine[:4] + _fresh_seq(g, V, 56, first_avoid=[spine[4]])
            seqs.append(hint)
            sources.append(hint)
            divergent[(id(spine), 4)] = [spine[4], hint[4]]
        seqs.append(spine)
        sources.append(spine)
        new_tokens = sum(len(s) for s in seqs) - (4 if step >= 30 else 0)
        # retrieved calls: share a prefix of the spine (or of an earlier
        # branch), then diverge; keep adding until the budget overflows
        while new_tokens < cfg.max_nodes + 40:
            src = sources[int(g.integers(0, len(sources)))]
            r = int(g.integers(0, max(1, len(src) - 4)))
            length = int(g.integers(r + 2, cfg.max_depth + 1))
            key = (id(src), r)
            used = divergent.setdefault(key, [src[r]] if r < len(src) else [])
            tail = _fresh_seq(g, V, length - r, first_avoid=used)
            used.append(tail[0])
            br = src[:r] + tail
            seqs.append(br)
            sources.append(br)
            new_tokens += len(tail)
        plant_seq = seqs[0]
        d = min(int(gp.integers(0, 65)), len(plant_seq))
        return Candidates(root, seqs, 0, d, cfg.max_nodes, cfg.max_depth)

    raise KeyError(cfg.name)


# ----------------------------------------------------------------------------
# designated greedy tokens and hidden rows (planted acceptance)


def node_prefixes(token: np.ndarray, parent: np.ndarray) -> List[Tuple[int, ...]]:
    """Token path (excluding the root) of every node of a packed trie."""
    n = len(token)
    pre: List[Tuple[int, ...]] = [()] * n
    for i in range(1, n):
        p = int(parent[i])
        pre[i] = pre[p] + (int(token[i]),)
    return pre


def designated_tokens(cfg: VerifyConfig, seed: int, step: int, cands: Candidates,
                      token: np.ndarray, parent: np.ndarray, island_prob: float = 0.5) -> Tuple[np.ndarray, int]:
    """Greedy token each node's hidden row is built to select.

    Returns ``(tau, planted_depth)``; ``planted_depth`` is the plant depth
    clipped to what the packed trie actually holds of the plant branch.
    """
    n = len(token)
    g = rng(cfg, seed, step, S_TAU)
    pre = node_prefixes(token, parent)
    index = {p: i for i, p in enumerate(pre)}
    children: List[List[int]] = [[] for _ in range(n)]
    for i in range(1, n):
        children[int(parent[i])].append(int(token[i]))
    plant = cands.seqs[cands.plant_index] if cands.seqs else []
    d = min(cands.plant_depth, len(plant), cands.max_depth)
    while d > 0 and tuple(plant[:d]) not in index:
        d -= 1
    on_path = {index[tuple(plant[:k])]: k for k in range(d + 1)}
    tau = np.empty(n, dtype=np.int64)
    for i in range(n):
        ch = children[i]
        if i in on_path:
            k = on_path[i]
            tau[i] = plant[k] if k < d else _fresh(g, cfg.vocab, ch)
        elif ch and g.random() < island_prob:
            # a matching child below a rejected ancestor: must not be accepted
            tau[i] = ch[int(g.integers(0, len(ch)))]
        else:
            tau[i] = _fresh(g, cfg.vocab, ch)
    return tau, d


def lm_head_weight(cfg: VerifyConfig, seed: int) -> np.ndarray:
    """W[V][H] ~ N(0, 0.02^2), stored in ``cfg.dtype``."""
    return draw(cfg, seed, 0, S_LMW, (cfg.vocab, cfg.hidden), std=0.02)


def hidden_rows(cfg: VerifyConfig, seed: int, step: int, w_stored: np.ndarray,
                tau: Optional[np.ndarray], n_nodes: int, boost: float = HIDDEN_BOOST) -> np.ndarray:
    """X[N][H]: N(0,1) rows (unit-RMS stand-in for the final norm's output),
    each pushed along its designated token's weight direction when ``tau``
    is given."""
    x = normal(cfg, seed, step, S_HIDDEN, (n_nodes, cfg.hidden))
    if tau is not None and boost != 0.0:
        wrows = to_f64(w_stored[np.asarray(tau, dtype=np.int64)], cfg.dtype)
        norms = np.sqrt((wrows * wrows).sum(axis=1, keepdims=True))
        x = (x.astype(np.float64) + boost * wrows / norms).astype(np.float32)
    return store(x, cfg.dtype)


# ----------------------------------------------------------------------------
# attention inputs


def queries(cfg: VerifyConfig, seed: int, step: int, layer: int, n_nodes: int) -> np.ndarray:
    """Q[N][Hq][D] for one layer (post-RoPE stand-in)."""
    return draw(cfg, seed, step, S_QUERY, (n_nodes, cfg.n_q_heads, cfg.head_dim), extra=(layer,))


def prefix_kv(cfg: VerifyConfig, seed: int, layer: int, prefix_len: Optional[int] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Committed prefix rows K,V[Hkv][P][D] of one layer."""
    P = cfg.prefix_len if prefix_len is None else prefix_len
    shp = (cfg.n_kv_heads, P, cfg.head_dim)
    return draw(cfg, seed, 0, S_KPRE, shp, extra=(layer,)), draw(cfg, seed, 0, S_VPRE, shp, extra=(layer,))


def tree_kv(cfg: VerifyConfig, seed: int, step: int, layer: int, n_nodes: int) -> Tuple[np.ndarray, np.ndarray]:
    """This step's node rows K,V[Hkv][N][D] of one layer (row i = node i)."""
    shp = (cfg.n_kv_heads, n_nodes, cfg.head_dim)
    return draw(cfg, seed, step, S_KTREE, shp, extra=(layer,)), draw(cfg, seed, step, S_VTREE, shp, extra=(layer,))


def layer_cache(cfg: VerifyConfig, seed: int, layer: int, n_nodes: int, step: int = 0,
                prefix_len: Optional[int] = None) -> Tuple[np.ndarray, np.ndarray]:
    """One layer's K and V cache [Hkv][cap][D]: prefix rows, then this step's
    node rows at [P, P+N), zero beyond."""
    P = cfg.prefix_len if prefix_len is None else prefix_len
    dt = np.uint16 if cfg.dtype == "bf16" else np.float32
    k = np.zeros((cfg.n_kv_heads, cfg.cap, cfg.head_dim), dtype=dt)
    v = np.zeros_like(k)
    kp, vp = prefix_kv(cfg, seed, layer, P)
    kt, vt = tree_kv(cfg, seed, step, layer, n_nodes)
    k[:, :P] = kp
    v[:, :P] = vp
    k[:, P:P + n_nodes] = kt
    v[:, P:P + n_nodes] = vt
    return k, v
