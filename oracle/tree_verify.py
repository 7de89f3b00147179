"""Plain CPU reference for OoO-Spec's target tree-verification step.

TEST INFRASTRUCTURE ONLY.  This module is the slow, obviously-correct
definition the native library is checked against.  Only the test suite, the
smoke check and the benchmark's CPU-baseline leg may import it; the product
path never does, and it shares no code with the native library.

Everything is float64 NumPy on the exact stored input values (bf16 inputs
are widened without rounding by the caller).  Where the paper fixes a result
with a plain definition, that definition is written out:

* Section 3 (Target authority, Eq. 1): with greedy decoding, the next
  output token is the target distribution's most likely token, and drafts
  never add output on their own.
* Section 3 (ToolSpec loop) and Section 4.5 (Verify and commit): all draft
  continuations form one tree that a single target pass scores; the output
  grows by the longest run of draft tokens that agree with the target's own
  greedy choices, then by the target's choice at the point of disagreement;
  the KV cache keeps the states of agreeing nodes and nothing else.

Because greedy tree verification is a faster schedule of sequential greedy
decoding, each node's attention is ordinary causal attention of the sequence
[committed prefix; root .. node]; the tree is never encoded as a mask here,
only walked through parent pointers.

Readings where the paper is silent (all are listed with the design notes):
the root is the previous step's bonus token and is always committed; node
order is first appearance over priority-ordered candidates; attention scale
is 1/sqrt(head_dim) with query head h reading KV head h // (Hq/Hkv); argmax
ties go to the lowest index; the accepted node at depth d moves to cache row
P + d.

Parity pins: none of these functions is pinned by a value the paper prints
(the paper gives no worked example for this path).  They are pinned by brute
force, closed forms, library routines and sequential greedy decoding in the
test suite.
"""

from __future__ import annotations

import math
from typing import Dict, List, Sequence, Tuple

import numpy as np


# ----------------------------------------------------------------------------
# O1: candidate trie (Section 3, ToolSpec loop; Section 4.4, Merge_B keeps a
# fixed candidate budget, hint lanes first; Section 4.5, one candidate tree)


def pack_tree(root_token: int, candidates: Sequence[Sequence[int]], max_nodes: int, max_depth: int) -> Dict:
    """Merge priority-ordered candidate continuations into one token trie.

    Node 0 is the root (the token the target committed last).  Candidates are
    walked in the given order; a token equal to an existing child is shared,
    otherwise a new node is appended while fewer than ``max_nodes`` exist.
    Tokens past ``max_depth``, and every token of a candidate from the first
    one that could not be placed, are dropped and counted in ``n_truncated``.
    """
    token: List[int] = [int(root_token)]
    parent: List[int] = [-1]
    depth: List[int] = [0]
    children: List[Dict[int, int]] = [{}]
    n_truncated = 0
    for cand in candidates:
        cur = 0
        for pos, t in enumerate(cand):
            t = int(t)
            if pos >= max_depth:
                n_truncated += len(cand) - pos
                break
            if t in children[cur]:
                cur = children[cur][t]
                continue
            if len(token) >= max_nodes:
                n_truncated += len(cand) - pos
                break
            node = len(token)
            token.append(t)
            parent.append(cur)
            depth.append(depth[cur] + 1)
            children.append({})
            children[cur][t] = node
            cur = node
    return {
        "token": np.array(token, dtype=np.int32),
        "parent": np.array(parent, dtype=np.int32),
        "depth": np.array(depth, dtype=np.int32),
        "n_nodes": len(token),
        "n_truncated": n_truncated,
    }


def chain(parent: np.ndarray, i: int) -> List[int]:
    """Root .. node ``i`` by following parent pointers."""
    out = []
    while i >= 0:
        out.append(int(i))
        i = int(parent[i])
    return out[::-1]


def ancestor_masks(parent: np.ndarray, mask_words: int) -> np.ndarray:
    """Bit j of row i set iff node j is an ancestor of i or i itself.  Only
    used to compare with the library's packed mask."""
    n = len(parent)
    m = np.zeros((n, mask_words), dtype=np.uint64)
    for i in range(n):
        for j in chain(parent, i):
            m[i, j // 64] |= np.uint64(1) << np.uint64(j % 64)
    return m


# ----------------------------------------------------------------------------
# O2: attention of every node against the committed prefix and its own
# ancestors (Section 4.5: the whole tree in one target forward pass, each
# node seeing exactly what sequential decoding of its path would see)


def tree_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, prefix_len: int,
                   parent: np.ndarray, n_kv_heads: int) -> np.ndarray:
    """Attention output O[N][Hq][D] of one layer.

    q: [N][Hq][D]; k, v: [Hkv][rows][D] with the committed prefix at rows
    [0, P) and node i's own key/value at row P + i.  Query head h reads KV
    head h // (Hq / Hkv).  For node i the keys are the P prefix rows followed
    by the rows of chain(i); scores are q.k / sqrt(D); softmax; weighted sum
    of the matching value rows.
    """
    N, Hq, D = q.shape
    G = Hq // n_kv_heads
    P = prefix_len
    scale = 1.0 / math.sqrt(D)
    out = np.zeros((N, Hq, D), dtype=np.float64)
    for g in range(n_kv_heads):
        heads = list(range(g * G, (g + 1) * G))
        kp, vp = k[g, :P], v[g, :P]
        # prefix scores of every (node, head of the group): one library matmul
        qg = q[:, heads, :].reshape(N * G, D)
        s_pre = (qg @ kp.T) * scale  # [N*G][P]
        for i in range(N):
            rows = [P + j for j in chain(parent, i)]
            kt, vt = k[g, rows], v[g, rows]
            for a, h in enumerate(heads):
                sp = s_pre[i * G + a]
                st = (kt @ q[i, h]) * scale
                m = max(sp.max() if P > 0 else -np.inf, st.max())
                pp = np.exp(sp - m)
                pt = np.exp(st - m)
                den = pp.sum() + pt.sum()
                out[i, h] = (pp @ vp + pt @ vt) / den
    return out


def attention_row(q: np.ndarray, k: np.ndarray, v: np.ndarray, prefix_len: int,
                  parent: np.ndarray, n_kv_heads: int, node: int, head: int) -> np.ndarray:
    """One output row O[node][head] of ``tree_attention``, for sampled checks
    at sizes where the whole layer is too slow."""
    N, Hq, D = q.shape
    g = head // (Hq // n_kv_heads)
    rows = list(range(prefix_len)) + [prefix_len + j for j in chain(parent, node)]
    kk, vv = k[g, rows], v[g, rows]
    s = (kk @ q[node, head]) / math.sqrt(D)
    p = np.exp(s - s.max())
    return (p @ vv) / p.sum()


# ----------------------------------------------------------------------------
# O3: LM head and greedy token (Eq. 1)


def lm_head_logits(x: np.ndarray, w: np.ndarray, rows_per_chunk: int = 8192) -> np.ndarray:
    """logits[i][v] = sum_k X[i][k] W[v][k]  (W in nn.Linear layout [V][H])."""
    V = w.shape[0]
    out = np.empty((x.shape[0], V), dtype=np.float64)
    for a in range(0, V, rows_per_chunk):
        b = min(V, a + rows_per_chunk)
        out[:, a:b] = x @ np.asarray(w[a:b], dtype=np.float64).T
    return out


def greedy_tokens(logits: np.ndarray) -> Dict[str, np.ndarray]:
    """Greedy token per node (lowest index among equal maxima), its logit and
    the gap to the runner-up logit."""
    ids = np.argmax(logits, axis=1)  # first occurrence of the maximum
    n = logits.shape[0]
    top1 = logits[np.arange(n), ids]
    rest = logits.copy()
    rest[np.arange(n), ids] = -np.inf
    top2 = rest.max(axis=1) if logits.shape[1] > 1 else np.full(n, -np.inf)
    return {"ids": ids.astype(np.int32), "max_logit": top1, "margin": top1 - top2}


# ----------------------------------------------------------------------------
# O4: keep the longest run of agreeing draft tokens (Section 4.5, Verify and commit)


def accept_walk(token: np.ndarray, parent: np.ndarray, ids: np.ndarray) -> Dict:
    """Sequential walk from the root: move to the child whose token equals
    the target's greedy token at the current node; stop when there is none.
    ``L`` counts accepted draft nodes; the step commits their tokens followed
    by the bonus token ids[path[L]] (the target's own next token)."""
    n = len(token)
    children: List[Dict[int, int]] = [{} for _ in range(n)]
    for i in range(1, n):
        children[int(parent[i])][int(token[i])] = i
    path = [0]
    cur = 0
    while int(ids[cur]) in children[cur]:
        cur = children[cur][int(ids[cur])]
        path.append(cur)
    L = len(path) - 1
    bonus = int(ids[path[-1]])
    committed = [int(token[p]) for p in path[1:]] + [bonus]
    return {"path": np.array(path, dtype=np.int32), "L": L, "bonus": bonus,
            "committed": np.array(committed, dtype=np.int32)}


# ----------------------------------------------------------------------------
# O5: commit accepted states into the KV cache (Section 4.5: the cache keeps
# the rows of agreeing nodes, rejected nodes leave no trace)


def kv_compact(caches: Sequence[np.ndarray], prefix_len: int, path: np.ndarray) -> List[Tuple[int, int]]:
    """In place, for every cache array shaped [..., rows, D]: row P + path[d]
    moves to row P + d for d = 0..L, in increasing d.  Returns the (src, dst)
    row pairs.  The committed length becomes P + L + 1."""
    pairs = [(prefix_len + int(path[d]), prefix_len + d) for d in range(len(path))]
    for c in caches:
        for src, dst in pairs:
            c[..., dst, :] = c[..., src, :]
    return pairs


# ----------------------------------------------------------------------------
# O6: hint continuations and lane filling in front of the trie (Section 4.4:
# suffix matching against the request's hint bank, n = 7 down to 1; hint
# continuations take the candidate lanes first, the native candidates fill
# the rest; an empty bank leaves the native candidates alone)


def hint_continuations(bank: Sequence[int], eos: int, committed: Sequence[int], max_suffix: int,
                       max_len: int) -> Dict:
    """Continuations the hint bank proposes for the next position.

    For n = min(max_suffix, len(committed)) down to 1, every occurrence of the
    last n committed tokens in the bank proposes the tokens that follow it,
    up to the next EOS (exclusive) and at most ``max_len`` of them.  The first
    n that proposes at least one non-empty continuation is used; its
    continuations are returned in bank order, each distinct one once.
    """
    bank = [int(t) for t in bank]
    committed = [int(t) for t in committed]
    for n in range(min(max_suffix, len(committed)), 0, -1):
        suffix = committed[len(committed) - n:]
        found: List[List[int]] = []
        for j in range(0, len(bank) - n + 1):
            if bank[j:j + n] != suffix:
                continue
            cont: List[int] = []
            k = j + n
            while k < len(bank) and bank[k] != eos and len(cont) < max_len:
                cont.append(bank[k])
                k += 1
            if cont and cont not in found:
                found.append(cont)
        if found:
            return {"n": n, "continuations": found}
    return {"n": 0, "continuations": []}


def merge_lanes(hints: Sequence[Sequence[int]], native: Sequence[Sequence[int]], n_lanes: int) -> List[List[int]]:
    """Merge_B's lane filling: hint continuations first, then the native
    candidates in their priority order, ``n_lanes`` candidates at most.  The
    node budget itself is applied by pack_tree."""
    lanes = [list(h) for h in hints][:n_lanes]
    for c in native:
        if len(lanes) >= n_lanes:
            break
        lanes.append(list(c))
    return lanes


# ----------------------------------------------------------------------------
# the whole step


def verify_step(root_token: int, candidates: Sequence[Sequence[int]], max_nodes: int, max_depth: int,
                layers: Sequence[Tuple[np.ndarray, np.ndarray, np.ndarray]], prefix_len: int,
                n_kv_heads: int, x: np.ndarray, w: np.ndarray) -> Dict:
    """Pack, attend every layer, greedy tokens, accept.  ``layers`` holds
    (q, k, v) per layer; ``x`` the node hidden rows feeding the LM head."""
    tree = pack_tree(root_token, candidates, max_nodes, max_depth)
    outs = [tree_attention(q, k, v, prefix_len, tree["parent"], n_kv_heads) for (q, k, v) in layers]
    logits = lm_head_logits(x, w)
    greedy = greedy_tokens(logits)
    acc = accept_walk(tree["token"], tree["parent"], greedy["ids"])
    return {"tree": tree, "attn": outs, "logits": logits, **greedy, **acc}
