"""Checks that pin the CPU reference to things other than itself.

Each ``check_*`` takes the reference module as an argument and raises
AssertionError on a mismatch, so the same checks run against the committed
reference (they must pass) and against copies with a planted mistake (some
check must fail).  What each check leans on:

* hand-derived fixtures under ``golden/`` (pack, accept, compact, hint-bank
  continuations and lane filling);
* brute force: distinct-prefix enumeration for packing; causal decoding of
  every root-to-leaf path as an ordinary sequence for attention; a regular-
  expression search of the hint bank for every suffix length;
* a library routine: torch's scaled_dot_product_attention (float64, CPU)
  with an explicit boolean mask and repeat_interleave for grouped heads;
  numpy's matmul/argmax for the LM head;
* closed forms: constant values, zero keys;
* sequential greedy decoding of a tiny transformer-like model, the audit the
  paper applies to every method (Section 5.3): tree verification must commit
  exactly the tokens plain greedy decoding produces, step after step,
  including the cache rows compaction leaves behind.
"""

from __future__ import annotations

import json
import math
import os

import numpy as np
import torch
import torch.nn.functional as F

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# ----------------------------------------------------------------------------
# packing


def brute_pack(root, cands, max_nodes, max_depth):
    """Node i>0 is the i-th distinct candidate prefix in scan order (within
    the depth cap), keeping the first max_nodes-1 of them."""
    prefixes, seen = [], set()
    for c in cands:
        for k in range(1, min(len(c), max_depth) + 1):
            p = tuple(int(t) for t in c[:k])
            if p not in seen:
                seen.add(p)
                prefixes.append(p)
    kept = prefixes[: max_nodes - 1]
    index = {(): 0}
    for i, p in enumerate(kept):
        index[p] = i + 1
    token = [int(root)] + [p[-1] for p in kept]
    parent = [-1] + [index[p[:-1]] for p in kept]
    depth = [0] + [len(p) for p in kept]
    trunc = 0
    for c in cands:
        trunc += max(0, len(c) - max_depth)
        trunc += sum(1 for k in range(1, min(len(c), max_depth) + 1) if tuple(c[:k]) not in index)
    return token, parent, depth, trunc


def random_candidate_sets(seed, count=60):
    rs = np.random.default_rng(seed)
    for _ in range(count):
        V = int(rs.choice([3, 5, 50]))
        n_c = int(rs.integers(0, 7))
        cands = []
        for _ in range(n_c):
            kind = rs.random()
            if cands and kind < 0.25:
                base = cands[int(rs.integers(0, len(cands)))]
                c = list(base[: int(rs.integers(0, len(base) + 1))])  # a prefix of an earlier one
            elif cands and kind < 0.4:
                c = list(cands[int(rs.integers(0, len(cands)))])  # duplicate
            else:
                c = [int(t) for t in rs.integers(0, V, size=int(rs.integers(0, 12)))]
            if rs.random() < 0.3:
                c = c + [int(t) for t in rs.integers(0, V, size=int(rs.integers(0, 5)))]
            cands.append(c)
        max_nodes = int(rs.choice([1, 2, 5, 17, 64, 65, 200]))
        max_depth = int(rs.choice([1, 3, 8, 64]))
        yield int(rs.integers(0, V)), cands, max_nodes, max_depth


def check_pack_golden(ov):
    for case in _load("pack_cases.json")["cases"]:
        t = ov.pack_tree(case["root"], case["candidates"], case["max_nodes"], case["max_depth"])
        assert t["token"].tolist() == case["token"]
        assert t["parent"].tolist() == case["parent"]
        assert t["depth"].tolist() == case["depth"]
        assert t["n_truncated"] == case["n_truncated"]
        m = ov.ancestor_masks(t["parent"], 1)
        assert m[:, 0].tolist() == case["anc_mask"]


def check_pack_bruteforce(ov):
    for root, cands, max_nodes, max_depth in random_candidate_sets(11):
        t = ov.pack_tree(root, cands, max_nodes, max_depth)
        tok, par, dep, trunc = brute_pack(root, cands, max_nodes, max_depth)
        assert t["token"].tolist() == tok, (cands, max_nodes, max_depth)
        assert t["parent"].tolist() == par
        assert t["depth"].tolist() == dep
        assert t["n_truncated"] == trunc
        n = t["n_nodes"]
        assert n == len(tok)
        # invariants: parents precede children, siblings carry distinct tokens
        for i in range(1, n):
            assert 0 <= par[i] < i and dep[i] == dep[par[i]] + 1
        sib = {}
        for i in range(1, n):
            key = (par[i], tok[i])
            assert key not in sib
            sib[key] = i


# ----------------------------------------------------------------------------
# attention


def _random_trie(ov, rs, n_cand=4, max_len=6, vocab=4, max_nodes=64):
    cands = [[int(t) for t in rs.integers(0, vocab, size=int(rs.integers(1, max_len + 1)))] for _ in range(n_cand)]
    return ov.pack_tree(0, cands, max_nodes, 64), cands


def _attn_inputs(rs, N, P, Hq, Hkv, D, rows_extra=3):
    q = rs.normal(size=(N, Hq, D))
    k = rs.normal(size=(Hkv, P + N + rows_extra, D))
    v = rs.normal(size=(Hkv, P + N + rows_extra, D))
    return q, k, v


def _sdpa(q_rows, keys, vals, allowed, G):
    """q_rows [T][Hq][D]; keys/vals [Hkv][S][D]; allowed [T][S] bool."""
    qt = torch.from_numpy(q_rows).permute(1, 0, 2).unsqueeze(0)  # [1][Hq][T][D]
    kt = torch.from_numpy(keys).repeat_interleave(G, dim=0).unsqueeze(0)
    vt = torch.from_numpy(vals).repeat_interleave(G, dim=0).unsqueeze(0)
    m = torch.from_numpy(allowed).unsqueeze(0).unsqueeze(0)
    o = F.scaled_dot_product_attention(qt, kt, vt, attn_mask=m)
    return o[0].permute(1, 0, 2).numpy()  # [T][Hq][D]


def check_attention_causal_paths(ov):
    """Every root-to-leaf path, decoded as an ordinary causal sequence after
    the prefix, gives each node the output the tree pass gives it."""
    rs = np.random.default_rng(3)
    for trial in range(12):
        Hkv = int(rs.choice([1, 2]))
        G = int(rs.choice([1, 2, 3]))
        Hq, D = Hkv * G, int(rs.choice([4, 8]))
        P = int(rs.choice([0, 1, 5]))
        tree, _ = _random_trie(ov, rs, n_cand=int(rs.integers(1, 5)))
        N = tree["n_nodes"]
        parent = tree["parent"]
        q, k, v = _attn_inputs(rs, N, P, Hq, Hkv, D)
        out = ov.tree_attention(q, k, v, P, parent, Hkv)
        leaves = [i for i in range(N) if i not in set(parent.tolist())]
        for leaf in leaves:
            path = []
            j = leaf
            while j >= 0:
                path.append(j)
                j = int(parent[j])
            path = path[::-1]
            T = len(path)
            rows = list(range(P)) + [P + a for a in path]
            allowed = np.zeros((T, P + T), dtype=bool)
            for t in range(T):
                allowed[t, : P + t + 1] = True
            ref = _sdpa(q[path], k[:, rows], v[:, rows], allowed, G)
            np.testing.assert_allclose(out[path], ref, rtol=1e-11, atol=1e-12)


def check_attention_sdpa_root_and_chain(ov):
    """Root-only tree (plain decode) and a single chain (causal suffix)."""
    rs = np.random.default_rng(4)
    for Hkv, G, D, P, N in [(2, 2, 8, 7, 1), (1, 4, 16, 9, 6), (2, 3, 8, 0, 5), (4, 1, 4, 1, 4)]:
        Hq = Hkv * G
        parent = np.array([-1] + list(range(N - 1)), dtype=np.int32)
        q, k, v = _attn_inputs(rs, N, P, Hq, Hkv, D, rows_extra=0)
        allowed = np.zeros((N, P + N), dtype=bool)
        for i in range(N):
            allowed[i, : P + i + 1] = True
        ref = _sdpa(q, k, v, allowed, G)
        out = ov.tree_attention(q, k, v, P, parent, Hkv)
        np.testing.assert_allclose(out, ref, rtol=1e-11, atol=1e-12)
        for i in range(N):
            for h in range(Hq):
                np.testing.assert_allclose(ov.attention_row(q, k, v, P, parent, Hkv, i, h), ref[i, h],
                                           rtol=1e-11, atol=1e-12)


def check_attention_closed_forms(ov):
    rs = np.random.default_rng(5)
    tree, _ = _random_trie(ov, rs, n_cand=5)
    N, parent = tree["n_nodes"], tree["parent"]
    Hkv, G, D, P = 2, 2, 8, 6
    Hq = Hkv * G
    q, k, v = _attn_inputs(rs, N, P, Hq, Hkv, D)
    # every value row equal -> output equals that row
    vc = np.broadcast_to(rs.normal(size=(Hkv, 1, D)), v.shape).copy()
    out = ov.tree_attention(q, k, vc, P, parent, Hkv)
    for h in range(Hq):
        np.testing.assert_allclose(out[:, h], np.broadcast_to(vc[h // G, 0], (N, D)), rtol=1e-12, atol=1e-12)
    # zero keys -> uniform weights: mean of the prefix rows and the chain rows
    out = ov.tree_attention(q, np.zeros_like(k), v, P, parent, Hkv)
    for i in range(N):
        anc = []
        j = i
        while j >= 0:
            anc.append(P + j)
            j = int(parent[j])
        rows = list(range(P)) + anc
        for h in range(Hq):
            np.testing.assert_allclose(out[i, h], v[h // G, rows].mean(axis=0), rtol=1e-12, atol=1e-12)


def check_attention_renumbering(ov):
    """Packing the same candidates in another priority order renumbers the
    nodes; each token path keeps its output."""
    rs = np.random.default_rng(6)
    cands = [[int(t) for t in rs.integers(0, 3, size=int(rs.integers(1, 6)))] for _ in range(5)]
    t1 = ov.pack_tree(0, cands, 64, 64)
    t2 = ov.pack_tree(0, cands[::-1], 64, 64)
    assert t1["n_nodes"] == t2["n_nodes"]
    N = t1["n_nodes"]

    def paths(t):
        out = []
        for i in range(N):
            p, j = [], i
            while j > 0:
                p.append(int(t["token"][j]))
                j = int(t["parent"][j])
            out.append(tuple(p[::-1]))
        return out

    p1, p2 = paths(t1), paths(t2)
    perm = [p2.index(p) for p in p1]  # node i of t1 is node perm[i] of t2
    Hkv, G, D, P = 2, 2, 8, 4
    q1, k1, v1 = _attn_inputs(rs, N, P, Hkv * G, Hkv, D, rows_extra=0)
    q2 = np.empty_like(q1)
    k2, v2 = k1.copy(), v1.copy()
    for i in range(N):
        q2[perm[i]] = q1[i]
        k2[:, P + perm[i]] = k1[:, P + i]
        v2[:, P + perm[i]] = v1[:, P + i]
    o1 = ov.tree_attention(q1, k1, v1, P, t1["parent"], Hkv)
    o2 = ov.tree_attention(q2, k2, v2, P, t2["parent"], Hkv)
    np.testing.assert_allclose(o1, o2[perm], rtol=1e-12, atol=1e-13)


# ----------------------------------------------------------------------------
# LM head, greedy token, accept, compact


def check_lm_head_library(ov):
    rs = np.random.default_rng(8)
    x = rs.normal(size=(7, 32))
    w = rs.normal(size=(301, 32)) * 0.1
    logits = ov.lm_head_logits(x, w, rows_per_chunk=64)
    np.testing.assert_allclose(logits, x @ w.T, rtol=1e-12, atol=1e-12)
    g = ov.greedy_tokens(logits)
    assert g["ids"].tolist() == np.argmax(x @ w.T, axis=1).tolist()
    srt = np.sort(x @ w.T, axis=1)
    np.testing.assert_allclose(g["margin"], srt[:, -1] - srt[:, -2], rtol=1e-12, atol=1e-12)
    # exact ties go to the lowest index
    w2 = w.copy()
    w2[250] = w2[17] = x[0] * 10.0
    g2 = ov.greedy_tokens(ov.lm_head_logits(x[:1], w2))
    assert int(g2["ids"][0]) == 17 and g2["margin"][0] == 0.0


def check_lm_head_closed_forms(ov):
    """Logits with a closed form: a hidden row c*e_j reads column j of W
    (one nonzero product per logit); weight rows v*u give logits v*(x.u),
    so the greedy token is the last row when x.u > 0 and row 0 when x.u < 0."""
    rs = np.random.default_rng(21)
    V, H = 203, 48
    w = rs.normal(size=(V, H))
    x = np.zeros((3, H))
    for i, (j, c) in enumerate(((0, 2.0), (17, -0.5), (47, 3.0))):
        x[i, j] = c
    logits = ov.lm_head_logits(x, w, rows_per_chunk=50)
    for i, (j, c) in enumerate(((0, 2.0), (17, -0.5), (47, 3.0))):
        assert logits[i].tolist() == (c * w[:, j]).tolist()
    u = rs.normal(size=H)
    wl = np.arange(V, dtype=np.float64)[:, None] * u[None, :]
    xs = np.stack([u, -u])
    g = ov.greedy_tokens(ov.lm_head_logits(xs, wl, rows_per_chunk=64))
    assert g["ids"].tolist() == [V - 1, 0]
    uu = float(u @ u)
    assert abs(g["max_logit"][0] - (V - 1) * uu) <= 1e-9 * V * uu
    assert abs(g["margin"][0] - uu) <= 1e-9 * V * uu


def check_accept_golden(ov):
    data = _load("accept_cases.json")
    token = np.array(data["token"], dtype=np.int32)
    parent = np.array(data["parent"], dtype=np.int32)
    for case in data["cases"]:
        a = ov.accept_walk(token, parent, np.array(case["ids"], dtype=np.int32))
        assert a["path"].tolist() == case["path"]
        assert a["L"] == case["L"] and a["bonus"] == case["bonus"]
        assert a["committed"].tolist() == case["committed"]


def check_compact_golden(ov):
    for case in _load("compact_cases.json")["cases"]:
        rows = np.array(case["rows"], dtype=np.float64).reshape(1, -1, 1)
        ov.kv_compact([rows], case["prefix_len"], np.array(case["path"]))
        assert rows.reshape(-1).tolist() == case["after"]


def check_compact_gather_scatter(ov):
    """In-place compaction equals reading every source row first and then
    writing all destinations (no hazard between overlapping rows)."""
    rs = np.random.default_rng(9)
    for trial in range(40):
        P = int(rs.integers(0, 6))
        N = int(rs.integers(1, 12))
        # an increasing path from node 0 (parent < child along any path)
        L = int(rs.integers(0, N))
        path = [0] + sorted(rs.choice(np.arange(1, N), size=L, replace=False).tolist()) if N > 1 else [0]
        path = np.array(path)
        cache = rs.normal(size=(2, 3, P + N + 2, 4))
        before = cache.copy()
        src = cache[..., P + path, :].copy()
        expect = cache.copy()
        expect[..., P + np.arange(len(path)), :] = src
        ov.kv_compact([cache], P, path)
        assert np.array_equal(cache, expect)
        assert np.array_equal(cache[..., :P, :], before[..., :P, :])


# ----------------------------------------------------------------------------
# sequential greedy decoding of a tiny model


class TinyModel:
    """Embedding + position -> per-head q, k, v; one attention layer; the
    node's hidden row is the RMS-normalised concatenation of its head
    outputs; an LM head maps it to logits."""

    def __init__(self, seed, vocab=40, emb=24, Hq=4, Hkv=2, D=8, max_pos=128):
        rs = np.random.default_rng(seed)
        self.V, self.Hq, self.Hkv, self.D = vocab, Hq, Hkv, D
        self.emb = rs.normal(size=(vocab, emb))
        self.pos = rs.normal(size=(max_pos, emb)) * 0.5
        self.wq = rs.normal(size=(Hq * D, emb)) / math.sqrt(emb)
        self.wk = rs.normal(size=(Hkv * D, emb)) / math.sqrt(emb)
        self.wv = rs.normal(size=(Hkv * D, emb)) / math.sqrt(emb)
        self.wlm = rs.normal(size=(vocab, Hq * D))

    def qkv(self, tok, p):
        x = self.emb[tok] + self.pos[p]
        return ((self.wq @ x).reshape(self.Hq, self.D), (self.wk @ x).reshape(self.Hkv, self.D),
                (self.wv @ x).reshape(self.Hkv, self.D))

    @staticmethod
    def hidden(o):
        h = o.reshape(-1)
        return h / math.sqrt(float((h * h).mean()) + 1e-6)


def _greedy_decode(model, prefix_tokens, root, steps):
    """Plain sequential greedy decoding with torch SDPA per token."""
    ks, vs = [], []
    for j, t in enumerate(prefix_tokens):
        _, k, v = model.qkv(int(t), j)
        ks.append(k)
        vs.append(v)
    seq = [int(root)]
    G = model.Hq // model.Hkv
    for s in range(steps):
        pos = len(prefix_tokens) + s
        q, k, v = model.qkv(seq[-1], pos)
        ks.append(k)
        vs.append(v)
        K = np.stack(ks, axis=1)  # [Hkv][T][D]
        Vv = np.stack(vs, axis=1)
        o = _sdpa(q[None], K, Vv, np.ones((1, K.shape[1]), dtype=bool), G)[0]
        logits = model.wlm @ model.hidden(o)
        seq.append(int(np.argmax(logits)))
    return seq[1:], np.stack(ks, axis=1), np.stack(vs, axis=1)


def check_sequential_greedy(ov):
    """Three chained verify steps (pack, tree attention, LM head, accept,
    compact) commit exactly the tokens, and leave exactly the cache rows,
    that plain greedy decoding produces."""
    model = TinyModel(seed=12)
    rs = np.random.default_rng(13)
    P0 = 5
    prefix = [int(t) for t in rs.integers(0, model.V, size=P0)]
    root0 = int(rs.integers(0, model.V))
    truth, Kseq, Vseq = _greedy_decode(model, prefix, root0, 40)
    cap = 96
    kc = np.zeros((model.Hkv, cap, model.D))
    vc = np.zeros_like(kc)
    for j, t in enumerate(prefix):
        _, kc[:, j], vc[:, j] = model.qkv(t, j)
    P, root, done = P0, root0, 0
    plants = [5, 0, 3]
    for step, d in enumerate(plants):
        future = truth[done:]
        wrong = [(t + 1 + int(rs.integers(0, model.V - 1))) % model.V for t in future[:12]]
        cands = [future[:d] + [wrong[d]] + [int(t) for t in rs.integers(0, model.V, size=2)],
                 future[:1] + [wrong[1]] + [int(rs.integers(0, model.V))],
                 [wrong[0], int(rs.integers(0, model.V))]]
        if d == 0:
            cands = cands[2:]
        tree = ov.pack_tree(root, cands, 64, 16)
        N = tree["n_nodes"]
        q = np.zeros((N, model.Hq, model.D))
        for i in range(N):
            q[i], kc[:, P + i], vc[:, P + i] = model.qkv(int(tree["token"][i]), P + int(tree["depth"][i]))
        out = ov.tree_attention(q, kc, vc, P, tree["parent"], model.Hkv)
        x = np.stack([model.hidden(out[i]) for i in range(N)])
        greedy = ov.greedy_tokens(ov.lm_head_logits(x, model.wlm))
        acc = ov.accept_walk(tree["token"], tree["parent"], greedy["ids"])
        assert acc["L"] == d, (step, acc["L"], d)
        assert acc["committed"].tolist() == future[: d + 1]
        ov.kv_compact([kc, vc], P, acc["path"])
        P += acc["L"] + 1
        root = acc["bonus"]
        done += d + 1
        # rows [0, P) now hold the states sequential decoding built for the
        # prefix, the old root and the accepted tokens
        np.testing.assert_allclose(kc[:, :P], Kseq[:, :P], rtol=0, atol=0)
        np.testing.assert_allclose(vc[:, :P], Vseq[:, :P], rtol=0, atol=0)


# ----------------------------------------------------------------------------
# the whole step on the tiny workload (Section 4.5, verify and commit)


def _path_sdpa(q, k, v, P, parent, G):
    """Each node's output by causal SDPA over [prefix; its root path]."""
    N = len(parent)
    out = np.empty_like(q)
    for i in range(N):
        chain = []
        j = i
        while j >= 0:
            chain.append(j)
            j = int(parent[j])
        chain = chain[::-1]
        rows = list(range(P)) + [P + a for a in chain]
        allowed = np.ones((1, len(rows)), dtype=bool)
        out[i] = _sdpa(q[i:i + 1], k[:, rows], v[:, rows], allowed, G)[0]
    return out


def check_verify_step(ov):
    """The composed oracle step on the fp32 workload (two layers' draws) returns what
    its inputs fix independently of it: the trie of brute-force prefix
    enumeration; the greedy token each node's hidden row was built to select
    (a margin wide enough that no other token competes); the planted
    acceptance depth, the plant branch's nodes as the path, and the bonus the
    deepest of them selects; and per-node attention equal to causal SDPA over
    the prefix and the node's own root path."""
    import sys
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    from paper_2608_00814_amd import workload as wl
    cfg = wl.CONFIGS["tiny-fp32"]
    for seed in range(2):
        cands = wl.candidates_for(cfg, seed, 0)
        token, parent, _, _ = brute_pack(cands.root_token, cands.seqs, cands.max_nodes, cands.max_depth)
        token, parent = np.array(token), np.array(parent)
        N = len(token)
        tau, d = wl.designated_tokens(cfg, seed, 0, cands, token, parent)
        w = wl.lm_head_weight(cfg, seed)
        x = wl.to_f64(wl.hidden_rows(cfg, seed, 0, w, tau, N), cfg.dtype)
        layers = []
        for layer in range(2):  # two layers of the workload's draws, so a mix-up of layers shows
            k, v = wl.layer_cache(cfg, seed, layer, N)
            q = wl.queries(cfg, seed, 0, layer, N)
            layers.append((wl.to_f64(q, cfg.dtype), wl.to_f64(k, cfg.dtype), wl.to_f64(v, cfg.dtype)))
        res = ov.verify_step(cands.root_token, cands.seqs, cands.max_nodes, cands.max_depth, layers,
                             cfg.prefix_len, cfg.n_kv_heads, x, wl.to_f64(w, cfg.dtype))
        assert res["tree"]["token"].tolist() == token.tolist()
        assert res["tree"]["parent"].tolist() == parent.tolist()
        assert np.asarray(res["ids"]).tolist() == tau.tolist()
        # the plant branch's first d tokens are nodes of the trie, in order
        plant = cands.seqs[cands.plant_index]
        index = {(): 0}
        for i in range(1, N):
            chain = []
            j = i
            while j > 0:
                chain.append(int(token[j]))
                j = int(parent[j])
            index[tuple(chain[::-1])] = i
        path = [index[tuple(plant[:kk])] for kk in range(d + 1)]
        assert res["L"] == d
        assert np.asarray(res["path"]).tolist()[: d + 1] == path
        assert res["bonus"] == int(tau[path[-1]])
        assert np.asarray(res["committed"]).tolist() == [int(t) for t in plant[:d]] + [int(tau[path[-1]])]
        G = cfg.n_q_heads // cfg.n_kv_heads
        assert len(res["attn"]) == len(layers)
        for (ql, kl, vl), got in zip(layers, res["attn"]):
            ref = _path_sdpa(ql, kl, vl, cfg.prefix_len, parent, G)
            np.testing.assert_allclose(got, ref, rtol=1e-10, atol=1e-12)


# ----------------------------------------------------------------------------
# hint-bank continuations and lane filling (Section 4.4)


def check_hint_golden(ov):
    g = _load("hint_cases.json")
    for c in g["hint_cases"]:
        r = ov.hint_continuations(c["bank"], 0, c["committed"], c["max_suffix"], c["max_len"])
        assert r["n"] == c["n"], c["name"]
        assert [list(x) for x in r["continuations"]] == c["continuations"], c["name"]
    for c in g["lane_cases"]:
        assert [list(x) for x in ov.merge_lanes(c["hints"], c["native"], c["n_lanes"])] == c["lanes"]


def _occurrences(bank, pattern):
    """Start positions of every (overlapping) occurrence of ``pattern`` in
    ``bank``, found by a regular-expression search over a text encoding of
    the tokens (a different search from the reference's slicing)."""
    import re
    text = "".join(f"<{t}>" for t in bank)
    pat = "".join(f"<{t}>" for t in pattern)
    starts = [m.start() for m in re.finditer("(?=" + re.escape(pat) + ")", text)]
    # map character offsets back to token positions
    pos_of = {}
    off = 0
    for i, t in enumerate(bank):
        pos_of[off] = i
        off += len(f"<{t}>")
    return [pos_of[s] for s in starts]


def brute_hints(bank, eos, committed, max_suffix, max_len):
    """Every n's proposals first, then the largest n that has any."""
    per_n = {}
    for n in range(1, min(max_suffix, len(committed)) + 1):
        props = []
        for j in _occurrences(bank, committed[-n:]):
            tail = []
            for t in bank[j + n:]:
                if t == eos or len(tail) == max_len:
                    break
                tail.append(t)
            if tail and tail not in props:
                props.append(tail)
        per_n[n] = props
    best = max([n for n, props in per_n.items() if props], default=0)
    return best, per_n.get(best, [])


def check_hint_bruteforce(ov):
    rs = np.random.default_rng(11)
    for trial in range(300):
        vocab = int(rs.integers(2, 6))  # small alphabets make long matches common
        L = int(rs.integers(0, 60))
        eos = 0
        bank = [int(t) for t in rs.integers(0, vocab + 1, size=L)]  # token 0 = EOS
        committed = [int(t) for t in rs.integers(1, vocab + 1, size=int(rs.integers(1, 10)))]
        max_suffix = int(rs.integers(1, 8))
        max_len = int(rs.integers(1, 6))
        r = ov.hint_continuations(bank, eos, committed, max_suffix, max_len)
        n, props = brute_hints(bank, eos, committed, max_suffix, max_len)
        assert r["n"] == n, (trial, r["n"], n)
        assert [list(x) for x in r["continuations"]] == props, trial
        for cont in r["continuations"]:
            assert 1 <= len(cont) <= max_len and eos not in cont
        lanes = ov.merge_lanes(props, [[9, 9], [8]], 3)
        assert lanes[:min(3, len(props))] == [list(x) for x in props[:3]]
        assert len(lanes) == min(3, len(props) + 2)


ALL_CHECKS = [
    check_pack_golden,
    check_pack_bruteforce,
    check_attention_causal_paths,
    check_attention_sdpa_root_and_chain,
    check_attention_closed_forms,
    check_lm_head_closed_forms,
    check_attention_renumbering,
    check_lm_head_library,
    check_accept_golden,
    check_compact_golden,
    check_compact_gather_scatter,
    check_sequential_greedy,
    check_verify_step,
    check_hint_golden,
    check_hint_bruteforce,
]
