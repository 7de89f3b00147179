"""Checks that pin the decoder reference (``oracle/target_model.py``) to
things other than itself.

Each ``check_*`` takes the reference module and raises AssertionError on a
mismatch, so the same checks run against the committed reference (they must
pass) and against copies with a planted mistake (some check must fail).
What each check leans on:

* library routines in float64 on the CPU: torch's ``rms_norm``, ``silu``,
  complex multiplication (``torch.polar``) for the rotation and
  ``scaled_dot_product_attention`` with a causal mask and repeated KV heads;
* closed forms of the rotation: the identity at position 0, unchanged pair
  norms, scores that depend only on the position difference, and
  hand-computed angles;
* a dense causal forward of every root-to-leaf path of a trie, written with
  those library routines: each node's hidden rows must equal the dense
  forward's rows at its position;
* sequential greedy decoding with the dense forward (the paper's audit,
  Section 5.3): chained verify steps of the reference commit exactly the
  greedy tokens and leave exactly the dense forward's K/V rows in the cache.
"""

from __future__ import annotations

import math

import numpy as np
import torch
import torch.nn.functional as F

from oracle import tree_verify as tv

T = torch.float64


def tiny_model(seed, layers=2, H=24, Hq=4, Hkv=2, D=8, I=40, V=50, theta=100.0, eps=1e-6, om=None):
    """Random float64 model (weights, embeddings, norms, LM head)."""
    rs = np.random.default_rng(seed)
    n = lambda *s, std=0.3: rs.normal(0, std, size=s)
    lws = []
    for _ in range(layers):
        lws.append(om.LayerWeights(
            in_norm=1 + n(H, std=0.1), w_qkv=n((Hq + 2 * Hkv) * D, H), q_norm=1 + n(D, std=0.1),
            k_norm=1 + n(D, std=0.1), w_o=n(H, Hq * D), post_norm=1 + n(H, std=0.1), w_gate=n(I, H),
            w_up=n(I, H), w_down=n(H, I)))
    shp = om.ModelShape(hidden=H, n_q_heads=Hq, n_kv_heads=Hkv, head_dim=D, intermediate=I, rope_theta=theta,
                        eps=eps)
    return {"layers": lws, "shp": shp, "emb": n(V, H, std=1.0), "final": 1 + n(H, std=0.1),
            "lm": n(V, H, std=0.5), "V": V}


# ----------------------------------------------------------------------------
# the dense causal forward, written with library routines


def _t(a):
    return torch.as_tensor(np.asarray(a, dtype=np.float64), dtype=T)


def _rope_complex(x, pos, theta):
    """x [T][heads][D]: pairs (j, j + D/2) as complex numbers times
    exp(i * pos * theta^(-2j/D))."""
    D = x.shape[-1]
    half = D // 2
    freqs = _t(pos)[:, None] * theta ** (-(2.0 * torch.arange(half, dtype=T)) / D)[None, :]
    rot = torch.polar(torch.ones_like(freqs), freqs)[:, None, :]
    z = torch.complex(x[..., :half], x[..., half:]) * rot
    return torch.cat([z.real, z.imag], dim=-1)


def dense_forward(model, tokens):
    """Ordinary causal forward of one token sequence (positions 0..T-1).
    Returns the final-norm rows, the residual rows after every layer and the
    per-layer rotated keys and values."""
    shp = model["shp"]
    H, Hq, Hkv, D = shp.hidden, shp.n_q_heads, shp.n_kv_heads, shp.head_dim
    x = _t(model["emb"])[torch.as_tensor(tokens)]
    Tn = len(tokens)
    pos = np.arange(Tn)
    hs, ks, vs = [], [], []
    for lw in model["layers"]:
        a = F.rms_norm(x, (H,), weight=_t(lw.in_norm), eps=shp.eps)
        qkv = a @ _t(lw.w_qkv).T
        q = qkv[:, :Hq * D].view(Tn, Hq, D)
        k = qkv[:, Hq * D:(Hq + Hkv) * D].view(Tn, Hkv, D)
        v = qkv[:, (Hq + Hkv) * D:].view(Tn, Hkv, D)
        q = _rope_complex(F.rms_norm(q, (D,), weight=_t(lw.q_norm), eps=shp.eps), pos, shp.rope_theta)
        k = _rope_complex(F.rms_norm(k, (D,), weight=_t(lw.k_norm), eps=shp.eps), pos, shp.rope_theta)
        ks.append(k.numpy().copy())
        vs.append(v.numpy().copy())
        kx = k.repeat_interleave(Hq // Hkv, dim=1)
        vx = v.repeat_interleave(Hq // Hkv, dim=1)
        o = F.scaled_dot_product_attention(q.transpose(0, 1)[None], kx.transpose(0, 1)[None],
                                           vx.transpose(0, 1)[None], is_causal=True)[0].transpose(0, 1)
        x = x + o.reshape(Tn, Hq * D) @ _t(lw.w_o).T
        b = F.rms_norm(x, (H,), weight=_t(lw.post_norm), eps=shp.eps)
        x = x + (F.silu(b @ _t(lw.w_gate).T) * (b @ _t(lw.w_up).T)) @ _t(lw.w_down).T
        hs.append(x.numpy().copy())
    out = F.rms_norm(x, (H,), weight=_t(model["final"]), eps=shp.eps)
    return {"x": out.numpy(), "h": hs, "k": ks, "v": vs}


def _prefix_caches(model, prefix_tokens, cap):
    """Per-layer caches [Hkv][cap][D] holding the dense forward's K/V of the
    prefix at rows [0, P)."""
    shp = model["shp"]
    P = len(prefix_tokens)
    d = dense_forward(model, prefix_tokens)
    kcs, vcs = [], []
    for l in range(len(model["layers"])):
        kc = np.zeros((shp.n_kv_heads, cap, shp.head_dim))
        vc = np.zeros_like(kc)
        kc[:, :P] = d["k"][l].transpose(1, 0, 2)
        vc[:, :P] = d["v"][l].transpose(1, 0, 2)
        kcs.append(kc)
        vcs.append(vc)
    return kcs, vcs


# ----------------------------------------------------------------------------
# building blocks


def check_rmsnorm_library(om):
    rs = np.random.default_rng(1)
    for shape in [(5, 24), (3, 4, 8), (1, 64)]:
        x = rs.normal(0, 3, size=shape)
        w = rs.normal(1, 0.2, size=shape[-1])
        for eps in (1e-6, 0.5):
            ref = F.rms_norm(_t(x), (shape[-1],), weight=_t(w), eps=eps).numpy()
            assert np.allclose(om.rmsnorm(x, w, eps), ref, rtol=1e-12, atol=1e-12)


def check_silu_library(om):
    x = np.linspace(-30, 30, 601)
    assert np.allclose(om.silu(x), F.silu(_t(x)).numpy(), rtol=1e-12, atol=1e-300)


def check_rope_closed_forms(om):
    rs = np.random.default_rng(2)
    N, Hh, D, theta = 6, 3, 16, 1000.0
    x = rs.normal(size=(N, Hh, D))
    # position 0 is the identity
    assert np.allclose(om.rope(x, np.zeros(N), theta), x, rtol=0, atol=1e-15)
    # pairs (j, j + D/2) keep their norm
    pos = rs.integers(0, 5000, size=N)
    y = om.rope(x, pos, theta)
    h = D // 2
    assert np.allclose(x[..., :h] ** 2 + x[..., h:] ** 2, y[..., :h] ** 2 + y[..., h:] ** 2, rtol=1e-12)
    # complex multiplication by exp(i pos theta^(-2j/D))
    ref = _rope_complex(_t(x), pos, theta).numpy()
    assert np.allclose(y, ref, rtol=1e-11, atol=1e-11)
    # scores depend only on the position difference
    q, k = rs.normal(size=(1, 1, D)), rs.normal(size=(1, 1, D))
    for m, n in [(7, 3), (1000, 998), (5, 5), (3, 40)]:
        a = float(np.sum(om.rope(q, [m], theta) * om.rope(k, [n], theta)))
        b = float(np.sum(om.rope(q, [m - n], theta) * om.rope(k, [0], theta)))
        assert abs(a - b) < 1e-10 * (1 + abs(a))
    # hand-computed: D = 4, theta = 100, position 1: angles 1 and 1/10
    e = np.array([[[1.0, 2.0, 3.0, 4.0]]])
    c1, s1, c2, s2 = math.cos(1.0), math.sin(1.0), math.cos(0.1), math.sin(0.1)
    want = [1 * c1 - 3 * s1, 2 * c2 - 4 * s2, 3 * c1 + 1 * s1, 4 * c2 + 2 * s2]
    assert np.allclose(om.rope(e, [1], 100.0)[0, 0], want, rtol=1e-14, atol=1e-14)


# ----------------------------------------------------------------------------
# the decoder over a trie against the dense forward of every root path


def _random_tree(rs, V, n_cand=4, max_len=5, max_nodes=16, max_depth=6):
    cands = []
    for _ in range(n_cand):
        L = int(rs.integers(1, max_len + 1))
        # small token range so candidates share prefixes and branch
        cands.append([int(t) for t in rs.integers(0, min(V, 4), size=L)])
    return tv.pack_tree(int(rs.integers(0, V)), cands, max_nodes, max_depth)


def check_model_paths(om):
    rs = np.random.default_rng(3)
    for seed in range(3):
        model = tiny_model(10 + seed, om=om)
        shp = model["shp"]
        P = int(rs.integers(0, 7))
        prefix = [int(t) for t in rs.integers(0, model["V"], size=P)]
        tree = _random_tree(rs, model["V"])
        N = tree["n_nodes"]
        assert N >= 4 and tree["depth"].max() >= 2
        cap = P + N + 2
        kcs, vcs = _prefix_caches(model, prefix, cap) if P else (
            [np.zeros((shp.n_kv_heads, cap, shp.head_dim)) for _ in model["layers"]],
            [np.zeros((shp.n_kv_heads, cap, shp.head_dim)) for _ in model["layers"]])
        fw = om.forward_tree(tree["token"], tree["parent"], tree["depth"], P, model["emb"], model["layers"],
                             model["final"], shp, kcs, vcs)
        for i in range(N):
            path = tv.chain(tree["parent"], i)
            seq = prefix + [int(tree["token"][j]) for j in path]
            d = dense_forward(model, seq)
            assert np.allclose(fw["x"][i], d["x"][-1], rtol=1e-9, atol=1e-9), (seed, i)
            for l in range(len(model["layers"])):
                assert np.allclose(fw["layers"][l]["h"][i], d["h"][l][-1], rtol=1e-9, atol=1e-9)
                # node i's own key/value sit in cache row P + i
                assert np.allclose(kcs[l][:, P + i], d["k"][l][-1], rtol=1e-9, atol=1e-9)
                assert np.allclose(vcs[l][:, P + i], d["v"][l][-1], rtol=1e-9, atol=1e-9)


def _dense_greedy(model, tokens, n):
    out = list(tokens)
    margins = []
    for _ in range(n):
        x = dense_forward(model, out)["x"][-1]
        logits = _t(model["lm"]).numpy() @ x
        srt = np.sort(logits)
        margins.append(srt[-1] - srt[-2])
        out.append(int(np.argmax(logits)))
    return out[len(tokens):], min(margins)


def check_model_sequential_greedy(om):
    """Three chained verify steps with compaction commit the dense forward's
    greedy tokens, and leave its K/V rows in the cache."""
    rs = np.random.default_rng(4)
    model = tiny_model(21, om=om)
    shp = model["shp"]
    V = model["V"]
    prefix = [int(t) for t in rs.integers(0, V, size=5)]
    root = int(rs.integers(0, V))
    greedy, margin = _dense_greedy(model, prefix + [root], 12)
    assert margin > 1e-6
    cap = 64
    kcs, vcs = _prefix_caches(model, prefix, cap)
    P = len(prefix)
    committed = []
    g = 0  # greedy tokens committed so far (the root of step s is greedy[g - 1] or root)
    for s, depth in enumerate([3, 0, 4]):
        chain = greedy[g:g + depth]
        wrong = [t for t in range(V) if t != greedy[g + depth]][int(rs.integers(0, V - 1))]
        cands = [chain + [wrong], [int((greedy[g] + 1) % V), 3], chain[:1] + [int((greedy[g + 1] + 2) % V)]]
        r = om.verify_step(root, cands, 32, 8, P, model["emb"], model["layers"], model["final"], model["lm"], shp,
                           kcs, vcs)
        assert r["L"] == depth, (s, r["L"], depth)
        assert list(r["committed"]) == greedy[g:g + depth + 1]
        committed += list(r["committed"])
        # the cache now holds the dense forward's rows for [prefix; root; accepted]
        seq = prefix + [root] + greedy[g:g + depth]
        d = dense_forward(model, seq)
        for l in range(len(model["layers"])):
            assert np.allclose(kcs[l][:, :len(seq)], d["k"][l].transpose(1, 0, 2), rtol=1e-9, atol=1e-9)
            assert np.allclose(vcs[l][:, :len(seq)], d["v"][l].transpose(1, 0, 2), rtol=1e-9, atol=1e-9)
        P = len(seq)
        root = int(r["bonus"])
        prefix = seq
        g += depth + 1
    assert committed == greedy[:g]


ALL_CHECKS = [
    check_rmsnorm_library,
    check_silu_library,
    check_rope_closed_forms,
    check_model_paths,
    check_model_sequential_greedy,
]
