"""Plain CPU reference for the target decoder around the verification path.

TEST INFRASTRUCTURE ONLY.  Like ``tree_verify``, this module is the slow,
obviously-correct definition the native library is checked against; only the
test suite, the smoke check and the benchmark's CPU-baseline leg may import
it, the product path never does, and it shares no code with the native
library.  Everything is float64 NumPy on the exact stored values.

The paper verifies with the target model itself (Section 3, Target
authority: only the target's greedy choice commits; Section 4.5: the whole
candidate tree is scored in one target forward pass; Section 5: the targets
are Qwen3 models run under HF Transformers).  It does not restate the
architecture, so the standard Qwen3 decoder layer is written out here:

    h   <- h + o_proj(attn(rope(q_norm(q)), rope(k_norm(k)), v)),
           with (q, k, v) = split(qkv_proj(rmsnorm(h)))
    h   <- h + down(silu(gate(x)) * up(x)),   x = rmsnorm(h)
    out  = rmsnorm_final(h)  -> LM head

The one point that is specific to tree verification: node i sits at the
position it would hold if its own root path were decoded sequentially, so
its rotary position is P + depth[i] (P committed rows before the root), and
its attention sees the committed prefix plus its ancestors-or-self
(``tree_verify.tree_attention``).

Readings where the paper is silent (listed with the design notes): RMSNorm
with epsilon 1e-6 over the last axis; per-head RMSNorm of q and k before the
rotation; rotate-half RoPE with base theta and frequencies
theta^(-2j/head_dim); SiLU-gated MLP; untied input embeddings.

Parity pins: none of these functions is pinned by a value the paper prints.
The test suite pins them by library routines (torch's rms_norm, silu and
scaled_dot_product_attention in float64), closed forms of the rotation, and
a dense causal forward of every root-to-leaf path.
"""

from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Dict, List, Sequence

import numpy as np

from oracle import tree_verify as tv


@dataclass
class LayerWeights:
    """One decoder layer, nn.Linear layout ([out][in]) for the projections."""

    in_norm: np.ndarray    # [H]
    w_qkv: np.ndarray      # [(Hq + 2 Hkv) * D][H]: q rows, then k rows, then v rows
    q_norm: np.ndarray     # [D]
    k_norm: np.ndarray     # [D]
    w_o: np.ndarray        # [H][Hq * D]
    post_norm: np.ndarray  # [H]
    w_gate: np.ndarray     # [I][H]
    w_up: np.ndarray       # [I][H]
    w_down: np.ndarray     # [H][I]


@dataclass
class ModelShape:
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    intermediate: int
    rope_theta: float = 1.0e6
    eps: float = 1.0e-6


# ----------------------------------------------------------------------------
# building blocks


def rmsnorm(x: np.ndarray, w: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * w over the last axis."""
    x = np.asarray(x, dtype=np.float64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * w


def rope(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotary embedding, rotate-half pairing: for j < D/2 the pair
    (x[j], x[j + D/2]) is rotated by the angle pos * theta^(-2j/D).
    x: [N][heads][D]; pos: [N]."""
    N, _, D = x.shape
    half = D // 2
    inv_freq = theta ** (-(2.0 * np.arange(half)) / D)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv_freq[None, :]  # [N][D/2]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def embed(table, tokens: Sequence[int]) -> np.ndarray:
    """Rows of the embedding table (widened after the lookup, so a table
    object that widens on indexing can stand in for a large one)."""
    return np.asarray(table[np.asarray(tokens, dtype=np.int64)], dtype=np.float64)


# ----------------------------------------------------------------------------
# one decoder layer over the trie (Section 4.5: one forward pass scores every
# node; node i is at rotary position P + depth[i])


def project_qkv(x: np.ndarray, lw: LayerWeights, shp: ModelShape, pos: np.ndarray):
    """q [N][Hq][D] and k, v [N][Hkv][D] of the normalised input rows x,
    after the per-head norms and the rotation of q and k."""
    N = x.shape[0]
    Hq, Hkv, D = shp.n_q_heads, shp.n_kv_heads, shp.head_dim
    qkv = x @ lw.w_qkv.T
    q = qkv[:, :Hq * D].reshape(N, Hq, D)
    k = qkv[:, Hq * D:(Hq + Hkv) * D].reshape(N, Hkv, D)
    v = qkv[:, (Hq + Hkv) * D:].reshape(N, Hkv, D)
    q = rope(rmsnorm(q, lw.q_norm, shp.eps), pos, shp.rope_theta)
    k = rope(rmsnorm(k, lw.k_norm, shp.eps), pos, shp.rope_theta)
    return q, k, v


def decoder_layer(h: np.ndarray, lw: LayerWeights, shp: ModelShape, k_cache: np.ndarray, v_cache: np.ndarray,
                  prefix_len: int, parent: np.ndarray, depth: np.ndarray) -> Dict[str, np.ndarray]:
    """Residual rows h [N][H] -> next layer's rows.  Writes node i's key and
    value into cache row P + i (k_cache, v_cache: [Hkv][rows][D], modified in
    place) and attends with ``tree_verify.tree_attention``."""
    N = h.shape[0]
    P = prefix_len
    pos = P + np.asarray(depth, dtype=np.int64)
    x = rmsnorm(h, lw.in_norm, shp.eps)
    q, k, v = project_qkv(x, lw, shp, pos)
    for i in range(N):
        k_cache[:, P + i] = k[i]
        v_cache[:, P + i] = v[i]
    o = tv.tree_attention(q, k_cache, v_cache, P, parent, shp.n_kv_heads)
    h = h + o.reshape(N, -1) @ lw.w_o.T
    x2 = rmsnorm(h, lw.post_norm, shp.eps)
    h = h + (silu(x2 @ lw.w_gate.T) * (x2 @ lw.w_up.T)) @ lw.w_down.T
    return {"h": h, "q": q, "k": k, "v": v, "attn": o}


def forward_tree(tokens: Sequence[int], parent: np.ndarray, depth: np.ndarray, prefix_len: int,
                 emb: np.ndarray, layers: Sequence[LayerWeights], final_norm: np.ndarray, shp: ModelShape,
                 k_caches: Sequence[np.ndarray], v_caches: Sequence[np.ndarray]) -> Dict:
    """All layers over the trie; returns the LM-head input rows X (final
    norm) plus per-layer records.  Caches are modified in place (node rows)."""
    h = embed(emb, tokens)
    recs: List[Dict[str, np.ndarray]] = []
    for lw, kc, vc in zip(layers, k_caches, v_caches):
        r = decoder_layer(h, lw, shp, kc, vc, prefix_len, parent, depth)
        recs.append(r)
        h = r["h"]
    return {"x": rmsnorm(h, final_norm, shp.eps), "h": h, "layers": recs}


def verify_step(root_token: int, candidates: Sequence[Sequence[int]], max_nodes: int, max_depth: int,
                prefix_len: int, emb: np.ndarray, layers: Sequence[LayerWeights], final_norm: np.ndarray,
                lm_head: np.ndarray, shp: ModelShape, k_caches: Sequence[np.ndarray],
                v_caches: Sequence[np.ndarray]) -> Dict:
    """The whole verify-and-commit step of the target model: pack, forward
    the trie, greedy tokens, accept, compact (caches modified in place)."""
    tree = tv.pack_tree(root_token, candidates, max_nodes, max_depth)
    fw = forward_tree(tree["token"], tree["parent"], tree["depth"], prefix_len, emb, layers, final_norm, shp,
                      k_caches, v_caches)
    greedy = tv.greedy_tokens(tv.lm_head_logits(fw["x"], lm_head))
    acc = tv.accept_walk(tree["token"], tree["parent"], greedy["ids"])
    moves = []
    for kc, vc in zip(k_caches, v_caches):
        moves = tv.kv_compact([kc, vc], prefix_len, acc["path"])
    return {"tree": tree, **fw, **greedy, **acc, "moves": moves}
