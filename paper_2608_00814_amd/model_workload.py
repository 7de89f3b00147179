"""Seeded synthetic weights and inputs for the target decoder around the
verification path.

Like ``workload``, this module only draws inputs (no normalisation, no
projection, no rotation, no attention, no logits); the native library's tests
and benchmark and the plain CPU reference consume what it produces.

Shapes are the decoder shapes of the targets the paper evaluates (Section 5:
Qwen3 models): hidden size, query / KV heads, head size, MLP width and
vocabulary of Qwen3-8B, plus small shapes for parity tests.  The paper's
checkpoints are not used; random weights of the same shapes stand in:
projection and embedding weights N(0, 0.02^2) and N(0, 1), norm weights
1 + N(0, 0.1^2), all rounded to bf16 and held as uint16 bit patterns.  The
committed prefix's K/V rows are N(0, 1) draws, like the path's own
workloads, unless a test builds them with the model.
"""

from __future__ import annotations

import dataclasses
from typing import Dict, List

import numpy as np

from . import workload as wl

# stream ids inside the seed key (distinct from the path workloads' streams)
S_EMB = 20
S_LAYER = 21
S_FINAL = 22
S_LMHEAD = 23
S_PREFIX_KV = 24
S_TOKENS = 25


@dataclasses.dataclass(frozen=True)
class ModelConfig:
    """A decoder shape.  ``prefix_len`` committed rows, ``cap`` cache rows per
    (layer, KV head); tries of up to ``max_nodes`` nodes and depth
    ``max_depth``."""

    name: str
    cfg_id: int
    n_layers: int
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    intermediate: int
    vocab: int
    prefix_len: int
    cap: int
    max_nodes: int
    max_depth: int
    rope_theta: float = 1.0e6
    eps: float = 1.0e-6
    description: str = ""

    @property
    def qkv_rows(self) -> int:
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim

    @property
    def mask_words(self) -> int:
        return (self.max_nodes + 63) // 64

    def weight_bytes(self) -> int:
        """bf16 bytes of the layer weights streamed per forward pass."""
        per_layer = (self.qkv_rows * self.hidden + self.hidden * self.n_q_heads * self.head_dim +
                     3 * self.intermediate * self.hidden)
        return 2 * self.n_layers * per_layer


MODEL_CONFIGS: Dict[str, ModelConfig] = {
    c.name: c
    for c in [
        ModelConfig("small-model", 10, n_layers=2, hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64,
                    intermediate=512, vocab=1000, prefix_len=100, cap=140, max_nodes=32, max_depth=12,
                    rope_theta=1.0e4, description="2-layer parity shape"),
        ModelConfig("qwen3-0.6b-model", 11, n_layers=28, hidden=1024, n_q_heads=16, n_kv_heads=8, head_dim=128,
                    intermediate=3072, vocab=151936, prefix_len=1024, cap=1056, max_nodes=32, max_depth=12,
                    description="Qwen3-0.6B decoder, 32-node trie, 1k prefix"),
        ModelConfig("qwen3-8b-model", 12, n_layers=36, hidden=4096, n_q_heads=32, n_kv_heads=8, head_dim=128,
                    intermediate=12288, vocab=151936, prefix_len=4096, cap=4160, max_nodes=64, max_depth=40,
                    description="Qwen3-8B decoder, 64-node trie, 4k prefix"),
    ]
}


def _key_cfg(cfg: ModelConfig) -> wl.VerifyConfig:
    # the path workloads' random streams are keyed by a VerifyConfig's cfg_id
    return dataclasses.replace(wl.CONFIGS["tiny-fp32"], cfg_id=cfg.cfg_id)


def _normal(cfg: ModelConfig, seed: int, stream: int, shape, std: float, extra=()) -> np.ndarray:
    return wl.normal(_key_cfg(cfg), seed, 0, stream, shape, std, extra=extra, stored="bf16")


def _norm_weight(cfg: ModelConfig, seed: int, stream: int, n: int, extra=()) -> np.ndarray:
    g = wl.rng(_key_cfg(cfg), seed, 0, stream, *extra)
    return wl.to_bf16_bits(1.0 + 0.1 * g.standard_normal(n, dtype=np.float32))


def layer_weights(cfg: ModelConfig, seed: int, layer: int) -> Dict[str, np.ndarray]:
    """bf16 bit patterns of one layer, nn.Linear layout.  ``w_qkv`` stacks the
    q rows, then the k rows, then the v rows; ``w_gate`` and ``w_up`` are
    separate [I][H] matrices."""
    H, D, I = cfg.hidden, cfg.head_dim, cfg.intermediate
    ex = lambda j: (layer, j)
    return {
        "in_norm": _norm_weight(cfg, seed, S_LAYER, H, ex(0)),
        "w_qkv": _normal(cfg, seed, S_LAYER, (cfg.qkv_rows, H), 0.02, ex(1)),
        "q_norm": _norm_weight(cfg, seed, S_LAYER, D, ex(2)),
        "k_norm": _norm_weight(cfg, seed, S_LAYER, D, ex(3)),
        "w_o": _normal(cfg, seed, S_LAYER, (H, cfg.n_q_heads * D), 0.02, ex(4)),
        "post_norm": _norm_weight(cfg, seed, S_LAYER, H, ex(5)),
        "w_gate": _normal(cfg, seed, S_LAYER, (I, H), 0.02, ex(6)),
        "w_up": _normal(cfg, seed, S_LAYER, (I, H), 0.02, ex(7)),
        "w_down": _normal(cfg, seed, S_LAYER, (H, I), 0.02, ex(8)),
    }


def embedding(cfg: ModelConfig, seed: int) -> np.ndarray:
    return _normal(cfg, seed, S_EMB, (cfg.vocab, cfg.hidden), 1.0)


def final_norm(cfg: ModelConfig, seed: int) -> np.ndarray:
    return _norm_weight(cfg, seed, S_FINAL, cfg.hidden)


def lm_head(cfg: ModelConfig, seed: int) -> np.ndarray:
    return _normal(cfg, seed, S_LMHEAD, (cfg.vocab, cfg.hidden), 0.02)


def prefix_kv(cfg: ModelConfig, seed: int, layer: int):
    """N(0, 1) K and V of the committed rows [0, P) of one layer, in a
    [Hkv][cap][D] cache (rows from P on are zero)."""
    shp = (cfg.n_kv_heads, cfg.cap, cfg.head_dim)
    k = np.zeros(shp, np.uint16)
    v = np.zeros(shp, np.uint16)
    P = cfg.prefix_len
    k[:, :P] = _normal(cfg, seed, S_PREFIX_KV, (cfg.n_kv_heads, P, cfg.head_dim), 1.0, (layer, 0))
    v[:, :P] = _normal(cfg, seed, S_PREFIX_KV, (cfg.n_kv_heads, P, cfg.head_dim), 1.0, (layer, 1))
    return k, v


def random_tokens(cfg: ModelConfig, seed: int, n: int, extra: int = 0) -> List[int]:
    g = wl.rng(_key_cfg(cfg), seed, 0, S_TOKENS, extra)
    return [int(t) for t in g.integers(0, cfg.vocab, size=n)]
