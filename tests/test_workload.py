"""Seeded input generator: determinism, shapes of each workload's trie,
bf16 rounding, and planted acceptance confirmed by the CPU reference."""

import numpy as np
import pytest
import torch

from oracle import tree_verify as ov
from paper_2608_00814_amd import workload as wl


def test_bf16_rounding_matches_torch():
    rs = np.random.default_rng(0)
    x = np.concatenate([rs.normal(size=10000).astype(np.float32) * 10.0 ** rs.integers(-8, 8, size=10000),
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.01171875, 3.4e38, -1e-40], dtype=np.float32)]).astype(np.float32)
    ours = wl.to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    assert np.array_equal(wl.bf16_to_f32(ours), torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_draws_are_deterministic_and_thread_independent():
    cfg = wl.CONFIGS["qwen3-0.6b"]
    a = wl.normal(cfg, 3, 0, wl.S_KPRE, (8, 1024, 128), extra=(5,))
    b = wl.normal(cfg, 3, 0, wl.S_KPRE, (8, 1024, 128), extra=(5,))
    c = wl.normal(cfg, 4, 0, wl.S_KPRE, (8, 1024, 128), extra=(5,))
    assert np.array_equal(a, b) and not np.array_equal(a, c)
    assert abs(float(a.std()) - 1.0) < 0.01


EXPECTED_SHAPE = {
    # name: (nodes, max depth, max branching, truncated tokens or None)
    "tiny-fp32": (None, 8, None, 0),
    "qwen3-0.6b": (32, 12, 2, 8),
    "qwen3-8b": (64, 40, 2, 0),
    "qwen2.5-32b": (128, 48, 6, 0),
}


@pytest.mark.parametrize("name", list(EXPECTED_SHAPE))
@pytest.mark.parametrize("seed", range(5))
def test_trie_shapes(name, seed):
    cfg = wl.CONFIGS[name]
    c = wl.candidates_for(cfg, seed)
    t = ov.pack_tree(c.root_token, c.seqs, c.max_nodes, c.max_depth)
    nodes, depth, branch, trunc = EXPECTED_SHAPE[name]
    if nodes is None:
        assert t["n_nodes"] <= 25
    else:
        assert t["n_nodes"] == nodes
    assert int(t["depth"].max()) == depth
    if branch is not None:
        assert int(np.bincount(t["parent"][1:]).max()) == branch
    assert t["n_truncated"] == trunc


@pytest.mark.parametrize("step", [0, 29, 30, 31, 199])
def test_decode_trie_shape(step):
    cfg = wl.CONFIGS["llama3.1-8b-decode"]
    c = wl.candidates_for(cfg, 0, step, root_token=17)
    t = ov.pack_tree(c.root_token, c.seqs, c.max_nodes, c.max_depth)
    assert t["n_nodes"] == 256 and t["n_truncated"] > 0
    assert int(t["depth"].max()) <= 64
    assert c.root_token == 17
    if step >= 30:
        assert len(c.seqs[0]) == 60 and c.seqs[0][:4] == c.seqs[1][:4] and c.seqs[0][4] != c.seqs[1][4]
    else:
        assert len(c.seqs[0]) == 64


@pytest.mark.parametrize("seed", range(5))
def test_planted_acceptance_tiny(seed):
    """tiny-fp32: the reference's greedy walk accepts exactly the planted 5
    tokens of candidate 0, with every node's logit margin >= 1e-2."""
    cfg = wl.CONFIGS["tiny-fp32"]
    c = wl.candidates_for(cfg, seed)
    t = ov.pack_tree(c.root_token, c.seqs, c.max_nodes, c.max_depth)
    tau, d = wl.designated_tokens(cfg, seed, 0, c, t["token"], t["parent"])
    assert d == 5
    w = wl.lm_head_weight(cfg, seed)
    x = wl.hidden_rows(cfg, seed, 0, w, tau, t["n_nodes"])
    g = ov.greedy_tokens(ov.lm_head_logits(wl.to_f64(x, cfg.dtype), wl.to_f64(w, cfg.dtype)))
    assert np.array_equal(g["ids"], tau)
    assert g["margin"].min() >= 1e-2
    a = ov.accept_walk(t["token"], t["parent"], g["ids"])
    assert a["L"] == 5
    assert a["committed"].tolist() == c.seqs[0][:5] + [int(tau[a["path"][-1]])]


def test_unboosted_hidden_rows_are_plain_normal():
    cfg = wl.CONFIGS["tiny-fp32"]
    w = wl.lm_head_weight(cfg, 0)
    x = wl.hidden_rows(cfg, 0, 0, w, None, 25)
    assert x.dtype == np.float32 and x.shape == (25, 256)
    assert abs(float(x.std()) - 1.0) < 0.05
