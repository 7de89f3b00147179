"""The decoder reference around the verification path against library
routines, closed forms, the dense causal forward of every root path and
sequential greedy decoding; planted mistakes in copies of it must each fail
one of those pins (CPU only)."""

import os
import sys
import types

import pytest

import model_checks as mc
from oracle import target_model as om


@pytest.mark.parametrize("check", mc.ALL_CHECKS, ids=lambda c: c.__name__)
def test_model_reference_pin(check):
    check(om)


SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle", "target_model.py")

# (name, original text, mutated text)
MUTATIONS = [
    ("rope_interleaved_pairs", "    a, b = x[..., :half], x[..., half:]", "    a, b = x[..., 0::2], x[..., 1::2]"),
    ("rope_frequency_exponent", "    inv_freq = theta ** (-(2.0 * np.arange(half)) / D)",
     "    inv_freq = theta ** (-(1.0 * np.arange(half)) / D)"),
    ("rope_sign", "    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)",
     "    return np.concatenate([a * c + b * s, b * c - a * s], axis=-1)"),
    ("position_by_node_index", "    pos = P + np.asarray(depth, dtype=np.int64)", "    pos = P + np.arange(N)"),
    ("position_without_prefix", "    pos = P + np.asarray(depth, dtype=np.int64)",
     "    pos = np.asarray(depth, dtype=np.int64)"),
    ("no_q_norm", "    q = rope(rmsnorm(q, lw.q_norm, shp.eps), pos, shp.rope_theta)", "    q = rope(q, pos, shp.rope_theta)"),
    ("k_norm_weight_of_q", "    k = rope(rmsnorm(k, lw.k_norm, shp.eps), pos, shp.rope_theta)",
     "    k = rope(rmsnorm(k, lw.q_norm, shp.eps), pos, shp.rope_theta)"),
    ("kv_rows_swapped", "    k = qkv[:, Hq * D:(Hq + Hkv) * D].reshape(N, Hkv, D)\n    v = qkv[:, (Hq + Hkv) * D:].reshape(N, Hkv, D)",
     "    v = qkv[:, Hq * D:(Hq + Hkv) * D].reshape(N, Hkv, D)\n    k = qkv[:, (Hq + Hkv) * D:].reshape(N, Hkv, D)"),
    ("rmsnorm_eps_outside", "    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * w",
     "    return x / (np.sqrt(np.mean(x * x, axis=-1, keepdims=True)) + eps) * w"),
    ("rmsnorm_no_weight", "    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * w",
     "    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)"),
    ("silu_is_sigmoid", "    return x / (1.0 + np.exp(-x))", "    return 1.0 / (1.0 + np.exp(-x))"),
    ("mlp_without_residual", "    h = h + (silu(x2 @ lw.w_gate.T) * (x2 @ lw.w_up.T)) @ lw.w_down.T",
     "    h = (silu(x2 @ lw.w_gate.T) * (x2 @ lw.w_up.T)) @ lw.w_down.T"),
    ("gate_up_swapped", "    h = h + (silu(x2 @ lw.w_gate.T) * (x2 @ lw.w_up.T)) @ lw.w_down.T",
     "    h = h + (silu(x2 @ lw.w_up.T) * (x2 @ lw.w_gate.T)) @ lw.w_down.T"),
    ("mlp_reads_pre_attention_rows", "    x2 = rmsnorm(h, lw.post_norm, shp.eps)\n", "    x2 = rmsnorm(h - o.reshape(N, -1) @ lw.w_o.T, lw.post_norm, shp.eps)\n"),
    ("no_final_norm", "    return {\"x\": rmsnorm(h, final_norm, shp.eps), \"h\": h, \"layers\": recs}",
     "    return {\"x\": h, \"h\": h, \"layers\": recs}"),
    ("cache_row_by_depth", "        k_cache[:, P + i] = k[i]\n        v_cache[:, P + i] = v[i]",
     "        k_cache[:, P + int(depth[i])] = k[i]\n        v_cache[:, P + int(depth[i])] = v[i]"),
]


def _mutant(name, old, new):
    with open(SRC) as f:
        text = f.read()
    assert text.count(old) == 1, f"mutation {name}: anchor text not found exactly once"
    mod = types.ModuleType(f"mutant_{name}")
    sys.modules[mod.__name__] = mod  # dataclasses resolve annotations through the module
    exec(compile(text.replace(old, new), f"<mutant {name}>", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_model_mutation_is_caught(name, old, new):
    mod = _mutant(name, old, new)
    caught = []
    for check in mc.ALL_CHECKS:
        try:
            check(mod)
        except Exception as e:  # AssertionError or a crash both count as caught
            caught.append((check.__name__, type(e).__name__))
    assert caught, f"no pin fails for planted mistake {name}"
