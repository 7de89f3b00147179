"""Plausible mistakes planted in copies of the CPU reference (on the CPU)
must each fail at least one pin: evidence that the pins constrain every part
of the reference, not just its happy path."""

import importlib.util
import os
import types

import pytest

import oracle_checks as oc

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle", "tree_verify.py")

# (name, original text, mutated text)
MUTATIONS = [
    ("pack_never_shares", "            if t in children[cur]:\n", "            if False:\n"),
    ("pack_depth_cap_off_by_one", "            if pos >= max_depth:", "            if pos > max_depth:"),
    ("pack_budget_off_by_one", "            if len(token) >= max_nodes:", "            if len(token) > max_nodes:"),
    ("pack_truncation_uncounted", "                n_truncated += len(cand) - pos\n                break\n            node",
     "                break\n            node"),
    ("attn_scale_1_over_d", "    scale = 1.0 / math.sqrt(D)\n", "    scale = 1.0 / D\n"),
    ("attn_strided_gqa", "        heads = list(range(g * G, (g + 1) * G))", "        heads = list(range(g, Hq, n_kv_heads))"),
    ("attn_chain_without_self", "            rows = [P + j for j in chain(parent, i)]",
     "            rows = [P + j for j in chain(parent, i)[:-1]] or [P]"),
    ("attn_no_prefix_in_denominator", "                den = pp.sum() + pt.sum()", "                den = pt.sum()"),
    ("attn_row_uses_parent_chain", "    rows = list(range(prefix_len)) + [prefix_len + j for j in chain(parent, node)]",
     "    rows = list(range(prefix_len)) + [prefix_len + j for j in chain(parent, max(0, int(parent[node])))]"),
    ("argmax_last_on_tie", "    ids = np.argmax(logits, axis=1)  # first occurrence of the maximum",
     "    ids = logits.shape[1] - 1 - np.argmax(logits[:, ::-1], axis=1)"),
    ("lm_head_transposed_chunk", "        out[:, a:b] = x @ np.asarray(w[a:b], dtype=np.float64).T",
     "        out[:, a:b] = x @ np.asarray(w[a:b], dtype=np.float64).T[::-1].T[:, ::-1]"),
    ("walk_from_root_only", "    while int(ids[cur]) in children[cur]:\n        cur = children[cur][int(ids[cur])]",
     "    while int(ids[cur]) in children[0] and cur == 0:\n        cur = children[0][int(ids[cur])]"),
    ("bonus_from_parent", "    bonus = int(ids[path[-1]])", "    bonus = int(ids[path[-2] if len(path) > 1 else 0])"),
    ("compact_reverse_order", "        for src, dst in pairs:", "        for src, dst in reversed(pairs):"),
    ("hint_shortest_first", "    for n in range(min(max_suffix, len(committed)), 0, -1):",
     "    for n in range(1, min(max_suffix, len(committed)) + 1):"),
    ("hint_runs_through_eos", "            while k < len(bank) and bank[k] != eos and len(cont) < max_len:",
     "            while k < len(bank) and len(cont) < max_len:"),
    ("hint_duplicates_kept", "            if cont and cont not in found:", "            if cont:"),
    ("hint_skips_first_token", "            k = j + n\n", "            k = j + n + 1\n"),
    ("hint_suffix_shifted", "        suffix = committed[len(committed) - n:]",
     "        suffix = committed[max(0, len(committed) - n - 1):len(committed) - 1]"),
    ("hint_one_token_too_many", "and len(cont) < max_len:", "and len(cont) <= max_len:"),
    ("lanes_native_first", "    lanes = [list(h) for h in hints][:n_lanes]\n    for c in native:",
     "    lanes = [list(h) for h in native][:n_lanes]\n    for c in hints:"),
    ("step_accepts_on_own_tokens", "    acc = accept_walk(tree[\"token\"], tree[\"parent\"], greedy[\"ids\"])",
     "    acc = accept_walk(tree[\"token\"], tree[\"parent\"], tree[\"token\"])"),
    ("step_first_layer_only", "    outs = [tree_attention(q, k, v, prefix_len, tree[\"parent\"], n_kv_heads) for (q, k, v) in layers]",
     "    outs = [tree_attention(q, layers[0][1], v, prefix_len, tree[\"parent\"], n_kv_heads) for (q, k, v) in layers]"),
    ("step_logits_of_attention_input", "    logits = lm_head_logits(x, w)", "    logits = lm_head_logits(x[::-1], w)"),
    ("compact_dest_by_node", "    pairs = [(prefix_len + int(path[d]), prefix_len + d) for d in range(len(path))]",
     "    pairs = [(prefix_len + int(path[d]), prefix_len + int(path[d])) for d in range(len(path))]"),
]


def _mutant(name, old, new):
    with open(SRC) as f:
        text = f.read()
    assert text.count(old) == 1, f"mutation {name}: anchor text not found exactly once"
    mod = types.ModuleType(f"mutant_{name}")
    exec(compile(text.replace(old, new), f"<mutant {name}>", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_mutation_is_caught(name, old, new):
    mod = _mutant(name, old, new)
    caught = []
    for check in oc.ALL_CHECKS:
        try:
            check(mod)
        except Exception as e:  # AssertionError or a crash both count as caught
            caught.append((check.__name__, type(e).__name__))
    assert caught, f"no pin fails for planted mistake {name}"
