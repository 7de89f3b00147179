"""Parity of the HIP path (called through the C ABI) with the CPU reference.

Integers must match exactly; attention outputs and logits within a per-row
relative error of 1e-2 (see gpu_harness).  Every case prints its name before
it touches the GPU.
"""

import math
import os

import numpy as np
import pytest
import torch

import gpu_harness as gh
from oracle import tree_verify as ov
from paper_2608_00814_amd import ooo
from paper_2608_00814_amd import workload as wl

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _bf16(x):
    return wl.to_bf16_bits(np.asarray(x, dtype=np.float32))


def _store(x, dt):
    return _bf16(x) if dt == "bf16" else np.asarray(x, dtype=np.float32)


# ----------------------------------------------------------------------------
# full verification steps of each workload


@pytest.mark.parametrize("seed", range(5))
def test_step_tiny_fp32(seed):
    print(f"case tiny-fp32 seed={seed}", flush=True)
    r = gh.run_and_check("tiny-fp32", seed=seed, verbose=True)
    assert r["L"] == 5


@pytest.mark.parametrize("seed", range(2))
def test_step_qwen3_0p6b(seed):
    print(f"case qwen3-0.6b seed={seed}", flush=True)
    gh.run_and_check("qwen3-0.6b", seed=seed, verbose=True)


def test_step_qwen3_8b():
    print("case qwen3-8b seed=0 (all 36 layers)", flush=True)
    gh.run_and_check("qwen3-8b", seed=0, verbose=True)


def test_step_qwen3_8b_second_seed_sampled():
    print("case qwen3-8b seed=1 (layers 0, 35 full; sampled rows elsewhere)", flush=True)
    gh.run_and_check("qwen3-8b", seed=1, layers=[0, 35], sample_rows=4, verbose=True)


def test_decode_llama31_8b_200_steps():
    """Llama-3.1-8B shape: 200 consecutive verify steps with compaction from a
    32768-row prefix (256-node tries, a hint branch from step 30)."""
    print("case decode llama3.1-8b 200 steps", flush=True)
    r = gh.run_decode("llama3.1-8b-decode", seed=0, verbose=True)
    assert r["steps"] == 200 and r["final_prefix"] == 32768 + r["tokens"]


def test_decode_llama31_8b_graph_replay_device_prefix():
    """The same steps with one captured graph per trie size replayed with the
    prefix length in device memory (what the decode loop and bench.py --loop
    do): 40 steps, across the hint branch's start at step 30."""
    print("case decode llama3.1-8b 40 steps, graphs + device prefix", flush=True)
    r = gh.run_decode("llama3.1-8b-decode", seed=1, steps=40, attn_steps=(0, 29, 30, 39), verbose=True, graphs=True)
    assert r["steps"] == 40 and r["final_prefix"] == 32768 + r["tokens"]


def test_step_qwen25_32b_sampled():
    print("case qwen2.5-32b seed=0 (layers 0, 63 full; sampled rows elsewhere)", flush=True)
    gh.run_and_check("qwen2.5-32b", seed=0, layers=[0, 63], sample_rows=4, verbose=True)


# ----------------------------------------------------------------------------
# attention edge sweep


def _trie(kind, N, rs, vocab=50000):
    if kind == "chain":
        cands = [list(range(1, N))]
    elif kind == "star":
        cands = [[i] for i in range(1, N)]
    elif kind == "deep":
        spine = list(range(1, N))
        cands = [spine] + [spine[:int(rs.integers(0, N - 1))] + [vocab + i] for i in range(N)]
    else:
        cands = [[int(t) for t in rs.integers(0, 3, size=int(rs.integers(1, 40)))] for _ in range(4 * N)]
    t = ov.pack_tree(0, cands, N, 10 ** 6)
    assert t["n_nodes"] == N, (kind, t["n_nodes"], N)
    return t


ATTN_CASES = [
    # (P, N, G, Hkv, D, kind, dtype)
    (0, 1, 1, 1, 64, "chain", "bf16"),
    (1, 2, 2, 1, 128, "chain", "bf16"),
    (63, 25, 4, 1, 64, "random", "bf16"),
    (64, 63, 4, 2, 128, "random", "bf16"),
    (65, 64, 5, 2, 128, "star", "bf16"),
    (1000, 65, 8, 1, 128, "random", "bf16"),
    (4097, 128, 5, 2, 128, "deep", "bf16"),
    (130, 256, 4, 2, 64, "random", "bf16"),
    (0, 256, 1, 2, 128, "chain", "bf16"),
    (64, 1, 8, 4, 128, "chain", "bf16"),
    (0, 64, 2, 1, 64, "star", "bf16"),
    (200, 200, 3, 3, 128, "random", "bf16"),
    (4096, 64, 4, 8, 128, "random", "bf16"),
    (77, 300, 2, 1, 64, "random", "bf16"),
    (500, 40, 16, 1, 128, "random", "bf16"),
    (100, 9, 12, 2, 64, "deep", "bf16"),
    # the largest tries the boundary takes (16 ancestor-mask words)
    (100, 1024, 1, 1, 64, "random", "bf16"),
    (37, 700, 2, 1, 128, "deep", "bf16"),
    (128, 25, 4, 1, 64, "random", "f32"),
    (1, 40, 2, 2, 128, "deep", "f32"),
    (0, 3, 1, 1, 64, "star", "f32"),
    (3000, 70, 4, 2, 128, "random", "f32"),
    (255, 2, 2, 1, 64, "chain", "f32"),
    (10, 1000, 1, 1, 64, "random", "f32"),
]


def _attn_inputs(P, N, G, Hkv, D, dt, seed, pad=3):
    rs = np.random.default_rng(seed)
    Hq = G * Hkv
    cap = P + N + pad
    q = _store(rs.normal(size=(N, Hq, D)), dt)
    k = _store(rs.normal(size=(Hkv, cap, D)), dt)
    v = _store(rs.normal(size=(Hkv, cap, D)), dt)
    return rs, q, k, v, cap


def _run_attn(q, k, v, P, N, mask, Hq, Hkv, D, dt, force_splits=0, variant=0):
    tdt = gh.torch_dtype(dt)
    code = ooo.BF16 if dt == "bf16" else ooo.F32
    qd, kd, vd = gh.to_dev(q, dt, DEV), gh.to_dev(k, dt, DEV), gh.to_dev(v, dt, DEV)
    md = torch.from_numpy(mask.view(np.int64)).to(DEV)
    out = torch.full((N, Hq, D), float("nan"), dtype=tdt, device=DEV)
    ws_n = ooo.tree_attn_workspace(N, Hq, Hkv, D, P, code, force_splits)
    ws = torch.zeros(max(ws_n, 4) // 4 + 1, dtype=torch.float32, device=DEV)
    ooo.tree_attn(qd, kd, vd, P, N, md, Hq, Hkv, 1.0 / math.sqrt(D), out, ws, force_splits=force_splits,
                  variant=variant)
    torch.cuda.synchronize()
    return gh.wl.to_f64(gh.to_host(out, dt), dt)


@pytest.mark.parametrize("case", ATTN_CASES, ids=[f"P{c[0]}-N{c[1]}-G{c[2]}-Hkv{c[3]}-D{c[4]}-{c[5]}-{c[6]}"
                                                   for c in ATTN_CASES])
def test_attention_edges(case):
    P, N, G, Hkv, D, kind, dt = case
    print(f"case attention {case}", flush=True)
    rs, q, k, v, cap = _attn_inputs(P, N, G, Hkv, D, dt, seed=sum(case[:5]))
    t = _trie(kind, N, rs)
    W = (N + 63) // 64
    mask = ov.ancestor_masks(t["parent"], W)
    got = _run_attn(q, k, v, P, N, mask, G * Hkv, Hkv, D, dt)
    ref = ov.tree_attention(wl.to_f64(q, dt), wl.to_f64(k, dt), wl.to_f64(v, dt), P, t["parent"], Hkv)
    tol = gh.ATTN_TOL if dt == "bf16" else 1e-5
    assert gh.row_rel_err(got, ref) <= tol


ONE_WAVE_CASES = [c for c in ATTN_CASES if c[4] == 128 and c[6] == "bf16"][:6]


@pytest.mark.parametrize("case", ONE_WAVE_CASES, ids=[f"P{c[0]}-N{c[1]}-G{c[2]}-Hkv{c[3]}-{c[5]}"
                                                      for c in ONE_WAVE_CASES])
def test_attention_one_wave_kernel(case):
    """head_dim 128 has two kernels (two waves per row group splitting each
    key tile, the default, and one wave per row group); both match the
    oracle."""
    P, N, G, Hkv, D, kind, dt = case
    print(f"case attention one-wave kernel {case}", flush=True)
    rs, q, k, v, cap = _attn_inputs(P, N, G, Hkv, D, dt, seed=sum(case[:5]) + 1)
    t = _trie(kind, N, rs)
    mask = ov.ancestor_masks(t["parent"], (N + 63) // 64)
    got = _run_attn(q, k, v, P, N, mask, G * Hkv, Hkv, D, dt, variant=1)
    ref = ov.tree_attention(wl.to_f64(q, dt), wl.to_f64(k, dt), wl.to_f64(v, dt), P, t["parent"], Hkv)
    assert gh.row_rel_err(got, ref) <= gh.ATTN_TOL


@pytest.mark.parametrize("splits", [1, 3, 32])
def test_attention_split_counts_agree(splits):
    """The split-KV decomposition does not change the result beyond rounding,
    and each setting is bitwise reproducible."""
    print(f"case attention splits={splits}", flush=True)
    P, N, G, Hkv, D = 1500, 64, 4, 2, 128
    rs, q, k, v, cap = _attn_inputs(P, N, G, Hkv, D, "bf16", seed=7)
    t = _trie("random", N, rs)
    mask = ov.ancestor_masks(t["parent"], 1)
    a = _run_attn(q, k, v, P, N, mask, G * Hkv, Hkv, D, "bf16", force_splits=splits)
    b = _run_attn(q, k, v, P, N, mask, G * Hkv, Hkv, D, "bf16", force_splits=splits)
    assert np.array_equal(a, b)
    ref = ov.tree_attention(wl.to_f64(q, "bf16"), wl.to_f64(k, "bf16"), wl.to_f64(v, "bf16"), P, t["parent"], Hkv)
    assert gh.row_rel_err(a, ref) <= gh.ATTN_TOL


# (P, N, G, Hkv, D, splits, variant): a split whose first key tile crosses
# the end of the prefix (the last prefix tile is partly masked) and which
# goes on to further tiles, in the key-split kernel (variant 0) and the
# one-wave kernel (variant 1 at head_dim 128, and head_dim 64)
BOUNDARY_SPLITS = [
    (150, 64, 4, 2, 128, 2, 0),   # tiles [0,1] [2,3]: split 1 starts at tile 2 (rows 128..191, prefix 150)
    (150, 64, 4, 2, 128, 2, 1),
    (190, 130, 4, 1, 128, 3, 0),  # tiles [0,1] [2,3] [4,5]: 3 mask words, the last tree tile partial too
    (190, 130, 2, 2, 64, 3, 0),
]


@pytest.mark.parametrize("case", BOUNDARY_SPLITS, ids=[f"P{c[0]}-N{c[1]}-G{c[2]}-Hkv{c[3]}-D{c[4]}-S{c[5]}-v{c[6]}"
                                                       for c in BOUNDARY_SPLITS])
def test_attention_split_starting_at_a_boundary_tile(case):
    P, N, G, Hkv, D, splits, variant = case
    print(f"case attention boundary split {case}", flush=True)
    rs, q, k, v, cap = _attn_inputs(P, N, G, Hkv, D, "bf16", seed=P * N + splits)
    t = _trie("random", N, rs)
    W = (N + 63) // 64
    mask = ov.ancestor_masks(t["parent"], W)
    got = _run_attn(q, k, v, P, N, mask, G * Hkv, Hkv, D, "bf16", force_splits=splits, variant=variant)
    ref = ov.tree_attention(wl.to_f64(q, "bf16"), wl.to_f64(k, "bf16"), wl.to_f64(v, "bf16"), P, t["parent"], Hkv)
    assert gh.row_rel_err(got, ref) <= gh.ATTN_TOL


def test_attention_workspace_reuse_across_shapes():
    """One workspace serves calls of different shapes, head sizes and split
    counts in a row: nothing a call reads from it is left over from another
    (the workspace starts out as NaN)."""
    print("case attention workspace reuse", flush=True)
    shapes = [(1500, 64, 4, 2, 128, 16), (300, 33, 2, 3, 64, 5), (4096, 64, 4, 8, 128, 16), (700, 100, 4, 1, 128, 7),
              (4096, 64, 4, 8, 128, 13)]
    need = 0
    for P, N, G, Hkv, D, splits in shapes:
        need = max(need, ooo.tree_attn_workspace(N, G * Hkv, Hkv, D, P, ooo.BF16, splits))
    ws = torch.full((need // 4 + 1,), float("nan"), dtype=torch.float32, device=DEV)
    for P, N, G, Hkv, D, splits in shapes:
        rs, q, k, v, cap = _attn_inputs(P, N, G, Hkv, D, "bf16", seed=P + N)
        t = _trie("random", N, rs)
        W = (N + 63) // 64
        mask = ov.ancestor_masks(t["parent"], W)
        qd, kd, vd = gh.to_dev(q, "bf16", DEV), gh.to_dev(k, "bf16", DEV), gh.to_dev(v, "bf16", DEV)
        md = torch.from_numpy(mask.view(np.int64)).to(DEV)
        out = torch.full((N, G * Hkv, D), float("nan"), dtype=torch.bfloat16, device=DEV)
        ooo.tree_attn(qd, kd, vd, P, N, md, G * Hkv, Hkv, 1.0 / math.sqrt(D), out, ws, force_splits=splits)
        torch.cuda.synchronize()
        got = gh.wl.to_f64(gh.to_host(out, "bf16"), "bf16")
        ref = ov.tree_attention(wl.to_f64(q, "bf16"), wl.to_f64(k, "bf16"), wl.to_f64(v, "bf16"), P, t["parent"], Hkv)
        assert gh.row_rel_err(got, ref) <= gh.ATTN_TOL


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_attention_ignores_rows_outside_prefix_and_tree(dt):
    """Cache rows at and beyond P + N hold NaN; the output must not see
    them."""
    print(f"case attention NaN rows {dt}", flush=True)
    P, N, G, Hkv, D = 100, 20, 4, 2, 128
    rs, q, k, v, cap = _attn_inputs(P, N, G, Hkv, D, dt, seed=11, pad=300)
    nan = np.uint16(0x7FC0) if dt == "bf16" else np.float32("nan")
    k[:, P + N:] = nan
    v[:, P + N:] = nan
    t = _trie("chain", N, rs)
    mask = ov.ancestor_masks(t["parent"], 1)
    got = _run_attn(q, k, v, P, N, mask, G * Hkv, Hkv, D, dt)
    assert np.isfinite(got).all()
    ref = ov.tree_attention(wl.to_f64(q, dt), wl.to_f64(k, dt), wl.to_f64(v, dt), P, t["parent"], Hkv)
    assert gh.row_rel_err(got, ref) <= gh.ATTN_TOL


# ----------------------------------------------------------------------------
# LM head


LM_CASES = [
    # (N, H, V, dtype)
    (1, 64, 1000, "bf16"),
    (31, 256, 4097, "bf16"),
    (32, 1024, 151936, "bf16"),
    (33, 128, 5000, "bf16"),
    (64, 4096, 151936, "bf16"),
    (65, 192, 3001, "bf16"),
    (128, 512, 9999, "bf16"),
    (129, 64, 1000, "bf16"),
    (256, 256, 20000, "bf16"),
    # more 128-row tiles than compute units with a partial last round: some
    # blocks' last tile has only some of its 32-row groups (wide node tiles
    # give a wave two groups, of which one, both or neither may be empty)
    (128, 128, 40000, "bf16"),
    (200, 64, 35000, "bf16"),
    (256, 64, 70000, "bf16"),
    (25, 256, 1024, "f32"),
    (3, 100, 777, "f32"),
]


def _run_lm(x, w, dt, want_logits=True, packed=False):
    N, H = x.shape
    V = w.shape[0]
    code = ooo.BF16 if dt == "bf16" else ooo.F32
    xd, wd = gh.to_dev(x, dt, DEV), gh.to_dev(w, dt, DEV)
    if packed:
        wd = ooo.lmhead_pack(wd)
    ids = torch.full((N,), -7, dtype=torch.int32, device=DEV)
    mx = torch.empty(N, dtype=torch.float32, device=DEV)
    lg = torch.empty(N, V, dtype=torch.float32, device=DEV) if want_logits else None
    ws = torch.empty(ooo.lmhead_workspace(N, H, V, code) // 4 + 1, dtype=torch.float32, device=DEV)
    ooo.lmhead_argmax(xd, wd, ids, mx, lg, ws)
    torch.cuda.synchronize()
    return ids.cpu().numpy(), mx.cpu().numpy(), (lg.cpu().numpy() if want_logits else None)


LM_RUNS = [(c, False) for c in LM_CASES] + [(c, True) for c in LM_CASES if c[3] == "bf16"]


@pytest.mark.parametrize("case,packed", LM_RUNS,
                         ids=[f"N{c[0]}-H{c[1]}-V{c[2]}-{c[3]}{'-packed' if p else ''}" for c, p in LM_RUNS])
def test_lmhead_edges(case, packed):
    N, H, V, dt = case
    print(f"case lmhead {case} packed={packed}", flush=True)
    rs = np.random.default_rng(N * 7 + H + V)
    x = _store(rs.normal(size=(N, H)), dt)
    # logit spread of about one unit so most nodes clear the tie-exclusion margin
    w = _store(rs.normal(size=(V, H)) * max(0.02, 1.0 / math.sqrt(H)), dt)
    ids, mx, lg = _run_lm(x, w, dt, packed=packed)
    ref = ov.lm_head_logits(wl.to_f64(x, dt), wl.to_f64(w, dt))
    g = ov.greedy_tokens(ref)
    tol = gh.LOGIT_TOL if dt == "bf16" else 1e-5
    assert gh.row_rel_err(lg, ref) <= tol
    clear = g["margin"] >= gh.MIN_MARGIN  # ties excluded by the margin bound
    assert clear.sum() >= 0.7 * N
    assert np.array_equal(ids[clear], g["ids"][clear])
    assert np.allclose(mx[clear], g["max_logit"][clear], rtol=1e-3, atol=1e-3)


@pytest.mark.parametrize("packed", [False, True])
def test_lmhead_exact_ties_go_to_lowest_index(packed):
    """Identical weight rows in different blocks give identical logits; the
    lowest vocabulary index must win for every node."""
    print(f"case lmhead ties packed={packed}", flush=True)
    N, H, V = 64, 256, 70001
    rs = np.random.default_rng(5)
    x = _bf16(rs.normal(size=(N, H)))
    w = _bf16(rs.normal(size=(V, H)) * 0.02)
    xf = wl.to_f64(x, "bf16")
    for n in range(N):
        # make rows a < b < c identical and dominant for node n
        a, b, c = sorted(rs.choice(V, size=3, replace=False).tolist())
        row = _bf16(xf[n] * 0.05)
        w[a] = w[b] = w[c] = row
    ids, mx, _ = _run_lm(x, w, "bf16", want_logits=False, packed=packed)
    ref = ov.greedy_tokens(ov.lm_head_logits(xf, wl.to_f64(w, "bf16")))
    # the reference breaks exact ties to the lowest index too
    assert np.array_equal(ids, ref["ids"])


@pytest.mark.parametrize("V,H", [(1000, 64), (128, 128), (300, 192)])
def test_lmhead_pack_layout(V, H):
    """The packed weight is a pure re-layout: tile t, chunk kc, row r and
    physical 16-byte piece p hold columns kc*64 + 8*(p ^ (r//2)%8) .. +8 of row
    t*128 + r, and rows past the vocabulary are zero."""
    print(f"case lmhead pack V={V} H={H}", flush=True)
    rs = np.random.default_rng(V + H)
    w = _bf16(rs.normal(size=(V, H)))
    pw = ooo.lmhead_pack(gh.to_dev(w, "bf16", DEV))
    torch.cuda.synchronize()
    got = pw.data.cpu().numpy().view(np.uint16)
    T, C = (V + 127) // 128, H // 64
    full = np.zeros((T * 128, H), np.uint16)
    full[:V] = w  # bf16 bit patterns
    want = np.empty((T, C, 128, 8, 8), np.uint16)
    for r in range(128):
        for p in range(8):
            q = p ^ ((r // 2) % 8)
            for kc in range(C):
                want[:, kc, r, p, :] = full[r::128][:T, kc * 64 + 8 * q:kc * 64 + 8 * q + 8]
    assert np.array_equal(got, want.reshape(-1))


@pytest.mark.parametrize("O,K", [(384, 64), (300, 192)])
def test_linear_pack_layout(O, K):
    """The packed projection weight is a pure re-layout: tile t, chunk kc,
    row r and physical 16-byte piece p hold columns kc*64 + 8*(p ^ (r//2)%8) .. +8
    of row t*128 + r, and rows past out_dim are zero."""
    print(f"case linear pack O={O} K={K}", flush=True)
    rs = np.random.default_rng(O + K)
    w = _bf16(rs.normal(size=(O, K)))
    pw = ooo.linear_pack(gh.to_dev(w, "bf16", DEV))
    torch.cuda.synchronize()
    got = pw.data.cpu().numpy().view(np.uint16)
    T, C = (O + 127) // 128, K // 64
    full = np.zeros((T * 128, K), np.uint16)
    full[:O] = w
    want = np.empty((T, C, 128, 8, 8), np.uint16)
    for r in range(128):
        for p in range(8):
            q = p ^ ((r // 2) % 8)
            for kc in range(C):
                want[:, kc, r, p, :] = full[r::128][:T, kc * 64 + 8 * q:kc * 64 + 8 * q + 8]
    assert np.array_equal(got, want.reshape(-1))


# ----------------------------------------------------------------------------
# accept and compact


def _upload_trie(t, W):
    N = t["n_nodes"]
    to = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(DEV)
    mask = torch.from_numpy(ov.ancestor_masks(t["parent"], W).view(np.int64)).to(DEV)
    return to(t["token"]), to(t["parent"]), to(t["depth"]), mask


@pytest.mark.parametrize("N,kind,target", [
    (1, "chain", "max"), (2, "chain", 0), (25, "random", 1), (64, "chain", "max"), (65, "deep", "leaf"),
    (128, "random", "max"), (256, "star", 1), (256, "deep", "max"), (1024, "random", "leaf"), (1000, "chain", 0),
])
def test_accept_planted(N, kind, target):
    print(f"case accept N={N} {kind} target={target}", flush=True)
    rs = np.random.default_rng(N)
    t = _trie(kind, N, rs)
    parent, token, depth = t["parent"], t["token"], t["depth"]
    children = [[] for _ in range(N)]
    for i in range(1, N):
        children[parent[i]].append(i)
    # choose a root path to plant
    path = [0]
    while children[path[-1]]:
        path.append(children[path[-1]][int(rs.integers(0, len(children[path[-1]])))])
    if target == "max" or target == "leaf":
        d = len(path) - 1
    else:
        d = min(int(target), len(path) - 1)
    ids = np.empty(N, np.int32)
    for i in range(N):
        ch = [int(token[c]) for c in children[i]]
        # islands: half the off-path nodes match one of their children
        ids[i] = ch[int(rs.integers(0, len(ch)))] if (ch and rs.random() < 0.5) else 10 ** 6 + i
    for k in range(len(path)):
        ids[path[k]] = token[path[k + 1]] if k < d else 10 ** 6 + 7
    W = (N + 63) // 64
    tok_d, par_d, dep_d, mask_d = _upload_trie(t, W)
    ids_d = torch.from_numpy(ids).to(DEV)
    cap = int(depth.max()) + 1
    pth = torch.full((cap,), 99, dtype=torch.int32, device=DEV)
    L = torch.full((1,), -5, dtype=torch.int32, device=DEV)
    bonus = torch.full((1,), -5, dtype=torch.int32, device=DEV)
    ooo.accept(tok_d, par_d, dep_d, mask_d, ids_d, N, pth, L, bonus)
    torch.cuda.synchronize()
    ref = ov.accept_walk(token, parent, ids)
    assert ref["L"] == d
    assert int(L.item()) == ref["L"] and int(bonus.item()) == ref["bonus"]
    p = pth.cpu().numpy()
    assert np.array_equal(p[:d + 1], ref["path"]) and np.all(p[d + 1:] == -1)


@pytest.mark.parametrize("planted", [3, 10])
def test_accept_reports_a_path_deeper_than_declared(planted):
    """A chain of depth 10 verified with a path buffer of 5 entries (declared
    max_depth 4): an accepted path that fits is returned as usual; one that
    runs deeper is reported (accept_len -1, path all -1) rather than
    shortened, and compaction then moves no row."""
    print(f"case accept overflow planted={planted}", flush=True)
    N = 11
    rs = np.random.default_rng(5)
    t = _trie("chain", N, rs)
    token = t["token"]
    ids = np.full(N, 10 ** 6, np.int32)
    for k in range(planted):
        ids[k] = token[k + 1]
    tok_d, par_d, dep_d, mask_d = _upload_trie(t, 1)
    ids_d = torch.from_numpy(ids).to(DEV)
    pth = torch.full((5,), 99, dtype=torch.int32, device=DEV)
    L = torch.full((1,), -5, dtype=torch.int32, device=DEV)
    bonus = torch.full((1,), -5, dtype=torch.int32, device=DEV)
    ooo.accept(tok_d, par_d, dep_d, mask_d, ids_d, N, pth, L, bonus, max_depth=4)
    P, Hkv, D = 7, 2, 64
    cache = torch.randn(2, 1, Hkv, P + N + 1, D, device=DEV).to(torch.bfloat16)
    before = cache.clone()
    ooo.kv_compact(cache[0], cache[1], P, N, pth, L)
    torch.cuda.synchronize()
    if planted <= 4:
        ref = ov.accept_walk(token, t["parent"], ids)
        assert int(L.item()) == ref["L"] == planted and int(bonus.item()) == ref["bonus"]
        assert pth.cpu().numpy()[:planted + 1].tolist() == list(range(planted + 1))
    else:
        assert int(L.item()) == -1 and int(bonus.item()) == -1
        assert (pth.cpu().numpy() == -1).all()
        assert torch.equal(cache, before)


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("path", [[0], [0, 2, 3], [0, 1, 5, 6], [0, 1, 2, 3, 4], list(range(0, 130, 2)),
                                  [0, 9, 10, 11, 40, 41, 63]])
def test_compact_hazards(path, dt):
    print(f"case compact {dt} path={path[:8]}... len={len(path)}", flush=True)
    rs = np.random.default_rng(len(path))
    Lm, Hkv, D, P = 3, 2, 128, 37
    N = max(path) + 1 + 5
    cap = P + N + 4
    k = _store(rs.normal(size=(Lm, Hkv, cap, D)), dt)
    v = _store(rs.normal(size=(Lm, Hkv, cap, D)), dt)
    kd, vd = gh.to_dev(k, dt, DEV), gh.to_dev(v, dt, DEV)
    pcap = len(path) + 3
    pth = torch.tensor(path + [-1] * 3, dtype=torch.int32, device=DEV)
    Ld = torch.tensor([len(path) - 1], dtype=torch.int32, device=DEV)
    ooo.kv_compact(kd, vd, P, N, pth, Ld)
    torch.cuda.synchronize()
    kr, vr = k.copy(), v.copy()
    ov.kv_compact([kr, vr], P, np.array(path))
    assert np.array_equal(gh.to_host(kd, dt), kr)
    assert np.array_equal(gh.to_host(vd, dt), vr)
    assert pcap > 0


# ----------------------------------------------------------------------------
# determinism


def test_step_is_bitwise_reproducible():
    print("case determinism qwen3-0.6b", flush=True)
    cfg = wl.CONFIGS["qwen3-0.6b"]
    outs = []
    for _ in range(2):
        P, N, G, Hkv, D = cfg.prefix_len, 32, cfg.group, cfg.n_kv_heads, cfg.head_dim
        rs, q, k, v, cap = _attn_inputs(P, N, G, Hkv, D, "bf16", seed=3)
        t = _trie("random", N, rs)
        a = _run_attn(q, k, v, P, N, ov.ancestor_masks(t["parent"], 1), G * Hkv, Hkv, D, "bf16")
        x = _bf16(rs.normal(size=(N, 1024)))
        w = _bf16(rs.normal(size=(20000, 1024)) * 0.02)
        ids, mx, lg = _run_lm(x, w, "bf16")
        outs.append((a, ids, mx, lg))
    for u, w_ in zip(outs[0], outs[1]):
        assert np.array_equal(u, w_)
