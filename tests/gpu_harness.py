"""Run verification steps on the GPU through the C ABI and compare them with
the CPU reference.  Used by the GPU parity tests and by the smoke check.

Tolerances: attention outputs and logits are compared per row as
max|gpu - ref| / max|ref| <= 1e-2 (bf16 inputs, float32 accumulation, bf16
outputs); every integer (trie arrays, greedy tokens, accepted length, path,
bonus, compacted cache rows) must match exactly.
"""

from __future__ import annotations

import math
import time
from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

from oracle import tree_verify as ov
from paper_2608_00814_amd import ooo
from paper_2608_00814_amd import workload as wl
from paper_2608_00814_amd.step import VerifyRunner

ATTN_TOL = 1e-2
LOGIT_TOL = 1e-2
MIN_MARGIN = 1e-2


def to_dev(arr: np.ndarray, dtype: str, device="cuda") -> torch.Tensor:
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).to(device)


def to_host(t: torch.Tensor, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def torch_dtype(dtype: str) -> torch.dtype:
    return torch.bfloat16 if dtype == "bf16" else torch.float32


def row_rel_err(g: np.ndarray, r: np.ndarray) -> float:
    """max over rows (last axis) of max|g - r| / max|r|."""
    g = np.asarray(g, dtype=np.float64).reshape(-1, g.shape[-1])
    r = np.asarray(r, dtype=np.float64).reshape(-1, r.shape[-1])
    num = np.abs(g - r).max(axis=1)
    den = np.maximum(np.abs(r).max(axis=1), 1e-30)
    return float((num / den).max())


def log(msg: str, verbose: bool) -> None:
    if verbose:
        print(msg, flush=True)


def run_and_check(name: str, seed: int = 0, layers: Optional[Sequence[int]] = None, step: int = 0,
                  sample_rows: int = 0, verbose: bool = False, check: bool = True) -> Dict:
    """One full verification step of workload ``name`` on cuda:0, checked
    against the reference.  ``layers`` limits the full attention comparison
    to those layers (None: all); ``sample_rows`` (node, head) rows of every
    other layer are checked one by one."""
    t0 = time.time()
    cfg = wl.CONFIGS[name]
    dt = cfg.dtype
    cands = wl.candidates_for(cfg, seed, step)
    tree = ov.pack_tree(cands.root_token, cands.seqs, cands.max_nodes, cands.max_depth)
    N = tree["n_nodes"]
    P = cfg.prefix_len
    tau, planted = wl.designated_tokens(cfg, seed, step, cands, tree["token"], tree["parent"])
    w = wl.lm_head_weight(cfg, seed)
    x = wl.hidden_rows(cfg, seed, step, w, tau, N)
    log(f"[{name} seed={seed}] inputs: N={N} P={P} planted={planted} ({time.time() - t0:.1f}s)", verbose)

    dev = torch.device("cuda:0")
    tdt = torch_dtype(dt)
    runner = VerifyRunner(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cfg.hidden, cfg.vocab,
                          cfg.max_nodes, cfg.max_depth, tdt, dev, max_prefix=P)
    toks, offs = cands.csr()
    packed = runner.pack(cands.root_token, toks, offs)
    if check:
        assert packed["n_nodes"] == N
        assert np.array_equal(packed["token"], tree["token"])
        assert np.array_equal(packed["parent"], tree["parent"])
        assert np.array_equal(packed["depth"], tree["depth"])
        assert packed["n_truncated"] == tree["n_truncated"]
        assert np.array_equal(packed["anc_mask"], ov.ancestor_masks(tree["parent"], cfg.mask_words))
    runner.ensure_workspace(P)

    shp = (cfg.n_layers, cfg.n_kv_heads, cfg.cap, cfg.head_dim)
    k_dev = torch.empty(shp, dtype=tdt, device=dev)
    v_dev = torch.empty(shp, dtype=tdt, device=dev)
    q_host: List[np.ndarray] = []
    cache_host = {}
    check_layers = list(range(cfg.n_layers)) if layers is None else list(layers)
    for l in range(cfg.n_layers):
        kc, vc = wl.layer_cache(cfg, seed, l, N, step)
        k_dev[l].copy_(to_dev(kc, dt, dev))
        v_dev[l].copy_(to_dev(vc, dt, dev))
        q_host.append(wl.queries(cfg, seed, step, l, N))
        if l in check_layers or sample_rows:
            cache_host[l] = (kc, vc)
    q_dev = [to_dev(q, dt, dev) for q in q_host]
    x_dev = to_dev(x, dt, dev)
    w_dev = to_dev(w, dt, dev)
    runner.set_weight(w_dev)
    logits_dev = torch.empty(N, cfg.vocab, dtype=torch.float32, device=dev)
    torch.cuda.synchronize()
    log(f"[{name}] uploaded ({time.time() - t0:.1f}s)", verbose)

    runner.device_step(q_dev, k_dev, v_dev, x_dev, P, logits=logits_dev, compact=True)
    torch.cuda.synchronize()
    res = runner.result()
    ids = runner.ids[:N].cpu().numpy()
    max_logit = runner.max_logit[:N].cpu().numpy()
    logits = logits_dev.cpu().numpy()
    log(f"[{name}] gpu step done: L={res.L} bonus={res.bonus} ({time.time() - t0:.1f}s)", verbose)
    out = {"n_nodes": N, "L": res.L, "bonus": res.bonus, "path": res.path, "planted": planted,
           "attn_rel": 0.0, "logit_rel": 0.0}
    if not check:
        return out

    # LM head and greedy tokens
    ref_logits = ov.lm_head_logits(wl.to_f64(x, dt), wl.to_f32(w, dt))
    g = ov.greedy_tokens(ref_logits)
    assert g["margin"].min() >= MIN_MARGIN, "input margin below the tie-exclusion bound"
    assert np.array_equal(ids, g["ids"]), (ids, g["ids"])
    out["logit_rel"] = row_rel_err(logits, ref_logits)
    assert out["logit_rel"] <= LOGIT_TOL, out["logit_rel"]
    assert np.all(np.abs(max_logit - g["max_logit"]) <= LOGIT_TOL * np.abs(ref_logits).max(axis=1))

    # accept
    acc = ov.accept_walk(tree["token"], tree["parent"], g["ids"])
    assert res.L == acc["L"] == planted, (res.L, acc["L"], planted)
    assert res.bonus == acc["bonus"]
    assert np.array_equal(res.path, acc["path"])
    full_path = runner.path.cpu().numpy()
    assert np.all(full_path[acc["L"] + 1:] == -1)

    # attention
    worst = 0.0
    rs = np.random.default_rng(seed + 1000)
    for l in range(cfg.n_layers):
        if l not in check_layers and not sample_rows:
            continue
        kc, vc = cache_host[l]
        k64, v64 = wl.to_f64(kc, dt), wl.to_f64(vc, dt)
        q64 = wl.to_f64(q_host[l], dt)
        got = wl.to_f64(to_host(runner.out[l, :N], dt), dt)
        if l in check_layers:
            ref = ov.tree_attention(q64, k64, v64, P, tree["parent"], cfg.n_kv_heads)
            e = row_rel_err(got, ref)
        else:
            e = 0.0
            for _ in range(sample_rows):
                i, h = int(rs.integers(0, N)), int(rs.integers(0, cfg.n_q_heads))
                ref = ov.attention_row(q64, k64, v64, P, tree["parent"], cfg.n_kv_heads, i, h)
                e = max(e, row_rel_err(got[i, h][None], ref[None]))
        worst = max(worst, e)
        assert e <= ATTN_TOL, (l, e)
    out["attn_rel"] = worst
    log(f"[{name}] attention checked, worst rel {worst:.2e} ({time.time() - t0:.1f}s)", verbose)

    # compaction: reference applied to the host copy of each checked layer
    for l in check_layers:
        kc, vc = cache_host[l]
        kr, vr = kc.copy(), vc.copy()
        ov.kv_compact([kr, vr], P, acc["path"])
        kg = to_host(k_dev[l], dt)
        vg = to_host(v_dev[l], dt)
        assert np.array_equal(kg, kr) and np.array_equal(vg, vr), f"compaction differs in layer {l}"
    log(f"[{name}] all checks passed ({time.time() - t0:.1f}s)", verbose)
    return out


def _par(fn, items):
    """Map fn over items on a thread pool (numpy releases the GIL while it draws)."""
    from concurrent.futures import ThreadPoolExecutor
    with ThreadPoolExecutor(8) as ex:
        return list(ex.map(fn, items))


def run_decode(name: str = "llama3.1-8b-decode", seed: int = 0, steps: Optional[int] = None,
               attn_steps: Sequence[int] = (0, 29, 30, 199), attn_layers: Sequence[int] = (0, 15, 31),
               sample_rows: int = 6, verbose: bool = False, graphs: bool = False) -> Dict:
    """Consecutive verification steps with compaction, each step's root the
    previous step's bonus token and the prefix growing by L+1.  Every step:
    the trie matches the reference packing, the greedy token of every node
    is the designated one (planted by construction), and L, path and bonus
    match the reference walk.  At ``attn_steps``: the LM head against the
    reference logits and sampled attention rows of ``attn_layers`` against
    the reference, with the committed prefix rebuilt from generator rows.
    At the end: the committed cache rows of ``attn_layers`` equal the
    prefix followed by the accepted nodes' rows, bit for bit."""
    t0 = time.time()
    cfg = wl.CONFIGS[name]
    dt = cfg.dtype
    steps = cfg.steps if steps is None else steps
    dev = torch.device("cuda:0")
    tdt = torch_dtype(dt)
    P = cfg.prefix_len
    runner = VerifyRunner(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cfg.hidden, cfg.vocab,
                          cfg.max_nodes, cfg.max_depth, tdt, dev, max_prefix=cfg.cap - cfg.max_nodes)
    w = wl.lm_head_weight(cfg, seed)
    runner.set_weight(to_dev(w, dt, dev))
    shp = (cfg.n_layers, cfg.n_kv_heads, cfg.cap, cfg.head_dim)
    k_dev = torch.zeros(shp, dtype=tdt, device=dev)
    v_dev = torch.zeros(shp, dtype=tdt, device=dev)
    exp_k: Dict[int, np.ndarray] = {}
    exp_v: Dict[int, np.ndarray] = {}

    def load_prefix(l):
        return l, wl.prefix_kv(cfg, seed, l)

    for l, (kp, vp) in _par(load_prefix, range(cfg.n_layers)):
        k_dev[l, :, :P].copy_(to_dev(kp, dt, dev))
        v_dev[l, :, :P].copy_(to_dev(vp, dt, dev))
        if l in attn_layers:
            exp_k[l] = np.zeros(shp[1:], dtype=kp.dtype)
            exp_v[l] = np.zeros(shp[1:], dtype=vp.dtype)
            exp_k[l][:, :P] = kp
            exp_v[l][:, :P] = vp
    torch.cuda.synchronize()
    log(f"[{name}] prefix of {P} rows uploaded ({time.time() - t0:.1f}s)", verbose)

    root = None
    total_tokens = 0
    worst_attn = worst_logit = 0.0
    rs = np.random.default_rng(seed + 2000)
    if graphs:
        # one captured step per trie size, replayed with the prefix length in
        # device memory; the step's inputs go to fixed buffers first
        bound = cfg.cap - cfg.max_nodes
        for n in range(1, cfg.max_nodes + 1):
            runner.ensure_workspace(bound, n)
        q_fix = [torch.empty(cfg.max_nodes, cfg.n_q_heads, cfg.head_dim, dtype=tdt, device=dev)
                 for _ in range(cfg.n_layers)]
        x_fix = torch.empty(cfg.max_nodes, cfg.hidden, dtype=tdt, device=dev)
        logits_fix = torch.empty(cfg.max_nodes, cfg.vocab, dtype=torch.float32, device=dev)
        captured: Dict[int, torch.cuda.CUDAGraph] = {}
        gstream = torch.cuda.Stream(device=dev)
    for step in range(steps):
        cands = wl.candidates_for(cfg, seed, step, root_token=root)
        tree = ov.pack_tree(cands.root_token, cands.seqs, cands.max_nodes, cands.max_depth)
        N = tree["n_nodes"]
        toks, offs = cands.csr()
        packed = runner.pack(cands.root_token, toks, offs)
        assert packed["n_nodes"] == N and packed["n_truncated"] == tree["n_truncated"], step
        assert np.array_equal(packed["token"], tree["token"]) and np.array_equal(packed["parent"], tree["parent"])
        tau, planted = wl.designated_tokens(cfg, seed, step, cands, tree["token"], tree["parent"])
        acc = ov.accept_walk(tree["token"], tree["parent"], tau)
        assert acc["L"] == planted, (step, acc["L"], planted)
        x = wl.hidden_rows(cfg, seed, step, w, tau, N)
        qs = _par(lambda l: wl.queries(cfg, seed, step, l, N), range(cfg.n_layers))
        kvs = _par(lambda l: wl.tree_kv(cfg, seed, step, l, N), range(cfg.n_layers))
        for l in range(cfg.n_layers):
            k_dev[l, :, P:P + N].copy_(to_dev(kvs[l][0], dt, dev))
            v_dev[l, :, P:P + N].copy_(to_dev(kvs[l][1], dt, dev))
        q_dev = [to_dev(q, dt, dev) for q in qs]
        check_now = step in attn_steps
        logits_dev = torch.empty(N, cfg.vocab, dtype=torch.float32, device=dev) if check_now else None
        if graphs:
            for l in range(cfg.n_layers):
                q_fix[l][:N].copy_(q_dev[l])
            x_fix[:N].copy_(to_dev(x, dt, dev))
            runner.set_prefix(P)
            torch.cuda.synchronize()
            with torch.cuda.stream(gstream):
                gr = captured.get(N)
                if gr is None:
                    gr = torch.cuda.CUDAGraph()
                    with torch.cuda.graph(gr, stream=gstream):
                        runner.device_step(q_fix, k_dev, v_dev, x_fix, bound, logits=logits_fix[:N], compact=True,
                                           prefix_dev=runner.prefix_dev)
                    captured[N] = gr
                gr.replay()
            torch.cuda.synchronize()
            if logits_dev is not None:
                logits_dev.copy_(logits_fix[:N])
        else:
            runner.ensure_workspace(P)
            runner.device_step(q_dev, k_dev, v_dev, to_dev(x, dt, dev), P, logits=logits_dev, compact=True)
        torch.cuda.synchronize()
        res = runner.result()
        ids = runner.ids[:N].cpu().numpy()
        assert np.array_equal(ids, tau.astype(np.int32)), f"step {step}: greedy tokens differ from the planted ones"
        assert res.L == acc["L"] and res.bonus == acc["bonus"], (step, res.L, acc["L"], res.bonus, acc["bonus"])
        assert np.array_equal(res.path, acc["path"]), step
        if check_now:
            ref_logits = ov.lm_head_logits(wl.to_f64(x, dt), wl.to_f32(w, dt))
            g = ov.greedy_tokens(ref_logits)
            assert g["margin"].min() >= MIN_MARGIN and np.array_equal(g["ids"], ids), step
            worst_logit = max(worst_logit, row_rel_err(logits_dev.cpu().numpy(), ref_logits))
            assert worst_logit <= LOGIT_TOL, (step, worst_logit)
            for l in attn_layers:
                k64 = wl.to_f64(exp_k[l][:, :P + N], dt)
                v64 = wl.to_f64(exp_v[l][:, :P + N], dt)
                k64[:, P:P + N] = wl.to_f64(kvs[l][0], dt)
                v64[:, P:P + N] = wl.to_f64(kvs[l][1], dt)
                q64 = wl.to_f64(qs[l], dt)
                got = wl.to_f64(to_host(runner.out[l, :N], dt), dt)
                for _ in range(sample_rows):
                    i, h = int(rs.integers(0, N)), int(rs.integers(0, cfg.n_q_heads))
                    ref = ov.attention_row(q64, k64, v64, P, tree["parent"], cfg.n_kv_heads, i, h)
                    e = row_rel_err(got[i, h][None], ref[None])
                    worst_attn = max(worst_attn, e)
                    assert e <= ATTN_TOL, (step, l, i, h, e)
            log(f"[{name}] step {step}: P={P} N={N} L={res.L} checked ({time.time() - t0:.1f}s)", verbose)
        # expected committed rows: accepted node at depth d lands in row P + d
        for l in attn_layers:
            for d, node in enumerate(acc["path"]):
                exp_k[l][:, P + d] = kvs[l][0][:, node]
                exp_v[l][:, P + d] = kvs[l][1][:, node]
        P += res.L + 1
        total_tokens += res.L + 1
        root = res.bonus
    for l in attn_layers:
        assert np.array_equal(to_host(k_dev[l, :, :P], dt), exp_k[l][:, :P]), f"committed K rows differ, layer {l}"
        assert np.array_equal(to_host(v_dev[l, :, :P], dt), exp_v[l][:, :P]), f"committed V rows differ, layer {l}"
    log(f"[{name}] {steps} steps, {total_tokens} tokens committed, final P={P} ({time.time() - t0:.1f}s)", verbose)
    return {"steps": steps, "tokens": total_tokens, "final_prefix": P, "attn_rel": worst_attn,
            "logit_rel": worst_logit}
