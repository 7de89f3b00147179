"""Decoder layers around the verification path on the GPU against the CPU
reference (``oracle/target_model.py``), through the C ABI.

Per-kernel parity (norms, projections, the rotation at P + depth with the
cache writes, the MLP activation, embedding rows) and whole verify steps of
a 2-layer model and of 2 layers at the Qwen3-8B decoder's sizes.  Float
outputs are compared per row (max abs error / max abs reference <= 1e-2);
greedy tokens, the accepted length, the path and the bonus token exactly on
nodes whose reference margin is at least 1e-2.
"""

from __future__ import annotations

import math

import numpy as np
import pytest
import torch

import gpu_harness as gh
from oracle import target_model as om
from oracle import tree_verify as ov
from paper_2608_00814_amd import model_workload as mw
from paper_2608_00814_amd import ooo
from paper_2608_00814_amd import workload as wl
from paper_2608_00814_amd.model import ModelRunner

pytestmark = pytest.mark.gpu
DEV = "cuda"
TOL = gh.ATTN_TOL
# fp32 outputs of the streaming projection: the stream-K partial sums pass
# through the workspace as fp16 (times a power of two per 32 rows), so each
# partial element carries a relative rounding error of at most 2^-11; over a
# row the error is at most 2^-11 * ||sum_s |p_s| || / ||sum_s p_s||, which is
# about 2^-11 * sqrt(S) for S independent partials (S <= 16 slots per tile
# at these shapes): 2e-3.  Measured: 3.6e-4 at N=64, K=4096, O=6144.
F32_OUT_TOL = 2e-3
f64 = wl.bf16_to_f64


def _bits(rs, shape, std=1.0):
    return wl.to_bf16_bits(rs.normal(0, std, size=shape).astype(np.float32))


def _dev_bf16(bits):
    return gh.to_dev(bits, "bf16", DEV)


def _host_f64(t):
    return f64(gh.to_host(t, "bf16"))


@pytest.mark.parametrize("N,H", [(1, 64), (37, 4096), (64, 5120)])
def test_rmsnorm(N, H):
    print(f"case rmsnorm N={N} H={H}", flush=True)
    rs = np.random.default_rng(N + H)
    h = (rs.normal(0, 3, size=(N, H))).astype(np.float32)
    w = _bits(rs, H, 0.3)
    out = torch.empty(N, H, dtype=torch.bfloat16, device=DEV)
    ooo.rmsnorm(torch.from_numpy(h).to(DEV), _dev_bf16(w), 1e-6, out)
    ref = om.rmsnorm(h.astype(np.float64), f64(w), 1e-6)
    assert gh.row_rel_err(_host_f64(out), ref) <= TOL


@pytest.mark.parametrize("N,K,O", [(64, 4096, 6144), (64, 4096, 4096), (37, 4096, 24576), (64, 12288, 4096),
                                   (1, 256, 1152), (5, 512, 256), (200, 1024, 3000), (33, 64, 130),
                                   (256, 512, 768), (129, 320, 512)])
@pytest.mark.parametrize("packed", [True, False], ids=["packed", "rows"])
def test_linear(N, K, O, packed):
    """Every epilogue of the streaming projection, both weight layouts, and
    bitwise-repeatable results."""
    print(f"case linear N={N} K={K} O={O} packed={packed}", flush=True)
    rs = np.random.default_rng(N + K + O)
    x, w = _bits(rs, (N, K)), _bits(rs, (O, K), 0.02)
    xd, wd = _dev_bf16(x), _dev_bf16(w)
    wl_ = ooo.linear_pack(wd) if packed else wd
    ref = f64(x) @ f64(w).T
    ws = torch.zeros(ooo.linear_workspace(N, K, O), dtype=torch.uint8, device=DEV)
    y32 = torch.full((N, O), float("nan"), dtype=torch.float32, device=DEV)
    ooo.linear(xd, wl_, y32, ooo.EPI_STORE_F32, ws)
    assert gh.row_rel_err(y32.double().cpu().numpy(), ref) <= F32_OUT_TOL
    again = torch.empty_like(y32)
    ooo.linear(xd, wl_, again, ooo.EPI_STORE_F32, ws)
    assert torch.equal(y32, again)
    y16 = torch.empty(N, O, dtype=torch.bfloat16, device=DEV)
    ooo.linear(xd, wl_, y16, ooo.EPI_STORE_BF16, ws)
    assert gh.row_rel_err(_host_f64(y16), ref) <= TOL
    base = rs.normal(size=(N, O)).astype(np.float32)
    acc = torch.from_numpy(base).to(DEV)
    ooo.linear(xd, wl_, acc, ooo.EPI_ADD_F32, ws)
    assert gh.row_rel_err(acc.double().cpu().numpy(), ref + base) <= F32_OUT_TOL
    if O % 256 == 0:
        I = O // 2
        act = torch.empty(N, I, dtype=torch.bfloat16, device=DEV)
        ooo.linear(xd, wl_, act, ooo.EPI_SWIGLU_BF16, ws)
        assert gh.row_rel_err(_host_f64(act), om.silu(ref[:, :I]) * ref[:, I:]) <= TOL
    torch.cuda.synchronize()


@pytest.mark.parametrize("scale", [3e4, 0.0])
def test_linear_partials_beyond_fp16_range(scale):
    """The stream-K partial sums pass through the workspace in fp16 with a
    power-of-two factor per 32 rows: sums far beyond fp16's largest value
    (65504) come back finite and within the fp32-output tolerance, and an
    all-zero weight gives exact zeros."""
    print(f"case linear partials scale={scale}", flush=True)
    N, K, O = 16, 4096, 256
    rs = np.random.default_rng(11)
    x = _bits(rs, (N, K), max(scale, 1.0))
    w = _bits(rs, (O, K), 1.0 if scale else 0.0)
    ref = f64(x) @ f64(w).T
    wp = ooo.linear_pack(_dev_bf16(w))
    ws = torch.zeros(ooo.linear_workspace(N, K, O), dtype=torch.uint8, device=DEV)
    y = torch.full((N, O), float("nan"), dtype=torch.float32, device=DEV)
    ooo.linear(_dev_bf16(x), wp, y, ooo.EPI_STORE_F32, ws)
    got = y.double().cpu().numpy()
    assert np.isfinite(got).all()
    if scale:
        assert np.abs(ref).max() > 1e6  # every 64-column partial exceeds fp16's range
        assert gh.row_rel_err(got, ref) <= F32_OUT_TOL
    else:
        assert (got == 0).all()


def test_linear_partials_keep_finite_rows_beside_an_infinite_one():
    """An infinite input in one node's row makes that row's outputs
    infinite or NaN; the other rows, whose partial sums share the fp16 scale
    of the same 32 output columns, stay finite and accurate."""
    print("case linear partials with an infinite row", flush=True)
    N, K, O = 8, 1024, 128
    rs = np.random.default_rng(12)
    x = _bits(rs, (N, K))
    w = _bits(rs, (O, K), 0.5)
    x[3, 5] = np.uint16(0x7F80)  # +inf in bf16
    wp = ooo.linear_pack(_dev_bf16(w))
    ws = torch.zeros(ooo.linear_workspace(N, K, O), dtype=torch.uint8, device=DEV)
    y = torch.full((N, O), float("nan"), dtype=torch.float32, device=DEV)
    ooo.linear(_dev_bf16(x), wp, y, ooo.EPI_STORE_F32, ws)
    got = y.double().cpu().numpy()
    assert not np.isfinite(got[3]).any()
    rows = [n for n in range(N) if n != 3]
    ref = f64(x[rows]) @ f64(w).T
    assert np.isfinite(got[rows]).all()
    assert gh.row_rel_err(got[rows], ref) <= F32_OUT_TOL


@pytest.mark.parametrize("N,K,O", [(64, 4096, 4096), (37, 12288, 4096), (1, 256, 256), (5, 512, 1024),
                                   (64, 1024, 8192)])
def test_linear_add_rmsnorm(N, K, O):
    """The projection added into the residual rows and the following RMSNorm
    in one call: the residual rows bitwise equal to ooo_linear's add
    epilogue, the normalised rows within tolerance of the reference."""
    print(f"case linear_add_rmsnorm N={N} K={K} O={O}", flush=True)
    rs = np.random.default_rng(N + K + O + 1)
    x, w = _bits(rs, (N, K)), _bits(rs, (O, K), 0.02)
    nw = wl.to_bf16_bits(1.0 + 0.2 * rs.normal(size=O).astype(np.float32))
    base = rs.normal(size=(N, O)).astype(np.float32)
    xd, wp = _dev_bf16(x), ooo.linear_pack(_dev_bf16(w))
    ws = torch.zeros(ooo.linear_workspace(N, K, O), dtype=torch.uint8, device=DEV)
    h_fused = torch.from_numpy(base).to(DEV)
    h_ref = h_fused.clone()
    out = torch.empty(N, O, dtype=torch.bfloat16, device=DEV)
    ooo.linear_add_rmsnorm(xd, wp, h_fused, _dev_bf16(nw), 1e-6, out, ws)
    ooo.linear(xd, wp, h_ref, ooo.EPI_ADD_F32, ws)
    torch.cuda.synchronize()
    assert torch.equal(h_fused, h_ref)
    ref_h = base.astype(np.float64) + f64(x) @ f64(w).T
    assert gh.row_rel_err(h_fused.double().cpu().numpy(), ref_h) <= F32_OUT_TOL
    assert gh.row_rel_err(_host_f64(out), om.rmsnorm(h_fused.double().cpu().numpy(), f64(nw), 1e-6)) <= TOL


@pytest.mark.parametrize("N,Hq,Hkv,D,P,bound", [(64, 32, 8, 128, 4096, None), (33, 4, 2, 64, 100, None),
                                                (1, 8, 2, 128, 0, None), (20, 16, 8, 128, 700, 2000)])
def test_linear_qk_norm_rope(N, Hq, Hkv, D, P, bound):
    """The q/k/v projection fused with the norms, the rotation at P + depth
    and the cache writes, against the reference layer's projection; with a
    device prefix below the bound when ``bound`` is set."""
    print(f"case linear_qk_norm_rope N={N} Hq={Hq} Hkv={Hkv} D={D} P={P} bound={bound}", flush=True)
    rs = np.random.default_rng(N + Hq + D + P + 3)
    H = 1024
    O = (Hq + 2 * Hkv) * D
    x, w = _bits(rs, (N, H)), _bits(rs, (O, H), 0.05)
    qn = wl.to_bf16_bits(1.0 + 0.2 * rs.normal(size=D).astype(np.float32))
    kn = wl.to_bf16_bits(1.0 + 0.2 * rs.normal(size=D).astype(np.float32))
    depth = rs.integers(0, 40, size=N).astype(np.int32)
    depth[0] = 0
    theta = 1.0e6
    cap = (bound if bound is not None else P) + N + 3
    kc = torch.full((Hkv, cap, D), 1.0, dtype=torch.bfloat16, device=DEV)
    vc = torch.full((Hkv, cap, D), 1.0, dtype=torch.bfloat16, device=DEV)
    q_out = torch.empty(N, Hq, D, dtype=torch.bfloat16, device=DEV)
    ws = torch.zeros(ooo.linear_workspace(N, H, O), dtype=torch.uint8, device=DEV)
    pdev = None if bound is None else torch.tensor([P], dtype=torch.int32, device=DEV)
    ooo.linear_qk_norm_rope(_dev_bf16(x), ooo.linear_pack(_dev_bf16(w)), _dev_bf16(qn), _dev_bf16(kn), 1e-6,
                            torch.from_numpy(depth).to(DEV), N, P if bound is None else bound, theta, Hq, Hkv,
                            q_out, kc, vc, ws, prefix_dev=pdev)
    torch.cuda.synchronize()
    lw = om.LayerWeights(in_norm=None, w_qkv=f64(w), q_norm=f64(qn), k_norm=f64(kn), w_o=None, post_norm=None,
                         w_gate=None, w_up=None, w_down=None)
    shp = om.ModelShape(hidden=H, n_q_heads=Hq, n_kv_heads=Hkv, head_dim=D, intermediate=0, rope_theta=theta)
    q_ref, k_ref, v_ref = om.project_qkv(f64(x), lw, shp, P + depth.astype(np.int64))
    assert gh.row_rel_err(_host_f64(q_out).reshape(N * Hq, D), q_ref.reshape(N * Hq, D)) <= TOL
    kh, vh = gh.to_host(kc, "bf16"), gh.to_host(vc, "bf16")
    assert gh.row_rel_err(f64(kh[:, P:P + N].transpose(1, 0, 2)).reshape(-1, D), k_ref.reshape(-1, D)) <= TOL
    assert gh.row_rel_err(f64(vh[:, P:P + N].transpose(1, 0, 2)).reshape(-1, D), v_ref.reshape(-1, D)) <= TOL
    sentinel = np.uint16(0x3F80)
    for arr in (kh, vh):
        assert (arr[:, :P] == sentinel).all() and (arr[:, P + N:] == sentinel).all()


def test_model_fused_matches_separate_calls():
    """The decoder with fused projection epilogues against the same decoder
    issued as separate calls: LM-head input rows within tolerance, equal
    greedy tokens where the reference margin allows, and the same accepted
    path."""
    print("case model fused vs separate calls (qwen3-8b-model, 2 layers)", flush=True)
    import dataclasses
    cfg = dataclasses.replace(mw.MODEL_CONFIGS["qwen3-8b-model"], n_layers=2)
    seed = 4
    lws, emb, fin, lm, _, _ = _model(cfg, seed, cfg.n_layers)
    kv = [mw.prefix_kv(cfg, seed, l) for l in range(cfg.n_layers)]
    toks = mw.random_tokens(cfg, seed, 80)
    cands = [toks[1:41], toks[41:53], toks[1:5] + toks[53:63], toks[63:75]]
    offs = np.zeros(len(cands) + 1, np.int32)
    offs[1:] = np.cumsum([len(c) for c in cands])
    flat = np.array([t for c in cands for t in c], np.int32)
    outs = []
    for fused in (True, False):
        runner = ModelRunner(cfg, lws, emb, fin, lm, DEV, fused=fused)
        kc = torch.stack([_dev_bf16(k) for k, _ in kv])
        vc = torch.stack([_dev_bf16(v) for _, v in kv])
        runner.pack(toks[0], flat, offs)
        logits = torch.empty(runner.vr.n_nodes, cfg.vocab, dtype=torch.float32, device=DEV)
        runner.device_step(kc, vc, cfg.prefix_len, logits=logits)
        torch.cuda.synchronize()
        outs.append((_host_f64(runner.xf[:runner.vr.n_nodes]), logits.cpu().numpy(), runner.result()))
        del runner, kc, vc
    (xa, la, ra), (xb, lb, rb) = outs
    assert gh.row_rel_err(xa, xb) <= TOL
    top = np.sort(lb, axis=1)
    safe = (top[:, -1] - top[:, -2]) >= 1e-2
    assert np.array_equal(la.argmax(1)[safe], lb.argmax(1)[safe])
    if safe[rb.path].all():
        assert ra.L == rb.L and np.array_equal(ra.path, rb.path) and ra.bonus == rb.bonus


@pytest.mark.parametrize("N,Hq,Hkv,D,P,norm", [(64, 32, 8, 128, 4096, True), (33, 4, 2, 64, 100, True),
                                                (7, 40, 8, 128, 8192, False), (1, 2, 1, 64, 0, True),
                                                (16, 8, 2, 128, 45000, True)])
def test_qk_norm_rope(N, Hq, Hkv, D, P, norm):
    """Queries, and the node keys/values in the cache rows P .. P + N - 1,
    match the reference norms and rotation at positions P + depth; every
    other cache row is left untouched."""
    print(f"case qk_norm_rope N={N} Hq={Hq} Hkv={Hkv} D={D} P={P} norm={norm}", flush=True)
    rs = np.random.default_rng(N + Hq + D + P)
    theta = 1.0e6
    qkv = _bits(rs, (N, (Hq + 2 * Hkv) * D))
    qn = kn = None
    if norm:
        qn = wl.to_bf16_bits(1.0 + 0.2 * rs.normal(size=D).astype(np.float32))
        kn = wl.to_bf16_bits(1.0 + 0.2 * rs.normal(size=D).astype(np.float32))
    depth = rs.integers(0, 50, size=N).astype(np.int32)
    depth[0] = 0
    cap = P + N + 5
    sentinel = np.uint16(0x3F80)  # 1.0
    kc = torch.full((Hkv, cap, D), 1.0, dtype=torch.bfloat16, device=DEV)
    vc = torch.full((Hkv, cap, D), 1.0, dtype=torch.bfloat16, device=DEV)
    q_out = torch.empty(N, Hq, D, dtype=torch.bfloat16, device=DEV)
    ooo.qk_norm_rope(_dev_bf16(qkv), _dev_bf16(qn) if norm else None, _dev_bf16(kn) if norm else None, 1e-6,
                     torch.from_numpy(depth).to(DEV), N, P, theta, Hq, Hkv, q_out, kc, vc)
    q = f64(qkv[:, :Hq * D]).reshape(N, Hq, D)
    k = f64(qkv[:, Hq * D:(Hq + Hkv) * D]).reshape(N, Hkv, D)
    if norm:
        q, k = om.rmsnorm(q, f64(qn), 1e-6), om.rmsnorm(k, f64(kn), 1e-6)
    pos = P + depth.astype(np.int64)
    q_ref, k_ref = om.rope(q, pos, theta), om.rope(k, pos, theta)
    assert gh.row_rel_err(_host_f64(q_out), q_ref) <= TOL
    kh, vh = gh.to_host(kc, "bf16"), gh.to_host(vc, "bf16")
    assert gh.row_rel_err(f64(kh[:, P:P + N].transpose(1, 0, 2)), k_ref) <= TOL
    assert np.array_equal(vh[:, P:P + N].transpose(1, 0, 2).reshape(N, -1), qkv[:, (Hq + Hkv) * D:])
    for arr in (kh, vh):
        assert (arr[:, :P] == sentinel).all() and (arr[:, P + N:] == sentinel).all()


def test_swiglu_and_embedding():
    print("case swiglu and embedding rows", flush=True)
    rs = np.random.default_rng(5)
    N, I, V, H = 19, 3072, 500, 1024
    gu = (rs.normal(0, 4, size=(N, 2 * I))).astype(np.float32)
    out = torch.empty(N, I, dtype=torch.bfloat16, device=DEV)
    ooo.swiglu(torch.from_numpy(gu).to(DEV), out)
    g, u = gu[:, :I].astype(np.float64), gu[:, I:].astype(np.float64)
    assert gh.row_rel_err(_host_f64(out), om.silu(g) * u) <= TOL
    table = _bits(rs, (V, H))
    toks = rs.integers(0, V, size=N).astype(np.int32)
    h = torch.empty(N, H, dtype=torch.float32, device=DEV)
    ooo.embed_rows(_dev_bf16(table), torch.from_numpy(toks).to(DEV), N, h)
    assert np.array_equal(h.cpu().numpy().astype(np.float64), f64(table[toks]))


# ----------------------------------------------------------------------------
# whole verify steps of the model


class _Widen:
    """A bf16 table that widens the rows it is indexed with."""

    def __init__(self, bits):
        self.bits = bits
        self.shape = bits.shape

    def __getitem__(self, idx):
        return f64(self.bits[idx])


def _model(cfg, seed, n_layers):
    lws = [mw.layer_weights(cfg, seed, l) for l in range(n_layers)]
    emb, fin, lm = mw.embedding(cfg, seed), mw.final_norm(cfg, seed), mw.lm_head(cfg, seed)
    ref_layers = [om.LayerWeights(**{k: f64(v) for k, v in lw.items()}) for lw in lws]
    shp = om.ModelShape(hidden=cfg.hidden, n_q_heads=cfg.n_q_heads, n_kv_heads=cfg.n_kv_heads,
                        head_dim=cfg.head_dim, intermediate=cfg.intermediate, rope_theta=cfg.rope_theta, eps=cfg.eps)
    return lws, emb, fin, lm, ref_layers, shp


def _greedy_chain(cfg, shp, ref_layers, emb, fin, lm, kcs, vcs, root, P, d):
    """The reference's own greedy continuation of length d + 1 after root
    (teacher-forced chains of growing length; caches are copied)."""
    chain = []
    for _ in range(d + 1):
        tree = ov.pack_tree(root, [chain] if chain else [], 64, 64)
        fw = om.forward_tree(tree["token"], tree["parent"], tree["depth"], P, _Widen(emb), ref_layers, f64(fin),
                             shp, [k.copy() for k in kcs], [v.copy() for v in vcs])
        g = ov.greedy_tokens(ov.lm_head_logits(fw["x"], _Widen(lm)))
        chain.append(int(g["ids"][-1]))
    return chain


@pytest.mark.parametrize("name,n_layers,depth", [("small-model", 2, 5), ("qwen3-8b-model", 2, 2)])
def test_model_verify_step(name, n_layers, depth):
    """Pack, all layers, LM head, accept and compact on the GPU against the
    reference step, with candidates that contain the reference's own greedy
    continuation for `depth` tokens (so exactly that many are accepted)."""
    print(f"case model verify step {name} layers={n_layers} depth={depth}", flush=True)
    base = mw.MODEL_CONFIGS[name]
    import dataclasses
    cfg = dataclasses.replace(base, n_layers=n_layers)
    seed = 3
    lws, emb, fin, lm, ref_layers, shp = _model(cfg, seed, n_layers)
    P = cfg.prefix_len
    kv = [mw.prefix_kv(cfg, seed, l) for l in range(n_layers)]
    kcs = [f64(k) for k, _ in kv]
    vcs = [f64(v) for _, v in kv]
    toks = mw.random_tokens(cfg, seed, 40)
    root = toks[0]
    chain = _greedy_chain(cfg, shp, ref_layers, emb, fin, lm, kcs, vcs, root, P, depth)
    wrong = (chain[depth] + 1) % cfg.vocab
    cands = [chain[:depth] + [wrong] + toks[1:4], toks[4:9], chain[:1] + toks[9:12], toks[12:15]]
    ref = om.verify_step(root, cands, cfg.max_nodes, cfg.max_depth, P, _Widen(emb), ref_layers, f64(fin), _Widen(lm),
                         shp, kcs, vcs)
    assert ref["L"] == depth
    # GPU
    runner = ModelRunner(cfg, lws, emb, fin, lm, DEV)
    kc = torch.stack([_dev_bf16(k) for k, _ in kv])
    vc = torch.stack([_dev_bf16(v) for _, v in kv])
    offs = np.zeros(len(cands) + 1, np.int32)
    for i, c in enumerate(cands):
        offs[i + 1] = offs[i] + len(c)
    flat = np.array([t for c in cands for t in c], np.int32)
    packed = runner.pack(root, flat, offs)
    N = packed["n_nodes"]
    assert N == ref["tree"]["n_nodes"] and np.array_equal(packed["token"], ref["tree"]["token"])
    logits = torch.empty(N, cfg.vocab, dtype=torch.float32, device=DEV)
    runner.device_step(kc, vc, P, logits=logits)
    torch.cuda.synchronize()
    res = runner.result()
    x_gpu = _host_f64(runner.xf[:N])
    assert gh.row_rel_err(x_gpu, ref["x"]) <= TOL
    ids = runner.vr.ids[:N].cpu().numpy()
    ok = ref["margin"] >= 1e-2
    assert ok[ref["path"]].all()
    assert np.array_equal(ids[ok], ref["ids"][ok])
    assert res.L == ref["L"] and res.bonus == ref["bonus"]
    assert np.array_equal(res.path, ref["path"])
    # the cache: prefix rows unchanged, rows P .. P + L hold the accepted
    # nodes' keys/values (bf16 rounding of the reference)
    for l in range(n_layers):
        kh = gh.to_host(kc[l], "bf16")
        vh = gh.to_host(vc[l], "bf16")
        assert np.array_equal(kh[:, :P], kv[l][0][:, :P]) and np.array_equal(vh[:, :P], kv[l][1][:, :P])
        rows = slice(P, P + ref["L"] + 1)
        assert gh.row_rel_err(f64(kh[:, rows]), kcs[l][:, rows]) <= TOL
        assert gh.row_rel_err(f64(vh[:, rows]), vcs[l][:, rows]) <= TOL


def test_model_chained_steps():
    """Three verify steps in a row on the 2-layer model, each compacting the
    accepted rows and moving the prefix on.  The GPU and the reference each
    keep their own cache and see the same candidates (built from the
    reference's own greedy continuation); the GPU commits exactly the
    reference's tokens at every step, and its cache rows stay within
    tolerance of the reference's."""
    print("case model chained verify steps", flush=True)
    import dataclasses
    cfg = dataclasses.replace(mw.MODEL_CONFIGS["small-model"], cap=160)
    seed = 5
    lws, emb, fin, lm, ref_layers, shp = _model(cfg, seed, cfg.n_layers)
    P = cfg.prefix_len
    kv = [mw.prefix_kv(cfg, seed, l) for l in range(cfg.n_layers)]
    kcs = [np.concatenate([f64(k), np.zeros((cfg.n_kv_heads, cfg.cap - k.shape[1], cfg.head_dim))], axis=1)
           if k.shape[1] < cfg.cap else f64(k) for k, _ in kv]
    vcs = [np.concatenate([f64(v), np.zeros((cfg.n_kv_heads, cfg.cap - v.shape[1], cfg.head_dim))], axis=1)
           if v.shape[1] < cfg.cap else f64(v) for _, v in kv]
    runner = ModelRunner(cfg, lws, emb, fin, lm, DEV)
    kc = torch.zeros(cfg.n_layers, cfg.n_kv_heads, cfg.cap, cfg.head_dim, dtype=torch.bfloat16, device=DEV)
    vc = torch.zeros_like(kc)
    for l, (k, v) in enumerate(kv):
        kc[l, :, :k.shape[1]] = _dev_bf16(k)
        vc[l, :, :v.shape[1]] = _dev_bf16(v)
    toks = mw.random_tokens(cfg, seed, 200)
    root = toks[0]
    for step, depth in enumerate([3, 0, 4]):
        chain = _greedy_chain(cfg, shp, ref_layers, emb, fin, lm, kcs, vcs, root, P, depth)
        wrong = (chain[depth] + 1) % cfg.vocab
        o = 10 * step
        # other lanes: random tokens whose first token is not the greedy one,
        # and (when depth >= 1) a lane sharing the greedy first token only
        other = [t if t != chain[0] else (t + 1) % cfg.vocab for t in toks[o + 3:o + 7]]
        cands = [chain[:depth] + [wrong] + toks[o + 1:o + 3], other]
        if depth >= 1:
            cands.append(chain[:1] + [(chain[1] + 2) % cfg.vocab] + toks[o + 7:o + 9])
        ref = om.verify_step(root, cands, cfg.max_nodes, cfg.max_depth, P, _Widen(emb), ref_layers, f64(fin),
                             _Widen(lm), shp, kcs, vcs)
        assert ref["L"] == depth
        offs = np.zeros(len(cands) + 1, np.int32)
        for i, c in enumerate(cands):
            offs[i + 1] = offs[i] + len(c)
        runner.pack(root, np.array([t for c in cands for t in c], np.int32), offs)
        runner.device_step(kc, vc, P)
        torch.cuda.synchronize()
        res = runner.result()
        assert res.L == ref["L"] and res.bonus == ref["bonus"], (step, res.L, ref["L"])
        assert np.array_equal(res.path, ref["path"])
        newP = P + res.L + 1
        for l in range(cfg.n_layers):
            kh, vh = gh.to_host(kc[l], "bf16"), gh.to_host(vc[l], "bf16")
            assert gh.row_rel_err(f64(kh[:, :newP]), kcs[l][:, :newP]) <= TOL
            assert gh.row_rel_err(f64(vh[:, :newP]), vcs[l][:, :newP]) <= TOL
        P = newP
        root = res.bonus
