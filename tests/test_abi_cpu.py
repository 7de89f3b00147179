"""The C ABI on the CPU: the library loads, exports exactly what
include/ooo.h declares, packs tries identically to the CPU reference, and
rejects bad arguments before touching a device."""

import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

import oracle_checks as oc
from oracle import tree_verify as ov
from paper_2608_00814_amd import ooo
from paper_2608_00814_amd import workload as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ooo.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ooo_[a-z_0-9]+)\s*\(", text)))


def test_exports_match_header():
    names = declared_functions()
    assert len(names) == 26
    assert set(names) == set(ooo.SIGNATURES)
    lib = ooo.lib()
    for n in names:
        assert getattr(lib, n) is not None
    out = subprocess.run(["nm", "-D", "--defined-only", ooo.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    exported = set(re.findall(r"\bT (ooo_[a-z_0-9]+)$", out, re.M))
    assert set(names) <= exported
    assert ooo.version() == 1


def _pack_both(root, cands, max_nodes, max_depth, mask_words=None):
    offs = np.zeros(len(cands) + 1, np.int32)
    for i, c in enumerate(cands):
        offs[i + 1] = offs[i] + len(c)
    toks = np.array([t for c in cands for t in c], dtype=np.int32)
    lib_res = ooo.pack_tree(root, toks, offs, max_nodes, max_depth, mask_words)
    ref = ov.pack_tree(root, cands, max_nodes, max_depth)
    return lib_res, ref


def _assert_same(lib_res, ref):
    assert lib_res["n_nodes"] == ref["n_nodes"]
    assert np.array_equal(lib_res["token"], ref["token"])
    assert np.array_equal(lib_res["parent"], ref["parent"])
    assert np.array_equal(lib_res["depth"], ref["depth"])
    assert lib_res["n_truncated"] == ref["n_truncated"]
    assert np.array_equal(lib_res["anc_mask"], ov.ancestor_masks(ref["parent"], lib_res["mask_words"]))


def test_pack_matches_reference_on_random_sets():
    for root, cands, mn, md in oc.random_candidate_sets(21, count=300):
        _assert_same(*_pack_both(root, cands, mn, md))


@pytest.mark.parametrize("mask_words", [1, 2, 4, 5])
def test_pack_mask_word_boundaries(mask_words):
    rs = np.random.default_rng(mask_words)
    for n_max in (63, 64, 65, 128, 256, 257, 64 * mask_words):
        if n_max > 64 * mask_words:
            continue
        cands = [[int(t) for t in rs.integers(0, 1000, size=int(rs.integers(1, 80)))] for _ in range(12)]
        _assert_same(*_pack_both(5, cands, n_max, 200, mask_words))


@pytest.mark.parametrize("name", list(wl.CONFIGS))
def test_pack_matches_reference_on_workloads(name):
    cfg = wl.CONFIGS[name]
    steps = [0, 30, 199] if cfg.steps > 1 else [0]
    for seed in range(3):
        for step in steps:
            c = wl.candidates_for(cfg, seed, step)
            _assert_same(*_pack_both(c.root_token, c.seqs, c.max_nodes, c.max_depth, cfg.mask_words))


def test_pack_into_caller_buffers_matches_reference():
    """The in-place packer (writing into one reused staging buffer, as the
    per-step runner does) gives the same trie as the oracle for a sequence of
    different candidate sets, whatever the buffer held before."""
    max_nodes, W = 64, 1
    buf = np.full(3 * max_nodes + 2 * max_nodes * W, -7, np.int32)
    m = 2 * max_nodes * W
    mask = buf[0:m].view(np.uint64).reshape(max_nodes, W)
    tok, par, dep = buf[m:m + max_nodes], buf[m + max_nodes:m + 2 * max_nodes], buf[m + 2 * max_nodes:]
    for root, cands, _, md in oc.random_candidate_sets(5, count=60):
        offs = np.zeros(len(cands) + 1, np.int32)
        for i, c in enumerate(cands):
            offs[i + 1] = offs[i] + len(c)
        toks = np.array([t for c in cands for t in c], dtype=np.int32)
        n, trunc = ooo.pack_tree_into(root, toks, offs, max_nodes, md, tok, par, dep, mask)
        ref = ov.pack_tree(root, cands, max_nodes, md)
        assert n == ref["n_nodes"] and trunc == ref["n_truncated"]
        assert np.array_equal(tok[:n], ref["token"]) and np.array_equal(par[:n], ref["parent"])
        assert np.array_equal(dep[:n], ref["depth"])
        assert np.array_equal(mask[:n], ov.ancestor_masks(ref["parent"], W))
    with pytest.raises(ValueError):
        ooo.pack_tree_into(1, np.array([2], np.int32), np.array([0, 1], np.int32), max_nodes, 4,
                           tok[:10], par, dep, mask)


def test_pack_degenerate_inputs():
    r, ref = _pack_both(3, [], 1, 0)
    _assert_same(r, ref)
    assert r["n_nodes"] == 1 and r["anc_mask"].tolist() == [[1]]
    r, ref = _pack_both(3, [[1, 2], [1, 2], [1]], 1, 5)  # budget of one: root only
    _assert_same(r, ref)
    assert r["n_truncated"] == 5
    r, ref = _pack_both(3, [[1, 2, 3]], 10, 0)  # depth cap 0
    _assert_same(r, ref)
    assert r["n_nodes"] == 1 and r["n_truncated"] == 3


def _call_pack(root=1, toks=(1, 2), offs=(0, 2), max_nodes=4, max_depth=4, W=1, null_out=False):
    toks = np.array(toks, np.int32)
    offs = np.array(offs, np.int32)
    o = [np.zeros(max(max_nodes, 1), np.int32) for _ in range(3)]
    m = np.zeros(max(max_nodes, 1) * max(W, 1), np.uint64)
    n = ctypes.c_int32(0)
    t = ctypes.c_int32(0)
    P = ctypes.POINTER(ctypes.c_int32)
    return ooo.lib().ooo_pack_tree(
        root, toks.ctypes.data_as(P), offs.ctypes.data_as(P), len(offs) - 1, max_nodes, max_depth,
        None if null_out else o[0].ctypes.data_as(P), o[1].ctypes.data_as(P), o[2].ctypes.data_as(P),
        m.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64)), W, ctypes.byref(n), ctypes.byref(t))


@pytest.mark.parametrize("kwargs", [
    dict(max_nodes=0), dict(max_depth=-1), dict(W=0), dict(max_nodes=65, W=1),
    dict(offs=(1, 2)), dict(toks=(1, -2)), dict(root=-1), dict(null_out=True), dict(offs=(0, 2, 1), toks=(1, 2)),
])
def test_pack_rejects_bad_arguments(kwargs):
    st = _call_pack(**kwargs)
    assert st == ooo.ERR_INVALID
    assert ooo.last_error() != ""


def test_pack_node_limit_and_no_state_between_calls():
    """The 1024-node limit of the device kernels is reported; a full-size
    pack after a small one (and the reverse) gives the reference trie each
    time: nothing carries over between calls."""
    assert _call_pack(max_nodes=1025, W=17) == ooo.ERR_UNSUPPORTED
    assert "exceeds 1024" in ooo.last_error()
    rs = np.random.default_rng(21)
    big = [[int(t) for t in rs.integers(0, 3, size=int(rs.integers(1, 30)))] for _ in range(200)]
    small = [[5, 6], [5, 7]]
    for cands, nodes in [(big, 1024), (small, 8), (big, 1024), (small, 3)]:
        r, ref = _pack_both(2, cands, nodes, 64)
        _assert_same(r, ref)


def test_layer_entry_points_validate_on_host():
    L = ooo.lib()
    fake = ctypes.c_void_p(256)  # never dereferenced: every call below fails validation first
    assert L.ooo_embed_rows(None, fake, 4, 64, 100, fake, None) == ooo.ERR_INVALID
    assert L.ooo_embed_rows(fake, fake, 0, 64, 100, fake, None) == ooo.ERR_INVALID
    assert L.ooo_rmsnorm(fake, None, 4, 64, 1e-6, fake, None) == ooo.ERR_INVALID
    assert L.ooo_rmsnorm(fake, fake, 4, 64, -1.0, fake, None) == ooo.ERR_INVALID
    assert L.ooo_rmsnorm(fake, fake, 4, 66, 1e-6, fake, None) == ooo.ERR_UNSUPPORTED
    assert L.ooo_rmsnorm(fake, fake, 4, 8196, 1e-6, fake, None) == ooo.ERR_UNSUPPORTED
    assert L.ooo_embed_rows(fake, fake, 4, 60, 100, fake, None) == ooo.ERR_UNSUPPORTED
    lin = lambda n=4, k=64, o=64, lay=ooo.W_PACKED, epi=ooo.EPI_STORE_F32, x=fake, ws=fake, wsb=1 << 30: \
        L.ooo_linear(x, fake, n, k, o, lay, epi, fake, ws, wsb, None)
    assert lin(n=0) == ooo.ERR_INVALID
    assert lin(x=None) == ooo.ERR_INVALID
    assert lin(lay=7) == ooo.ERR_INVALID
    assert lin(epi=9) == ooo.ERR_INVALID
    assert lin(k=96) == ooo.ERR_UNSUPPORTED
    assert lin(n=300) == ooo.ERR_UNSUPPORTED
    assert lin(o=384, epi=ooo.EPI_SWIGLU_BF16) == ooo.ERR_UNSUPPORTED
    assert lin(wsb=16) == ooo.ERR_CAPACITY
    assert lin(ws=None) == ooo.ERR_CAPACITY
    assert ooo.linear_workspace(64, 4096, 6144) > 0 and ooo.linear_workspace(64, 100, 64) == 0
    assert ooo.lib().ooo_linear_packed_bytes(300, 128) == 384 * 128 * 2
    args = dict(qkv=fake, qn=fake, kn=fake, eps=1e-6, depth=fake, N=4, P=10, theta=1e6, Hq=4, Hkv=2, D=128,
                q=fake, kc=fake, vc=fake, cap=100)

    def qk(**kw):
        a = {**args, **kw}
        return L.ooo_qk_norm_rope(a["qkv"], a["qn"], a["kn"], a["eps"], a["depth"], a["N"], a["P"], None,
                                  a["theta"], a["Hq"], a["Hkv"], a["D"], a["q"], a["kc"], a["vc"], a["cap"], None)
    assert qk(qkv=None) == ooo.ERR_INVALID
    assert qk(depth=None) == ooo.ERR_INVALID
    assert qk(P=97) == ooo.ERR_INVALID  # P + N > cap
    assert qk(theta=0.0) == ooo.ERR_INVALID
    assert qk(N=0) == ooo.ERR_INVALID
    assert qk(D=96) == ooo.ERR_UNSUPPORTED
    assert L.ooo_swiglu(None, 4, 64, fake, None) == ooo.ERR_INVALID
    assert L.ooo_swiglu(fake, 4, 0, fake, None) == ooo.ERR_INVALID
    # fused projection epilogues: rejected on the host, nothing enqueued
    ws_need = ooo.linear_workspace(64, 4096, 4096)
    assert L.ooo_linear_add_rmsnorm(fake, fake, 64, 4096, 4096, ooo.W_PACKED, None, fake, 1e-6, fake, fake,
                                    ws_need, None) == ooo.ERR_INVALID
    assert L.ooo_linear_add_rmsnorm(fake, fake, 64, 4096, 8196, ooo.W_PACKED, fake, fake, 1e-6, fake, fake,
                                    1 << 30, None) == ooo.ERR_UNSUPPORTED
    assert L.ooo_linear_add_rmsnorm(fake, fake, 64, 4096, 4096, ooo.W_PACKED, fake, fake, -1.0, fake, fake,
                                    ws_need, None) == ooo.ERR_INVALID
    assert L.ooo_linear_add_rmsnorm(fake, fake, 64, 4096, 4096, ooo.W_PACKED, fake, fake, 1e-6, fake, fake,
                                    ws_need - 1, None) == ooo.ERR_CAPACITY
    qk = lambda **kw: L.ooo_linear_qk_norm_rope(
        fake, fake, kw.get("N", 64), 4096, ooo.W_PACKED, fake, fake, 1e-6, kw.get("depth", fake), kw.get("P", 10),
        None, 1e6, 32, 8, kw.get("D", 128), fake, fake, fake, kw.get("cap", 5000), fake, kw.get("ws", 1 << 30), None)
    assert qk(depth=None) == ooo.ERR_INVALID
    assert qk(P=4990) == ooo.ERR_INVALID  # P + N > cap
    assert qk(D=96) == ooo.ERR_UNSUPPORTED
    assert qk(ws=16) == ooo.ERR_CAPACITY


def test_device_entry_points_validate_on_host():
    L = ooo.lib()
    fake = ctypes.c_void_p(256)  # never dereferenced: every call below fails validation first
    # null pointers
    assert L.ooo_tree_attn(None, fake, fake, 100, 10, None, 4, fake, 1, 4, 1, 64, 0.1, ooo.BF16, fake, None, 0, None) \
        == ooo.ERR_INVALID
    assert "null" in ooo.last_error()
    assert L.ooo_lmhead_argmax(fake, None, 4, 64, 100, ooo.BF16, ooo.W_ROWS, fake, fake, None, fake, 1 << 20, None) \
        == ooo.ERR_INVALID
    assert L.ooo_accept(fake, fake, fake, fake, 1, fake, 4, 7, 8, None, fake, fake, None) == ooo.ERR_INVALID
    assert L.ooo_kv_compact(fake, fake, 2, 2, 100, 64, ooo.BF16, 10, None, 4, None, fake, 8, None) == ooo.ERR_INVALID
    # inconsistent shapes
    assert L.ooo_tree_attn(fake, fake, fake, 100, 97, None, 4, fake, 1, 4, 1, 64, 0.1, ooo.BF16, fake, None, 0, None) \
        == ooo.ERR_INVALID  # P + N > cap
    assert L.ooo_tree_attn(fake, fake, fake, 100, 10, None, 4, fake, 1, 6, 4, 64, 0.1, ooo.BF16, fake, None, 0, None) \
        == ooo.ERR_INVALID  # Hq % Hkv
    assert L.ooo_tree_attn(fake, fake, fake, 100, 10, None, 65, fake, 1, 4, 1, 64, 0.1, ooo.BF16, fake, None, 0, None) \
        == ooo.ERR_INVALID  # too few mask words
    assert L.ooo_tree_attn(fake, fake, fake, 100, 10, None, 0, fake, 1, 4, 1, 64, 0.1, ooo.BF16, fake, None, 0, None) \
        == ooo.ERR_INVALID
    assert L.ooo_accept(fake, fake, fake, fake, 1, fake, 65, 7, 8, fake, fake, fake, None) == ooo.ERR_INVALID
    assert L.ooo_accept(fake, fake, fake, fake, 1, fake, 4, 0, 0, fake, fake, fake, None) == ooo.ERR_INVALID
    assert L.ooo_accept(fake, fake, fake, fake, 1, fake, 4, -1, 8, fake, fake, fake, None) == ooo.ERR_INVALID
    # a path buffer that cannot hold a root path of the declared depth
    assert L.ooo_accept(fake, fake, fake, fake, 1, fake, 4, 8, 8, fake, fake, fake, None) == ooo.ERR_CAPACITY
    assert "cannot hold" in ooo.last_error()
    assert L.ooo_kv_compact(fake, fake, 2, 2, 100, 64, ooo.BF16, 97, None, 4, fake, fake, 8, None) == ooo.ERR_INVALID
    # unsupported but valid
    assert L.ooo_tree_attn(fake, fake, fake, 100, 10, None, 4, fake, 1, 4, 1, 96, 0.1, ooo.BF16, fake, None, 0, None) \
        == ooo.ERR_UNSUPPORTED
    assert L.ooo_lmhead_argmax(fake, fake, 4, 100, 1000, ooo.BF16, ooo.W_ROWS, fake, fake, None, fake, 1 << 20, None) \
        == ooo.ERR_UNSUPPORTED
    assert L.ooo_lmhead_argmax(fake, fake, 300, 128, 1000, ooo.BF16, ooo.W_ROWS, fake, fake, None, fake, 1 << 20, None) \
        == ooo.ERR_UNSUPPORTED
    assert L.ooo_kv_compact(fake, fake, 2, 2, 100, 4, ooo.BF16, 10, None, 4, fake, fake, 8, None) == ooo.ERR_UNSUPPORTED
    # weight layouts
    assert L.ooo_lmhead_argmax(fake, fake, 4, 64, 1000, ooo.BF16, 2, fake, fake, None, fake, 1 << 20, None) \
        == ooo.ERR_INVALID
    assert L.ooo_lmhead_argmax(fake, fake, 4, 64, 1000, ooo.F32, ooo.W_PACKED, fake, fake, None, fake, 1 << 20,
                               None) == ooo.ERR_UNSUPPORTED
    assert L.ooo_lmhead_packed_bytes(1000, 64, ooo.BF16) == 8 * 128 * 64 * 2  # 8 tiles of 128 rows
    assert L.ooo_lmhead_packed_bytes(1000, 100, ooo.BF16) == 0
    assert L.ooo_lmhead_packed_bytes(1000, 64, ooo.F32) == 0
    assert L.ooo_lmhead_pack(fake, 1000, 64, ooo.BF16, None, 1 << 20, None) == ooo.ERR_INVALID
    assert L.ooo_lmhead_pack(fake, 1000, 64, ooo.F32, fake, 1 << 20, None) == ooo.ERR_UNSUPPORTED
    assert L.ooo_lmhead_pack(fake, 1000, 100, ooo.BF16, fake, 1 << 20, None) == ooo.ERR_UNSUPPORTED
    assert L.ooo_lmhead_pack(fake, 1000, 64, ooo.BF16, fake, 8 * 128 * 64 * 2 - 1, None) == ooo.ERR_CAPACITY
    # workspace too small
    need = L.ooo_lmhead_workspace(4, 64, 1000, ooo.BF16)
    assert need > 0
    assert L.ooo_lmhead_argmax(fake, fake, 4, 64, 1000, ooo.BF16, ooo.W_ROWS, fake, fake, None, fake, need - 1, None) \
        == ooo.ERR_CAPACITY
    need = L.ooo_tree_attn_workspace(64, 32, 8, 128, 4096, ooo.BF16)
    assert need > 0
    assert L.ooo_tree_attn(fake, fake, fake, 4160, 4096, None, 64, fake, 1, 32, 8, 128, 0.1, ooo.BF16, fake, fake,
                           need - 1, None) == ooo.ERR_CAPACITY
    assert ooo.last_error() != ""
