"""ooo_tree_attn_noalloc (the attention entry point that allocates nothing)
against ooo_tree_attn with a caller workspace, through the C ABI: bitwise the
same output (same kernels, same plan) and within the oracle tolerance, on two
calls in a row, the second with a smaller input."""

import math

import numpy as np
import pytest
import torch

import gpu_harness as gh
from oracle import tree_verify as ov
from paper_2608_00814_amd import ooo
from paper_2608_00814_amd import workload as wl

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _inputs(P, N, G, Hkv, D, seed):
    rs = np.random.default_rng(seed)
    cap = P + N + 3
    q = wl.to_bf16_bits(rs.normal(size=(N, G * Hkv, D)).astype(np.float32))
    k = wl.to_bf16_bits(rs.normal(size=(Hkv, cap, D)).astype(np.float32))
    v = wl.to_bf16_bits(rs.normal(size=(Hkv, cap, D)).astype(np.float32))
    cands = [[int(t) for t in rs.integers(0, 3, size=int(rs.integers(1, 20)))] for _ in range(4 * N)]
    t = ov.pack_tree(0, cands, N, 10 ** 6)
    assert t["n_nodes"] == N
    return q, k, v, t


def test_noalloc_matches_the_workspace_entry_point():
    for P, N, G, Hkv, D in [(4096, 64, 4, 8, 128), (700, 20, 4, 2, 128)]:
        print(f"case noalloc P={P} N={N} G={G} Hkv={Hkv} D={D}", flush=True)
        q, k, v, t = _inputs(P, N, G, Hkv, D, seed=P + N)
        W = (N + 63) // 64
        mask = ov.ancestor_masks(t["parent"], W)
        qd, kd, vd = gh.to_dev(q, "bf16", DEV), gh.to_dev(k, "bf16", DEV), gh.to_dev(v, "bf16", DEV)
        md = torch.from_numpy(mask.view(np.int64)).to(DEV)
        Hq = G * Hkv
        need = ooo.tree_attn_workspace(N, Hq, Hkv, D, P, ooo.BF16)
        assert 0 < need <= ooo.lib().ooo_tree_attn_noalloc_scratch_bytes()
        ws = torch.zeros(need // 4 + 1, dtype=torch.float32, device=DEV)
        a = torch.full((N, Hq, D), float("nan"), dtype=torch.bfloat16, device=DEV)
        b = torch.full_like(a, float("nan"))
        ooo.tree_attn(qd, kd, vd, P, N, md, Hq, Hkv, 1.0 / math.sqrt(D), a, ws)
        ooo.tree_attn_noalloc(qd, kd, vd, P, N, md, Hq, Hkv, 1.0 / math.sqrt(D), b)
        torch.cuda.synchronize()
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))
        got = wl.to_f64(gh.to_host(b, "bf16"), "bf16")
        ref = ov.tree_attention(wl.to_f64(q, "bf16"), wl.to_f64(k, "bf16"), wl.to_f64(v, "bf16"), P, t["parent"], Hkv)
        assert gh.row_rel_err(got, ref) <= gh.ATTN_TOL
