"""One verification step as a sequence of libooo calls.

The runner owns the per-step device buffers (trie arrays, per-layer
attention outputs, greedy tokens, accepted path, workspaces) for one
workload shape and issues, on one stream:

    H2D of the packed trie  ->  n_layers x ooo_tree_attn  ->  ooo_lmhead_argmax
    ->  ooo_accept  ->  ooo_kv_compact  ->  D2H of (L, bonus, path)

Packing runs on the host through ``ooo_pack_tree``.  The node queries, the
node K/V rows written into the cache and the hidden rows feeding the LM head
are the model's job (its projections); the caller stages them.
"""

from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Optional, Sequence

import numpy as np
import torch

from . import ooo


@dataclass
class StepResult:
    n_nodes: int
    n_truncated: int
    L: int
    bonus: int
    path: np.ndarray

    @property
    def committed_count(self) -> int:
        return self.L + 1


class VerifyRunner:
    def __init__(self, n_layers: int, n_q_heads: int, n_kv_heads: int, head_dim: int, hidden: int, vocab: int,
                 max_nodes: int, max_depth: int, dtype: torch.dtype, device="cuda", max_prefix: int = 0):
        self.L_m, self.Hq, self.Hkv, self.D = n_layers, n_q_heads, n_kv_heads, head_dim
        self.H, self.V = hidden, vocab
        self.max_nodes, self.max_depth = max_nodes, max_depth
        self.W = max(1, (max_nodes + 63) // 64)
        self.dtype = dtype
        self.device = torch.device(device)
        self.code = ooo.BF16 if dtype == torch.bfloat16 else ooo.F32
        dev = self.device
        self.path_cap = max_depth + 1
        # trie on the device, filled from pinned host staging; the last
        # entries are a header (the prefix length the step runs at, read on
        # the device when one captured step is replayed at a growing prefix)
        self.h_tree = torch.zeros(3 * max_nodes + 2 * max_nodes * self.W + 4, dtype=torch.int32).pin_memory()
        self.d_tree = torch.zeros_like(self.h_tree, device=dev)
        n = max_nodes
        m = 2 * n * self.W  # mask first so its int64 view stays 8-byte aligned
        self.mask = self.d_tree[0:m].view(torch.int64).view(n, self.W)
        self.token = self.d_tree[m:m + n]
        self.parent = self.d_tree[m + n:m + 2 * n]
        self.depth = self.d_tree[m + 2 * n:m + 3 * n]
        self.prefix_dev = self.d_tree[m + 3 * n:m + 3 * n + 1]
        h = self.h_tree.numpy()
        self._h_mask = h[0:m].view(np.uint64).reshape(n, self.W)
        self._h_token = h[m:m + n]
        self._h_parent = h[m + n:m + 2 * n]
        self._h_depth = h[m + 2 * n:m + 3 * n]
        self._h_hdr = h[m + 3 * n:m + 3 * n + 4]
        self.out = torch.empty(n_layers, max_nodes, n_q_heads, head_dim, dtype=dtype, device=dev)
        self.ids = torch.empty(max_nodes, dtype=torch.int32, device=dev)
        self.max_logit = torch.empty(max_nodes, dtype=torch.float32, device=dev)
        self.res = torch.zeros(2 + self.path_cap, dtype=torch.int32, device=dev)  # L, bonus, path
        self.accept_len = self.res[0:1]
        self.bonus = self.res[1:2]
        self.path = self.res[2:]
        self.h_res = torch.zeros_like(self.res, device="cpu").pin_memory()
        self.attn_ws = torch.zeros(64, dtype=torch.float32, device=dev)
        for nn in sorted({1, max(1, max_nodes // 2), max_nodes}):
            self.ensure_workspace(max(max_prefix, 1), nn)
        lws = ooo.lmhead_workspace(max_nodes, hidden, vocab, self.code)
        self.lm_ws = torch.empty(max(lws, 256) // 4 + 1, dtype=torch.float32, device=dev)
        self.scale = 1.0 / math.sqrt(head_dim)
        self.n_nodes = 0
        self.n_truncated = 0
        self.packed = None
        self._packer = ooo.StagedPacker(max_nodes, max_depth, self._h_token, self._h_parent, self._h_depth,
                                        self._h_mask)

    # -- host ---------------------------------------------------------------
    def pack(self, root_token: int, cand_tokens: np.ndarray, cand_offsets: np.ndarray,
             keep: bool = True) -> Optional[dict]:
        """Pack the candidates straight into the pinned staging buffer.  With
        keep, also return copies of the trie arrays (the buffer is rewritten
        by the next pack); without, return None (the per-step path)."""
        k, trunc = self._packer(root_token, cand_tokens, cand_offsets)
        self.n_nodes = k
        self.n_truncated = trunc
        self.packed = None
        if keep:
            self.packed = {"token": self._h_token[:k].copy(), "parent": self._h_parent[:k].copy(),
                           "depth": self._h_depth[:k].copy(), "anc_mask": self._h_mask[:k].copy(),
                           "n_nodes": k, "n_truncated": trunc, "mask_words": self.W}
        return self.packed

    def set_prefix(self, prefix_len: int) -> None:
        """Stage the prefix length that the next upload carries to
        ``prefix_dev`` (for steps that read it on the device)."""
        self._h_hdr[0] = prefix_len

    def ensure_workspace(self, prefix_len: int, n_nodes: Optional[int] = None) -> None:
        """Grow the attention workspace (outside any timed or captured region)."""
        n = self.n_nodes if n_nodes is None else n_nodes
        need = ooo.tree_attn_workspace(max(n, 1), self.Hq, self.Hkv, self.D, prefix_len, self.code)
        if need > self.attn_ws.numel() * 4:
            self.attn_ws = torch.zeros(need // 4 + 1, dtype=torch.float32, device=self.device)

    # -- device -------------------------------------------------------------
    def upload_tree(self, stream=None) -> None:
        self.d_tree.copy_(self.h_tree, non_blocking=True)

    def attention(self, layer: int, q, k_layer, v_layer, prefix_len: int, stream=None, prefix_dev=None) -> None:
        N = self.n_nodes
        ooo.tree_attn(q, k_layer, v_layer, prefix_len, N, self.mask[:N], self.Hq, self.Hkv, self.scale,
                      self.out[layer, :N], self.attn_ws, stream, prefix_dev=prefix_dev)

    def lm_head(self, hidden, logits=None, stream=None) -> None:
        N = self.n_nodes
        ooo.lmhead_argmax(hidden[:N], self._weight, self.ids[:N], self.max_logit[:N], logits, self.lm_ws, stream)

    def accept(self, stream=None) -> None:
        N = self.n_nodes
        ooo.accept(self.token[:N], self.parent[:N], self.depth[:N], self.mask[:N], self.ids[:N], N, self.path,
                   self.accept_len, self.bonus, stream, max_depth=self.max_depth)

    def compact(self, k_cache, v_cache, prefix_len: int, stream=None, prefix_dev=None) -> None:
        ooo.kv_compact(k_cache, v_cache, prefix_len, self.n_nodes, self.path, self.accept_len, stream,
                       prefix_dev=prefix_dev)

    def download(self) -> None:
        self.h_res.copy_(self.res, non_blocking=True)

    def result(self) -> StepResult:
        r = self.h_res.numpy()
        L = int(r[0])
        if L < 0:
            raise ooo.OooError(ooo.ERR_CAPACITY, f"accepted path deeper than max_depth {self.max_depth}: "
                               "nothing was committed")
        return StepResult(self.n_nodes, self.n_truncated, L, int(r[1]), r[2:2 + L + 1].copy())

    def set_weight(self, weight, packed: Optional[bool] = None) -> None:
        """Binds the LM-head weight [V][H].  bf16 weights are re-laid out once
        for streaming (ooo_lmhead_pack) unless packed=False; the row-major
        tensor is then no longer referenced."""
        if packed is None:
            packed = self.code == ooo.BF16 and weight.shape[1] % 64 == 0
        self._weight = ooo.lmhead_pack(weight) if packed else weight

    def device_step(self, q_layers: Sequence, k_cache, v_cache, hidden, prefix_len: int,
                    logits=None, compact: bool = True, prefix_dev=None) -> None:
        """Everything after packing, enqueued on the current stream.  With
        ``prefix_dev`` the kernels read P from the device (``prefix_len``
        bounds it)."""
        self.upload_tree()
        for l in range(self.L_m):
            self.attention(l, q_layers[l], k_cache[l], v_cache[l], prefix_len, prefix_dev=prefix_dev)
        self.lm_head(hidden, logits)
        self.accept()
        if compact:
            self.compact(k_cache, v_cache, prefix_len, prefix_dev=prefix_dev)
        self.download()
