"""Full target verify step: the decoder layers around the verification path.

``ModelRunner`` owns a Qwen3-shaped decoder's device weights and per-step
buffers and issues, on one stream, for a packed trie (``VerifyRunner``
supplies the trie arrays, the attention, the LM head, acceptance and
compaction):

    h = embedding[token]                                  ooo_embed_rows
    per layer:
        x   = rmsnorm(h)                                  ooo_rmsnorm
        qkv = x Wqkv^T                                    ooo_linear (bf16 out)
        q, cache[P + i] <- k, v  (norms, rotation at P + depth)   ooo_qk_norm_rope
        o   = tree attention                              ooo_tree_attn
        h  += o Wo^T                                      ooo_linear (add into h)
        x   = rmsnorm(h)                                  ooo_rmsnorm
        a   = silu(x Wg^T) * (x Wu^T)                     ooo_linear (SwiGLU epilogue)
        h  += a Wd^T                                      ooo_linear (add into h)
    X = rmsnorm(h); greedy tokens; accept; compact        (VerifyRunner)

By default the projections' epilogues are fused into their consumers: the
qkv projection with the norms, rotation and cache writes
(ooo_linear_qk_norm_rope), o_proj and down with the residual add and the
following RMSNorm (ooo_linear_add_rmsnorm); 10 launches per layer instead of
13.

The residual rows stay in float32; every projection reads bf16 operands and
accumulates in float32.  Projection weights are packed once, at load, into
the streaming layout of ooo_linear_pack.
"""

from __future__ import annotations

from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

from . import ooo
from .model_workload import ModelConfig
from .step import VerifyRunner


def _bits_to_dev(a: np.ndarray, dev) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)


class ModelRunner:
    def __init__(self, cfg: ModelConfig, layers: Sequence[Dict[str, np.ndarray]], embedding: np.ndarray,
                 final_norm: np.ndarray, lm_head: np.ndarray, device="cuda", fused: bool = True):
        """Weights as bf16 bit patterns (uint16, ``model_workload`` layout).
        ``fused``: projections with their consumers fused into the epilogue
        (ooo_linear_qk_norm_rope, ooo_linear_add_rmsnorm); False issues the
        separate calls."""
        self.cfg = cfg
        self.fused = fused
        dev = torch.device(device)
        self.device = dev
        self.vr = VerifyRunner(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cfg.hidden, cfg.vocab,
                               cfg.max_nodes, cfg.max_depth, torch.bfloat16, dev, max_prefix=cfg.cap - cfg.max_nodes)
        self.vr.set_weight(_bits_to_dev(lm_head, dev))
        self.emb = _bits_to_dev(embedding, dev)
        self.final_norm = _bits_to_dev(final_norm, dev)
        self.layers: List[Dict[str, object]] = []
        pk = lambda a: ooo.linear_pack(_bits_to_dev(a, dev))
        for lw in layers:
            self.layers.append({
                "in_norm": _bits_to_dev(lw["in_norm"], dev),
                "w_qkv": pk(lw["w_qkv"]),
                "q_norm": _bits_to_dev(lw["q_norm"], dev),
                "k_norm": _bits_to_dev(lw["k_norm"], dev),
                "w_o": pk(lw["w_o"]),
                "post_norm": _bits_to_dev(lw["post_norm"], dev),
                # gate rows, then up rows: the SwiGLU epilogue pairs them
                "w_gu": pk(np.concatenate([lw["w_gate"], lw["w_up"]], axis=0)),
                "w_down": pk(lw["w_down"]),
            })
            torch.cuda.synchronize(dev)  # the row-major copies can go
        n, H = cfg.max_nodes, cfg.hidden
        self.h = torch.zeros(n, H, dtype=torch.float32, device=dev)
        self.x = torch.zeros(n, H, dtype=torch.bfloat16, device=dev)
        self.xf = torch.zeros(n, H, dtype=torch.bfloat16, device=dev)  # LM-head input
        self.qkv = torch.zeros(n, cfg.qkv_rows, dtype=torch.bfloat16, device=dev)
        self.q = torch.zeros(n, cfg.n_q_heads, cfg.head_dim, dtype=torch.bfloat16, device=dev)
        self.act = torch.zeros(n, cfg.intermediate, dtype=torch.bfloat16, device=dev)
        H, I, A = cfg.hidden, cfg.intermediate, cfg.n_q_heads * cfg.head_dim
        need = max(ooo.linear_workspace(nn, k, o) for nn in range(1, n + 1)
                   for k, o in ((H, cfg.qkv_rows), (A, H), (H, 2 * I), (I, H)))
        self.lin_ws = torch.empty(need, dtype=torch.uint8, device=dev)

    # -- host ---------------------------------------------------------------
    def pack(self, root_token: int, cand_tokens: np.ndarray, cand_offsets: np.ndarray, keep: bool = True):
        return self.vr.pack(root_token, cand_tokens, cand_offsets, keep=keep)

    # -- device -------------------------------------------------------------
    def forward(self, k_cache: torch.Tensor, v_cache: torch.Tensor, prefix_len: int, prefix_dev=None) -> None:
        """Decoder layers over the packed trie (already uploaded): leaves the
        LM-head input rows in ``self.xf`` and each layer's attention output
        in ``self.vr.out``; node k/v rows go to the caches' rows [P, P + N).
        With ``prefix_dev`` (an int32 device scalar) the kernels read P from
        it and ``prefix_len`` is only its upper bound."""
        cfg, vr = self.cfg, self.vr
        N, P = vr.n_nodes, prefix_len
        vr.ensure_workspace(P)  # allocates only for a larger shape than seen before (never inside a capture)
        ws = self.lin_ws
        ooo.embed_rows(self.emb, vr.token, N, self.h)
        if not self.fused:
            for l, w in enumerate(self.layers):
                ooo.rmsnorm(self.h, w["in_norm"], cfg.eps, self.x, n_rows=N)
                ooo.linear(self.x, w["w_qkv"], self.qkv, ooo.EPI_STORE_BF16, ws, n_rows=N)
                ooo.qk_norm_rope(self.qkv, w["q_norm"], w["k_norm"], cfg.eps, vr.depth, N, P, cfg.rope_theta,
                                 cfg.n_q_heads, cfg.n_kv_heads, self.q, k_cache[l], v_cache[l], prefix_dev=prefix_dev)
                vr.attention(l, self.q, k_cache[l], v_cache[l], P, prefix_dev=prefix_dev)
                o = vr.out[l].view(cfg.max_nodes, cfg.n_q_heads * cfg.head_dim)
                ooo.linear(o, w["w_o"], self.h, ooo.EPI_ADD_F32, ws, n_rows=N)
                ooo.rmsnorm(self.h, w["post_norm"], cfg.eps, self.x, n_rows=N)
                ooo.linear(self.x, w["w_gu"], self.act, ooo.EPI_SWIGLU_BF16, ws, n_rows=N)
                ooo.linear(self.act, w["w_down"], self.h, ooo.EPI_ADD_F32, ws, n_rows=N)
            ooo.rmsnorm(self.h, self.final_norm, cfg.eps, self.xf, n_rows=N)
            return
        # The same layers with the projections' epilogues fused into their
        # consumers: qkv + norms/rotation/cache writes, o_proj + residual add
        # + post-attention norm, down + residual add + the next layer's input
        # norm (the final norm after the last layer).
        ooo.rmsnorm(self.h, self.layers[0]["in_norm"], cfg.eps, self.x, n_rows=N)
        for l, w in enumerate(self.layers):
            ooo.linear_qk_norm_rope(self.x, w["w_qkv"], w["q_norm"], w["k_norm"], cfg.eps, vr.depth, N, P,
                                    cfg.rope_theta, cfg.n_q_heads, cfg.n_kv_heads, self.q, k_cache[l], v_cache[l],
                                    ws, prefix_dev=prefix_dev)
            vr.attention(l, self.q, k_cache[l], v_cache[l], P, prefix_dev=prefix_dev)
            o = vr.out[l].view(cfg.max_nodes, cfg.n_q_heads * cfg.head_dim)
            ooo.linear_add_rmsnorm(o, w["w_o"], self.h, w["post_norm"], cfg.eps, self.x, ws, n_rows=N)
            ooo.linear(self.x, w["w_gu"], self.act, ooo.EPI_SWIGLU_BF16, ws, n_rows=N)
            last = l + 1 == len(self.layers)
            nxt = self.final_norm if last else self.layers[l + 1]["in_norm"]
            ooo.linear_add_rmsnorm(self.act, w["w_down"], self.h, nxt, cfg.eps, self.xf if last else self.x, ws,
                                   n_rows=N)

    def device_step(self, k_cache: torch.Tensor, v_cache: torch.Tensor, prefix_len: int,
                    logits: Optional[torch.Tensor] = None, compact: bool = True, prefix_dev=None) -> None:
        """Everything after packing, enqueued on the current stream."""
        vr = self.vr
        vr.upload_tree()
        self.forward(k_cache, v_cache, prefix_len, prefix_dev)
        vr.lm_head(self.xf, logits)
        vr.accept()
        if compact:
            vr.compact(k_cache, v_cache, prefix_len, prefix_dev=prefix_dev)
        vr.download()

    def result(self):
        return self.vr.result()
