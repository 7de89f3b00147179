"""ctypes binding of libooo (C ABI declared in include/ooo.h).

Argument marshalling only: every computation happens in the native library.
Device arguments are torch tensors on the ROCm device (their ``data_ptr()``
is passed through); host arguments of ``pack_tree`` are NumPy arrays.  The
library must be built (``python -m paper_2608_00814_amd.build``); loading
fails loudly when it is missing.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libooo.so")

OK, ERR_INVALID, ERR_UNSUPPORTED, ERR_CAPACITY, ERR_HIP = 0, -1, -2, -3, -4
F32, BF16 = 0, 1
W_ROWS, W_PACKED = 0, 1  # ooo_weight_layout
EPI_STORE_F32, EPI_STORE_BF16, EPI_ADD_F32, EPI_SWIGLU_BF16 = 0, 1, 2, 3  # ooo_epilogue

_c_i32p = ctypes.POINTER(ctypes.c_int32)
_c_u64p = ctypes.POINTER(ctypes.c_uint64)
_vp = ctypes.c_void_p
_i32 = ctypes.c_int32
_i64 = ctypes.c_int64
_sz = ctypes.c_size_t

# name -> (restype, argtypes); mirrors include/ooo.h
SIGNATURES = {
    "ooo_last_error": (ctypes.c_char_p, []),
    "ooo_version": (ctypes.c_int, []),
    "ooo_pack_tree": (ctypes.c_int, [_i32, _c_i32p, _c_i32p, _i32, _i32, _i32, _c_i32p, _c_i32p, _c_i32p,
                                     _c_u64p, _i32, _c_i32p, _c_i32p]),
    "ooo_hint_merge": (ctypes.c_int, [_c_i32p, _i64, _i32, _c_i32p, _i32, _i32, _i32, _c_i32p, _c_i32p, _i32,
                                      _i32, _c_i32p, _i64, _c_i32p, _c_i32p, _c_i32p, _c_i32p]),
    "ooo_tree_attn_workspace": (_sz, [_i32, _i32, _i32, _i32, _i32, ctypes.c_int]),
    "ooo_tree_attn": (ctypes.c_int, [_vp, _vp, _vp, _i64, _i32, _vp, _i32, _vp, _i32, _i32, _i32, _i32,
                                     ctypes.c_float, ctypes.c_int, _vp, _vp, _sz, _vp]),
    "ooo_tree_attn_workspace_ex": (_sz, [_i32, _i32, _i32, _i32, _i32, ctypes.c_int, _i32]),
    "ooo_tree_attn_noalloc": (ctypes.c_int, [_vp, _vp, _vp, _i64, _i32, _vp, _i32, _vp, _i32, _i32, _i32, _i32,
                                             ctypes.c_float, ctypes.c_int, _vp, _vp]),
    "ooo_tree_attn_noalloc_scratch_bytes": (_sz, []),
    "ooo_tree_attn_ex": (ctypes.c_int, [_vp, _vp, _vp, _i64, _i32, _vp, _i32, _vp, _i32, _i32, _i32, _i32,
                                        ctypes.c_float, ctypes.c_int, _vp, _vp, _sz, _vp, _i32, _i32]),
    "ooo_lmhead_workspace": (_sz, [_i32, _i32, _i32, ctypes.c_int]),
    "ooo_lmhead_packed_bytes": (_sz, [_i32, _i32, ctypes.c_int]),
    "ooo_lmhead_pack": (ctypes.c_int, [_vp, _i32, _i32, ctypes.c_int, _vp, _sz, _vp]),
    "ooo_lmhead_argmax": (ctypes.c_int, [_vp, _vp, _i32, _i32, _i32, ctypes.c_int, _i32, _vp, _vp, _vp, _vp, _sz,
                                         _vp]),
    "ooo_accept": (ctypes.c_int, [_vp, _vp, _vp, _vp, _i32, _vp, _i32, _i32, _i32, _vp, _vp, _vp, _vp]),
    "ooo_kv_compact": (ctypes.c_int, [_vp, _vp, _i32, _i32, _i64, _i32, ctypes.c_int, _i32, _vp, _i32, _vp, _vp,
                                      _i32, _vp]),
    "ooo_embed_rows": (ctypes.c_int, [_vp, _vp, _i32, _i32, _i32, _vp, _vp]),
    "ooo_rmsnorm": (ctypes.c_int, [_vp, _vp, _i32, _i32, ctypes.c_float, _vp, _vp]),
    "ooo_linear_workspace": (_sz, [_i32, _i32, _i32]),
    "ooo_linear_packed_bytes": (_sz, [_i32, _i32]),
    "ooo_linear_pack": (ctypes.c_int, [_vp, _i32, _i32, _vp, _sz, _vp]),
    "ooo_linear": (ctypes.c_int, [_vp, _vp, _i32, _i32, _i32, _i32, ctypes.c_int, _vp, _vp, _sz, _vp]),
    "ooo_qk_norm_rope": (ctypes.c_int, [_vp, _vp, _vp, ctypes.c_float, _vp, _i32, _i32, _vp, ctypes.c_double, _i32,
                                        _i32, _i32, _vp, _vp, _vp, _i64, _vp]),
    "ooo_swiglu": (ctypes.c_int, [_vp, _i32, _i32, _vp, _vp]),
    "ooo_linear_add_rmsnorm": (ctypes.c_int, [_vp, _vp, _i32, _i32, _i32, _i32, _vp, _vp, ctypes.c_float, _vp, _vp,
                                              _sz, _vp]),
    "ooo_linear_qk_norm_rope": (ctypes.c_int, [_vp, _vp, _i32, _i32, _i32, _vp, _vp, ctypes.c_float, _vp, _i32, _vp,
                                               ctypes.c_double, _i32, _i32, _i32, _vp, _vp, _vp, _i64, _vp, _sz,
                                               _vp]),
}


class OooError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"[{status}] {message}")
        self.status = status


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise OSError(f"{LIB_PATH} is missing: build it with `python -m paper_2608_00814_amd.build`")
        h = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(h, name)
            f.restype = res
            f.argtypes = args
        _lib = h
    return _lib


def last_error() -> str:
    return lib().ooo_last_error().decode()


def version() -> int:
    return int(lib().ooo_version())


def _check(status: int) -> None:
    if status != OK:
        raise OooError(status, last_error())


def dtype_code(t) -> int:
    import torch

    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _prefix_ptr(t) -> Optional[int]:
    """Device prefix length: None, or an int32 device tensor (its first element)."""
    if t is None:
        return None
    import torch

    if not t.is_cuda or t.dtype != torch.int32 or t.numel() < 1:
        raise ValueError("prefix_dev must be an int32 device tensor with at least one element")
    return t.data_ptr()


def _dev(t, name: str, contiguous: bool = True):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if contiguous and not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch

        return torch.cuda.current_stream().cuda_stream
    return int(stream) if not hasattr(stream, "cuda_stream") else stream.cuda_stream


# ----------------------------------------------------------------------------
# host


def pack_tree(root_token: int, cand_tokens: np.ndarray, cand_offsets: np.ndarray, max_nodes: int, max_depth: int,
              mask_words: Optional[int] = None) -> dict:
    """ooo_pack_tree on NumPy arrays; outputs trimmed to n_nodes."""
    W = mask_words if mask_words is not None else max(1, (max_nodes + 63) // 64)
    toks = np.ascontiguousarray(cand_tokens, dtype=np.int32)
    offs = np.ascontiguousarray(cand_offsets, dtype=np.int32)
    cap = max(int(max_nodes), 1)
    token = np.zeros(cap, np.int32)
    parent = np.zeros(cap, np.int32)
    depth = np.zeros(cap, np.int32)
    mask = np.zeros(cap * W, np.uint64)
    n = ctypes.c_int32(0)
    trunc = ctypes.c_int32(0)
    st = lib().ooo_pack_tree(int(root_token), toks.ctypes.data_as(_c_i32p) if toks.size else None,
                             offs.ctypes.data_as(_c_i32p), len(offs) - 1, int(max_nodes), int(max_depth),
                             token.ctypes.data_as(_c_i32p), parent.ctypes.data_as(_c_i32p),
                             depth.ctypes.data_as(_c_i32p), mask.ctypes.data_as(_c_u64p), int(W),
                             ctypes.byref(n), ctypes.byref(trunc))
    _check(st)
    k = n.value
    return {"token": token[:k].copy(), "parent": parent[:k].copy(), "depth": depth[:k].copy(),
            "anc_mask": mask.reshape(cap, W)[:k].copy(), "n_nodes": k, "n_truncated": trunc.value,
            "mask_words": W}


def pack_tree_into(root_token: int, cand_tokens: np.ndarray, cand_offsets: np.ndarray, max_nodes: int,
                   max_depth: int, token: np.ndarray, parent: np.ndarray, depth: np.ndarray,
                   anc_mask: np.ndarray) -> tuple:
    """ooo_pack_tree writing straight into caller arrays (for example views
    of a pinned staging buffer): token/parent/depth int32 [>= max_nodes],
    anc_mask uint64 [>= max_nodes][W], all C-contiguous.  Returns
    (n_nodes, n_truncated)."""
    for a, nm, dt in ((token, "token", np.int32), (parent, "parent", np.int32), (depth, "depth", np.int32),
                      (anc_mask, "anc_mask", np.uint64)):
        if a.dtype != dt or not a.flags.c_contiguous or a.shape[0] < max_nodes:
            raise ValueError(f"{nm} must be a C-contiguous {np.dtype(dt).name} array of >= {max_nodes} rows")
    W = 1 if anc_mask.ndim == 1 else int(anc_mask.shape[1])
    toks = np.ascontiguousarray(cand_tokens, dtype=np.int32)
    offs = np.ascontiguousarray(cand_offsets, dtype=np.int32)
    n = ctypes.c_int32(0)
    trunc = ctypes.c_int32(0)
    _check(lib().ooo_pack_tree(int(root_token), toks.ctypes.data_as(_c_i32p) if toks.size else None,
                               offs.ctypes.data_as(_c_i32p), len(offs) - 1, int(max_nodes), int(max_depth),
                               token.ctypes.data_as(_c_i32p), parent.ctypes.data_as(_c_i32p),
                               depth.ctypes.data_as(_c_i32p), anc_mask.ctypes.data_as(_c_u64p), W,
                               ctypes.byref(n), ctypes.byref(trunc)))
    return n.value, trunc.value


class StagedPacker:
    """ooo_pack_tree bound to fixed output arrays (the per-step staging
    buffer): their addresses are resolved once, so a call only marshals the
    candidate arrays.  Returns (n_nodes, n_truncated)."""

    _proto = ctypes.CFUNCTYPE(ctypes.c_int, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                              ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                              ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p)

    def __init__(self, max_nodes: int, max_depth: int, token: np.ndarray, parent: np.ndarray, depth: np.ndarray,
                 anc_mask: np.ndarray):
        for a, nm, dt in ((token, "token", np.int32), (parent, "parent", np.int32), (depth, "depth", np.int32),
                          (anc_mask, "anc_mask", np.uint64)):
            if a.dtype != dt or not a.flags.c_contiguous or a.shape[0] < max_nodes:
                raise ValueError(f"{nm} must be a C-contiguous {np.dtype(dt).name} array of >= {max_nodes} rows")
        self._fn = self._proto(("ooo_pack_tree", lib()))
        self._keep = (token, parent, depth, anc_mask)  # the addresses below stay valid
        self._n, self._trunc = ctypes.c_int32(0), ctypes.c_int32(0)
        W = 1 if anc_mask.ndim == 1 else int(anc_mask.shape[1])
        self._fixed = (int(max_nodes), int(max_depth), token.ctypes.data, parent.ctypes.data, depth.ctypes.data,
                       anc_mask.ctypes.data, W, ctypes.addressof(self._n), ctypes.addressof(self._trunc))

    def __call__(self, root_token: int, cand_tokens: np.ndarray, cand_offsets: np.ndarray) -> tuple:
        if cand_tokens.dtype != np.int32 or not cand_tokens.flags.c_contiguous:
            cand_tokens = np.ascontiguousarray(cand_tokens, dtype=np.int32)
        if cand_offsets.dtype != np.int32 or not cand_offsets.flags.c_contiguous:
            cand_offsets = np.ascontiguousarray(cand_offsets, dtype=np.int32)
        mn, md, t, p, d, m, W, n, tr = self._fixed
        _check(self._fn(int(root_token), cand_tokens.ctypes.data if cand_tokens.size else None,
                        cand_offsets.ctypes.data, cand_offsets.shape[0] - 1, mn, md, t, p, d, m, W, n, tr))
        return self._n.value, self._trunc.value


def hint_merge(bank: np.ndarray, eos_token: int, committed: np.ndarray, native_tokens: np.ndarray,
               native_offsets: np.ndarray, n_lanes: int, max_suffix: int = 7, max_len: int = 64) -> dict:
    """ooo_hint_merge on NumPy arrays: the merged lanes as CSR (tokens,
    offsets), plus how many came from the bank and the suffix length used."""
    b = np.ascontiguousarray(bank, dtype=np.int32)
    cm = np.ascontiguousarray(committed, dtype=np.int32)
    nt = np.ascontiguousarray(native_tokens, dtype=np.int32)
    no = np.ascontiguousarray(native_offsets, dtype=np.int32)
    cap = int(nt.size) + int(n_lanes) * int(max_len)
    out = np.zeros(max(cap, 1), np.int32)
    offs = np.zeros(int(n_lanes) + 1, np.int32)
    n_out, n_hint, slen = ctypes.c_int32(0), ctypes.c_int32(0), ctypes.c_int32(0)
    p = lambda a: a.ctypes.data_as(_c_i32p) if a.size else None
    st = lib().ooo_hint_merge(p(b), int(b.size), int(eos_token), p(cm), int(cm.size), int(max_suffix),
                              int(max_len), p(nt), no.ctypes.data_as(_c_i32p), len(no) - 1, int(n_lanes),
                              out.ctypes.data_as(_c_i32p), cap, offs.ctypes.data_as(_c_i32p), ctypes.byref(n_out),
                              ctypes.byref(n_hint), ctypes.byref(slen))
    _check(st)
    k = n_out.value
    return {"tokens": out[:offs[k]].copy(), "offsets": offs[:k + 1].copy(), "n_out": k, "n_hint": n_hint.value,
            "suffix_len": slen.value}


# ----------------------------------------------------------------------------
# device


def tree_attn_workspace(n_nodes: int, n_q_heads: int, n_kv_heads: int, head_dim: int, prefix_len: int,
                        dtype: int, force_splits: int = 0) -> int:
    """Bytes of attention workspace (``force_splits`` as for ``tree_attn``)."""
    return int(lib().ooo_tree_attn_workspace_ex(n_nodes, n_q_heads, n_kv_heads, head_dim, prefix_len, dtype,
                                                force_splits))


def tree_attn(q, k_cache, v_cache, prefix_len: int, n_nodes: int, anc_mask, n_q_heads: int, n_kv_heads: int,
              scale: float, out, workspace=None, stream=None, prefix_dev=None, force_splits: int = 0,
              variant: int = 0) -> None:
    """q [N][Hq][D]; k_cache/v_cache one layer [Hkv][cap][D]; anc_mask
    [N][W] int64/uint64 device tensor; out [N][Hq][D].  ``prefix_dev``: an
    int32 device tensor whose first element is the prefix length used at run
    time (``prefix_len`` bounds it), or None.  ``force_splits`` (> 0) and
    ``variant`` (1: one wave per row group at head_dim 128) override the
    planner, for tests and tuning."""
    for t, nm in ((q, "q"), (k_cache, "k_cache"), (v_cache, "v_cache"), (anc_mask, "anc_mask"), (out, "out")):
        _dev(t, nm)
    Hkv, cap, D = k_cache.shape
    W = anc_mask.shape[-1]
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().ooo_tree_attn_ex(q.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(), cap, prefix_len,
                                  _prefix_ptr(prefix_dev), n_nodes,
                                  anc_mask.data_ptr(), W, n_q_heads, n_kv_heads, D, float(scale), dtype_code(q),
                                  out.data_ptr(), _ptr(workspace), ws_bytes, _stream(stream), force_splits,
                                  variant))


def tree_attn_noalloc(q, k_cache, v_cache, prefix_len: int, n_nodes: int, anc_mask, n_q_heads: int,
                      n_kv_heads: int, scale: float, out, stream=None, prefix_dev=None) -> None:
    """tree_attn with the library's built-in per-GPU scratch instead of a
    workspace (the call allocates nothing)."""
    for t, nm in ((q, "q"), (k_cache, "k_cache"), (v_cache, "v_cache"), (anc_mask, "anc_mask"), (out, "out")):
        _dev(t, nm)
    Hkv, cap, D = k_cache.shape
    W = anc_mask.shape[-1]
    _check(lib().ooo_tree_attn_noalloc(q.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(), cap, prefix_len,
                                       _prefix_ptr(prefix_dev), n_nodes, anc_mask.data_ptr(), W, n_q_heads,
                                       n_kv_heads, D, float(scale), dtype_code(q), out.data_ptr(), _stream(stream)))


def lmhead_workspace(n_nodes: int, hidden_dim: int, vocab: int, dtype: int) -> int:
    return int(lib().ooo_lmhead_workspace(n_nodes, hidden_dim, vocab, dtype))


class PackedWeight:
    """LM-head weight in the streaming layout of ooo_lmhead_pack: a flat
    uint8 device tensor plus the logical [vocab][hidden_dim] shape."""

    def __init__(self, data, vocab: int, hidden_dim: int, dtype: int):
        self.data, self.vocab, self.hidden_dim, self.dtype = data, vocab, hidden_dim, dtype


def lmhead_pack(weight, stream=None) -> PackedWeight:
    """Packs a [V][H] bf16 device weight (allocates the packed copy)."""
    import torch
    _dev(weight, "weight")
    V, H = weight.shape
    code = dtype_code(weight)
    need = int(lib().ooo_lmhead_packed_bytes(V, H, code))
    if need == 0:
        raise OooError(ERR_UNSUPPORTED, f"no packed layout for {tuple(weight.shape)} {weight.dtype}")
    data = torch.empty(need, dtype=torch.uint8, device=weight.device)
    _check(lib().ooo_lmhead_pack(weight.data_ptr(), V, H, code, data.data_ptr(), need, _stream(stream)))
    return PackedWeight(data, V, H, code)


def lmhead_argmax(hidden, weight, argmax_ids, max_logit, logits=None, workspace=None, stream=None) -> None:
    """hidden [N][H]; weight [V][H] device tensor or a PackedWeight;
    argmax_ids int32 [N]; max_logit float32 [N]; logits optional float32 [N][V]."""
    packed = isinstance(weight, PackedWeight)
    wt = weight.data if packed else weight
    for t, nm in ((hidden, "hidden"), (wt, "weight"), (argmax_ids, "argmax_ids"), (max_logit, "max_logit")):
        _dev(t, nm)
    if logits is not None:
        _dev(logits, "logits")
    N, H = hidden.shape
    if packed:
        if weight.hidden_dim != H or weight.dtype != dtype_code(hidden):
            raise OooError(ERR_INVALID, "packed weight does not match the hidden rows")
        V = weight.vocab
    else:
        V = weight.shape[0]
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().ooo_lmhead_argmax(hidden.data_ptr(), wt.data_ptr(), N, H, V, dtype_code(hidden),
                                   W_PACKED if packed else W_ROWS, argmax_ids.data_ptr(), max_logit.data_ptr(),
                                   _ptr(logits), _ptr(workspace), ws_bytes, _stream(stream)))


def accept(token, parent, depth, anc_mask, argmax_ids, n_nodes: int, path, accept_len, bonus_token,
           stream=None, max_depth: Optional[int] = None) -> None:
    """All device int32 tensors (anc_mask int64 [N][W]); path [path_cap];
    ``max_depth`` defaults to path_cap - 1.  accept_len comes back -1 when
    the accepted path runs deeper than path_cap - 1 (nothing committed)."""
    for t, nm in ((token, "token"), (parent, "parent"), (depth, "depth"), (anc_mask, "anc_mask"),
                  (argmax_ids, "argmax_ids"), (path, "path"), (accept_len, "accept_len"),
                  (bonus_token, "bonus_token")):
        _dev(t, nm)
    W = anc_mask.shape[-1]
    md = path.numel() - 1 if max_depth is None else max_depth
    _check(lib().ooo_accept(token.data_ptr(), parent.data_ptr(), depth.data_ptr(), anc_mask.data_ptr(), W,
                            argmax_ids.data_ptr(), n_nodes, md, path.numel(), path.data_ptr(),
                            accept_len.data_ptr(), bonus_token.data_ptr(), _stream(stream)))


def kv_compact(k_cache, v_cache, prefix_len: int, n_nodes: int, path, accept_len, stream=None,
               prefix_dev=None) -> None:
    """k_cache/v_cache [L][Hkv][cap][D] contiguous, updated in place;
    ``prefix_dev`` as for ``tree_attn``."""
    for t, nm in ((k_cache, "k_cache"), (v_cache, "v_cache"), (path, "path"), (accept_len, "accept_len")):
        _dev(t, nm)
    L, Hkv, cap, D = k_cache.shape
    _check(lib().ooo_kv_compact(k_cache.data_ptr(), v_cache.data_ptr(), L, Hkv, cap, D, dtype_code(k_cache),
                                prefix_len, _prefix_ptr(prefix_dev), n_nodes, path.data_ptr(), accept_len.data_ptr(),
                                path.numel(),
                                _stream(stream)))


# ----------------------------------------------------------------------------
# decoder layer around the path


def embed_rows(table, tokens, n_nodes: int, h, stream=None) -> None:
    """table [V][H] bf16; tokens [>= n_nodes] int32; h [>= n_nodes][H] float32."""
    for t, nm in ((table, "table"), (tokens, "tokens"), (h, "h")):
        _dev(t, nm)
    V, H = table.shape
    _check(lib().ooo_embed_rows(table.data_ptr(), tokens.data_ptr(), n_nodes, H, V, h.data_ptr(), _stream(stream)))


def rmsnorm(h, weight, eps: float, out, n_rows: Optional[int] = None, stream=None) -> None:
    """h [rows][dim] float32; weight [dim] bf16; out [rows][dim] bf16."""
    for t, nm in ((h, "h"), (weight, "weight"), (out, "out")):
        _dev(t, nm)
    n = h.shape[0] if n_rows is None else n_rows
    _check(lib().ooo_rmsnorm(h.data_ptr(), weight.data_ptr(), n, h.shape[-1], float(eps), out.data_ptr(),
                             _stream(stream)))


def linear_workspace(n_rows: int, in_dim: int, out_dim: int) -> int:
    return int(lib().ooo_linear_workspace(n_rows, in_dim, out_dim))


class PackedLinear:
    """A projection weight in the streaming layout of ooo_linear_pack: a flat
    uint8 device tensor plus the logical [out_dim][in_dim] shape."""

    def __init__(self, data, out_dim: int, in_dim: int):
        self.data, self.out_dim, self.in_dim = data, out_dim, in_dim
        self.shape = (out_dim, in_dim)


def linear_pack(weight, stream=None) -> PackedLinear:
    """Packs a [out][in] bf16 device weight (allocates the packed copy)."""
    import torch
    _dev(weight, "weight")
    O, K = weight.shape
    need = int(lib().ooo_linear_packed_bytes(O, K))
    if need == 0:
        raise OooError(ERR_UNSUPPORTED, f"ooo_linear_pack: cannot pack a [{O}][{K}] weight")
    data = torch.empty(need, dtype=torch.uint8, device=weight.device)
    _check(lib().ooo_linear_pack(weight.data_ptr(), O, K, data.data_ptr(), need, _stream(stream)))
    return PackedLinear(data, O, K)


def linear(x, weight, out, epilogue: int, workspace, n_rows: Optional[int] = None, stream=None) -> None:
    """out (epilogue)= x[:n] @ weight.T: x bf16 [rows][in]; weight bf16
    [out][in] or a PackedLinear; out float32 or bf16 per the epilogue."""
    _dev(x, "x")
    _dev(out, "out")
    n = x.shape[0] if n_rows is None else n_rows
    if isinstance(weight, PackedLinear):
        wptr, layout, (O, K) = weight.data.data_ptr(), W_PACKED, weight.shape
    else:
        _dev(weight, "weight")
        wptr, layout, (O, K) = weight.data_ptr(), W_ROWS, weight.shape
    ws_bytes = workspace.numel() * workspace.element_size()
    _check(lib().ooo_linear(x.data_ptr(), wptr, n, K, O, layout, int(epilogue), out.data_ptr(), workspace.data_ptr(),
                            ws_bytes, _stream(stream)))


def _weight_args(weight):
    if isinstance(weight, PackedLinear):
        return weight.data.data_ptr(), W_PACKED, weight.shape
    _dev(weight, "weight")
    return weight.data_ptr(), W_ROWS, tuple(weight.shape)


def linear_add_rmsnorm(x, weight, residual, norm_weight, eps: float, normed_out, workspace,
                       n_rows: Optional[int] = None, stream=None) -> None:
    """residual[:n] += x[:n] @ weight.T (float32 rows, in place), then
    normed_out[:n] = rmsnorm(residual[:n]) * norm_weight in bf16."""
    for t, nm in ((x, "x"), (residual, "residual"), (norm_weight, "norm_weight"), (normed_out, "normed_out")):
        _dev(t, nm)
    n = x.shape[0] if n_rows is None else n_rows
    wptr, layout, (O, K) = _weight_args(weight)
    ws_bytes = workspace.numel() * workspace.element_size()
    _check(lib().ooo_linear_add_rmsnorm(x.data_ptr(), wptr, n, K, O, layout, residual.data_ptr(),
                                        norm_weight.data_ptr(), float(eps), normed_out.data_ptr(),
                                        workspace.data_ptr(), ws_bytes, _stream(stream)))


def linear_qk_norm_rope(x, weight, q_norm, k_norm, eps: float, depth, n_nodes: int, prefix_len: int,
                        rope_theta: float, n_q_heads: int, n_kv_heads: int, q_out, k_cache, v_cache, workspace,
                        stream=None, prefix_dev=None) -> None:
    """The fused q/k/v projection of x[:n] followed by the q/k norms, the
    rotation at P + depth and the cache writes (as ``qk_norm_rope`` on the
    projection's float32 sums)."""
    for t, nm in ((x, "x"), (depth, "depth"), (q_out, "q_out"), (k_cache, "k_cache"), (v_cache, "v_cache")):
        _dev(t, nm)
    wptr, layout, (O, K) = _weight_args(weight)
    _, cap, D = k_cache.shape
    if O != (n_q_heads + 2 * n_kv_heads) * D:
        raise ValueError(f"weight has {O} rows, expected (Hq + 2 Hkv) * D = {(n_q_heads + 2 * n_kv_heads) * D}")
    ws_bytes = workspace.numel() * workspace.element_size()
    _check(lib().ooo_linear_qk_norm_rope(x.data_ptr(), wptr, n_nodes, K, layout, _ptr(q_norm), _ptr(k_norm),
                                         float(eps), depth.data_ptr(), prefix_len, _prefix_ptr(prefix_dev),
                                         float(rope_theta), n_q_heads, n_kv_heads, D, q_out.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(), cap,
                                         workspace.data_ptr(), ws_bytes, _stream(stream)))


def qk_norm_rope(qkv, q_norm, k_norm, eps: float, depth, n_nodes: int, prefix_len: int, rope_theta: float,
                 n_q_heads: int, n_kv_heads: int, q_out, k_cache, v_cache, stream=None, prefix_dev=None) -> None:
    """qkv [N][(Hq + 2 Hkv) D] bf16; q_norm/k_norm [D] bf16 or None; depth
    [>= N] int32; q_out [N][Hq][D]; k_cache/v_cache one layer [Hkv][cap][D];
    ``prefix_dev`` as for ``tree_attn``."""
    for t, nm in ((qkv, "qkv"), (depth, "depth"), (q_out, "q_out"), (k_cache, "k_cache"), (v_cache, "v_cache")):
        _dev(t, nm)
    _, cap, D = k_cache.shape
    _check(lib().ooo_qk_norm_rope(qkv.data_ptr(), _ptr(q_norm), _ptr(k_norm), float(eps), depth.data_ptr(), n_nodes,
                                  prefix_len, _prefix_ptr(prefix_dev), float(rope_theta), n_q_heads, n_kv_heads, D,
                                  q_out.data_ptr(),
                                  k_cache.data_ptr(), v_cache.data_ptr(), cap, _stream(stream)))


def swiglu(gate_up, out, n_rows: Optional[int] = None, stream=None) -> None:
    """gate_up [rows][2 I] float32 (gate rows, then up rows) -> out [rows][I] bf16."""
    _dev(gate_up, "gate_up")
    _dev(out, "out")
    n = gate_up.shape[0] if n_rows is None else n_rows
    _check(lib().ooo_swiglu(gate_up.data_ptr(), n, out.shape[-1], out.data_ptr(), _stream(stream)))
