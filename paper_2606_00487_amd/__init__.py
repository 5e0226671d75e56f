"""TAPS draft-tree verification hot path on MI355X (gfx950).

Thin Python binding over libtaps.so (include/taps.h): argument marshalling
only, every step of the path runs in the HIP kernels.  PyTorch provides device
memory and the current stream.

    sel = Selector(batch, block, vocab, K, budget, dtype=BF16, kind=LOGITS)
    tree = sel(marginals)                       # taps_select
    att = TreeAttention(batch, budget, Hq, Hkv, head_dim, max_ctx)
    O = att(Q, K, V, kv_offset, ctx_len, tree.parent, tree.n_nodes)   # tree_verify_attn
    walk = AcceptWalk(batch, budget, block)
    path, path_len, bonus = walk(tree, target_tokens)                 # accept_walk
    com = KVCommit(batch, budget, block, Hkv, head_dim, max_ctx)
    new_ctx, tokens, n = com(K, V, kv_offset, ctx_len, tree, path, path_len, bonus)  # kv_commit
    lay = VerifyLayer(batch, budget, Hq, Hkv, head_dim, hidden, max_ctx)
    Y = lay(X, LayerWeights(Wq, Wk, Wv, Wo, q_norm, k_norm), K, V, kv_offset, ctx_len, tree)
"""
from __future__ import annotations

import ctypes
import dataclasses

import torch

from . import _lib
from ._lib import (TAPS_BF16 as BF16, TAPS_FP32 as FP32, TAPS_LOGITS as LOGITS,  # noqa: F401
                   TAPS_PROBS as PROBS, TAPS_SCORER_LEARNED as LEARNED,
                   TAPS_SCORER_MARGINAL as MARGINAL, TAPS_SCORER_SIBLING as SIBLING, TapsError,
                   load)

_TORCH_DT = {BF16: torch.bfloat16, FP32: torch.float32}


def _ptr(t: torch.Tensor | None) -> int | None:
    return None if t is None else t.data_ptr()


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def _need(t: torch.Tensor, name: str, dtype, shape=None):
    if t.dtype != dtype:
        raise TypeError(f"{name}: expected {dtype}, got {t.dtype}")
    if not t.is_cuda:
        raise TypeError(f"{name}: expected a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name}: must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: expected shape {tuple(shape)}, got {tuple(t.shape)}")


@dataclasses.dataclass
class TreeBuffers:
    """Device arrays of taps_tree (see include/taps.h)."""
    parent: torch.Tensor
    token: torch.Tensor
    depth: torch.Tensor
    rank: torch.Tensor
    q_reach: torch.Tensor
    n_nodes: torch.Tensor
    topk_idx: torch.Tensor
    topk_val: torch.Tensor

    @staticmethod
    def empty(batch, block, K, budget, device="cuda"):
        i32 = dict(dtype=torch.int32, device=device)
        return TreeBuffers(
            parent=torch.empty(batch, budget, **i32), token=torch.empty(batch, budget, **i32),
            depth=torch.empty(batch, budget, **i32), rank=torch.empty(batch, budget, **i32),
            q_reach=torch.empty(batch, budget, dtype=torch.float64, device=device),
            n_nodes=torch.empty(batch, **i32), topk_idx=torch.empty(batch, block, K, **i32),
            topk_val=torch.empty(batch, block, K, dtype=torch.float32, device=device))

    def struct(self) -> _lib.Tree:
        return _lib.Tree(_ptr(self.parent), _ptr(self.token), _ptr(self.depth), _ptr(self.rank),
                         _ptr(self.q_reach), _ptr(self.n_nodes), _ptr(self.topk_idx),
                         _ptr(self.topk_val))


@dataclasses.dataclass
class ScorerWeights:
    """Device weights of the learned-scorer hook (taps_scorer_mlp): float32 emb [vocab][d],
    W1 [h][2d+3], b1 [h], w2 [h], the float b2 and int32 root_token [batch]."""
    emb: torch.Tensor
    W1: torch.Tensor
    b1: torch.Tensor
    w2: torch.Tensor
    b2: float
    root_token: torch.Tensor

    def struct(self) -> _lib.ScorerMLP:
        d, h = self.emb.shape[1], self.W1.shape[0]
        _need(self.emb, "emb", torch.float32)
        _need(self.W1, "W1", torch.float32, (h, 2 * d + 3))
        _need(self.b1, "b1", torch.float32, (h,))
        _need(self.w2, "w2", torch.float32, (h,))
        _need(self.root_token, "root_token", torch.int32)
        return _lib.ScorerMLP(_ptr(self.emb), _ptr(self.W1), _ptr(self.b1), _ptr(self.w2),
                              float(self.b2), _ptr(self.root_token), d, h)


class Selector:
    """taps_select: top-K, Eq. 1-3 and the budgeted prefix-closed selection of Alg. 1."""

    def __init__(self, batch, block, vocab, K, budget, dtype=BF16, kind=LOGITS, lambda1=1.0,
                 lambda2=0.125, tau=0.0, beta=1.0, scorer=SIBLING, mlp=None, device="cuda"):
        """scorer: SIBLING (sibling softmax over the K candidates), MARGINAL (the drafter's
        full-vocabulary marginal: the scoring ablation) or LEARNED (the learned-scorer hook,
        whose weights `mlp` (ScorerWeights) must stay alive while the Selector is used)."""
        self.lib = load()
        self.mlp = mlp
        self._mlp_struct = mlp.struct() if mlp is not None else None
        self.p = _lib.SelectParams(batch, block, vocab, K, budget, dtype, kind, lambda1, lambda2,
                                   tau, beta, scorer,
                                   ctypes.pointer(self._mlp_struct) if mlp is not None else None)
        _lib.check(self.lib, "taps_select_validate", self.lib.taps_select_validate(ctypes.byref(self.p)))
        self.ws_bytes = self.lib.taps_select_workspace_bytes(ctypes.byref(self.p))
        self.ws = torch.empty(max(self.ws_bytes, 8), dtype=torch.uint8, device=device)
        self.tree = TreeBuffers.empty(batch, block, K, budget, device)
        self._tree_struct = self.tree.struct()

    def __call__(self, marginals: torch.Tensor, tree: TreeBuffers | None = None) -> TreeBuffers:
        p = self.p
        _need(marginals, "marginals", _TORCH_DT[p.dtype], (p.batch, p.block, p.vocab))
        t = tree or self.tree
        st = t.struct() if tree is not None else self._tree_struct
        _lib.check(self.lib, "taps_select",
                   self.lib.taps_select(_ptr(marginals), ctypes.byref(p), ctypes.byref(st),
                                        _ptr(self.ws), self.ws_bytes, _stream()))
        return t

    def noalloc(self, marginals: torch.Tensor, tree: TreeBuffers | None = None) -> TreeBuffers:
        """taps_select_noalloc: the same selection with the library's static scratch instead
        of this Selector's workspace (for callers that cannot allocate)."""
        p = self.p
        _need(marginals, "marginals", _TORCH_DT[p.dtype], (p.batch, p.block, p.vocab))
        t = tree or self.tree
        st = t.struct() if tree is not None else self._tree_struct
        _lib.check(self.lib, "taps_select_noalloc",
                   self.lib.taps_select_noalloc(_ptr(marginals), ctypes.byref(p),
                                                ctypes.byref(st), _stream()))
        return t


class TreeAttention:
    """tree_verify_attn: tree-masked verification attention."""

    def __init__(self, batch, budget, Hq, Hkv, head_dim, max_ctx, dtype=BF16, scale=None,
                 device="cuda"):
        self.lib = load()
        self.shape = (batch, budget, Hq, Hkv, head_dim, max_ctx, dtype)
        self.scale = float(scale if scale is not None else head_dim ** -0.5)
        _lib.check(self.lib, "tree_verify_attn_validate",
                   self.lib.tree_verify_attn_validate(batch, budget, Hq, Hkv, head_dim, max_ctx,
                                                      dtype, self.scale))
        self.ws_bytes = self.lib.tree_verify_attn_workspace_bytes(batch, budget, Hq, Hkv,
                                                                  head_dim, max_ctx, dtype)
        self.ws = torch.empty(max(self.ws_bytes, 16), dtype=torch.uint8, device=device)

    def __call__(self, Q, K, V, kv_offset, ctx_len, parent, n_nodes, out=None, events=None):
        """events: optional (begin, end) torch.cuda.Event pair recorded around the main
        attention kernel only (tree_verify_attn_timed)."""
        batch, budget, Hq, Hkv, hd, max_ctx, dtype = self.shape
        tdt = _TORCH_DT[dtype]
        _need(Q, "Q_tree", tdt, (batch, budget, Hq, hd))
        _need(K, "K_cache", tdt)
        _need(V, "V_cache", tdt, tuple(K.shape))
        if K.dim() != 3 or K.shape[1:] != (Hkv, hd):
            raise ValueError(f"K_cache: expected [rows, {Hkv}, {hd}], got {tuple(K.shape)}")
        _need(kv_offset, "kv_offset", torch.int64, (batch,))
        _need(ctx_len, "ctx_len", torch.int32, (batch,))
        _need(parent, "tree_parent", torch.int32, (batch, budget))
        _need(n_nodes, "n_nodes", torch.int32, (batch,))
        O = out if out is not None else torch.empty_like(Q)
        _need(O, "O", tdt, (batch, budget, Hq, hd))
        args = (_ptr(Q), _ptr(K), _ptr(V), _ptr(kv_offset), _ptr(ctx_len), _ptr(parent),
                _ptr(n_nodes), batch, budget, Hq, Hkv, hd, max_ctx, dtype, self.scale, _ptr(O),
                _ptr(self.ws), self.ws_bytes, _stream())
        if events is None:
            _lib.check(self.lib, "tree_verify_attn", self.lib.tree_verify_attn(*args))
        else:
            _lib.check(self.lib, "tree_verify_attn_timed", self.lib.tree_verify_attn_timed(
                *args, events[0].cuda_event, events[1].cuda_event))
        return O


class PagedTreeAttention:
    """tree_verify_attn_paged: tree_verify_attn over a paged KV cache (bf16, head_dim 128)."""

    def __init__(self, batch, budget, Hq, Hkv, max_ctx, page_rows, scale=None, device="cuda"):
        self.lib = load()
        hd = 128
        self.shape = (batch, budget, Hq, Hkv, hd, max_ctx)
        self.page_rows = int(page_rows)
        self.scale = float(scale if scale is not None else hd ** -0.5)
        self.ws_bytes = self.lib.tree_verify_attn_paged_workspace_bytes(
            batch, budget, Hq, Hkv, hd, max_ctx, self.page_rows)
        self.ws = torch.empty(max(self.ws_bytes, 16), dtype=torch.uint8, device=device)

    def __call__(self, Q, K_pages, V_pages, block_table, ctx_len, parent, n_nodes, out=None,
                 events=None):
        """K_pages, V_pages: [num_pages, page_rows, Hkv, 128] bf16; block_table: [batch,
        max_pages] int32 page ids (request b's logical row r at page block_table[b, r //
        page_rows], slot r % page_rows).  events: optional (begin, end) pair recorded around
        the main attention kernel only (tree_verify_attn_paged_timed)."""
        batch, budget, Hq, Hkv, hd, max_ctx = self.shape
        _need(Q, "Q_tree", torch.bfloat16, (batch, budget, Hq, hd))
        _need(K_pages, "K_pages", torch.bfloat16)
        if K_pages.dim() != 4 or K_pages.shape[1:] != (self.page_rows, Hkv, hd):
            raise ValueError(f"K_pages: expected [pages, {self.page_rows}, {Hkv}, {hd}], "
                             f"got {tuple(K_pages.shape)}")
        _need(V_pages, "V_pages", torch.bfloat16, tuple(K_pages.shape))
        _need(block_table, "block_table", torch.int32)
        if block_table.dim() != 2 or block_table.shape[0] != batch:
            raise ValueError(f"block_table: expected [{batch}, max_pages], "
                             f"got {tuple(block_table.shape)}")
        _need(ctx_len, "ctx_len", torch.int32, (batch,))
        _need(parent, "tree_parent", torch.int32, (batch, budget))
        _need(n_nodes, "n_nodes", torch.int32, (batch,))
        O = out if out is not None else torch.empty_like(Q)
        _need(O, "O", torch.bfloat16, (batch, budget, Hq, hd))
        args = (_ptr(Q), _ptr(K_pages), _ptr(V_pages), K_pages.shape[0], self.page_rows,
                _ptr(block_table), block_table.shape[1], _ptr(ctx_len), _ptr(parent),
                _ptr(n_nodes), batch, budget, Hq, Hkv, hd, max_ctx, BF16, self.scale, _ptr(O),
                _ptr(self.ws), self.ws_bytes, _stream())
        if events is None:
            _lib.check(self.lib, "tree_verify_attn_paged", self.lib.tree_verify_attn_paged(*args))
        else:
            _lib.check(self.lib, "tree_verify_attn_paged_timed",
                       self.lib.tree_verify_attn_paged_timed(*args, events[0].cuda_event,
                                                             events[1].cuda_event))
        return O


class AcceptWalk:
    """accept_walk: greedy acceptance of the longest matching root path."""

    def __init__(self, batch, budget, block, device="cuda"):
        self.lib = load()
        self.batch, self.budget, self.block = batch, budget, block
        self.path = torch.empty(batch, block + 1, dtype=torch.int32, device=device)
        self.path_len = torch.empty(batch, dtype=torch.int32, device=device)
        self.bonus = torch.empty(batch, dtype=torch.int32, device=device)

    def __call__(self, tree: TreeBuffers, target_tokens: torch.Tensor):
        _need(target_tokens, "target_tokens", torch.int32, (self.batch, self.budget))
        st = tree.struct()
        _lib.check(self.lib, "accept_walk", self.lib.accept_walk(
            ctypes.byref(st), self.batch, self.budget, self.block, _ptr(target_tokens),
            _ptr(self.path), _ptr(self.path_len), _ptr(self.bonus), _stream()))
        return self.path, self.path_len, self.bonus


class KVCommit:
    """kv_commit: the accepted path's tree K/V rows move to the rows after the context
    (in place), and the round's emitted tokens."""

    def __init__(self, batch, budget, block, Hkv, head_dim, max_ctx, dtype=BF16, device="cuda"):
        self.lib = load()
        self.shape = (batch, budget, block, Hkv, head_dim, max_ctx, dtype)
        self.new_ctx = torch.empty(batch, dtype=torch.int32, device=device)
        self.committed = torch.empty(batch, block + 1, dtype=torch.int32, device=device)
        self.n_committed = torch.empty(batch, dtype=torch.int32, device=device)

    def __call__(self, K, V, kv_offset, ctx_len, tree: TreeBuffers, path, path_len, bonus):
        batch, budget, block, Hkv, hd, max_ctx, dtype = self.shape
        tdt = _TORCH_DT[dtype]
        _need(K, "K_cache", tdt)
        _need(V, "V_cache", tdt, tuple(K.shape))
        if K.dim() != 3 or K.shape[1:] != (Hkv, hd):
            raise ValueError(f"K_cache: expected [rows, {Hkv}, {hd}], got {tuple(K.shape)}")
        _need(kv_offset, "kv_offset", torch.int64, (batch,))
        _need(ctx_len, "ctx_len", torch.int32, (batch,))
        _need(tree.token, "tree.token", torch.int32, (batch, budget))
        _need(path, "path", torch.int32, (batch, block + 1))
        _need(path_len, "path_len", torch.int32, (batch,))
        _need(bonus, "bonus", torch.int32, (batch,))
        st = tree.struct()
        _lib.check(self.lib, "kv_commit", self.lib.kv_commit(
            _ptr(K), _ptr(V), _ptr(kv_offset), _ptr(ctx_len), ctypes.byref(st), _ptr(path),
            _ptr(path_len), _ptr(bonus), batch, budget, block, Hkv, hd, max_ctx, dtype,
            _ptr(self.new_ctx), _ptr(self.committed), _ptr(self.n_committed), _stream()))
        return self.new_ctx, self.committed, self.n_committed


class PagedKVCommit:
    """kv_commit_paged: kv_commit on a paged cache (pools [num_pages, page_rows, Hkv,
    head_dim] and a block table [batch, max_pages], as for PagedTreeAttention)."""

    def __init__(self, batch, budget, block, Hkv, head_dim, max_ctx, page_rows, dtype=BF16,
                 device="cuda"):
        self.lib = load()
        self.shape = (batch, budget, block, Hkv, head_dim, max_ctx, dtype)
        self.page_rows = int(page_rows)
        self.new_ctx = torch.empty(batch, dtype=torch.int32, device=device)
        self.committed = torch.empty(batch, block + 1, dtype=torch.int32, device=device)
        self.n_committed = torch.empty(batch, dtype=torch.int32, device=device)

    def __call__(self, K_pages, V_pages, block_table, ctx_len, tree: TreeBuffers, path, path_len,
                 bonus):
        batch, budget, block, Hkv, hd, max_ctx, dtype = self.shape
        tdt = _TORCH_DT[dtype]
        _need(K_pages, "K_pages", tdt)
        _need(V_pages, "V_pages", tdt, tuple(K_pages.shape))
        if K_pages.dim() != 4 or K_pages.shape[1:] != (self.page_rows, Hkv, hd):
            raise ValueError(f"K_pages: expected [pages, {self.page_rows}, {Hkv}, {hd}], "
                             f"got {tuple(K_pages.shape)}")
        _need(block_table, "block_table", torch.int32)
        if block_table.dim() != 2 or block_table.shape[0] != batch:
            raise ValueError(f"block_table: expected [{batch}, max_pages], "
                             f"got {tuple(block_table.shape)}")
        _need(ctx_len, "ctx_len", torch.int32, (batch,))
        _need(tree.token, "tree.token", torch.int32, (batch, budget))
        _need(path, "path", torch.int32, (batch, block + 1))
        _need(path_len, "path_len", torch.int32, (batch,))
        _need(bonus, "bonus", torch.int32, (batch,))
        st = tree.struct()
        _lib.check(self.lib, "kv_commit_paged", self.lib.kv_commit_paged(
            _ptr(K_pages), _ptr(V_pages), K_pages.shape[0], self.page_rows, _ptr(block_table),
            block_table.shape[1], _ptr(ctx_len), ctypes.byref(st), _ptr(path), _ptr(path_len),
            _ptr(bonus), batch, budget, block, Hkv, hd, max_ctx, dtype, _ptr(self.new_ctx),
            _ptr(self.committed), _ptr(self.n_committed), _stream()))
        return self.new_ctx, self.committed, self.n_committed


@dataclasses.dataclass
class LayerWeights:
    """Device bf16 weights of one attention layer (taps_layer_weights), row-major [out][in]:
    Wq [Hq*hd][hidden], Wk and Wv [Hkv*hd][hidden], Wo [hidden][Hq*hd], q_norm and k_norm
    [hd]."""
    Wq: torch.Tensor
    Wk: torch.Tensor
    Wv: torch.Tensor
    Wo: torch.Tensor
    q_norm: torch.Tensor
    k_norm: torch.Tensor
    rope_theta: float = 1e6
    norm_eps: float = 1e-6

    def struct(self) -> _lib.LayerWeights:
        hidden = self.Wq.shape[1]
        for name in ("Wq", "Wk", "Wv", "Wo", "q_norm", "k_norm"):
            _need(getattr(self, name), name, torch.bfloat16)
        _need(self.Wo, "Wo", torch.bfloat16, (hidden, self.Wq.shape[0]))
        return _lib.LayerWeights(_ptr(self.Wq), _ptr(self.Wk), _ptr(self.Wv), _ptr(self.Wo),
                                 _ptr(self.q_norm), _ptr(self.k_norm), float(self.rope_theta),
                                 float(self.norm_eps), hidden)


class VerifyLayer:
    """verify_layer: one attention layer of the target over the selected trees
    (projections, per-head RMSNorm, rotary positions by tree depth, tree attention,
    output projection)."""

    def __init__(self, batch, budget, Hq, Hkv, head_dim, hidden, max_ctx, scale=None,
                 device="cuda"):
        self.lib = load()
        self.scale = float(scale if scale is not None else head_dim ** -0.5)
        self.shape = (batch, budget, Hq, Hkv, head_dim, hidden, max_ctx)
        nbytes = self.lib.verify_layer_workspace_bytes(batch, budget, Hq, Hkv, head_dim, hidden,
                                                       max_ctx)
        if batch > 0 and nbytes == 0:
            raise TapsError("verify_layer_workspace_bytes", _lib.TAPS_ERR_UNSUPPORTED)
        self.ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
        self.Y = torch.empty((batch, budget, hidden), dtype=torch.bfloat16, device=device)

    def __call__(self, X, w: LayerWeights, K, V, kv_offset, ctx_len, tree: TreeBuffers):
        batch, budget, Hq, Hkv, hd, hidden, max_ctx = self.shape
        _need(X, "X", torch.bfloat16, (batch, budget, hidden))
        _need(K, "K_cache", torch.bfloat16)
        _need(V, "V_cache", torch.bfloat16, tuple(K.shape))
        _need(kv_offset, "kv_offset", torch.int64, (batch,))
        _need(ctx_len, "ctx_len", torch.int32, (batch,))
        ws = w.struct()
        if ws.hidden != hidden:
            raise ValueError(f"weights: hidden {ws.hidden}, expected {hidden}")
        st = tree.struct()
        _lib.check(self.lib, "verify_layer", self.lib.verify_layer(
            _ptr(X), ctypes.byref(ws), _ptr(K), _ptr(V), _ptr(kv_offset), _ptr(ctx_len),
            ctypes.byref(st), batch, budget, Hq, Hkv, hd, max_ctx, self.scale, _ptr(self.Y),
            _ptr(self.ws), self.ws.numel(), _stream()))
        return self.Y


class PagedVerifyLayer:
    """verify_layer_paged: verify_layer over a paged KV cache (pools [num_pages, page_rows,
    Hkv, head_dim] and a block table [batch, max_pages], as for PagedTreeAttention)."""

    def __init__(self, batch, budget, Hq, Hkv, head_dim, hidden, max_ctx, page_rows, scale=None,
                 device="cuda"):
        self.lib = load()
        self.scale = float(scale if scale is not None else head_dim ** -0.5)
        self.shape = (batch, budget, Hq, Hkv, head_dim, hidden, max_ctx)
        self.page_rows = int(page_rows)
        nbytes = self.lib.verify_layer_paged_workspace_bytes(batch, budget, Hq, Hkv, head_dim,
                                                             hidden, max_ctx, self.page_rows)
        if batch > 0 and nbytes == 0:
            raise TapsError("verify_layer_paged_workspace_bytes", _lib.TAPS_ERR_UNSUPPORTED)
        self.ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
        self.Y = torch.empty((batch, budget, hidden), dtype=torch.bfloat16, device=device)

    def __call__(self, X, w: LayerWeights, K_pages, V_pages, block_table, ctx_len,
                 tree: TreeBuffers):
        batch, budget, Hq, Hkv, hd, hidden, max_ctx = self.shape
        _need(X, "X", torch.bfloat16, (batch, budget, hidden))
        _need(K_pages, "K_pages", torch.bfloat16)
        if K_pages.dim() != 4 or K_pages.shape[1:] != (self.page_rows, Hkv, hd):
            raise ValueError(f"K_pages: expected [pages, {self.page_rows}, {Hkv}, {hd}], "
                             f"got {tuple(K_pages.shape)}")
        _need(V_pages, "V_pages", torch.bfloat16, tuple(K_pages.shape))
        _need(block_table, "block_table", torch.int32)
        if block_table.dim() != 2 or block_table.shape[0] != batch:
            raise ValueError(f"block_table: expected [{batch}, max_pages], "
                             f"got {tuple(block_table.shape)}")
        _need(ctx_len, "ctx_len", torch.int32, (batch,))
        ws = w.struct()
        if ws.hidden != hidden:
            raise ValueError(f"weights: hidden {ws.hidden}, expected {hidden}")
        st = tree.struct()
        _lib.check(self.lib, "verify_layer_paged", self.lib.verify_layer_paged(
            _ptr(X), ctypes.byref(ws), _ptr(K_pages), _ptr(V_pages), K_pages.shape[0],
            self.page_rows, _ptr(block_table), block_table.shape[1], _ptr(ctx_len),
            ctypes.byref(st), batch, budget, Hq, Hkv, hd, max_ctx, self.scale, _ptr(self.Y),
            _ptr(self.ws), self.ws.numel(), _stream()))
        return self.Y
