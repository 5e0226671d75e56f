"""One attention layer of the target over the draft tree (the verification forward's
layer slice; Sec. 4.1 stage 3 and Sec. 4.3 run the target once over the selected tree
with tree attention) -- TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

The paper leaves the target model to the serving system; this follows a Qwen3-style
attention block, plain fp64 except where the stored tensors are bf16.  Reading (the
same on the GPU):

* Inputs: the tree nodes' hidden states X [B][N][H] (bf16 values), weights
  Wq [Hq*hd][H], Wk and Wv [Hkv*hd][H], Wo [H][Hq*hd] and the per-head RMSNorm weights
  q_norm, k_norm [hd] (bf16 values).
* q = X Wq^T, k = X Wk^T, v = X Wv^T, split into heads of hd values.
* RMSNorm of each query and key head: x / sqrt(mean(x^2) + eps) * weight.
* Rotary positions by tree depth: node i of request b sits at position ctx_b + depth_i,
  so the root takes the position right after the context and siblings share one.  For
  j < hd/2 the pair (x_j, x_{j+hd/2}) turns by the angle pos * theta^(-2j/hd).
* Q, K and V are stored as bf16 (the cache's type), rounded to nearest even; K and V of
  node i < n_b go to cache row ctx_b + i of request b.
* Tree attention (oracle.attention) over the bf16 cache; O is rounded to bf16.
* Y = O Wo^T.  Rows i >= n_b of Y, Q and O are not defined.
"""
from __future__ import annotations

import numpy as np

from .attention import tree_attention


def bf16_round(x) -> np.ndarray:
    """Round to the nearest bf16 value (8 significant bits), ties to even; normal range."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)                       # x = m 2^e with 0.5 <= |m| < 1
    return np.ldexp(np.round(m * 256.0) / 256.0, e)   # np.round: half to even


def rms_norm(x: np.ndarray, w: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm over the last axis."""
    x = np.asarray(x, dtype=np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(w, dtype=np.float64)


def rope(x: np.ndarray, pos, theta: float) -> np.ndarray:
    """Rotary position embedding in the half-split pairing; ``pos`` broadcasts against the
    leading axes of ``x`` [..., hd]."""
    x = np.asarray(x, dtype=np.float64)
    hd = x.shape[-1]
    half = hd // 2
    freq = theta ** (-2.0 * np.arange(half, dtype=np.float64) / hd)
    ang = np.asarray(pos, dtype=np.float64)[..., None] * freq
    c, s = np.cos(ang), np.sin(ang)
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def verify_layer(X, Wq, Wk, Wv, Wo, q_norm, k_norm, Kc, Vc, kv_offset, ctx_len, depth, parent,
                 n_nodes, Hq, Hkv, hd, theta, eps, scale, samples=None):
    """Y [B][N][H] (NaN on rows i >= n_b), the updated caches (copies), Q and O (bf16
    values).  ``samples``: optional (b, i, h) triples for the attention (others NaN)."""
    X = np.asarray(X, dtype=np.float64)
    B, N, H = X.shape
    q = (X @ np.asarray(Wq, np.float64).T).reshape(B, N, Hq, hd)
    k = (X @ np.asarray(Wk, np.float64).T).reshape(B, N, Hkv, hd)
    v = (X @ np.asarray(Wv, np.float64).T).reshape(B, N, Hkv, hd)
    pos = np.asarray(ctx_len, np.int64)[:, None] + np.asarray(depth, np.int64)   # [B][N]
    q = bf16_round(rope(rms_norm(q, q_norm, eps), pos[:, :, None], theta))
    k = bf16_round(rope(rms_norm(k, k_norm, eps), pos[:, :, None], theta))
    v = bf16_round(v)
    Kc = np.array(Kc, dtype=np.float64)
    Vc = np.array(Vc, dtype=np.float64)
    for b in range(B):
        r0 = int(kv_offset[b]) + int(ctx_len[b])
        n = int(n_nodes[b])
        Kc[r0:r0 + n] = k[b, :n]
        Vc[r0:r0 + n] = v[b, :n]
    O = tree_attention(q, Kc, Vc, kv_offset, ctx_len, [np.asarray(p) for p in parent],
                       [int(x) for x in n_nodes], scale, samples=samples)
    O = bf16_round(O)
    Y = O.reshape(B, N, Hq * hd) @ np.asarray(Wo, np.float64).T
    return Y, Kc, Vc, q, O


def verify_layer_paged(X, Wq, Wk, Wv, Wo, q_norm, k_norm, K_pages, V_pages, block_table,
                       page_rows, ctx_len, depth, parent, n_nodes, Hq, Hkv, hd, theta, eps,
                       scale, samples=None):
    """verify_layer over a paged cache (reading C20 of the layout: request b's logical row r
    is row r % page_rows of page block_table[b][r // page_rows]): the logical rows are
    gathered into a contiguous cache, the layer runs as defined above, and the rows are put
    back.  Returns (Y, K_pages', V_pages', Q, O)."""
    B, N = np.asarray(X).shape[:2]
    where, offs, Ks, Vs = [], [], [], []
    base = 0
    for b in range(B):
        rows = np.arange(int(ctx_len[b]) + N)
        pg = np.asarray(block_table[b])[rows // page_rows]
        sl = rows % page_rows
        where.append((pg, sl))
        Ks.append(np.asarray(K_pages)[pg, sl])
        Vs.append(np.asarray(V_pages)[pg, sl])
        offs.append(base)
        base += len(rows)
    Y, Kc, Vc, q, O = verify_layer(X, Wq, Wk, Wv, Wo, q_norm, k_norm, np.concatenate(Ks),
                                   np.concatenate(Vs), np.asarray(offs, np.int64), ctx_len, depth,
                                   parent, n_nodes, Hq, Hkv, hd, theta, eps, scale, samples)
    Kp = np.array(K_pages, dtype=np.float64)
    Vp = np.array(V_pages, dtype=np.float64)
    for b in range(B):
        pg, sl = where[b]
        Kp[pg, sl] = Kc[offs[b]:offs[b] + len(pg)]
        Vp[pg, sl] = Vc[offs[b]:offs[b] + len(pg)]
    return Y, Kp, Vp, q, O
