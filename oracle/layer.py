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
