"""Pins of oracle.layer (the verification layer slice) against properties fixed by the
mathematics of RMSNorm, rotary embeddings and attention, and against torch's bf16."""
import numpy as np
import pytest
import torch

from oracle.attention import tree_attention
from oracle.layer import bf16_round, rms_norm, rope, verify_layer


def test_bf16_round_equals_torch_conversion():
    rng = np.random.default_rng(1)
    x = (rng.standard_normal(20000) * np.exp(rng.uniform(-20, 20, 20000))).astype(np.float32)
    # exact ties: bf16 value plus half an ulp, both parities
    base = torch.from_numpy(x[:2000]).to(torch.bfloat16).float().numpy()
    ties = (base.view(np.uint32) | np.uint32(0x8000)).view(np.float32)
    x = np.concatenate([x, ties])
    want = torch.from_numpy(x).to(torch.bfloat16).double().numpy()
    assert np.array_equal(bf16_round(x.astype(np.float64)), want)


def test_rms_norm_unit_rms_and_scale_invariance():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((7, 128))
    y = rms_norm(x, np.ones(128), 0.0)
    assert np.allclose(np.sqrt(np.mean(y * y, axis=-1)), 1.0, rtol=1e-14)
    assert np.allclose(rms_norm(3.5 * x, np.ones(128), 0.0), y, rtol=1e-13)
    w = rng.standard_normal(128)
    assert np.allclose(rms_norm(x, w, 0.0), y * w, rtol=1e-14)


def test_rope_is_a_complex_rotation():
    rng = np.random.default_rng(3)
    hd, theta = 128, 1e6
    x = rng.standard_normal((5, hd))
    pos = np.array([0, 1, 17, 8191, 40000])
    got = rope(x, pos, theta)
    assert np.array_equal(got[0], x[0])                              # position 0: identity
    z = x[:, :hd // 2] + 1j * x[:, hd // 2:]
    freq = np.exp(-np.log(theta) * np.arange(hd // 2) * 2.0 / hd)
    z = z * np.exp(1j * pos[:, None] * freq)
    assert np.allclose(got, np.concatenate([z.real, z.imag], axis=-1), atol=1e-9)
    assert np.allclose(np.linalg.norm(got, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-13)


def test_rope_scores_depend_only_on_the_position_difference():
    rng = np.random.default_rng(4)
    q, k = rng.standard_normal(128), rng.standard_normal(128)
    s1 = rope(q, 1005, 1e6) @ rope(k, 1000, 1e6)
    s2 = rope(q, 8197, 1e6) @ rope(k, 8192, 1e6)
    assert abs(s1 - s2) < 1e-9
    assert abs(rope(q, 7, 1e6) @ rope(k, 7, 1e6) - q @ k) < 1e-9


def _case(rng, B=2, N=6, H=256, Hq=4, Hkv=2, hd=128, ctx=(5, 0)):
    f = lambda *s: bf16_round(rng.standard_normal(s))
    X = f(B, N, H)
    Wq, Wk, Wv = f(Hq * hd, H) / 16, f(Hkv * hd, H) / 16, f(Hkv * hd, H) / 16
    Wo = f(H, Hq * hd) / 16
    qn, kn = bf16_round(1 + 0.1 * rng.standard_normal(hd)), bf16_round(1 + 0.1 * rng.standard_normal(hd))
    ctx = np.array(ctx, dtype=np.int32)
    off = np.array([0, ctx[0] + N + 3], dtype=np.int64)
    rows = int(off[-1] + ctx[-1] + N)
    Kc, Vc = f(rows, Hkv, hd), f(rows, Hkv, hd)
    parent = np.array([[-1, 0, 0, 1, 1, 2]] * B, dtype=np.int32)[:, :N]
    depth = np.array([[0, 1, 1, 2, 2, 2]] * B, dtype=np.int32)[:, :N]
    return dict(X=X, Wq=Wq, Wk=Wk, Wv=Wv, Wo=Wo, q_norm=qn, k_norm=kn, Kc=Kc, Vc=Vc,
                kv_offset=off, ctx_len=ctx, depth=depth, parent=parent,
                n_nodes=np.array([N, N - 2]), Hq=Hq, Hkv=Hkv, hd=hd, theta=1e6, eps=1e-6,
                scale=1 / np.sqrt(hd))


def test_single_node_without_context_returns_its_own_value_row():
    """n = 1 and no context: the root attends only to itself, so O = V of the root and
    Y = bf16(v) Wo^T with query head h reading KV head h // (Hq/Hkv)."""
    rng = np.random.default_rng(5)
    c = _case(rng, ctx=(0, 0))
    c["n_nodes"] = np.array([1, 1])
    Y, Kc, Vc, q, O = verify_layer(**c)
    v = bf16_round(c["X"] @ c["Wv"].T).reshape(2, -1, c["Hkv"], c["hd"])
    G = c["Hq"] // c["Hkv"]
    want_O = np.repeat(v[:, 0], G, axis=1)                 # [B][Hq][hd]
    assert np.array_equal(O[:, 0], want_O)
    assert np.allclose(Y[:, 0], want_O.reshape(2, -1) @ c["Wo"].T, rtol=1e-13, atol=1e-13)


def test_cache_rows_and_positions():
    rng = np.random.default_rng(6)
    c = _case(rng)
    Y, Kc, Vc, q, O = verify_layer(**c)
    keep = np.ones(len(Kc), bool)
    for b in range(2):
        r0 = int(c["kv_offset"][b] + c["ctx_len"][b])
        keep[r0:r0 + int(c["n_nodes"][b])] = False
    # rows outside every request's [ctx, ctx + n) are untouched
    assert np.array_equal(Kc[keep], c["Kc"][keep]) and np.array_equal(Vc[keep], c["Vc"][keep])
    for b in range(2):
        r0 = int(c["kv_offset"][b] + c["ctx_len"][b])
        n = int(c["n_nodes"][b])
        # the written key of node i is the normed key rotated to position ctx + depth_i
        k = (c["X"][b] @ c["Wk"].T).reshape(-1, c["Hkv"], c["hd"])
        for i in range(n):
            pos = int(c["ctx_len"][b] + c["depth"][b, i])
            want = bf16_round(rope(rms_norm(k[i], c["k_norm"], c["eps"]), pos, c["theta"]))
            assert np.array_equal(Kc[r0 + i], want)
    # siblings (same depth) share a position: equal hidden states give equal keys
    c2 = _case(np.random.default_rng(7))
    c2["X"][:, 2] = c2["X"][:, 1]
    _, K2, _, q2, _ = verify_layer(**c2)
    r0 = int(c2["ctx_len"][0])
    assert np.array_equal(K2[r0 + 1], K2[r0 + 2]) and np.array_equal(q2[0, 1], q2[0, 2])


def test_layer_equals_attention_with_identity_output_projection():
    """With Wo = I (H = Hq*hd), Y is the attention output over the written cache."""
    rng = np.random.default_rng(8)
    c = _case(rng, H=512)
    c["Wo"] = np.eye(512)
    Y, Kc, Vc, q, O = verify_layer(**c)
    O2 = bf16_round(tree_attention(q, Kc, Vc, c["kv_offset"], c["ctx_len"], list(c["parent"]),
                                   [int(x) for x in c["n_nodes"]], c["scale"]))
    for b in range(2):
        n = int(c["n_nodes"][b])
        assert np.array_equal(Y[b, :n], O2[b, :n].reshape(n, -1))


def test_paged_layer_equals_contiguous():
    """The paged layer is the contiguous one seen through the block table: same Y, and the
    pools hold the contiguous result's rows (the written node rows included); pages of no
    request keep their contents."""
    from oracle.layer import verify_layer, verify_layer_paged
    rng = np.random.default_rng(31)
    B, N, H, Hq, Hkv, hd, P = 2, 6, 64, 2, 1, 128, 4
    ctx = np.array([5, 0], np.int32)
    rnd = lambda *s: bf16_round(rng.standard_normal(s) * 0.5)   # noqa: E731
    X = rnd(B, N, H)
    Wq, Wk, Wv = rnd(Hq * hd, H), rnd(Hkv * hd, H), rnd(Hkv * hd, H)
    Wo = rnd(H, Hq * hd)
    qn, kn = bf16_round(1 + 0.1 * rng.standard_normal(hd)), bf16_round(1 + 0.1 * rng.standard_normal(hd))
    parent = np.array([[-1, 0, 0, 1, 1, 2], [-1, 0, 1, 2, 3, 4]], np.int32)
    depth = np.array([[0, 1, 1, 2, 2, 2], [0, 1, 2, 3, 4, 5]], np.int32)
    n = np.array([6, 4], np.int32)
    off = np.array([0, int(ctx[0]) + N], np.int64)
    rows = int(off[-1] + ctx[-1] + N)
    Kc, Vc = rnd(rows, Hkv, hd), rnd(rows, Hkv, hd)
    Y, Ko, Vo, _, _ = verify_layer(X, Wq, Wk, Wv, Wo, qn, kn, Kc, Vc, off, ctx, depth, parent,
                                   n, Hq, Hkv, hd, 1e6, 1e-6, hd ** -0.5)
    need = [-(-(int(ctx[b]) + N) // P) for b in range(B)]
    ids = rng.permutation(sum(need) + 3)
    Kp = rnd(len(ids), P, Hkv, hd)
    Vp = rnd(len(ids), P, Hkv, hd)
    table = np.zeros((B, max(need)), np.int32)
    k = 0
    for b in range(B):
        for p in range(need[b]):
            table[b, p] = ids[k]
            for r in range(p * P, min(int(ctx[b]) + N, (p + 1) * P)):
                Kp[ids[k], r - p * P] = Kc[int(off[b]) + r]
                Vp[ids[k], r - p * P] = Vc[int(off[b]) + r]
            k += 1
    Yp, Kp2, Vp2, _, _ = verify_layer_paged(X, Wq, Wk, Wv, Wo, qn, kn, Kp, Vp, table, P, ctx,
                                            depth, parent, n, Hq, Hkv, hd, 1e6, 1e-6, hd ** -0.5)
    for b in range(B):
        assert np.array_equal(Yp[b, :n[b]], Y[b, :n[b]])
        for r in range(int(ctx[b]) + N):
            pg, sl = table[b, r // P], r % P
            assert np.array_equal(Kp2[pg, sl], Ko[int(off[b]) + r])
            assert np.array_equal(Vp2[pg, sl], Vo[int(off[b]) + r])
    for x in ids[k:]:
        assert np.array_equal(Kp2[x], Kp[x]) and np.array_equal(Vp2[x], Vp[x])
