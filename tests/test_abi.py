"""The C-ABI library on the CPU: it loads, exports every symbol include/taps.h
declares, validates arguments before touching the device, and its fp64
exponential (the host instance of the device function) matches the oracle bit
for bit.  No kernel is launched here."""
import ctypes
import math
import os
import re

import numpy as np
import pytest

from paper_2606_00487_amd import _lib
from oracle.specexp import spec_exp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "taps.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b([a-z_]+)\s*\(", src)) - {"defined"})


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert set(names) == set(_lib.EXPORTED), names
    for name in names:
        assert hasattr(lib, name), name


def params(**kw):
    base = dict(batch=2, block=16, vocab=151936, K=8, budget=64, dtype=_lib.TAPS_BF16,
                kind=_lib.TAPS_LOGITS, lambda1=1.0, lambda2=0.125, tau=0.0, beta=1.0)
    base.update(kw)
    return _lib.SelectParams(**base)


@pytest.mark.parametrize("kw,status", [
    ({}, _lib.TAPS_OK),
    ({"batch": 0}, _lib.TAPS_OK),
    ({"batch": -1}, _lib.TAPS_ERR_INVALID_ARG),
    ({"K": 17}, _lib.TAPS_ERR_UNSUPPORTED),
    ({"K": 0}, _lib.TAPS_ERR_INVALID_ARG),
    ({"budget": 513}, _lib.TAPS_ERR_UNSUPPORTED),
    ({"budget": 512}, _lib.TAPS_OK),
    ({"budget": 0}, _lib.TAPS_ERR_INVALID_ARG),
    ({"block": 33}, _lib.TAPS_ERR_UNSUPPORTED),
    ({"block": 0}, _lib.TAPS_ERR_INVALID_ARG),
    ({"vocab": 4, "K": 8}, _lib.TAPS_ERR_INVALID_ARG),
    ({"vocab": 2_000_000}, _lib.TAPS_ERR_UNSUPPORTED),
    ({"lambda1": 0.0}, _lib.TAPS_ERR_INVALID_ARG),
    ({"lambda1": math.inf}, _lib.TAPS_ERR_INVALID_ARG),
    ({"lambda2": -0.5}, _lib.TAPS_ERR_UNSUPPORTED),
    ({"lambda2": math.nan}, _lib.TAPS_ERR_INVALID_ARG),
    ({"tau": math.nan}, _lib.TAPS_ERR_INVALID_ARG),
    ({"tau": math.inf}, _lib.TAPS_OK),
    ({"beta": -1.0}, _lib.TAPS_ERR_INVALID_ARG),
    ({"kind": _lib.TAPS_PROBS, "beta": 2.0}, _lib.TAPS_ERR_UNSUPPORTED),
    ({"kind": _lib.TAPS_PROBS, "dtype": _lib.TAPS_FP32}, _lib.TAPS_OK),
    ({"dtype": 7}, _lib.TAPS_ERR_INVALID_ARG),
    ({"kind": 5}, _lib.TAPS_ERR_INVALID_ARG),
])
def test_select_validation(lib, kw, status):
    p = params(**kw)
    assert lib.taps_select_validate(ctypes.byref(p)) == status
    if status != _lib.TAPS_OK:
        # the entry point returns the same status without touching its (null) buffers
        assert lib.taps_select(None, ctypes.byref(p), None, None, 0, None) == status


def test_select_scorer_validation_and_workspace(lib):
    assert lib.taps_select_validate(ctypes.byref(params(scorer=1))) == _lib.TAPS_OK
    assert lib.taps_select_validate(ctypes.byref(params(scorer=2))) == _lib.TAPS_ERR_INVALID_ARG
    assert lib.taps_select_validate(ctypes.byref(params(scorer=1, beta=2.0))) == \
        _lib.TAPS_ERR_UNSUPPORTED
    base = lib.taps_select_workspace_bytes(ctypes.byref(params()))
    marg = lib.taps_select_workspace_bytes(ctypes.byref(params(scorer=1)))
    assert marg == base + 2 * 16 * 10 * 4 * 8    # four int64 partials per (row, chunk)
    probs = params(scorer=1, kind=_lib.TAPS_PROBS)
    assert lib.taps_select_workspace_bytes(ctypes.byref(probs)) == base   # no normaliser


def test_select_learned_scorer_validation_and_workspace(lib):
    fake = 1 << 20
    w = _lib.ScorerMLP(fake, fake, fake, fake, 0.5, fake, 16, 32)

    def p(**kw):
        q = params(scorer=2, **kw)
        q.mlp = ctypes.pointer(w)
        return q

    assert lib.taps_select_validate(ctypes.byref(p())) == _lib.TAPS_OK
    assert lib.taps_select_validate(ctypes.byref(p(kind=_lib.TAPS_PROBS))) == \
        _lib.TAPS_ERR_UNSUPPORTED
    assert lib.taps_select_validate(ctypes.byref(p(block=32, K=16))) == \
        _lib.TAPS_ERR_UNSUPPORTED                     # a 32 x 16 x 16 table exceeds the LDS
    assert lib.taps_select_validate(ctypes.byref(params(scorer=2))) == \
        _lib.TAPS_ERR_INVALID_ARG                     # no weights
    w.emb_dim = 33
    assert lib.taps_select_validate(ctypes.byref(p())) == _lib.TAPS_ERR_UNSUPPORTED
    w.emb_dim, w.hidden = 16, 0
    assert lib.taps_select_validate(ctypes.byref(p())) == _lib.TAPS_ERR_INVALID_ARG
    w.hidden = 32
    base = lib.taps_select_workspace_bytes(ctypes.byref(params()))
    assert lib.taps_select_workspace_bytes(ctypes.byref(p())) == base + 2 * (2 * 16 * 10 * 4 * 8)
    # the largest tables of each K fit the scratch area at the largest weights
    w.emb_dim, w.hidden = 32, 64
    for blk, k in ((32, 8), (28, 16), (32, 4)):
        assert lib.taps_select_validate(ctypes.byref(p(block=blk, K=k))) == _lib.TAPS_OK


def test_select_rejects_null_buffers_and_small_workspace(lib):
    p = params()
    assert lib.taps_select(None, ctypes.byref(p), None, None, 0, None) == _lib.TAPS_ERR_INVALID_ARG
    fake = 1 << 20  # aligned, never dereferenced: validation stops before any launch
    t = _lib.Tree(fake, fake, fake, fake, fake, fake, fake, fake)
    need = lib.taps_select_workspace_bytes(ctypes.byref(p))
    assert need == 2 * 16 * 10 * 8 * 8     # 32 rows x 10 chunks of 16384 x K keys of 8 bytes
    assert lib.taps_select(fake, ctypes.byref(p), ctypes.byref(t), fake, need - 1, None) == \
        _lib.TAPS_ERR_WORKSPACE
    assert lib.taps_select(fake + 2, ctypes.byref(p), ctypes.byref(t), fake, need, None) == \
        _lib.TAPS_ERR_INVALID_ARG            # marginals must be 16-byte aligned
    assert lib.taps_select(None, ctypes.byref(params(batch=0)), None, None, 0, None) == _lib.TAPS_OK


@pytest.mark.parametrize("args,status", [
    ((1, 64, 32, 8, 128, 8192, 0, 0.088), _lib.TAPS_OK),
    ((1, 64, 32, 7, 128, 8192, 0, 0.088), _lib.TAPS_ERR_INVALID_ARG),
    ((1, 64, 32, 8, 96, 8192, 0, 0.088), _lib.TAPS_ERR_UNSUPPORTED),
    ((1, 600, 32, 8, 128, 8192, 0, 0.088), _lib.TAPS_ERR_UNSUPPORTED),
    ((1, 300, 32, 8, 128, 8192, 0, 0.088), _lib.TAPS_OK),
    ((1, 64, 32, 8, 128, -1, 0, 0.088), _lib.TAPS_ERR_INVALID_ARG),
    ((1, 64, 32, 8, 128, 8192, 3, 0.088), _lib.TAPS_ERR_INVALID_ARG),
    ((1, 64, 32, 8, 128, 8192, 0, math.inf), _lib.TAPS_ERR_INVALID_ARG),
    ((1, 64, 32, 8, 128, 8192, 0, 0.0), _lib.TAPS_ERR_INVALID_ARG),
    ((1, 64, 32, 8, 128, 8192, 0, -0.5), _lib.TAPS_ERR_INVALID_ARG),
    ((0, 64, 32, 8, 128, 8192, 0, 0.088), _lib.TAPS_OK),
    ((1, 16, 4, 2, 64, 256, 1, 0.125), _lib.TAPS_OK),
])
def test_attention_validation(lib, args, status):
    assert lib.tree_verify_attn_validate(*args) == status
    b, n, hq, hkv, hd, mc, dt, sc = args
    if status != _lib.TAPS_OK:
        assert lib.tree_verify_attn(None, None, None, None, None, None, None, b, n, hq, hkv, hd,
                                    mc, dt, sc, None, None, 0, None) == status


def test_attention_workspace_is_a_pure_function(lib):
    a = lib.tree_verify_attn_workspace_bytes(1, 64, 32, 8, 128, 8192, 0)
    assert a > 0 and a == lib.tree_verify_attn_workspace_bytes(1, 64, 32, 8, 128, 8192, 0)
    assert lib.tree_verify_attn_workspace_bytes(1, 16, 4, 2, 64, 256, 1) == 0   # fp32: none
    fake = 1 << 20
    assert lib.tree_verify_attn(fake, fake, fake, fake, fake, fake, fake, 1, 64, 32, 8, 128, 8192,
                                0, 0.088, fake, fake, a - 1, None) == _lib.TAPS_ERR_WORKSPACE


@pytest.mark.parametrize("page_rows,hd,dtype,max_pages,num_pages,status", [
    (64, 128, 0, 130, 200, _lib.TAPS_OK),
    (32, 128, 0, 260, 1, _lib.TAPS_OK),
    (4096, 128, 0, 3, 1, _lib.TAPS_OK),
    (48, 128, 0, 200, 200, _lib.TAPS_ERR_INVALID_ARG),       # not a power of two
    (16, 128, 0, 600, 600, _lib.TAPS_ERR_INVALID_ARG),       # below 32 rows
    (8192, 128, 0, 2, 2, _lib.TAPS_ERR_INVALID_ARG),         # above 4096 rows
    (64, 64, 0, 130, 200, _lib.TAPS_ERR_UNSUPPORTED),        # head_dim 64
    (64, 128, 1, 130, 200, _lib.TAPS_ERR_UNSUPPORTED),       # fp32
    (64, 128, 0, 128, 200, _lib.TAPS_ERR_INVALID_ARG),       # 128 * 64 < 8192 + 64 rows
    (64, 128, 0, 129, 200, _lib.TAPS_OK),                    # 129 * 64 = 8192 + 64 rows
    (64, 128, 0, 130, 0, _lib.TAPS_ERR_INVALID_ARG),         # no pages
])
def test_paged_attention_validation(lib, page_rows, hd, dtype, max_pages, num_pages, status):
    """tree_verify_attn_paged checks its page geometry on the host; every case stops
    before a launch (the pointers are never dereferenced)."""
    fake = 1 << 20
    need = lib.tree_verify_attn_paged_workspace_bytes(1, 64, 32, 8, hd, 8192, page_rows)
    args = (fake, fake, fake, num_pages, page_rows, fake, max_pages, fake, fake, fake, 1, 64,
            32, 8, hd, 8192, dtype, 0.088, fake, fake)
    if status == _lib.TAPS_OK:
        assert need > 0
        # a valid geometry gets as far as the workspace check
        assert lib.tree_verify_attn_paged(*args, need - 1, None) == _lib.TAPS_ERR_WORKSPACE
    else:
        assert lib.tree_verify_attn_paged(*args, 1 << 30, None) == status


def test_paged_attention_workspace_matches_contiguous_plan(lib):
    """Below the paged split cap the paged plan is the contiguous one, so the workspaces
    agree; without a valid page size there is none."""
    a = lib.tree_verify_attn_workspace_bytes(1, 64, 32, 8, 128, 8192, 0)
    assert lib.tree_verify_attn_paged_workspace_bytes(1, 64, 32, 8, 128, 8192, 64) == a
    assert lib.tree_verify_attn_paged_workspace_bytes(1, 64, 32, 8, 128, 8192, 48) == 0
    assert lib.tree_verify_attn_paged_workspace_bytes(0, 64, 32, 8, 128, 8192, 64) == 0


def test_paged_commit_validation(lib):
    fake = 1 << 20          # aligned, never dereferenced: every case stops before a launch
    t = _lib.Tree(fake, fake, fake, fake, fake, fake, fake, fake)

    def call(num_pages=100, page_rows=64, max_pages=129, sizes=(1, 64, 16, 8, 128, 8192, 0),
             new_ctx=fake + 64):
        return lib.kv_commit_paged(fake, fake, num_pages, page_rows, fake, max_pages, fake,
                                   ctypes.byref(t), fake, fake, fake, *sizes, new_ctx,
                                   fake + 128, fake + 192, None)

    assert call(sizes=(0, 64, 16, 8, 128, 8192, 0)) == _lib.TAPS_OK            # nothing to do
    assert call(page_rows=48) == _lib.TAPS_ERR_INVALID_ARG
    assert call(page_rows=16) == _lib.TAPS_ERR_INVALID_ARG
    assert call(max_pages=128) == _lib.TAPS_ERR_INVALID_ARG    # 128 * 64 < 8192 + 64 rows
    assert call(num_pages=0) == _lib.TAPS_ERR_INVALID_ARG
    assert call(new_ctx=fake) == _lib.TAPS_ERR_INVALID_ARG      # new_ctx_len is ctx_len
    assert call(sizes=(1, 513, 16, 8, 128, 8192, 0)) == _lib.TAPS_ERR_UNSUPPORTED
    assert call(sizes=(1, 64, 16, 8, 96, 8192, 0)) == _lib.TAPS_ERR_UNSUPPORTED


def test_paged_layer_validation(lib):
    """verify_layer_paged checks the page geometry before anything else; the workspace
    query matches the contiguous one below the paged split cap."""
    fake = 1 << 20
    w = _lib.LayerWeights(fake, fake, fake, fake, fake, fake, 1e6, 1e-6, 4096)
    t = _lib.Tree(fake, fake, fake, fake, fake, fake, fake, fake)

    def call(num_pages=200, page_rows=64, max_pages=129):
        return lib.verify_layer_paged(fake, ctypes.byref(w), fake, fake, num_pages, page_rows,
                                      fake, max_pages, fake, ctypes.byref(t), 1, 64, 32, 8, 128,
                                      8192, 0.088, fake, fake, 1 << 40, None)

    assert call(page_rows=48) == _lib.TAPS_ERR_INVALID_ARG
    assert call(max_pages=128) == _lib.TAPS_ERR_INVALID_ARG
    assert call(num_pages=0) == _lib.TAPS_ERR_INVALID_ARG
    a = lib.verify_layer_workspace_bytes(1, 64, 32, 8, 128, 4096, 8192)
    assert lib.verify_layer_paged_workspace_bytes(1, 64, 32, 8, 128, 4096, 8192, 64) == a > 0
    assert lib.verify_layer_paged_workspace_bytes(1, 64, 32, 8, 128, 4096, 8192, 48) == 0


def test_walk_validation(lib):
    assert lib.accept_walk(None, 1, 64, 16, None, None, None, None, None) == _lib.TAPS_ERR_INVALID_ARG
    assert lib.accept_walk(None, 1, 64, 33, None, None, None, None, None) == _lib.TAPS_ERR_UNSUPPORTED
    assert lib.accept_walk(None, 0, 64, 16, None, None, None, None, None) == _lib.TAPS_OK


def test_commit_validation(lib):
    fake = 1 << 20          # aligned, never dereferenced: every case stops before a launch
    t = _lib.Tree(fake, fake, fake, fake, fake, fake, fake, fake)
    ok = (fake, fake, fake, fake, ctypes.byref(t), fake, fake, fake)
    outs = (fake + 64, fake + 128, fake + 192, None)

    def call(ptrs=ok, sizes=(1, 64, 16, 8, 128, 8192, 0), out=outs):
        return lib.kv_commit(*ptrs, *sizes, *out)

    assert call(sizes=(0, 64, 16, 8, 128, 8192, 0)) == _lib.TAPS_OK            # nothing to do
    assert call(sizes=(-1, 64, 16, 8, 128, 8192, 0)) == _lib.TAPS_ERR_INVALID_ARG
    assert call(sizes=(1, 513, 16, 8, 128, 8192, 0)) == _lib.TAPS_ERR_UNSUPPORTED
    assert call(sizes=(1, 64, 33, 8, 128, 8192, 0)) == _lib.TAPS_ERR_UNSUPPORTED
    assert call(sizes=(1, 64, 16, 8, 96, 8192, 0)) == _lib.TAPS_ERR_UNSUPPORTED
    assert call(sizes=(1, 64, 16, 8, 128, 8192, 5)) == _lib.TAPS_ERR_INVALID_ARG
    assert call(sizes=(1, 64, 16, 8, 128, -1, 0)) == _lib.TAPS_ERR_INVALID_ARG
    # new_ctx_len may not be the ctx_len array; buffers must be present and aligned
    assert call(out=(fake, fake + 128, fake + 192, None)) == _lib.TAPS_ERR_INVALID_ARG
    assert call(ptrs=(None,) + ok[1:]) == _lib.TAPS_ERR_INVALID_ARG
    assert call(ptrs=(fake + 8,) + ok[1:]) == _lib.TAPS_ERR_INVALID_ARG
    assert call(out=(None, fake + 128, fake + 192, None)) == _lib.TAPS_ERR_INVALID_ARG


def test_status_strings(lib):
    assert lib.taps_status_string(0) == b"TAPS_OK"
    assert lib.taps_status_string(-3) == b"TAPS_ERR_WORKSPACE"
    assert lib.taps_status_string(42) == b"TAPS_UNKNOWN_STATUS"


def test_library_exponential_matches_oracle_bitwise(lib):
    rng = np.random.default_rng(11)
    ts = np.concatenate([-rng.uniform(0, 1, 20000), -rng.uniform(0, 50, 20000),
                         -rng.uniform(0, 708, 5000), [0.0, -0.0, -1e-300, -708.0, -708.5,
                                                      -math.inf, math.nan, -0.5 * math.log(2)]])
    # every bf16 gap a row of logits can produce near the top of a row
    from workloads import bf16_bits_to_f32
    v = bf16_bits_to_f32(np.arange(0x3F00, 0x4180, dtype=np.uint16)).astype(np.float64)
    ts = np.concatenate([ts, (v[:, None] - v[None, :]).ravel()])
    ts = ts[~(ts > 0)]
    for t in ts:
        a, b = lib.taps_spec_exp_host(float(t)), spec_exp(float(t))
        assert a == b or (math.isnan(a) and math.isnan(b)), (t, a, b)
        assert np.float64(a).view(np.int64) == np.float64(b).view(np.int64), t


def test_layer_validation_and_workspace(lib):
    fake = 1 << 20          # aligned, never dereferenced: every case stops before a launch
    t = _lib.Tree(fake, fake, fake, fake, fake, fake, fake, fake)
    w = _lib.LayerWeights(fake, fake, fake, fake, fake, fake, 1e6, 1e-6, 4096)
    ws_need = lib.verify_layer_workspace_bytes(1, 64, 32, 8, 128, 4096, 8192)
    assert ws_need > 2 * 64 * 32 * 128 * 2          # at least Q and O in bf16
    assert lib.verify_layer_workspace_bytes(0, 64, 32, 8, 128, 4096, 8192) == 0
    assert lib.verify_layer_workspace_bytes(1, 64, 32, 8, 64, 4096, 8192) == 0    # head_dim 128
    assert lib.verify_layer_workspace_bytes(1, 64, 32, 8, 128, 4000, 8192) == 0   # hidden % 64

    def call(batch=1, hidden=4096, hd=128, scale=0.088, ws=fake, ws_bytes=ws_need, X=fake,
             tree=ctypes.byref(t), weights=None):
        w.hidden = hidden
        return lib.verify_layer(X, weights if weights is not None else ctypes.byref(w), fake,
                                fake, fake, fake, tree, batch, 64, 32, 8, hd, 8192, scale,
                                fake, ws, ws_bytes, None)

    assert call(batch=0) == _lib.TAPS_OK
    assert call(hidden=4000) == _lib.TAPS_ERR_INVALID_ARG
    assert call(hidden=32768) == _lib.TAPS_ERR_UNSUPPORTED
    assert call(hd=64) == _lib.TAPS_ERR_UNSUPPORTED
    assert call(scale=0.0) == _lib.TAPS_ERR_INVALID_ARG
    assert call(X=fake + 8) == _lib.TAPS_ERR_INVALID_ARG            # misaligned
    assert call(X=None) == _lib.TAPS_ERR_INVALID_ARG
    assert call(tree=None) == _lib.TAPS_ERR_INVALID_ARG
    assert call(ws_bytes=ws_need - 1) == _lib.TAPS_ERR_WORKSPACE
    assert call(ws=fake + 16) == _lib.TAPS_ERR_WORKSPACE             # 256-byte aligned
    w.rope_theta = 1.0
    assert call() == _lib.TAPS_ERR_INVALID_ARG
    w.rope_theta, w.norm_eps = 1e6, float("nan")
    assert call() == _lib.TAPS_ERR_INVALID_ARG
    w.norm_eps, w.Wo = 1e-6, None
    assert call() == _lib.TAPS_ERR_INVALID_ARG


def test_noalloc_select_validates_before_touching_the_device(lib):
    """taps_select_noalloc refuses bad parameters, missing outputs and selections larger
    than its static scratch on the host, before any device call (this runs without a GPU)."""
    import ctypes
    fake = 4096                       # never dereferenced: every case returns before
    tree = _lib.Tree(fake, fake, fake, fake, fake, fake, fake, fake)
    big = params(batch=4096, block=32, K=16)
    assert lib.taps_select_workspace_bytes(ctypes.byref(big)) > _lib.SELECT_SCRATCH_BYTES
    assert lib.taps_select_noalloc(fake, ctypes.byref(big), ctypes.byref(tree), None) == \
        _lib.TAPS_ERR_WORKSPACE
    assert lib.taps_select_noalloc(fake, ctypes.byref(params(K=17)), ctypes.byref(tree),
                                   None) == _lib.TAPS_ERR_UNSUPPORTED
    assert lib.taps_select_noalloc(None, ctypes.byref(params()), ctypes.byref(tree), None) == \
        _lib.TAPS_ERR_INVALID_ARG
    assert lib.taps_select_noalloc(fake, ctypes.byref(params(batch=0)), None, None) == _lib.TAPS_OK
    assert lib.taps_select_workspace_bytes(ctypes.byref(params(batch=16))) <= \
        _lib.SELECT_SCRATCH_BYTES
