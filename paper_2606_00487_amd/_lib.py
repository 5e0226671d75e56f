"""ctypes view of libtaps.so (declarations mirror include/taps.h).

Loading never builds: a missing library raises, so nothing can silently fall
back to another implementation.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libtaps.so")

TAPS_OK = 0
TAPS_ERR_INVALID_ARG = -1
TAPS_ERR_UNSUPPORTED = -2
TAPS_ERR_WORKSPACE = -3
TAPS_ERR_HIP = -4
TAPS_BF16 = 0
TAPS_FP32 = 1
TAPS_LOGITS = 0
TAPS_PROBS = 1
TAPS_SCORER_SIBLING = 0
TAPS_SCORER_MARGINAL = 1
TAPS_SCORER_LEARNED = 2
MAX_BLOCK = 32
MAX_K = 16
MAX_BUDGET = 512

EXPORTED = [
    "taps_select_workspace_bytes", "taps_select_validate", "taps_select",
    "tree_verify_attn_workspace_bytes", "tree_verify_attn_validate", "tree_verify_attn",
    "tree_verify_attn_timed", "accept_walk", "kv_commit", "taps_status_string",
    "taps_spec_exp_host", "verify_layer_workspace_bytes", "verify_layer", "taps_select_noalloc",
    "tree_verify_attn_paged_workspace_bytes", "tree_verify_attn_paged",
    "tree_verify_attn_paged_timed", "kv_commit_paged", "verify_layer_paged_workspace_bytes",
    "verify_layer_paged",
]
SELECT_SCRATCH_BYTES = 8 << 20   # TAPS_SELECT_SCRATCH_BYTES


class LayerWeights(ctypes.Structure):
    _fields_ = [("Wq", ctypes.c_void_p), ("Wk", ctypes.c_void_p), ("Wv", ctypes.c_void_p),
                ("Wo", ctypes.c_void_p), ("q_norm", ctypes.c_void_p), ("k_norm", ctypes.c_void_p),
                ("rope_theta", ctypes.c_double), ("norm_eps", ctypes.c_float),
                ("hidden", ctypes.c_int32)]


class ScorerMLP(ctypes.Structure):
    _fields_ = [("emb", ctypes.c_void_p), ("W1", ctypes.c_void_p), ("b1", ctypes.c_void_p),
                ("w2", ctypes.c_void_p), ("b2", ctypes.c_float), ("root_token", ctypes.c_void_p),
                ("emb_dim", ctypes.c_int32), ("hidden", ctypes.c_int32)]


class SelectParams(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("block", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("K", ctypes.c_int32), ("budget", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("kind", ctypes.c_int32), ("lambda1", ctypes.c_double),
                ("lambda2", ctypes.c_double), ("tau", ctypes.c_double), ("beta", ctypes.c_double),
                ("scorer", ctypes.c_int32), ("mlp", ctypes.POINTER(ScorerMLP))]


class Tree(ctypes.Structure):
    _fields_ = [("parent", ctypes.c_void_p), ("token", ctypes.c_void_p),
                ("depth", ctypes.c_void_p), ("rank", ctypes.c_void_p),
                ("q_reach", ctypes.c_void_p), ("n_nodes", ctypes.c_void_p),
                ("topk_idx", ctypes.c_void_p), ("topk_val", ctypes.c_void_p)]


class TapsError(RuntimeError):
    def __init__(self, call: str, status: int, lib=None):
        name = lib.taps_status_string(status).decode() if lib is not None else str(status)
        super().__init__(f"{call} failed: {name} ({status})")
        self.status = status


_LIB = None


def load(path: str = LIB_PATH):
    """Load the built library (raises if it is not built)."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with __graft_entry__.build() "
                           "(python -m paper_2606_00487_amd.build)")
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER
    vp, i32, i64, f32, f64, sz = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                                  ctypes.c_float, ctypes.c_double, ctypes.c_size_t)
    lib.taps_select_workspace_bytes.argtypes = [P(SelectParams)]
    lib.taps_select_workspace_bytes.restype = sz
    lib.taps_select_validate.argtypes = [P(SelectParams)]
    lib.taps_select_validate.restype = i32
    lib.taps_select.argtypes = [vp, P(SelectParams), P(Tree), vp, sz, vp]
    lib.taps_select.restype = i32
    lib.taps_select_noalloc.argtypes = [vp, P(SelectParams), P(Tree), vp]
    lib.taps_select_noalloc.restype = i32
    lib.tree_verify_attn_workspace_bytes.argtypes = [i32, i32, i32, i32, i32, i32, i32]
    lib.tree_verify_attn_workspace_bytes.restype = sz
    lib.tree_verify_attn_validate.argtypes = [i32, i32, i32, i32, i32, i32, i32, f32]
    lib.tree_verify_attn_validate.restype = i32
    lib.tree_verify_attn.argtypes = [vp, vp, vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32,
                                     i32, f32, vp, vp, sz, vp]
    lib.tree_verify_attn.restype = i32
    lib.tree_verify_attn_timed.argtypes = lib.tree_verify_attn.argtypes + [vp, vp]
    lib.tree_verify_attn_timed.restype = i32
    lib.tree_verify_attn_paged_workspace_bytes.argtypes = [i32, i32, i32, i32, i32, i32, i32]
    lib.tree_verify_attn_paged_workspace_bytes.restype = sz
    lib.tree_verify_attn_paged.argtypes = [vp, vp, vp, i32, i32, vp, i32, vp, vp, vp, i32, i32,
                                           i32, i32, i32, i32, i32, f32, vp, vp, sz, vp]
    lib.tree_verify_attn_paged.restype = i32
    lib.tree_verify_attn_paged_timed.argtypes = lib.tree_verify_attn_paged.argtypes + [vp, vp]
    lib.tree_verify_attn_paged_timed.restype = i32
    lib.accept_walk.argtypes = [P(Tree), i32, i32, i32, vp, vp, vp, vp, vp]
    lib.accept_walk.restype = i32
    lib.kv_commit.argtypes = [vp, vp, vp, vp, P(Tree), vp, vp, vp, i32, i32, i32, i32, i32, i32,
                              i32, vp, vp, vp, vp]
    lib.kv_commit.restype = i32
    lib.kv_commit_paged.argtypes = [vp, vp, i32, i32, vp, i32, vp, P(Tree), vp, vp, vp, i32, i32,
                                    i32, i32, i32, i32, i32, vp, vp, vp, vp]
    lib.kv_commit_paged.restype = i32
    lib.verify_layer_workspace_bytes.argtypes = [i32] * 7
    lib.verify_layer_workspace_bytes.restype = ctypes.c_size_t
    lib.verify_layer.argtypes = [vp, P(LayerWeights), vp, vp, vp, vp, P(Tree), i32, i32, i32, i32,
                                 i32, i32, ctypes.c_float, vp, vp, ctypes.c_size_t, vp]
    lib.verify_layer.restype = i32
    lib.verify_layer_paged_workspace_bytes.argtypes = [i32] * 8
    lib.verify_layer_paged_workspace_bytes.restype = ctypes.c_size_t
    lib.verify_layer_paged.argtypes = [vp, P(LayerWeights), vp, vp, i32, i32, vp, i32, vp,
                                       P(Tree), i32, i32, i32, i32, i32, i32, f32, vp, vp, sz,
                                       vp]
    lib.verify_layer_paged.restype = i32
    lib.taps_status_string.argtypes = [i32]
    lib.taps_status_string.restype = ctypes.c_char_p
    lib.taps_spec_exp_host.argtypes = [f64]
    lib.taps_spec_exp_host.restype = f64
    _LIB = lib
    return lib


def check(lib, call: str, status: int):
    if status != TAPS_OK:
        raise TapsError(call, status, lib)
