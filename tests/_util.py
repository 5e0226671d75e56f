"""Helpers shared by the GPU tests: upload seeded inputs, run the oracle, compare."""
from __future__ import annotations

import numpy as np
import torch

import oracle
from workloads import BF16, Config, RoundInputs, target_tokens


def to_dev(a: np.ndarray, bf16: bool) -> torch.Tensor:
    if bf16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def oracle_trees(inp: RoundInputs, **over) -> list[oracle.Tree]:
    c = inp.cfg
    kw = dict(kind=c.kind, lambda1=c.lambda1, lambda2=c.lambda2, tau=c.tau, beta=c.beta)
    kw.update(over)
    x = inp.marginals_f64()
    return [oracle.select_request(x[b], c.K, c.budget, **kw) for b in range(c.batch)]


def assert_tree_equal(gpu, trees: list[oracle.Tree], cfg: Config):
    par = gpu.parent.cpu().numpy()
    tok = gpu.token.cpu().numpy()
    dep = gpu.depth.cpu().numpy()
    rnk = gpu.rank.cpu().numpy()
    q = gpu.q_reach.cpu().numpy()
    n = gpu.n_nodes.cpu().numpy()
    tidx = gpu.topk_idx.cpu().numpy()
    tval = gpu.topk_val.cpu().numpy()
    for b, t in enumerate(trees):
        assert n[b] == t.n, (b, n[b], t.n)
        np.testing.assert_array_equal(tidx[b], t.topk_idx, err_msg=f"topk_idx b={b}")
        ov = t.topk_val.astype(np.float32)
        same = (tval[b] == ov) | (np.isnan(tval[b]) & np.isnan(ov))
        assert same.all(), f"topk_val b={b}"
        np.testing.assert_array_equal(par[b], t.parent, err_msg=f"parent b={b}")
        np.testing.assert_array_equal(tok[b], t.token, err_msg=f"token b={b}")
        np.testing.assert_array_equal(dep[b], t.depth, err_msg=f"depth b={b}")
        np.testing.assert_array_equal(rnk[b], t.rank, err_msg=f"rank b={b}")
        assert np.array_equal(q[b].view(np.int64), t.q_reach.view(np.int64)), f"q_reach bits b={b}"


def targets_for(inp: RoundInputs, trees: list[oracle.Tree], branch: bool = False) -> np.ndarray:
    c = inp.cfg
    out = np.stack([target_tokens(c, b, t.parent, t.rank, t.n, t.topk_idx[:, 0], inp.p_acc[b],
                                  seed=inp.seed, branch=branch, token=t.token)
                    for b, t in enumerate(trees)])
    return out.astype(np.int32)


def tree_device(trees: list[oracle.Tree]):
    parent = torch.from_numpy(np.stack([t.parent for t in trees]).astype(np.int32)).cuda()
    token = torch.from_numpy(np.stack([t.token for t in trees]).astype(np.int32)).cuda()
    n = torch.tensor([t.n for t in trees], dtype=torch.int32).cuda()
    return parent, token, n


def attention_inputs(inp: RoundInputs):
    bf = inp.cfg.dtype == BF16
    return (to_dev(inp.Q, bf), to_dev(inp.K, bf), to_dev(inp.V, bf),
            torch.from_numpy(inp.kv_offset).cuda(), torch.from_numpy(inp.ctx_len).cuda())


def gpu_o_as_f64(O: torch.Tensor) -> np.ndarray:
    return O.float().cpu().numpy().astype(np.float64)
