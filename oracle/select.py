"""Target-aware selection of one request's draft tree (Sec. 4.1-4.3, Alg. 1).

Readings taken where the paper is silent (each one is listed with its reason
in the design notes):

* Row i of the drafter marginals describes the token at depth i+1; the root
  (depth 0) is the current position and carries no drafted token.
* The candidate tree is the full implicit K-ary trie of depth D: a depth-d
  node's children are the top-K tokens of row d (Sec. 4.1, Stage 1).
* Scorer stand-in: the edge logit is beta times the drafter logit of the child
  token (LOGITS input) or the child's probability is used directly (PROBS
  input).  The sibling softmax of Eq. 1 then depends only on (row, rank).
* Marginal-confidence scorer (the scoring ablation of Sec. 5: the scorer is
  removed and selection falls back to the drafter's marginal confidence, with
  the same candidate pool and procedure): q_cond is the child's full-vocabulary
  marginal probability, without the sibling renormalisation.  LOGITS:
  EXP(x_r - M) / Z with M the row maximum and Z the sum over the whole row of
  EXP(x_j - M), each term rounded to a multiple of 2^-42 and summed exactly (an
  integer sum, so no summation order enters); PROBS: the probability itself,
  clamped into [0, 1] (NaN counts 0), which keeps q_cond <= 1 as Alg. 1's
  one-node-per-iteration property needs.
* Top-K order: value descending, then vocabulary index ascending; -0 equals
  +0; NaN ranks below -inf.
* Ties in the greedy argmax of Alg. 1 are broken by the total order
  u descending, then depth ascending, then rank path lexicographically
  ascending.  The root counts toward the budget; the stop test is the strict
  ``u > tau`` of Alg. 1.
* Arithmetic is IEEE fp64 with round-to-nearest-even and no fused
  multiply-add; sums run in rank order, products in path order.
"""
from __future__ import annotations

import dataclasses
import heapq
import itertools
from fractions import Fraction

import numpy as np

from .specexp import spec_exp, spec_exp_array

LOGITS = 0
PROBS = 1
SIBLING = 0     # scorer: sibling softmax over the K candidates (Eq. 1 stand-in)
MARGINAL = 1    # scorer: the drafter's full-vocabulary marginal (Sec. 5 ablation)
LEARNED = 2     # scorer: the learned-scorer hook, an MLP on edge features (Sec. 4.2)
Z_GRID = 2.0 ** 42   # terms of the marginal normaliser are rounded to multiples of 1/Z_GRID


@dataclasses.dataclass
class Tree:
    """Selected subtree S of one request, breadth first: nodes ordered by depth, then by
    rank path (so every parent precedes its children).

    Slots n..budget-1 hold parent = token = depth = rank = -1 and q_reach = 0.
    """
    parent: np.ndarray    # int32 [budget]; -1 at the root
    token: np.ndarray     # int32 [budget]; -1 at the root
    depth: np.ndarray     # int32 [budget]; 0 at the root
    rank: np.ndarray      # int32 [budget]; -1 at the root
    q_reach: np.ndarray   # float64 [budget]; 1.0 at the root
    n: int
    topk_idx: np.ndarray  # int32 [D][K]
    topk_val: np.ndarray  # float64 [D][K]
    utility: np.ndarray   # float64 [budget]; u of every emitted node (root: 1/den[0])

    def paths(self) -> list[tuple[int, ...]]:
        out: list[tuple[int, ...]] = [()]
        for i in range(1, self.n):
            out.append(out[int(self.parent[i])] + (int(self.rank[i]),))
        return out


# ------------------------------------------------------------ Stage 1: top-K
def topk_row(x: np.ndarray, K: int) -> tuple[np.ndarray, np.ndarray]:
    """The K largest entries of one marginal row: indices and exact values.

    A stable ascending sort of -x orders values descending with ties kept in
    index order; NaN sorts last (below -inf), and -0.0 / +0.0 compare equal.
    """
    x = np.asarray(x, dtype=np.float64)
    order = np.argsort(-x, kind="stable")[:K]
    return order.astype(np.int32), x[order]


# ------------------------------------------------------------ Eq. 1
def edge_factors(vals: np.ndarray, kind: int, beta: float) -> np.ndarray:
    """q_cond of a rank-r child of any depth-i node, c[i][r] (Eq. 1).

    Sibling softmax over the K children.  LOGITS: e_r = EXP(beta*(x_r - x_0));
    PROBS: e_r = x_r when positive, else 0.  Z is summed in rank order;
    c = e/Z, or 0 for the whole row when Z is zero or not finite.
    """
    D, K = vals.shape
    c = np.zeros((D, K), dtype=np.float64)
    for i in range(D):
        if kind == LOGITS:
            x0 = float(vals[i, 0])
            e = [spec_exp(beta * (float(vals[i, r]) - x0)) for r in range(K)]
        else:
            e = [float(v) if float(v) > 0.0 else 0.0 for v in vals[i]]
        Z = 0.0
        for r in range(K):
            Z = Z + e[r]
        if Z > 0.0 and np.isfinite(Z):
            for r in range(K):
                c[i, r] = e[r] / Z
    return c


def marginal_normaliser(row: np.ndarray, M: float) -> float:
    """Z of the marginal scorer for one row of logits with maximum M: the sum over every
    vocabulary entry of EXP(x_j - M) rounded to the nearest multiple of 2^-42 (half to
    even), summed exactly as integers, then converted to the nearest double."""
    with np.errstate(invalid="ignore"):     # inf - inf: NaN, which contributes 0
        t = spec_exp_array(np.asarray(row, dtype=np.float64) - M)
    z = int(np.rint(t * Z_GRID).astype(np.int64).sum(dtype=np.int64))
    return float(Fraction(z) / Fraction(int(Z_GRID)))


def marginal_factors(vals: np.ndarray, rows: np.ndarray | None, kind: int) -> np.ndarray:
    """q_cond of the marginal scorer, c[i][r]: the full-vocabulary probability of the
    rank-r candidate of row i (0 for a row whose normaliser is 0 or not finite)."""
    D, K = vals.shape
    c = np.zeros((D, K), dtype=np.float64)
    for i in range(D):
        if kind == PROBS:   # the probability, clamped into [0, 1] (NaN: 0)
            c[i] = [min(float(v), 1.0) if float(v) > 0.0 else 0.0 for v in vals[i]]
            continue
        M = float(vals[i, 0])
        Z = marginal_normaliser(rows[i], M)
        if Z > 0.0 and np.isfinite(Z):
            for r in range(K):
                c[i, r] = spec_exp(float(vals[i, r]) - M) / Z
    return c


# ------------------------------------------------------------ Eq. 3 denominator
def denominators(D: int, lambda1: float, lambda2: float) -> np.ndarray:
    return np.array([lambda1 + lambda2 * d for d in range(D + 1)], dtype=np.float64)


def _order_key(u: float, depth: int, path: tuple[int, ...]):
    # larger key = earlier in the total order: u desc, depth asc, path lex asc
    return (u, -depth, tuple(-r for r in path))


# ------------------------------------------------------------ Alg. 1 (best-first form)
def select_request(marg_rows: np.ndarray, K: int, budget: int, kind: int = LOGITS,
                   lambda1: float = 1.0, lambda2: float = 0.125, tau: float = 0.0,
                   beta: float = 1.0, scorer: int = SIBLING, mlp=None, req: int = 0) -> Tree:
    """Greedy prefix-closed selection of Alg. 1 for one request.

    The argmax of Alg. 1 over all unselected trie nodes always lies among the
    children of already-selected nodes: q_cond <= 1 and a non-decreasing
    denominator make u(child) <= u(parent) in floating point, and the depth
    tie-break puts a parent first on equal u.  So every iteration adds exactly
    one node whose ancestors are already in S; this loop keeps all children of
    selected nodes in a priority queue and pops the best one.  Alg. 1 returns a
    set; it is emitted breadth first (depth, then rank path).
    """
    D = marg_rows.shape[0]
    idx = np.zeros((D, K), dtype=np.int32)
    val = np.zeros((D, K), dtype=np.float64)
    for i in range(D):
        idx[i], val[i] = topk_row(marg_rows[i], K)
    if scorer == MARGINAL:
        c = marginal_factors(val, marg_rows, kind)
    elif scorer == LEARNED:        # c[depth][parent rank][child rank] (oracle.scorer)
        from .scorer import scorer_table
        c = scorer_table(mlp, req, marg_rows, idx, val)
    else:
        c = edge_factors(val, kind, beta)
    den = denominators(D, lambda1, lambda2)

    parent = [-1]
    token = [-1]
    depth = [0]
    rank = [-1]
    q = [1.0]
    util = [1.0 / den[0]]
    paths: list[tuple[int, ...]] = [()]

    heap: list = []
    tie = itertools.count()

    def push_children(pos: int):
        d = depth[pos]
        if d >= D:
            return
        for r in range(K):
            qc = q[pos] * edge_q(c, d, paths[pos], r)
            uc = qc / den[d + 1]
            p = paths[pos] + (r,)
            k = _order_key(uc, d + 1, p)
            # heapq is a min-heap: negate the order so the best node pops first
            heapq.heappush(heap, ((-k[0], -k[1], tuple(-x for x in k[2])), next(tie),
                                  (pos, r, qc, uc, p)))

    push_children(0)
    while len(parent) < budget and heap:
        _, _, (pos, r, qc, uc, p) = heap[0]
        if not uc > tau:
            break
        heapq.heappop(heap)
        parent.append(pos)
        token.append(int(idx[depth[pos], r]))
        depth.append(depth[pos] + 1)
        rank.append(r)
        q.append(qc)
        util.append(uc)
        paths.append(p)
        push_children(len(parent) - 1)

    # emit S breadth first: by depth, then by rank path (parents still precede children)
    n = len(parent)
    order = sorted(range(n), key=lambda i: (depth[i], paths[i]))
    new = {old: k for k, old in enumerate(order)}
    pad = budget - n
    return Tree(
        parent=np.array([-1 if parent[i] < 0 else new[parent[i]] for i in order] + [-1] * pad,
                        dtype=np.int32),
        token=np.array([token[i] for i in order] + [-1] * pad, dtype=np.int32),
        depth=np.array([depth[i] for i in order] + [-1] * pad, dtype=np.int32),
        rank=np.array([rank[i] for i in order] + [-1] * pad, dtype=np.int32),
        q_reach=np.array([q[i] for i in order] + [0.0] * pad, dtype=np.float64),
        n=n, topk_idx=idx, topk_val=val,
        utility=np.array([util[i] for i in order] + [0.0] * pad, dtype=np.float64),
    )


def select_batch(marginals_f64: np.ndarray, K: int, budget: int, **kw) -> list[Tree]:
    return [select_request(marginals_f64[b], K, budget, **kw) for b in range(marginals_f64.shape[0])]


def edge_q(c: np.ndarray, d: int, parent_path: tuple[int, ...], r: int) -> float:
    """q_cond of the rank-r child of the node at rank path parent_path (depth d): c[d][r]
    for the scorers whose factor depends on (row, rank) only, c[d][parent rank][r] for
    the learned scorer's table (the root's parent rank is 0)."""
    if c.ndim == 3:
        return c[d, parent_path[-1] if parent_path else 0, r]
    return c[d, r]


# ------------------------------------------------------------ pins: literal Alg. 1 and brute force
def enumerate_trie(c: np.ndarray, den: np.ndarray, max_depth: int | None = None):
    """Every node of the implicit trie: dict path -> (q_reach, utility)."""
    D, K = c.shape[0], c.shape[-1]
    max_depth = D if max_depth is None else max_depth
    nodes = {(): (1.0, 1.0 / den[0])}
    level = [()]
    for d in range(max_depth):
        nxt = []
        for p in level:
            qp = nodes[p][0]
            for r in range(K):
                qc = qp * edge_q(c, d, p, r)
                nodes[p + (r,)] = (qc, qc / den[d + 1])
                nxt.append(p + (r,))
        level = nxt
    return nodes


def select_literal_alg1(c: np.ndarray, den: np.ndarray, budget: int, tau: float):
    """Alg. 1 as printed: q for every trie node, then repeatedly add the
    argmax-utility node outside S together with its ancestors.

    Returns the list of rank paths in the order they entered S, and whether
    any iteration had to add an ancestor (the lemma says it never does).
    """
    nodes = enumerate_trie(c, den)
    S = [()]
    in_S = {()}
    added_ancestor = False
    while len(S) < budget:
        best = None
        for p, (qv, uv) in nodes.items():
            if p in in_S:
                continue
            if best is None or _order_key(uv, len(p), p) > _order_key(nodes[best][1], len(best), best):
                best = p
        if best is None or not nodes[best][1] > tau:
            break
        for j in range(1, len(best)):
            a = best[:j]
            if a not in in_S:
                added_ancestor = True
                S.append(a)
                in_S.add(a)
        S.append(best)
        in_S.add(best)
    return S, added_ancestor


def _connected_subtrees(children, root, max_size):
    """All node sets that contain ``root``, are closed under parent, and have size <= max_size."""
    out = []

    def extend(current, frontier):
        out.append(frozenset(current))
        if len(current) == max_size:
            return
        frontier = list(frontier)
        for i, v in enumerate(frontier):
            # include v; later frontier entries stay optional, earlier ones are excluded
            extend(current + [v], frontier[i + 1:] + children.get(v, []))

    extend([root], children.get(root, []))
    return out


def brute_force_best_set(c: np.ndarray, den: np.ndarray, budget: int, tau: float):
    """Maximum of sum(u - tau) over prefix-closed sets with the root and <= budget
    nodes, in exact rational arithmetic on the fp64 utilities; also returns every
    maximising set."""
    nodes = enumerate_trie(c, den)
    children: dict = {}
    for p in nodes:
        if p:
            children.setdefault(p[:-1], []).append(p)
    best_val = None
    best_sets = []
    for s in _connected_subtrees(children, (), budget):
        val = sum((Fraction(nodes[p][1]) - Fraction(tau) for p in s if p), Fraction(0))
        if best_val is None or val > best_val:
            best_val, best_sets = val, [s]
        elif val == best_val:
            best_sets.append(s)
    return best_val, best_sets, nodes
