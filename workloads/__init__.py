"""Seeded synthetic inputs for one TAPS verification round.

This module only draws random numbers and lays them out; it holds none of the
method's arithmetic (no top-K, no scores, no selection, no attention).  Both the
CPU oracle and the HIP path take their inputs from here.

Workload recipe (shapes follow the paper's setting: Qwen3 vocabulary of 151,936
tokens, a draft block of 16 positions (Sec. 5.1, Baselines), trees of about 64
verification nodes (Sec. 5.2, Budget-Controlled Verification), Qwen3-8B-style
grouped-query attention with 32 query heads, 8 KV heads and head_dim 128):

* ``tiny``      [8, 1000] fp32 probabilities (N(0,1) logits plus +4 at one
  seeded token per row, softmaxed); K=4, budget 16; 4/2/64 heads over 256
  context rows; Q, K, V are N(0,1)/8 in fp32.
* ``qwen3_4b``  [16, 151936] bf16 logits 3*N(0,1) plus a spike at one seeded
  token per row decaying linearly from +8 (row 0) to +2 (last row); K=8,
  budget 32; 32/8/128 heads over 2048 context rows, N(0,1) bf16.
* ``qwen3_8b``  as qwen3_4b with budget 64 over 8192 context rows.
* ``serve16``   16 requests shaped like qwen3_8b with budget 128, contexts
  drawn log-uniform in [512, 16384], a ragged KV cache indexed by row offsets,
  and a per-request acceptance probability drawn uniform in [0.4, 0.9].
* ``stress``    4 requests, [32, 151936] bf16 logits 1.5*N(0,1) plus +3 at the
  spike; K=16, budget 256; 32/8/128 heads over 32768 context rows.

Target tokens (the target model's greedy choice after each node) are the
draft's top-1 at the next position with probability ``p_acc``, else uniform over
the vocabulary; the draws are keyed by a SplitMix64 hash of (seed, config,
request, rank path) so they do not depend on the order nodes are emitted in.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

BASE_SEED = 20260601

# stream ids for the per-purpose generators
_S_NOISE, _S_SPIKE, _S_Q, _S_K, _S_V, _S_CTX, _S_PACC = range(7)

LOGITS = 0
PROBS = 1
BF16 = 0
FP32 = 1


@dataclasses.dataclass(frozen=True)
class Config:
    name: str
    cfg_id: int
    batch: int
    block: int
    vocab: int
    K: int
    budget: int
    Hq: int
    Hkv: int
    head_dim: int
    ctx: int | None           # fixed context length, or None for the ragged draw
    kind: int                 # LOGITS or PROBS
    dtype: int                # BF16 or FP32
    noise_sigma: float
    spike_first: float
    spike_last: float
    p_acc: float | None       # fixed acceptance probability, or None for the per-request draw
    ctx_lo: int = 512
    ctx_hi: int = 16384
    lambda1: float = 1.0
    lambda2: float = 0.125
    tau: float = 0.0
    beta: float = 1.0

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim)


CONFIGS = {
    "tiny": Config("tiny", 0, 1, 8, 1000, 4, 16, 4, 2, 64, 256, PROBS, FP32,
                   1.0, 4.0, 4.0, 0.7),
    "qwen3_4b": Config("qwen3_4b", 1, 1, 16, 151936, 8, 32, 32, 8, 128, 2048, LOGITS, BF16,
                       3.0, 8.0, 2.0, 0.7),
    "qwen3_8b": Config("qwen3_8b", 2, 1, 16, 151936, 8, 64, 32, 8, 128, 8192, LOGITS, BF16,
                       3.0, 8.0, 2.0, 0.7),
    "serve16": Config("serve16", 3, 16, 16, 151936, 8, 128, 32, 8, 128, None, LOGITS, BF16,
                      3.0, 8.0, 2.0, None),
    "stress": Config("stress", 4, 4, 32, 151936, 16, 256, 32, 8, 128, 32768, LOGITS, BF16,
                     1.5, 3.0, 3.0, 0.7),
}


def rng(cfg_id: int, b: int, stream: int, seed: int = BASE_SEED) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([seed, cfg_id, b, stream]))


# ---------------------------------------------------------------- bf16 storage
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round to nearest even; NaN -> 0x7FC0."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)).astype(np.uint16)
    nan = np.isnan(np.asarray(x, dtype=np.float32))
    r[nan] = np.uint16(0x7FC0)
    return r


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


# ---------------------------------------------------------------- SplitMix64
_M64 = (1 << 64) - 1


def splitmix64(x: int) -> int:
    """One SplitMix64 output step (Steele, Lea, Flood 2014) applied to state x."""
    z = (x + 0x9E3779B97F4A7C15) & _M64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _M64
    return z ^ (z >> 31)


def path_hash(seed: int, cfg_id: int, b: int, path: tuple[int, ...], salt: int) -> int:
    h = splitmix64(seed)
    for x in (cfg_id, b, salt, len(path), *path):
        h = splitmix64(h ^ (x & _M64))
    return h


def unit_from_hash(h: int) -> float:
    return (h >> 11) * (1.0 / (1 << 53))


# ---------------------------------------------------------------- inputs
@dataclasses.dataclass
class RoundInputs:
    cfg: Config
    marginals: np.ndarray     # [B][D][V]: uint16 bf16 bits, or float32
    ctx_len: np.ndarray       # [B] int32
    kv_offset: np.ndarray     # [B] int64, first KV row of each request
    p_acc: np.ndarray         # [B] float64
    Q: np.ndarray | None      # [B][N][Hq][hd]: uint16 bf16 bits, or float32
    K: np.ndarray | None      # [rows][Hkv][hd]
    V: np.ndarray | None
    seed: int

    @property
    def total_rows(self) -> int:
        return int(self.kv_offset[-1] + self.ctx_len[-1] + self.cfg.budget)

    def marginals_f64(self) -> np.ndarray:
        if self.cfg.dtype == BF16:
            return bf16_bits_to_f32(self.marginals).astype(np.float64)
        return self.marginals.astype(np.float64)

    def qkv_f64(self):
        conv = (lambda a: bf16_bits_to_f32(a).astype(np.float64)) if self.cfg.dtype == BF16 \
            else (lambda a: a.astype(np.float64))
        return conv(self.Q), conv(self.K), conv(self.V)


def _store(x32: np.ndarray, dtype: int) -> np.ndarray:
    return f32_to_bf16_bits(x32) if dtype == BF16 else np.ascontiguousarray(x32, dtype=np.float32)


def gen_marginals(cfg: Config, seed: int = BASE_SEED) -> np.ndarray:
    D, V = cfg.block, cfg.vocab
    rows = []
    for b in range(cfg.batch):
        noise = rng(cfg.cfg_id, b, _S_NOISE, seed).standard_normal((D, V), dtype=np.float32)
        x = noise * np.float32(cfg.noise_sigma)
        spike_tok = rng(cfg.cfg_id, b, _S_SPIKE, seed).integers(0, V, size=D)
        for i in range(D):
            t = i / (D - 1) if D > 1 else 0.0
            x[i, spike_tok[i]] += np.float32(cfg.spike_first + (cfg.spike_last - cfg.spike_first) * t)
        if cfg.kind == PROBS:
            z = x.astype(np.float64)
            z = np.exp(z - z.max(axis=1, keepdims=True))
            x = (z / z.sum(axis=1, keepdims=True)).astype(np.float32)
        rows.append(x)
    return _store(np.stack(rows), cfg.dtype)


def gen_ctx(cfg: Config, seed: int = BASE_SEED) -> np.ndarray:
    if cfg.ctx is not None:
        return np.full(cfg.batch, cfg.ctx, dtype=np.int32)
    out = np.empty(cfg.batch, dtype=np.int32)
    for b in range(cfg.batch):
        u = rng(cfg.cfg_id, b, _S_CTX, seed).uniform(math.log(cfg.ctx_lo), math.log(cfg.ctx_hi))
        out[b] = int(round(math.exp(u)))
    return out


def gen_p_acc(cfg: Config, seed: int = BASE_SEED) -> np.ndarray:
    if cfg.p_acc is not None:
        return np.full(cfg.batch, cfg.p_acc, dtype=np.float64)
    return np.array([rng(cfg.cfg_id, b, _S_PACC, seed).uniform(0.4, 0.9) for b in range(cfg.batch)])


def kv_offsets(ctx_len: np.ndarray, budget: int) -> np.ndarray:
    rows = ctx_len.astype(np.int64) + budget
    return np.concatenate([[0], np.cumsum(rows)[:-1]]).astype(np.int64)


def gen_round(cfg: Config | str, seed: int = BASE_SEED, with_attention: bool = True) -> RoundInputs:
    if isinstance(cfg, str):
        cfg = CONFIGS[cfg]
    marg = gen_marginals(cfg, seed)
    ctx = gen_ctx(cfg, seed)
    off = kv_offsets(ctx, cfg.budget)
    p = gen_p_acc(cfg, seed)
    Q = K = V = None
    if with_attention:
        sig = np.float32(1.0 / math.sqrt(cfg.head_dim)) if cfg.dtype == FP32 else np.float32(1.0)
        total = int(off[-1] + ctx[-1] + cfg.budget)
        qs, ks, vs = [], [], []
        for b in range(cfg.batch):
            qs.append(rng(cfg.cfg_id, b, _S_Q, seed).standard_normal(
                (cfg.budget, cfg.Hq, cfg.head_dim), dtype=np.float32) * sig)
            rows_b = int(ctx[b]) + cfg.budget
            ks.append(rng(cfg.cfg_id, b, _S_K, seed).standard_normal(
                (rows_b, cfg.Hkv, cfg.head_dim), dtype=np.float32) * sig)
            vs.append(rng(cfg.cfg_id, b, _S_V, seed).standard_normal(
                (rows_b, cfg.Hkv, cfg.head_dim), dtype=np.float32) * sig)
        Q = _store(np.stack(qs), cfg.dtype)
        K = _store(np.concatenate(ks), cfg.dtype)
        V = _store(np.concatenate(vs), cfg.dtype)
        assert K.shape[0] == total
    return RoundInputs(cfg, marg, ctx, off, p, Q, K, V, seed)


def gen_scorer_weights(rng: np.random.Generator, vocab: int, d: int, h: int, batch: int) -> dict:
    """Seeded random weights for the learned-scorer hook (no trained weights exist here):
    float32 emb [vocab][d], W1 [h][2d+3], b1 [h], w2 [h], the float32 b2 and int32 root
    tokens [batch]."""
    F = 2 * d + 3
    return dict(
        emb=(rng.standard_normal((vocab, d)) * 0.5).astype(np.float32),
        W1=(rng.standard_normal((h, F)) / np.sqrt(F)).astype(np.float32),
        b1=(rng.standard_normal(h) * 0.1).astype(np.float32),
        w2=(rng.standard_normal(h) / np.sqrt(h)).astype(np.float32),
        b2=float(np.float32(rng.standard_normal() * 0.1)),
        root_token=rng.integers(0, vocab, size=batch).astype(np.int32))


def rank_paths(parent: np.ndarray, rank: np.ndarray, n: int) -> list[tuple[int, ...]]:
    """Rank path of every emitted node, read off parent pointers (node 0 is the root)."""
    paths: list[tuple[int, ...]] = [()]
    for i in range(1, n):
        paths.append(paths[int(parent[i])] + (int(rank[i]),))
    return paths


def target_tokens(cfg: Config, b: int, parent: np.ndarray, rank: np.ndarray, n: int,
                  top1_next: np.ndarray, p_acc: float, seed: int = BASE_SEED,
                  branch: bool = False, token: np.ndarray | None = None) -> np.ndarray:
    """Synthetic greedy target choice after each of the n nodes (rest of the budget: -1).

    ``top1_next[d]`` is the draft's top-1 token at draft position d (the token a
    depth-d node's child would carry at rank 0).  With ``branch`` set, an
    accepted draw picks one of the node's emitted children uniformly instead,
    so walks leave the rank-0 chain (needs ``token``).
    """
    out = np.full(cfg.budget, -1, dtype=np.int32)
    paths = rank_paths(parent, rank, n)
    kids: dict[int, list[int]] = {}
    for i in range(1, n):
        kids.setdefault(int(parent[i]), []).append(i)
    D = len(top1_next)
    for i in range(n):
        path = paths[i]
        u = unit_from_hash(path_hash(seed, cfg.cfg_id, b, path, 1))
        uni = int(path_hash(seed, cfg.cfg_id, b, path, 2) % cfg.vocab)
        pick = path_hash(seed, cfg.cfg_id, b, path, 3)
        if u < p_acc:
            if branch and i in kids:
                out[i] = int(token[kids[i][pick % len(kids[i])]])
            elif len(path) < D:
                out[i] = int(top1_next[len(path)])
            else:
                out[i] = uni
        else:
            out[i] = uni
    return out
