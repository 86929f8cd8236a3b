"""Seeded synthetic inputs for DARTree draft-tree construction.

This module only draws random numbers and packs them into the input layout of
the library (drafter logits, drafter hidden states, prefix state, correction-head
weights). It holds none of the method's arithmetic; both the HIP path and the
CPU oracle consume what it produces.

Inputs stand in for the drafter outputs of the paper's workload (a DFlash-style
block drafter with a gamma=16 block over the Qwen3 vocabulary, Sec. 4.1); trained
drafters and benchmark prompts are not available,
so every tensor is drawn from a fixed distribution:

* weights ``A`` [h][h] and ``U`` [V][h] ~ N(0, sigma_w^2)
* prefix state ``r0`` [b][h] ~ N(0, 1), drafter hidden ``H`` [b][L][h] ~ N(0, 1)
* drafter logits ``Lb`` [b][L][V] ~ N(0, sigma_l^2) plus a ranked boost on a few
  distinct uniformly drawn tokens per position (``peak`` for a single planted
  token, or ``boost_max * rank**-zipf_s`` for ranks 1..n_boost).

Draw order is fixed: A from ``Generator(PCG64(SeedSequence([seed, 0])))``; row
block c of U (rows 4096*c onwards) from ``SeedSequence([seed, 2, c])`` so blocks
can be drawn on several threads; then, for request i, from ``Generator(PCG64(SeedSequence([seed, 1, i])))``: Lb
noise, boosted token ids (without replacement, per position), H, r0.  Every
request has its own stream, so a request draws the same values alone or in a
batch.  bf16 tensors are drawn in fp32 and rounded
to bfloat16 with round-to-nearest-even; they are returned as uint16 bit patterns.
"""
from __future__ import annotations

import concurrent.futures
import dataclasses
import os
from typing import Optional

import numpy as np

FP32 = 0
BF16 = 1
U_BLOCK_ROWS = 4096


@dataclasses.dataclass(frozen=True)
class Config:
    """One workload: tree shape, precision and input distribution."""

    name: str
    batch: int
    vocab: int
    hidden: int
    depth: int
    width: int
    branch: int
    budget: int
    temperature: float
    precision: int
    seed: int
    candidates: int = 0           # 0: full vocabulary; K > 0: shared C_d = TopK(L_d^base, K)
    head: int = 0                 # 0: recurrent (Elman) correction head; 1: Markov head
    depth_bonus: float = -0.2
    sigma_w: float = 0.02
    sigma_l: float = 2.0
    n_boost: int = 32
    boost_max: float = 10.0
    zipf_s: float = 1.1
    peak: Optional[float] = None  # single planted peak instead of a Zipf boost

    def replace(self, **kw) -> "Config":
        return dataclasses.replace(self, **kw)

    def level_sizes(self) -> list[int]:
        """n_d = min(W, n_{d-1} * k), n_0 = 1 (data independent)."""
        n, out = 1, []
        for _ in range(self.depth):
            n = min(self.width, n * self.branch)
            out.append(n)
        return out

    def supertree_size(self) -> int:
        return sum(self.level_sizes())


# The five workloads: a tiny fp32 case and four Qwen3-shaped bf16 cases
# (vocab 151936, hidden 2560 / 4096 / 5120, block depth 16).
CONFIGS = {
    "tiny": Config("tiny", batch=1, vocab=1024, hidden=64, depth=4, width=4,
                   branch=4, budget=16, temperature=0.0, precision=FP32, seed=0,
                   sigma_w=0.05, sigma_l=3.0, n_boost=1, peak=8.0),
    "qwen3-4b": Config("qwen3-4b", batch=1, vocab=151936, hidden=2560, depth=16,
                       width=8, branch=8, budget=64, temperature=0.0,
                       precision=BF16, seed=1),
    "qwen3-4b-wide": Config("qwen3-4b-wide", batch=1, vocab=151936, hidden=2560,
                            depth=16, width=32, branch=8, budget=256,
                            temperature=0.0, precision=BF16, seed=2),
    "qwen3-8b-x4": Config("qwen3-8b-x4", batch=4, vocab=151936, hidden=4096,
                          depth=16, width=16, branch=8, budget=128,
                          temperature=1.0, precision=BF16, seed=3),
    "stress-x16": Config("stress-x16", batch=16, vocab=151936, hidden=5120,
                         depth=16, width=64, branch=8, budget=512,
                         temperature=1.0, precision=BF16, seed=4, n_boost=64),
}
# The paper's default candidate set (Alg. 1 as printed; Sec. 4.1 "DARTree
# (pruned)": K = 64 candidates per position, width 12, B = 64, beta = -0.2):
# every node of a depth is scored over the same C_d = TopK(L_d^base, 64) and
# keeps all of it (branching k = K).
CONFIGS["qwen3-4b-shared"] = Config("qwen3-4b-shared", batch=1, vocab=151936, hidden=2560, depth=16,
                                    width=12, branch=64, budget=64, temperature=0.0,
                                    precision=BF16, seed=5, candidates=64)
CONFIGS["qwen3-8b-shared-x4"] = Config("qwen3-8b-shared-x4", batch=4, vocab=151936, hidden=4096,
                                       depth=16, width=12, branch=64, budget=64,
                                       temperature=1.0, precision=BF16, seed=6, candidates=64)
# The Markov correction head (DSpark-Markov, Table 3: Qwen3-4B, the same
# DARTree settings): the state is the previous token's embedding only.
CONFIGS["qwen3-4b-markov"] = Config("qwen3-4b-markov", batch=1, vocab=151936, hidden=2560, depth=16,
                                    width=12, branch=64, budget=64, temperature=0.0,
                                    precision=BF16, seed=7, candidates=64, head=1)
CONFIG_ORDER = ["tiny", "qwen3-4b", "qwen3-4b-wide", "qwen3-8b-x4", "stress-x16",
                "qwen3-4b-shared", "qwen3-8b-shared-x4", "qwen3-4b-markov"]


def fp32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bfloat16 (nearest, ties to even); return uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_fp32(bits: np.ndarray) -> np.ndarray:
    """Widen bfloat16 bit patterns to fp32 (exact)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclasses.dataclass
class Inputs:
    """Host copies of one round's inputs.

    For BF16 configs ``A``, ``U``, ``H`` and ``r0`` are uint16 bfloat16 bit
    patterns; for FP32 configs they are float32.  ``Lb`` is always float32.
    """

    cfg: Config
    Lb: np.ndarray   # [b][L][V] fp32
    H: np.ndarray    # [b][L][h]
    r0: np.ndarray   # [b][h]
    A: np.ndarray    # [h][h]
    U: np.ndarray    # [V][h]


def _normal(rng: np.random.Generator, shape, sigma: float) -> np.ndarray:
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if sigma != 1.0:
        x *= np.float32(sigma)
    return x


def _normal_blocks(seed: int, shape, sigma: float, precision: int) -> np.ndarray:
    """Draw a large 2-D weight block of rows at a time, one stream per block."""
    rows, cols = shape
    out = np.empty(shape, dtype=np.uint16 if precision == BF16 else np.float32)

    def fill(c: int) -> None:
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 2, c])))
        r = c * U_BLOCK_ROWS
        n = min(U_BLOCK_ROWS, rows - r)
        x = _normal(rng, (n, cols), sigma)
        out[r:r + n] = fp32_to_bf16_bits(x) if precision == BF16 else x

    nblocks = (rows + U_BLOCK_ROWS - 1) // U_BLOCK_ROWS
    workers = max(1, min(16, len(os.sched_getaffinity(0))))
    with concurrent.futures.ThreadPoolExecutor(workers) as pool:
        list(pool.map(fill, range(nblocks)))
    return out


def _pack(x: np.ndarray, precision: int) -> np.ndarray:
    return fp32_to_bf16_bits(x) if precision == BF16 else np.ascontiguousarray(x, np.float32)


def make_weights(cfg: Config):
    """Draw the shared correction-head weights (A, U) for ``cfg``."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([cfg.seed, 0])))
    A = _pack(_normal(rng, (cfg.hidden, cfg.hidden), cfg.sigma_w), cfg.precision)
    U = _normal_blocks(cfg.seed, (cfg.vocab, cfg.hidden), cfg.sigma_w, cfg.precision)
    return A, U


def boost_values(cfg: Config) -> np.ndarray:
    """Boost added to the ranked tokens of each position (rank 1 first)."""
    if cfg.peak is not None:
        return np.full(cfg.n_boost, cfg.peak, dtype=np.float32)
    ranks = np.arange(1, cfg.n_boost + 1, dtype=np.float64)
    return (cfg.boost_max * ranks ** (-cfg.zipf_s)).astype(np.float32)


def make_request(cfg: Config, i: int):
    """Draw request ``i``'s drafter logits, drafter hidden states and prefix state."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([cfg.seed, 1, i])))
    L, V, h = cfg.depth, cfg.vocab, cfg.hidden
    Lb = _normal(rng, (L, V), cfg.sigma_l)
    boost = boost_values(cfg)
    nb = min(cfg.n_boost, V)
    for d in range(L):
        ids = rng.choice(V, size=nb, replace=False)
        Lb[d, ids] += boost[:nb]
    H = _pack(_normal(rng, (L, h), 1.0), cfg.precision)
    r0 = _pack(_normal(rng, (h,), 1.0), cfg.precision)
    return Lb, H, r0


def make_inputs(cfg: Config, requests: Optional[list[int]] = None,
                weights=None) -> Inputs:
    """All inputs of one round for ``cfg``.

    ``requests`` selects which request indices to draw (default: all
    ``cfg.batch``); the returned batch holds them in that order, so a sampled
    subset of a large batch reproduces exactly the rows of the full batch.
    """
    if requests is None:
        requests = list(range(cfg.batch))
    A, U = weights if weights is not None else make_weights(cfg)
    parts = [make_request(cfg, i) for i in requests]
    Lb = np.stack([p[0] for p in parts])
    H = np.stack([p[1] for p in parts])
    r0 = np.stack([p[2] for p in parts])
    sub = cfg.replace(batch=len(requests))
    return Inputs(cfg=sub, Lb=Lb, H=H, r0=r0, A=A, U=U)


# ---------------------------------------------------------------------------
# The consumer of the emitted tree: one tree-attention layer's inputs
# ---------------------------------------------------------------------------
@dataclasses.dataclass
class AttentionInputs:
    """bf16 bit patterns (uint16) of one attention layer over a flattened tree:
    q [b][B][Hq][D], k_ctx / v_ctx [b][max_ctx][Hkv][D], k_tree / v_tree
    [b][B][Hkv][D]; ctx_len int32 [b]."""

    q: np.ndarray
    k_ctx: np.ndarray
    v_ctx: np.ndarray
    k_tree: np.ndarray
    v_tree: np.ndarray
    ctx_len: np.ndarray


# Qwen3-4B's attention shape (32 query heads, 8 key/value heads, head size
# 128) over a 2048-position verified context: the layer the paper's target
# runs on every verified tree.
ATTENTION_QWEN3_4B = dict(heads_q=32, heads_kv=8, head_dim=128, max_ctx=2048)


def make_attention_inputs(batch: int, budget: int, max_ctx: int, heads_q: int, heads_kv: int,
                          head_dim: int = 128, seed: int = 0, ctx_len=None) -> AttentionInputs:
    """Unit-normal queries, keys and values rounded to bf16, one stream per
    tensor (SeedSequence([seed, 3, tensor]))."""
    def draw(t, shape):
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 3, t])))
        return fp32_to_bf16_bits(rng.standard_normal(shape, dtype=np.float32))

    lens = np.full(batch, max_ctx, np.int32) if ctx_len is None else np.asarray(ctx_len, np.int32)
    return AttentionInputs(q=draw(0, (batch, budget, heads_q, head_dim)),
                           k_ctx=draw(1, (batch, max_ctx, heads_kv, head_dim)),
                           v_ctx=draw(2, (batch, max_ctx, heads_kv, head_dim)),
                           k_tree=draw(3, (batch, budget, heads_kv, head_dim)),
                           v_tree=draw(4, (batch, budget, heads_kv, head_dim)), ctx_len=lens)
