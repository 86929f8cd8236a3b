"""The consumer of the emitted tree on the GPU against the oracle: the
acceptance walk (bit-exact: it is integer work) and one tree-attention layer.

Tolerance of the attention output.  Scores q.k are bf16 products accumulated
in fp32 (relative error ~1e-6 at head size 128, negligible here); the softmax
weights p_j = exp(s_j - m) are rounded to bf16 (relative error <= 2^-9) before
the weighted sum of values, while the normaliser sums the unrounded weights.
The rounding moves the output by at most 2^-9 sum_j p_j |v_j| / sum_j p_j <=
2^-9 max|v|, and the unrounded normaliser by the same bound again, so every
element must agree within 2^-8 max|v| (plus 1e-5 for the fp32 sums)."""
import numpy as np
import pytest
import torch

import oracle.dartree_ref as R
from paper_2608_13524_amd import dartree as D
from paper_2608_13524_amd import workloads as W
from tests.gpu_util import device, run_build, say, to_dev
from tests.pins import run_oracle, tiny
from tests.test_gpu_heap import run_heap
from tests.test_gpu_parity import small

pytestmark = pytest.mark.gpu


def targets_for(tokens, parents, num_nodes, V, rng, p_match=0.85):
    """Target tokens per position that continue into a random child with
    probability p_match (else a random, possibly absent, token)."""
    b, B = tokens.shape
    t = rng.integers(0, V, size=(b, B + 1)).astype(np.int32)
    for q in range(b):
        n = int(num_nodes[q])
        for pos in range(-1, n):
            kids = np.nonzero(parents[q, :n] == pos)[0]
            if len(kids) and rng.random() < p_match:
                t[q, pos + 1] = tokens[q, rng.choice(kids)]
    return t


def run_walk(tree, target, max_len):
    dev = device()
    b = tree["tokens"].shape[0]
    acc = torch.empty(b, max_len, dtype=torch.int32, device=dev)
    n = torch.empty(b, dtype=torch.int32, device=dev)
    bonus = torch.empty(b, dtype=torch.int32, device=dev)
    say(f"accept_walk b={b} B={tree['tokens'].shape[1]} max_len={max_len}")
    D.accept_walk(to_dev(tree["tokens"]), to_dev(tree["parents"]), to_dev(tree["num_nodes"]), to_dev(target),
                  acc, n, bonus)
    torch.cuda.synchronize()
    return acc.cpu().numpy(), n.cpu().numpy(), bonus.cpu().numpy()


@pytest.mark.parametrize("kind", ["dartree", "heap", "chain"])
def test_accept_walk_bit_exact(kind):
    cfg = {"dartree": small(seed=90, batch=4), "heap": small(seed=91, batch=4, budget=40),
           "chain": small(seed=92, batch=4, width=1, budget=5)}[kind]
    inputs = W.make_inputs(cfg)
    tree = run_heap(cfg, inputs, states=False)[0] if kind == "heap" else run_build(cfg, inputs, export=False)[0]
    rng = np.random.default_rng(93)
    for trial in range(6):
        target = targets_for(tree["tokens"], tree["parents"], tree["num_nodes"], cfg.vocab, rng,
                             p_match=1.0 if trial == 0 else 0.85)
        for max_len in (cfg.depth, 2):
            acc, n, bonus = run_walk(tree, target, max_len)
            for q in range(cfg.batch):
                path, want_bonus = R.acceptance_walk(tree["tokens"][q], tree["parents"][q], tree["num_nodes"][q],
                                                     target[q])
                m = min(len(path), max_len)           # a walk stops after max_len nodes
                assert int(n[q]) == m
                assert acc[q, :m].tolist() == path[:m] and (acc[q, m:] == -1).all()
                want = want_bonus if m == len(path) else int(target[q, path[m - 1] + 1])
                assert int(bonus[q]) == want


def run_attention(ai: W.AttentionInputs, mask, budget, heads_q, heads_kv, scale, use_ctx_len=True):
    dev = device()
    b, max_ctx = ai.k_ctx.shape[0], ai.k_ctx.shape[1]
    p = D.AttnParams(b, budget, max_ctx, heads_q, heads_kv, 128, scale)
    nws = D.tree_attention_workspace_size(p)
    ws = torch.empty(nws, dtype=torch.uint8, device=dev) if nws else None
    out = torch.full((b, budget, heads_q, 128), float("nan"), dtype=torch.float32, device=dev)
    kc = to_dev(ai.k_ctx) if max_ctx else None
    vc = to_dev(ai.v_ctx) if max_ctx else None
    say(f"tree_attention b={b} B={budget} ctx={max_ctx} Hq={heads_q} Hkv={heads_kv}")
    D.tree_attention(p, to_dev(ai.q), kc, vc, to_dev(ai.k_tree), to_dev(ai.v_tree),
                     to_dev(np.ascontiguousarray(mask).view(np.int64)), to_dev(ai.ctx_len) if use_ctx_len else None,
                     out, ws)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def check_attention(ai, masks, got, scale, rows=None):
    f = lambda x: W.bf16_bits_to_fp32(x).astype(np.float64)
    vmax = max(np.abs(f(ai.v_ctx)).max() if ai.v_ctx.size else 0.0, np.abs(f(ai.v_tree)).max())
    tol = 2.0 ** -8 * vmax + 1e-5
    worst = 0.0
    for q in range(ai.q.shape[0]):
        want = R.tree_attention(f(ai.q[q]), f(ai.k_ctx[q]), f(ai.v_ctx[q]), f(ai.k_tree[q]), f(ai.v_tree[q]),
                                masks[q], int(ai.ctx_len[q]), scale)
        sel = slice(None) if rows is None else rows
        err = np.abs(got[q][sel] - want[sel])
        worst = max(worst, float(err.max()))
    assert worst <= tol, (worst, tol)
    return worst, tol


def tree_masks(b, budget, seed, vocab=60, depth=6, width=24, branch=5):
    cfg = tiny(seed=seed, batch=b, vocab=vocab, depth=depth, width=width, branch=branch, budget=budget)
    _, tree, _ = run_oracle(cfg)
    return tree.mask


ATTN = {
    # b, B, max_ctx, ctx_len, Hq, Hkv
    "ragged": (2, 20, 300, [300, 123], 8, 2),      # two context segments, 80 query rows (2 row tiles)
    "tree-only": (1, 37, 0, [0], 4, 4),            # no context; group of 1
    "wide-tree": (1, 130, 64, [64], 4, 1),         # 3 mask words, 3 key steps in the tree segment
    "single-node": (2, 1, 70, [70, 1], 8, 8),
    "empty-context-row": (2, 12, 256, [0, 256], 16, 4),
    "tree-only-pads": (1, 140, 0, [0], 4, 2),      # rows 125.. are pad slots that see nothing: zero
    # >= 512 (request, kv head, row tile) blocks: one block covers all keys, no merge
    "fused-ragged": (8, 130, 300, [300, 0, 17, 256, 299, 1, 64, 200], 32, 8),   # 8 x 8 x 9 tiles
    "fused-tree-only": (16, 200, 0, [0] * 16, 16, 2),                          # 16 x 2 x 25 tiles
}


@pytest.mark.parametrize("name", list(ATTN))
def test_tree_attention_matches_oracle(name):
    b, B, ctx, lens, Hq, Hkv = ATTN[name]
    ai = W.make_attention_inputs(b, B, ctx, Hq, Hkv, seed=94, ctx_len=lens)
    masks = tree_masks(b, B, seed=95)
    scale = 1.0 / np.sqrt(128)
    got = run_attention(ai, masks, B, Hq, Hkv, scale)
    worst, tol = check_attention(ai, masks, got, scale)
    print(name, "max err", worst, "tol", tol)


def test_tree_attention_qwen3_4b_shape():
    """Qwen3-4B's layer shape over a 2048-position context and a 64-node tree
    emitted by the GPU for the qwen3-4b workload (all rows checked)."""
    cfg = W.CONFIGS["qwen3-4b"]
    tree, _, _ = run_build(cfg, W.make_inputs(cfg), export=False)
    s = W.ATTENTION_QWEN3_4B
    ai = W.make_attention_inputs(1, cfg.budget, s["max_ctx"], s["heads_q"], s["heads_kv"], seed=96)
    scale = 1.0 / np.sqrt(128)
    got = run_attention(ai, tree["mask"], cfg.budget, s["heads_q"], s["heads_kv"], scale, use_ctx_len=False)
    worst, tol = check_attention(ai, tree["mask"], got, scale)
    print("qwen3-4b layer max err", worst, "tol", tol)
