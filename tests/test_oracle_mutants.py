"""Every plausible mistake planted in the oracle must fail at least one pin.

Each mutant replaces one oracle function (on the CPU, inside this test only)
with a copy carrying a single bug: a transposed operand, a dropped term, a
wrong sign or index, a reversed tie-break.
"""
import numpy as np
import pytest

import oracle.dartree_ref as R
from tests import pins

_orig = {name: getattr(R, name) for name in (
    "head_features", "vocab_logits", "log_softmax", "topk_ids", "select_level",
    "child_states", "path_score", "prune", "emit_tree", "rnd_bf16", "candidate_set",
    "candidate_logits", "heap_entry", "markov_states", "next_states", "acceptance_walk", "tree_attention",
    "mask_bit")}


def _head_transposed(r, A, H_d, precision):
    t = r @ A
    return t, R._rounder(precision)(np.tanh(t + H_d[None, :]))


def _head_no_hidden(r, A, H_d, precision):
    t = r @ A.T
    return t, R._rounder(precision)(np.tanh(t))


def _head_no_round(r, A, H_d, precision):
    t = r @ A.T
    return t, np.tanh(t + H_d[None, :])


def _logits_no_base(a, U, Lb_d, chunk=16384):
    return a @ U.T


def _logits_sign(a, U, Lb_d, chunk=16384):
    return Lb_d[None, :] - a @ U.T


def _lsm_no_norm(z, tau):
    return (z - z.max(axis=-1, keepdims=True)) / tau


def _lsm_no_tau(z, tau):
    return _orig["log_softmax"](z, 1.0)


def _topk_id_desc(z_row, k):
    order = np.lexsort((-np.arange(len(z_row)), -z_row))
    return order[:k]


def _topk_ascending(z_row, k):
    return np.lexsort((np.arange(len(z_row)), z_row))[:k]


def _select_token_first(parent, token, score, n_keep):
    return np.lexsort((parent, token, -score))[:n_keep]


def _child_no_scale(t_parent, U_tok, e, precision):
    return R._rounder(precision)(np.tanh(t_parent + U_tok))


def _child_no_parent(t_parent, U_tok, e, precision):
    return R._rounder(precision)(np.tanh(e * U_tok))


def _score_no_beta(s_parent, logp, beta):
    return s_parent + logp


def _score_no_parent(s_parent, logp, beta):
    return logp + beta


def _prune_depth_desc(levels, budget):
    depth = np.concatenate([np.full(len(l.token), d + 1) for d, l in enumerate(levels)])
    slot = np.concatenate([np.arange(len(l.token)) for l in levels])
    score = np.concatenate([l.score for l in levels])
    order = np.lexsort((slot, -depth, -score))[:min(budget, len(score))]
    return [(int(depth[i]), int(slot[i])) for i in order]


def _prune_off_by_one(levels, budget):
    return _orig["prune"](levels, budget - 1)


def _emit_token_order(levels, kept, budget):
    out = _orig["emit_tree"](levels, kept, budget)
    tokens, parents, depths, scores, mask, n = out
    # forget the mask's ancestor bits: self only
    m2 = np.zeros_like(mask)
    for i in range(n):
        m2[i, i // 64] |= np.uint64(1) << np.uint64(i % 64)
    return tokens, parents, depths, scores, m2, n


def _rnd_truncate(x):
    u = np.asarray(x, np.float64).astype(np.float32).view(np.uint32) & np.uint32(0xFFFF0000)
    return u.view(np.float32).astype(np.float64)


def _cset_lowest(Lb_d, K):
    return np.lexsort((np.arange(len(Lb_d)), Lb_d))[:K]


def _cset_id_order(Lb_d, K):
    return np.arange(K)


def _cand_logits_full_vocab(a, U, Lb_d, cset):
    return R.vocab_logits(a, U, Lb_d)


def _cand_logits_no_base(a, U, Lb_d, cset):
    z = np.full((a.shape[0], U.shape[0]), -np.inf)
    z[:, cset] = a @ U[cset].T
    return z


def _heap_breadth_first(score, depth, parent, rank, token):
    return (depth, parent, rank, token)


def _heap_prefers_descendants(score, depth, parent, rank, token):
    return (-score, -depth, parent, rank, token)


def _heap_min_first(score, depth, parent, rank, token):
    return (score, depth, parent, rank, token)


def _markov_no_scale(U_tok, e, precision):
    return R._rounder(precision)(U_tok)


def _next_ignores_head(p, t_parent, U_tok):
    return R.child_states(t_parent, U_tok, p.embed_scale, p.precision)


def _walk_own_target(tokens, parents, num_nodes, target):
    # reads the target at the child's own index instead of its parent's position
    cur, path = -1, []
    while True:
        kids = [j for j in range(int(num_nodes)) if int(parents[j]) == cur]
        match = [j for j in kids if int(tokens[j]) == int(target[j + 1])]
        if not match:
            return path, int(target[cur + 1])
        cur = match[0]
        path.append(cur)


def _walk_no_bonus(tokens, parents, num_nodes, target):
    path, bonus = _orig["acceptance_walk"](tokens, parents, num_nodes, target)
    return path, int(target[0])


def _attn_all_nodes(q, k_ctx, v_ctx, k_tree, v_tree, mask, ctx_len, scale):
    full = np.full_like(mask, np.uint64(0xFFFFFFFFFFFFFFFF))
    return _orig["tree_attention"](q, k_ctx, v_ctx, k_tree, v_tree, full, ctx_len, scale)


def _attn_no_scale(q, k_ctx, v_ctx, k_tree, v_tree, mask, ctx_len, scale):
    return _orig["tree_attention"](q, k_ctx, v_ctx, k_tree, v_tree, mask, ctx_len, 1.0)


def _mask_bit_transposed(mask, i, j):
    return bool((int(mask[j, i // 64]) >> (i % 64)) & 1) if j < mask.shape[0] else False


MUTANTS = {
    "walk_reads_child_target": ("acceptance_walk", _walk_own_target),
    "walk_bonus_always_first": ("acceptance_walk", _walk_no_bonus),
    "attention_ignores_mask": ("tree_attention", _attn_all_nodes),
    "attention_unscaled": ("tree_attention", _attn_no_scale),
    "attention_mask_transposed": ("mask_bit", _mask_bit_transposed),
    "markov_embedding_unscaled": ("markov_states", _markov_no_scale),
    "markov_head_ignored": ("next_states", _next_ignores_head),
    "heap_breadth_first": ("heap_entry", _heap_breadth_first),
    "heap_prefers_descendants": ("heap_entry", _heap_prefers_descendants),
    "heap_pops_worst": ("heap_entry", _heap_min_first),
    "cset_lowest_values": ("candidate_set", _cset_lowest),
    "cset_first_ids": ("candidate_set", _cset_id_order),
    "cand_logits_full_vocab": ("candidate_logits", _cand_logits_full_vocab),
    "cand_logits_drop_base": ("candidate_logits", _cand_logits_no_base),
    "head_transposed_A": ("head_features", _head_transposed),
    "head_drops_hidden": ("head_features", _head_no_hidden),
    "head_skips_bf16_rounding": ("head_features", _head_no_round),
    "logits_drop_base": ("vocab_logits", _logits_no_base),
    "logits_wrong_sign": ("vocab_logits", _logits_sign),
    "log_softmax_unnormalised": ("log_softmax", _lsm_no_norm),
    "log_softmax_ignores_tau": ("log_softmax", _lsm_no_tau),
    "topk_ties_id_desc": ("topk_ids", _topk_id_desc),
    "topk_ascending": ("topk_ids", _topk_ascending),
    "select_tiebreak_swapped": ("select_level", _select_token_first),
    "child_no_embed_scale": ("child_states", _child_no_scale),
    "child_ignores_parent": ("child_states", _child_no_parent),
    "score_drops_beta": ("path_score", _score_no_beta),
    "score_drops_parent": ("path_score", _score_no_parent),
    "prune_prefers_descendants": ("prune", _prune_depth_desc),
    "prune_budget_off_by_one": ("prune", _prune_off_by_one),
    "mask_without_ancestors": ("emit_tree", _emit_token_order),
    "bf16_truncates": ("rnd_bf16", _rnd_truncate),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(R, attr, fn)
    caught = []
    for pin in pins.PINS:
        try:
            pin()
        except AssertionError:
            caught.append(pin.__name__)
        except Exception as exc:  # a crash also exposes the mutant
            caught.append(f"{pin.__name__}:{type(exc).__name__}")
    assert caught, f"mutant {name} passed every pin"
