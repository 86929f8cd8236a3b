"""The sequential-heap replay comparator on the CPU: a trace made from the
oracle's own run passes with no events, and planted mistakes in a trace
(a pop out of order, a wrong score, a wrong child set, a wrong state, a
state or feature rounded to the wrong side away from a near-tie, a normaliser
beyond its fp32 bound) fail."""
import numpy as np
import pytest

import oracle.dartree_ref as R
from paper_2608_13524_amd import workloads as W
from tests import replay
from tests.pins import tiny


def trace_of(dec, runs):
    """The arrays dartree_export_heap would hold for these runs."""
    p = dec.p
    b, B, k, h = len(runs), p.budget, min(p.branch, p.vocab), p.hidden
    t = dict(tokens=np.full((b, B + 1), -1, np.int32), parents=np.full((b, B + 1), -1, np.int32),
             depths=np.zeros((b, B + 1), np.int32), scores=np.zeros((b, B + 1), np.float32),
             num_popped=np.zeros(b, np.int32), lse=np.zeros((B, b), np.float32),
             cand_logp=np.zeros((B, b, k), np.float32), cand_ids=np.zeros((B, b, k), np.int32),
             states=np.zeros((B + 1, b, h)))
    for q, run in enumerate(runs):
        n = len(run.token) - 1
        t["num_popped"][q] = n
        for s in range(1, n + 1):
            t["tokens"][q, s], t["parents"][q, s] = run.token[s], run.parent[s]
            t["depths"][q, s], t["scores"][q, s] = run.depth[s], run.score[s]
        for node, ex in run.expansions.items():
            t["lse"][node, q] = ex.lse
            t["cand_logp"][node, q] = ex.cand_logp
            t["cand_ids"][node, q] = ex.cand_ids
    if p.candidates > 0:
        t["csets"] = np.stack([[R.candidate_set(dec.Lb[q, d], p.candidates) for d in range(p.depth)]
                               for q in range(b)]).astype(np.int32)
    return t


def states_of(dec, runs):
    """Each expanded slot's state and feature row, recomputed along the
    oracle's own pops: (states [B+1][b][h], features [B][b][h])."""
    p = dec.p
    out = np.zeros((p.budget + 1, len(runs), p.hidden))
    feat = np.zeros((p.budget, len(runs), p.hidden))
    for q, run in enumerate(runs):
        t0, a0 = R.head_features(dec.r0[q][None, :], dec.A, dec.H[q, 0], p.precision)
        t_of = {0: t0[0]}
        feat[0, q] = a0[0]
        for n in sorted(run.expansions):
            if n == 0:
                continue
            r = R.next_states(p, t_of[run.parent[n]][None, :], dec.U[run.token[n]][None, :])[0]
            out[n, q] = r
            t, a = R.head_features(r[None, :], dec.A, dec.H[q, run.depth[n]], p.precision)
            t_of[n] = t[0]
            feat[n, q] = a[0]
    return out, feat


def tree_dict(tree):
    return {"tokens": tree.tokens, "parents": tree.parents, "depths": tree.depths,
            "scores": tree.scores.astype(np.float32), "mask": tree.mask, "num_nodes": tree.num_nodes}


def _setup(**kw):
    cfg = tiny(**{**dict(batch=2, vocab=9, depth=3, branch=3, budget=8, precision=W.BF16, seed=80), **kw})
    dec = R.prepare(W.make_inputs(cfg))
    tree, runs = R.sequential_heap_tree(dec)
    return dec, runs, trace_of(dec, runs), tree_dict(tree)


@pytest.mark.parametrize("kw", [dict(), dict(candidates=5, branch=4), dict(precision=W.FP32, temperature=0.7),
                                dict(budget=60, depth=2)])   # 60 > 3 + 9: the heap runs dry
def test_oracle_trace_passes(kw):
    dec, runs, trace, tree = _setup(**kw)
    st, ft = states_of(dec, runs)
    rep = replay.follow_heap(dec, trace, tree, [0, 1], [0, 1], gpu_states=st, gpu_features=ft)
    assert rep.events == 0 and rep.max_score_err < 1e-6 and rep.state_ties == 0 and rep.feature_ties == 0
    assert rep.state_elems > 0 and rep.feature_elems > 0 and rep.max_lse_ratio <= 1 and rep.max_logp_ratio <= 1
    rep = replay.follow_heap(dec, trace, tree, [0, 1], [0, 1])
    assert rep.events == 0


def _swap_pops(trace, tree, runs, q):
    """Exchange the first two pops that are siblings with scores more than
    1e-3 apart (the emitted tree is unchanged, the pop order is wrong)."""
    run = runs[q]
    for s in range(1, len(run.token) - 1):
        if run.parent[s] == run.parent[s + 1] and run.score[s] - run.score[s + 1] > 1e-2:
            for f in ("tokens", "scores"):
                trace[f][q, s], trace[f][q, s + 1] = trace[f][q, s + 1], trace[f][q, s]
            return True
    return False


def test_planted_mistakes_fail():
    dec, runs, trace, tree = _setup()
    assert _swap_pops(trace, tree, runs, 1)
    with pytest.raises(replay.ParityError):
        replay.follow_heap(dec, trace, tree, [0, 1], [0, 1])

    dec, runs, trace, tree = _setup()
    trace["scores"][0, 3] += 0.05
    with pytest.raises(replay.ParityError, match="score"):
        replay.follow_heap(dec, trace, tree, [0, 1], [0, 1])

    dec, runs, trace, tree = _setup()
    ids = trace["cand_ids"][0, 0].copy()
    trace["cand_ids"][0, 0, -1] = next(v for v in range(dec.p.vocab) if v not in ids)   # a worse child
    with pytest.raises(replay.ParityError):
        replay.follow_heap(dec, trace, tree, [0, 1], [0, 1])

    dec, runs, trace, tree = _setup()
    st, ft = states_of(dec, runs)
    node = max(n for n in runs[0].expansions if n > 0)
    st[node, 0, :4] += 0.25
    with pytest.raises(replay.ParityError, match="state"):
        replay.follow_heap(dec, trace, tree, [0, 1], [0, 1], gpu_states=st, gpu_features=ft)

    # one state element moved to its neighbouring bf16 value far from a rounding midpoint
    dec, runs, trace, tree = _setup()
    st, ft = states_of(dec, runs)
    j = int(np.argmax(np.abs(st[node, 0])))
    dn, up = replay._bf16_neighbours(st[node, 0, j:j + 1])
    st[node, 0, j] = up[0]
    with pytest.raises(replay.ParityError, match="near-ties"):
        replay.follow_heap(dec, trace, tree, [0, 1], [0, 1], gpu_states=st, gpu_features=ft)

    # a feature element one step off
    dec, runs, trace, tree = _setup()
    st, ft = states_of(dec, runs)
    j = int(np.argmax(np.abs(ft[0, 1])))
    dn, up = replay._bf16_neighbours(ft[0, 1, j:j + 1])
    ft[0, 1, j] = dn[0]
    with pytest.raises(replay.ParityError, match="features"):
        replay.follow_heap(dec, trace, tree, [0, 1], [0, 1], gpu_states=st, gpu_features=ft)

    # a normaliser off by more than its fp32 bound (the child ranking is unchanged)
    dec, runs, trace, tree = _setup()
    st, ft = states_of(dec, runs)
    trace["lse"][0, 0] += 1e-3
    with pytest.raises(replay.ParityError, match="lse"):
        replay.follow_heap(dec, trace, tree, [0, 1], [0, 1], gpu_states=st, gpu_features=ft)

    dec, runs, trace, tree = _setup()
    trace["num_popped"][1] -= 1
    with pytest.raises(replay.ParityError):
        replay.follow_heap(dec, trace, tree, [0, 1], [0, 1])

    dec, runs, trace, tree = _setup()
    tree["mask"] = tree["mask"].copy()
    tree["mask"][0, 3, 0] ^= np.uint64(1)
    with pytest.raises(replay.ParityError, match="mask"):
        replay.follow_heap(dec, trace, tree, [0, 1], [0, 1])
