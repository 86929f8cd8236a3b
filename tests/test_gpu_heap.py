"""The sequential heap on the GPU (dartree_build_tree_heap) against the
oracle's node-at-a-time construction, by the heap replay comparator.

Small cases cover every branch of the step kernel (segment records merged,
rows written in place by the softmax pass, the softmax over a shared set, a
heap that runs dry, pops at depth L, more slots than one wavefront scans at
once) with the oracle on every request; full-size workloads run the launch
sequence the benchmark times on sampled requests."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle.dartree_ref as R
from paper_2608_13524_amd import dartree as D
from paper_2608_13524_amd import workloads as W
from tests import replay
from tests.gpu_util import device, say
from tests.test_gpu_parity import _log_report, small

pytestmark = pytest.mark.gpu


def run_heap(cfg, inputs, states=True):
    """dartree_build_tree_heap on cuda:0; returns (tree dict, trace dict)."""
    dev = device()
    p = D.Params.of(cfg)
    di = D.DeviceInputs.from_host(inputs, dev)
    ws = D.alloc_heap_workspace(p, dev)
    out = D.DeviceTree.alloc(cfg.batch, cfg.budget, dev)
    say(f"build_tree_heap {cfg.name} b={cfg.batch} V={cfg.vocab} h={cfg.hidden} L={cfg.depth} "
        f"k={cfg.branch} K={cfg.candidates} B={cfg.budget} T={cfg.temperature}")
    D.build_tree_heap(p, di, ws, out)
    tr = D.DeviceHeapTrace.alloc(p, states=states, device=dev)
    D.export_heap(p, ws, tr)
    torch.cuda.synchronize()
    return out.host(), tr.host()


SMALL = {
    "heap-bf16": small(),                                              # 3 segments per row: records merged
    "heap-T0.7": small(temperature=0.7, seed=60),
    "heap-beta0": small(depth_bonus=0.0, seed=61),
    "heap-k12": small(branch=12, budget=40, seed=62),                  # top-k bucket 16
    "heap-k20": small(branch=20, budget=40, seed=63),                  # top-k bucket 32
    "heap-wide-B": small(batch=2, branch=8, budget=300, depth=6, seed=64),   # > 64 slots per arg-min
    "heap-max-B": small(batch=2, vocab=1031, hidden=64, branch=8, depth=8, budget=1024, seed=77),   # the most pops
    "heap-dry": small(vocab=7, hidden=64, branch=2, depth=3, budget=40, seed=65),   # 14 prefixes exist
    "heap-depth1": small(depth=1, budget=6, seed=66),                  # every pop at depth L
    "heap-B1": small(budget=1, seed=67),
    "heap-k1": small(branch=1, budget=8, seed=68),                     # the chain
    "heap-fp32": small(precision=W.FP32, hidden=48, sigma_w=0.1, seed=69),
    "heap-fp32-in-place": small(precision=W.FP32, vocab=1024, hidden=64, sigma_w=0.1, seed=70),   # one segment
    "heap-shared": small(candidates=12, branch=12, budget=30, seed=71),
    "heap-shared-k<K": small(candidates=20, branch=5, seed=72),
    "heap-shared-T0.7": small(candidates=16, branch=16, temperature=0.7, seed=73),
    "heap-shared-K200": small(batch=2, candidates=200, branch=64, budget=100, hidden=128, seed=74),
    "heap-shared-fp32": small(precision=W.FP32, hidden=48, candidates=9, branch=9, sigma_w=0.1, seed=75),
    "heap-markov": small(head=1, seed=79),
    "heap-markov-shared": small(head=1, candidates=16, branch=8, budget=30, seed=81),
}


@pytest.mark.parametrize("name", list(SMALL))
def test_heap_small_parity(name):
    cfg = SMALL[name]
    inputs = W.make_inputs(cfg)
    tree, trace = run_heap(cfg, inputs)
    dec = R.prepare(inputs)
    reqs = list(range(cfg.batch))
    gs = replay.decode_states(trace["states"], cfg.precision)
    gf = replay.decode_states(trace["features"], cfg.precision)
    rep = replay.follow_heap(dec, trace, tree, reqs, reqs, gpu_states=gs, gpu_features=gf)
    _log_report(name, "heap-follow-states", rep)
    assert rep.max_lse_ratio <= 1 and rep.max_logp_ratio <= 1
    free = replay.follow_heap(dec, trace, tree, reqs, reqs)
    _log_report(name, "heap-free-running", free)
    if free.events == 0:   # then the GPU equals the free-running oracle outright
        want, _ = R.sequential_heap_tree(dec)
        assert np.array_equal(tree["tokens"], want.tokens) and np.array_equal(tree["mask"], want.mask)


def test_heap_zeroed_correction_is_ddtree():
    """U = 0 and k = V: the heap pops DDTree's optimum, the top-B prefixes by
    factorised marginal mass plus beta*d; checked by rescoring every emitted
    prefix from the marginals."""
    cfg = small(vocab=30, hidden=64, branch=30, budget=25, seed=76)
    inputs = W.make_inputs(cfg)
    inputs.U[:] = 0
    tree, trace = run_heap(cfg, inputs, states=False)
    Lb = inputs.Lb.astype(np.float64)
    for q in range(cfg.batch):
        want, _ = R.sequential_heap_tree(R.prepare(inputs), requests=[q])
        n = int(tree["num_nodes"][q])
        assert n == cfg.budget
        for name in ("tokens", "parents", "depths", "mask"):
            assert np.array_equal(tree[name][q], getattr(want, name)[0]), name
        for o in range(n):
            path, j = [], o
            while j >= 0:
                path.append(int(tree["tokens"][q, j]))
                j = int(tree["parents"][q, j])
            path.reverse()
            s = sum(R.log_softmax(Lb[q, i][None, :], 1.0)[0, v] + cfg.depth_bonus for i, v in enumerate(path))
            assert abs(s - tree["scores"][q, o]) < 1e-4


# Full-size workloads at their own budgets: the requests the oracle re-derives.
FULL = {"tiny": [0], "qwen3-4b": [0], "qwen3-4b-wide": [0], "qwen3-4b-shared": [0], "qwen3-8b-x4": [1],
        "qwen3-8b-shared-x4": [0, 3], "stress-x16": [5], "qwen3-4b-markov": [0]}


@pytest.mark.parametrize("name", list(FULL))
def test_heap_full_size_parity(name):
    reqs = FULL[name]
    cfg = W.CONFIGS[name]
    weights = W.make_weights(cfg)
    inputs = W.make_inputs(cfg, weights=weights)
    tree, trace = run_heap(cfg, inputs)
    for q in range(cfg.batch):
        n = int(tree["num_nodes"][q])
        assert n == min(cfg.budget, int(trace["num_popped"][q]))
        assert (tree["parents"][q, :n] < np.arange(n)).all()
        s = trace["scores"][q, 1:n + 1]
        assert (np.diff(s) <= 1e-6).all()           # pops in non-increasing score order
    sub = W.make_inputs(cfg, requests=reqs, weights=weights)
    states = trace["states"][:, reqs]
    feats = trace["features"][:, reqs]
    trace = {k: (v[:, reqs] if k in ("lse", "cand_logp", "cand_ids") else v[reqs])
             for k, v in trace.items() if k not in ("states", "features")}
    tree = {k: v[reqs] for k, v in tree.items()}
    del inputs
    dec = R.prepare(sub)
    idx = list(range(len(reqs)))
    # every differing state or feature element must be a proven rounding near-tie
    # (replay.check_rounded), and every normaliser and log-probability within its
    # fp32 bound; the comparator raises otherwise
    rep = replay.follow_heap(dec, trace, tree, idx, idx, gpu_states=replay.decode_states(states, cfg.precision),
                             gpu_features=replay.decode_states(feats, cfg.precision))
    _log_report(name, "heap-follow-states", rep)
    assert rep.max_lse_ratio <= 1 and rep.max_logp_ratio <= 1 and rep.max_tie_ratio <= 1
    assert rep.max_score_err < replay.SCORE_TOL


def test_heap_graph_replay_matches_eager():
    """One heap round captured in a HIP graph: every replay, with eager rounds
    on other inputs in between, gives the eager result bit for bit."""
    for cfg in (small(seed=77, batch=2, budget=24), small(seed=78, batch=2, candidates=16, branch=8)):
        inputs = W.make_inputs(cfg)
        other = W.make_inputs(cfg.replace(seed=cfg.seed + 100))
        dev = device()
        p = D.Params.of(cfg)
        di = D.DeviceInputs.from_host(inputs, dev)
        do = D.DeviceInputs.from_host(other, dev)
        ws = D.alloc_heap_workspace(p, dev)
        out = D.DeviceTree.alloc(cfg.batch, cfg.budget, dev)
        say(f"graph capture of build_tree_heap K={cfg.candidates}")
        D.build_tree_heap(p, di, ws, out)
        torch.cuda.synchronize()
        want = out.host()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            D.build_tree_heap(p, di, ws, out)
        for rep in range(3):
            D.build_tree_heap(p, do, ws, out)
            torch.cuda.synchronize()
            for f in dataclasses.fields(out):
                getattr(out, f.name).fill_(-7)
            g.replay()
            torch.cuda.synchronize()
            got = out.host()
            for k in want:
                assert np.array_equal(got[k], want[k]), (rep, k)
