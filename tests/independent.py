"""Second, independent constructions used to pin the oracle on tiny inputs.

Nothing here calls the oracle's arithmetic: the correction head is evaluated
with scalar Python loops (``math``), bf16 rounding uses torch's conversion, and
the tree is built by algorithms the paper states separately from Alg. 1:

* ``heap_best_first``      - best-first max-heap over a materialised prefix tree
                              (Lemma 1 and its proof, Appendix C);
* ``sequential_heap``      - the sequential correction with a heap: pop the best prefix,
                              run the head on it, push its children (Sec. 3.1);
* ``brute_force``          - global top-B over every prefix of length <= L;
* ``marginal_top_b``       - DDTree's optimum for a zeroed correction: top-B
                              prefixes by factorised mass (Sec. 2.3, eq. (4));
* ``greedy_chain``         - the corrected single chain (W = 1);
* ``viterbi``              - Markov head: the best full-depth path by dynamic
                              programming over the previous token;
* ``canonical_arrays``     - the flattened tree and mask from a set of paths.
"""
from __future__ import annotations

import heapq
import math

import numpy as np
import torch

FP32, BF16 = 0, 1


def _widen(x, precision):
    if precision == BF16:
        t = torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16)
        return t.to(torch.float64).numpy()
    return np.asarray(x, np.float32).astype(np.float64)


def _bf16(v: float) -> float:
    return torch.tensor(v, dtype=torch.float64).to(torch.float32).to(torch.bfloat16).to(torch.float64).item()


class ScalarHead:
    """The correction head evaluated element by element.

    t_i = sum_k A[i][k] r[k];  a_i = rnd(tanh(t_i + H_d[i]));
    z_v = Lb_d[v] + sum_i U[v][i] a_i;  r'_i = rnd(tanh(t_i + e U[u][i])).
    """

    def __init__(self, inputs, cfg):
        self.cfg = cfg
        self.prec = cfg.precision
        self.A = _widen(inputs.A, self.prec).tolist()
        self.U = _widen(inputs.U, self.prec).tolist()
        self.H = _widen(inputs.H, self.prec).tolist()
        self.r0 = _widen(inputs.r0, self.prec).tolist()
        self.Lb = np.asarray(inputs.Lb, np.float32).astype(np.float64).tolist()
        self.h, self.V = cfg.hidden, cfg.vocab
        self.e = float(np.float32(math.sqrt(cfg.hidden)))
        self.tau = cfg.temperature if cfg.temperature > 0 else 1.0
        self.markov = getattr(cfg, "head", 0) == 1

    def _rnd(self, v):
        return _bf16(v) if self.prec == BF16 else v

    def step(self, b, d, r):
        """Parent state r at depth d-1 -> (t, z, logp) for depth d (1-based)."""
        h, V = self.h, self.V
        t = [math.fsum(self.A[i][k] * r[k] for k in range(h)) for i in range(h)]
        a = [self._rnd(math.tanh(t[i] + self.H[b][d - 1][i])) for i in range(h)]
        z = [self.Lb[b][d - 1][v] + math.fsum(self.U[v][i] * a[i] for i in range(h)) for v in range(V)]
        m = max(z)
        lse = math.log(math.fsum(math.exp((zv - m) / self.tau) for zv in z))
        logp = [(zv - m) / self.tau - lse for zv in z]
        return t, z, logp

    def child(self, t, v):
        """State of a child with token v: tanh(t + e U[v]), or with the Markov
        head e U[v] alone (the previous token's embedding), rounded."""
        if self.markov:
            return [self._rnd(self.e * self.U[v][i]) for i in range(self.h)]
        return [self._rnd(math.tanh(t[i] + self.e * self.U[v][i])) for i in range(self.h)]

    def step_over(self, b, d, r, cset):
        """As ``step`` with the head scoring only the tokens of ``cset`` and
        q~ normalised over them: returns (t, {v: z_v}, {v: log q~_v})."""
        h = self.h
        t = [math.fsum(self.A[i][k] * r[k] for k in range(h)) for i in range(h)]
        a = [self._rnd(math.tanh(t[i] + self.H[b][d - 1][i])) for i in range(h)]
        z = {v: self.Lb[b][d - 1][v] + math.fsum(self.U[v][i] * a[i] for i in range(h)) for v in cset}
        m = max(z.values())
        lse = math.log(math.fsum(math.exp((zv - m) / self.tau) for zv in z.values()))
        return t, z, {v: (zv - m) / self.tau - lse for v, zv in z.items()}

    def cset(self, b, d, K):
        """C_d = TopK(L_d^base, K) by a full sort of the drafter's base logits."""
        return _ranked(self.Lb[b][d - 1], K)


def _ranked(z, k):
    """Ids of the k best entries by (z desc, id asc), via a full sort."""
    return [v for _, v in sorted((-zv, v) for v, zv in enumerate(z))][:k]


def heap_best_first(levels, budget):
    """Best-first heap over a supertree: start from the depth-1 nodes, pop the best
    (score desc, depth asc, slot asc), push the popped node's children.

    ``levels[d-1]`` has ``token``, ``parent`` (slot at d-1) and ``score``.
    Returns the pop order as (depth, slot) pairs.
    """
    children = {}
    for d, lvl in enumerate(levels, start=1):
        for sl in range(len(lvl.score)):
            children.setdefault((d - 1, int(lvl.parent[sl]) if d > 1 else 0), []).append((d, sl))
    heap = [(-float(levels[0].score[sl]), 1, sl) for sl in range(len(levels[0].score))]
    heapq.heapify(heap)
    out = []
    while heap and len(out) < budget:
        negs, d, sl = heapq.heappop(heap)
        out.append((d, sl))
        for (cd, csl) in children.get((d, sl), []):
            heapq.heappush(heap, (-float(levels[cd - 1].score[csl]), cd, csl))
    return out


def sequential_heap(head: ScalarHead, b, budget, branch, beta):
    """Node-at-a-time construction: each pop runs the head on the popped prefix
    and pushes its top-k children (Sec. 3.1).  Returns {path: score}."""
    L = head.cfg.depth
    heap = []

    def expand(path, state, score):
        d = len(path) + 1
        t, z, logp = head.step(b, d, state)
        for v in _ranked(z, branch):
            s = (score + logp[v]) + beta
            heapq.heappush(heap, (-s, d, path + (v,), t))

    expand((), head.r0[b], 0.0)
    out = {}
    while heap and len(out) < budget:
        negs, d, path, t_parent = heapq.heappop(heap)
        out[path] = -negs
        if d < L:
            expand(path, head.child(t_parent, path[-1]), -negs)
    return out


def brute_force(head: ScalarHead, b, budget, beta):
    """Every prefix of length 1..L scored along its own path; global top-B by
    (score desc, depth asc, path asc).  Exponential: tiny V and L only."""
    L, V = head.cfg.depth, head.V
    scored = {}
    frontier = [((), head.r0[b], 0.0)]
    for d in range(1, L + 1):
        nxt = []
        for path, state, score in frontier:
            t, z, logp = head.step(b, d, state)
            for v in range(V):
                s = (score + logp[v]) + beta
                scored[path + (v,)] = s
                nxt.append((path + (v,), head.child(t, v), s))
        frontier = nxt
    best = sorted(scored, key=lambda p: (-scored[p], len(p), p))[:budget]
    return {p: scored[p] for p in best}


def brute_force_shared(head: ScalarHead, b, budget, beta, K):
    """Shared candidate sets: every prefix whose token at depth d lies in
    C_d = TopK(L_d^base, K), scored along its own path with q~ normalised over
    C_d; global top-B by (score desc, depth asc, path asc)."""
    L = head.cfg.depth
    scored = {}
    frontier = [((), head.r0[b], 0.0)]
    for d in range(1, L + 1):
        cset = head.cset(b, d, K)
        nxt = []
        for path, state, score in frontier:
            t, z, logp = head.step_over(b, d, state, cset)
            for v in cset:
                s = (score + logp[v]) + beta
                scored[path + (v,)] = s
                nxt.append((path + (v,), head.child(t, v), s))
        frontier = nxt
    best = sorted(scored, key=lambda p: (-scored[p], len(p), p))[:budget]
    return {p: scored[p] for p in best}


def sequential_heap_shared(head: ScalarHead, b, budget, branch, beta, K):
    """Node-at-a-time construction over shared candidate sets: each pop runs
    the head on the popped prefix over C_d and pushes its k best children."""
    L = head.cfg.depth
    heap = []

    def expand(path, state, score):
        d = len(path) + 1
        cset = head.cset(b, d, K)
        t, z, logp = head.step_over(b, d, state, cset)
        best = [v for _, v in sorted((-z[v], v) for v in cset)][:branch]
        for v in best:
            heapq.heappush(heap, (-((score + logp[v]) + beta), d, path + (v,), t))

    expand((), head.r0[b], 0.0)
    out = {}
    while heap and len(out) < budget:
        negs, d, path, t_parent = heapq.heappop(heap)
        out[path] = -negs
        if d < L:
            expand(path, head.child(t_parent, path[-1]), -negs)
    return out


def marginal_top_b(Lb, tau, L, budget, beta, K=None):
    """Zeroed correction: s(u) = sum_i log q_i(u_i) + beta*d with the drafter's
    marginals q_i = softmax(Lb_i / tau); top-B prefixes by brute force.  With
    K, tokens at position i range over TopK(Lb_i, K) and q_i is the softmax
    restricted to those K tokens (a shared candidate set)."""
    Lb = np.asarray(Lb, np.float64)
    V = Lb.shape[1]
    logq, allowed = [], []
    for d in range(L):
        ids = list(range(V)) if K is None else _ranked(Lb[d].tolist(), K)
        m = max(Lb[d][v] for v in ids)
        lse = math.log(math.fsum(math.exp((Lb[d][v] - m) / tau) for v in ids))
        logq.append({v: (Lb[d][v] - m) / tau - lse for v in ids})
        allowed.append(ids)
    scored = {}
    frontier = [((), 0.0)]
    for d in range(L):
        nxt = []
        for path, score in frontier:
            for v in allowed[d]:
                s = (score + logq[d][v]) + beta
                scored[path + (v,)] = s
                nxt.append((path + (v,), s))
        frontier = nxt
    best = sorted(scored, key=lambda p: (-scored[p], len(p), p))[:budget]
    return {p: scored[p] for p in best}, logq


def greedy_chain(head: ScalarHead, b, beta):
    """W = 1: follow the single best corrected token at every depth."""
    path, state, score, scores = (), head.r0[b], 0.0, []
    for d in range(1, head.cfg.depth + 1):
        t, z, logp = head.step(b, d, state)
        v = _ranked(z, 1)[0]
        score = (score + logp[v]) + beta
        path += (v,)
        scores.append(score)
        state = head.child(t, v)
    return path, scores


def viterbi(head: ScalarHead, b, beta):
    """Markov head: the best full-depth path by dynamic programming over the
    last token (its score is a sum of one-step transition log-probabilities,
    log q_d(v | u) of the head run on u's embedding).  Returns (score, path)."""
    L, V = head.cfg.depth, head.V
    _, _, lp = head.step(b, 1, head.r0[b])
    best = {v: ((0.0 + lp[v]) + beta, (v,)) for v in range(V)}
    for d in range(2, L + 1):
        nxt = {}
        for u, (su, pu) in best.items():
            _, _, lp = head.step(b, d, head.child(None, u))
            for v in range(V):
                s = (su + lp[v]) + beta
                if v not in nxt or s > nxt[v][0]:
                    nxt[v] = (s, pu + (v,))
        best = nxt
    return max(best.values())


def canonical_arrays(paths, budget):
    """Flatten a prefix-closed set of token paths: order by (depth, path), parent
    = index of the path without its last token, mask bit j of row i set iff
    node j's path is a prefix of node i's path (itself included)."""
    order = sorted(paths, key=lambda p: (len(p), p))
    index = {p: i for i, p in enumerate(order)}
    words = (budget + 63) // 64
    tokens = np.full(budget, -1, np.int64)
    parents = np.full(budget, -1, np.int64)
    depths = np.zeros(budget, np.int64)
    mask = np.zeros((budget, words), np.uint64)
    for i, p in enumerate(order):
        tokens[i] = p[-1]
        parents[i] = index[p[:-1]] if len(p) > 1 else -1
        depths[i] = len(p)
        for n in range(1, len(p) + 1):
            j = index[p[:n]]
            mask[i, j // 64] |= np.uint64(1) << np.uint64(j % 64)
    return tokens, parents, depths, mask, len(order)


def tree_paths(tokens, parents, num_nodes):
    """Token paths of an emitted tree (follows parent indices)."""
    paths = []
    for i in range(int(num_nodes)):
        path, j = [], i
        while j >= 0:
            path.append(int(tokens[j]))
            j = int(parents[j])
        paths.append(tuple(reversed(path)))
    return paths
