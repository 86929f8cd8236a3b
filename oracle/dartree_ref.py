"""Plain, slow CPU oracle of DARTree fixed-width draft-tree construction.

TEST INFRASTRUCTURE ONLY (see the package docstring): nothing on the product
path may import, call or link this module.

What it computes (paper: Sec. 3.2, Algorithm 1, Sec. 3.3, eq. (5) and
Lemma 1), for each request independently:

  root level S_0 = {empty prefix}, state r_0, score 0              (Alg. 1, init)
  for d = 1 .. L:                                                 (Alg. 1, depth loop)
      for every parent j of S_{d-1}:
          t_j = A r_j                                  (correction head, state part)
          a_j = rnd(tanh(t_j + H_d))                   (correction feature)
          z_j = L_d^base + U a_j                       (corrected logits, full vocab)
          l_j = log_softmax(z_j / tau)                 (log q~_d(. | u_<d), tau = T or 1)
          C_j = top-k ids of z_j by (z desc, id asc)   (per-parent candidate set)
      candidates (j, v in C_j), score s = (s_j + l_j[v]) + beta   (eq. (5), one step)
      S_d = first n_d candidates by (s desc, j asc, v asc)        (global top-W)
      r_child = rnd(tanh(t_j + e * U[v])), e = fp32(sqrt(h))      (state update)
  T = first min(B, |S|) nodes of S by (s desc, depth asc, slot asc)   (top-B, Lemma 1)

With a shared candidate set (``candidates`` = K > 0; Alg. 1 as printed, the
paper's default K = 64 of Sec. 4.1): C_d = TopK(L_d^base, K) by (value desc,
id asc) for each request and depth, the head scores only C_d
(z_j[v] = L_d^base[v] + U[v] a_j for v in C_d) and q~_d is normalised over
C_d, i.e. the tokens outside C_d take z = -inf; the rest is unchanged (the
per-parent cap k <= K, k = K keeping every token of C_d as in Alg. 1).
  emit T in canonical breadth-first order with parent indices and the
  ancestor-or-self tree-attention mask (Sec. 2.3).

Readings where the paper is silent:
  * the head form g and the state update (Alg. 1 gives only the signature
    g(H_d, r(u_<d)) and says that a child's state follows from its parent's
    state and its token): the Elman residual head above;
  * the candidate set is the per-parent top-k of the full-vocabulary corrected
    logits (the full-vocabulary variant of Appendix D) with branching cap k,
    or, with ``candidates`` = K, the shared C_d above with q~ normalised over
    C_d (Alg. 1 writes q~_d(C_d | u_<d) = g_{C_d}(...) without stating the
    normaliser; normalising over C_d keeps log q~ <= 0, which Lemma 1 needs);
  * tau = T for T > 0 and tau = 1 at T = 0 (q_T is defined for T > 0 only);
  * rounding points: with bf16 inputs, a and r are rounded to bf16 (through
    fp32, nearest-even) because they are operands of bf16 matrix products;
    everything else is fp64 here.  With fp32 inputs nothing is rounded;
  * n_d = min(W, n_{d-1} * k); the top-W that Alg. 1 calls global is taken
    per request;
  * tie-breaks: top-k (z desc, id asc); top-W (s desc, parent slot asc, id asc);
    top-B (s desc, depth asc, slot asc) - depth ascending is Lemma 1's tie
    rule, under which a prefix wins a tie with its extensions;
  * the root is not a node of T and does not count toward B.

The node-at-a-time baseline DARTree replaces (Sec. 3.1, the sequential
correction with a heap of Table 2) is ``sequential_heap``: a max-heap over candidate prefixes;
the head is run on the root and its k best children are pushed; each pop adds
the best prefix to the tree, runs the head on it under its own token history
(state from its parent's t and its token) and pushes its k best children,
until B prefixes have been popped.  Pop order: (s desc, depth asc, parent node
asc, child rank asc) - depth asc again prefers ancestors, the last two fields
make the order total.  The popped prefixes are emitted like DARTree's tree.

With the Markov correction head (``head`` = MARKOV; the DSpark-Markov head of
Sec. 2.2 and Table 3, which models the one-step transition y_{d-1} -> y_d) the
state of a prefix is the embedding of its last token only,
r(u_1:d) = rnd(e * U[u_d]) (r_0: the embedding of the last verified token);
t, a, z and everything after them are unchanged, so the children's
distribution depends on the path through its last token and depth alone.

The consumer of the emitted tree (Sec. 2.1, Sec. 2.3, Sec. 4.1):
  * ``acceptance_walk``: verification accepts, from the root, the child whose
    token equals the target's token at the current position (its greedy
    prediction at T = 0, its sample at T = 1: exact target-sample matching),
    and at the first position with no such child emits the target's token as
    the bonus; tau = accepted + 1 tokens advance per round;
  * ``tree_attention``: one attention layer over the flattened tree - node
    i's query attends to every position of the verified context and to the
    tree nodes j whose bit is set in mask row i (its root-to-node path).

Parity status: every function here is pinned by the CPU tests (brute force,
Lemma 1's heap, the sequential-heap algorithm of Sec. 3.1, special cases and
library routines).  The head form itself is this oracle's reading of a passage
the paper leaves open; its arithmetic is pinned by scalar-loop evaluation only.
"""
from __future__ import annotations

import dataclasses
import heapq
from typing import Callable, Optional

import numpy as np

FP32 = 0
BF16 = 1

RNN = 0      # Elman residual head: the state summarises the whole prefix
MARKOV = 1   # the state is the last token's embedding (a first-order transition)


# ----------------------------------------------------------------------------
# Parameters and decoded inputs
# ----------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class Params:
    """Alg. 1 inputs that are not tensors: depth L (= gamma), width W, branching
    cap k, budget B, temperature T and depth bonus beta (<= 0, Lemma 1)."""

    batch: int
    vocab: int
    hidden: int
    depth: int
    width: int
    branch: int
    budget: int
    temperature: float
    depth_bonus: float
    precision: int
    candidates: int = 0   # K of a shared C_d = TopK(L_d^base, K); 0 = the full vocabulary
    head: int = RNN       # RNN or MARKOV correction head

    @staticmethod
    def of(cfg) -> "Params":
        return Params(cfg.batch, cfg.vocab, cfg.hidden, cfg.depth, cfg.width,
                      cfg.branch, cfg.budget, float(cfg.temperature),
                      float(cfg.depth_bonus), int(cfg.precision), int(getattr(cfg, "candidates", 0)),
                      int(getattr(cfg, "head", RNN)))

    @property
    def tau(self) -> float:
        return self.temperature if self.temperature > 0 else 1.0

    @property
    def embed_scale(self) -> float:
        """e = fp32(sqrt(h)), the scale of the token input of the state update."""
        return float(np.float32(np.sqrt(np.float64(self.hidden))))

    def level_sizes(self) -> list[int]:
        n, out = 1, []
        for _ in range(self.depth):
            n = min(self.width, n * min(self.branch, self.vocab))
            out.append(n)
        return out


def _decode(x: np.ndarray, precision: int) -> np.ndarray:
    """Input values as fp64: bf16 bit patterns are widened exactly."""
    if precision == BF16:
        return (np.asarray(x, np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    return np.asarray(x, np.float32).astype(np.float64)


@dataclasses.dataclass
class Decoded:
    p: Params
    Lb: np.ndarray  # [b][L][V]
    H: np.ndarray   # [b][L][h]
    r0: np.ndarray  # [b][h]
    A: np.ndarray   # [h][h]
    U: np.ndarray   # [V][h]


def prepare(inputs, params: Optional[Params] = None) -> Decoded:
    """Decode one round's inputs (any object with Lb, H, r0, A, U and cfg)."""
    p = params if params is not None else Params.of(inputs.cfg)
    return Decoded(p, np.asarray(inputs.Lb, np.float32).astype(np.float64),
                   _decode(inputs.H, p.precision), _decode(inputs.r0, p.precision),
                   _decode(inputs.A, p.precision), _decode(inputs.U, p.precision))


def rnd_bf16(x: np.ndarray) -> np.ndarray:
    """fp64 -> fp32 (nearest-even) -> bf16 (nearest-even), returned as fp64."""
    u = np.asarray(x, np.float64).astype(np.float32).view(np.uint32)
    u = (u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))) & np.uint32(0xFFFF0000)
    return u.view(np.float32).astype(np.float64)


def _rounder(precision: int) -> Callable[[np.ndarray], np.ndarray]:
    return rnd_bf16 if precision == BF16 else (lambda x: x)


# ----------------------------------------------------------------------------
# One depth (Alg. 1, loop body)
# ----------------------------------------------------------------------------

def head_preimage(r: np.ndarray, A: np.ndarray, H_d: np.ndarray):
    """Correction head before the feature is rounded: t_j = A r_j and
    tanh(t_j + H_d), both [R][h] for ``r`` [R][h]."""
    t = r @ A.T
    return t, np.tanh(t + H_d[None, :])


def head_features(r: np.ndarray, A: np.ndarray, H_d: np.ndarray, precision: int):
    """Correction head, state part: t_j = A r_j and a_j = rnd(tanh(t_j + H_d)).

    ``r`` is [R][h] (one parent state per row); returns (t, a), both [R][h].
    """
    t, pre = head_preimage(r, A, H_d)
    return t, _rounder(precision)(pre)


def vocab_logits(a: np.ndarray, U: np.ndarray, Lb_d: np.ndarray, chunk: int = 16384) -> np.ndarray:
    """Corrected logits over the whole vocabulary: z_j = L_d^base + U a_j ([R][V])."""
    R, V = a.shape[0], U.shape[0]
    z = np.empty((R, V), np.float64)
    for c in range(0, V, chunk):
        z[:, c:c + chunk] = Lb_d[None, c:c + chunk] + a @ U[c:c + chunk].T
    return z


def candidate_set(Lb_d: np.ndarray, K: int) -> np.ndarray:
    """C_d = TopK(L_d^base, K) (Alg. 1): the K ids of the drafter's base logits
    at position d, ordered by (value desc, id asc)."""
    return topk_ids(Lb_d, K)


def candidate_logits(a: np.ndarray, U: np.ndarray, Lb_d: np.ndarray, cset: np.ndarray) -> np.ndarray:
    """Corrected logits on a shared candidate set (Alg. 1, g over C_d):
    z_j[v] = L_d^base[v] + U[v] a_j for v in C_d and -inf elsewhere ([R][V]),
    so that a softmax over the row is normalised over C_d."""
    z = np.full((a.shape[0], U.shape[0]), -np.inf)
    z[:, cset] = Lb_d[None, cset] + a @ U[cset].T
    return z


def log_softmax(z: np.ndarray, tau: float) -> np.ndarray:
    """log q_T: (z - m)/tau - log sum_v exp((z_v - m)/tau), row-wise."""
    m = z.max(axis=-1, keepdims=True)
    y = (z - m) / tau
    return y - np.log(np.exp(y).sum(axis=-1, keepdims=True))


def topk_ids(z_row: np.ndarray, k: int) -> np.ndarray:
    """The first k ids of one row ordered by (z desc, id asc)."""
    V = z_row.shape[0]
    k = min(k, V)
    kth = np.partition(z_row, V - k)[V - k]          # k-th largest value
    cand = np.nonzero(z_row >= kth)[0]               # contains every id of the top-k
    order = np.lexsort((cand, -z_row[cand]))
    return cand[order[:k]]


def select_level(parent: np.ndarray, token: np.ndarray, score: np.ndarray, n_keep: int) -> np.ndarray:
    """Indices of the first n_keep candidates by (score desc, parent asc, token asc)."""
    order = np.lexsort((token, parent, -score))
    return order[:n_keep]


def path_score(s_parent: np.ndarray, logp: np.ndarray, beta: float) -> np.ndarray:
    """Eq. (5) one depth at a time: s(u_1:d) = (s(u_<d) + log q~_d(u_d)) + beta."""
    return (s_parent + logp) + beta


def child_states(t_parent: np.ndarray, U_tok: np.ndarray, e: float, precision: int) -> np.ndarray:
    """State update r(u_1:d) = rnd(tanh(t(u_<d) + e * U[u_d])) for kept children."""
    return _rounder(precision)(np.tanh(t_parent + e * U_tok))


def markov_states(U_tok: np.ndarray, e: float, precision: int) -> np.ndarray:
    """Markov head: the state of u_1:d is its last token's embedding rnd(e * U[u_d])."""
    return _rounder(precision)(e * U_tok)


def state_preimage(p: Params, t_parent: np.ndarray, U_tok: np.ndarray) -> np.ndarray:
    """The kept children's states before they are rounded: tanh(t + e U[u_d])
    (recurrent head) or e U[u_d] (Markov head)."""
    e = p.embed_scale
    return e * U_tok if p.head == MARKOV else np.tanh(t_parent + e * U_tok)


def next_states(p: Params, t_parent: np.ndarray, U_tok: np.ndarray) -> np.ndarray:
    """The state of each kept child under the configured head."""
    if p.head == MARKOV:
        return markov_states(U_tok, p.embed_scale, p.precision)
    return child_states(t_parent, U_tok, p.embed_scale, p.precision)


# ----------------------------------------------------------------------------
# Whole construction
# ----------------------------------------------------------------------------

@dataclasses.dataclass
class Level:
    """S_d of one request: n_d nodes in slot order."""

    token: np.ndarray    # int64 [n_d]
    parent: np.ndarray   # int64 [n_d], slot in S_{d-1} (0 = the root at d = 1)
    score: np.ndarray    # fp64 [n_d], s_beta(u_1:d)
    # per-parent rows of this depth (for comparison with a second implementation)
    lse: Optional[np.ndarray] = None        # [n_{d-1}] log sum_v exp(z_v / tau)
    cand_ids: Optional[np.ndarray] = None   # [n_{d-1}][k] top-k ids of each parent
    cand_logp: Optional[np.ndarray] = None  # [n_{d-1}][k] their log q~
    logp: Optional[np.ndarray] = None       # [n_{d-1}][V] full log q~ (kept on demand)
    cset: Optional[np.ndarray] = None       # [K] shared candidate set C_d (candidates > 0)


@dataclasses.dataclass
class Supertree:
    p: Params
    levels: list  # levels[i][d-1] = Level of request i at depth d


Chooser = Callable[..., np.ndarray]


def _default_choose(req: int, d: int, parent, token, score, n_keep: int, level_rows) -> np.ndarray:
    return select_level(parent, token, score, n_keep)


def build_supertree(dec: Decoded, requests=None, choose: Optional[Chooser] = None,
                    choose_topk: Optional[Callable] = None, keep_logp: bool = False,
                    adopt_states: Optional[Callable] = None,
                    adopt_features: Optional[Callable] = None) -> Supertree:
    """Alg. 1's depth loop for every request (slow: full fp64 vocabulary products).

    ``choose`` / ``choose_topk`` let a caller replace the two selections (used
    to follow another implementation's choices); by default the oracle makes
    its own.  ``choose_topk(req, d, j, z_row, logp_row, k)`` returns the ids of
    parent j's candidate set.  ``adopt_states(req, d, r, pre)`` may replace the
    states of S_d computed here, and ``adopt_features(req, d, a, pre)`` the
    features a of depth d's parent rows (to follow another implementation's
    rounding); ``pre`` is the value before rounding (fp64).
    """
    p = dec.p
    choose = choose or _default_choose
    tau, e, beta = p.tau, p.embed_scale, p.depth_bonus
    k = min(p.branch, p.vocab)
    sizes = p.level_sizes()
    reqs = range(p.batch) if requests is None else requests
    out = []
    for b in reqs:
        r = dec.r0[b][None, :]            # states of S_0
        s = np.zeros(1)                   # scores of S_0
        levels = []
        for d in range(1, p.depth + 1):
            t, a = head_features(r, dec.A, dec.H[b, d - 1], p.precision)
            if adopt_features is not None:
                a = adopt_features(b, d, a, head_preimage(r, dec.A, dec.H[b, d - 1])[1])
            cset = None
            if p.candidates > 0:
                cset = candidate_set(dec.Lb[b, d - 1], p.candidates)
                z = candidate_logits(a, dec.U, dec.Lb[b, d - 1], cset)
            else:
                z = vocab_logits(a, dec.U, dec.Lb[b, d - 1])
            lp = log_softmax(z, tau)
            m = z.max(axis=1)
            lse = m / tau + np.log(np.exp((z - m[:, None]) / tau).sum(axis=1))
            R = z.shape[0]
            cids = np.empty((R, k), np.int64)
            for j in range(R):
                cids[j] = (choose_topk(b, d, j, z[j], lp[j], k) if choose_topk
                           else topk_ids(z[j], k))
            clp = np.take_along_axis(lp, cids, axis=1)
            par = np.repeat(np.arange(R), k)
            tok = cids.reshape(-1)
            sc = path_score(s[par], clp.reshape(-1), beta)
            keep = choose(b, d, par, tok, sc, sizes[d - 1], None)
            lvl = Level(token=tok[keep], parent=par[keep], score=sc[keep], lse=lse,
                        cand_ids=cids, cand_logp=clp, logp=lp if keep_logp else None, cset=cset)
            levels.append(lvl)
            r = next_states(p, t[lvl.parent], dec.U[lvl.token])
            if adopt_states is not None and d < p.depth:
                r = adopt_states(b, d, r, state_preimage(p, t[lvl.parent], dec.U[lvl.token]))
            s = lvl.score
        out.append(levels)
    return Supertree(p, out)


def prune(levels: list, budget: int):
    """Global top-B over the supertree by (s desc, depth asc, slot asc).

    Returns the kept nodes as a list of (depth, slot) in that order.
    """
    depth = np.concatenate([np.full(len(l.token), d + 1) for d, l in enumerate(levels)])
    slot = np.concatenate([np.arange(len(l.token)) for l in levels])
    score = np.concatenate([l.score for l in levels])
    order = np.lexsort((slot, depth, -score))[:min(budget, len(score))]
    return [(int(depth[i]), int(slot[i])) for i in order]


@dataclasses.dataclass
class Tree:
    """Emitted verification trees of a batch (pad slots: -1 / -1 / 0 / -inf / 0)."""

    tokens: np.ndarray     # int32 [b][B]
    parents: np.ndarray    # int32 [b][B], output index of the parent, -1 under the root
    depths: np.ndarray     # int32 [b][B], 1..L
    scores: np.ndarray     # fp64 [b][B]
    mask: np.ndarray       # uint64 [b][B][ceil(B/64)], bit j of row i: j is an ancestor-or-self of i
    num_nodes: np.ndarray  # int32 [b]


def emit_tree(levels: list, kept, budget: int):
    """Flatten the kept nodes of one request in canonical breadth-first order.

    Order: depth asc, then the parent's output index asc, then token asc.
    The ancestor-or-self mask row of a node is its parent's row plus itself.
    """
    words = (budget + 63) // 64
    tokens = np.full(budget, -1, np.int32)
    parents = np.full(budget, -1, np.int32)
    depths = np.zeros(budget, np.int32)
    scores = np.full(budget, -np.inf)
    mask = np.zeros((budget, words), np.uint64)
    out_index = {}  # (depth, slot) -> output index
    kept_by_depth = {}
    for (d, sl) in kept:
        kept_by_depth.setdefault(d, []).append(sl)
    n = 0
    for d in sorted(kept_by_depth):
        lvl = levels[d - 1]
        rows = []
        for sl in kept_by_depth[d]:
            pidx = -1 if d == 1 else out_index[(d - 1, int(lvl.parent[sl]))]
            rows.append((pidx, int(lvl.token[sl]), sl))
        rows.sort()
        for pidx, tok, sl in rows:
            out_index[(d, sl)] = n
            tokens[n], parents[n], depths[n], scores[n] = tok, pidx, d, lvl.score[sl]
            if pidx >= 0:
                mask[n] = mask[pidx]
            mask[n, n // 64] |= np.uint64(1) << np.uint64(n % 64)
            n += 1
    return tokens, parents, depths, scores, mask, n


def build_tree(dec: Decoded, requests=None) -> tuple[Tree, Supertree]:
    """Alg. 1 end to end: supertree, top-B prune, emitted trees."""
    st = build_supertree(dec, requests)
    return emit_batch(st), st


def emit_batch(st: Supertree, kept_sets=None) -> Tree:
    B = st.p.budget
    outs = []
    for i, levels in enumerate(st.levels):
        kept = prune(levels, B) if kept_sets is None else kept_sets[i]
        outs.append(emit_tree(levels, kept, B))
    return Tree(tokens=np.stack([o[0] for o in outs]), parents=np.stack([o[1] for o in outs]),
                depths=np.stack([o[2] for o in outs]), scores=np.stack([o[3] for o in outs]),
                mask=np.stack([o[4] for o in outs]), num_nodes=np.array([o[5] for o in outs], np.int32))


# ----------------------------------------------------------------------------
# Sequential correction with a best-first heap (Sec. 3.1; Table 2's baseline)
# ----------------------------------------------------------------------------

@dataclasses.dataclass
class Expansion:
    """The head's output on one expanded node (its children's distribution)."""

    lse: float                 # log sum_v exp(z_v / tau) of the node's row
    cand_ids: np.ndarray       # [k] its k best children, (z desc, id asc)
    cand_logp: np.ndarray      # [k] their log q~
    cset: Optional[np.ndarray] = None   # C_d scored for it (candidates > 0)


@dataclasses.dataclass
class HeapRun:
    """One request's node-at-a-time construction.  Node 0 is the root, node
    i >= 1 the i-th popped prefix."""

    token: list       # token of node i (-1 for the root)
    parent: list      # node index of its parent (-1 for the root)
    depth: list       # 0 for the root
    score: list       # s_beta(u) (0 for the root)
    expansions: dict  # node index -> Expansion, for every node the head ran on


def heap_entry(score: float, depth: int, parent: int, rank: int, token: int) -> tuple:
    """Ordering key of a candidate prefix in the heap; the smallest key is
    popped first: (s desc, depth asc, parent node asc, child rank asc)."""
    return (-score, depth, parent, rank, token)


def sequential_heap(dec: Decoded, requests=None, choose_topk: Optional[Callable] = None,
                    choose_pop: Optional[Callable] = None,
                    adopt_states: Optional[Callable] = None,
                    adopt_features: Optional[Callable] = None) -> list:
    """Sec. 3.1's exact best-first construction with the correction head run
    once per popped prefix (B pops per request).

    ``choose_topk(req, node, d, z_row, logp_row, k)`` may replace a node's
    k best children, ``choose_pop(req, step, heap)`` the index of the heap
    item popped at a step (items are (key, (score, depth, parent, token))),
    ``adopt_states(req, node, r, pre)`` a popped node's state and
    ``adopt_features(req, node, a, pre)`` the feature row the head computed on
    it (to follow another implementation's choices and rounding; ``pre`` is
    the value before rounding).
    """
    p = dec.p
    tau, e, beta = p.tau, p.embed_scale, p.depth_bonus
    k = min(p.branch, p.vocab)
    reqs = range(p.batch) if requests is None else requests
    runs = []
    for b in reqs:
        run = HeapRun(token=[-1], parent=[-1], depth=[0], score=[0.0], expansions={})
        t_of = {}
        heap: list = []

        def expand(n: int, r: np.ndarray):
            d = run.depth[n] + 1
            t, a = head_features(r[None, :], dec.A, dec.H[b, d - 1], p.precision)
            if adopt_features is not None:
                a = adopt_features(b, n, a, head_preimage(r[None, :], dec.A, dec.H[b, d - 1])[1])
            t_of[n] = t[0]
            cset = None
            if p.candidates > 0:
                cset = candidate_set(dec.Lb[b, d - 1], p.candidates)
                z = candidate_logits(a, dec.U, dec.Lb[b, d - 1], cset)[0]
            else:
                z = vocab_logits(a, dec.U, dec.Lb[b, d - 1])[0]
            lp = log_softmax(z[None, :], tau)[0]
            m = z.max()
            lse = m / tau + np.log(np.exp((z - m) / tau).sum())
            ids = (np.asarray(choose_topk(b, n, d, z, lp, k), np.int64) if choose_topk
                   else topk_ids(z, k))
            run.expansions[n] = Expansion(lse=float(lse), cand_ids=ids, cand_logp=lp[ids], cset=cset)
            for rank, v in enumerate(ids):
                sc = float(path_score(run.score[n], lp[v], beta))
                heapq.heappush(heap, (heap_entry(sc, d, n, rank, int(v)), (sc, d, n, int(v))))

        expand(0, dec.r0[b])
        while heap and len(run.token) - 1 < p.budget:
            step = len(run.token) - 1
            i = choose_pop(b, step, heap) if choose_pop else 0
            entry = heap[i]
            heap[i] = heap[-1]
            heap.pop()
            heapq.heapify(heap)
            sc, d, par, v = entry[1]
            n = len(run.token)
            run.token.append(v)
            run.parent.append(par)
            run.depth.append(d)
            run.score.append(sc)
            if d < p.depth and len(run.token) - 1 < p.budget:   # the last pop's children are never popped
                r = next_states(p, t_of[par][None, :], dec.U[v][None, :])[0]
                if adopt_states is not None:
                    r = adopt_states(b, n, r, state_preimage(p, t_of[par][None, :], dec.U[v][None, :])[0])
                expand(n, r)
        runs.append(run)
    return runs


def heap_levels(run: HeapRun):
    """The popped prefixes as levels (depth by depth, in pop order) and the
    (depth, slot) list of every node, for ``emit_tree``."""
    slot_of, by_depth = {}, {}
    for n in range(1, len(run.token)):
        lst = by_depth.setdefault(run.depth[n], [])
        slot_of[n] = len(lst)
        lst.append(n)
    levels = []
    for d in range(1, max(by_depth, default=0) + 1):
        ns = by_depth[d]   # prefix-closed: every depth up to the deepest is present
        levels.append(Level(token=np.array([run.token[n] for n in ns], np.int64),
                            parent=np.array([slot_of[run.parent[n]] if d > 1 else 0 for n in ns], np.int64),
                            score=np.array([run.score[n] for n in ns], np.float64)))
    kept = [(run.depth[n], slot_of[n]) for n in range(1, len(run.token))]
    return levels, kept


def emit_heap(runs: list, budget: int) -> Tree:
    outs = [emit_tree(*heap_levels(run), budget) for run in runs]
    return Tree(tokens=np.stack([o[0] for o in outs]), parents=np.stack([o[1] for o in outs]),
                depths=np.stack([o[2] for o in outs]), scores=np.stack([o[3] for o in outs]),
                mask=np.stack([o[4] for o in outs]), num_nodes=np.array([o[5] for o in outs], np.int32))


def sequential_heap_tree(dec: Decoded, requests=None) -> tuple[Tree, list]:
    """Sec. 3.1's baseline end to end: B pops per request, emitted trees."""
    runs = sequential_heap(dec, requests)
    return emit_heap(runs, dec.p.budget), runs


# ----------------------------------------------------------------------------
# The consumer: verification of the emitted tree (Sec. 2.1, 2.3, 4.1)
# ----------------------------------------------------------------------------

def acceptance_walk(tokens: np.ndarray, parents: np.ndarray, num_nodes: int, target: np.ndarray):
    """The accepted path of one flattened tree and the bonus token.

    ``target[0]`` is the target's token after the verified context and
    ``target[i + 1]`` its token after node i's path.  From the root, move to
    the child whose token is the target's token at the current position;
    stop at the first position without one.  Returns (output indices of the
    accepted nodes in path order, bonus token).
    """
    cur, path = -1, []
    while True:
        want = int(target[cur + 1])
        child = [j for j in range(int(num_nodes)) if int(parents[j]) == cur and int(tokens[j]) == want]
        if not child:
            return path, want
        cur = child[0]
        path.append(cur)


def mask_bit(mask: np.ndarray, i: int, j: int) -> bool:
    """Bit (i, j) of a packed ancestor-or-self mask [B][ceil(B/64)] (u64)."""
    return bool((int(mask[i, j // 64]) >> (j % 64)) & 1)


def tree_attention(q: np.ndarray, k_ctx: np.ndarray, v_ctx: np.ndarray, k_tree: np.ndarray,
                   v_tree: np.ndarray, mask: np.ndarray, ctx_len: int, scale: float) -> np.ndarray:
    """One attention layer over a flattened tree, one request (Sec. 2.3).

    q [B][Hq][D]; k_ctx, v_ctx [n_ctx][Hkv][D] (the first ctx_len positions
    are the verified context); k_tree, v_tree [B][Hkv][D] (each node's own key
    and value); mask [B][ceil(B/64)] u64.  Query head h reads key/value head
    h // (Hq / Hkv).  Node i attends to context positions 0..ctx_len-1 and to
    the nodes j with mask bit (i, j) set:
        out[i][h] = sum_j softmax_j(scale q[i][h] . k_j) v_j      (fp64),
    and a row that sees nothing is zero.
    """
    B, Hq, D = q.shape
    G = Hq // k_ctx.shape[1]
    out = np.zeros((B, Hq, D))
    for i in range(B):
        nodes = [j for j in range(B) if mask_bit(mask, i, j)]
        for h in range(Hq):
            kv = h // G
            keys = np.concatenate([k_ctx[:ctx_len, kv], k_tree[nodes, kv]], axis=0)
            vals = np.concatenate([v_ctx[:ctx_len, kv], v_tree[nodes, kv]], axis=0)
            if len(keys) == 0:      # nothing visible (a pad row without context): zero
                continue
            s = scale * (keys @ q[i, h])
            w = np.exp(s - s.max())
            out[i, h] = (w / w.sum()) @ vals
    return out
