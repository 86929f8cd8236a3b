"""Replay comparator: run the oracle along the GPU's choices and check them.

Exact parity is not well defined where two candidates' scores differ by less
than the arithmetic noise (fp32 accumulation on the GPU, fp64 in the oracle).
So, at every selection the GPU made (each parent's top-k, each depth's
top-W, the final top-B), the oracle recomputes the values in fp64 along the
GPU's tree and requires:

  every chosen item's oracle value >= the best unchosen item's value - EPS

(EPS = 1e-3, in log-probability units for top-k and score units otherwise).
A differing set within that window is a near-tie event: the oracle adopts
the GPU's set and continues.  A larger gap fails.  Afterwards the emitted
arrays (tokens, parents, depths, mask, node counts) must equal the oracle's
flattening of the followed supertree bit for bit, and every score must agree
within SCORE_TOL (2e-2 absolute).  With no near-tie events this is plain
equality with the free-running oracle.

Recurrent state and features.  States r and features a are rounded to bf16
(they are operands of bf16 products).  Two correct implementations that
accumulate t = A r in a different order round a few of them to neighbouring
bf16 values; a one-step change in r moves every element of t at the next
depth, so free-running states drift apart until they differ by about one
step per element.  The strict check therefore follows the GPU's states and
features (``gpu_states``, ``gpu_features``), and accepts a GPU element that
differs from the oracle's only at a rounding near-tie:

  * the GPU's value g is the oracle's rounded value r = rnd(x), or
  * g is the rounding of a value within delta of the oracle's unrounded
    fp64 value x (rnd(x - delta) <= g <= rnd(x + delta)), where delta bounds
    the GPU's fp32 error before rounding: x lies within delta of a bf16
    rounding midpoint (for |x| of the order of delta the window can span
    several bf16 steps).

delta (``Bounds.preimage``): the GPU computes y = tanh(t + c) in fp32 with
c = H_d[i] (feature) or e U[u][i] (state).  t_i = sum_j A_ij r_j is a sum of
h products, exact in fp32 for bf16 operands, accumulated in fp32 in some
order.  Its error is sum_k eps_k s_k over the partial sums s_k with
|eps_k| <= u = 2^-24; with |s_k| of the order of ||w||_2 (w_j = A_ij r_j,
random-walk partial sums) and independent roundings the error has rms below
u sqrt(h) ||w||_2, and ACC_LAMBDA = 16 of those bound it (the model assumes
one rounding per product; an MFMA rounds once per 16 products).  The
rounding of the sums t + c and e U adds u (|c| + |t + c|); tanh's slope is at
most min(1, 1 - x^2 + 2 Din); tanhf is within 4 ulp (2^-21 |x|).  Each such
element is a near-tie event (``state_ties``, ``feature_ties``); any other
difference fails.  In fp32 mode nothing is rounded and |g - x| <= delta is
required outright.

With the GPU's features adopted, the oracle's z differs from the GPU's only
by the GPU's fp32 accumulation, so the log-probabilities and normalisers are
asserted: |dz_v| <= ACC_LAMBDA u sqrt(h) ||a o U_v||_2 + u |z_v| (the bias
add; max over v bounded with ||a o U_v|| <= max|a| ||U_v||); |d lse| <=
max_v |dz_v| / tau (lse is 1-Lipschitz in the max norm) plus the fp32 error
of the normaliser: at most 2 ceil(n / 64) + 64 sequential additions and
rescalings of positive terms (n scored tokens over at least 64 lanes) and
the exponentials' argument and evaluation errors (2^-19 relative).  Without
``gpu_states`` the comparator runs free (a whole-round check with a wider
window; nothing is adopted and these bounds do not apply).
"""
from __future__ import annotations

import dataclasses

import numpy as np

import oracle.dartree_ref as R

EPS = 1e-3
SCORE_TOL = 2e-2
U32 = 2.0 ** -24        # unit roundoff of fp32
ACC_LAMBDA = 16.0       # multiple of the rms accumulation error taken as its bound
TANH_REL = 2.0 ** -21   # tanhf: 4 ulp


@dataclasses.dataclass
class Report:
    topk_events: int = 0
    topw_events: int = 0
    topb_events: int = 0
    pop_events: int = 0          # sequential heap: a pop other than the oracle's own best
    max_logp_err: float = 0.0
    max_lse_err: float = 0.0
    max_score_err: float = 0.0
    max_logp_ratio: float = 0.0  # largest error / its bound (asserted <= 1 when features are followed)
    max_lse_ratio: float = 0.0
    checked_rows: int = 0
    state_elems: int = 0
    state_ties: int = 0          # state elements on the other side of a bf16 rounding near-tie
    feature_elems: int = 0
    feature_ties: int = 0
    max_tie_ratio: float = 0.0   # largest |x - midpoint| / delta over the ties (<= 1)
    max_fp32_ratio: float = 0.0  # fp32 mode: largest |g - x| / delta (<= 1)

    @property
    def events(self) -> int:
        return self.topk_events + self.topw_events + self.topb_events + self.pop_events


class ParityError(AssertionError):
    pass


def _valid_choice(chosen_vals: np.ndarray, unchosen_best: float, what: str, eps: float = EPS):
    if chosen_vals.size and unchosen_best > -np.inf and chosen_vals.min() < unchosen_best - eps:
        raise ParityError(f"{what}: chosen value {chosen_vals.min():.6f} below unchosen "
                          f"{unchosen_best:.6f} by more than {eps}")


def decode_states(bits_or_f32: np.ndarray, precision: int) -> np.ndarray:
    # exported buffers may hold slots no kernel wrote (never compared): any bits
    with np.errstate(invalid="ignore", over="ignore"):
        if precision == R.BF16:
            return (np.asarray(bits_or_f32).view(np.uint16).astype(np.uint32) << np.uint32(16)).view(
                np.float32).astype(np.float64)
        return np.asarray(bits_or_f32, np.float32).astype(np.float64)


def free_running_tol(p) -> float:
    """Window for the free-running comparison of a bf16 round, in units of
    sigma_U (the caller multiplies by the weights' standard deviation).

    Free-running states differ by up to one bf16 step (2^-7 relative) per
    element; a 1-step change of the feature a moves z_v by sum_i U_vi da_i,
    whose rms is at most sigma_U 2^-7 sqrt(h) (|a_i| <= 1, independent signs).
    Scores add one such difference per depth (plus the same order from the
    normaliser), so after L depths the rms is at most
    2 sqrt(L) sigma_U 2^-7 sqrt(h)."""
    if p.precision != R.BF16:
        return EPS
    return 2.0 * np.sqrt(p.depth) * 2.0 ** -7 * np.sqrt(p.hidden)


class Bounds:
    """fp32 error bounds of the GPU's arithmetic for one decoded round."""

    def __init__(self, dec):
        self.p = dec.p
        self.h = dec.p.hidden
        self.A2 = dec.A * dec.A
        self.U = dec.U
        # ||U_v||_2 per token (the bound of ||a o U_v|| for |a_i| <= max|a|)
        self.unorm = np.sqrt(np.einsum("vh,vh->v", dec.U, dec.U))

    def acc(self, wnorm):
        """Bound of the fp32 accumulation error of h exact products with
        ||w||_2 = wnorm."""
        return ACC_LAMBDA * U32 * np.sqrt(self.h) * wnorm

    def row_norms(self, r):
        """||A_i o r_j||_2 for every parent row j ([R][h]) and output i."""
        return np.sqrt(np.maximum((r * r) @ self.A2.T, 0.0))

    def preimage(self, x, tnorm, t_plus_c, c, markov=False):
        """delta: bound of |y_gpu - x| for y = tanh(t + c) computed in fp32
        (Markov: y = fl(e U), only the product's rounding)."""
        if markov:
            return U32 * np.abs(x) + 1e-30
        din = self.acc(tnorm) + U32 * (np.abs(c) + np.abs(t_plus_c))
        slope = np.minimum(1.0, 1.0 - x * x + 2.0 * din)
        return slope * din + TANH_REL * np.abs(x) + 2.0 ** -40


def _bf16_neighbours(r):
    """The bf16 values just below and just above each bf16 value r (fp64)."""
    bits = (np.asarray(r, np.float64).astype(np.float32).view(np.uint32) >> np.uint32(16)).astype(np.int64)
    mag, neg = bits & 0x7FFF, (bits & 0x8000) != 0
    away = np.where(neg, 0x8000, 0) | (mag + 1)                       # one step away from zero
    toward = np.where(mag == 0, np.where(neg, 0x0001, 0x8001),         # through zero
                      np.where(neg, 0x8000, 0) | (mag - 1))
    up = np.where(neg, toward, away)
    dn = np.where(neg, away, toward)

    def val(b):
        return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    return val(dn), val(up)


def check_rounded(r, g, x, delta, precision, what):
    """The GPU's element g against the oracle's r = rnd(x) (x unrounded).

    bf16: g must be the rounding of some y with |y - x| <= delta, i.e.
    rnd(x - delta) <= g <= rnd(x + delta) (rounding is monotone).  Where the
    window holds no rounding midpoint that leaves g == r; a g != r is a
    near-tie (counted), its ratio the distance from x to the nearest y that
    rounds to g, over delta (for |x| of the order of delta the window can
    span several bf16 steps).  fp32 (no rounding): |g - x| <= delta.
    Returns (number of near-ties, max tie ratio, max fp32 ratio)."""
    r, g, x, delta = (np.asarray(v, np.float64) for v in (r, g, x, delta))
    delta = np.broadcast_to(delta, x.shape)
    if precision != R.BF16:
        ratio = np.abs(g - x) / delta
        if not (ratio <= 1.0).all():
            i = np.unravel_index(int(np.argmax(ratio)), ratio.shape)
            raise ParityError(f"{what}: fp32 element {i} differs by {abs(g[i] - x[i]):.3e} > bound {delta[i]:.3e}")
        return 0, 0.0, float(ratio.max(initial=0.0))
    diff = g != r
    if not diff.any():
        return 0, 0.0, 0.0
    rd, gd, xd, dd = r[diff], g[diff], x[diff], delta[diff]
    inside = (gd >= R.rnd_bf16(xd - dd)) & (gd <= R.rnd_bf16(xd + dd))
    dn, up = _bf16_neighbours(gd)
    # nearest value that rounds to g: the midpoint on x's side of g
    edge = np.where(gd > rd, 0.5 * (gd + dn), 0.5 * (gd + up))
    tie = np.abs(edge - xd) / dd
    if not inside.all():
        j = int(np.argmax(~inside))
        raise ParityError(f"{what}: {int((~inside).sum())} of {int(diff.sum())} differing elements are not rounding "
                          f"near-ties (e.g. GPU {gd[j]!r}, oracle {rd[j]!r}, unrounded {xd[j]!r}, "
                          f"delta {dd[j]:.3e})")
    return int(diff.sum()), float(np.minimum(tie, 1.0).max()), 0.0


def _record(rep, kind, n, res):
    ties, tie_ratio, fp32_ratio = res
    if kind == "state":
        rep.state_elems += n
        rep.state_ties += ties
    else:
        rep.feature_elems += n
        rep.feature_ties += ties
    rep.max_tie_ratio = max(rep.max_tie_ratio, tie_ratio)
    rep.max_fp32_ratio = max(rep.max_fp32_ratio, fp32_ratio)


def _check_topk(ids, glp, glse, z_row, lp_row, kk, tau, what, eps, rep, bounds=None, a_row=None, n_scored=None):
    """A node's k children chosen by the GPU against the oracle's row.  With
    ``a_row`` (the GPU's feature row, adopted) the log-probabilities and the
    normaliser are asserted against their fp32 bounds."""
    if len(set(ids.tolist())) != kk or ids.min() < 0 or ids.max() >= len(z_row):
        raise ParityError(f"{what}: malformed candidate ids {ids}")
    mine = set(ids.tolist())
    ref = R.topk_ids(z_row, min(kk + 1, len(z_row)))
    best_un = next((lp_row[v] for v in ref if v not in mine), -np.inf)
    _valid_choice(lp_row[ids], best_un, f"top-k {what}", eps)
    if mine != set(ref[:kk].tolist()):
        rep.topk_events += 1
    lp_err = np.abs(glp - lp_row[ids])
    rep.max_logp_err = max(rep.max_logp_err, float(lp_err.max()))
    fin = np.isfinite(z_row)
    m = z_row[fin].max()
    lse = m / tau + np.log(np.exp((z_row[fin] - m) / tau).sum())
    lse_err = abs(float(glse) - lse)
    rep.max_lse_err = max(rep.max_lse_err, lse_err)
    rep.checked_rows += 1
    if bounds is None or a_row is None:
        return
    scored = np.nonzero(fin)[0]
    zmax_err = bounds.acc(np.abs(a_row).max() * bounds.unorm[scored].max()) + U32 * np.abs(z_row[fin]).max()
    n = len(scored) if n_scored is None else n_scored
    sum_rel = (2 * -(-n // 64) + 64) * U32 + 2.0 ** -19
    log_s = lse - m / tau
    lse_bound = zmax_err / tau + sum_rel / (1 - sum_rel) + 4 * U32 * (abs(m / tau) + abs(log_s))
    U_ids = bounds.U[ids]
    z_err = bounds.acc(np.sqrt(((a_row[None, :] * U_ids) ** 2).sum(axis=1))) + U32 * np.abs(z_row[ids])
    lp_bound = z_err / tau + lse_bound + 8 * U32 * (np.abs(lp_row[ids]) + abs(lse))
    rep.max_lse_ratio = max(rep.max_lse_ratio, lse_err / lse_bound)
    rep.max_logp_ratio = max(rep.max_logp_ratio, float((lp_err / lp_bound).max()))
    if lse_err > lse_bound:
        raise ParityError(f"{what}: lse error {lse_err:.3e} above its fp32 bound {lse_bound:.3e}")
    if (lp_err > lp_bound).any():
        raise ParityError(f"{what}: log q~ error {lp_err.max():.3e} above its fp32 bound")


def _check_emitted(tree, q, b, want, n, score_tol, rep):
    tok, par, dep, sco, mask, nn = want
    for name, arr in (("tokens", tok), ("parents", par), ("depths", dep)):
        if not np.array_equal(tree[name][q], arr):
            raise ParityError(f"request {b}: {name} differ\nGPU    {tree[name][q][:n]}\noracle {arr[:n]}")
    if not np.array_equal(tree["mask"][q], mask):
        raise ParityError(f"request {b}: mask differs")
    if nn != n:
        raise ParityError(f"request {b}: num_nodes {n} vs {nn}")
    fin = np.isfinite(sco)
    if not np.array_equal(fin, np.isfinite(tree["scores"][q])):
        raise ParityError(f"request {b}: padding of scores differs")
    err = float(np.abs(tree["scores"][q][fin] - sco[fin]).max()) if fin.any() else 0.0
    rep.max_score_err = max(rep.max_score_err, err)
    if err > score_tol:
        raise ParityError(f"request {b}: emitted score error {err}")


def follow(dec, sup: dict, tree: dict, batch_index: list, requests: list, gpu_states: dict | None = None,
           gpu_features: dict | None = None, eps: float = EPS, score_tol: float = SCORE_TOL,
           rep: Report | None = None) -> Report:
    """Check GPU results against the oracle.

    dec           oracle.prepare(...) of inputs holding the requests in ``requests``
                  (row i of dec is request requests[i])
    sup, tree     host copies of the GPU's exported supertree and emitted tree
    batch_index   position of each checked request in the GPU's batch
    gpu_states    {d: states of S_d as exported, [b * n_d][h]} for d = 1..L-1
    gpu_features  {d: features of depth d's parent rows, [b * n_{d-1}][h]}
                  for d = 1..L (both decoded with decode_states), or both
                  None to run free
    """
    rep = rep or Report()
    p = dec.p
    sizes = p.level_sizes()
    W, k = p.width, min(p.branch, p.vocab)
    strict = gpu_states is not None
    if strict and gpu_features is None:
        raise ValueError("the strict comparison follows both the GPU's states and its features")
    bounds = Bounds(dec) if strict else None
    n_scored = p.candidates if p.candidates > 0 else p.vocab
    is_markov = p.head == R.MARKOV

    followed = []
    for i, b in enumerate(requests):
        q = batch_index[i]
        cur = {"par_states": dec.r0[i][None, :], "a": None, "t": None, "tnorm": None}

        def choose_topk(req, d, j, z_row, lp_row, kk, q=q):
            row = q * sizes[d - 2] + j if d > 1 else q  # parent row of this depth
            ids = sup["cand_ids"][d - 1, row, :kk].astype(np.int64)
            glp = sup["cand_logp"][d - 1, row, :kk].astype(np.float64)
            _check_topk(ids, glp, sup["lse"][d - 1, row], z_row, lp_row, kk, p.tau, f"depth {d} row {row}", eps, rep,
                        bounds, None if cur["a"] is None else cur["a"][j], n_scored)
            return ids

        def choose(req, d, par, tok, sc, n_keep, _unused, q=q):
            gtok = sup["tokens"][d - 1, q, :n_keep].astype(np.int64)
            gpar = sup["parents"][d - 1, q, :n_keep].astype(np.int64)
            index = {(int(a), int(t)): c for c, (a, t) in enumerate(zip(par, tok))}
            try:
                keep = np.array([index[(int(a), int(t))] for a, t in zip(gpar, gtok)], np.int64)
            except KeyError as e:
                raise ParityError(f"depth {d}: GPU kept a child that is not a candidate: {e}")
            if len(set(keep.tolist())) != n_keep:
                raise ParityError(f"depth {d}: duplicate children in the GPU level")
            un = np.ones(len(sc), bool)
            un[keep] = False
            _valid_choice(sc[keep], sc[un].max() if un.any() else -np.inf, f"top-W depth {d}", eps)
            if set(keep.tolist()) != set(R.select_level(par, tok, sc, n_keep).tolist()):
                rep.topw_events += 1
            gs = sup["scores"][d - 1, q, :n_keep].astype(np.float64)
            err = float(np.abs(gs - sc[keep]).max())
            rep.max_score_err = max(rep.max_score_err, err)
            if err > score_tol:
                raise ParityError(f"depth {d}: score error {err}")
            return keep

        def adopt_features(req, d, a, pre, q=q):
            n = sizes[d - 2] if d > 1 else 1
            g = gpu_features[d][q * n:(q + 1) * n]
            t = cur["par_states"] @ dec.A.T
            tnorm = bounds.row_norms(cur["par_states"])
            H = dec.H[req, d - 1][None, :]
            delta = bounds.preimage(pre, tnorm, t + H, H)
            _record(rep, "feature", a.size, check_rounded(a, g, pre, delta, p.precision, f"depth {d} features"))
            cur["a"], cur["t"], cur["tnorm"] = g, t, tnorm
            return g

        def adopt_states(req, d, r, pre, q=q):
            n = sizes[d - 1]
            g = gpu_states[d][q * n:(q + 1) * n]
            gpar = sup["parents"][d - 1, q, :n].astype(np.int64)
            gtok = sup["tokens"][d - 1, q, :n].astype(np.int64)
            c = p.embed_scale * dec.U[gtok]
            if is_markov:
                delta = bounds.preimage(pre, None, None, None, markov=True)
            else:
                delta = bounds.preimage(pre, cur["tnorm"][gpar], cur["t"][gpar] + c, c)
            _record(rep, "state", r.size, check_rounded(r, g, pre, delta, p.precision, f"depth {d} states"))
            cur["par_states"] = g
            return g

        st = R.build_supertree(dec, requests=[i], choose=choose, choose_topk=choose_topk,
                               adopt_states=adopt_states if strict else None,
                               adopt_features=adopt_features if strict else None)
        followed.append(st.levels[0])
        if p.candidates > 0:   # shared sets depend on the drafter logits only: bit-exact
            for d, lvl in enumerate(st.levels[0], start=1):
                if not np.array_equal(sup["csets"][q, d - 1].astype(np.int64), lvl.cset):
                    raise ParityError(f"request {b} depth {d}: shared candidate set differs")

        # top-B: the GPU's kept set, read back from its emitted tree
        levels = st.levels[0]
        n = int(tree["num_nodes"][q])
        slot_of = {}
        for d, lvl in enumerate(levels, start=1):
            for sl in range(len(lvl.token)):
                slot_of[(d, int(lvl.parent[sl]) if d > 1 else 0, int(lvl.token[sl]))] = sl
        out_slot = []
        kept = []
        for o in range(n):
            d = int(tree["depths"][q, o])
            po = int(tree["parents"][q, o])
            ps = 0 if po < 0 else out_slot[po][1]
            key = (d, ps, int(tree["tokens"][q, o]))
            if key not in slot_of or (po >= 0 and out_slot[po][0] != d - 1) or (po < 0 and d != 1):
                raise ParityError(f"emitted node {o} {key} is not in the supertree")
            out_slot.append((d, slot_of[key]))
            kept.append((d, slot_of[key]))
        if len(set(kept)) != n or n != min(p.budget, sum(sizes)):
            raise ParityError(f"emitted tree has {n} nodes / duplicates")
        all_nodes = [(d, sl) for d, lvl in enumerate(levels, start=1) for sl in range(len(lvl.token))]
        score = {(d, sl): levels[d - 1].score[sl] for d, sl in all_nodes}
        ks = set(kept)
        _valid_choice(np.array([score[x] for x in kept]),
                      max((score[x] for x in all_nodes if x not in ks), default=-np.inf), "top-B", eps)
        if ks != set(R.prune(levels, p.budget)):
            rep.topb_events += 1
        _check_emitted(tree, q, b, R.emit_tree(levels, kept, p.budget), n, score_tol, rep)
    return rep


def follow_heap(dec, trace: dict, tree: dict, batch_index: list, requests: list, gpu_states=None,
                gpu_features=None, eps: float = EPS, score_tol: float = SCORE_TOL,
                rep: Report | None = None) -> Report:
    """The sequential heap (oracle.sequential_heap) along the GPU's choices.

    trace         host copy of dartree_export_heap (slot i = the i-th pop; step
                  i ran the head on slot i)
    gpu_states    decoded states [B+1][b][h] (slot order) and
    gpu_features  decoded features [B][b][h] (step order), or both None to run free
    At every pop the GPU's prefix must be a candidate whose oracle score is
    within ``eps`` of the best candidate's (else a failure; a different
    choice within the window is a near-tie event the oracle adopts), and
    every expanded node's k children are checked like a top-k of the
    depth-wise construction.  States and features are checked and adopted as
    in ``follow``.  The emitted tree must then equal the oracle's flattening
    of the followed pops bit for bit, scores within score_tol.
    """
    rep = rep or Report()
    p = dec.p
    strict = gpu_states is not None
    if strict and gpu_features is None:
        raise ValueError("the strict comparison follows both the GPU's states and its features")
    bounds = Bounds(dec) if strict else None
    n_scored = p.candidates if p.candidates > 0 else p.vocab
    is_markov = p.head == R.MARKOV
    for i, b in enumerate(requests):
        q = batch_index[i]
        n_gpu = int(trace["num_popped"][q])
        state_of = {0: dec.r0[i]}          # adopted state of each expanded slot
        t_of, tnorm_of = {}, {}            # t = A r and ||A_i o r|| of each expanded slot
        a_of = {}

        def choose_topk(req, node, d, z_row, lp_row, kk, q=q):
            ids = trace["cand_ids"][node, q, :kk].astype(np.int64)
            glp = trace["cand_logp"][node, q, :kk].astype(np.float64)
            _check_topk(ids, glp, trace["lse"][node, q], z_row, lp_row, kk, p.tau, f"slot {node}", eps, rep,
                        bounds, a_of.get(node), n_scored)
            return ids

        def choose_pop(req, step, heap, q=q):
            slot = step + 1
            if slot > n_gpu:
                raise ParityError(f"request {b}: the GPU stopped after {n_gpu} pops with {len(heap)} candidates left")
            gp, gt = int(trace["parents"][q, slot]), int(trace["tokens"][q, slot])
            match = [j for j, (_, (sc, d, par, v)) in enumerate(heap) if par == gp and v == gt]
            if not match:
                raise ParityError(f"request {b} pop {slot}: (parent slot {gp}, token {gt}) is not a candidate")
            j = match[0]
            best = min(range(len(heap)), key=lambda x: heap[x][0])
            chosen, top = heap[j][1][0], heap[best][1][0]
            _valid_choice(np.array([chosen]), top, f"pop {slot}", eps)
            if j != best:
                rep.pop_events += 1
            if int(trace["depths"][q, slot]) != heap[j][1][1]:
                raise ParityError(f"request {b} pop {slot}: depth {trace['depths'][q, slot]} vs {heap[j][1][1]}")
            err = abs(float(trace["scores"][q, slot]) - chosen)
            rep.max_score_err = max(rep.max_score_err, err)
            if err > score_tol:
                raise ParityError(f"request {b} pop {slot}: score error {err}")
            return j

        def adopt_features(req, node, a, pre, q=q):
            d = int(trace["depths"][q, node]) + 1 if node > 0 else 1
            g = gpu_features[node, q][None, :]
            t = state_of[node][None, :] @ dec.A.T
            tnorm = bounds.row_norms(state_of[node][None, :])
            H = dec.H[req, d - 1][None, :]
            delta = bounds.preimage(pre, tnorm, t + H, H)
            _record(rep, "feature", a.size, check_rounded(a, g, pre, delta, p.precision, f"slot {node} features"))
            t_of[node], tnorm_of[node], a_of[node] = t[0], tnorm[0], g[0]
            return g

        def adopt_states(req, node, r, pre, q=q):
            g = gpu_states[node, q]
            par, tok = int(trace["parents"][q, node]), int(trace["tokens"][q, node])
            if is_markov:
                delta = bounds.preimage(pre, None, None, None, markov=True)
            else:
                c = p.embed_scale * dec.U[tok]
                delta = bounds.preimage(pre, tnorm_of[par], t_of[par] + c, c)
            _record(rep, "state", r.size, check_rounded(r, g, pre, delta, p.precision, f"slot {node} state"))
            state_of[node] = g
            return g

        run = R.sequential_heap(dec, requests=[i], choose_topk=choose_topk, choose_pop=choose_pop,
                                adopt_states=adopt_states if strict else None,
                                adopt_features=adopt_features if strict else None)[0]
        n = len(run.token) - 1
        if n != n_gpu:
            raise ParityError(f"request {b}: the GPU popped {n_gpu} prefixes, the oracle {n}")
        if p.candidates > 0:
            for d in {run.depth[x] + 1 for x in run.expansions}:
                if not np.array_equal(trace["csets"][q, d - 1].astype(np.int64),
                                      R.candidate_set(dec.Lb[i, d - 1], p.candidates)):
                    raise ParityError(f"request {b} depth {d}: shared candidate set differs")
        _check_emitted(tree, q, b, R.emit_tree(*R.heap_levels(run), p.budget), n, score_tol, rep)
    return rep
