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

Recurrent state.  States are rounded to bf16 after every depth (they are
operands of bf16 products).  Two correct implementations that accumulate in
a different order round a few state elements to neighbouring bf16 values; a
1-ulp change in r moves every element of t = A r, which flips more roundings
at the next depth, so free-running states drift apart until they differ by
about one ulp per element (corrected logits then differ by ~1e-3 at
h = 4096-5120).  The strict check therefore follows the GPU's states too
(``gpu_states``): each depth is recomputed in fp64 from the GPU's parent
states, and the GPU's state update is checked element by element against the
oracle's (equal, or the neighbouring bf16 value).  Without ``gpu_states`` the
comparator runs free (used with a wider window as a whole-round check).
"""
from __future__ import annotations

import dataclasses

import numpy as np

import oracle.dartree_ref as R

EPS = 1e-3
SCORE_TOL = 2e-2
STATE_ABS_TOL = 1e-5   # fp32 error of t + e U[v] before the state is rounded


@dataclasses.dataclass
class Report:
    topk_events: int = 0
    topw_events: int = 0
    topb_events: int = 0
    pop_events: int = 0          # sequential heap: a pop other than the oracle's own best
    max_logp_err: float = 0.0
    max_lse_err: float = 0.0
    max_score_err: float = 0.0
    checked_rows: int = 0
    state_elems: int = 0
    state_mismatch: int = 0

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
    """Window for the free-running comparison of a bf16 round.

    Free-running states differ by up to one bf16 step (2^-7 relative) per
    element; a 1-step change of the feature a moves z_v by sum_i U_vi da_i,
    whose rms is at most sigma_U 2^-7 sqrt(h) (|a_i| <= 1, independent signs).
    Scores add one such difference per depth (plus the same order from the
    normaliser), so after L depths the rms is at most
    2 sqrt(L) sigma_U 2^-7 sqrt(h); sigma_U is taken from the weights."""
    if p.precision != R.BF16:
        return EPS
    return 2.0 * np.sqrt(p.depth) * 2.0 ** -7 * np.sqrt(p.hidden)


def _check_topk(ids, glp, glse, z_row, lp_row, kk, tau, what, eps, rep):
    """A node's k children chosen by the GPU against the oracle's row."""
    if len(set(ids.tolist())) != kk or ids.min() < 0 or ids.max() >= len(z_row):
        raise ParityError(f"{what}: malformed candidate ids {ids}")
    mine = set(ids.tolist())
    ref = R.topk_ids(z_row, min(kk + 1, len(z_row)))
    best_un = next((lp_row[v] for v in ref if v not in mine), -np.inf)
    _valid_choice(lp_row[ids], best_un, f"top-k {what}", eps)
    if mine != set(ref[:kk].tolist()):
        rep.topk_events += 1
    rep.max_logp_err = max(rep.max_logp_err, float(np.abs(glp - lp_row[ids]).max()))
    m = z_row.max()
    lse = m / tau + np.log(np.exp((z_row - m) / tau).sum())
    rep.max_lse_err = max(rep.max_lse_err, abs(float(glse) - lse))
    rep.checked_rows += 1


def _check_state(r, g, precision, what, rep):
    """The GPU's bf16 state against the oracle's: equal or one rounding step
    apart (fp32 mode: the fp32 noise alone)."""
    err = np.abs(r - g)
    if precision == R.BF16:
        diff = err > 0
        far = err > 2.0 ** -7 * np.maximum(np.abs(r), np.abs(g)) + STATE_ABS_TOL
    else:
        diff = err > 1e-6
        far = err > STATE_ABS_TOL
    if far.any():
        raise ParityError(f"{what}: {int(far.sum())} state elements differ by more than one rounding step")
    rep.state_elems += r.size
    rep.state_mismatch += int(diff.sum())


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
           eps: float = EPS, score_tol: float = SCORE_TOL, rep: Report | None = None) -> Report:
    """Check GPU results against the oracle.

    dec          oracle.prepare(...) of inputs holding the requests in ``requests``
                 (row i of dec is request requests[i])
    sup, tree    host copies of the GPU's exported supertree and emitted tree
    batch_index  position of each checked request in the GPU's batch
    gpu_states   {d: states of S_d as exported, [b * n_d][h]} for d = 1..L-1
                 (decoded with decode_states), or None to run free
    """
    rep = rep or Report()
    p = dec.p
    sizes = p.level_sizes()
    W, k = p.width, min(p.branch, p.vocab)

    followed = []
    for i, b in enumerate(requests):
        q = batch_index[i]

        def choose_topk(req, d, j, z_row, lp_row, kk, q=q):
            row = q * sizes[d - 2] + j if d > 1 else q  # parent row of this depth
            ids = sup["cand_ids"][d - 1, row, :kk].astype(np.int64)
            glp = sup["cand_logp"][d - 1, row, :kk].astype(np.float64)
            _check_topk(ids, glp, sup["lse"][d - 1, row], z_row, lp_row, kk, p.tau, f"depth {d} row {row}", eps, rep)
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

        def adopt(req, d, r, q=q):
            n = sizes[d - 1]
            g = gpu_states[d][q * n:(q + 1) * n]
            _check_state(r, g, p.precision, f"depth {d}", rep)
            return g

        st = R.build_supertree(dec, requests=[i], choose=choose, choose_topk=choose_topk,
                               adopt_states=adopt if gpu_states is not None else None)
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
                eps: float = EPS, score_tol: float = SCORE_TOL, rep: Report | None = None) -> Report:
    """The sequential heap (oracle.sequential_heap) along the GPU's choices.

    trace        host copy of dartree_export_heap (slot i = the i-th pop; step
                 i ran the head on slot i)
    gpu_states   decoded states [B+1][b][h] (slot order), or None to run free
    At every pop the GPU's prefix must be a candidate whose oracle score is
    within ``eps`` of the best candidate's (else a failure; a different
    choice within the window is a near-tie event the oracle adopts), and
    every expanded node's k children are checked like a top-k of the
    depth-wise construction.  The emitted tree must then equal the oracle's
    flattening of the followed pops bit for bit, scores within score_tol.
    """
    rep = rep or Report()
    p = dec.p
    for i, b in enumerate(requests):
        q = batch_index[i]
        n_gpu = int(trace["num_popped"][q])

        def choose_topk(req, node, d, z_row, lp_row, kk, q=q):
            ids = trace["cand_ids"][node, q, :kk].astype(np.int64)
            glp = trace["cand_logp"][node, q, :kk].astype(np.float64)
            _check_topk(ids, glp, trace["lse"][node, q], z_row, lp_row, kk, p.tau, f"slot {node}", eps, rep)
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

        def adopt(req, node, r, q=q):
            g = gpu_states[node, q]
            _check_state(r, g, p.precision, f"slot {node}", rep)
            return g

        run = R.sequential_heap(dec, requests=[i], choose_topk=choose_topk, choose_pop=choose_pop,
                                adopt_states=adopt if gpu_states is not None else None)[0]
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
