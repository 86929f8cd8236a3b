"""The depth-wise replay comparator on the CPU: the oracle's own round, laid
out as the GPU's exports, passes with no events; planted mistakes fail; and
the rounding near-tie test accepts a flip only next to a bf16 midpoint."""
import numpy as np
import pytest

import oracle.dartree_ref as R
from paper_2608_13524_amd import workloads as W
from tests import replay
from tests.pins import tiny


def exports_of(dec):
    """What dartree_export_supertree / _states / _features would hold after a
    round equal to the oracle's: (sup, tree, states {d}, features {d})."""
    p = dec.p
    b, L, Wd, k = p.batch, p.depth, p.width, min(p.branch, p.vocab)
    sizes = p.level_sizes()
    states, feats = {}, {}

    def keep_f(req, d, a, pre):
        feats.setdefault(d, []).append(a)
        return a

    def keep_s(req, d, r, pre):
        states.setdefault(d, []).append(r)
        return r

    st = R.build_supertree(dec, adopt_states=keep_s, adopt_features=keep_f)
    tree = R.emit_batch(st)
    sup = dict(tokens=np.zeros((L, b, Wd), np.int32), parents=np.zeros((L, b, Wd), np.int32),
               scores=np.zeros((L, b, Wd), np.float32), lse=np.zeros((L, b * Wd), np.float32),
               cand_logp=np.zeros((L, b * Wd, k), np.float32), cand_ids=np.zeros((L, b * Wd, k), np.int32))
    if p.candidates > 0:
        sup["csets"] = np.zeros((b, L, p.candidates), np.int32)
    for q, levels in enumerate(st.levels):
        for d, lvl in enumerate(levels, start=1):
            n, npar = sizes[d - 1], (sizes[d - 2] if d > 1 else 1)
            sup["tokens"][d - 1, q, :n] = lvl.token
            sup["parents"][d - 1, q, :n] = lvl.parent
            sup["scores"][d - 1, q, :n] = lvl.score
            sup["lse"][d - 1, q * npar:(q + 1) * npar] = lvl.lse
            sup["cand_logp"][d - 1, q * npar:(q + 1) * npar] = lvl.cand_logp
            sup["cand_ids"][d - 1, q * npar:(q + 1) * npar] = lvl.cand_ids
            if p.candidates > 0:
                sup["csets"][q, d - 1] = lvl.cset
    tr = {"tokens": tree.tokens, "parents": tree.parents, "depths": tree.depths,
          "scores": tree.scores.astype(np.float32), "mask": tree.mask, "num_nodes": tree.num_nodes}
    return sup, tr, {d: np.concatenate(v) for d, v in states.items()}, {d: np.concatenate(v) for d, v in feats.items()}


def _setup(**kw):
    cfg = tiny(**{**dict(batch=2, vocab=11, hidden=64, depth=4, width=5, branch=3, budget=9, precision=W.BF16,
                         seed=81), **kw})
    dec = R.prepare(W.make_inputs(cfg))
    return (dec,) + exports_of(dec)


def _follow(dec, sup, tree, st, ft):
    return replay.follow(dec, sup, tree, [0, 1], [0, 1], gpu_states=st, gpu_features=ft)


@pytest.mark.parametrize("kw", [dict(), dict(candidates=6, branch=4), dict(precision=W.FP32, temperature=0.7),
                                dict(head=R.MARKOV), dict(budget=100)])
def test_oracle_round_passes(kw):
    dec, sup, tree, st, ft = _setup(**kw)
    rep = _follow(dec, sup, tree, st, ft)
    assert rep.events == 0 and rep.state_ties == 0 and rep.feature_ties == 0
    assert rep.state_elems > 0 and rep.feature_elems > 0
    assert rep.max_lse_ratio <= 1 and rep.max_logp_ratio <= 1 and rep.max_score_err < 1e-6
    free = replay.follow(dec, sup, tree, [0, 1], [0, 1])
    assert free.events == 0


def test_planted_mistakes_fail():
    dec, sup, tree, st, ft = _setup()
    with pytest.raises(ValueError):   # the strict mode needs both
        replay.follow(dec, sup, tree, [0, 1], [0, 1], gpu_states=st)

    # a state element on the other side of a rounding step, far from the midpoint
    # (a large element: its step is far wider than the fp32 window)
    st2 = {d: v.copy() for d, v in st.items()}
    j = int(np.argmax(np.abs(st2[2][3])))
    dn, up = replay._bf16_neighbours(st2[2][3, j:j + 1])
    st2[2][3, j] = up[0]
    with pytest.raises(replay.ParityError, match="near-ties"):
        _follow(dec, sup, tree, st2, ft)

    # a state element two steps off
    st2 = {d: v.copy() for d, v in st.items()}
    dn, up = replay._bf16_neighbours(st2[1][0, :1])
    dn2, _ = replay._bf16_neighbours(dn)
    st2[1][0, 0] = dn2[0]
    with pytest.raises(replay.ParityError, match="states"):
        _follow(dec, sup, tree, st2, ft)

    # a feature element one step off
    ft2 = {d: v.copy() for d, v in ft.items()}
    j = int(np.argmax(np.abs(ft2[3][1])))
    dn, up = replay._bf16_neighbours(ft2[3][1, j:j + 1])
    ft2[3][1, j] = dn[0]
    with pytest.raises(replay.ParityError, match="features"):
        _follow(dec, sup, tree, st, ft2)

    # truncation instead of nearest-even rounding on a fraction of the states
    st2 = {d: v.copy() for d, v in st.items()}
    x = st2[1]
    trunc = (x.astype(np.float32).view(np.uint32) & np.uint32(0xFFFF0000)).view(np.float32).astype(np.float64)
    st2[1] = trunc
    if not np.array_equal(trunc, x):
        with pytest.raises(replay.ParityError):
            _follow(dec, sup, tree, st2, ft)

    # a normaliser and a log-probability beyond their fp32 bounds
    sup2 = {k: v.copy() for k, v in sup.items()}
    sup2["lse"][2, 1] += 5e-4
    with pytest.raises(replay.ParityError, match="lse"):
        _follow(dec, sup2, tree, st, ft)
    sup2 = {k: v.copy() for k, v in sup.items()}
    sup2["cand_logp"][1, 0, 1] -= 5e-4
    with pytest.raises(replay.ParityError, match="log q~"):
        _follow(dec, sup2, tree, st, ft)


def test_rounded_near_tie():
    """check_rounded on hand-made values around the midpoint of two bf16 neighbours."""
    lo, hi = 1.0, 1.0 + 2.0 ** -7
    mid = 0.5 * (lo + hi)
    delta = np.array([1e-6])
    # x just below the midpoint rounds to lo; the GPU's hi is a near-tie
    x = np.array([mid - 5e-7])
    r = R.rnd_bf16(x)
    assert r[0] == lo
    assert replay.check_rounded(r, np.array([hi]), x, delta, R.BF16, "t")[0] == 1
    assert replay.check_rounded(r, np.array([lo]), x, delta, R.BF16, "t")[0] == 0
    # outside the window: fails
    x = np.array([mid - 3e-6])
    with pytest.raises(replay.ParityError):
        replay.check_rounded(R.rnd_bf16(x), np.array([hi]), x, delta, R.BF16, "t")
    # two steps away with a window far narrower than a step: fails
    with pytest.raises(replay.ParityError):
        replay.check_rounded(np.array([lo]), np.array([hi + 2.0 ** -7]), np.array([mid]), delta, R.BF16, "t")
    # a value near zero whose window spans several bf16 steps: any rounding inside it passes
    x = np.array([2.6e-7])
    r = R.rnd_bf16(x)
    g = R.rnd_bf16(np.array([2.6e-7 + 3e-8]))
    assert g[0] != r[0]
    assert replay.check_rounded(r, g, x, np.array([3.5e-5]), R.BF16, "t")[0] == 1
    with pytest.raises(replay.ParityError):
        replay.check_rounded(r, g, x, np.array([1e-8]), R.BF16, "t")
    # negative values and a binade edge (neighbours of -1: -1 - 2^-7 and -1 + 2^-8)
    dn, up = replay._bf16_neighbours(np.array([-1.0, 1.0, 0.0]))
    assert dn[0] == -1.0 - 2.0 ** -7 and up[0] == -1.0 + 2.0 ** -8
    assert dn[1] == 1.0 - 2.0 ** -8 and up[1] == 1.0 + 2.0 ** -7
    assert dn[2] < 0 < up[2]
    # fp32 mode: within delta of x
    assert replay.check_rounded(np.array([0.3]), np.array([0.3 + 5e-7]), np.array([0.3]), delta, R.FP32, "t")[2] <= 1
    with pytest.raises(replay.ParityError):
        replay.check_rounded(np.array([0.3]), np.array([0.3 + 5e-6]), np.array([0.3]), delta, R.FP32, "t")
