"""Each kernel of one depth on injected inputs, through the C ABI, against the
oracle's routines on the same values.

Selections (top-k, top-W, top-B and the emitted tree) are integer work on the
same fp32 values on both sides and must agree bit for bit, ties included.
Products and normalisers are checked against fp64 with error bounds."""
import numpy as np
import pytest
import torch

import oracle.dartree_ref as R
from paper_2608_13524_amd import dartree as D
from paper_2608_13524_amd import workloads as W
from tests.gpu_util import device, say, to_dev

pytestmark = pytest.mark.gpu


# ---------------------------------------------------------------------------
# log-softmax normaliser + per-row top-k
# ---------------------------------------------------------------------------

LSE_CASES = [
    # rows, vocab, k, T, distribution
    (1, 151936, 8, 0.0, "normal"),      # split over many segments + merge
    (8, 151936, 8, 1.0, "normal"),
    (64, 151936, 8, 0.7, "normal"),
    (1024, 4096, 8, 1.0, "normal"),     # one segment per row
    (3, 1001, 4, 0.7, "normal"),        # vocab not a multiple of 4: scalar path
    (5, 1024, 32, 1.0, "ties"),         # coarse values: many exact ties
    (7, 151936, 16, 0.0, "ties"),
    (2, 40, 1, 0.0, "ties"),
    (4, 9, 9, 2.0, "normal"),           # k = V
    # a segment held in registers where fewer than k threads hold values
    (3, 16, 8, 1.0, "ties"), (2, 28, 8, 0.0, "normal"),
    # 17..511 rows: segments of at most 8192 held in registers (13 ragged
    # segments with exact ties; one segment per row; k = 16; 300 rows)
    (24, 100000, 8, 1.0, "ties"), (40, 5000, 8, 0.7, "normal"), (17, 151936, 16, 0.0, "normal"),
    (300, 20004, 8, 1.0, "normal"),
]


@pytest.mark.parametrize("rows,vocab,k,T,dist", LSE_CASES)
def test_lse_topk(rows, vocab, k, T, dist):
    rng = np.random.default_rng(rows * 7919 + vocab + k)
    z = rng.normal(0, 2, size=(rows, vocab)).astype(np.float32)
    if dist == "ties":
        z = (np.round(z * 4) / 4).astype(np.float32)
    dev = device()
    zd = to_dev(z)
    lse = torch.empty(rows, dtype=torch.float32, device=dev)
    lp = torch.empty(rows, k, dtype=torch.float32, device=dev)
    ids = torch.empty(rows, k, dtype=torch.int32, device=dev)
    need = D.lse_topk_workspace_size(rows, vocab, k)
    ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    say(f"lse_topk rows={rows} vocab={vocab} k={k} T={T} {dist}")
    D.lse_topk(zd, k, T, lse, lp, ids, ws)
    torch.cuda.synchronize()
    lse, lp, ids = lse.cpu().numpy(), lp.cpu().numpy(), ids.cpu().numpy()
    tau = T if T > 0 else 1.0
    z64 = z.astype(np.float64)
    ref_lp = R.log_softmax(z64, tau)
    m = z64.max(axis=1)
    ref_lse = m / tau + np.log(np.exp((z64 - m[:, None]) / tau).sum(axis=1))
    for r in range(rows):
        want = R.topk_ids(z64[r], k)
        assert np.array_equal(ids[r], want), (r, ids[r], want)
    assert np.allclose(lse, ref_lse, rtol=2e-6, atol=2e-5)
    got = np.take_along_axis(ref_lp, ids.astype(np.int64), axis=1)
    assert np.abs(lp - got).max() < 2e-5
    assert (lp <= 0).all()


# ---------------------------------------------------------------------------
# corrected-logit products
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("rows,vocab,hidden,group", [
    (1, 4099, 2560, 1), (8, 4099, 2560, 8), (13, 5000, 512, 5), (16, 151936, 2560, 8),
    (33, 3001, 1024, 11), (64, 4099, 4096, 16), (100, 4099, 512, 25), (128, 4103, 1024, 64),
    (200, 3000, 256, 50),
    # 17..64 rows against a long vocabulary, K a multiple of 128: the sweep,
    # one wave per run of 16-row weight tiles (on 256 CUs 6, 8, 10, 13 and 16
    # tiles per wave); ragged last tile and last wave; 1 to 4 128-deep chunks
    # (a single chunk fills only its own stages); groups of 4, 6, 8, 10, 11,
    # 16 and 25 rows (bias rows with an odd stride: scalar epilogue)
    (20, 65600, 384, 4), (33, 70000, 256, 11), (64, 66000, 512, 16),
    (24, 65536, 256, 8), (18, 110000, 128, 6), (48, 100000, 128, 16), (40, 128300, 128, 8),
    (30, 90000, 256, 10), (50, 80000, 128, 25), (24, 170000, 128, 8),
    # 17..64 rows with K not a multiple of 128: the 128-row-block stream kernel
    (20, 65600, 320, 4), (40, 70000, 192, 8),
    (1, 151936, 64, 1),
    # <= 16 rows against a long vocabulary, K a multiple of 128: 128-deep
    # chunk pairs, 4 waves over K (some waves with no pairs; one pair)
    (5, 70001, 384, 5), (12, 100003, 1152, 4), (9, 65536, 128, 3),
    # >= 512 rows against >= 16384 columns: the 512x128-tile kernel where the
    # rows are a multiple of 512 (512, 1024, 2048), else the 256x256-tile one;
    # ragged in the vocabulary, and in the rows for the 256x256 tiles
    (512, 16400, 256, 64), (600, 16390, 128, 75), (1024, 20000, 512, 64),
    # one, three and five 64-deep K steps: every depth of the load pipelines'
    # prologues, an odd step count (the 512-row kernel runs steps in pairs)
    (512, 16384, 64, 64), (520, 16500, 192, 13), (2048, 16500, 320, 64),
    # a last partial wave of tiles split along K (on 256 CUs, 512-row tiles:
    # 58 tiles in 4 pieces of 4 steps, in 2 pieces of 5 steps; 256x256 tiles:
    # 69 tiles in 3 pieces, ragged in M and N)
    (1024, 20000, 1024, 64), (1024, 20000, 640, 32), (1030, 16400, 768, 103),
])
def test_project_bf16_within_error_bound(rows, vocab, hidden, group):
    check_project_bf16(rows, vocab, hidden, group, pad=3)


@pytest.mark.parametrize("rows,vocab,hidden,group", [(24, 100000, 256, 8), (40, 151936, 128, 20), (8, 151936, 256, 8)])
def test_project_bf16_aligned_bias(rows, vocab, hidden, group):
    """Bias rows with a stride of the vocabulary (16-byte aligned): the vector epilogues."""
    check_project_bf16(rows, vocab, hidden, group, pad=0)


def check_project_bf16(rows, vocab, hidden, group, pad):
    rng = np.random.default_rng(rows + vocab + hidden)
    x = W.fp32_to_bf16_bits(np.tanh(rng.normal(0, 1.4, size=(rows, hidden))).astype(np.float32))
    U = W.fp32_to_bf16_bits(rng.normal(0, 0.02, size=(vocab, hidden)).astype(np.float32))
    groups = (rows + group - 1) // group
    bias = rng.normal(0, 2, size=(groups, vocab + pad)).astype(np.float32)  # stride vocab + pad
    dev = device()
    z = torch.empty(rows, vocab, dtype=torch.float32, device=dev)
    nws = D.project_workspace_size(D.BF16, rows, vocab, hidden)
    ws = torch.empty(nws, dtype=torch.uint8, device=dev) if nws else None
    say(f"project bf16 rows={rows} vocab={vocab} hidden={hidden} group={group} ws={nws}")
    xd, Ud, bd = to_dev(x), to_dev(U), to_dev(bias)
    D.project(D.BF16, xd, Ud, bd, vocab + pad, z, group, ws)
    if ws is not None:  # deterministic: a second call (stale scratch) gives the same bits
        z2 = torch.empty_like(z)
        ws.fill_(0x7F)
        D.project(D.BF16, xd, Ud, bd, vocab + pad, z2, group, ws)
        torch.cuda.synchronize()
        assert torch.equal(z, z2)
    torch.cuda.synchronize()
    z = z.cpu().numpy().astype(np.float64)
    xf = W.bf16_bits_to_fp32(x).astype(np.float64)
    Uf = W.bf16_bits_to_fp32(U).astype(np.float64)
    g = np.arange(rows) // group
    ref = bias[g, :vocab].astype(np.float64) + xf @ Uf.T
    # fp32 accumulation of `hidden` exact products, then one fp32 add of the bias
    bound = 1.01 * hidden * 2.0 ** -24 * (np.abs(xf) @ np.abs(Uf).T) + 2.0 ** -23 * np.abs(ref)
    err = np.abs(z - ref)
    assert (err <= bound + 1e-7).all(), float((err - bound).max())


def test_project_fp32():
    rng = np.random.default_rng(5)
    rows, vocab, hidden = 7, 1030, 64
    x = rng.normal(0, 1, size=(rows, hidden)).astype(np.float32)
    U = rng.normal(0, 0.05, size=(vocab, hidden)).astype(np.float32)
    bias = rng.normal(0, 3, size=(1, vocab)).astype(np.float32)
    z = torch.empty(rows, vocab, dtype=torch.float32, device=device())
    say("project fp32")
    D.project(D.FP32, to_dev(x), to_dev(U), to_dev(bias), 0, z, rows)
    torch.cuda.synchronize()
    ref = bias.astype(np.float64) + x.astype(np.float64) @ U.astype(np.float64).T
    assert np.abs(z.cpu().numpy() - ref).max() < 1e-4


# ---------------------------------------------------------------------------
# segmented top-W
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("batch,n_parent,k,n_keep,beta,ties", [
    (1, 1, 8, 8, -0.2, False), (1, 8, 8, 8, -0.2, False), (3, 32, 8, 32, -0.2, True),
    (16, 64, 8, 64, 0.0, True), (2, 5, 3, 7, -1.0, True), (4, 512, 8, 100, -0.2, False),
    (1, 128, 32, 2048, -0.2, True),
])
def test_select_topw_bit_exact(batch, n_parent, k, n_keep, beta, ties):
    rng = np.random.default_rng(batch * 100 + n_parent + k)
    sp = rng.normal(-5, 2, size=(batch, n_parent)).astype(np.float32)
    lp = -np.abs(rng.normal(0, 3, size=(batch * n_parent, k))).astype(np.float32)
    if ties:
        sp = (np.round(sp * 2) / 2).astype(np.float32)
        lp = (np.round(lp * 2) / 2).astype(np.float32)
    ids = np.stack([rng.choice(151936, size=k, replace=False) for _ in range(batch * n_parent)]).astype(np.int32)
    dev = device()
    tok = torch.empty(batch, n_keep, dtype=torch.int32, device=dev)
    par = torch.empty(batch, n_keep, dtype=torch.int32, device=dev)
    sc = torch.empty(batch, n_keep, dtype=torch.float32, device=dev)
    say(f"select_topw batch={batch} n_parent={n_parent} k={k} n_keep={n_keep}")
    D.select_topw(batch, n_parent, k, n_keep, beta, to_dev(sp), to_dev(lp), to_dev(ids), tok, par, sc)
    torch.cuda.synchronize()
    tok, par, sc = tok.cpu().numpy(), par.cpu().numpy(), sc.cpu().numpy()
    for q in range(batch):
        parent = np.repeat(np.arange(n_parent), k)
        token = ids[q * n_parent:(q + 1) * n_parent].reshape(-1).astype(np.int64)
        # the same two fp32 additions as the kernel
        s32 = (sp[q][parent] + lp[q * n_parent:(q + 1) * n_parent].reshape(-1)) + np.float32(beta)
        keep = R.select_level(parent, token, s32.astype(np.float64), n_keep)
        assert np.array_equal(tok[q], token[keep])
        assert np.array_equal(par[q], parent[keep])
        assert np.array_equal(sc[q], s32[keep])


def test_select_topw_root_scores_null():
    dev = device()
    lp = np.array([[-0.1, -2.0, -0.5]], np.float32)
    ids = np.array([[5, 9, 2]], np.int32)
    tok = torch.empty(1, 3, dtype=torch.int32, device=dev)
    par = torch.empty(1, 3, dtype=torch.int32, device=dev)
    sc = torch.empty(1, 3, dtype=torch.float32, device=dev)
    say("select_topw root")
    D.select_topw(1, 1, 3, 3, -0.2, None, to_dev(lp), to_dev(ids), tok, par, sc)
    torch.cuda.synchronize()
    assert tok.cpu().tolist() == [[5, 2, 9]]
    assert par.cpu().tolist() == [[0, 0, 0]]
    assert np.array_equal(sc.cpu().numpy()[0], (lp[0][[0, 2, 1]] + np.float32(0)) + np.float32(-0.2))


# ---------------------------------------------------------------------------
# deferred top-B prune + emission
# ---------------------------------------------------------------------------

def _random_supertree(rng, batch, L, Wd, k, ties):
    sizes, n = [], 1
    for _ in range(L):
        n = min(Wd, n * k)
        sizes.append(n)
    tok = np.full((L, batch, Wd), -7, np.int32)
    par = np.full((L, batch, Wd), -7, np.int32)
    sco = np.full((L, batch, Wd), np.nan, np.float32)
    levels = []
    for q in range(batch):
        lv, prev = [], np.zeros(1, np.float32)
        for d in range(L):
            nd = sizes[d]
            pp = rng.integers(0, len(prev), size=nd) if d > 0 else np.zeros(nd, np.int64)
            # distinct tokens among siblings: draw without replacement per level
            tt = rng.choice(50000, size=nd, replace=False)
            drop = (np.round(rng.exponential(1.0, nd) * 2) / 2 if ties else rng.exponential(1.0, nd))
            s = (prev[pp] - drop.astype(np.float32)).astype(np.float32)
            tok[d, q, :nd], par[d, q, :nd], sco[d, q, :nd] = tt, pp, s
            lv.append(R.Level(token=tt.astype(np.int64), parent=pp.astype(np.int64), score=s.astype(np.float64)))
            prev = s
        levels.append(lv)
    return sizes, tok, par, sco, levels


@pytest.mark.parametrize("batch,L,Wd,k,B,ties", [
    (1, 4, 4, 4, 16, False), (1, 16, 8, 8, 64, True), (1, 16, 32, 8, 256, True),
    (4, 16, 16, 8, 128, False), (16, 16, 64, 8, 512, True), (2, 5, 3, 2, 100, False),
    (3, 6, 5, 3, 1, True), (1, 64, 64, 2, 4096, False), (2, 7, 9, 4, 20, True),
])
def test_prune_levels_bit_exact(batch, L, Wd, k, B, ties):
    rng = np.random.default_rng(batch * 1000 + L * 10 + Wd + B)
    sizes, tok, par, sco, levels = _random_supertree(rng, batch, L, Wd, k, ties)
    cfg = W.Config("prune", batch=batch, vocab=50000, hidden=64, depth=L, width=Wd, branch=k, budget=B,
                   temperature=0.0, precision=W.FP32, seed=0)
    p = D.Params.of(cfg)
    dev = device()
    out = D.DeviceTree.alloc(batch, B, dev)
    say(f"prune_levels batch={batch} L={L} W={Wd} k={k} B={B}")
    D.prune_levels(p, to_dev(tok), to_dev(par), to_dev(sco), out)
    torch.cuda.synchronize()
    got = out.host()
    for q in range(batch):
        kept = R.prune(levels[q], B)
        t, pa, de, s, m, n = R.emit_tree(levels[q], kept, B)
        assert got["num_nodes"][q] == n
        assert np.array_equal(got["tokens"][q], t)
        assert np.array_equal(got["parents"][q], pa)
        assert np.array_equal(got["depths"][q], de)
        assert np.array_equal(got["mask"][q], m)
        assert np.array_equal(got["scores"][q].astype(np.float64), s)


def test_lse_topk_workspace_reuse():
    """Consecutive calls on one workspace (row tickets must come back to zero),
    with a different number of rows each time."""
    dev = device()
    vocab, k = 151936, 8
    need = max(D.lse_topk_workspace_size(r, vocab, k) for r in (8, 3, 8))
    ws = torch.empty(need, dtype=torch.uint8, device=dev)
    for rep, rows in enumerate((8, 3, 8)):
        z = np.random.default_rng(100 + rep).normal(0, 2, size=(rows, vocab)).astype(np.float32)
        lse = torch.empty(rows, dtype=torch.float32, device=dev)
        lp = torch.empty(rows, k, dtype=torch.float32, device=dev)
        ids = torch.empty(rows, k, dtype=torch.int32, device=dev)
        say(f"lse_topk reuse rows={rows}")
        D.lse_topk(to_dev(z), k, 0.0, lse, lp, ids, ws)
        torch.cuda.synchronize()
        for r in range(rows):
            assert np.array_equal(ids.cpu().numpy()[r], R.topk_ids(z[r].astype(np.float64), k))


def test_calibration_kernels():
    """The calibration kernels do the work they state: the copy is exact, the
    streaming read sums every element, the MFMA loop gives the closed-form sum."""
    dev = device()
    g = torch.Generator().manual_seed(7)
    n = (1 << 20) + 4 * 37                        # ragged against the grid
    src = torch.randint(-8, 8, (n,), generator=g).float().to(dev)
    dst = torch.zeros_like(src)
    sink = torch.zeros(D.CALIB_SINK_FLOATS, device=dev)
    say("calib copy/read/mfma")
    D.calib_copy(dst, src)
    torch.cuda.synchronize()
    assert torch.equal(dst, src)
    D.calib_read(src, sink)
    torch.cuda.synchronize()
    assert float(sink.double().sum()) == float(src.double().sum())   # small integers: exact in fp32
    sink.zero_()
    D.calib_mfma(3, 5, sink)
    torch.cuda.synchronize()
    # accumulator (i, j) adds the tile a_i b_j^T every round: 4 waves, 5 rounds.
    # The operands are pseudo-random bf16 values: element e of lane l of slot
    # s (a_i: slot i, b_j: slot 8 + j) comes from an integer hash of
    # (s * 64 + l) * 8 + e, regenerated here from the same published steps.
    M32 = 0xFFFFFFFF

    def mix(h):
        h ^= h >> 15
        h = (h * 0x2C1B3C6D) & M32
        h ^= h >> 12
        h = (h * 0x297A2D39) & M32
        h ^= h >> 15
        return h

    def operand(slot):                             # lane l holds row l % 16, k-group l // 16
        M = np.zeros((16, 32))
        for l in range(64):
            for e in range(8):
                h = mix((((slot * 64 + l) * 8 + e) * 0x9E3779B1 + 0x3C6EF372) & M32)
                bits = ((h >> 31) << 15) | ((119 + (h >> 8) % 8) << 7) | (h & 0x7F)
                M[l % 16, 8 * (l // 16) + e] = W.bf16_bits_to_fp32(np.array([bits], np.uint16))[0]
        return M

    A = [operand(i) for i in range(8)]
    B = [operand(8 + j) for j in range(8)]
    want = 4 * 5 * sum(float((A[i] @ B[j].T).sum()) for i in range(8) for j in range(8))
    # fp32 accumulation: every product passes through at most ~30 roundings at
    # 2^-24 (5 rounds of 32-term sums, the lane, wave and block reductions)
    scale = 4 * 5 * sum(float((np.abs(A[i]) @ np.abs(B[j]).T).sum()) for i in range(8) for j in range(8))
    got = sink[:3].cpu().double().numpy()
    assert np.all(np.abs(got - want) <= 2e-6 * scale), (got, want, scale)
    assert got[0] == got[1] == got[2]


def test_sync_calibration_kernels():
    """The launch and grid-barrier calibrations: every workgroup passes every
    barrier (each counter ends at the number of workgroups, nothing gives up),
    and a launch of empty workgroups completes."""
    dev = device()
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    counters = torch.zeros(D.CALIB_MAX_BARRIERS, dtype=torch.int32, device=dev)
    fail = torch.zeros(1, dtype=torch.int32, device=dev)
    for blocks, nbar in ((1, 1), (cus, 3), (cus // 2, D.CALIB_MAX_BARRIERS)):
        counters.zero_()
        say(f"calib grid barrier blocks={blocks} nbar={nbar}")
        D.calib_grid_barrier(blocks, nbar, counters, fail)
        torch.cuda.synchronize()
        assert int(fail.item()) == 0
        got = counters.cpu().numpy()
        assert (got[:nbar] == blocks).all() and (got[nbar:] == 0).all(), got[:8]
    D.calib_grid_barrier(cus, 0, counters, fail)
    say("calib empty launches")
    for _ in range(3):
        D.calib_empty(cus)
    torch.cuda.synchronize()
    with pytest.raises(D.DartreeError):
        D.calib_grid_barrier(cus + 1, 1, counters, fail)   # not every workgroup could be resident


@pytest.mark.parametrize("rows,vocab,K,dist", [
    (3, 151936, 64, "normal"), (2, 151936, 256, "ties"), (4, 20001, 17, "ties"), (2, 8193, 64, "normal"),
    (5, 100, 7, "ties"), (3, 8192, 1, "normal"), (2, 40, 40, "ties"),
])
def test_candidate_sets_bit_exact(rows, vocab, K, dist):
    """C = TopK(row, K) by (value desc, id asc), bit for bit, ties included."""
    g = np.random.default_rng(rows * 1000 + K)
    if dist == "ties":
        x = g.integers(-3, 4, size=(rows, vocab)).astype(np.float32)
    else:
        x = g.standard_normal((rows, vocab)).astype(np.float32)
    dev = device()
    xd = torch.from_numpy(x).to(dev)
    ids = torch.empty(rows, K, dtype=torch.int32, device=dev)
    ws = torch.empty(max(D.candidate_sets_workspace_size(rows, vocab, K), 16), dtype=torch.uint8, device=dev)
    say(f"candidate sets rows={rows} V={vocab} K={K} {dist}")
    D.candidate_sets(xd, K, ids, ws)
    torch.cuda.synchronize()
    got = ids.cpu().numpy()
    for r in range(rows):
        want = np.lexsort((np.arange(vocab), -x[r]))[:K]
        assert np.array_equal(got[r], want), (r, got[r][:10], want[:10])
