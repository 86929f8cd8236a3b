#!/usr/bin/env python3
"""Draft-tree build latency of one DARTree round on one MI355X.

A step is one full round of Algorithm 1 plus the deferred prune
(dartree_build_tree) over one batch of synthetic drafter outputs already
resident in HBM.  Default workload: the Qwen3-4B-shaped one (vocab 151936,
hidden 2560, L=16, W=8, k=8, B=64, T=0, batch 1).

    python bench.py [--steps K] [--warmup W] [--config NAME] [--no-cpu-baseline]

Prints one JSON line: latency per round (value, us), nodes scored per second,
per-kernel average durations, the roofline fraction of the dominant kernel,
and the CPU oracle timed on a bounded sample on the host cores.
"""
from __future__ import annotations

import argparse
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2608_13524_amd import dartree as D  # noqa: E402
from paper_2608_13524_amd import workloads as W  # noqa: E402

METRIC = "draft-tree build latency µs/round; nodes scored/s; % of MFMA/HBM peak"
HBM_PEAK_GBS = 8000.0        # MI355X HBM3E, GB/s
MFMA_BF16_PEAK_TFS = 2500.0  # dense bf16 MFMA, TFLOP/s
FP32_VECTOR_PEAK_TFS = 157.3
RIDGE = MFMA_BF16_PEAK_TFS * 1e12 / (HBM_PEAK_GBS * 1e9)


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def measured_traffic(workload: str, kernel: str):
    """The committed counter summary of this workload and kernel (HBM bytes
    per launch, over the round and at the steady-state depths), or None if
    there is none or the kernel's source has changed since the counters were
    taken."""
    import hashlib
    import re
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.md")
    if not os.path.exists(path):
        return None
    m = re.search(r"```json\s*(\{.*?\})\s*```", open(path).read(), re.S)
    if not m:
        return None
    rec = json.loads(m.group(1))
    if rec.get("kernel") != kernel:
        return None
    src = os.path.join(ROOT, rec["source"])
    if not os.path.exists(src) or hashlib.sha256(open(src, "rb").read()).hexdigest() != rec["source_sha256"]:
        return None
    return rec


def kernel_work(cfg, kind: str, d: int):
    """Algorithmic (bytes, flops) of one launch at depth d.

    logits : per vocabulary row, U row (2h B) + the bias row read once per
             request (4b B) + one fp32 logit written per parent row (4R B);
             plus the R feature rows (2hR B).  flops 2 R h V.
    lse_topk: one fp32 read of z (4 R V B).
    head   : A (2h^2 B) + R state rows in, t (4hR) and a (2hR) out, H rows.
    """
    sizes = [1] + cfg.level_sizes()
    R = cfg.batch * sizes[d - 1]
    h, V, b = cfg.hidden, cfg.vocab, cfg.batch
    act = 2 if cfg.precision == W.BF16 else 4
    K = getattr(cfg, "candidates", 0)
    if K and kind == "logits":
        # shared set: the K gathered rows of U and the bias entries once per
        # request, the R feature rows, one fp32 logit per (row, candidate)
        return b * K * (act * h + 4) + act * h * R + 4 * R * K, 2.0 * R * h * K
    if K and kind == "lse_topk":
        # the candidate sets of all depths, built at d = 1: one read of L^base
        return (4 * b * cfg.depth * V, 0.0) if d == 1 else (0, 0.0)
    if kind == "logits":
        return V * (act * h + 4 * b + 4 * R) + act * h * R, 2.0 * R * h * V
    if kind == "lse_topk":
        return 4 * R * V, 0.0
    if kind == "head":
        return act * h * h + act * h * R + 4 * h * R + act * h * R + act * h * b, 2.0 * R * h * h
    if kind == "select":
        # the rows' candidates in (segment records, or the logits over C_d),
        # parent scores, the level and per-row candidates out, and the state
        # update of the kept children (parent t rows, U rows in, states out)
        k, nk = cfg.branch, b * sizes[d]
        if K:
            rows_in = 4 * R * K + 4 * b * K
        else:
            nseg = max(1, min(-(-1024 // R), -(-V // 2048), 64))
            bucket = next(x for x in (1, 2, 4, 8, 16, 32) if x >= k)
            rows_in = 4 * R * nseg * ((4 + 2 * bucket + 3) & ~3) if nseg > 1 else 8 * R * k
        state = nk * (4 * h + 2 * act * h) if d < cfg.depth else 0
        return rows_in + 4 * R + 12 * nk + R * (4 + 8 * k) + state, 0.0
    return 0, 0.0


def calibrate(torch, dev, U, stream, reps: int = 5) -> dict:
    """Measured ceilings on this GPU: one streaming read of U, a 1 GiB copy and
    an MFMA-only loop (one wave per SIMD), each the mean of `reps` launches."""
    sink = torch.zeros(D.CALIB_SINK_FLOATS, device=dev)
    src = torch.empty(1 << 28, dtype=torch.float32, device=dev).fill_(1.0)
    dst = torch.empty_like(src)

    def mean_us(fn):
        fn()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        for _ in range(reps):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e3 / reps

    u_bytes = U.numel() * U.element_size()
    read_us = mean_us(lambda: D.calib_read(U, sink))
    copy_us = mean_us(lambda: D.calib_copy(dst, src))
    blocks, iters = 256, 2048
    flops = D.calib_mfma(blocks, iters, sink)
    mfma_us = mean_us(lambda: D.calib_mfma(blocks, iters, sink))
    out = {"read_GBs": u_bytes / read_us / 1e3, "read_bytes": u_bytes,
           "copy_GBs": 2 * src.numel() * 4 / copy_us / 1e3, "copy_bytes": src.numel() * 4,
           "mfma_TFs": flops / mfma_us / 1e6}
    out.update(sync_costs(torch, dev, stream, reps))
    return out


def sync_costs(torch, dev, stream, reps: int = 5) -> dict:
    """The two ways the steps of a round can be ordered, priced on this GPU
    with one workgroup of 1024 threads per compute unit: the boundary between
    consecutive launches replayed from a graph, and a grid-wide barrier
    inside one launch (what a single persistent kernel per round would need)."""
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    n = 20
    D.calib_empty(cus)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for _ in range(n):
            D.calib_empty(cus)
    graph.replay()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    launch = []
    for _ in range(reps):
        a.record(stream)
        graph.replay()
        b.record(stream)
        torch.cuda.synchronize()
        launch.append(a.elapsed_time(b) * 1e3 / n)
    counters = torch.zeros(D.CALIB_MAX_BARRIERS, dtype=torch.int32, device=dev)
    fail = torch.zeros(1, dtype=torch.int32, device=dev)

    def kernel_us(nbar):
        ts = []
        for _ in range(reps):
            counters.zero_()
            a.record(stream)
            D.calib_grid_barrier(cus, nbar, counters, fail)
            b.record(stream)
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b) * 1e3)
        return float(np.mean(ts))

    nbar = 16
    t0, tn = kernel_us(0), kernel_us(nbar)
    ok = int(fail.item()) == 0
    return {"sync_blocks": cus, "launch_us": float(np.mean(launch)),
            "grid_barrier_us": (tn - t0) / nbar if ok else None}


def time_heap(torch, cfg, di, stream, steps: int, timed) -> dict:
    """The node-at-a-time baseline (Sec. 3.1, the sequential correction with a
    heap of Table 2) on the same inputs: one round is B pops, each after a head,
    logits and softmax pass on the popped prefix, captured in a HIP graph."""
    p = D.Params.of(cfg)
    dev = di.U.device
    ws = D.alloc_heap_workspace(p, dev)
    out = D.DeviceTree.alloc(cfg.batch, cfg.budget, dev)
    for _ in range(2):
        D.build_tree_heap(p, di, ws, out)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        D.build_tree_heap(p, di, ws, out)
    graph.replay()
    torch.cuda.synchronize()
    per_ms, total_ms, _ = timed(graph.replay, steps)
    pops = int(out.num_nodes.max().item())
    del graph
    return {"us_per_round": total_ms * 1e3 / steps, "us_per_round_p50": float(np.percentile(per_ms, 50) * 1e3),
            "steps": steps, "pops_per_round": pops, "head_evaluations_per_round": cfg.budget,
            "timing": "HIP graph replay of dartree_build_tree_heap"}


def time_consumer(torch, cfg, out, stream, reps: int = 50) -> dict:
    """The step after the path on the tree just built: one tree-attention
    layer of Qwen3-4B's shape over a 2048-position context (the target's
    verification pass reads the emitted mask) and the acceptance walk, each
    the mean of `reps` launches replayed from a HIP graph."""
    dev = out.tokens.device
    s = W.ATTENTION_QWEN3_4B
    ai = W.make_attention_inputs(cfg.batch, cfg.budget, s["max_ctx"], s["heads_q"], s["heads_kv"], seed=7)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16) if a.dtype == np.uint16 else a).to(dev)
    q, kc, vc, kt, vt = t(ai.q), t(ai.k_ctx), t(ai.v_ctx), t(ai.k_tree), t(ai.v_tree)
    p = D.AttnParams(cfg.batch, cfg.budget, s["max_ctx"], s["heads_q"], s["heads_kv"], s["head_dim"],
                     1.0 / np.sqrt(s["head_dim"]))
    nws = D.tree_attention_workspace_size(p)
    ws = torch.empty(nws, dtype=torch.uint8, device=dev) if nws else None
    o = torch.empty(cfg.batch, cfg.budget, s["heads_q"], s["head_dim"], dtype=torch.float32, device=dev)
    target = torch.randint(0, cfg.vocab, (cfg.batch, cfg.budget + 1), dtype=torch.int32, device=dev,
                           generator=torch.Generator(device=dev).manual_seed(7))
    acc = torch.empty(cfg.batch, cfg.depth, dtype=torch.int32, device=dev)
    na = torch.empty(cfg.batch, dtype=torch.int32, device=dev)
    bonus = torch.empty(cfg.batch, dtype=torch.int32, device=dev)

    def mean_us(fn):
        # `reps` launches captured in one HIP graph and replayed, so the host's
        # launch rate does not starve the device between these short kernels
        fn()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(reps):
                fn()
        g.replay()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        g.replay()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e3 / reps

    attn_us = mean_us(lambda: D.tree_attention(p, q, kc, vc, kt, vt, out.mask, None, o, ws))
    walk_us = mean_us(lambda: D.accept_walk(out.tokens, out.parents, out.num_nodes, target, acc, na, bonus))
    # algorithmic work of the layer: context and tree keys/values once, the
    # queries once, fp32 outputs written; 4 flop per (query row, key, dim)
    b, B, n, Hq, Hkv, Dh = cfg.batch, cfg.budget, s["max_ctx"], s["heads_q"], s["heads_kv"], s["head_dim"]
    nbytes = 2 * 2 * b * (n + B) * Hkv * Dh + 2 * b * B * Hq * Dh + 4 * b * B * Hq * Dh
    flops = 4.0 * b * B * Hq * (n + B) * Dh
    # the bound by arithmetic intensity against the spec balance (2.5 PFLOP/s / 8 TB/s = 312 flop/B)
    if flops / nbytes > MFMA_BF16_PEAK_TFS * 1e12 / (HBM_PEAK_GBS * 1e9):
        roof = {"bound": "mfma", "achieved": flops / attn_us / 1e6, "peak": MFMA_BF16_PEAK_TFS, "unit": "TFLOP/s",
                "frac": flops / attn_us / 1e6 / MFMA_BF16_PEAK_TFS}
    else:
        roof = {"bound": "hbm", "achieved": nbytes / attn_us / 1e3, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": nbytes / attn_us / 1e3 / HBM_PEAK_GBS}
    roof.update({"algorithmic_bytes": nbytes, "flops": flops})
    if nbytes < 64e6:
        roof["note"] = (f"latency-bound: {nbytes / 1e6:.0f} MB and {flops / 1e9:.1f} GFLOP per layer "
                        f"({b} request(s) x {B} nodes)")
    return {"tree_attention_us": attn_us, "accept_walk_us": walk_us,
            "shape": {"heads_q": Hq, "heads_kv": Hkv, "head_dim": Dh, "context": n, "nodes": B},
            "attention_roofline": roof}


# The per-kernel targets are stated for the throughput-stress shape: 16
# requests x 64 nodes = 1024 parent rows against the 151936-token vocabulary
# at hidden 5120 (the only shape above the MFMA ridge).
TARGET_SHAPE = dict(rows=1024, vocab=151936, hidden=5120, k=8, rows_per_group=64)


def time_targets(torch, dev, stream, reps: int = 10, calibration: bool = False) -> dict:
    """The projection and the softmax/top-k pass at the stress shape, through
    dartree_project and dartree_lse_topk on device buffers filled with random
    bf16 features (tanh of normals, like the head's output) and weights
    N(0, 0.02^2) (random operands: the matrix cores' power draw, and so their
    clock, depends on the data).  No host inputs and no oracle.  Each launch is
    timed by its own event pair on the stream it runs on; the projection and
    the pass alternate as in a round, so the pass reads logits the projection
    has just written."""
    s = TARGET_SHAPE
    R, V, h, k = s["rows"], s["vocab"], s["hidden"], s["k"]
    g = torch.Generator(device=dev).manual_seed(11)
    x = torch.tanh(torch.randn(R, h, device=dev, generator=g) * 1.4).to(torch.bfloat16)
    U = (torch.randn(V, h, device=dev, generator=g) * 0.02).to(torch.bfloat16)
    groups = R // s["rows_per_group"]
    bias = torch.randn(groups, V, device=dev, generator=g) * 2.0
    z = torch.empty(R, V, dtype=torch.float32, device=dev)
    nws = D.project_workspace_size(D.BF16, R, V, h)
    pws = torch.empty(max(nws, 1), dtype=torch.uint8, device=dev)
    lse = torch.empty(R, dtype=torch.float32, device=dev)
    lp = torch.empty(R, k, dtype=torch.float32, device=dev)
    ids = torch.empty(R, k, dtype=torch.int32, device=dev)
    lws = torch.empty(max(D.lse_topk_workspace_size(R, V, k), 1), dtype=torch.uint8, device=dev)
    xi, Ui = x.view(torch.int16), U.view(torch.int16)

    def proj():
        D.project(D.BF16, xi, Ui, bias, V, z, s["rows_per_group"], pws)

    def soft():
        D.lse_topk(z, k, 1.0, lse, lp, ids, lws)

    for _ in range(2):
        proj()
        soft()
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(2 * reps)]
    for i in range(reps):
        ev[2 * i][0].record(stream)
        proj()
        ev[2 * i][1].record(stream)
        ev[2 * i + 1][0].record(stream)
        soft()
        ev[2 * i + 1][1].record(stream)
    torch.cuda.synchronize()
    pt = np.array([a.elapsed_time(b) * 1e3 for a, b in ev[0::2]])
    st = np.array([a.elapsed_time(b) * 1e3 for a, b in ev[1::2]])
    flops = 2.0 * R * h * V
    pbytes = V * (2 * h + 4 * groups + 4 * R) + 2 * h * R
    lbytes = 4.0 * R * V
    p_tf = flops / pt.mean() / 1e6
    l_gb = lbytes / st.mean() / 1e3
    out = {
        "shape": {"rows": R, "vocab": V, "hidden": h, "k": k, "bias_rows": groups},
        "projection": {"avg_launch_us": float(pt.mean()), "min_launch_us": float(pt.min()),
                       "algorithmic_flops_per_launch": flops, "algorithmic_bytes_per_launch": pbytes,
                       "achieved_TFs": p_tf, "peak_TFs": MFMA_BF16_PEAK_TFS, "frac": p_tf / MFMA_BF16_PEAK_TFS,
                       "target_frac": 0.5, "launches": reps,
                       "note": "includes the fix-up launch of the split last wave when the split applies"},
        "lse_topk": {"avg_launch_us": float(st.mean()), "min_launch_us": float(st.min()),
                     "algorithmic_bytes_per_launch": lbytes, "achieved_GBs": l_gb, "peak_GBs": HBM_PEAK_GBS,
                     "frac": l_gb / HBM_PEAK_GBS, "target_frac": 0.6, "launches": reps},
        "timing": "HIP events around each dartree_project / dartree_lse_topk call on the launch stream",
    }
    out["projection_mfma_frac"] = out["projection"]["frac"]
    out["lse_topk_hbm_frac"] = out["lse_topk"]["frac"]
    del x, bias, z, pws, lws
    if calibration:   # the copy of known size that scales the traffic counters, in the same process
        out["calibration"] = calibrate(torch, dev, U, stream)
    del U
    torch.cuda.empty_cache()
    return out


def gpu_env(torch) -> dict:
    """Device, HIP runtime and the shader clock, read from the device's
    pp_dpm_sclk file in sysfs (the level marked current), sampled right after
    the timed replays; null where the file is not readable."""
    props = torch.cuda.get_device_properties(0)
    env = {"device": torch.cuda.get_device_name(0), "arch": getattr(props, "gcnArchName", None),
           "compute_units": props.multi_processor_count, "hip": torch.version.hip, "sclk_mhz": None}
    try:
        pci = f"{props.pci_domain_id:04x}:{props.pci_bus_id:02x}:{props.pci_device_id:02x}.0"
        with open(f"/sys/bus/pci/devices/{pci}/pp_dpm_sclk") as f:
            for line in f:                  # e.g. "1: 2400Mhz *"
                m = re.search(r"(\d+)\s*mhz\s*\*", line, re.I)
                if m:
                    env["sclk_mhz"] = int(m.group(1))
    except (OSError, AttributeError, ValueError):
        pass
    return env


def cpu_baseline(cfg, inputs, budget_s: float = 20.0) -> dict:
    """The oracle (fp64 NumPy) on the host cores, on the first D depths of
    request 0 with D chosen to take ~budget_s; scaled to us per full round."""
    import threadpoolctl

    import oracle.dartree_ref as R
    sub = W.Inputs(cfg=cfg.replace(batch=1), Lb=inputs.Lb[:1], H=inputs.H[:1], r0=inputs.r0[:1],
                   A=inputs.A, U=inputs.U)
    dec = R.prepare(sub)
    rows = [1] + cfg.level_sizes()[:-1]          # parent rows per depth, one request
    info = threadpoolctl.threadpool_info()
    threads = max([i.get("num_threads", 1) for i in info if i.get("user_api") == "blas"] or [1])

    def run(depth: int) -> float:
        p = R.Params.of(cfg.replace(batch=1, depth=depth))
        d2 = R.Decoded(p, dec.Lb[:, :depth], dec.H[:, :depth], dec.r0, dec.A, dec.U)
        t0 = time.perf_counter()
        R.build_tree(d2)
        return time.perf_counter() - t0

    t1 = run(1)
    per_row = t1 / rows[0]
    depth = 1
    while depth < cfg.depth and per_row * sum(rows[:depth + 1]) < budget_s:
        depth += 1
    t = run(depth) if depth > 1 else t1
    reps = 1
    while depth == cfg.depth and reps * t < budget_s / 2:   # whole rounds: repeat, report the mean
        t = (t * reps + run(depth)) / (reps + 1)
        reps += 1
    scale = sum(rows) / sum(rows[:depth]) * cfg.batch
    blas = ",".join(sorted({i.get("internal_api", "?") for i in info if i.get("user_api") == "blas"})) or None
    return {"value": t * scale * 1e6, "unit": "us/round", "cores": int(threads), "kind": "oracle",
            "blas": blas, "host_cpus_available": len(os.sched_getaffinity(0)),
            "sample": f"request 0, depths 1..{depth} of {cfg.depth} (mean of {reps} run(s), {t:.2f} s each), "
                      f"scaled by parent rows to the full round of {cfg.batch} request(s)"}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="qwen3-4b", choices=W.CONFIG_ORDER)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-heap", action="store_true", help="skip the sequential-heap comparison")
    ap.add_argument("--schedule", default="dartree", choices=["dartree", "heap"],
                    help="heap: time only the sequential-heap baseline (for a kernel trace of it alone)")
    ap.add_argument("--width", type=int, default=None, help="override the workload's layer width W (sweeps)")
    ap.add_argument("--budget", type=int, default=None, help="override the workload's budget B (sweeps)")
    ap.add_argument("--no-targets", action="store_true",
                    help="skip the per-kernel target leg at the stress shape")
    ap.add_argument("--targets-only", action="store_true",
                    help="run only the per-kernel target leg (for its counter runs)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only (--gpus 1): the library builds trees on one device. Requests "
              "are independent trees, so several GPUs would each take their own requests with no exchange.",
              file=sys.stderr)
        return 2

    import torch
    assert torch.cuda.is_available(), "bench.py needs a ROCm GPU"
    dev = torch.device("cuda:0")
    cfg = W.CONFIGS[args.config]
    if args.width is not None or args.budget is not None:
        cfg = cfg.replace(width=args.width if args.width is not None else cfg.width,
                          budget=args.budget if args.budget is not None else cfg.budget)
    log(f"workload {cfg.name}: generating inputs")
    inputs = W.make_inputs(cfg)
    p = D.Params.of(cfg)
    di = D.DeviceInputs.from_host(inputs, dev)
    stream = torch.cuda.current_stream()

    def timed(run_round, K):
        """K rounds, an event pair around each; returns (per-round ms, total ms, wall s)."""
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(K + 1)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ev[0].record(stream)
        for i in range(K):
            run_round()
            ev[i + 1].record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        return np.array([ev[i].elapsed_time(ev[i + 1]) for i in range(K)]), ev[0].elapsed_time(ev[K]), wall

    if args.targets_only:
        log("per-kernel targets at the stress shape only")
        tg = time_targets(torch, dev, torch.cuda.current_stream(), reps=max(args.steps, 1), calibration=True)
        log(f"  projection {tg['projection']['avg_launch_us']:.1f} us ({tg['projection_mfma_frac']:.3f} of MFMA), "
            f"softmax/top-k {tg['lse_topk']['avg_launch_us']:.1f} us ({tg['lse_topk_hbm_frac']:.3f} of HBM)")
        print(json.dumps({"targets": tg, "env": gpu_env(torch)}), flush=True)
        return 0

    if args.schedule == "heap":
        log(f"sequential heap only: {args.steps} rounds")
        heap = time_heap(torch, cfg, di, stream, args.steps, timed)
        log(f"  {heap['us_per_round']:.1f} us/round")
        print(json.dumps({
            "metric": METRIC, "value": heap["us_per_round"], "unit": "us/round", "n_gpus": 1, "steps": args.steps,
            "warmup": 2, "ms_per_step": heap["us_per_round"] / 1e3, "higher_is_better": False, "scaling": "weak",
            "vs_baseline": None, "dtype": "bf16" if cfg.precision == W.BF16 else "f32", "data": "synthetic",
            "config": {"workload": cfg.name, "schedule": "sequential-heap", "batch": cfg.batch, "budget": cfg.budget,
                       "branch": cfg.branch, "candidates": getattr(cfg, "candidates", 0),
                       "head": "markov" if getattr(cfg, "head", 0) == 1 else "rnn"},
            "sequential_heap": heap, "roofline": None, "cpu_baseline": None}), flush=True)
        return 0

    ws = D.alloc_workspace(p, dev)
    out = D.DeviceTree.alloc(cfg.batch, cfg.budget, dev)
    log(f"warmup {args.warmup}")
    for _ in range(args.warmup):
        D.build_tree(p, di, ws, out)
    torch.cuda.synchronize()

    # the round captured once in a HIP graph; a replay equals an eager call
    # (kernel launches only: no copies, fills or host synchronisation inside)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        D.build_tree(p, di, ws, out)
    torch.cuda.synchronize()
    for _ in range(2):
        graph.replay()
    torch.cuda.synchronize()

    # timed region: exactly K graph replays (the value), then K eager calls
    K = args.steps
    per_step_ms, total_ms, wall = timed(graph.replay, K)
    us_round = total_ms * 1e3 / K
    env = gpu_env(torch)
    log(f"timed {K} graph replays: {us_round:.1f} us/round (wall {wall * 1e3 / K:.1f} ms/round)")
    eager_ms, eager_total, _ = timed(lambda: D.build_tree(p, di, ws, out), K)
    eager_us = eager_total * 1e3 / K
    log(f"timed {K} eager calls:   {eager_us:.1f} us/round")

    # kernel durations: the same K rounds through the instrumented launch
    # sequence, an event pair around every launch
    nk = len(D.KERNEL_NAMES)
    n_ev = 2 * (nk * cfg.depth + 1)
    kev = [[torch.cuda.Event(enable_timing=True) for _ in range(n_ev)] for _ in range(K)]
    for e in kev[0]:
        e.record(stream)                     # creates the underlying hipEvent_t
    for evs in kev[1:]:
        for e in evs:
            e.record(stream)
    torch.cuda.synchronize()
    for i in range(K):
        D.build_tree_timed(p, di, ws, out, [e.cuda_event for e in kev[i]])
    torch.cuda.synchronize()
    dur = {name: [] for name in D.KERNEL_NAMES + ["prune"]}
    work = {name: [0.0, 0.0] for name in D.KERNEL_NAMES + ["prune"]}
    # the steady-state depths: those with the most parent rows (every depth
    # after the level sizes stop growing)
    sizes = [1] + cfg.level_sizes()
    steady = [d for d in range(1, cfg.depth + 1) if sizes[d - 1] == max(sizes[:cfg.depth])]
    steady_t = {name: 0.0 for name in D.KERNEL_NAMES}
    steady_w = {name: [0.0, 0.0] for name in D.KERNEL_NAMES}
    for i in range(K):
        for d in range(1, cfg.depth + 1):
            for c, name in enumerate(D.KERNEL_NAMES):
                j = (d - 1) * nk + c
                t_ = kev[i][2 * j].elapsed_time(kev[i][2 * j + 1]) * 1e3
                dur[name].append(t_)
                b_, f_ = kernel_work(cfg, name, d)
                if d in steady:
                    steady_t[name] += t_
                    steady_w[name][0] += b_
                    steady_w[name][1] += f_
                if i == 0:
                    work[name][0] += b_
                    work[name][1] += f_
        j = cfg.depth * nk
        dur["prune"].append(kev[i][2 * j].elapsed_time(kev[i][2 * j + 1]) * 1e3)
    kernels = {}
    for name, v in dur.items():
        per_round = sum(v) / K
        kernels[name] = {"us_per_round": per_round, "launches_per_round": len(v) // K,
                         "avg_us_per_launch": per_round / max(len(v) // K, 1)}
        log(f"  {name:9s} {per_round:9.1f} us/round  ({len(v) // K} launches)")
    instrumented_us = sum(k["us_per_round"] for k in kernels.values())

    dom = max(kernels, key=lambda n: kernels[n]["us_per_round"])
    bytes_round, flops_round = work[dom]
    t_round = kernels[dom]["us_per_round"] * 1e-6
    intensity = flops_round / bytes_round if bytes_round else 0.0
    launches = kernels[dom]["launches_per_round"]
    if cfg.precision == W.BF16 and dom == "logits" and intensity > RIDGE:
        roof = {"bound": "mfma", "achieved": flops_round / t_round / 1e12, "peak": MFMA_BF16_PEAK_TFS,
                "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": bytes_round / t_round / 1e9, "peak": HBM_PEAK_GBS, "unit": "GB/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    if roof["frac"] < 0.1:
        roof["note"] = ("latency-bound: each launch moves little data, so its duration is launch and "
                        "dependent-load latency, not bandwidth")
    traffic = measured_traffic(cfg.name, dom)
    roof["traffic"] = float(traffic["traffic_bytes_per_launch"]) if traffic else None
    roof["kernel"] = dom
    roof["algorithmic_bytes_per_launch"] = bytes_round / launches
    roof["algorithmic_flops_per_launch"] = flops_round / launches
    roof["avg_launch_us"] = kernels[dom]["avg_us_per_launch"]

    def steady_state(name, bound):
        t_ = steady_t[name] * 1e-6
        if t_ <= 0:
            return None
        b_, f_ = steady_w[name]
        ach = f_ / t_ / 1e12 if bound == "mfma" else b_ / t_ / 1e9
        peak = MFMA_BF16_PEAK_TFS if bound == "mfma" else HBM_PEAK_GBS
        n = len(steady) * K
        return {"depths": [steady[0], steady[-1]], "rows": cfg.batch * sizes[steady[0] - 1],
                "avg_launch_us": steady_t[name] / n, "algorithmic_bytes_per_launch": b_ / n,
                "algorithmic_flops_per_launch": f_ / n, "achieved": ach, "frac": ach / peak}

    if dom in steady_t:
        roof["steady_state"] = steady_state(dom, roof["bound"])
        if roof["steady_state"]:
            roof["steady_state"]["traffic"] = (float(traffic.get("steady_traffic_bytes_per_launch",
                                                                 traffic["traffic_bytes_per_launch"]))
                                               if traffic else None)
    # second roofline of the per-row softmax/top-k pass (HBM); with a shared
    # candidate set this slot is the candidate-set pass over L^base at d = 1
    # (over the depths that launch it)
    lse_d = [d for d in range(1, cfg.depth + 1) if kernel_work(cfg, "lse_topk", d)[0] > 0]
    lse_roof = None
    if lse_d:
        lb = sum(kernel_work(cfg, "lse_topk", d)[0] for d in lse_d)
        lse_t = sum(dur["lse_topk"][i * cfg.depth + d - 1] for i in range(K) for d in lse_d) / K * 1e-6
        lse_roof = {"bound": "hbm", "achieved": lb / lse_t / 1e9, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": lb / lse_t / 1e9 / HBM_PEAK_GBS, "depths": lse_d,
                    "note": ("candidate sets TopK(L^base, K) of every depth, built once per round"
                             if getattr(cfg, "candidates", 0) else
                             "z is written by the projection just before; below ~256 MB it can be served "
                             "from the Infinity Cache rather than HBM")}
    proj_flops = work["logits"][1] / (kernels["logits"]["us_per_round"] * 1e-6) / 1e12

    # achievable ceilings measured in this job: stream U once (the projection's
    # access pattern), copy 1 GiB, and a register-only MFMA loop
    cal = calibrate(torch, dev, di.U, stream)
    gb = cal["grid_barrier_us"]
    log(f"calibration: read {cal['read_GBs']:.0f} GB/s, copy {cal['copy_GBs']:.0f} GB/s, "
        f"mfma {cal['mfma_TFs']:.0f} TFLOP/s; launch boundary {cal['launch_us']:.2f} us, grid barrier "
        + (f"{gb:.2f} us" if gb is not None else "gave up"))
    meas = cal["mfma_TFs"] if roof["bound"] == "mfma" else cal["read_GBs"]
    roof["measured_peak"] = meas
    roof["frac_of_measured"] = roof["achieved"] / meas
    if lse_roof:
        lse_roof["measured_peak"] = cal["read_GBs"]
        lse_roof["frac_of_measured"] = lse_roof["achieved"] / cal["read_GBs"]
        if not getattr(cfg, "candidates", 0) and steady_w["lse_topk"][0] > 0:
            lse_roof["steady_state"] = steady_state("lse_topk", "hbm")
            if lse_roof["steady_state"]:
                lse_roof["steady_state"]["frac_of_measured"] = (lse_roof["steady_state"]["achieved"] /
                                                                cal["read_GBs"])
    if roof.get("steady_state"):
        roof["steady_state"]["frac_of_measured"] = roof["steady_state"]["achieved"] / meas

    sizes = [1] + cfg.level_sizes()
    nodes = cfg.batch * sum(sizes[d - 1] * cfg.branch for d in range(1, cfg.depth + 1))
    per_row = getattr(cfg, "candidates", 0) or cfg.vocab   # entries scored per parent row
    vocab_entries = cfg.batch * sum(sizes[d - 1] for d in range(1, cfg.depth + 1)) * per_row

    # the node-at-a-time baseline DARTree's depth-wise schedule replaces,
    # a few rounds (each is B head evaluations)
    heap = None
    if cfg.budget <= D.MAX_HEAP_BUDGET and not args.no_heap:
        heap_steps = max(3, min(K, int(2e6 / max(us_round * cfg.budget / cfg.depth, 1.0))))
        log(f"sequential heap: {heap_steps} rounds")
        heap = time_heap(torch, cfg, di, stream, heap_steps, timed)
        heap["vs_dartree"] = heap["us_per_round"] / us_round
        log(f"  {heap['us_per_round']:.1f} us/round, {heap['vs_dartree']:.2f}x DARTree's round")

    targets = None
    if not args.no_targets and cfg.precision == W.BF16:
        log("per-kernel targets at the stress shape (1024 x 151936 x 5120)")
        targets = time_targets(torch, dev, stream)
        log(f"  projection {targets['projection']['avg_launch_us']:.1f} us/launch = "
            f"{targets['projection']['achieved_TFs']:.0f} TFLOP/s ({targets['projection_mfma_frac']:.3f} of MFMA); "
            f"softmax/top-k {targets['lse_topk']['avg_launch_us']:.1f} us/launch = "
            f"{targets['lse_topk']['achieved_GBs']:.0f} GB/s ({targets['lse_topk_hbm_frac']:.3f} of HBM)")

    consumer = None
    if cfg.precision == W.BF16:
        consumer = time_consumer(torch, cfg, out, stream)
        log(f"consumer: tree attention {consumer['tree_attention_us']:.1f} us, "
            f"acceptance walk {consumer['accept_walk_us']:.1f} us")

    cpu = None
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle on host cores)")
        cpu = cpu_baseline(cfg, inputs)
        log(f"  oracle {cpu['value'] / 1e6:.2f} s/round on {cpu['cores']} threads ({cpu['sample']})")

    line = {
        "metric": METRIC, "value": us_round, "unit": "us/round", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": total_ms / K, "higher_is_better": False, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16" if cfg.precision == W.BF16 else "f32", "data": "synthetic",
        "config": {"workload": cfg.name, "batch": cfg.batch, "vocab": cfg.vocab, "hidden": cfg.hidden,
                   "depth": cfg.depth, "width": cfg.width, "branch": cfg.branch, "budget": cfg.budget,
                   "temperature": cfg.temperature, "depth_bonus": cfg.depth_bonus,
                   "candidates": getattr(cfg, "candidates", 0),
                   "head": "markov" if getattr(cfg, "head", 0) == 1 else "rnn"},
        "timing": "HIP graph replay of dartree_build_tree",
        "eager_us_per_round": eager_us,
        "us_per_round_p10": float(np.percentile(per_step_ms, 10) * 1e3),
        "us_per_round_p50": float(np.percentile(per_step_ms, 50) * 1e3),
        "us_per_round_p90": float(np.percentile(per_step_ms, 90) * 1e3),
        "nodes_scored_per_s": nodes / (us_round * 1e-6),
        "vocab_entries_scored_per_s": vocab_entries / (us_round * 1e-6),
        "projection_tflops": proj_flops,
        "projection_mfma_frac": proj_flops / MFMA_BF16_PEAK_TFS,
        "kernels": kernels, "instrumented_us_per_round": instrumented_us,
        "roofline": roof, "lse_topk_roofline": lse_roof, "targets": targets, "calibration": cal,
        "sequential_heap": heap,
        "consumer": consumer, "env": env,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
