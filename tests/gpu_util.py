"""Helpers for the GPU tests: run the HIP path on host inputs and copy back."""
from __future__ import annotations

import sys

import numpy as np
import torch

from paper_2608_13524_amd import dartree as D


def device():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    return torch.device("cuda:0")


def say(msg: str) -> None:
    """Name the case before a GPU step (visible even if the process dies)."""
    print(f"[gpu] {msg}", file=sys.stderr, flush=True)


def run_build(cfg, inputs, export=True):
    """dartree_build_tree on cuda:0; returns (tree dict, supertree dict, params)."""
    dev = device()
    p = D.Params.of(cfg)
    di = D.DeviceInputs.from_host(inputs, dev)
    ws = D.alloc_workspace(p, dev)
    out = D.DeviceTree.alloc(cfg.batch, cfg.budget, dev)
    say(f"build_tree {cfg.name} b={cfg.batch} V={cfg.vocab} h={cfg.hidden} L={cfg.depth} "
        f"W={cfg.width} k={cfg.branch} B={cfg.budget} T={cfg.temperature}")
    D.build_tree(p, di, ws, out)
    sup = None
    if export:
        st = D.DeviceSupertree.alloc(p, dev)
        D.export_supertree(p, ws, st)
        torch.cuda.synchronize()
        sup = st.host()
    torch.cuda.synchronize()
    return out.host(), sup, p


def to_dev(a: np.ndarray):
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).to(device())


def run_stepwise(cfg, inputs):
    """expand_depth(1..L) with the features and states of every depth
    exported, then prune.  Returns (tree dict, supertree dict, {d: host
    states of S_d}, {d: host features of depth d's parent rows})."""
    dev = device()
    p = D.Params.of(cfg)
    di = D.DeviceInputs.from_host(inputs, dev)
    ws = D.alloc_workspace(p, dev)
    out = D.DeviceTree.alloc(cfg.batch, cfg.budget, dev)
    sizes = p.level_sizes()
    act = torch.int16 if cfg.precision == D.BF16 else torch.float32
    states, feats = {}, {}
    say(f"stepwise {cfg.name} b={cfg.batch} V={cfg.vocab} h={cfg.hidden} L={cfg.depth} W={cfg.width}")
    for d in range(1, cfg.depth + 1):
        D.expand_depth(p, di, d, ws)
        fb = torch.empty(cfg.batch * (sizes[d - 2] if d > 1 else 1), cfg.hidden, dtype=act, device=dev)
        D.export_features(p, ws, d, fb)
        feats[d] = fb.cpu().numpy()
        if d < cfg.depth:
            buf = torch.empty(cfg.batch * sizes[d - 1], cfg.hidden, dtype=act, device=dev)
            D.export_states(p, ws, d, buf)
            states[d] = buf.cpu().numpy()
    D.prune(p, ws, out)
    st = D.DeviceSupertree.alloc(p, dev)
    D.export_supertree(p, ws, st)
    torch.cuda.synchronize()
    return out.host(), st.host(), states, feats


def decoded(exports: dict, precision: int) -> dict:
    """Decode exported state or feature buffers ({d: bits}) to fp64."""
    from tests import replay
    return {d: replay.decode_states(v, precision) for d, v in exports.items()}
