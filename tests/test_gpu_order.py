"""Algorithm 1's depth order through the C ABI on the GPU: calls that would
read levels no earlier call produced are reported (DARTREE_ERR_ORDER) and
write nothing; with DARTREE_DEBUG=1 the device record in the workspace and
the depth's normalisers are checked as well."""
import os
import subprocess
import sys

import numpy as np
import pytest
import torch

from paper_2608_13524_amd import dartree as D
from paper_2608_13524_amd import workloads as W
from tests.gpu_util import device, say
from tests.test_gpu_parity import small

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _status(fn, *args):
    try:
        fn(*args)
    except D.DartreeError as e:
        return e.status
    return D.OK


@pytest.mark.parametrize("shared", [0, 16])
def test_out_of_order_calls_write_nothing(shared):
    # a budget no other test uses: the library keys its order record by the
    # workspace's address and the parameters, and the allocator may hand this
    # test memory where another test completed a round of the same parameters
    cfg = small(seed=91, candidates=shared, branch=8 if shared else 4, budget=19)
    dev = device()
    p = D.Params.of(cfg)
    di = D.DeviceInputs.from_host(W.make_inputs(cfg), dev)
    ws = D.alloc_workspace(p, dev)
    ws.fill_(0x5A)
    out = D.DeviceTree.alloc(cfg.batch, cfg.budget, dev)
    for f in ("tokens", "parents", "depths", "num_nodes"):
        getattr(out, f).fill_(-7)
    torch.cuda.synchronize()
    say(f"order checks shared={shared}")
    before = ws.clone()
    # a fresh workspace: nothing but depth 1 may run, and nothing is enqueued
    assert _status(D.expand_depth, p, di, 2, ws) == D.ERR_ORDER
    assert _status(D.expand_depth, p, di, cfg.depth, ws) == D.ERR_ORDER
    assert _status(D.prune, p, ws, out) == D.ERR_ORDER
    torch.cuda.synchronize()
    assert torch.equal(ws, before)
    assert (out.tokens == -7).all() and (out.num_nodes == -7).all()
    # depth 1, then skipping depth 2
    D.expand_depth(p, di, 1, ws)
    torch.cuda.synchronize()
    after1 = ws.clone()
    assert _status(D.expand_depth, p, di, 3, ws) == D.ERR_ORDER
    assert _status(D.prune, p, ws, out) == D.ERR_ORDER
    torch.cuda.synchronize()
    assert torch.equal(ws, after1)
    # other parameters on the same workspace do not continue its round
    q = D.Params.of(cfg.replace(depth_bonus=-0.3))
    assert _status(D.expand_depth, q, di, 2, ws) == D.ERR_ORDER
    # in order, the round completes and prunes
    for d in range(2, cfg.depth + 1):
        D.expand_depth(p, di, d, ws)
    D.prune(p, ws, out)
    torch.cuda.synchronize()
    assert (out.num_nodes == min(cfg.budget, cfg.supertree_size())).all()
    # a new round starts at depth 1 at any time
    D.expand_depth(p, di, 1, ws)
    assert _status(D.prune, p, ws, out) == D.ERR_ORDER


_DEBUG_CHILD = r"""
import sys, torch
sys.path.insert(0, {root!r})
from paper_2608_13524_amd import dartree as D
from paper_2608_13524_amd import workloads as W
from tests.test_gpu_parity import small

def status(fn, *a):
    try:
        fn(*a)
    except D.DartreeError as e:
        return e.status
    return D.OK

cfg = small(seed=92)
p = D.Params.of(cfg)
dev = torch.device("cuda:0")
inputs = W.make_inputs(cfg)
di = D.DeviceInputs.from_host(inputs, dev)
ws = D.alloc_workspace(p, dev)
ws.zero_()
# the host record says depth 3 (a captured graph that was never replayed),
# the device record says nothing: the debug check reports the order
g = torch.cuda.CUDAGraph()
with torch.cuda.graph(g):
    for d in (1, 2, 3):
        D.expand_depth(p, di, d, ws)
torch.cuda.synchronize()
print("device-record", status(D.expand_depth, p, di, 4, ws), flush=True)
# after a replay the device record holds depth 3 and the round continues
g.replay()
print("after-replay", status(D.expand_depth, p, di, 4, ws), flush=True)
# an infinite drafter logit at depth 2 makes that depth's normaliser non-finite
bad = W.make_inputs(cfg)
bad.Lb[0, 1, 17] = float("inf")
db = D.DeviceInputs.from_host(bad, dev)
print("depth1", status(D.expand_depth, p, db, 1, ws), flush=True)
print("nonfinite", status(D.expand_depth, p, db, 2, ws), flush=True)
torch.cuda.synchronize()
"""


def test_debug_mode_device_checks():
    """DARTREE_DEBUG=1 (read once per process, so in a child process)."""
    env = dict(os.environ, DARTREE_DEBUG="1")
    say("debug-mode order and finiteness checks (child process)")
    res = subprocess.run([sys.executable, "-c", _DEBUG_CHILD.format(root=ROOT)], env=env, capture_output=True,
                         text=True, timeout=300)
    print(res.stdout, res.stderr[-2000:])
    assert res.returncode == 0
    got = dict(line.split() for line in res.stdout.splitlines() if line.strip())
    assert int(got["device-record"]) == D.ERR_ORDER
    assert int(got["after-replay"]) == D.OK
    assert int(got["depth1"]) == D.OK
    assert int(got["nonfinite"]) == D.ERR_NONFINITE
