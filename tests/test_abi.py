"""The C ABI without a GPU: the library loads, exports every declared entry
point, and rejects bad arguments on the host before touching the device."""
import ctypes
import math
import re
import os

import pytest

from paper_2608_13524_amd import dartree as D
from paper_2608_13524_amd import workloads as W

INCLUDE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include")
HEADERS = sorted(os.path.join(INCLUDE, f) for f in os.listdir(INCLUDE) if f.endswith(".h"))
FAKE = 0x10000  # 16-byte aligned address that is never dereferenced


def declared_symbols():
    text = "".join(open(h).read() for h in HEADERS)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\**\s+\**(dartree_\w+)\s*\(", text, re.M)))


def test_library_exports_every_declared_symbol():
    syms = declared_symbols()
    assert len(syms) == 31, syms
    lib = D.lib()
    for s in syms:
        assert hasattr(lib, s), s
    assert sorted(D.SYMBOLS) == syms


def test_abi_version_and_status_strings():
    assert D.abi_version() == D.ABI_VERSION == 8
    for s in range(7):
        assert D.status_string(s)
    assert D.status_string(99) == "unknown status"


def _p(**kw):
    cfg = W.CONFIGS["qwen3-4b"]
    p = D.Params.of(cfg)
    for k, v in kw.items():
        setattr(p, k, v)
    return p


@pytest.mark.parametrize("field,value,code", [
    ("batch", 0, D.ERR_INVALID_ARG), ("vocab", 0, D.ERR_INVALID_ARG), ("hidden", 0, D.ERR_INVALID_ARG),
    ("depth", 0, D.ERR_INVALID_ARG), ("width", 0, D.ERR_INVALID_ARG), ("branch", 0, D.ERR_INVALID_ARG),
    ("budget", 0, D.ERR_INVALID_ARG), ("precision", 7, D.ERR_INVALID_ARG),
    ("temperature", -0.5, D.ERR_INVALID_ARG), ("temperature", math.nan, D.ERR_INVALID_ARG),
    ("temperature", math.inf, D.ERR_INVALID_ARG), ("depth_bonus", 0.1, D.ERR_INVALID_ARG),
    ("depth_bonus", math.nan, D.ERR_INVALID_ARG), ("branch", 151937, D.ERR_INVALID_ARG),
    ("vocab", (1 << 20) + 1, D.ERR_UNSUPPORTED), ("depth", 65, D.ERR_UNSUPPORTED),
    ("width", 2049, D.ERR_UNSUPPORTED), ("branch", 33, D.ERR_UNSUPPORTED),
    ("budget", 4097, D.ERR_UNSUPPORTED), ("hidden", 2560 + 32, D.ERR_UNSUPPORTED),
    ("width", 1024, D.ERR_UNSUPPORTED),   # 1024 parents x 8 candidates > 4096
    ("head", 2, D.ERR_INVALID_ARG), ("head", -1, D.ERR_INVALID_ARG),
])
def test_validate_rejects(field, value, code):
    assert D.validate(_p(**{field: value})) == code


def test_validate_accepts_all_workloads_and_edges():
    for name in W.CONFIG_ORDER:
        assert D.validate(D.Params.of(W.CONFIGS[name])) == D.OK, name
    assert D.validate(_p(depth_bonus=0.0, temperature=0.0)) == D.OK
    assert D.validate(_p(depth_bonus=-0.0)) == D.OK
    assert D.validate(_p(width=1, branch=1, budget=1)) == D.OK
    assert D.validate(_p(head=D.HEAD_MARKOV)) == D.OK
    fp = D.Params.of(W.CONFIGS["tiny"])
    fp.hidden = 7                      # any hidden size in fp32 mode
    assert D.validate(fp) == D.OK
    assert D.validate(None) == D.ERR_INVALID_ARG


def test_workspace_size():
    p = D.Params.of(W.CONFIGS["stress-x16"])
    n = D.workspace_size(p)
    R, V, h = 16 * 64, 151936, 5120
    assert n >= R * V * 4 + 2 * R * h * 2 + R * h * 4   # logits, states, features
    assert n % 256 == 0
    assert D.workspace_size(D.Params.of(W.CONFIGS["qwen3-4b"])) < n
    with pytest.raises(D.DartreeError) as e:
        D.workspace_size(_p(batch=0))
    assert e.value.status == D.ERR_INVALID_ARG


def _inputs():
    return D.InputsC(FAKE, FAKE, FAKE, FAKE, FAKE)


def _tree():
    return D.TreeC(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE)


def test_entry_points_reject_before_any_launch():
    lib = D.lib()
    p = _p()
    need = D.workspace_size(p)
    byref = ctypes.byref
    # null / misaligned pointers
    bad_in = D.InputsC(FAKE, FAKE, None, FAKE, FAKE)
    assert lib.dartree_build_tree(byref(p), byref(bad_in), FAKE, need, byref(_tree()), None) == D.ERR_INVALID_ARG
    mis = D.InputsC(FAKE + 4, FAKE, FAKE, FAKE, FAKE)
    assert lib.dartree_build_tree(byref(p), byref(mis), FAKE, need, byref(_tree()), None) == D.ERR_INVALID_ARG
    bad_tree = D.TreeC(FAKE, FAKE, FAKE, FAKE, None, FAKE)
    assert lib.dartree_build_tree(byref(p), byref(_inputs()), FAKE, need, byref(bad_tree), None) == D.ERR_INVALID_ARG
    # workspace: too small, misaligned, missing
    assert lib.dartree_build_tree(byref(p), byref(_inputs()), FAKE, need - 1, byref(_tree()), None) == D.ERR_WORKSPACE
    assert lib.dartree_build_tree(byref(p), byref(_inputs()), FAKE + 16, need, byref(_tree()), None) == D.ERR_WORKSPACE
    assert lib.dartree_build_tree(byref(p), byref(_inputs()), None, need, byref(_tree()), None) == D.ERR_WORKSPACE
    # depth index out of range
    assert lib.dartree_expand_depth(byref(p), byref(_inputs()), 0, FAKE, need, None) == D.ERR_INVALID_ARG
    assert lib.dartree_expand_depth(byref(p), byref(_inputs()), 17, FAKE, need, None) == D.ERR_INVALID_ARG
    assert lib.dartree_prune(byref(p), FAKE, need - 256, byref(_tree()), None) == D.ERR_WORKSPACE
    assert lib.dartree_export_supertree(byref(p), FAKE, need, None, None) == D.ERR_INVALID_ARG
    assert lib.dartree_export_states(byref(p), FAKE, need, 16, FAKE, None) == D.ERR_INVALID_ARG
    assert lib.dartree_export_states(byref(p), FAKE, need, 0, FAKE, None) == D.ERR_INVALID_ARG
    assert lib.dartree_export_states(byref(p), FAKE, need - 1, 3, FAKE, None) == D.ERR_WORKSPACE
    # single-step calls
    assert lib.dartree_project(1, 8, 100, 65, 8, FAKE, FAKE, FAKE, 100, FAKE, None, 0, None) == D.ERR_UNSUPPORTED
    assert lib.dartree_project(1, 0, 100, 64, 8, FAKE, FAKE, FAKE, 100, FAKE, None, 0, None) == D.ERR_INVALID_ARG
    assert lib.dartree_project(1, 8, 100, 64, 8, FAKE + 2, FAKE, FAKE, 100, FAKE, None, 0, None) == D.ERR_INVALID_ARG
    # split scratch: none for few rows or fp32; 64 MB of split partials for the
    # many-row tilings, plus the node rows in fragment order for the 512-row
    # tiles (row counts that are multiples of 512, as 1024)
    assert D.project_workspace_size(D.BF16, 64, 151936, 2560) == 0
    assert D.project_workspace_size(D.FP32, 1024, 151936, 2560) == 0
    assert D.project_workspace_size(D.BF16, 768, 151936, 5120) == 256 * 256 * 256 * 4
    assert D.project_workspace_size(D.BF16, 1000, 151936, 5120) == 256 * 256 * 256 * 4
    split = D.project_workspace_size(D.BF16, 1024, 151936, 5120)
    assert split == 256 * 256 * 256 * 4 + 1024 * 5120 * 2
    assert lib.dartree_project(1, 1024, 151936, 5120, 64, FAKE, FAKE, FAKE, 0, FAKE, None, 0, None) == D.ERR_WORKSPACE
    assert lib.dartree_project(1, 1024, 151936, 5120, 64, FAKE, FAKE, FAKE, 0, FAKE, FAKE, split - 1,
                               None) == D.ERR_WORKSPACE
    assert lib.dartree_project(1, 1024, 151936, 5120, 64, FAKE, FAKE, FAKE, 0, FAKE, FAKE + 16, split,
                               None) == D.ERR_WORKSPACE
    assert lib.dartree_lse_topk(FAKE, 4, 100, 101, 1.0, FAKE, FAKE, FAKE, None, 0, None) == D.ERR_INVALID_ARG
    assert lib.dartree_lse_topk(FAKE, 4, 100, 4, -1.0, FAKE, FAKE, FAKE, None, 0, None) == D.ERR_INVALID_ARG
    big = D.lse_topk_workspace_size(1, 151936, 8)
    assert big > 0
    assert lib.dartree_lse_topk(FAKE, 1, 151936, 8, 1.0, FAKE, FAKE, FAKE, None, 0, None) == D.ERR_WORKSPACE
    assert lib.dartree_select_topw(1, 8, 8, 65, -0.2, None, FAKE, FAKE, FAKE, FAKE, FAKE, None) == D.ERR_INVALID_ARG
    assert lib.dartree_select_topw(1, 8, 8, 8, 0.5, None, FAKE, FAKE, FAKE, FAKE, FAKE, None) == D.ERR_INVALID_ARG
    assert lib.dartree_select_topw(1, 1024, 8, 8, -0.2, None, FAKE, FAKE, FAKE, FAKE, FAKE, None) == D.ERR_UNSUPPORTED
    assert lib.dartree_prune_levels(byref(p), None, FAKE, FAKE, byref(_tree()), None) == D.ERR_INVALID_ARG


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(D, "_lib", None)
    monkeypatch.setattr(D, "LIB_PATH", str(tmp_path / "absent.so"))
    with pytest.raises(RuntimeError, match="no fallback"):
        D.lib()


def test_calibration_kernels_reject_bad_arguments():
    lib = D.lib()
    sink = ctypes.c_void_p(FAKE)
    assert lib.dartree_calib_read(None, 1024, sink, None) == D.ERR_INVALID_ARG
    assert lib.dartree_calib_read(ctypes.c_void_p(FAKE), 1000, sink, None) == D.ERR_INVALID_ARG   # not 16 B units
    assert lib.dartree_calib_read(ctypes.c_void_p(FAKE + 4), 1024, sink, None) == D.ERR_INVALID_ARG
    assert lib.dartree_calib_read(ctypes.c_void_p(FAKE), 0, sink, None) == D.ERR_INVALID_ARG
    assert lib.dartree_calib_read(ctypes.c_void_p(FAKE), 1024, None, None) == D.ERR_INVALID_ARG
    assert lib.dartree_calib_copy(ctypes.c_void_p(FAKE), ctypes.c_void_p(FAKE + 512), 1024, None) == D.ERR_INVALID_ARG
    assert lib.dartree_calib_copy(ctypes.c_void_p(FAKE), ctypes.c_void_p(FAKE + 4096), 1000, None) == D.ERR_INVALID_ARG
    assert lib.dartree_calib_copy(None, ctypes.c_void_p(FAKE), 1024, None) == D.ERR_INVALID_ARG
    assert lib.dartree_calib_mfma(0, 10, sink, None) == D.ERR_INVALID_ARG
    assert lib.dartree_calib_empty(0, None) == D.ERR_INVALID_ARG
    assert lib.dartree_calib_empty(D.CALIB_SINK_FLOATS + 1, None) == D.ERR_INVALID_ARG
    cnt = ctypes.c_void_p(FAKE)
    assert lib.dartree_calib_grid_barrier(0, 1, cnt, cnt, None) == D.ERR_INVALID_ARG
    assert lib.dartree_calib_grid_barrier(8, -1, cnt, cnt, None) == D.ERR_INVALID_ARG
    assert lib.dartree_calib_grid_barrier(8, D.CALIB_MAX_BARRIERS + 1, cnt, cnt, None) == D.ERR_INVALID_ARG
    assert lib.dartree_calib_grid_barrier(8, 1, None, cnt, None) == D.ERR_INVALID_ARG
    assert lib.dartree_calib_grid_barrier(8, 1, cnt, None, None) == D.ERR_INVALID_ARG
    assert lib.dartree_calib_mfma(D.CALIB_SINK_FLOATS + 1, 10, sink, None) == D.ERR_INVALID_ARG
    assert lib.dartree_calib_mfma(4, 0, sink, None) == D.ERR_INVALID_ARG
    assert lib.dartree_calib_mfma(4, 10, None, None) == D.ERR_INVALID_ARG


def test_validate_shared_candidate_sets():
    p = D.Params.of(W.CONFIGS["qwen3-4b-shared"])
    assert D.validate(p) == D.OK
    assert D.validate(_p(candidates=-1)) == D.ERR_INVALID_ARG
    assert D.validate(_p(candidates=4, branch=8)) == D.ERR_INVALID_ARG        # k > K
    assert D.validate(_p(candidates=64, branch=64)) == D.OK                   # k may exceed 32 with a shared set
    assert D.validate(_p(candidates=0, branch=64)) == D.ERR_UNSUPPORTED       # not over the full vocabulary
    assert D.validate(_p(candidates=257, branch=8)) == D.ERR_UNSUPPORTED
    small = D.Params.of(W.CONFIGS["tiny"])
    small.candidates = small.vocab + 1
    assert D.validate(small) == D.ERR_INVALID_ARG                              # K > V
    big = _p(candidates=256, branch=8)
    big.vocab = 1 << 20
    assert D.validate(big) == D.OK
    assert D.workspace_size(p) < D.workspace_size(D.Params.of(W.CONFIGS["qwen3-4b"]))   # logits over C_d only


def test_candidate_sets_reject_bad_arguments():
    lib = D.lib()
    n = ctypes.c_size_t(0)
    assert lib.dartree_candidate_sets_workspace_size(4, 100, 0, ctypes.byref(n)) == D.ERR_INVALID_ARG
    assert lib.dartree_candidate_sets_workspace_size(4, 100, 101, ctypes.byref(n)) == D.ERR_INVALID_ARG
    assert lib.dartree_candidate_sets_workspace_size(4, 100000, 257, ctypes.byref(n)) == D.ERR_UNSUPPORTED
    assert lib.dartree_candidate_sets_workspace_size(4, 151936, 64, ctypes.byref(n)) == D.OK
    assert n.value == 4 * 64 * 4               # one maximum per group, K groups per row
    ws = ctypes.c_void_p(FAKE)
    assert lib.dartree_candidate_sets(None, 4, 151936, 64, ctypes.c_void_p(FAKE), ws, n.value, None) == D.ERR_INVALID_ARG
    assert lib.dartree_candidate_sets(ctypes.c_void_p(FAKE), 4, 151936, 64, ctypes.c_void_p(FAKE), ws, n.value - 1,
                                      None) == D.ERR_WORKSPACE


def test_sequential_heap_validation_and_rejects():
    lib = D.lib()
    byref = ctypes.byref
    for name in W.CONFIG_ORDER:
        cfg = W.CONFIGS[name]
        if cfg.budget <= D.MAX_HEAP_BUDGET:
            assert D.heap_workspace_size(D.Params.of(cfg)) > 0, name
    p = _p(width=0)                                  # the width is not used by the heap
    n = D.heap_workspace_size(p)
    b, B, h, V = p.batch, p.budget, p.hidden, p.vocab
    assert n >= (B + 1) * b * h * 2 + B * b * h * 4 + b * V * 4   # states, t per slot, one row of logits
    assert n % 256 == 0
    with pytest.raises(D.DartreeError) as e:
        D.heap_workspace_size(_p(budget=D.MAX_HEAP_BUDGET + 1))
    assert e.value.status == D.ERR_UNSUPPORTED
    with pytest.raises(D.DartreeError) as e:
        D.heap_workspace_size(_p(depth_bonus=0.5))
    assert e.value.status == D.ERR_INVALID_ARG
    assert D.heap_workspace_size(_p(candidates=64, branch=64)) < n          # logits over C_d only
    assert lib.dartree_build_tree_heap(byref(p), byref(_inputs()), FAKE, n - 1, byref(_tree()), None) == D.ERR_WORKSPACE
    assert lib.dartree_build_tree_heap(byref(p), byref(_inputs()), FAKE + 16, n, byref(_tree()), None) == D.ERR_WORKSPACE
    bad_in = D.InputsC(FAKE, None, FAKE, FAKE, FAKE)
    assert lib.dartree_build_tree_heap(byref(p), byref(bad_in), FAKE, n, byref(_tree()), None) == D.ERR_INVALID_ARG
    bad_tree = D.TreeC(FAKE, FAKE, FAKE + 8, FAKE, FAKE, FAKE)
    assert lib.dartree_build_tree_heap(byref(p), byref(_inputs()), FAKE, n, byref(bad_tree), None) == D.ERR_INVALID_ARG
    assert lib.dartree_build_tree_heap(byref(_p(batch=0)), byref(_inputs()), FAKE, n, byref(_tree()),
                                       None) == D.ERR_INVALID_ARG
    assert lib.dartree_export_heap(byref(p), FAKE, n, None, None) == D.ERR_INVALID_ARG
    assert lib.dartree_export_heap(byref(p), FAKE, n - 1, byref(D.HeapTraceC()), None) == D.ERR_WORKSPACE


def test_consumer_rejects_bad_arguments():
    lib = D.lib()
    F = ctypes.c_void_p(FAKE)
    args = [F] * 7
    assert lib.dartree_accept_walk(0, 8, 4, *args, None) == D.ERR_INVALID_ARG
    assert lib.dartree_accept_walk(1, 8, 0, *args, None) == D.ERR_INVALID_ARG
    assert lib.dartree_accept_walk(1, 4097, 4, *args, None) == D.ERR_UNSUPPORTED
    assert lib.dartree_accept_walk(1, 8, 4, F, F, F, None, F, F, F, None) == D.ERR_INVALID_ARG
    p = D.AttnParams(batch=1, budget=64, max_ctx=2048, heads_q=32, heads_kv=8, head_dim=128, scale=0.0884)
    n = D.tree_attention_workspace_size(p)
    assert n >= 9 * 8 * 256 * 128 * 4          # one partial row per segment, kv head and query row
    edge = D.AttnParams(1, 64, 1023 * 256, 4, 1, 128, 0.0884)
    assert D.tree_attention_workspace_size(edge) > 0   # 1023 context segments + the tree: the limit
    # >= 512 (request, kv head, 64-row tile) blocks: every block covers all keys, no workspace
    assert D.tree_attention_workspace_size(D.AttnParams(16, 64, 2048, 32, 8, 128, 0.0884)) == 0   # 16*8*4
    assert D.tree_attention_workspace_size(D.AttnParams(15, 64, 2048, 32, 8, 128, 0.0884)) > 0    # 480
    for field, value, code in (("head_dim", 64, D.ERR_UNSUPPORTED), ("heads_q", 30, D.ERR_INVALID_ARG),
                               ("scale", 0.0, D.ERR_INVALID_ARG), ("budget", 0, D.ERR_INVALID_ARG),
                               ("max_ctx", -1, D.ERR_INVALID_ARG), ("budget", 4097, D.ERR_UNSUPPORTED),
                               ("max_ctx", 1023 * 256 + 1, D.ERR_UNSUPPORTED)):
        bad = D.AttnParams(1, 64, 2048, 32, 8, 128, 0.0884)
        setattr(bad, field, value)
        with pytest.raises(D.DartreeError) as e:
            D.tree_attention_workspace_size(bad)
        assert e.value.status == code, field
    call = lambda ws, nbytes, q=F, kc=F: lib.dartree_tree_attention(ctypes.byref(p), q, kc, F, F, F, F, None, F, ws,
                                                                    nbytes, None)
    assert call(F, n - 1) == D.ERR_WORKSPACE
    assert call(ctypes.c_void_p(FAKE + 16), n) == D.ERR_WORKSPACE
    assert call(F, n, q=None) == D.ERR_INVALID_ARG
    assert call(F, n, kc=None) == D.ERR_INVALID_ARG                 # context expected
    assert call(F, n, q=ctypes.c_void_p(FAKE + 2)) == D.ERR_INVALID_ARG


def test_depth_order_checked_before_any_launch():
    """Algorithm 1's depths run 1..L: a call that would read levels no earlier
    call produced returns DARTREE_ERR_ORDER with nothing enqueued (on a
    workspace address the library has never seen)."""
    lib = D.lib()
    p = _p()
    need = D.workspace_size(p)
    byref = ctypes.byref
    fresh = 0x7A000000   # never used as a workspace in this process
    assert D.status_string(D.ERR_ORDER) and D.status_string(D.ERR_NONFINITE)
    for d in (2, 5, 16):
        assert lib.dartree_expand_depth(byref(p), byref(_inputs()), d, fresh, need, None) == D.ERR_ORDER
    assert lib.dartree_prune(byref(p), fresh, need, byref(_tree()), None) == D.ERR_ORDER
    assert lib.dartree_export_states(byref(p), fresh, need, 3, FAKE, None) == D.ERR_ORDER
    assert lib.dartree_export_features(byref(p), fresh, need, 1, FAKE, None) == D.ERR_ORDER
    assert lib.dartree_export_supertree(byref(p), fresh, need, byref(D.SupertreeC()), None) == D.ERR_ORDER
    # argument errors still come first
    assert lib.dartree_export_features(byref(p), fresh, need, 0, FAKE, None) == D.ERR_INVALID_ARG
    assert lib.dartree_export_features(byref(p), fresh, need, 17, FAKE, None) == D.ERR_INVALID_ARG
    assert lib.dartree_export_features(byref(p), fresh, need - 1, 1, FAKE, None) == D.ERR_WORKSPACE
    assert lib.dartree_expand_depth(byref(p), byref(_inputs()), 2, fresh, need - 1, None) == D.ERR_WORKSPACE
