"""ctypes binding of libdartree (the C ABI in include/dartree.h).

Argument marshalling only: every step of tree construction runs in the HIP
kernels of ``libdartree.so``.  PyTorch supplies device memory and the stream.
If the library has not been built, :func:`lib` raises; there is no fallback.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Optional

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libdartree.so")

FP32 = 0
BF16 = 1
HEAD_RNN = 0
HEAD_MARKOV = 1

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP, ERR_ORDER, ERR_NONFINITE = range(7)

ABI_VERSION = 8   # DARTREE_ABI_VERSION of include/dartree.h this binding follows

MAX_VOCAB = 1 << 20
MAX_DEPTH = 64
MAX_WIDTH = 2048
MAX_BRANCH = 32
MAX_CANDIDATES = 256
MAX_SORT = 4096
MAX_HEAP_BUDGET = 1024
LSE_TOPK_STATIC_SCRATCH_BYTES = 576 * 1024

SYMBOLS = [
    "dartree_abi_version", "dartree_status_string", "dartree_validate",
    "dartree_workspace_size", "dartree_expand_depth", "dartree_prune",
    "dartree_build_tree", "dartree_build_tree_timed", "dartree_export_supertree", "dartree_export_states",
    "dartree_export_features", "dartree_project",
    "dartree_project_workspace_size",
    "dartree_lse_topk_workspace_size", "dartree_lse_topk", "dartree_lse_topk_noalloc", "dartree_select_topw",
    "dartree_prune_levels", "dartree_candidate_sets_workspace_size", "dartree_candidate_sets",
    "dartree_heap_workspace_size", "dartree_build_tree_heap", "dartree_export_heap",
    "dartree_accept_walk", "dartree_tree_attention_workspace_size", "dartree_tree_attention",
    "dartree_calib_read", "dartree_calib_copy", "dartree_calib_mfma", "dartree_calib_empty",
    "dartree_calib_grid_barrier",
]
CALIB_MAX_BARRIERS = 64
CALIB_SINK_FLOATS = 4096


class Params(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("vocab", ctypes.c_int32), ("hidden", ctypes.c_int32),
                ("depth", ctypes.c_int32), ("width", ctypes.c_int32), ("branch", ctypes.c_int32),
                ("budget", ctypes.c_int32), ("precision", ctypes.c_int32),
                ("temperature", ctypes.c_float), ("depth_bonus", ctypes.c_float),
                ("candidates", ctypes.c_int32), ("head", ctypes.c_int32)]

    @staticmethod
    def of(cfg) -> "Params":
        return Params(cfg.batch, cfg.vocab, cfg.hidden, cfg.depth, cfg.width, cfg.branch,
                      cfg.budget, cfg.precision, float(cfg.temperature), float(cfg.depth_bonus),
                      int(getattr(cfg, "candidates", 0)), int(getattr(cfg, "head", HEAD_RNN)))

    def level_sizes(self) -> list[int]:
        n, out = 1, []
        for _ in range(self.depth):
            n = min(self.width, n * self.branch)
            out.append(n)
        return out


class InputsC(ctypes.Structure):
    _fields_ = [("drafter_logits", ctypes.c_void_p), ("drafter_hidden", ctypes.c_void_p),
                ("prefix_state", ctypes.c_void_p), ("head_A", ctypes.c_void_p),
                ("head_U", ctypes.c_void_p)]


class TreeC(ctypes.Structure):
    _fields_ = [("tokens", ctypes.c_void_p), ("parents", ctypes.c_void_p), ("depths", ctypes.c_void_p),
                ("scores", ctypes.c_void_p), ("mask", ctypes.c_void_p), ("num_nodes", ctypes.c_void_p)]


class SupertreeC(ctypes.Structure):
    _fields_ = [("tokens", ctypes.c_void_p), ("parents", ctypes.c_void_p), ("scores", ctypes.c_void_p),
                ("lse", ctypes.c_void_p), ("cand_logp", ctypes.c_void_p), ("cand_ids", ctypes.c_void_p),
                ("csets", ctypes.c_void_p)]


class HeapTraceC(ctypes.Structure):
    _fields_ = [("tokens", ctypes.c_void_p), ("parents", ctypes.c_void_p), ("depths", ctypes.c_void_p),
                ("scores", ctypes.c_void_p), ("num_popped", ctypes.c_void_p), ("lse", ctypes.c_void_p),
                ("cand_logp", ctypes.c_void_p), ("cand_ids", ctypes.c_void_p), ("states", ctypes.c_void_p),
                ("csets", ctypes.c_void_p), ("features", ctypes.c_void_p)]


class AttnParams(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("budget", ctypes.c_int32), ("max_ctx", ctypes.c_int32),
                ("heads_q", ctypes.c_int32), ("heads_kv", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("scale", ctypes.c_float)]


class DartreeError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} (status {status})")


_lib: Optional[ctypes.CDLL] = None


def lib() -> ctypes.CDLL:
    """The loaded HIP library.  Raises if it is missing: build it first with
    ``python -m paper_2608_13524_amd.build``."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: the HIP library must be built "
                           "(python -m paper_2608_13524_amd.build); there is no fallback path")
    L = ctypes.CDLL(LIB_PATH)
    P, vp, i32, i64, f32, sz = (ctypes.POINTER(Params), ctypes.c_void_p, ctypes.c_int32,
                                ctypes.c_int64, ctypes.c_float, ctypes.c_size_t)
    L.dartree_abi_version.restype = i32
    L.dartree_abi_version.argtypes = []
    L.dartree_status_string.restype = ctypes.c_char_p
    L.dartree_status_string.argtypes = [ctypes.c_int]
    L.dartree_validate.argtypes = [P]
    L.dartree_workspace_size.argtypes = [P, ctypes.POINTER(sz)]
    L.dartree_expand_depth.argtypes = [P, ctypes.POINTER(InputsC), i32, vp, sz, vp]
    L.dartree_prune.argtypes = [P, vp, sz, ctypes.POINTER(TreeC), vp]
    L.dartree_build_tree.argtypes = [P, ctypes.POINTER(InputsC), vp, sz, ctypes.POINTER(TreeC), vp]
    L.dartree_build_tree_timed.argtypes = [P, ctypes.POINTER(InputsC), vp, sz, ctypes.POINTER(TreeC),
                                           ctypes.POINTER(vp), vp]
    L.dartree_export_supertree.argtypes = [P, vp, sz, ctypes.POINTER(SupertreeC), vp]
    L.dartree_export_states.argtypes = [P, vp, sz, i32, vp, vp]
    L.dartree_export_features.argtypes = [P, vp, sz, i32, vp, vp]
    L.dartree_project.argtypes = [i32, i32, i32, i32, i32, vp, vp, vp, i64, vp, vp, sz, vp]
    L.dartree_project_workspace_size.argtypes = [i32, i32, i32, i32, ctypes.POINTER(sz)]
    L.dartree_lse_topk_workspace_size.argtypes = [i32, i32, i32, ctypes.POINTER(sz)]
    L.dartree_lse_topk.argtypes = [vp, i32, i32, i32, f32, vp, vp, vp, vp, sz, vp]
    L.dartree_lse_topk_noalloc.argtypes = [vp, i32, i32, i32, f32, vp, vp, vp, vp]
    L.dartree_select_topw.argtypes = [i32, i32, i32, i32, f32, vp, vp, vp, vp, vp, vp, vp]
    L.dartree_prune_levels.argtypes = [P, vp, vp, vp, ctypes.POINTER(TreeC), vp]
    L.dartree_candidate_sets_workspace_size.argtypes = [i32, i32, i32, ctypes.POINTER(sz)]
    L.dartree_candidate_sets.argtypes = [vp, i32, i32, i32, vp, vp, sz, vp]
    L.dartree_heap_workspace_size.argtypes = [P, ctypes.POINTER(sz)]
    L.dartree_build_tree_heap.argtypes = [P, ctypes.POINTER(InputsC), vp, sz, ctypes.POINTER(TreeC), vp]
    L.dartree_export_heap.argtypes = [P, vp, sz, ctypes.POINTER(HeapTraceC), vp]
    L.dartree_accept_walk.argtypes = [i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp]
    L.dartree_tree_attention_workspace_size.argtypes = [ctypes.POINTER(AttnParams), ctypes.POINTER(sz)]
    L.dartree_tree_attention.argtypes = [ctypes.POINTER(AttnParams), vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    L.dartree_calib_read.argtypes = [vp, sz, vp, vp]
    L.dartree_calib_copy.argtypes = [vp, vp, sz, vp]
    L.dartree_calib_mfma.argtypes = [i32, i32, vp, vp]
    L.dartree_calib_empty.argtypes = [i32, vp]
    L.dartree_calib_grid_barrier.argtypes = [i32, i32, vp, vp, vp]
    for name in SYMBOLS:
        if name not in ("dartree_abi_version", "dartree_status_string"):
            getattr(L, name).restype = ctypes.c_int
    _lib = L
    return L


def status_string(status: int) -> str:
    return lib().dartree_status_string(int(status)).decode()


def _check(status: int, where: str) -> None:
    if status != OK:
        raise DartreeError(status, where)


def _ptr(t) -> Optional[int]:
    """Device address of a tensor (None for None)."""
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


# ---------------------------------------------------------------------------
# Host-only calls
# ---------------------------------------------------------------------------

def abi_version() -> int:
    return lib().dartree_abi_version()


def validate(p: Params) -> int:
    return lib().dartree_validate(None if p is None else ctypes.byref(p))


def workspace_size(p: Params) -> int:
    n = ctypes.c_size_t(0)
    _check(lib().dartree_workspace_size(ctypes.byref(p), ctypes.byref(n)), "dartree_workspace_size")
    return n.value


def heap_workspace_size(p: Params) -> int:
    n = ctypes.c_size_t(0)
    _check(lib().dartree_heap_workspace_size(ctypes.byref(p), ctypes.byref(n)), "dartree_heap_workspace_size")
    return n.value


def lse_topk_workspace_size(rows: int, vocab: int, k: int) -> int:
    n = ctypes.c_size_t(0)
    _check(lib().dartree_lse_topk_workspace_size(rows, vocab, k, ctypes.byref(n)),
           "dartree_lse_topk_workspace_size")
    return n.value


# ---------------------------------------------------------------------------
# Device buffers (torch allocations: plumbing only)
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class DeviceInputs:
    Lb: object
    H: object
    r0: object
    A: object
    U: object

    def c(self) -> InputsC:
        return InputsC(_ptr(self.Lb), _ptr(self.H), _ptr(self.r0), _ptr(self.A), _ptr(self.U))

    @staticmethod
    def from_host(inputs, device="cuda") -> "DeviceInputs":
        """Copy host inputs (numpy; bf16 given as uint16 bit patterns) to the device."""
        import numpy as np
        import torch

        def dev(x):
            x = np.ascontiguousarray(x)
            if x.dtype == np.uint16:
                x = x.view(np.int16)
            return torch.from_numpy(x).to(device)

        return DeviceInputs(dev(inputs.Lb), dev(inputs.H), dev(inputs.r0), dev(inputs.A), dev(inputs.U))


@dataclasses.dataclass
class DeviceTree:
    tokens: object
    parents: object
    depths: object
    scores: object
    mask: object
    num_nodes: object

    def c(self) -> TreeC:
        return TreeC(_ptr(self.tokens), _ptr(self.parents), _ptr(self.depths), _ptr(self.scores),
                     _ptr(self.mask), _ptr(self.num_nodes))

    @staticmethod
    def alloc(batch: int, budget: int, device="cuda") -> "DeviceTree":
        import torch
        words = (budget + 63) // 64
        i32 = dict(dtype=torch.int32, device=device)
        return DeviceTree(torch.empty(batch, budget, **i32), torch.empty(batch, budget, **i32),
                          torch.empty(batch, budget, **i32),
                          torch.empty(batch, budget, dtype=torch.float32, device=device),
                          torch.empty(batch, budget, words, dtype=torch.int64, device=device),
                          torch.empty(batch, **i32))

    def host(self) -> dict:
        """Numpy copies (mask as uint64)."""
        import numpy as np
        out = {f.name: getattr(self, f.name).cpu().numpy() for f in dataclasses.fields(self)}
        out["mask"] = out["mask"].view(np.uint64)
        return out


@dataclasses.dataclass
class DeviceSupertree:
    tokens: object
    parents: object
    scores: object
    lse: object
    cand_logp: object
    cand_ids: object
    csets: object = None   # [b][L][K] shared candidate sets (candidates > 0)

    def c(self) -> SupertreeC:
        return SupertreeC(*(_ptr(getattr(self, f.name)) for f in dataclasses.fields(self)))

    @staticmethod
    def alloc(p: Params, device="cuda") -> "DeviceSupertree":
        import torch
        L, b, W, k = p.depth, p.batch, p.width, p.branch
        i32 = dict(dtype=torch.int32, device=device)
        f32 = dict(dtype=torch.float32, device=device)
        K = p.candidates
        return DeviceSupertree(torch.empty(L, b, W, **i32), torch.empty(L, b, W, **i32),
                               torch.empty(L, b, W, **f32), torch.empty(L, b * W, **f32),
                               torch.empty(L, b * W, k, **f32), torch.empty(L, b * W, k, **i32),
                               torch.empty(b, L, K, **i32) if K > 0 else None)

    def host(self) -> dict:
        return {f.name: getattr(self, f.name).cpu().numpy() for f in dataclasses.fields(self)
                if getattr(self, f.name) is not None}


@dataclasses.dataclass
class DeviceHeapTrace:
    tokens: object
    parents: object
    depths: object
    scores: object
    num_popped: object
    lse: object
    cand_logp: object
    cand_ids: object
    states: object = None   # act [B+1][b][h] (int16 bit patterns in bf16 mode)
    csets: object = None    # [b][L][K] (candidates > 0)
    features: object = None  # act [B][b][h]

    def c(self) -> HeapTraceC:
        return HeapTraceC(*(_ptr(getattr(self, f.name)) for f in dataclasses.fields(self)))

    @staticmethod
    def alloc(p: Params, states: bool = True, device="cuda") -> "DeviceHeapTrace":
        """``states``: also the per-slot states and per-step features."""
        import torch
        b, B, k, h, L, K = p.batch, p.budget, p.branch, p.hidden, p.depth, p.candidates
        i32 = dict(dtype=torch.int32, device=device)
        f32 = dict(dtype=torch.float32, device=device)
        act = torch.int16 if p.precision == BF16 else torch.float32
        return DeviceHeapTrace(torch.empty(b, B + 1, **i32), torch.empty(b, B + 1, **i32),
                               torch.empty(b, B + 1, **i32), torch.empty(b, B + 1, **f32), torch.empty(b, **i32),
                               torch.empty(B, b, **f32), torch.empty(B, b, k, **f32), torch.empty(B, b, k, **i32),
                               torch.empty(B + 1, b, h, dtype=act, device=device) if states else None,
                               torch.empty(b, L, K, **i32) if K > 0 else None,
                               torch.empty(B, b, h, dtype=act, device=device) if states else None)

    def host(self) -> dict:
        return {f.name: getattr(self, f.name).cpu().numpy() for f in dataclasses.fields(self)
                if getattr(self, f.name) is not None}


def alloc_workspace(p: Params, device="cuda"):
    import torch
    # torch's caching allocator returns blocks aligned to at least 512 bytes
    return torch.empty(max(workspace_size(p), 1), dtype=torch.uint8, device=device)


def alloc_heap_workspace(p: Params, device="cuda"):
    import torch
    return torch.empty(max(heap_workspace_size(p), 1), dtype=torch.uint8, device=device)


# ---------------------------------------------------------------------------
# Device calls (enqueued on `stream`, default: torch's current stream)
# ---------------------------------------------------------------------------

def build_tree(p: Params, inputs: DeviceInputs, ws, out: DeviceTree, stream=None) -> None:
    ic, tc = inputs.c(), out.c()
    _check(lib().dartree_build_tree(ctypes.byref(p), ctypes.byref(ic), _ptr(ws), ws.numel(),
                                    ctypes.byref(tc), _stream(stream)), "dartree_build_tree")


def build_tree_heap(p: Params, inputs: DeviceInputs, ws, out: DeviceTree, stream=None) -> None:
    """Sequential correction with a best-first heap (the node-at-a-time baseline)."""
    ic, tc = inputs.c(), out.c()
    _check(lib().dartree_build_tree_heap(ctypes.byref(p), ctypes.byref(ic), _ptr(ws), ws.numel(),
                                         ctypes.byref(tc), _stream(stream)), "dartree_build_tree_heap")


def export_heap(p: Params, ws, dst: DeviceHeapTrace, stream=None) -> None:
    hc = dst.c()
    _check(lib().dartree_export_heap(ctypes.byref(p), _ptr(ws), ws.numel(), ctypes.byref(hc), _stream(stream)),
           "dartree_export_heap")


KERNEL_NAMES = ["head", "logits", "lse_topk", "select"]   # per depth, launch order


def build_tree_timed(p: Params, inputs: DeviceInputs, ws, out: DeviceTree, events, stream=None) -> None:
    """build_tree recording ``events`` (2 * (4 L + 1) raw hipEvent_t handles or
    None) around each launch; see dartree_build_tree_timed."""
    ic, tc = inputs.c(), out.c()
    n = 2 * (len(KERNEL_NAMES) * p.depth + 1)
    assert len(events) == n
    arr = (ctypes.c_void_p * n)(*events)
    _check(lib().dartree_build_tree_timed(ctypes.byref(p), ctypes.byref(ic), _ptr(ws), ws.numel(),
                                          ctypes.byref(tc), arr, _stream(stream)), "dartree_build_tree_timed")


def expand_depth(p: Params, inputs: DeviceInputs, d: int, ws, stream=None) -> None:
    ic = inputs.c()
    _check(lib().dartree_expand_depth(ctypes.byref(p), ctypes.byref(ic), d, _ptr(ws), ws.numel(),
                                      _stream(stream)), "dartree_expand_depth")


def prune(p: Params, ws, out: DeviceTree, stream=None) -> None:
    tc = out.c()
    _check(lib().dartree_prune(ctypes.byref(p), _ptr(ws), ws.numel(), ctypes.byref(tc), _stream(stream)),
           "dartree_prune")


def export_supertree(p: Params, ws, dst: DeviceSupertree, stream=None) -> None:
    sc = dst.c()
    _check(lib().dartree_export_supertree(ctypes.byref(p), _ptr(ws), ws.numel(), ctypes.byref(sc),
                                          _stream(stream)), "dartree_export_supertree")


def export_states(p: Params, ws, d: int, dst, stream=None) -> None:
    """States of S_d into dst (act [b * n_d][h]); see the header for validity."""
    _check(lib().dartree_export_states(ctypes.byref(p), _ptr(ws), ws.numel(), d, _ptr(dst), _stream(stream)),
           "dartree_export_states")


def export_features(p: Params, ws, d: int, dst, stream=None) -> None:
    """Features of depth d's parent rows into dst (act [b * n_{d-1}][h]),
    right after expand_depth(d)."""
    _check(lib().dartree_export_features(ctypes.byref(p), _ptr(ws), ws.numel(), d, _ptr(dst), _stream(stream)),
           "dartree_export_features")


def project_workspace_size(precision: int, rows: int, vocab: int, hidden: int) -> int:
    n = ctypes.c_size_t(0)
    _check(lib().dartree_project_workspace_size(precision, rows, vocab, hidden, ctypes.byref(n)),
           "dartree_project_workspace_size")
    return n.value


def project(precision: int, x, U, bias, bias_stride: int, z, rows_per_group: int, ws=None, stream=None) -> None:
    rows, hidden = x.shape
    vocab = U.shape[0]
    _check(lib().dartree_project(precision, rows, vocab, hidden, rows_per_group, _ptr(x), _ptr(U), _ptr(bias),
                                 bias_stride, _ptr(z), _ptr(ws), 0 if ws is None else ws.numel(), _stream(stream)),
           "dartree_project")


def lse_topk(z, k: int, temperature: float, lse, cand_logp, cand_ids, ws=None, stream=None) -> None:
    rows, vocab = z.shape
    _check(lib().dartree_lse_topk(_ptr(z), rows, vocab, k, temperature, _ptr(lse), _ptr(cand_logp),
                                  _ptr(cand_ids), _ptr(ws), 0 if ws is None else ws.numel(), _stream(stream)),
           "dartree_lse_topk")


def lse_topk_noalloc(z, k: int, temperature: float, lse, cand_logp, cand_ids, stream=None) -> None:
    """lse_topk with the library's static scratch (no workspace, nothing allocated)."""
    rows, vocab = z.shape
    _check(lib().dartree_lse_topk_noalloc(_ptr(z), rows, vocab, k, temperature, _ptr(lse), _ptr(cand_logp),
                                          _ptr(cand_ids), _stream(stream)), "dartree_lse_topk_noalloc")


def select_topw(batch: int, n_parent: int, k: int, n_keep: int, depth_bonus: float, parent_score,
                cand_logp, cand_ids, out_tokens, out_parents, out_scores, stream=None) -> None:
    _check(lib().dartree_select_topw(batch, n_parent, k, n_keep, depth_bonus, _ptr(parent_score),
                                     _ptr(cand_logp), _ptr(cand_ids), _ptr(out_tokens), _ptr(out_parents),
                                     _ptr(out_scores), _stream(stream)), "dartree_select_topw")


def prune_levels(p: Params, tokens, parents, scores, out: DeviceTree, stream=None) -> None:
    tc = out.c()
    _check(lib().dartree_prune_levels(ctypes.byref(p), _ptr(tokens), _ptr(parents), _ptr(scores),
                                      ctypes.byref(tc), _stream(stream)), "dartree_prune_levels")


# ---------------------------------------------------------------------------
# Calibration kernels (achievable ceilings; they compute nothing of the method)
def calib_read(src, sink, stream=None) -> None:
    """Stream src (any contiguous device tensor, size a multiple of 16 bytes) once."""
    nbytes = src.numel() * src.element_size()
    _check(lib().dartree_calib_read(_ptr(src), nbytes, _ptr(sink), _stream(stream)), "dartree_calib_read")


def calib_copy(dst, src, stream=None) -> None:
    nbytes = src.numel() * src.element_size()
    assert dst.numel() * dst.element_size() >= nbytes
    _check(lib().dartree_calib_copy(_ptr(dst), _ptr(src), nbytes, _stream(stream)), "dartree_calib_copy")


def calib_mfma(blocks: int, iters: int, sink, stream=None) -> float:
    """Launch the MFMA-only loop; returns its flop count."""
    _check(lib().dartree_calib_mfma(blocks, iters, _ptr(sink), _stream(stream)), "dartree_calib_mfma")
    return float(blocks) * 4 * iters * 64 * (2 * 16 * 16 * 32)


def calib_empty(blocks: int, stream=None) -> None:
    """One launch of `blocks` workgroups that does nothing."""
    _check(lib().dartree_calib_empty(blocks, _stream(stream)), "dartree_calib_empty")


def calib_grid_barrier(blocks: int, nbar: int, counters, fail, stream=None) -> None:
    """One launch passing `nbar` grid-wide barriers (counters: >= nbar zeroed
    int32 words on the device; fail: one int32 word set to 1 if a wait gave up)."""
    _check(lib().dartree_calib_grid_barrier(blocks, nbar, _ptr(counters) if nbar else None, _ptr(fail),
                                            _stream(stream)), "dartree_calib_grid_barrier")


def candidate_sets(logits, K: int, ids, ws=None, stream=None) -> None:
    """Shared candidate sets: ids [rows][K] = TopK of each fp32 row by (value desc, id asc)."""
    rows, vocab = logits.shape
    _check(lib().dartree_candidate_sets(_ptr(logits), rows, vocab, K, _ptr(ids), _ptr(ws),
                                        0 if ws is None else ws.numel(), _stream(stream)),
           "dartree_candidate_sets")


def candidate_sets_workspace_size(rows: int, vocab: int, K: int) -> int:
    n = ctypes.c_size_t(0)
    _check(lib().dartree_candidate_sets_workspace_size(rows, vocab, K, ctypes.byref(n)),
           "dartree_candidate_sets_workspace_size")
    return n.value


# ---------------------------------------------------------------------------
# The consumer of the emitted tree
# ---------------------------------------------------------------------------
def accept_walk(tokens, parents, num_nodes, target, accepted, num_accepted, bonus, stream=None) -> None:
    """tokens, parents [b][B] and num_nodes [b] of emitted trees, target [b][B+1];
    outputs accepted [b][max_len], num_accepted [b], bonus [b] (int32 device)."""
    batch, budget = tokens.shape
    _check(lib().dartree_accept_walk(batch, budget, accepted.shape[1], _ptr(tokens), _ptr(parents), _ptr(num_nodes),
                                     _ptr(target), _ptr(accepted), _ptr(num_accepted), _ptr(bonus),
                                     _stream(stream)), "dartree_accept_walk")


def tree_attention_workspace_size(p: AttnParams) -> int:
    n = ctypes.c_size_t(0)
    _check(lib().dartree_tree_attention_workspace_size(ctypes.byref(p), ctypes.byref(n)),
           "dartree_tree_attention_workspace_size")
    return n.value


def tree_attention(p: AttnParams, q, k_ctx, v_ctx, k_tree, v_tree, mask, ctx_len, out, ws, stream=None) -> None:
    _check(lib().dartree_tree_attention(ctypes.byref(p), _ptr(q), _ptr(k_ctx), _ptr(v_ctx), _ptr(k_tree),
                                        _ptr(v_tree), _ptr(mask), _ptr(ctx_len), _ptr(out), _ptr(ws),
                                        0 if ws is None else ws.numel(), _stream(stream)), "dartree_tree_attention")
