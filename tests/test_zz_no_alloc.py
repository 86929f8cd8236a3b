"""dartree_lse_topk_noalloc (the softmax/top-k pass with the library's static
scratch, for callers that cannot allocate) against dartree_lse_topk with a
caller workspace, through the C ABI: identical bits on consecutive calls, each
smaller than the one before, so stale records of a larger call sit in the
shared scratch."""
import numpy as np
import pytest
import torch

from paper_2608_13524_amd import dartree as D
from tests.gpu_util import device, say

pytestmark = pytest.mark.gpu

# rows, vocab, k, T: the largest split any call can make (1023 rows x 2 segments
# of 68-float records: 556784 bytes), then smaller splits, then no split
CALLS = [(1023, 151936, 32, 1.0), (8, 151936, 8, 0.0), (3, 50003, 5, 0.7), (2, 1001, 3, 1.0)]


def _run(fn, z, k, T, ws=None):
    rows = z.shape[0]
    dev = z.device
    lse = torch.full((rows,), -7.0, dtype=torch.float32, device=dev)
    lp = torch.full((rows, k), -7.0, dtype=torch.float32, device=dev)
    ids = torch.full((rows, k), -7, dtype=torch.int32, device=dev)
    if ws is None:
        fn(z, k, T, lse, lp, ids)
    else:
        fn(z, k, T, lse, lp, ids, ws)
    torch.cuda.synchronize()
    return lse.cpu().numpy(), lp.cpu().numpy(), ids.cpu().numpy()


def test_noalloc_matches_workspace_version():
    dev = device()
    rows, vocab, k, _ = CALLS[0]
    assert D.lse_topk_workspace_size(rows, vocab, k) <= D.LSE_TOPK_STATIC_SCRATCH_BYTES
    for rows, vocab, k, T in CALLS:
        rng = np.random.default_rng(rows * 31 + vocab + k)
        z = torch.from_numpy(rng.normal(0, 2, size=(rows, vocab)).astype(np.float32)).to(dev)
        need = D.lse_topk_workspace_size(rows, vocab, k)
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
        say(f"lse_topk_noalloc rows={rows} vocab={vocab} k={k} T={T} scratch={need}")
        want = _run(D.lse_topk, z, k, T, ws)
        got = _run(D.lse_topk_noalloc, z, k, T)
        for w, g in zip(want, got):
            assert np.array_equal(w, g)
        assert (got[2] >= 0).all() and (got[2] < vocab).all()
        del z, ws
        torch.cuda.empty_cache()


def test_noalloc_rejects_bad_arguments():
    lib = D.lib()
    fake = 0x10000
    assert lib.dartree_lse_topk_noalloc(fake, 4, 100, 101, 1.0, fake, fake, fake, None) == D.ERR_INVALID_ARG
    assert lib.dartree_lse_topk_noalloc(fake, 4, 100, 4, -1.0, fake, fake, fake, None) == D.ERR_INVALID_ARG
    assert lib.dartree_lse_topk_noalloc(None, 4, 100, 4, 1.0, fake, fake, fake, None) == D.ERR_INVALID_ARG
    assert lib.dartree_lse_topk_noalloc(fake, 4, 100, 33, 1.0, fake, fake, fake, None) == D.ERR_UNSUPPORTED
