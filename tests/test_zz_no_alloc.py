"""kv_evict_topk_indexed_noalloc (the eviction step over a slot-indexed cache
with the library's fixed scratch instead of a workspace, for callers that
cannot allocate) against kv_evict_topk_indexed with a workspace: two calls
in a row on the same GPU, the second on a smaller cache, then a cache with
broken invariants; every output bit for bit, the outcome word through the
caller's buffer."""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import DEV

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ds():
    import paper_2609_27470_amd as ds
    ds.lib()
    return ds


def _tables(chunk, pos, capacity, seed):
    n = len(chunk)
    rng = np.random.default_rng(seed)
    slot = rng.permutation(capacity)[:n].astype(np.int32)
    out = []
    for a in (np.asarray(pos, np.int32), np.asarray(chunk, np.int32), slot):
        t = torch.full((capacity,), -7, dtype=torch.int32, device=DEV)
        t[:n] = torch.as_tensor(a, device=DEV)
        out.append(t)
    return out


def _both(ds, chunk, pos, scores, M, ns, nw, nb, capacity, seed):
    """Run the workspace entry point and the one without on equal copies;
    return both results and the oracle's keep list."""
    n = len(chunk)
    sc = torch.as_tensor(scores, device=DEV)
    a = _tables(chunk, pos, capacity, seed)
    b = [t.clone() for t in a]
    keep_a = torch.full((M,), -1, dtype=torch.int32, device=DEV)
    keep_b = keep_a.clone()
    free_a = torch.full((n - M,), -1, dtype=torch.int32, device=DEV)
    free_b = free_a.clone()
    outcome = torch.full((1,), -5, dtype=torch.int32, device=DEV)
    la, ws, _ = ds.kv_evict_topk_indexed(*a, sc, n, M, ns, nw, nb, keep_out=keep_a, free_out=free_a)
    lb = ds.kv_evict_topk_indexed_noalloc(*b, sc, n, M, ns, nw, nb, keep_out=keep_b, free_out=free_b,
                                          outcome=outcome)
    torch.cuda.synchronize()
    return dict(la=la, lb=lb, a=a, b=b, keep_a=keep_a, keep_b=keep_b, free_a=free_a, free_b=free_b,
                outcome=int(outcome.item()), status_a=ds.kv_device_status(ws)[0])


def _check_equal(r, M):
    assert r["la"] == r["lb"] == M
    assert r["outcome"] == 0 and r["status_a"] == 0
    assert torch.equal(r["keep_a"], r["keep_b"])
    assert torch.equal(r["free_a"], r["free_b"])
    for ta, tb in zip(r["a"], r["b"]):
        assert torch.equal(ta[:M], tb[:M])


def test_noalloc_matches_workspace_entry_two_calls(ds):
    # call 1: the eviction-loop cache (17 chunks of 1024 tokens -> 16384, capacity 17408)
    rng = np.random.default_rng(31)
    chunk = np.repeat(np.arange(17), 1024).astype(np.int32)
    pos = (np.arange(17 * 1024) + 5000).astype(np.int32)
    scores = rng.random(17).astype(np.float32)
    r = _both(ds, chunk, pos, scores, 16384, 0, 0, 1, 17408, seed=1)
    _check_equal(r, 16384)
    ref = oracle.select_keep(chunk, pos, scores, len(chunk), 16384, 0, 0, 1)
    assert r["keep_b"].cpu().tolist() == ref
    # call 2, smaller: 60 chunks of 40-90 tokens, the paper's policy with spans
    lens = rng.integers(40, 91, 60)
    chunk2 = np.repeat(np.arange(60), lens).astype(np.int32)
    pos2 = np.cumsum(rng.integers(1, 3, len(chunk2))).astype(np.int32)
    scores2 = rng.choice([0.25, 0.5, 0.75, 1.0], 60).astype(np.float32)
    M2 = len(chunk2) * 2 // 3
    r2 = _both(ds, chunk2, pos2, scores2, M2, 4, 256, 4, len(chunk2) + 64, seed=2)
    _check_equal(r2, M2)
    ref2 = oracle.select_keep(chunk2, pos2, scores2, len(chunk2), M2, 4, 256, 4)
    assert r2["keep_b"].cpu().tolist() == ref2


def test_noalloc_reports_broken_invariants(ds):
    """Chunk ids that decrease: nothing is rewritten and the caller's outcome
    word reads 1 (the kernel's own invariant check)."""
    chunk = np.repeat(np.arange(6), 100).astype(np.int32)
    chunk[250] = 0
    pos = np.arange(600, dtype=np.int32)
    sc = torch.rand(6, generator=torch.Generator().manual_seed(3)).to(DEV)
    t = _tables(chunk, pos, 640, seed=5)
    before = [x.clone() for x in t]
    free = torch.full((100,), -1, dtype=torch.int32, device=DEV)
    outcome = torch.full((1,), -5, dtype=torch.int32, device=DEV)
    ds.kv_evict_topk_indexed_noalloc(*t, sc, 600, 500, 0, 0, 1, free_out=free, outcome=outcome)
    torch.cuda.synchronize()
    assert int(outcome.item()) == 1
    for x, y in zip(t, before):
        assert torch.equal(x, y)
    assert torch.all(free == -1)
