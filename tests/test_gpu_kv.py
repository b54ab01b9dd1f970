"""GPU parity of kv_evict_topk: the keep list is bit-exact with the oracle's
selection, and the compacted K/V rows, positions and chunk ids are bit-exact
with the oracle's gather (position-keyed rows regenerate the expected cache)."""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_helpers import DEV

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ds():
    import paper_2609_27470_amd as ds
    ds.lib()
    return ds


def make_cache(L, row_elems, capacity, chunk, pos):
    """K/V planes whose row at slot i is the hash row of position pos[i]."""
    n = len(pos)
    pos_t = torch.zeros(capacity, dtype=torch.int64, device=DEV)
    pos_t[:n] = torch.as_tensor(np.asarray(pos, np.int64), device=DEV)
    ks, vs = [], []
    for l in range(L):
        kk = torch.zeros((capacity, row_elems), dtype=torch.int16, device=DEV)
        vv = torch.zeros((capacity, row_elems), dtype=torch.int16, device=DEV)
        kk[:n] = synth.kv_row_bits_torch(l, 0, pos_t[:n], row_elems)
        vv[:n] = synth.kv_row_bits_torch(l, 1, pos_t[:n], row_elems)
        ks.append(kk)
        vs.append(vv)
    p = torch.zeros(capacity, dtype=torch.int32, device=DEV)
    c = torch.zeros(capacity, dtype=torch.int32, device=DEV)
    p[:n] = torch.as_tensor(np.asarray(pos, np.int32), device=DEV)
    c[:n] = torch.as_tensor(np.asarray(chunk, np.int32), device=DEV)
    return ks, vs, p, c


def check_cache(ks, vs, p, c, M, exp_pos, exp_chunk):
    assert np.array_equal(p[:M].cpu().numpy(), exp_pos)
    assert np.array_equal(c[:M].cpu().numpy(), exp_chunk)
    ep = torch.as_tensor(np.asarray(exp_pos, np.int64), device=DEV)
    for l, (kk, vv) in enumerate(zip(ks, vs)):
        assert torch.equal(kk[:M], synth.kv_row_bits_torch(l, 0, ep, kk.shape[1])), f"K layer {l}"
        assert torch.equal(vv[:M], synth.kv_row_bits_torch(l, 1, ep, vv.shape[1])), f"V layer {l}"


def one_event(ds, L, row_elems, chunk, pos, scores, M, ns, nw, nb, capacity=None):
    n = len(pos)
    capacity = capacity or n
    ks, vs, p, c = make_cache(L, row_elems, capacity, chunk, pos)
    sc = torch.as_tensor(np.asarray(scores, np.float32), device=DEV)
    keep = torch.full((max(M, 1),), -1, dtype=torch.int32, device=DEV)
    new_len, ws = ds.kv_evict_topk(ks, vs, p, c, sc, n, M, ns, nw, nb, keep_out=keep)
    torch.cuda.synchronize()
    ref = oracle.select_keep(chunk, pos, scores, n, M, ns, nw, nb)
    if n <= M:
        assert new_len == n
        check_cache(ks, vs, p, c, n, np.asarray(pos), np.asarray(chunk))
        return
    assert new_len == M
    assert keep[:M].cpu().tolist() == ref
    st = ds.kv_device_status(ws)
    assert st[0] == 0 and st[2] == 0, st
    check_cache(ks, vs, p, c, M, np.asarray(pos)[ref], np.asarray(chunk)[ref])


def random_cache(rng, n_chunks, lo, hi, thin=0.8):
    lens = rng.integers(lo, hi + 1, n_chunks)
    chunk = np.repeat(np.arange(n_chunks), lens)
    keep = rng.random(len(chunk)) < thin
    chunk = chunk[keep]
    pos = (np.nonzero(keep)[0] + 3).astype(np.int64)
    return chunk.astype(np.int32), pos.astype(np.int32)


@pytest.mark.parametrize("seed", range(12))
def test_random_small_caches(ds, seed):
    rng = np.random.default_rng(1000 + seed)
    chunk, pos = random_cache(rng, int(rng.integers(3, 40)), 1, 60)
    n = len(chunk)
    scores = rng.choice([0.1, 0.25, 0.5, 1.0, 2.0], size=int(chunk.max()) + 1).astype(np.float32)
    if seed % 3 == 0:
        scores[0] = np.inf
    ns = int(rng.integers(0, 5))
    nw = int(rng.integers(0, 40))
    M = int(rng.integers(ns + nw, n + 3))
    nb = int(rng.integers(0, 9))
    one_event(ds, 2, 64 * (1 + seed % 3), chunk, pos, scores, M, ns, nw, nb)


@pytest.mark.parametrize("n_chunks,lo,hi,nb,window", [(1024, 1, 20, 1, False), (1500, 1, 16, 5, True),
                                                      (2048, 2, 6, 3, False), (3000, 1, 8, 4, True)])
def test_many_runs(ds, n_chunks, lo, hi, nb, window):
    """About 1000 to 3000 runs: the ranking sorts up to 2048 runs in LDS (the
    2048-chunk case without sinks and window has exactly 2048 candidate runs)
    and compares every pair in global memory beyond that (the 3000-chunk
    case).  Scores from a small set, so many runs tie on the score and are
    ordered by chunk id."""
    rng = np.random.default_rng(n_chunks + nb)
    chunk, pos = random_cache(rng, n_chunks, lo, hi, thin=0.9)
    if n_chunks == 2048:  # every chunk present: exactly 2048 runs
        chunk = np.repeat(np.arange(n_chunks), 3).astype(np.int32)
        pos = np.arange(len(chunk), dtype=np.int32) * 2 + 1
    n = len(chunk)
    scores = rng.choice([0.1, 0.2, 0.3, 0.5, 1.0], size=int(chunk.max()) + 1).astype(np.float32)
    scores[rng.integers(0, len(scores), 3)] = np.inf
    ns, nw = (4, n // 10) if window else (0, 0)
    one_event(ds, 1, 8, chunk, pos, scores, n * 2 // 3, ns, nw, nb)


def test_golden_examples_on_gpu(ds):
    import json, math, os
    gd = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "select_examples.json")))
    chunk = np.array(gd["cache"]["chunk_id"], np.int32)
    pos = np.array(gd["cache"]["pos"], np.int32)
    for c in gd["cases"]:
        sc = [math.inf if s == "inf" else float(s) for s in c["chunk_scores"]]
        one_event(ds, 1, 8, chunk, pos, sc, c["M"], c["n_sink"], c["n_window"], c["n_buckets"])


def test_equal_scores_keep_newest(ds):
    chunk = np.repeat(np.arange(10), 50).astype(np.int32)
    pos = np.arange(500, dtype=np.int32)
    one_event(ds, 1, 64, chunk, pos, np.full(10, 0.5, np.float32), 123, 0, 0, 1)


@pytest.mark.parametrize("policy", [(0, 0, 1), (4, 1024, 4)])
def test_eviction_loop_shape(ds, policy):
    """The eviction-loop cache at full size: 8 layers x (K, V) x 8 heads x 256
    bf16 (4 KiB rows), 17 chunks of 1024 tokens, budget 16384, capacity 17408."""
    ns, nw, nb = policy
    rng = np.random.default_rng(5)
    chunk = np.repeat(np.arange(17), 1024).astype(np.int32)
    pos = np.arange(17 * 1024, dtype=np.int32) + 40000
    scores = rng.random(17).astype(np.float32)
    scores[3] = np.inf
    one_event(ds, 8, 2048, chunk, pos, scores, 16384, ns, nw, nb)


def test_staged_and_ticket_regions_in_one_event(ds):
    """64 KiB of rows per token (8 layers x 4 KiB K and V): the first moved
    rows shift by 512 slots (less than 64 MiB of rows: staged through the
    workspace) and the later ones by 1536 (the ticket-ordered gather), in one
    event: 512 oldest tokens of chunk 2 and all of chunk 12 are evicted."""
    chunk = np.concatenate([np.repeat(np.arange(17), 1024), np.full(512, 17)]).astype(np.int32)
    pos = np.arange(len(chunk), dtype=np.int32) + 7
    scores = np.linspace(0.5, 1.0, 18).astype(np.float32)
    scores[12] = 0.01
    scores[2] = 0.02
    one_event(ds, 8, 2048, chunk, pos, scores, 16384, 0, 0, 1)


def test_small_shifts_full_shape(ds):
    """The paper's policy on the eviction-loop shape with chunks of 125
    tokens: every event removes a few scattered tokens, so every moved row
    shifts by less than 1024 slots (all staged)."""
    rng = np.random.default_rng(9)
    chunk = np.repeat(np.arange(140), 125)[:16384 + 125].astype(np.int32)
    pos = np.arange(len(chunk), dtype=np.int32)
    scores = rng.random(140).astype(np.float32)
    one_event(ds, 8, 2048, chunk, pos, scores, 16384, 4, 1024, 4)


def test_repeated_events_stream(ds):
    """Append a chunk per step and evict down to M every time the cache
    overflows; after every step the cache equals the oracle's replay."""
    L, row, M, F, capacity = 3, 128, 700, 96, 700 + 96
    rng = np.random.default_rng(11)
    steps = 40
    scores_all = rng.random(steps).astype(np.float32)
    scores_all[0] = np.inf
    ks, vs, p, c = make_cache(L, row, capacity, [], [])
    sc = torch.as_tensor(scores_all, device=DEV)
    ref_pos, ref_chunk = np.zeros(0, np.int64), np.zeros(0, np.int64)
    n = 0
    ws = None
    for f in range(steps):
        new_pos = np.arange(f * F, (f + 1) * F, dtype=np.int64)
        pt = torch.as_tensor(new_pos, device=DEV)
        for l in range(L):
            ks[l][n:n + F] = synth.kv_row_bits_torch(l, 0, pt, row)
            vs[l][n:n + F] = synth.kv_row_bits_torch(l, 1, pt, row)
        p[n:n + F] = pt.to(torch.int32)
        c[n:n + F] = f
        n += F
        ref_pos = np.concatenate([ref_pos, new_pos])
        ref_chunk = np.concatenate([ref_chunk, np.full(F, f)])
        new_len, ws = ds.kv_evict_topk(ks, vs, p, c, sc, n, M, 4, 64, 4, workspace=ws)
        if n > M:
            keep = oracle.select_keep(ref_chunk, ref_pos, scores_all, n, M, 4, 64, 4)
            ref_pos, ref_chunk = ref_pos[keep], ref_chunk[keep]
        n = new_len
        torch.cuda.synchronize()
        check_cache(ks, vs, p, c, n, ref_pos, ref_chunk)


def test_broken_invariants_leave_cache_untouched(ds):
    chunk = np.repeat(np.arange(6), 20).astype(np.int32)
    chunk[50] = 0                                   # chunk ids go backwards
    pos = np.arange(120, dtype=np.int32)
    ks, vs, p, c = make_cache(1, 64, 120, chunk, pos)
    before = ks[0].clone()
    sc = torch.ones(6, dtype=torch.float32, device=DEV)
    new_len, ws = ds.kv_evict_topk(ks, vs, p, c, sc, 120, 60, 0, 0, 1)
    torch.cuda.synchronize()
    assert ds.kv_device_status(ws)[0] == 1
    assert torch.equal(ks[0], before)
    assert np.array_equal(p.cpu().numpy(), pos)


# ---------------------------------------------------------------- slot-indexed variant
def indexed_event(ds, chunk, pos, scores, M, ns, nw, nb, seed=0, capacity=None):
    """kv_evict_topk_indexed on a table whose rows are scattered over the
    physical cache; keep list, compacted table and free list bit-exact with
    the oracle."""
    n = len(pos)
    capacity = capacity or n + 5
    rng = np.random.default_rng(seed)
    slot = rng.permutation(capacity)[:n].astype(np.int32)
    mk = lambda a: torch.as_tensor(np.concatenate([np.asarray(a, np.int32),
                                                   np.full(capacity - n, -7, np.int32)]), device=DEV)
    p, c, s = mk(pos), mk(chunk), mk(slot)
    sc = torch.as_tensor(np.asarray(scores, np.float32), device=DEV)
    keep = torch.full((max(M, 1),), -1, dtype=torch.int32, device=DEV)
    new_len, ws, free = ds.kv_evict_topk_indexed(p, c, s, sc, n, M, ns, nw, nb, keep_out=keep)
    torch.cuda.synchronize()
    if n <= M:
        assert new_len == n
        assert np.array_equal(s[:n].cpu().numpy(), slot) and np.array_equal(p[:n].cpu().numpy(), pos)
        return
    ref = oracle.select_keep(chunk, pos, scores, n, M, ns, nw, nb)
    assert new_len == M
    assert ds.kv_device_status(ws)[0] == 0
    assert keep[:M].cpu().tolist() == ref
    ep, ec, es, efree = oracle.compact_indexed(pos, chunk, slot, ref, n)
    assert np.array_equal(p[:M].cpu().numpy(), ep)
    assert np.array_equal(c[:M].cpu().numpy(), ec)
    assert np.array_equal(s[:M].cpu().numpy(), es)
    assert np.array_equal(free[:n - M].cpu().numpy(), efree)
    assert np.array_equal(s[n:].cpu().numpy(), np.full(capacity - n, -7))   # beyond len: untouched


@pytest.mark.parametrize("seed", range(8))
def test_indexed_random_small_caches(ds, seed):
    rng = np.random.default_rng(2000 + seed)
    chunk, pos = random_cache(rng, int(rng.integers(3, 40)), 1, 60)
    n = len(chunk)
    scores = rng.choice([0.1, 0.25, 0.5, 1.0, 2.0], size=int(chunk.max()) + 1).astype(np.float32)
    ns = int(rng.integers(0, 5))
    nw = int(rng.integers(0, 40))
    M = int(rng.integers(ns + nw, n + 3))
    indexed_event(ds, chunk, pos, scores, M, ns, nw, int(rng.integers(0, 9)), seed=seed)


@pytest.mark.parametrize("policy", [(0, 0, 1), (4, 1024, 4)])
def test_indexed_eviction_loop_shape(ds, policy):
    """17 chunks of 1024 tokens down to 16384, capacity 17408."""
    rng = np.random.default_rng(6)
    chunk = np.repeat(np.arange(17), 1024).astype(np.int32)
    pos = np.arange(17 * 1024, dtype=np.int32) + 40000
    scores = rng.random(17).astype(np.float32)
    indexed_event(ds, chunk, pos, scores, 16384, *policy, seed=3, capacity=17408)


def test_indexed_long_cache_several_blocks(ds):
    """A cache of ~100k tokens, so that selection and the table compaction
    both run over several 32768-slot blocks."""
    rng = np.random.default_rng(8)
    chunk, pos = random_cache(rng, 90, 900, 1400, thin=0.9)
    scores = rng.random(90).astype(np.float32)
    n = len(chunk)
    indexed_event(ds, chunk, pos, scores, n // 2, 4, 1000, 5, seed=4)


@pytest.mark.parametrize("n_chunks", [1500, 2600])
def test_indexed_many_runs(ds, n_chunks):
    """The slot-indexed eviction over caches of 1500 and 2600 short chunks:
    its ranking takes the sorted path (up to 2048 runs) and the pairwise one
    over the global run table (beyond)."""
    rng = np.random.default_rng(70 + n_chunks)
    chunk, pos = random_cache(rng, n_chunks, 1, 12, thin=0.9)
    scores = rng.choice([0.1, 0.2, 0.5, 1.0], size=n_chunks).astype(np.float32)
    n = len(chunk)
    indexed_event(ds, chunk, pos, scores, n * 3 // 4, 4, 64, 3, seed=9)


def test_indexed_matches_gather_in_a_stream(ds):
    """Appends write each new chunk's K/V rows into the rows the previous
    eviction freed (an index_copy by the caller); after every step the rows
    read through the table equal the position-keyed rows of the gather-based
    cache, which the gather variant itself rebuilds in the same loop."""
    L, row, M, F, capacity = 2, 128, 700, 96, 700 + 96
    rng = np.random.default_rng(12)
    steps = 30
    scores_all = rng.random(steps).astype(np.float32)
    scores_all[0] = np.inf
    sc = torch.as_tensor(scores_all, device=DEV)
    # gather-based cache
    ks, vs, p, c = make_cache(L, row, capacity, [], [])
    # indexed cache: physical rows + table
    kx = [torch.zeros((capacity, row), dtype=torch.int16, device=DEV) for _ in range(L)]
    tp = torch.zeros(capacity, dtype=torch.int32, device=DEV)
    tc = torch.zeros(capacity, dtype=torch.int32, device=DEV)
    ts = torch.zeros(capacity, dtype=torch.int32, device=DEV)
    free = torch.arange(capacity, dtype=torch.int32, device=DEV)
    n, ws_g, ws_x = 0, None, None
    for f in range(steps):
        pt = torch.arange(f * F, (f + 1) * F, dtype=torch.int64, device=DEV) + 77
        dst = free[:F].to(torch.int64)
        for l in range(L):
            rows_k = synth.kv_row_bits_torch(l, 0, pt, row)
            ks[l][n:n + F] = rows_k
            vs[l][n:n + F] = synth.kv_row_bits_torch(l, 1, pt, row)
            kx[l].index_copy_(0, dst, rows_k)
        p[n:n + F] = pt.to(torch.int32)
        c[n:n + F] = f
        tp[n:n + F] = pt.to(torch.int32)
        tc[n:n + F] = f
        ts[n:n + F] = dst.to(torch.int32)
        n += F
        kg = torch.empty(M, dtype=torch.int32, device=DEV)
        kxk = torch.empty(M, dtype=torch.int32, device=DEV)
        new_len, ws_g = ds.kv_evict_topk(ks, vs, p, c, sc, n, M, 4, 64, 4, keep_out=kg, workspace=ws_g)
        new_x, ws_x, freed = ds.kv_evict_topk_indexed(tp, tc, ts, sc, n, M, 4, 64, 4, keep_out=kxk,
                                                      workspace=ws_x)
        assert new_x == new_len
        free = free[F:]                              # rows never used so far
        if n > M:
            assert torch.equal(kg, kxk)
            free = torch.cat([free, freed[:n - M]])
        n = new_len
        torch.cuda.synchronize()
        assert torch.equal(tp[:n], p[:n]) and torch.equal(tc[:n], c[:n])
        idx = ts[:n].to(torch.int64)
        for l in range(L):
            assert torch.equal(kx[l][idx], ks[l][:n]), f"step {f} layer {l}"
        assert sorted(torch.cat([ts[:n], free]).cpu().tolist()) == list(range(capacity))


def test_indexed_broken_invariants_leave_table_untouched(ds):
    chunk = np.repeat(np.arange(6), 20).astype(np.int32)
    pos = np.arange(120, dtype=np.int32)
    pos[70] = pos[69]                                # positions not increasing
    p = torch.as_tensor(pos, device=DEV)
    c = torch.as_tensor(chunk, device=DEV)
    s = torch.arange(120, dtype=torch.int32, device=DEV)
    free = torch.full((60,), -3, dtype=torch.int32, device=DEV)
    sc = torch.ones(6, dtype=torch.float32, device=DEV)
    new_len, ws, _ = ds.kv_evict_topk_indexed(p, c, s, sc, 120, 60, 0, 0, 1, free_out=free)
    torch.cuda.synchronize()
    assert ds.kv_device_status(ws)[0] == 1
    assert np.array_equal(p.cpu().numpy(), pos) and np.array_equal(c.cpu().numpy(), chunk)
    assert torch.equal(s, torch.arange(120, dtype=torch.int32, device=DEV))
    assert torch.equal(free, torch.full((60,), -3, dtype=torch.int32, device=DEV))


@pytest.mark.parametrize("na,nb,T,n,row", [(50, 30, 40, 10, 64), (50, 30, 70, 20, 4096), (0, 80, 80, 0, 16),
                                           (80, 0, 0, 7, 64), (300, 700, 257, 600, 4096), (1024, 0, 1, 0, 48)])
def test_append_indexed_matches_indexing(ds, na, nb, T, n, row):
    """kv_append_indexed against plain tensor indexing: each plane's rows at
    the first T entries of free_a ++ free_b hold the new rows, every other row
    keeps its bytes; pos, chunk_id and slot [n, n + T) hold the positions,
    the chunk id and those rows, the rest of each table is untouched; the
    rest of the list lands in free_rest.  Bit for bit, spanning several
    256-entry blocks of the list copy and both list segments."""
    capacity = 1024 + 64
    g = torch.Generator(device=DEV).manual_seed(na * 7 + nb + T)
    L = 3
    kp = torch.randint(-30000, 30000, (L, capacity, row // 2), dtype=torch.int16, device=DEV, generator=g)
    vp = torch.randint(-30000, 30000, (L, capacity, row // 2), dtype=torch.int16, device=DEV, generator=g)
    kn = torch.randint(-30000, 30000, (L, T + 5, row // 2), dtype=torch.int16, device=DEV, generator=g)
    vn = torch.randint(-30000, 30000, (L, T + 5, row // 2), dtype=torch.int16, device=DEV, generator=g)
    perm = torch.randperm(capacity, generator=torch.Generator().manual_seed(T)).to(torch.int32).to(DEV)
    fa, fb = perm[:na].clone(), perm[na:na + nb].clone()
    rest = torch.full((capacity,), -9, dtype=torch.int32, device=DEV)
    tabs = [torch.randint(-100, 100, (capacity,), dtype=torch.int32, device=DEV, generator=g) for _ in range(3)]
    exp_k, exp_v, exp_tabs = kp.clone(), vp.clone(), [t.clone() for t in tabs]
    lst = torch.cat([fa, fb]).to(torch.int64)
    dst = lst[:T]
    exp_k[:, dst] = kn[:, :T]
    exp_v[:, dst] = vn[:, :T]
    exp_tabs[0][n:n + T] = torch.arange(5000, 5000 + T, dtype=torch.int32, device=DEV)
    exp_tabs[1][n:n + T] = 37
    exp_tabs[2][n:n + T] = dst.to(torch.int32)
    ds.kv_append_indexed(kp, vp, kn, vn, fa if na else None, na, fb if nb else None, nb, rest, T, n, 5000, 37,
                         *tabs)
    torch.cuda.synchronize()
    assert torch.equal(kp, exp_k) and torch.equal(vp, exp_v)
    for t, e in zip(tabs, exp_tabs):
        assert torch.equal(t, e)
    r = na + nb - T
    assert torch.equal(rest[:r], lst[T:].to(torch.int32)) and bool((rest[r:] == -9).all())
