"""Pins for the fp64 oracle: closed forms, invariants, an independent
chunkwise formulation, Eq. 1 vs Eq. 2, and hand-worked selection examples.

Everything here runs on the CPU; nothing touches the HIP library.
"""
import json
import math
import os

import numpy as np
import pytest

import oracle
import synth
from chunkwise_ref import chunkwise_forward, eq1_forward
from synth import bf16_bits_to_f64, to_bf16_bits

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand_inputs(seed, T, H_k, H_v, d, lengths=None):
    rng = np.random.default_rng(seed)
    if lengths is None:
        lengths = [T]
    T = sum(lengths)
    q = rng.standard_normal((T, H_k, d))
    k = rng.standard_normal((T, H_k, d))
    q /= np.linalg.norm(q, axis=-1, keepdims=True)
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((T, H_v, d))
    g = (-np.logaddexp(0, rng.standard_normal((T, H_v)))).astype(np.float32)
    beta = (1 / (1 + np.exp(-rng.standard_normal((T, H_v))))).astype(np.float32)
    cu = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    return to_bf16_bits(q), to_bf16_bits(k), to_bf16_bits(v), g, beta, cu


# ---------------------------------------------------------------- P1
def test_no_decay_no_write_keeps_state():
    """g = 0 and beta = 0: alpha = 1 and every write is zero, so S_T = S0
    exactly, o_t = S0 q_t and the drift sums are exactly zero."""
    q, k, v, _, _, cu = _rand_inputs(1, 300, 2, 4, 16)
    T, H_v = v.shape[0], v.shape[1]
    g = np.zeros((T, H_v), np.float32)
    beta = np.zeros((T, H_v), np.float32)
    S0 = np.random.default_rng(2).standard_normal((1, H_v, 16, 16))
    r = oracle.gdn_forward(q, k, v, g, beta, cu, 64, S0=S0)
    assert np.array_equal(r["S"], S0)
    qf = bf16_bits_to_f64(q)
    for j in range(H_v):
        ref = qf[:, j // 2] @ S0[0, j].T
        np.testing.assert_allclose(r["o"][:, j], ref, rtol=1e-13, atol=1e-13)
    assert np.all(r["partials"][:, :, 0] == 0.0)
    # den of the first frame is ||S0||^2, later frames the same state
    np.testing.assert_allclose(r["partials"][:, :, 1],
                               np.broadcast_to(np.sum(S0[0] ** 2, axis=(1, 2)), r["partials"][:, :, 1].shape),
                               rtol=1e-14)


# ---------------------------------------------------------------- P2
def test_full_write_retrieves_value_for_any_decay():
    """beta = 1 with a unit key: S_t k_t = alpha S k + (v - alpha S k) = v_t for
    any alpha, so reading with q_t = k_t returns o_t = v_t."""
    d, T, H = 64, 200, 2
    rng = np.random.default_rng(3)
    keys = synth.orthonormal_keys(d)
    idx = rng.integers(0, d, size=(T, H))
    sign = rng.choice([-1.0, 1.0], size=(T, H))
    kk = keys[idx] * sign[..., None]          # exactly unit, exact in bf16
    k = to_bf16_bits(kk)
    q = k.copy()
    v = to_bf16_bits(rng.standard_normal((T, H, d)))
    g = (-rng.uniform(0, 3, size=(T, H))).astype(np.float32)
    beta = np.ones((T, H), np.float32)
    cu = np.array([0, T], np.int32)
    r = oracle.gdn_forward(q, k, v, g, beta, cu, 0)
    np.testing.assert_allclose(r["o"], bf16_bits_to_f64(v), rtol=0, atol=1e-12)


def test_orthonormal_keys_store_every_pair():
    """g = 0, beta = 1, d orthonormal keys written once each: S_T k_i = v_i for
    every written pair (the keys do not interfere)."""
    d = 128
    keys = synth.orthonormal_keys(d)
    rng = np.random.default_rng(4)
    perm = rng.permutation(d)
    k = to_bf16_bits(keys[perm][:, None, :])
    q = to_bf16_bits(rng.standard_normal((d, 1, d)))
    vv = rng.standard_normal((d, 1, d))
    v = to_bf16_bits(vv)
    g = np.zeros((d, 1), np.float32)
    beta = np.ones((d, 1), np.float32)
    r = oracle.gdn_forward(q, k, v, g, beta, np.array([0, d], np.int32), 32)
    S = r["S"][0, 0]
    K = bf16_bits_to_f64(k)[:, 0]
    np.testing.assert_allclose(K @ S.T, bf16_bits_to_f64(v)[:, 0], rtol=0, atol=1e-12)


# ---------------------------------------------------------------- P3
def test_represented_pairs_give_zero_drift():
    """A frame that re-presents pairs the state already stores (g = 0) has a
    zero residual, hence writes nothing and has drift exactly 0."""
    d = 64
    keys = synth.orthonormal_keys(d)
    rng = np.random.default_rng(5)
    n = 32
    sel = rng.choice(d, size=n, replace=False)
    k1 = keys[sel]
    v1 = rng.standard_normal((n, d))
    order = rng.permutation(n)
    kk = np.concatenate([k1, k1[order]])[:, None, :]
    vv = np.concatenate([v1, v1[order]])[:, None, :]
    k = to_bf16_bits(kk)
    v = to_bf16_bits(vv)
    q = to_bf16_bits(rng.standard_normal((2 * n, 1, d)))
    g = np.zeros((2 * n, 1), np.float32)
    beta = np.concatenate([np.ones(n), rng.uniform(0.1, 1, n)]).astype(np.float32)[:, None]
    r = oracle.gdn_forward(q, k, v, g, beta, np.array([0, 2 * n], np.int32), n)
    assert r["partials"][0, 0, 0] > 0           # the first frame wrote
    assert r["partials"][1, 0, 0] == 0.0        # the second frame did not
    assert r["partials"][1, 0, 1] > 0
    sc = oracle.drift_scores(r["partials"][None], oracle.LAYER_FROB)
    assert sc[1] == 0.0 and math.isinf(sc[0])


# ---------------------------------------------------------------- P4
def test_pure_decay_drift_closed_form():
    """beta = 0 after the first frame: S_end = exp(sum_frame g) S_start, so the
    per-head drift of that frame is 1 - exp(sum g)."""
    q, k, v, g, beta, cu = _rand_inputs(6, 5 * 64, 2, 4, 32)
    beta[64:] = 0.0
    g[64:] *= 0.05                      # keep the state well above underflow
    r = oracle.gdn_forward(q, k, v, g, beta, cu, 64)
    ph = oracle.drift_scores(r["partials"][None], oracle.PER_HEAD)[0]
    for f in range(1, 5):
        sg = np.sum(g[64 * f:64 * (f + 1)].astype(np.float64), axis=0)
        np.testing.assert_allclose(ph[f], 1.0 - np.exp(sg), rtol=1e-10)


# ---------------------------------------------------------------- P5
def test_single_token_frame_drift_is_write_norm():
    """One-token frames, g = 0, unit keys: ||S_after - S_before||_F equals
    beta ||v - S k||_2 (the rank-one write has that norm, Appendix on the
    beta||e|| signal)."""
    d, T = 64, 40
    rng = np.random.default_rng(7)
    keys = synth.orthonormal_keys(d)
    k = to_bf16_bits(keys[rng.integers(0, d, T)][:, None, :])
    q = to_bf16_bits(rng.standard_normal((T, 1, d)))
    v = to_bf16_bits(rng.standard_normal((T, 1, d)))
    g = np.zeros((T, 1), np.float32)
    beta = rng.uniform(0.05, 1, (T, 1)).astype(np.float32)
    r = oracle.gdn_forward(q, k, v, g, beta, np.array([0, T], np.int32), 1, snapshots=True)
    K = bf16_bits_to_f64(k)[:, 0]
    V = bf16_bits_to_f64(v)[:, 0]
    prev = np.zeros((d, d))
    for t in range(T):
        expect = float(beta[t, 0]) * np.linalg.norm(V[t] - prev @ K[t])
        np.testing.assert_allclose(math.sqrt(r["partials"][t, 0, 0]), expect, rtol=1e-12, atol=1e-14)
        prev = r["snapshots"][t, 0]


# ---------------------------------------------------------------- scalar closed form
def test_scalar_state_sum_product_form():
    """d = 1, k = +-1: S_t = (1 - beta_t) alpha_t S_{t-1} + beta_t k_t v_t, whose
    solution is S_T = sum_t beta_t k_t v_t prod_{s>t} (1-beta_s) alpha_s + S0 prod_s (...)."""
    rng = np.random.default_rng(8)
    T = 50
    ks = rng.choice([-1.0, 1.0], T)
    k = to_bf16_bits(ks[:, None, None])
    q = to_bf16_bits(rng.standard_normal((T, 1, 1)))
    vv = bf16_bits_to_f64(to_bf16_bits(rng.standard_normal((T, 1, 1))))
    v = to_bf16_bits(vv)
    g = (-rng.uniform(0, 1, (T, 1))).astype(np.float32)
    beta = rng.uniform(0, 1, (T, 1)).astype(np.float32)
    S0 = np.array([[[[0.7]]]])
    r = oracle.gdn_forward(q, k, v, g, beta, np.array([0, T], np.int32), 0, S0=S0)
    a = np.exp(g[:, 0].astype(np.float64))
    b = beta[:, 0].astype(np.float64)
    f = (1 - b) * a
    tot = S0[0, 0, 0, 0] * np.prod(f)
    for t in range(T):
        tot += b[t] * ks[t] * vv[t, 0, 0] * np.prod(f[t + 1:])
    np.testing.assert_allclose(r["S"][0, 0, 0, 0], tot, rtol=1e-12)


# ---------------------------------------------------------------- P6
def test_eq1_matches_eq2():
    """Eq. 1 (explicit d_k x d_k product) and Eq. 2 (residual form) agree."""
    q, k, v, g, beta, cu = _rand_inputs(9, 90, 2, 4, 16)
    S0 = np.random.default_rng(10).standard_normal((1, 4, 16, 16))
    r = oracle.gdn_forward(q, k, v, g, beta, cu, 0, S0=S0)
    o1, S1 = eq1_forward(q, k, v, g, beta, 90, 2, 4, S0=S0[0])
    np.testing.assert_allclose(r["o"], o1, rtol=0, atol=1e-13 * max(1, np.abs(o1).max()))
    np.testing.assert_allclose(r["S"][0], S1, rtol=0, atol=1e-13 * max(1, np.abs(S1).max()))


# ---------------------------------------------------------------- P7
@pytest.mark.parametrize("C", [1, 2, 3, 8, 64])
@pytest.mark.parametrize("grp", [1, 2])
def test_chunkwise_matches_recurrence(C, grp):
    """The tile-parallel form (derived from Eq. 2) reproduces the token
    recurrence on ragged streams, with zero and non-zero entry states."""
    lengths = [1, 63, 65, 130]
    H_k = 2
    H_v = H_k * grp
    q, k, v, g, beta, cu = _rand_inputs(11 + C + grp, 0, H_k, H_v, 8, lengths=lengths)
    for S0 in (None, np.random.default_rng(12).standard_normal((4, H_v, 8, 8))):
        r = oracle.gdn_forward(q, k, v, g, beta, cu, 64, S0=S0)
        c = chunkwise_forward(q, k, v, g, beta, cu, 64, C=C, S0=S0)
        np.testing.assert_allclose(r["o"], c["o"], rtol=0, atol=1e-12)
        np.testing.assert_allclose(r["S"], c["S"], rtol=0, atol=1e-12)
        np.testing.assert_allclose(r["partials"], c["partials"], rtol=1e-11, atol=1e-12)


# ---------------------------------------------------------------- P8
def test_power_of_two_scaling_invariance():
    """Scaling v and S0 by 2^j scales o and S by 2^j exactly and leaves the
    drift bit-identical; scaling q scales o only."""
    q, k, v, g, beta, cu = _rand_inputs(13, 200, 1, 2, 16)
    S0 = np.random.default_rng(14).standard_normal((1, 2, 16, 16))
    r0 = oracle.gdn_forward(q, k, v, g, beta, cu, 64, S0=S0)
    v4 = to_bf16_bits(bf16_bits_to_f64(v) * 4.0)
    r1 = oracle.gdn_forward(q, k, v4, g, beta, cu, 64, S0=S0 * 4.0)
    assert np.array_equal(r1["o"], 4.0 * r0["o"])
    assert np.array_equal(r1["S"], 4.0 * r0["S"])
    s0 = oracle.drift_scores(r0["partials"][None], oracle.PER_HEAD)
    s1 = oracle.drift_scores(r1["partials"][None], oracle.PER_HEAD)
    assert np.array_equal(s0, s1)
    q2 = to_bf16_bits(bf16_bits_to_f64(q) * 0.5)
    r2 = oracle.gdn_forward(q2, k, v, g, beta, cu, 64, S0=S0)
    assert np.array_equal(r2["o"], 0.5 * r0["o"]) and np.array_equal(r2["S"], r0["S"])


def test_head_permutation_equivariance():
    """Permuting (qk-head, v-head) groups permutes every output the same way."""
    q, k, v, g, beta, cu = _rand_inputs(15, 150, 2, 4, 16)
    r0 = oracle.gdn_forward(q, k, v, g, beta, cu, 64)
    hp = [1, 0]
    vp = [2, 3, 0, 1]
    r1 = oracle.gdn_forward(q[:, hp], k[:, hp], v[:, vp], g[:, vp], beta[:, vp], cu, 64)
    assert np.array_equal(r1["o"], r0["o"][:, vp])
    assert np.array_equal(r1["S"], r0["S"][:, vp])
    assert np.array_equal(r1["partials"], r0["partials"][:, vp])


# ---------------------------------------------------------------- P9 drift modes
def test_drift_modes_agree_on_single_and_identical_heads():
    rng = np.random.default_rng(16)
    p1 = rng.uniform(0.1, 2, (3, 5, 1, 2))
    lf = oracle.drift_scores(p1, oracle.LAYER_FROB)
    ph = oracle.drift_scores(p1, oracle.PER_HEAD)
    hm = oracle.drift_scores(p1, oracle.HEAD_MEAN)
    np.testing.assert_allclose(lf, ph[:, :, 0].mean(axis=0), rtol=1e-15)
    np.testing.assert_allclose(hm, lf, rtol=1e-15)
    p4 = np.repeat(p1, 4, axis=2)
    np.testing.assert_allclose(oracle.drift_scores(p4, oracle.LAYER_FROB), lf, rtol=1e-14)
    np.testing.assert_allclose(oracle.drift_scores(p4, oracle.HEAD_MEAN), lf, rtol=1e-14)


def test_drift_layer_frob_pools_heads():
    """Eq. 3 takes the Frobenius norm over all heads of a layer: two heads with
    (num, den) = (1, 1) and (9, 100) give sqrt(10/101), not the head mean."""
    p = np.array([[[[1.0, 1.0], [9.0, 100.0]]]])
    assert oracle.drift_scores(p, oracle.LAYER_FROB)[0] == pytest.approx(math.sqrt(10 / 101), rel=1e-15)
    assert oracle.drift_scores(p, oracle.HEAD_MEAN)[0] == pytest.approx(0.5 * (1 + 0.3), rel=1e-15)


def test_drift_zero_previous_state():
    p = np.array([[[[2.0, 0.0]], [[0.0, 0.0]]]])
    s = oracle.drift_scores(p, oracle.LAYER_FROB)
    assert math.isinf(s[0]) and s[1] == 0.0


# ---------------------------------------------------------------- selection (P10)
def _load_golden():
    with open(os.path.join(GOLDEN, "select_examples.json")) as f:
        return json.load(f)


@pytest.mark.parametrize("case", range(4))
def test_selection_golden(case):
    gd = _load_golden()
    c = gd["cases"][case]
    scores = [math.inf if s == "inf" else float(s) for s in c["chunk_scores"]]
    chunk = gd["cache"]["chunk_id"]
    pos = gd["cache"]["pos"]
    keep = oracle.select_keep(chunk, pos, scores, len(chunk), c["M"], c["n_sink"], c["n_window"],
                              c["n_buckets"])
    assert keep == c["keep"]


def _random_cache(rng, n_chunks, chunk_len_lo, chunk_len_hi):
    lens = rng.integers(chunk_len_lo, chunk_len_hi + 1, n_chunks)
    chunk = np.repeat(np.arange(n_chunks), lens)
    # a cache that has already been thinned: drop some tokens, keep order
    keep = rng.random(len(chunk)) < 0.8
    keep[:2] = True
    chunk = chunk[keep]
    pos = np.nonzero(keep)[0] + 7
    return chunk.astype(np.int32), pos.astype(np.int32)


def _key(scores, chunk, pos, i):
    return (-scores[chunk[i]], -chunk[i], -pos[i])


@pytest.mark.parametrize("seed", range(40))
def test_selection_properties(seed):
    rng = np.random.default_rng(100 + seed)
    chunk, pos = _random_cache(rng, int(rng.integers(2, 30)), 1, 12)
    n = len(chunk)
    scores = rng.choice([0.1, 0.2, 0.3, 0.5, 1.0], size=chunk.max() + 1).astype(np.float32)
    if rng.random() < 0.3:
        scores[0] = np.inf
    n_s = int(rng.integers(0, 4))
    n_w = int(rng.integers(0, 6))
    M = int(rng.integers(n_s + n_w, max(n_s + n_w + 1, n)))
    N = int(rng.integers(0, 5))
    keep = oracle.select_keep(chunk, pos, scores, n, M, n_s, n_w, N)
    if n <= M:
        assert keep == list(range(n))
        return
    assert len(keep) == M
    assert keep == sorted(set(keep))
    assert set(range(n_s)) <= set(keep)
    assert set(range(n - n_w, n)) <= set(keep)
    cand = list(range(n_s, n - n_w))
    kept_c = [i for i in cand if i in set(keep)]
    drop_c = [i for i in cand if i not in set(keep)]
    Nb = max(1, N)
    a_min = min(chunk[i] for i in cand)
    a_max = max(chunk[i] for i in cand)
    bucket = {i: (Nb * (chunk[i] - a_min)) // (a_max - a_min + 1) for i in cand}
    quota = (M - n_s - n_w) // Nb
    for b in range(Nb):
        mem = [i for i in cand if bucket[i] == b]
        kb = [i for i in mem if i in set(keep)]
        # each span keeps at least min(quota, |span|)
        assert len(kb) >= min(quota, len(mem))
        # inside a span the best min(quota, |span|) candidates are all kept
        best = sorted(mem, key=lambda i: _key(scores, chunk, pos, i))[:min(quota, len(mem))]
        assert set(best) <= set(kb)
    # every dropped candidate is beaten by every kept candidate that was kept
    # beyond its span quota (the fill is a global top)
    if drop_c:
        best_drop = min(drop_c, key=lambda i: _key(scores, chunk, pos, i))
        over = []
        for b in range(Nb):
            mem = sorted([i for i in kept_c if bucket[i] == b], key=lambda i: _key(scores, chunk, pos, i))
            over += mem[quota:]
        for i in over:
            assert _key(scores, chunk, pos, i) < _key(scores, chunk, pos, best_drop)


def test_selection_global_topM_and_equal_scores():
    rng = np.random.default_rng(7)
    chunk, pos = _random_cache(rng, 20, 3, 9)
    n = len(chunk)
    scores = rng.random(chunk.max() + 1).astype(np.float32)
    M = n // 2
    keep = oracle.select_keep(chunk, pos, scores, n, M, 0, 0, 1)
    order = sorted(range(n), key=lambda i: _key(scores, chunk, pos, i))
    assert keep == sorted(order[:M])
    eq = np.full_like(scores, 0.25)
    keep = oracle.select_keep(chunk, pos, eq, n, M, 0, 0, 1)
    assert keep == list(range(n - M, n))            # all equal -> newest kept


def test_compaction_keeps_positions_and_rows():
    """Position-keyed rows: after compaction row i is the row generated for
    the position now stored in slot i (positions are never rewritten)."""
    pos = np.arange(40, dtype=np.int32) + 1000
    rows = synth.kv_row_bits(3, 1, pos, 16)
    keep = [0, 1, 5, 6, 7, 20, 39]
    new_rows = oracle.compact(rows, keep)
    new_pos = oracle.compact(pos, keep)
    assert np.array_equal(new_rows, synth.kv_row_bits(3, 1, new_pos, 16))


def test_indexed_compaction_equals_gather_over_a_stream():
    """A slot-indexed cache evicts the same tokens as the gather and moves
    none of their rows: over a stream of appends (new tokens written into the
    freed rows) and evictions, the rows read through the table always equal
    the gathered cache, the table is a permutation of the rows in use, and the
    free list holds exactly the rows of the evicted tokens in logical order."""
    rng = np.random.default_rng(23)
    F, M, cap, steps, W = 37, 150, 150 + 37, 30, 8
    scores = rng.random(steps).astype(np.float32)
    # gather cache: rows in logical order; indexed cache: physical rows + table
    dt = synth.kv_row_bits(0, 0, np.zeros(1, np.int64), W).dtype
    g_rows = np.zeros((0, W), dt)
    g_pos = np.zeros(0, np.int64)
    g_chunk = np.zeros(0, np.int64)
    phys = np.zeros((cap, W), dt)
    t_pos, t_chunk, t_slot = np.zeros(0, np.int64), np.zeros(0, np.int64), np.zeros(0, np.int64)
    free = np.arange(cap)
    for f in range(steps):
        new_pos = np.arange(f * F, (f + 1) * F) + 500
        new_rows = synth.kv_row_bits(2, 0, new_pos, W)
        g_rows = np.concatenate([g_rows, new_rows])
        g_pos = np.concatenate([g_pos, new_pos])
        g_chunk = np.concatenate([g_chunk, np.full(F, f)])
        dst = free[:F]
        phys[dst] = new_rows
        t_pos = np.concatenate([t_pos, new_pos])
        t_chunk = np.concatenate([t_chunk, np.full(F, f)])
        t_slot = np.concatenate([t_slot, dst])
        free = free[F:]
        n = len(g_pos)
        if n > M:
            keep = oracle.select_keep(g_chunk, g_pos, scores, n, M, 2, 20, 3)
            assert keep == oracle.select_keep(t_chunk, t_pos, scores, n, M, 2, 20, 3)
            before, slot_before = phys.copy(), t_slot.copy()
            t_pos, t_chunk, t_slot, freed = oracle.compact_indexed(t_pos, t_chunk, t_slot, keep, n)
            assert np.array_equal(phys, before)                       # no row moved
            evicted = [i for i in range(n) if i not in set(keep)]
            assert freed.tolist() == [int(slot_before[i]) for i in evicted]
            assert len(freed) == n - M
            free = np.concatenate([free, freed])
            g_rows, g_pos, g_chunk = oracle.compact(g_rows, keep), g_pos[keep], g_chunk[keep]
        assert np.array_equal(t_pos, g_pos) and np.array_equal(t_chunk, g_chunk)
        assert np.array_equal(phys[t_slot], g_rows)
        assert sorted(np.concatenate([t_slot, free]).tolist()) == list(range(cap))


def test_indexed_free_list_by_hand():
    """A 6-token table with rows scattered in physical memory; keeping logical
    tokens 1, 2 and 4 frees the rows of tokens 0, 3 and 5, in that order."""
    pos = np.array([10, 11, 12, 13, 14, 15])
    chunk = np.array([0, 0, 1, 1, 2, 2])
    slot = np.array([7, 2, 9, 0, 4, 5])
    p2, c2, s2, free = oracle.compact_indexed(pos, chunk, slot, [1, 2, 4], 6)
    assert p2.tolist() == [11, 12, 14] and c2.tolist() == [0, 1, 2]
    assert s2.tolist() == [2, 9, 4] and free.tolist() == [7, 0, 5]


# ---------------------------------------------------------------- P12
def test_paper_size_constants():
    """48 MiB of recurrent state over 24 layers and 32 KiB of KV per token
    over 8 full-attention layers (Section 3.1 and the model description)."""
    assert 24 * 32 * 128 * 128 * 4 == 48 * 2 ** 20
    assert 8 * 4 * 256 * 2 * 2 == 32 * 2 ** 10


# ---------------------------------------------------------------- drift from two states
def test_drift_states_closed_forms():
    """drift_states against closed forms: an unchanged state gives num = 0; a
    zero state before gives den = 0 and num = ||S_after||^2; S_after = c S_before
    gives num = (c - 1)^2 den; a single changed entry gives num = delta^2."""
    rng = np.random.default_rng(5)
    S = rng.standard_normal((2, 3, 4, 8, 8))
    p = oracle.drift_states(S, S)
    assert np.all(p[..., 0] == 0.0)
    assert np.allclose(p[..., 1], np.einsum("...ij,...ij->...", S, S), rtol=1e-14)
    z = oracle.drift_states(np.zeros_like(S), S)
    assert np.all(z[..., 1] == 0.0)
    assert np.allclose(z[..., 0], (S ** 2).sum(axis=(-2, -1)), rtol=1e-14)
    c = 0.75
    q = oracle.drift_states(S, c * S)
    assert np.allclose(q[..., 0], (c - 1.0) ** 2 * q[..., 1], rtol=1e-12)
    T = S.copy()
    T[1, 2, 3, 5, 6] += 0.5
    one = oracle.drift_states(S, T)
    assert one[1, 2, 3, 0] == pytest.approx(0.25, rel=1e-12)
    mask = np.ones(one.shape[:-1], bool)
    mask[1, 2, 3] = False
    assert np.all(one[..., 0][mask] == 0.0)


def test_drift_states_matches_fused_sums():
    """The fused per-frame sums of the recurrence equal the sums taken from its
    own frame-end snapshots (the unfused way of Section 3.2)."""
    x = synth.workload_inputs("tiny")
    r = oracle.gdn_forward(x.q, x.k, x.v, x.g, x.beta, x.cu_seqlens, x.frame_len, snapshots=True)
    snaps = r["snapshots"]  # [F][H][d][d]
    before = np.concatenate([np.zeros_like(snaps[:1]), snaps[:-1]], axis=0)
    p = oracle.drift_states(before, snaps)
    assert np.allclose(p, r["partials"], rtol=1e-12, atol=1e-300)


# ---------------------------------------------------------------- write-magnitude signal
def _one_stream(T, H, d, rng, g=None, beta=None):
    q = to_bf16_bits(rng.standard_normal((T, H, d)))
    kk = rng.standard_normal((T, H, d))
    kk /= np.linalg.norm(kk, axis=-1, keepdims=True)
    k = to_bf16_bits(kk)
    v = to_bf16_bits(rng.standard_normal((T, H, d)))
    gg = np.full((T, H), -0.1, np.float32) if g is None else g
    bb = np.full((T, H), 0.7, np.float32) if beta is None else beta
    return q, k, v, gg.astype(np.float32), bb.astype(np.float32)


def test_write_signal_first_token_closed_form():
    """From a zero state the first write is beta v: ||e|| = beta ||v||."""
    rng = np.random.default_rng(21)
    q, k, v, g, b = _one_stream(1, 3, 16, rng)
    r = oracle.gdn_forward(q, k, v, g, b, np.array([0, 1], np.int32), 64)
    vv = bf16_bits_to_f64(v)[0]
    expect = b[0].astype(np.float64) * np.linalg.norm(vv, axis=-1)
    assert np.allclose(r["writes"][0, :, 0], expect, rtol=1e-14)
    assert np.all(r["writes"][0, :, 1] == 1.0)


def test_write_signal_equals_one_token_drift():
    """With g = 0 and unit keys a token's state change is the rank-one write
    e k^T, so ||Delta S||_F = ||e||: one-token frames make the frame drift num
    equal to the squared write sum (up to the bf16-rounded key norm)."""
    rng = np.random.default_rng(22)
    T, H, d = 40, 2, 32
    q, k, v, _, b = _one_stream(T, H, d, rng, g=np.zeros((T, H), np.float32),
                                beta=rng.uniform(0.1, 1.0, (T, H)))
    r = oracle.gdn_forward(q, k, v, np.zeros((T, H), np.float32), b, np.array([0, T], np.int32), 1)
    kn = np.linalg.norm(bf16_bits_to_f64(k), axis=-1)            # [T][H], 1 within bf16 rounding
    assert np.allclose(np.sqrt(r["partials"][..., 0]), r["writes"][..., 0] * kn, rtol=1e-12)
    assert np.all(r["writes"][..., 1] == 1.0)


def test_write_signal_zero_for_represented_pairs():
    """g = 0, beta = 1, exactly orthonormal keys: a frame that re-presents
    stored pairs writes nothing (e = 0 exactly)."""
    d, n = 64, 16
    keys = to_bf16_bits(synth.orthonormal_keys(d)[:n])   # bf16-exact rows, ||k|| = 1
    rng = np.random.default_rng(23)
    vals = to_bf16_bits(rng.standard_normal((n, 1, d)))
    kb = np.concatenate([keys, keys])[:, None, :]
    q = kb.copy()
    v = np.concatenate([vals, vals])
    T = 2 * n
    r = oracle.gdn_forward(q, kb, v, np.zeros((T, 1), np.float32), np.ones((T, 1), np.float32),
                           np.array([0, T], np.int32), n)
    assert r["writes"][0, 0, 0] > 0.0
    assert r["writes"][1, 0, 0] == 0.0
    assert r["writes"][1, 0, 1] == n


def test_write_mean_score_aggregation():
    """WRITE_MEAN averages sum / count over layers and heads."""
    p = np.zeros((2, 1, 2, 2))
    p[0, 0, 0] = (3.0, 2.0)
    p[0, 0, 1] = (1.0, 4.0)
    p[1, 0, 0] = (0.0, 2.0)
    p[1, 0, 1] = (10.0, 5.0)
    s = oracle.drift_scores(p, oracle.WRITE_MEAN)
    assert s[0] == pytest.approx((1.5 + 0.25 + 0.0 + 2.0) / 4, rel=1e-15)
