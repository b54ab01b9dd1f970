"""Streaming DeltaS with the paper's chunking and policy (Section 3.3,
Algorithm 1): variable chunks of 118-132 tokens, each one frame of every
linear-attention layer, sinks + recent window + 4 spans, and question-time
save/restore.

Parity: after every chunk the GPU chunk score matches the oracle's (fp64
recurrence per layer chained over the chunks, Eq. 3 over the layers) within
1e-3; every layer's output o of every chunk and the final states match within
2e-3; the cache (positions, chunk ids, K/V rows) equals the oracle selection
replayed on the GPU's own scores, bit for bit.  Both cache forms (rows
compacted in place, slot-indexed) are checked, eager and as a replayed HIP
graph, on a small shape and on the benchmark's streamed shape.

Save/restore: a stream that answers a question in the middle (extra tokens
and decode steps) and restores afterwards ends bit-identical to one that
never stopped."""
import math

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_helpers import DEV, dev_bf16, dev_f32, rel_fro, drift_rel_err

pytestmark = pytest.mark.gpu

L, H_K, H_V, D = 3, 2, 4, 64
KV_L, ROW = 2, 64
M, N_SINK, N_WIN, N_BKT = 640, 4, 256, 4


@pytest.fixture(scope="module")
def ds():
    import paper_2609_27470_amd as ds
    ds.lib()
    return ds


def chunk_lengths(n, seed=3):
    rng = np.random.default_rng(seed)
    return [int(x) for x in rng.integers(118, 133, n)]


def layer_streams(total, seed_cfg=97):
    return [synth.make_gdn_inputs([total], H_K, H_V, D, 128, True, config=seed_cfg, layer=l) for l in range(L)]


def chunk_inputs(xs, a, b):
    return [(dev_bf16(x.q[a:b]), dev_bf16(x.k[a:b]), dev_bf16(x.v[a:b]), dev_f32(x.g[a:b]), dev_f32(x.beta[a:b]))
            for x in xs]


def kv_rows(pos0, T):
    p = torch.arange(pos0, pos0 + T, dtype=torch.int64, device=DEV)
    k = torch.stack([synth.kv_row_bits_torch(l, 0, p, ROW) for l in range(KV_L)])
    v = torch.stack([synth.kv_row_bits_torch(l, 1, p, ROW) for l in range(KV_L)])
    return k, v


def new_stream(indexed=False, o_dtype=torch.bfloat16):
    from paper_2609_27470_amd.streaming import DeltaSStream
    return DeltaSStream(L, H_K, H_V, D, KV_L, ROW, M, 132, 128, N_SINK, N_WIN, N_BKT, device=DEV, indexed=indexed,
                        o_dtype=o_dtype)


class Fro:
    def __init__(self):
        self.num = self.den = 0.0

    def add(self, got, ref):
        self.num += float(np.sum((np.asarray(got, np.float64) - ref) ** 2))
        self.den += float(np.sum(np.asarray(ref, np.float64) ** 2))

    def err(self):
        return math.sqrt(self.num / self.den)


@pytest.mark.parametrize("indexed", [False, True])
def test_stream_matches_oracle_replay(ds, indexed):
    lens = chunk_lengths(24)
    xs = layer_streams(sum(lens))
    s = new_stream(indexed, o_dtype=torch.float32)
    S_ref = [np.zeros((1, H_V, D, D)) for _ in range(L)]
    ref_pos, ref_chunk = np.zeros(0, np.int64), np.zeros(0, np.int64)
    fo = Fro()
    off = 0
    for c, T in enumerate(lens):
        k_rows, v_rows = kv_rows(off, T)
        s.step(chunk_inputs(xs, off, off + T), k_rows, v_rows)
        parts = []
        for l, x in enumerate(xs):
            r = oracle.gdn_forward(x.q[off:off + T], x.k[off:off + T], x.v[off:off + T], x.g[off:off + T],
                                   x.beta[off:off + T], np.array([0, T], np.int32), 0, S0=S_ref[l])
            S_ref[l] = r["S"]
            parts.append(r["partials"])
            got = s.o[l, :T].cpu().numpy()
            assert rel_fro(got, r["o"]) <= 2e-3, (c, l)
            fo.add(got, r["o"])
        ref_score = oracle.drift_scores(np.stack(parts), oracle.LAYER_FROB)
        gpu_scores = s.scores[:c + 1].cpu().numpy()
        assert drift_rel_err(gpu_scores[c:c + 1], ref_score) <= 1e-3, (c, gpu_scores[c], ref_score)
        ref_pos = np.concatenate([ref_pos, np.arange(off, off + T)])
        ref_chunk = np.concatenate([ref_chunk, np.full(T, c)])
        if len(ref_pos) > M:
            keep = oracle.select_keep(ref_chunk, ref_pos, gpu_scores, len(ref_pos), M, N_SINK, N_WIN, N_BKT)
            ref_pos, ref_chunk = ref_pos[keep], ref_chunk[keep]
        off += T
        n = s.length
        assert n == len(ref_pos)
        assert np.array_equal(s.pos[:n].cpu().numpy(), ref_pos)
        assert np.array_equal(s.chunk_id[:n].cpu().numpy(), ref_chunk)
    ep = torch.as_tensor(ref_pos, device=DEV)
    kl, vl = s.logical_rows()
    for l in range(KV_L):
        assert torch.equal(kl[l], synth.kv_row_bits_torch(l, 0, ep, ROW))
        assert torch.equal(vl[l], synth.kv_row_bits_torch(l, 1, ep, ROW))
    for l in range(L):
        assert rel_fro(s.state[l].cpu().numpy(), S_ref[l]) <= 2e-3
    assert fo.err() <= 2e-3
    s.check()
    print(f"streamed o over {len(lens)} chunks x {L} layers: {fo.err():.2e}")


def test_question_save_restore_is_transparent(ds):
    lens = chunk_lengths(16, seed=4)
    xs = layer_streams(sum(lens) + 200, seed_cfg=98)
    offs = np.concatenate([[0], np.cumsum(lens)])
    a, b = new_stream(), new_stream()
    for c, T in enumerate(lens):
        k_rows, v_rows = kv_rows(int(offs[c]), T)
        a.step(chunk_inputs(xs, int(offs[c]), int(offs[c]) + T), k_rows, v_rows)
    stop = 9
    for c in range(stop):
        T = lens[c]
        k_rows, v_rows = kv_rows(int(offs[c]), T)
        b.step(chunk_inputs(xs, int(offs[c]), int(offs[c]) + T), k_rows, v_rows)
    snap = b.save()
    # the question: a chunk of other tokens, then decode steps on every layer
    q0 = int(offs[-1])
    k_rows, v_rows = kv_rows(10 ** 6, 40)
    b.step(chunk_inputs(xs, q0, q0 + 40), k_rows, v_rows)
    for t in range(5):
        for l, x in enumerate(xs):
            i = slice(q0 + 40 + t, q0 + 41 + t)
            ds.gdn_decode_step(dev_bf16(x.q[i]), dev_bf16(x.k[i]), dev_bf16(x.v[i]), dev_f32(x.g[i]),
                               dev_f32(x.beta[i]), state_in=b.state[l], state_out=b.state[l])
    b.restore(snap)
    for c in range(stop, len(lens)):
        T = lens[c]
        k_rows, v_rows = kv_rows(int(offs[c]), T)
        b.step(chunk_inputs(xs, int(offs[c]), int(offs[c]) + T), k_rows, v_rows)
    torch.cuda.synchronize()
    assert a.length == b.length and a.n_chunks == b.n_chunks and a.next_pos == b.next_pos
    n = a.length
    assert torch.equal(a.state, b.state)
    assert torch.equal(a.pos[:n], b.pos[:n]) and torch.equal(a.chunk_id[:n], b.chunk_id[:n])
    assert torch.equal(a.k[:, :n], b.k[:, :n]) and torch.equal(a.v[:, :n], b.v[:, :n])
    assert torch.equal(a.scores[:a.n_chunks], b.scores[:b.n_chunks])


def test_graph_replays_match_eager_steps(ds):
    """The captured graphs (all layers + score, lengths read on the device; one
    for chunks of at most two tiles, one for the full capacity) replayed for
    chunks of different lengths on both sides of 128 tokens, with eager work and
    synchronisations between replays, gives the eager steps' results bit for
    bit after every chunk."""
    lens = chunk_lengths(12, seed=5)
    xs = layer_streams(sum(lens), seed_cfg=99)
    a, b = new_stream(), new_stream()
    b.capture_graph()
    off = 0
    for c, T in enumerate(lens):
        k_rows, v_rows = kv_rows(off, T)
        ins = chunk_inputs(xs, off, off + T)
        a.step(ins, k_rows, v_rows)
        for i, buf in enumerate(b.inputs):
            for l in range(L):
                buf[l, :T].copy_(ins[l][i])
        b.step_inputs(T, k_rows, v_rows)
        torch.cuda.synchronize()
        n = a.length
        assert b.length == n
        assert torch.equal(a.state, b.state), c
        assert torch.equal(a.scores[:c + 1], b.scores[:c + 1]), c
        assert torch.equal(a.pos[:n], b.pos[:n]) and torch.equal(a.chunk_id[:n], b.chunk_id[:n])
        assert torch.equal(a.k[:, :n], b.k[:, :n])
        off += T


def test_indexed_stream_matches_gather_stream(ds):
    """The slot-indexed session (no K/V row moved at eviction, new chunks
    written into freed rows) keeps the same tokens, scores and states as the
    order-preserving one after every chunk, and its logical rows are the
    gathered cache bit for bit; save/restore is transparent in it too."""
    from paper_2609_27470_amd.streaming import DeltaSStream
    lens = chunk_lengths(14, seed=6)
    xs = layer_streams(sum(lens) + 64, seed_cfg=100)
    a = new_stream(indexed=False)
    b = DeltaSStream(L, H_K, H_V, D, KV_L, ROW, M, 132, 128, N_SINK, N_WIN, N_BKT, device=DEV, indexed=True)
    off = 0
    snap = None
    for c, T in enumerate(lens):
        k_rows, v_rows = kv_rows(off, T)
        ins = chunk_inputs(xs, off, off + T)
        a.step(ins, k_rows, v_rows)
        b.step(ins, k_rows, v_rows)
        if c == 8:
            snap = b.save()
            q0 = sum(lens)
            qk, qv = kv_rows(10 ** 6, 40)
            b.step(chunk_inputs(xs, q0, q0 + 40), qk, qv)
            b.restore(snap)
        torch.cuda.synchronize()
        n = a.length
        assert b.length == n
        assert torch.equal(a.state, b.state), c
        assert torch.equal(a.scores[:c + 1], b.scores[:c + 1])
        assert torch.equal(a.pos[:n], b.pos[:n]) and torch.equal(a.chunk_id[:n], b.chunk_id[:n])
        ka, va = a.logical_rows()
        kb, vb = b.logical_rows()
        assert torch.equal(ka, kb) and torch.equal(va, vb), c
        off += T


# ---------------------------------------------------------------------------
# the benchmark's streamed shape: 24 linear-attention layers of 16 qk / 32 v
# heads (d = 128), 8 full-attention layers of 8 KV heads x 256, budget 16384,
# the paper's policy, starting from a full cache of 128 earlier chunks
BL, BH_K, BH_V, BD = 24, 16, 32, 128
BKV_L, BROW, BM = 8, 8 * 256, 16384
PRE_CHUNK = 128


def _bench_kv_rows(pos0, T):
    p = torch.arange(pos0, pos0 + T, dtype=torch.int64, device=DEV)
    return (torch.stack([synth.kv_row_bits_torch(l, 0, p, BROW) for l in range(BKV_L)]),
            torch.stack([synth.kv_row_bits_torch(l, 1, p, BROW) for l in range(BKV_L)]))


@pytest.mark.timeout(300)
@pytest.mark.parametrize("mode", ["eager_gather", "graph_indexed"])
def test_stream_bench_shape(ds, mode):
    """Six chunks of 118-132 tokens through the benchmark's streamed shape,
    from a cache pre-filled with 16384 tokens (128 chunks with given scores):
    every chunk's score, every layer's o (fp32) and the final states against
    the oracle chained per layer; every eviction against the oracle selection
    replayed on the GPU's scores; the cached rows at the end against the rows
    of the kept positions."""
    from paper_2609_27470_amd.streaming import DeltaSStream
    lens = chunk_lengths(6, seed=21)
    total = sum(lens)
    xs = [synth.make_gdn_inputs([total], BH_K, BH_V, BD, 128, True, config=96, layer=l) for l in range(BL)]
    indexed = mode.endswith("indexed")
    s = DeltaSStream(BL, BH_K, BH_V, BD, BKV_L, BROW, BM, 132, BM // PRE_CHUNK + 16, 4, 1024, 4, device=DEV,
                     indexed=indexed, o_dtype=torch.float32)
    pre_scores = torch.rand(BM // PRE_CHUNK, generator=torch.Generator().manual_seed(5)).to(DEV)
    pk, pv = _bench_kv_rows(0, BM)
    s.k[:, :BM].copy_(pk)
    s.v[:, :BM].copy_(pv)
    del pk, pv
    s.pos[:BM] = torch.arange(BM, dtype=torch.int32, device=DEV)
    s.chunk_id[:BM] = torch.arange(BM, dtype=torch.int32, device=DEV) // PRE_CHUNK
    s.scores[:BM // PRE_CHUNK] = pre_scores
    s.length, s.n_chunks, s.next_pos = BM, BM // PRE_CHUNK, BM
    if indexed:
        s.slot[:BM] = torch.arange(BM, dtype=torch.int32, device=DEV)
        s.free = torch.arange(BM, s.capacity, dtype=torch.int32, device=DEV)
    if mode.startswith("graph"):
        s.capture_graph()
    ref_pos = np.arange(BM)
    ref_chunk = np.arange(BM) // PRE_CHUNK
    S_ref = [np.zeros((1, BH_V, BD, BD)) for _ in range(BL)]
    fo = Fro()
    off = 0
    for c, T in enumerate(lens):
        k_rows, v_rows = _bench_kv_rows(BM + off, T)
        ins = [(dev_bf16(x.q[off:off + T]), dev_bf16(x.k[off:off + T]), dev_bf16(x.v[off:off + T]),
                dev_f32(x.g[off:off + T]), dev_f32(x.beta[off:off + T])) for x in xs]
        if mode.startswith("graph"):
            for i, buf in enumerate(s.inputs):
                for l in range(BL):
                    buf[l, :T].copy_(ins[l][i])
            s.step_inputs(T, k_rows, v_rows)
        else:
            s.step(ins, k_rows, v_rows)
        parts = []
        for l, x in enumerate(xs):
            r = oracle.gdn_forward(x.q[off:off + T], x.k[off:off + T], x.v[off:off + T], x.g[off:off + T],
                                   x.beta[off:off + T], np.array([0, T], np.int32), 0, S0=S_ref[l])
            S_ref[l] = r["S"]
            parts.append(r["partials"])
            fo.add(s.o[l, :T].cpu().numpy(), r["o"])
        ref_score = oracle.drift_scores(np.stack(parts), oracle.LAYER_FROB)
        gpu_scores = s.scores[:s.n_chunks].cpu().numpy()
        assert drift_rel_err(gpu_scores[-1:], ref_score) <= 1e-3, (c, gpu_scores[-1], ref_score)
        ref_pos = np.concatenate([ref_pos, np.arange(BM + off, BM + off + T)])
        ref_chunk = np.concatenate([ref_chunk, np.full(T, BM // PRE_CHUNK + c)])
        keep = oracle.select_keep(ref_chunk, ref_pos, gpu_scores, len(ref_pos), BM, 4, 1024, 4)
        ref_pos, ref_chunk = ref_pos[keep], ref_chunk[keep]
        off += T
        n = s.length
        assert n == len(ref_pos) == BM
        assert np.array_equal(s.pos[:n].cpu().numpy(), ref_pos), c
        assert np.array_equal(s.chunk_id[:n].cpu().numpy(), ref_chunk), c
    assert fo.err() <= 2e-3, fo.err()
    for l in range(BL):
        assert rel_fro(s.state[l].cpu().numpy(), S_ref[l]) <= 2e-3, l
    kl, vl = s.logical_rows()
    ep = torch.as_tensor(ref_pos, device=DEV)
    for l in range(BKV_L):
        assert torch.equal(kl[l], synth.kv_row_bits_torch(l, 0, ep, BROW)), l
        assert torch.equal(vl[l], synth.kv_row_bits_torch(l, 1, ep, BROW)), l
    print(f"bench streamed shape ({mode}): o {fo.err():.2e} over {len(lens)} chunks x {BL} layers")
