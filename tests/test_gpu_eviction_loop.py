"""The eviction loop (Algorithm 1 over the stack, Section 3.3) scaled down in
heads: 24 linear-attention layers of one GQA group (1 qk / 2 v heads,
d = 128), 40 frames of 1024 tokens drawn from a per-layer pool of 8 frames
(stream frame f at layer l reads pool frame (f + 4 l) mod 8, which keeps the
novel frames aligned across layers), fp32 state carried in place, drift
pairs per state slice pooled by Eq. 3 over the layers, and after every frame
the frame's K/V rows of 8 full-attention layers (8 KV heads x 256 bf16)
appended and kv_evict_topk run at budget 16384 with whole chunks kept by
drift, ties to newer (24 events).

Against an oracle replay: every frame's score within 1e-3 of Eq. 3 over the
fp64 recurrence of each layer's stream; after every event the positions and
chunk ids equal the oracle selection replayed on the GPU's scores, bit for
bit; the final cache rows are the rows of the kept positions; final states
and a sample of the outputs within 2e-3."""
import math

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_helpers import DEV, dev_bf16, dev_f32, drift_rel_err, rel_fro

pytestmark = pytest.mark.gpu

L, H_K, H_V, D, FRAME, POOL, FRAMES = 24, 1, 2, 128, 1024, 8, 40
KV_L, ROW, M = 8, 8 * 256, 16384
CAP = M + FRAME


@pytest.fixture(scope="module")
def ds():
    import paper_2609_27470_amd as ds
    ds.lib()
    return ds


def _pool_index(f, l):
    return synth.pool_frame_index(f, l, POOL)


@pytest.mark.timeout(600)
def test_eviction_loop_against_oracle_replay(ds):
    pools = [synth.make_gdn_inputs([POOL * FRAME], H_K, H_V, D, FRAME, True, config=4, layer=l) for l in range(L)]
    dev_pools = [tuple(t(a) for t, a in ((dev_bf16, x.q), (dev_bf16, x.k), (dev_bf16, x.v), (dev_f32, x.g),
                                         (dev_f32, x.beta))) for x in pools]
    # the oracle's view: each layer's stream is its pool frames in stream order
    streams = []
    for l, x in enumerate(pools):
        idx = np.concatenate([np.arange(FRAME) + _pool_index(f, l) * FRAME for f in range(FRAMES)])
        streams.append(tuple(a[idx] for a in (x.q, x.k, x.v, x.g, x.beta)))
    # one oracle pass per layer, layers in parallel threads (each pass has only
    # two (stream, v-head) units to spread over cores)
    from concurrent.futures import ThreadPoolExecutor
    with ThreadPoolExecutor(max_workers=8) as ex:
        refs = list(ex.map(lambda s: oracle.gdn_forward(*s, np.array([0, FRAMES * FRAME], np.int32), FRAME,
                                                        n_threads=2), streams))
    ref_scores = oracle.drift_scores(np.stack([r["partials"] for r in refs]), oracle.LAYER_FROB)

    state = torch.zeros((L, 1, H_V, D, D), dtype=torch.float32, device=DEV)
    parts = torch.zeros((L, 1, H_V * D // 16, 2), dtype=torch.float32, device=DEV)
    o = torch.empty((FRAME, H_V, D), dtype=torch.float32, device=DEV)
    table = torch.zeros(FRAMES, dtype=torch.float32, device=DEV)
    k_cache = [torch.zeros((CAP, ROW), dtype=torch.int16, device=DEV) for _ in range(KV_L)]
    v_cache = [torch.zeros((CAP, ROW), dtype=torch.int16, device=DEV) for _ in range(KV_L)]
    pos = torch.zeros(CAP, dtype=torch.int32, device=DEV)
    chunk = torch.zeros(CAP, dtype=torch.int32, device=DEV)
    ws = None
    kv_ws = None
    fail = torch.zeros(1, dtype=torch.int32, device=DEV)
    n = 0
    ref_pos = np.zeros(0, np.int64)
    ref_chunk = np.zeros(0, np.int64)
    num = den = 0.0
    events = 0
    for f in range(FRAMES):
        for l in range(L):
            s = slice(_pool_index(f, l) * FRAME, (_pool_index(f, l) + 1) * FRAME)
            q, k, v, g, b = dev_pools[l]
            r = ds.gdn_chunk_fwd(q[s], k[s], v[s], g[s], b[s], [FRAME], FRAME, state_in=state[l], state_out=state[l],
                                 o=o, drift_partials=parts[l], workspace=ws, drift_per_slice=True)
            ws = r["workspace"]
            if f % 5 == 4:
                got = o.cpu().numpy()
                ref_o = refs[l]["o"][f * FRAME:(f + 1) * FRAME]
                num += float(np.sum((got - ref_o) ** 2))
                den += float(np.sum(ref_o ** 2))
        ds.deltas_drift(parts, ds.LAYER_FROB, scores=table[f:f + 1])
        # append the frame's rows, positions f * 1024 + i, chunk id f
        p = torch.arange(f * FRAME, (f + 1) * FRAME, dtype=torch.int64, device=DEV)
        for kv in range(KV_L):
            k_cache[kv][n:n + FRAME] = synth.kv_row_bits_torch(kv, 0, p, ROW)
            v_cache[kv][n:n + FRAME] = synth.kv_row_bits_torch(kv, 1, p, ROW)
        pos[n:n + FRAME] = p.to(torch.int32)
        chunk[n:n + FRAME] = f
        n += FRAME
        ref_pos = np.concatenate([ref_pos, np.arange(f * FRAME, (f + 1) * FRAME)])
        ref_chunk = np.concatenate([ref_chunk, np.full(FRAME, f)])
        if n > M:
            n, kv_ws = ds.kv_evict_topk(k_cache, v_cache, pos, chunk, table[:f + 1], n, M, 0, 0, 1, workspace=kv_ws)
            torch.maximum(fail, ds.kv_outcome_word(kv_ws), out=fail)
            gpu_scores = table[:f + 1].cpu().numpy()
            keep = oracle.select_keep(ref_chunk, ref_pos, gpu_scores, len(ref_pos), M, 0, 0, 1)
            ref_pos, ref_chunk = ref_pos[keep], ref_chunk[keep]
            events += 1
            assert np.array_equal(pos[:n].cpu().numpy(), ref_pos), f
            assert np.array_equal(chunk[:n].cpu().numpy(), ref_chunk), f
    torch.cuda.synchronize()
    assert events == FRAMES - 16 and int(fail.item()) == 0
    assert drift_rel_err(table.cpu().numpy(), ref_scores) <= 1e-3
    for l in range(L):
        assert rel_fro(state[l].cpu().numpy(), refs[l]["S"]) <= 2e-3, l
    assert math.sqrt(num / den) <= 2e-3
    ep = torch.as_tensor(ref_pos, device=DEV)
    for kv in range(KV_L):
        assert torch.equal(k_cache[kv][:n], synth.kv_row_bits_torch(kv, 0, ep, ROW)), kv
        assert torch.equal(v_cache[kv][:n], synth.kv_row_bits_torch(kv, 1, ep, ROW)), kv
    print(f"eviction loop: {events} events, o {math.sqrt(num / den):.2e}, kept chunks {sorted(set(ref_chunk.tolist()))}")
