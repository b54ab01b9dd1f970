"""The whole-head sequential kernel (one workgroup per (stream, v-head), used
when B * H_v reaches 256 at d = 128) against the fp64 oracle (Section 3.2,
Eq. 2 and Eq. 3), on batches of many short streams that select it: ragged,
empty and one-token streams, a non-zero entry state, snapshots, every drift
aggregation, per-slice drift pairs, bf16 o and the write signal; frame
split and determinism bit for bit; P (which this kernel forms itself) under a
non-default output scale and extreme gates.  The full varlen workload runs
through it in test_gpu_full_size.py."""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_helpers import DEV, bf16_round, dev_bf16, dev_f32, drift_rel_err, lengths_of, rel_fro, run_gpu

pytestmark = pytest.mark.gpu
TOL_O, TOL_DRIFT = 2e-3, 1e-3


@pytest.fixture(scope="module")
def ds():
    import paper_2609_27470_amd as ds
    ds.lib()
    return ds


def _batch(B, seed, lo=0, hi=400, frame_len=128, H_k=2, H_v=4):
    rng = np.random.default_rng(seed)
    lens = [int(x) for x in rng.integers(lo, hi + 1, B)]
    lens[:6] = [0, 1, 63, 64, 65, 129][:min(6, B)]
    return synth.make_gdn_inputs(lens, H_k, H_v, 128, frame_len, novelty=True, config=5, layer=seed)


def _check(ds, gpu, ref):
    eo, es = rel_fro(gpu["o"], ref["o"]), rel_fro(gpu["S"], ref["S"])
    assert eo <= TOL_O and es <= TOL_O, (eo, es)
    p = torch.from_numpy(gpu["partials"].astype(np.float32)).to(DEV)[None]
    for mode in (oracle.LAYER_FROB, oracle.HEAD_MEAN, oracle.PER_HEAD):
        ed = drift_rel_err(ds.deltas_drift(p, mode).cpu().numpy(), oracle.drift_scores(ref["partials"][None], mode))
        assert ed <= TOL_DRIFT, (mode, ed)
    return eo, es


def test_wide_many_streams_against_oracle(ds):
    x = _batch(64, 1)
    assert x.B * x.H_v >= 256
    S0 = (np.random.default_rng(2).standard_normal((64, 4, 128, 128)) * 0.1).astype(np.float32).astype(np.float64)
    gpu = run_gpu(ds, x, state_in=S0, snapshots=True)
    ref = oracle.gdn_forward(x.q, x.k, x.v, x.g, x.beta, x.cu_seqlens, x.frame_len, S0=S0, snapshots=True)
    eo, es = _check(ds, gpu, ref)
    assert rel_fro(gpu["snapshots"], ref["snapshots"]) <= TOL_O
    assert np.array_equal(gpu["S"][0], S0[0])          # the empty stream passes its state through
    print(f"wide, 64 streams: o {eo:.2e} S {es:.2e}")


def test_wide_full_heads_one_frame_per_stream(ds):
    """8 streams x 32 v-heads (the varlen head count) of short streams, each one
    frame (frame_len = 0), bf16 o against the bf16-rounded oracle."""
    lens = [300, 1, 64, 517, 128, 0, 77, 1000]
    x = synth.make_gdn_inputs(lens, 16, 32, 128, 0, novelty=True, config=3, layer=7)
    gpu = run_gpu(ds, x, o_dtype=torch.bfloat16)
    ref = oracle.gdn_forward(x.q, x.k, x.v, x.g, x.beta, x.cu_seqlens, 0)
    assert rel_fro(gpu["o"], bf16_round(ref["o"])) <= TOL_O
    assert rel_fro(gpu["S"], ref["S"]) <= TOL_O
    p = torch.from_numpy(gpu["partials"].astype(np.float32)).to(DEV)[None]
    assert drift_rel_err(ds.deltas_drift(p, 0).cpu().numpy(), oracle.drift_scores(ref["partials"][None], 0)) <= TOL_DRIFT


def test_wide_per_slice_pairs(ds):
    """Per-slice drift pairs from the whole-head kernel: added per head in slice
    order they are its per-head pairs bit for bit; Eq. 3 over them matches the
    oracle."""
    x = _batch(64, 3)
    q, k, v, g, beta = dev_bf16(x.q), dev_bf16(x.k), dev_bf16(x.v), dev_f32(x.g), dev_f32(x.beta)
    lens = lengths_of(x)
    head = ds.gdn_chunk_fwd(q, k, v, g, beta, lens, 128)
    sl = ds.gdn_chunk_fwd(q, k, v, g, beta, lens, 128, drift_per_slice=True)
    torch.cuda.synchronize()
    ph = head["drift_partials"].cpu().numpy()
    ps = sl["drift_partials"].cpu().numpy().reshape(ph.shape[0], 4, 8, 2)
    acc = np.zeros(ph.shape, np.float32)
    for s_ in range(8):
        acc += ps[:, :, s_, :]
    assert np.array_equal(acc, ph)
    assert torch.equal(head["o"], sl["o"]) and torch.equal(head["state"], sl["state"])
    ref = oracle.gdn_forward(x.q, x.k, x.v, x.g, x.beta, x.cu_seqlens, 128)
    sc = ds.deltas_drift(sl["drift_partials"][None], ds.LAYER_FROB).cpu().numpy()
    assert drift_rel_err(sc, oracle.drift_scores(ref["partials"][None], oracle.LAYER_FROB)) <= TOL_DRIFT


def test_wide_write_signal(ds):
    x = _batch(64, 4)
    r = ds.gdn_chunk_fwd(dev_bf16(x.q), dev_bf16(x.k), dev_bf16(x.v), dev_f32(x.g), dev_f32(x.beta), lengths_of(x),
                         128, write_partials=True)
    torch.cuda.synchronize()
    ref = oracle.gdn_forward(x.q, x.k, x.v, x.g, x.beta, x.cu_seqlens, 128)
    got = r["write_partials"].cpu().numpy().astype(np.float64)
    assert np.array_equal(got[..., 1], ref["writes"][..., 1])
    rel = np.abs(got[..., 0] - ref["writes"][..., 0]) / np.maximum(ref["writes"][..., 0], 1e-30)
    assert rel.max() <= 1e-3, rel.max()


def test_wide_frame_split_and_determinism(ds):
    """64 streams of 3 frames of 128 tokens in one call == three calls of one
    frame each carrying the state, bit for bit; two equal calls agree."""
    B, F = 64, 128
    x = synth.make_gdn_inputs([3 * F] * B, 2, 4, 128, F, novelty=True, config=5, layer=9)
    whole = run_gpu(ds, x)
    again = run_gpu(ds, x)
    assert np.array_equal(whole["o"], again["o"]) and np.array_equal(whole["partials"], again["partials"])
    S = None
    for f in range(3):
        idx = np.concatenate([np.arange(b * 3 * F + f * F, b * 3 * F + (f + 1) * F) for b in range(B)])
        xf = synth.GdnInputs(x.q[idx], x.k[idx], x.v[idx], x.g[idx], x.beta[idx],
                             np.arange(B + 1, dtype=np.int32) * F, F, 2, 4, 128)
        part = run_gpu(ds, xf, state_in=S)
        assert np.array_equal(part["o"], whole["o"][idx])
        assert np.array_equal(part["partials"], whole["partials"].reshape(B, 3, 4, 2)[:, f])
        S = part["S"]
    assert np.array_equal(S, whole["S"])


def test_wide_output_scale_and_extreme_gates(ds):
    """P = scale D (.) tril(Q K^T) is formed by this kernel's loaders from the
    staged K and q tiles: a non-default output scale (1 / sqrt(d)), streams
    with near-unity decay (g = -1e-4), streams with decay so strong that
    2^(gamma_i - gamma_j) underflows inside a tile (g = -30), and beta = 0 on
    some tokens, against the oracle with the same scale."""
    x = _batch(64, 6, lo=1, hi=300)
    cu = x.cu_seqlens
    for b in range(64):
        s0, e0 = int(cu[b]), int(cu[b + 1])
        if b % 3 == 0:
            x.g[s0:e0] = -1e-4
        elif b % 3 == 1:
            x.g[s0:e0] = -30.0
        if b % 5 == 0:
            x.beta[s0:e0:7] = 0.0
    scale = 1.0 / np.sqrt(128.0)
    S0 = (np.random.default_rng(7).standard_normal((64, 4, 128, 128)) * 0.05).astype(np.float32).astype(np.float64)
    r = ds.gdn_chunk_fwd(dev_bf16(x.q), dev_bf16(x.k), dev_bf16(x.v), dev_f32(x.g), dev_f32(x.beta), lengths_of(x),
                         x.frame_len, state_in=dev_f32(S0), scale=scale)
    torch.cuda.synchronize()
    ref = oracle.gdn_forward(x.q, x.k, x.v, x.g, x.beta, x.cu_seqlens, x.frame_len, S0=S0, scale=scale)
    o = r["o"].cpu().numpy().astype(np.float64)
    assert np.all(np.isfinite(o))
    eo, es = rel_fro(o, ref["o"]), rel_fro(r["state"].cpu().numpy(), ref["S"])
    assert eo <= TOL_O and es <= TOL_O, (eo, es)
    p = r["drift_partials"][None]
    ed = drift_rel_err(ds.deltas_drift(p, oracle.PER_HEAD).cpu().numpy(),
                       oracle.drift_scores(ref["partials"][None], oracle.PER_HEAD))
    assert ed <= TOL_DRIFT, ed
    print(f"wide, scale 1/sqrt(d), extreme gates: o {eo:.2e} S {es:.2e} drift {ed:.2e}")


def test_wide_split_launches_full_heads(ds):
    """8 streams x 32 v-heads of unequal lengths, frames of two tiles: the call
    runs as whole heads up to the cut (tile 8: from there 4 streams are left)
    and half heads from it; fp32 o, a non-zero entry state, per-head drift
    pairs (added over the two half heads) and snapshots against the oracle,
    and the per-slice pairs of the same call adding up to the per-head pairs
    bit for bit."""
    lens = [2000, 1900, 700, 600, 500, 300, 100, 0]
    x = synth.make_gdn_inputs(lens, 16, 32, 128, 128, novelty=True, config=3, layer=11)
    S0 = (np.random.default_rng(13).standard_normal((8, 32, 128, 128)) * 0.05).astype(np.float32).astype(np.float64)
    gpu = run_gpu(ds, x, state_in=S0, snapshots=True)
    ref = oracle.gdn_forward(x.q, x.k, x.v, x.g, x.beta, x.cu_seqlens, x.frame_len, S0=S0, snapshots=True)
    eo, es = _check(ds, gpu, ref)
    assert rel_fro(gpu["snapshots"], ref["snapshots"]) <= TOL_O
    sl = ds.gdn_chunk_fwd(dev_bf16(x.q), dev_bf16(x.k), dev_bf16(x.v), dev_f32(x.g), dev_f32(x.beta), lens, 128,
                          state_in=dev_f32(S0), drift_per_slice=True)
    torch.cuda.synchronize()
    ph = gpu["raw"]["drift_partials"].cpu().numpy()
    ps = sl["drift_partials"].cpu().numpy().reshape(ph.shape[0], 32, 8, 2)
    acc = np.zeros(ph.shape, np.float32)
    for s_ in range(8):
        acc += ps[:, :, s_, :]
    assert np.array_equal(acc, ph)
    assert torch.equal(sl["o"], gpu["raw"]["o"]) and torch.equal(sl["state"], gpu["raw"]["state"])
    print(f"wide, split launches: o {eo:.2e} S {es:.2e}")


def test_wide_state_in_place(ds):
    """The state updated in place (state_out aliasing state_in) on the
    whole-head kernel, including the split into whole-head and half-head
    launches (the second reads the states the first wrote): bit-equal to the
    call with a separate output state."""
    lens = [2000, 1900, 700, 600, 500, 300, 100, 0]
    x = synth.make_gdn_inputs(lens, 16, 32, 128, 128, novelty=True, config=3, layer=12)
    S0 = (np.random.default_rng(14).standard_normal((8, 32, 128, 128)) * 0.05).astype(np.float32).astype(np.float64)
    a = run_gpu(ds, x, state_in=S0)
    b = run_gpu(ds, x, state_in=S0, in_place=True)
    assert np.array_equal(a["o"], b["o"])
    assert np.array_equal(a["S"], b["S"])
    assert np.array_equal(a["partials"], b["partials"])
