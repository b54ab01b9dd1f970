"""Calls of at most two tiles on the per-slice sequential kernel (most
streamed chunks) form their prep inside it, in one launch, unless the per-head drift
sums are asked for (their slice counters are cleared by the separate prep
pass).  The same inputs through both paths give the same bits, and both match
the fp64 oracle (Section 3.2, Eq. 2; drift sums of Eq. 3); longer calls (up to
17 tiles, a packed pair) take the prep pass on every call and are held to the
same comparisons."""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_helpers import DEV, bf16_round, dev_bf16, dev_f32, drift_rel_err, rel_fro

pytestmark = pytest.mark.gpu

TOL_O = 2e-3
TOL_DRIFT = 1e-3


@pytest.fixture(scope="module")
def ds():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_27470_amd as m
    return m


# (lengths, H_k, H_v, d, frame_len): one-launch cases have (T + 63 B) / 64 <= 2
# tiles; the others (three tiles and up, to 1025 tokens) take the two launches
# on every call
CASES = [
    ([1], 2, 4, 128, 64),
    ([63], 2, 4, 128, 0),
    ([64], 2, 4, 128, 64),
    ([65], 2, 4, 128, 128),
    ([118], 16, 32, 128, 0),
    ([125], 16, 32, 128, 128),
    ([128], 2, 4, 128, 64),
    ([100], 2, 2, 64, 0),
    ([1, 1], 2, 2, 64, 64),
    ([132], 16, 32, 128, 0),
    ([129], 2, 4, 128, 64),
    ([1024], 16, 32, 128, 1024),
    ([1000], 2, 4, 128, 256),
    ([511], 2, 2, 64, 128),
    ([600, 300], 2, 4, 128, 256),
    ([1025], 2, 4, 128, 1024),
    ([520], 2, 2, 64, 0),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c[0])) + f"_h{c[2]}_d{c[3]}_f{c[4]}")
def test_one_launch_matches_two_launches_and_oracle(ds, case):
    lens, H_k, H_v, d, frame_len = case
    x = synth.make_gdn_inputs(lens, H_k, H_v, d, frame_len, novelty=True, config=1)
    rng = np.random.default_rng(sum(lens) + d)
    S0 = (rng.standard_normal((len(lens), H_v, d, d)) * 0.1).astype(np.float32).astype(np.float64)
    q, k, v = dev_bf16(x.q), dev_bf16(x.k), dev_bf16(x.v)
    g, beta, s_in = dev_f32(x.g), dev_f32(x.beta), dev_f32(S0)
    two = ds.gdn_chunk_fwd(q, k, v, g, beta, lens, frame_len, state_in=s_in)                        # per-head sums
    one = ds.gdn_chunk_fwd(q, k, v, g, beta, lens, frame_len, state_in=s_in, drift_per_slice=True)  # one launch
    bare = ds.gdn_chunk_fwd(q, k, v, g, beta, lens, frame_len, state_in=s_in, drift_partials=False)
    torch.cuda.synchronize()
    for r in (one, bare):
        assert torch.equal(r["o"], two["o"]) and torch.equal(r["state"], two["state"])
    ph = two["drift_partials"].cpu().numpy()
    ps = one["drift_partials"].cpu().numpy().reshape(ph.shape[0], H_v, d // 16, 2)
    acc = np.zeros(ph.shape, np.float32)
    for s_ in range(d // 16):
        acc += ps[:, :, s_, :]
    assert np.array_equal(acc, ph)
    ref = oracle.gdn_forward(x.q, x.k, x.v, x.g, x.beta, x.cu_seqlens, frame_len, S0=S0)
    assert rel_fro(one["o"].cpu().numpy().astype(np.float64), ref["o"]) <= TOL_O
    assert rel_fro(one["state"].cpu().numpy().astype(np.float64), ref["S"]) <= TOL_O
    if ph.shape[0] > 0:
        sc = ds.deltas_drift(one["drift_partials"][None], ds.LAYER_FROB).cpu().numpy()
        rs = oracle.drift_scores(ref["partials"][None], oracle.LAYER_FROB)
        assert drift_rel_err(sc, rs) <= TOL_DRIFT


def test_one_launch_bf16_snapshots_and_unreached_frames(ds):
    """bf16 o and frame snapshots through the one-launch path; the pairs of
    frames the device lengths do not reach read zero."""
    lens = [60]
    x = synth.make_gdn_inputs(lens, 2, 4, 128, 64, novelty=True, config=1)
    q, k, v = dev_bf16(x.q), dev_bf16(x.k), dev_bf16(x.v)
    g, beta = dev_f32(x.g), dev_f32(x.beta)
    r = ds.gdn_chunk_fwd(q, k, v, g, beta, lens, 64, o_dtype=torch.bfloat16, snapshots=True, drift_per_slice=True)
    torch.cuda.synchronize()
    ref = oracle.gdn_forward(x.q, x.k, x.v, x.g, x.beta, x.cu_seqlens, 64, snapshots=True)
    assert rel_fro(r["o"].float().cpu().numpy().astype(np.float64), bf16_round(ref["o"])) <= TOL_O
    assert rel_fro(r["snapshots"].cpu().numpy().astype(np.float64), ref["snapshots"]) <= TOL_O
    # capacity of 128 tokens (2 frames of 64), device lengths of 60 (1 frame)
    cap = [128]
    pad = lambda a: torch.cat([a, torch.zeros((128 - a.shape[0],) + tuple(a.shape[1:]), dtype=a.dtype, device=DEV)])
    cu = torch.tensor(np.asarray(x.cu_seqlens, np.int32), device=DEV)
    dp = torch.full((2, 4 * 8, 2), float("nan"), dtype=torch.float32, device=DEV)
    o2 = ds.gdn_chunk_fwd(pad(q), pad(k), pad(v), pad(g), pad(beta), cap, 64, cu_seqlens=cu, drift_partials=dp,
                          drift_per_slice=True)
    torch.cuda.synchronize()
    got = dp.cpu().numpy()
    assert np.array_equal(got[:1], r["drift_partials"].cpu().numpy())
    assert np.all(got[1:] == 0.0)
    assert torch.equal(o2["state"], r["state"])


def test_capacity_call_bf16_snapshots_and_unreached_frames(ds):
    """A call sized for 1024 tokens with 700 on the device (the prep pass and
    the sequential kernel read the length on the device): bf16 o and snapshots
    against the oracle, the pairs of frames the device length does not reach
    zero, and the result bit-equal to the call sized to the device length."""
    lens = [700]
    x = synth.make_gdn_inputs(lens, 2, 4, 128, 256, novelty=True, config=1)
    q, k, v = dev_bf16(x.q), dev_bf16(x.k), dev_bf16(x.v)
    g, beta = dev_f32(x.g), dev_f32(x.beta)
    r = ds.gdn_chunk_fwd(q, k, v, g, beta, lens, 256, o_dtype=torch.bfloat16, snapshots=True, drift_per_slice=True)
    torch.cuda.synchronize()
    ref = oracle.gdn_forward(x.q, x.k, x.v, x.g, x.beta, x.cu_seqlens, 256, snapshots=True)
    assert rel_fro(r["o"].float().cpu().numpy().astype(np.float64), bf16_round(ref["o"])) <= TOL_O
    assert rel_fro(r["snapshots"].cpu().numpy().astype(np.float64), ref["snapshots"]) <= TOL_O
    cap = [1024]
    pad = lambda a: torch.cat([a, torch.zeros((1024 - a.shape[0],) + tuple(a.shape[1:]), dtype=a.dtype, device=DEV)])
    cu = torch.tensor(np.asarray(x.cu_seqlens, np.int32), device=DEV)
    dp = torch.full((4, 4 * 8, 2), float("nan"), dtype=torch.float32, device=DEV)
    o2 = ds.gdn_chunk_fwd(pad(q), pad(k), pad(v), pad(g), pad(beta), cap, 256, cu_seqlens=cu, drift_partials=dp,
                          o_dtype=torch.bfloat16, drift_per_slice=True)
    torch.cuda.synchronize()
    got = dp.cpu().numpy()
    assert np.array_equal(got[:3], r["drift_partials"].cpu().numpy())
    assert np.all(got[3:] == 0.0)
    assert torch.equal(o2["state"], r["state"]) and torch.equal(o2["o"][:700], r["o"])
