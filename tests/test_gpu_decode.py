"""GPU parity of gdn_decode_step (one token per stream of Eq. 2, batched over
streams) against the fp64 oracle recurrence: single steps from random states,
chains of steps, and a prefill by gdn_chunk_fwd continued by decode steps.

The decode step runs in fp32 (no matrix cores): its error against the fp64
recurrence is a few fp32 roundings of d-term dot products (~1e-6 relative), so
the bar here is 1e-5 relative Frobenius, tighter than the 2e-3 of the chunked
forward (whose operands are fp16)."""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_helpers import DEV, dev_bf16, dev_f32, rel_fro, bf16_round

pytestmark = pytest.mark.gpu
TOL = 1e-5


@pytest.fixture(scope="module")
def ds():
    import paper_2609_27470_amd as ds
    ds.lib()
    return ds


def tokens(B, H_k, H_v, d, seed, gates="standard"):
    """B one-token streams, packed: q, k [B][H_k][d], v [B][H_v][d], g, beta [B][H_v]."""
    return synth.make_gdn_inputs([1] * B, H_k, H_v, d, 0, False, config=90 + seed, gates=gates)


def random_state(B, H_v, d, seed, scale=0.3):
    rng = np.random.default_rng(seed)
    return (scale * rng.standard_normal((B, H_v, d, d))).astype(np.float32)


def decode(ds, x, state, o_dtype=torch.float32, in_place=False):
    B, H_k, d = x.q.shape
    H_v = x.v.shape[1]
    s_in = None if state is None else dev_f32(state)
    r = ds.gdn_decode_step(dev_bf16(x.q), dev_bf16(x.k), dev_bf16(x.v), dev_f32(x.g), dev_f32(x.beta),
                           state_in=s_in, state_out=s_in if in_place else None, o_dtype=o_dtype)
    torch.cuda.synchronize()
    return r["o"].float().cpu().numpy().astype(np.float64), r["state"].cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("d,H_k,H_v", [(64, 2, 2), (128, 2, 4), (128, 16, 32)])
def test_one_step_matches_oracle(ds, d, H_k, H_v):
    B = 8 if H_v < 32 else 64
    x = tokens(B, H_k, H_v, d, seed=d + H_v)
    S0 = random_state(B, H_v, d, seed=d)
    o, S = decode(ds, x, S0)
    ref = oracle.gdn_forward(x.q, x.k, x.v, x.g, x.beta, x.cu_seqlens, 0, S0=S0.astype(np.float64))
    eo, es = rel_fro(o, ref["o"]), rel_fro(S, ref["S"])
    print(f"decode d={d} H=({H_k},{H_v}) B={B}: o {eo:.2e} S {es:.2e}")
    assert eo <= TOL and es <= TOL


def test_zero_state_bf16_output_and_in_place(ds):
    B, H_k, H_v, d = 5, 2, 4, 128
    x = tokens(B, H_k, H_v, d, seed=3)
    o, S = decode(ds, x, None, o_dtype=torch.bfloat16)
    ref = oracle.gdn_forward(x.q, x.k, x.v, x.g, x.beta, x.cu_seqlens, 0)
    assert rel_fro(o, bf16_round(ref["o"])) <= 2e-3
    assert rel_fro(S, ref["S"]) <= TOL
    S0 = random_state(B, H_v, d, seed=4)
    o2, S2 = decode(ds, x, S0, in_place=True)
    ref2 = oracle.gdn_forward(x.q, x.k, x.v, x.g, x.beta, x.cu_seqlens, 0, S0=S0.astype(np.float64))
    assert rel_fro(o2, ref2["o"]) <= TOL and rel_fro(S2, ref2["S"]) <= TOL


def test_no_decay_no_write_keeps_state_bits(ds):
    """g = 0, beta = 0: alpha = 1 and e = 0, so S' = S bit for bit and o = S q."""
    B, H_k, H_v, d = 4, 2, 4, 64
    x = tokens(B, H_k, H_v, d, seed=5)
    x.g[:] = 0.0
    x.beta[:] = 0.0
    S0 = random_state(B, H_v, d, seed=6)
    o, S = decode(ds, x, S0)
    assert np.array_equal(S.astype(np.float32), S0)
    qf = synth.bf16_bits_to_f64(x.q)
    grp = H_v // H_k
    ref_o = np.stack([np.einsum("bij,bj->bi", S0[:, j].astype(np.float64), qf[:, j // grp]) for j in range(H_v)], 1)
    assert rel_fro(o, ref_o) <= TOL


def test_chain_of_steps_equals_recurrence(ds):
    """40 decode steps over 3 streams equal the oracle over the 40-token streams."""
    B, H_k, H_v, d, N = 3, 2, 4, 128, 40
    xs = synth.make_gdn_inputs([N] * B, H_k, H_v, d, 0, False, config=95, gates="long_memory")
    ref = oracle.gdn_forward(xs.q, xs.k, xs.v, xs.g, xs.beta, xs.cu_seqlens, 0)
    state = torch.zeros((B, H_v, d, d), dtype=torch.float32, device=DEV)
    idx = lambda t: np.arange(B) * N + t
    outs = []
    for t in range(N):
        i = idx(t)
        r = ds.gdn_decode_step(dev_bf16(xs.q[i]), dev_bf16(xs.k[i]), dev_bf16(xs.v[i]), dev_f32(xs.g[i]),
                               dev_f32(xs.beta[i]), state_in=state, state_out=state)
        outs.append(r["o"].cpu().numpy().astype(np.float64))
    torch.cuda.synchronize()
    o = np.stack(outs, 1).reshape(B * N, H_v, d)
    assert rel_fro(o, ref["o"]) <= TOL
    assert rel_fro(state.cpu().numpy(), ref["S"]) <= TOL


def test_prefill_then_decode(ds):
    """gdn_chunk_fwd over two streams (300 and 200 tokens), then 10 decode
    steps from its final states, equal the oracle over 310 and 210 tokens."""
    H_k, H_v, d, n_dec = 2, 4, 128, 10
    lens = [310, 210]
    xs = synth.make_gdn_inputs(lens, H_k, H_v, d, 64, True, config=96)
    ref = oracle.gdn_forward(xs.q, xs.k, xs.v, xs.g, xs.beta, xs.cu_seqlens, 64)
    pre = [l - n_dec for l in lens]
    cu = xs.cu_seqlens
    sel = np.concatenate([np.arange(cu[b], cu[b] + pre[b]) for b in range(2)])
    r = ds.gdn_chunk_fwd(dev_bf16(xs.q[sel]), dev_bf16(xs.k[sel]), dev_bf16(xs.v[sel]), dev_f32(xs.g[sel]),
                         dev_f32(xs.beta[sel]), pre, 64, drift_partials=False)
    state = r["state"]
    outs = []
    for t in range(n_dec):
        i = np.array([cu[b] + pre[b] + t for b in range(2)])
        rr = ds.gdn_decode_step(dev_bf16(xs.q[i]), dev_bf16(xs.k[i]), dev_bf16(xs.v[i]), dev_f32(xs.g[i]),
                                dev_f32(xs.beta[i]), state_in=state, state_out=state)
        outs.append(rr["o"].cpu().numpy().astype(np.float64))
    torch.cuda.synchronize()
    o_dec = np.stack(outs, 1)                                  # [2][n_dec][H_v][d]
    ref_dec = np.stack([ref["o"][cu[b] + pre[b]:cu[b + 1]] for b in range(2)])
    # the prefix carries the chunked forward's fp16-operand error (<= 2e-3)
    assert rel_fro(o_dec, ref_dec) <= 2e-3
    assert rel_fro(state.cpu().numpy(), ref["S"]) <= 2e-3
