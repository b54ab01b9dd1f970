"""Helpers for the GPU parity tests: move synthetic inputs to the device,
run the HIP path through the binding and compare with the oracle."""
import numpy as np
import torch

DEV = torch.device("cuda:0")


def rel_fro(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    nb = np.linalg.norm(b)
    return np.linalg.norm(a - b) / (nb if nb > 0 else 1.0)


def dev_bf16(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(DEV).view(torch.bfloat16)


def dev_f32(x):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(DEV)


def lengths_of(x):
    cu = x.cu_seqlens
    return [int(cu[i + 1] - cu[i]) for i in range(len(cu) - 1)]


def run_gpu(ds, x, o_dtype=torch.float32, state_in=None, snapshots=False, in_place=False):
    q, k, v = dev_bf16(x.q), dev_bf16(x.k), dev_bf16(x.v)
    g, beta = dev_f32(x.g), dev_f32(x.beta)
    s_in = None if state_in is None else dev_f32(state_in)
    r = ds.gdn_chunk_fwd(q, k, v, g, beta, lengths_of(x), x.frame_len, state_in=s_in,
                         state_out=s_in if in_place else None, o_dtype=o_dtype, snapshots=snapshots)
    torch.cuda.synchronize()
    out = dict(o=r["o"].float().cpu().numpy().astype(np.float64),
               S=r["state"].cpu().numpy().astype(np.float64),
               partials=r["drift_partials"].cpu().numpy().astype(np.float64))
    if snapshots:
        out["snapshots"] = r["snapshots"].cpu().numpy().astype(np.float64)
    out["raw"] = r
    return out


def bf16_round(x):
    from synth import bf16_bits_to_f64, to_bf16_bits
    return bf16_bits_to_f64(to_bf16_bits(x))


def drift_rel_err(gpu_scores, ref_scores):
    """Max relative error over finite entries; +inf must match +inf exactly."""
    g = np.asarray(gpu_scores, np.float64)
    r = np.asarray(ref_scores, np.float64)
    assert np.array_equal(np.isinf(g), np.isinf(r)), (g, r)
    fin = np.isfinite(r)
    if not fin.any():
        return 0.0
    den = np.abs(r[fin])
    return float(np.max(np.abs(g[fin] - r[fin]) / np.where(den > 0, den, 1.0)))
