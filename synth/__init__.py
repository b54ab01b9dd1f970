"""Seeded synthetic inputs for the DeltaS hot path.

This module only draws numbers.  It holds none of the method's arithmetic
(no recurrence, no drift, no selection): both the fp64 oracle and the HIP
path read what it produces, so neither side can leak into the other here.

Recipe (stated once, used everywhere):

* generator: numpy ``PCG64`` seeded with ``SeedSequence([config, layer,
  stream, group])``, one generator per group of four frames (novelty streams)
  or per block of 1024 tokens (iid streams), so that groups are drawn in
  parallel threads; everything is drawn in fp64 and rounded to the stored
  dtype (fp64 -> fp32 round-to-nearest-even -> bf16 round-to-nearest-even);
* q, k ~ N(0, 1) per element, L2-normalised per (token, head) in fp64, then
  bf16 (the method takes unit keys, Section 3.2 after Eq. 1);
* v ~ N(0, 1), bf16;
* log-decay g = -softplus(N(0, 1)) and write strength beta = sigmoid(N(0, 1)),
  fp32, one value per (token, v-head);
* "novelty" streams: frames whose index is a multiple of 4 draw each
  qk-head's keys from a fresh random 32-dim subspace (QR of a Gaussian
  128x32 matrix, scaled by sqrt(d/32)) and fresh values; every other frame
  re-presents a token of the previous frame chosen uniformly with
  replacement (one source index per token, shared by all heads and by k and
  v) plus N(0, 0.05) noise added before normalisation.  q stays iid.

A novelty group is one novel frame followed by the three frames that
re-present it (frames 4 i .. 4 i + 3 of the stream).  Draw order inside one
frame: [basis per qk-head, z] or [src, k-noise], then v (or v-noise), q,
g_raw, beta_raw.  An iid block draws q, k, v, g_raw, beta_raw in that order.
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

# Shapes of the five workloads (tokens, heads, head dim, frame length).
WORKLOADS = {
    "tiny": dict(H_k=2, H_v=2, d=64, T=1024, frame_len=256, novelty=False),
    "single_layer": dict(H_k=16, H_v=32, d=128, T=32768, frame_len=1024, novelty=True),
    "stack": dict(H_k=16, H_v=32, d=128, T=262144, frame_len=1024, novelty=True, layers=24),
    "varlen": dict(H_k=16, H_v=32, d=128, B=8, len_lo=16384, len_hi=131072,
                   frame_len=1024, novelty=True),
    "eviction_loop": dict(H_k=16, H_v=32, d=128, T=1048576, frame_len=1024, novelty=True,
                          layers=24, kv_layers=8, kv_heads=8, kv_head_dim=256,
                          budget=16384, pool_frames=64),
}
CONFIG_INDEX = {"tiny": 0, "single_layer": 1, "stack": 2, "varlen": 3, "eviction_loop": 4}


# ----------------------------------------------------------------------------
# dtype helpers (bit patterns, so nothing depends on a bf16 numpy dtype)
# ----------------------------------------------------------------------------
def to_bf16_bits(x) -> np.ndarray:
    """fp64/fp32 array -> bf16 bit patterns (uint16), round to nearest even
    (finite values: the sum below stays inside 32 bits)."""
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    u = f.view(np.uint32)
    r = u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))
    return (r >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f64(b) -> np.ndarray:
    u = np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def _softplus(x):
    return np.logaddexp(0.0, x)


def _sigmoid(x):
    return 0.5 * (1.0 + np.tanh(0.5 * x))


def _unit_rows(x):
    n = np.sqrt(np.sum(x * x, axis=-1, keepdims=True))
    return x / np.where(n > 0, n, 1.0)


def rng_for(config: int, layer: int = 0, stream: int = 0, *more: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([config, layer, stream, *more])))


IID_BLOCK = 1024      # tokens per generator of an iid stream
NOVELTY_GROUP = 4     # frames per generator of a novelty stream (one novel frame, three re-presenting it)
_pool = None


def _executor():
    global _pool
    if _pool is None:
        _pool = ThreadPoolExecutor(max_workers=max(1, min(16, os.cpu_count() or 1)))
    return _pool


# ----------------------------------------------------------------------------
# GDN inputs
# ----------------------------------------------------------------------------
@dataclass
class GdnInputs:
    """One packed batch of streams (token-major layouts)."""
    q: np.ndarray          # uint16 bf16 bits [T_total][H_k][d_k]
    k: np.ndarray          # uint16 bf16 bits [T_total][H_k][d_k]
    v: np.ndarray          # uint16 bf16 bits [T_total][H_v][d_v]
    g: np.ndarray          # float32 [T_total][H_v]   (log decay, alpha = exp(g))
    beta: np.ndarray       # float32 [T_total][H_v]
    cu_seqlens: np.ndarray  # int32 [B+1]
    frame_len: int
    H_k: int
    H_v: int
    d: int
    meta: dict = field(default_factory=dict)

    @property
    def B(self) -> int:
        return len(self.cu_seqlens) - 1

    @property
    def T_total(self) -> int:
        return int(self.cu_seqlens[-1])

    def n_frames(self) -> int:
        return sum(frames_of_length(int(self.cu_seqlens[b + 1] - self.cu_seqlens[b]), self.frame_len)
                   for b in range(self.B))


def frames_of_length(n: int, frame_len: int) -> int:
    """Frames in a stream of n tokens: every frame_len tokens plus a ragged
    tail; frame_len == 0 makes the whole stream one frame; empty -> 0."""
    if n <= 0:
        return 0
    if frame_len <= 0:
        return 1
    return (n + frame_len - 1) // frame_len


def _gates(rng, n, H_v, gates="standard", head_x=None):
    if gates == "standard":
        g = -_softplus(rng.standard_normal((n, H_v)))
    elif gates == "long_memory":
        x = head_x[None, :] + 0.1 * rng.standard_normal((n, H_v))
        g = -_softplus(x)
    else:
        raise ValueError(gates)
    beta = _sigmoid(rng.standard_normal((n, H_v)))
    return g.astype(np.float32), beta.astype(np.float32)


def _plain_block(rng, n, H_k, H_v, d, gates="standard", head_x=None):
    """n iid tokens: fp64 q, k (normalised), v, and fp32 gates."""
    q = _unit_rows(rng.standard_normal((n, H_k, d)))
    k = _unit_rows(rng.standard_normal((n, H_k, d)))
    v = rng.standard_normal((n, H_v, d))
    g, beta = _gates(rng, n, H_v, gates, head_x)
    return q, k, v, g, beta


def _novelty_group(rng, lens, H_k, H_v, d, sub=32, sigma=0.05, gates="standard", head_x=None):
    """Yield (q, k, v, g, beta) for the frames of one novelty group (frame
    lengths `lens`): the first frame is novel, each later one re-presents
    tokens of the frame before it."""
    k_prev = v_prev = None
    for c, n in enumerate(lens):
        if c == 0:
            k_raw = np.empty((n, H_k, d))
            for h in range(H_k):
                basis, _ = np.linalg.qr(rng.standard_normal((d, sub)))
                z = rng.standard_normal((n, sub))
                k_raw[:, h, :] = (z @ basis.T) * math.sqrt(d / sub)
            v_raw = rng.standard_normal((n, H_v, d))
        else:
            src = rng.integers(0, k_prev.shape[0], size=n)
            k_raw = k_prev[src] + sigma * rng.standard_normal((n, H_k, d))
            v_raw = v_prev[src] + sigma * rng.standard_normal((n, H_v, d))
        q = rng.standard_normal((n, H_k, d))
        g, beta = _gates(rng, n, H_v, gates, head_x)
        k_prev, v_prev = k_raw, v_raw
        yield _unit_rows(q), _unit_rows(k_raw), v_raw, g, beta


def _store(out, t, part):
    """Round one generated piece into the packed arrays at token offset t."""
    q, k, v, g, beta = out
    pq, pk, pv, pg, pb = part
    n = pq.shape[0]
    q[t:t + n] = to_bf16_bits(pq)
    k[t:t + n] = to_bf16_bits(pk)
    v[t:t + n] = to_bf16_bits(pv)
    g[t:t + n] = pg
    beta[t:t + n] = pb


def _stream_tasks(out, t0, config, layer, stream, T, H_k, H_v, d, frame_len, novelty, gates):
    """Independent generation tasks that fill one stream's tokens [t0, t0 + T)."""
    head_x = None
    if gates == "long_memory":   # per-head gate offsets, drawn from the stream's own generator
        head_x = rng_for(config, layer, stream).uniform(-10.0, -2.0, size=H_v)
    tasks = []
    if novelty:
        F = frame_len if frame_len > 0 else T
        n_fr = frames_of_length(T, F)
        for grp in range((n_fr + NOVELTY_GROUP - 1) // NOVELTY_GROUP):
            f0 = grp * NOVELTY_GROUP
            lens = [min(F, T - f * F) for f in range(f0, min(f0 + NOVELTY_GROUP, n_fr))]

            def task(grp=grp, lens=lens, ts=t0 + f0 * F):
                rng = rng_for(config, layer, stream, grp)
                t = ts
                for part in _novelty_group(rng, lens, H_k, H_v, d, gates=gates, head_x=head_x):
                    _store(out, t, part)
                    t += part[0].shape[0]
            tasks.append(task)
    else:
        for blk in range((T + IID_BLOCK - 1) // IID_BLOCK):
            n = min(IID_BLOCK, T - blk * IID_BLOCK)

            def task(blk=blk, n=n):
                rng = rng_for(config, layer, stream, blk)
                _store(out, t0 + blk * IID_BLOCK, _plain_block(rng, n, H_k, H_v, d, gates, head_x))
            tasks.append(task)
    return tasks


def _run(tasks):
    for f in [_executor().submit(t) for t in tasks]:
        f.result()


def make_stream(config: int, layer: int, stream: int, T: int, H_k: int, H_v: int, d: int,
                frame_len: int, novelty: bool, gates: str = "standard"):
    """One stream's arrays (bf16 bits / fp32) from its own seeds."""
    out = (np.empty((T, H_k, d), np.uint16), np.empty((T, H_k, d), np.uint16), np.empty((T, H_v, d), np.uint16),
           np.empty((T, H_v), np.float32), np.empty((T, H_v), np.float32))
    _run(_stream_tasks(out, 0, config, layer, stream, T, H_k, H_v, d, frame_len, novelty, gates))
    return out


def make_gdn_inputs(lengths, H_k, H_v, d, frame_len, novelty, config=0, layer=0,
                    gates="standard") -> GdnInputs:
    """Packed varlen batch: stream b is drawn from seed (config, layer, b)."""
    lengths = [int(x) for x in lengths]
    cu = np.zeros(len(lengths) + 1, np.int32)
    cu[1:] = np.cumsum(lengths)
    T = int(cu[-1])
    q = np.empty((T, H_k, d), np.uint16)
    k = np.empty((T, H_k, d), np.uint16)
    v = np.empty((T, H_v, d), np.uint16)
    g = np.empty((T, H_v), np.float32)
    beta = np.empty((T, H_v), np.float32)
    tasks = []
    for b, n in enumerate(lengths):
        if n > 0:
            tasks += _stream_tasks((q, k, v, g, beta), int(cu[b]), config, layer, b, n, H_k, H_v, d, frame_len,
                                   novelty, gates)
    _run(tasks)
    return GdnInputs(q, k, v, g, beta, cu, frame_len, H_k, H_v, d,
                     meta=dict(config=config, layer=layer, novelty=novelty, gates=gates))


def workload_inputs(name: str, layer: int = 0, **override) -> GdnInputs:
    """Inputs of a named workload (optionally with smaller sizes for tests)."""
    w = dict(WORKLOADS[name])
    w.update(override)
    cfg = CONFIG_INDEX[name]
    if name == "varlen":
        lengths = w.get("lengths")
        if lengths is None:
            lengths = varlen_lengths(w["B"], w["len_lo"], w["len_hi"])
    else:
        lengths = [w["T"]]
    return make_gdn_inputs(lengths, w["H_k"], w["H_v"], w["d"], w["frame_len"], w["novelty"],
                           config=cfg, layer=layer, gates=w.get("gates", "standard"))


def varlen_lengths(B: int, lo: int, hi: int, seed_tag: int = 99) -> list:
    """Stream lengths drawn uniformly from the integers [lo, hi] (inclusive)."""
    rng = rng_for(CONFIG_INDEX["varlen"], seed_tag, 0)
    return [int(x) for x in rng.integers(lo, hi + 1, size=B)]


def pool_frame_index(frame: int, layer: int, pool_frames: int) -> int:
    """Eviction loop input pool: stream frame f at layer l reads pool frame (f + 4 l) mod P."""
    return (frame + 4 * layer) % pool_frames


# ----------------------------------------------------------------------------
# Closed-form inputs used by the pins (exact in bf16)
# ----------------------------------------------------------------------------
def hadamard(n: int) -> np.ndarray:
    h = np.array([[1.0]])
    while h.shape[0] < n:
        h = np.block([[h, h], [h, -h]])
    return h


def orthonormal_keys(d: int) -> np.ndarray:
    """d exactly orthonormal keys whose entries are 0 or +-1/8 (exact in bf16).

    d = 64: rows of H_64 / 8.  d = 128: rows of H_64 / 8 placed in coordinates
    0..63 and again in 64..127.
    """
    h = hadamard(64) / 8.0
    if d == 64:
        return h
    if d == 128:
        out = np.zeros((128, 128))
        out[:64, :64] = h
        out[64:, 64:] = h
        return out
    raise ValueError("d must be 64 or 128")


# ----------------------------------------------------------------------------
# KV-cache rows: a counter-based hash of (layer, K/V, position, element)
# ----------------------------------------------------------------------------
_M32 = 0xFFFFFFFF


def _fmix32_np(x):
    x = x.astype(np.uint64)
    x ^= x >> np.uint64(16)
    x = (x * np.uint64(0x85EBCA6B)) & np.uint64(_M32)
    x ^= x >> np.uint64(13)
    x = (x * np.uint64(0xC2B2AE35)) & np.uint64(_M32)
    x ^= x >> np.uint64(16)
    return x


def kv_row_bits(layer: int, kv: int, pos, row_elems: int) -> np.ndarray:
    """bf16 bit patterns [len(pos)][row_elems] for the rows at positions ``pos``.

    Each element is murmur3's 32-bit finaliser of a counter built from
    (layer, kv, pos, element); the top 16 bits become the bf16 pattern with the
    top exponent bit cleared, so every value is finite (|x| < 2).
    """
    pos = np.asarray(pos, dtype=np.uint64).reshape(-1, 1)
    e = np.arange(row_elems, dtype=np.uint64).reshape(1, -1)
    base = (pos * np.uint64(0x9E3779B1) + np.uint64((layer * 0x85EBCA77) & _M32)
            + np.uint64((kv * 0xC2B2AE3D) & _M32)) & np.uint64(_M32)
    x = (base + e * np.uint64(0x27D4EB2F)) & np.uint64(_M32)
    h = _fmix32_np(x)
    return ((h >> np.uint64(16)) & np.uint64(0xBFFF)).astype(np.uint16)


def kv_row_bits_torch(layer: int, kv: int, pos, row_elems: int):
    """Same values as ``kv_row_bits`` computed with torch int64 ops (any device).

    ``pos`` is an int64 tensor; returns an int16 tensor holding the bit patterns.
    """
    import torch
    m = 0xFFFFFFFF
    p = pos.to(torch.int64).reshape(-1, 1)
    e = torch.arange(row_elems, dtype=torch.int64, device=p.device).reshape(1, -1)
    base = (p * 0x9E3779B1 + ((layer * 0x85EBCA77) & m) + ((kv * 0xC2B2AE3D) & m)) & m
    x = (base + e * 0x27D4EB2F) & m
    x = x ^ (x >> 16)
    x = (x * 0x85EBCA6B) & m
    x = x ^ (x >> 13)
    x = (x * 0xC2B2AE35) & m
    x = x ^ (x >> 16)
    bits = (x >> 16) & 0xBFFF
    # reinterpret the low 16 bits as int16
    return (bits - ((bits & 0x8000) << 1)).to(torch.int16)


# ----------------------------------------------------------------------------
# The same recipe drawn on the device (benchmark inputs too large to draw on
# the host in a benchmark run: the per-layer frame pools of the stack and
# eviction-loop workloads, the varlen batch).  torch's generator, fp32
# arithmetic; the orthonormal bases of the novel frames come from numpy's QR
# on the host.  Values differ from the host generator's (parity tests use
# the host generator); the distributions and the novelty structure do not.
# ----------------------------------------------------------------------------
def device_novelty_frames(n_frames, frame_len, H_k, H_v, d, seed, device, sub=32, sigma=0.05):
    """(q, k, v, g, beta) for n_frames frames of frame_len tokens on `device`:
    q, k, v bf16 [n_frames * frame_len][H][d], g, beta fp32 [..][H_v].  Frames
    4 i are novel (keys from a fresh 32-dim subspace per qk-head, fresh
    values); the others re-present a uniformly chosen token of the frame
    before them (one source per token, shared by heads, k and v) plus
    N(0, 0.05) noise before normalisation; q iid; g = -softplus(N(0, 1)),
    beta = sigmoid(N(0, 1))."""
    import torch
    gen = torch.Generator(device=device).manual_seed(int(seed))
    hrng = rng_for(7000, int(seed) & 0x7FFFFFFF, 0)
    T = n_frames * frame_len
    q = torch.empty((T, H_k, d), dtype=torch.bfloat16, device=device)
    k = torch.empty((T, H_k, d), dtype=torch.bfloat16, device=device)
    v = torch.empty((T, H_v, d), dtype=torch.bfloat16, device=device)
    n = frame_len

    def unit(x):
        return x / x.norm(dim=-1, keepdim=True)

    k_prev = v_prev = None
    for f in range(n_frames):
        s = slice(f * n, (f + 1) * n)
        if f % 4 == 0:
            bases = np.stack([np.linalg.qr(hrng.standard_normal((d, sub)))[0] for _ in range(H_k)])
            B = torch.as_tensor(bases, dtype=torch.float32, device=device)           # [H_k][d][sub]
            z = torch.randn((H_k, n, sub), generator=gen, device=device)
            k_raw = (torch.matmul(z, B.transpose(1, 2).contiguous()) * math.sqrt(d / sub)).transpose(0, 1)
            v_raw = torch.randn((n, H_v, d), generator=gen, device=device)
        else:
            src = torch.randint(0, n, (n,), generator=gen, device=device)
            k_raw = k_prev[src] + sigma * torch.randn((n, H_k, d), generator=gen, device=device)
            v_raw = v_prev[src] + sigma * torch.randn((n, H_v, d), generator=gen, device=device)
        k[s] = unit(k_raw).to(torch.bfloat16)
        v[s] = v_raw.to(torch.bfloat16)
        q[s] = unit(torch.randn((n, H_k, d), generator=gen, device=device)).to(torch.bfloat16)
        k_prev, v_prev = k_raw.contiguous(), v_raw
    g = -torch.nn.functional.softplus(torch.randn((T, H_v), generator=gen, device=device))
    beta = torch.sigmoid(torch.randn((T, H_v), generator=gen, device=device))
    return q, k, v, g, beta
