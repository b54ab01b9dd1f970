"""fp64 CPU oracle for the DeltaS hot path.

TEST INFRASTRUCTURE ONLY: the slow, plain reference that the HIP path is
checked against.  Only the test suite, the smoke check and the benchmark's
CPU-baseline leg may import it.  It shares no code with the product library
(``paper_2609_27470_amd``) and never imports it.

Contents
  gdn_forward   token-by-token gated delta rule (Eq. 2) with frame drift sums
                (C, ``gdn_ref.c``, fp64, OpenMP over (stream, v-head))
  drift_scores  Eq. 3 and the two other aggregations of the per-head sums
  select_keep   retention policy of Section 3.3 / Algorithm 1 (plain Python)
  compact       the eviction gather KV <- KV[keep] (numpy fancy indexing)
  compact_indexed  the same eviction over a slot-indexed cache: only the
                (pos, chunk id, slot) table is gathered; freed rows listed

Readings of the paper that these functions take where it is silent are
listed in each function's docstring.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess
from pathlib import Path

import numpy as np

_HERE = Path(__file__).resolve().parent
_SRC = _HERE / "gdn_ref.c"
_LIB = _HERE / "libgdn_ref.so"
_lib = None

# drift aggregation modes
LAYER_FROB = 0   # Eq. 3: per layer ||dS||_F / ||S_before||_F over all heads, mean over layers
HEAD_MEAN = 1    # mean over layers and heads of the per-head ratio
PER_HEAD = 2     # the per-(layer, frame, head) ratios themselves
WRITE_MEAN = 3   # (sum, count) write pairs: mean over layers and heads of sum / count


def build(force: bool = False) -> Path:
    """Compile the C oracle with gcc (-O2, no fast-math, OpenMP)."""
    if force or not _LIB.exists() or _LIB.stat().st_mtime < _SRC.stat().st_mtime:
        tmp = _LIB.with_suffix(".so.tmp%d" % os.getpid())
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
                               str(_SRC), "-o", str(tmp), "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(str(_LIB))
        P = ctypes.c_void_p
        lib.ref_gdn_forward.argtypes = [ctypes.c_int, P, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                        ctypes.c_int, ctypes.c_int, P, P, P, P, P, P,
                                        ctypes.c_double, P, P, P, P, P, ctypes.c_int]
        lib.ref_gdn_forward.restype = ctypes.c_int
        lib.ref_max_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def max_threads() -> int:
    return int(_load().ref_max_threads())


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def n_frames(cu_seqlens, frame_len) -> int:
    tot = 0
    for b in range(len(cu_seqlens) - 1):
        n = int(cu_seqlens[b + 1]) - int(cu_seqlens[b])
        if n > 0:
            tot += 1 if frame_len <= 0 else (n + frame_len - 1) // frame_len
    return tot


def gdn_forward(q, k, v, g, beta, cu_seqlens, frame_len, S0=None, scale=1.0,
                snapshots=False, n_threads=0):
    """Gated delta rule, token by token (Section 3.2, Eq. 2), in fp64.

    q, k: uint16 bf16 bits [T][H_k][d_k]; v: uint16 bf16 bits [T][H_v][d_v];
    g (log decay, alpha = exp(g)) and beta: float32 [T][H_v];
    cu_seqlens: int32 [B+1]; S0: fp64 [B][H_v][d_v][d_k] or None (zeros).

    Readings: o_t = scale * S_t q_t is read after the token's update; v-head
    j reads qk-head j * H_k / H_v; the state is d_v x d_k (Eq. 1 multiplies
    S on the right by a d_k x d_k matrix); frames start at each stream's
    first token and the last frame may be partial.

    Returns dict(o [T][H_v][d_v], S [B][H_v][d_v][d_k],
                 partials [F][H_v][2] (num, den),
                 writes [F][H_v][2] (sum over the frame of beta_t ||v_t - alpha_t S k_t||_2,
                                     token count) -- the write-magnitude signal,
                 snapshots or None).
    
    """
    lib = _load()
    q = np.ascontiguousarray(q, dtype=np.uint16)
    k = np.ascontiguousarray(k, dtype=np.uint16)
    v = np.ascontiguousarray(v, dtype=np.uint16)
    g = np.ascontiguousarray(g, dtype=np.float32)
    beta = np.ascontiguousarray(beta, dtype=np.float32)
    cu = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
    T, H_k, d_k = q.shape
    H_v, d_v = v.shape[1], v.shape[2]
    B = len(cu) - 1
    F = n_frames(cu, frame_len)
    o = np.zeros((T, H_v, d_v), np.float64)
    S = np.zeros((B, H_v, d_v, d_k), np.float64)
    part = np.zeros((F, H_v, 2), np.float64)
    wr = np.zeros((F, H_v, 2), np.float64)
    snap = np.zeros((F, H_v, d_v, d_k), np.float64) if snapshots else None
    S0c = None if S0 is None else np.ascontiguousarray(S0, dtype=np.float64)
    rc = lib.ref_gdn_forward(B, _ptr(cu), H_k, H_v, d_k, d_v, int(frame_len), _ptr(q), _ptr(k),
                             _ptr(v), _ptr(g), _ptr(beta), _ptr(S0c), float(scale), _ptr(o),
                             _ptr(S), _ptr(part), _ptr(wr), _ptr(snap), int(n_threads))
    if rc != 0:
        raise ValueError("oracle rejected the arguments")
    return dict(o=o, S=S, partials=part, writes=wr, snapshots=snap)


def _ratio(num, den):
    """sqrt(num / den) with the reading den = 0 -> +inf if num > 0, else 0."""
    if den > 0.0:
        return math.sqrt(num / den)
    return math.inf if num > 0.0 else 0.0


def drift_scores(partials, mode=LAYER_FROB):
    """State drift from per-(layer, frame, head) sums (Section 3.2, Eq. 3).

    partials: [L][F][H][2] holding num = ||S_end - S_start||_F^2 and
    den = ||S_start||_F^2 of each head.
    LAYER_FROB: Eq. 3 -- the norm of layer i runs over all its heads, so
      per layer sqrt(sum_h num / sum_h den), then the mean over layers -> [F].
    HEAD_MEAN: mean over layers and heads of sqrt(num / den) -> [F].
    PER_HEAD: sqrt(num / den) -> [L][F][H].
    WRITE_MEAN: the pairs are the write-magnitude sums (sum over the frame's
      tokens of beta ||e||, token count) of gdn_forward; the chunk score of the
      beta ||e|| signal is the mean over layers, heads and tokens -> [F].
    A mean that contains +inf is +inf.
    """
    p = np.asarray(partials, dtype=np.float64)
    L, F, H, _ = p.shape
    if mode == PER_HEAD:
        out = np.zeros((L, F, H))
        for l in range(L):
            for f in range(F):
                for h in range(H):
                    out[l, f, h] = _ratio(p[l, f, h, 0], p[l, f, h, 1])
        return out
    out = np.zeros(F)
    for f in range(F):
        vals = []
        for l in range(L):
            if mode == LAYER_FROB:
                vals.append(_ratio(sum(p[l, f, :, 0]), sum(p[l, f, :, 1])))
            elif mode == WRITE_MEAN:
                vals.extend(p[l, f, h, 0] / p[l, f, h, 1] if p[l, f, h, 1] > 0 else 0.0 for h in range(H))
            elif mode == HEAD_MEAN:
                vals.extend(_ratio(p[l, f, h, 0], p[l, f, h, 1]) for h in range(H))
            else:
                raise ValueError(mode)
        out[f] = math.inf if any(math.isinf(x) for x in vals) else sum(vals) / len(vals)
    return out


def drift_states(S_before, S_after):
    """The two sums behind Eq. 3 (Section 3.2) from two copies of the state:
    num = ||S_after - S_before||_F^2 and den = ||S_before||_F^2 per head, for
    arrays [..., d_v, d_k] -> [..., 2], in fp64."""
    b = np.asarray(S_before, dtype=np.float64)
    a = np.asarray(S_after, dtype=np.float64)
    num = np.sum((a - b) ** 2, axis=(-2, -1))
    den = np.sum(b ** 2, axis=(-2, -1))
    return np.stack([num, den], axis=-1)


def select_keep(chunk_id, pos, chunk_scores, length, M, n_sink, n_window, n_buckets):
    """Cache slots kept by one eviction step (Section 3.3, Algorithm 1).

    When the cache holds more than M tokens: the first n_sink and the last
    n_window slots are always kept; the other slots are candidates, split
    into N equal spans of chunk arrival time; each span keeps its best
    floor((M - n_sink - n_window) / N) candidates and the slots left over
    (the remainder of the division and the quota of spans with too few
    candidates) go to the best candidates not yet kept.

    Readings: a token's score is its chunk's score; arrival time is the
    chunk index; span of chunk a is floor(N (a - a_min) / (a_max - a_min + 1))
    over the candidates' chunk range; N = 0 means one span; "best" orders by
    (score desc, chunk id desc, position desc) -- ties go to newer tokens.
    Returns the kept slot indices in ascending order (positions are never
    rewritten).
    """
    chunk_id = [int(x) for x in chunk_id[:length]]
    pos = [int(x) for x in pos[:length]]
    scores = [float(x) for x in chunk_scores]
    if length <= M:
        return list(range(length))
    if n_sink + n_window > M:
        raise ValueError("reserved regions exceed the budget")
    N = max(1, int(n_buckets))
    sink = list(range(0, n_sink))
    window = list(range(length - n_window, length))
    cand = list(range(n_sink, length - n_window))

    def key(i):
        return (-scores[chunk_id[i]], -chunk_id[i], -pos[i])

    taken = set()
    if cand:
        a_min = min(chunk_id[i] for i in cand)
        a_max = max(chunk_id[i] for i in cand)
        span = a_max - a_min + 1
        quota = (M - n_sink - n_window) // N
        for bkt in range(N):
            members = [i for i in cand if (N * (chunk_id[i] - a_min)) // span == bkt]
            members.sort(key=key)
            taken.update(members[:quota])
        fill = M - n_sink - n_window - len(taken)
        rest = sorted((i for i in cand if i not in taken), key=key)
        taken.update(rest[:fill])
    return sorted(set(sink) | taken | set(window))


def compact(rows, keep):
    """The eviction gather: new[i] = old[keep[i]] (rows of any dtype)."""
    rows = np.asarray(rows)
    return rows[np.asarray(keep, dtype=np.int64)]


def compact_indexed(pos, chunk_id, slot, keep, length):
    """Eviction over a slot-indexed cache (Section 3.3: same kept set as the
    gather, Z18 order kept through the table).

    Logical token i lives in physical row slot[i].  The table is gathered
    like the rows of the plain cache -- new[d] = old[keep[d]] -- and the rows
    of the tokens not kept are returned in ascending logical order as the
    free list.  Returns (pos', chunk_id', slot', free), each of the first
    three of length len(keep).
    """
    keep = np.asarray(keep, dtype=np.int64)
    pos = np.asarray(pos)[:length]
    chunk_id = np.asarray(chunk_id)[:length]
    slot = np.asarray(slot)[:length]
    kept = np.zeros(length, dtype=bool)
    kept[keep] = True
    return pos[keep], chunk_id[keep], slot[keep], slot[~kept]
