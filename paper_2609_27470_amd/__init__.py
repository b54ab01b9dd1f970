"""DeltaS hot path on MI355X: Python binding of libdeltas (C ABI in include/deltas.h).

The binding only marshals arguments: torch tensors provide device memory
and the current HIP stream; every step of the computation runs in the HIP
kernels of libdeltas.so.  There is no fallback -- if the library is not
built, every entry point raises.
"""
from __future__ import annotations

import ctypes
from pathlib import Path

import torch

PKG = Path(__file__).resolve().parent
LIB_PATH = PKG / "libdeltas.so"

DS_OK = 0
DS_BF16, DS_F32 = 0, 1
LAYER_FROB, HEAD_MEAN, PER_HEAD, WRITE_MEAN = 0, 1, 2, 3

EXPORTED = [
    "ds_status_string", "ds_last_error", "ds_gdn_workspace_bytes", "ds_gdn_write_workspace_bytes",
    "gdn_chunk_fwd", "deltas_drift",
    "deltas_drift_states", "ds_kv_workspace_bytes", "kv_evict_topk", "ds_kv_device_status",
    "ds_kv_indexed_workspace_bytes", "kv_evict_topk_indexed", "gdn_decode_step", "kv_evict_topk_indexed_noalloc",
    "kv_append_indexed",
]
NOALLOC_MAX_CAPACITY = 65536


class GdnShape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("B", "T_total", "H_k", "H_v", "d_k", "d_v", "frame_len", "n_frames", "drift_per_slice")]


class KvShape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("n_layers", "row_bytes", "capacity")]


class DeltasError(RuntimeError):
    def __init__(self, status, detail):
        super().__init__(f"status {status}: {detail}")
        self.status = status


_lib = None


def lib():
    """Load libdeltas.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not LIB_PATH.exists():
            raise RuntimeError(f"{LIB_PATH} is missing: build it with paper_2609_27470_amd.build.build()")
        L = ctypes.CDLL(str(LIB_PATH))
        P, I32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        L.ds_status_string.argtypes = [I32]
        L.ds_status_string.restype = ctypes.c_char_p
        L.ds_last_error.argtypes = []
        L.ds_last_error.restype = ctypes.c_char_p
        L.ds_gdn_workspace_bytes.argtypes = [ctypes.POINTER(GdnShape)]
        L.ds_gdn_workspace_bytes.restype = SZ
        L.ds_gdn_write_workspace_bytes.argtypes = [ctypes.POINTER(GdnShape)]
        L.ds_gdn_write_workspace_bytes.restype = SZ
        L.gdn_chunk_fwd.argtypes = [ctypes.POINTER(GdnShape), P, P, P, P, P, P, P, P, P, I32, ctypes.c_float,
                                    P, P, P, P, SZ, P]
        L.gdn_chunk_fwd.restype = I32
        L.gdn_decode_step.argtypes = [I32, I32, I32, I32, I32, P, P, P, P, P, P, P, P, I32, ctypes.c_float, P]
        L.gdn_decode_step.restype = I32
        L.deltas_drift.argtypes = [P, I32, I32, I32, I32, P, P]
        L.deltas_drift.restype = I32
        L.deltas_drift_states.argtypes = [P, P, I32, I32, I32, I32, I32, P, P]
        L.deltas_drift_states.restype = I32
        L.ds_kv_workspace_bytes.argtypes = [ctypes.POINTER(KvShape)]
        L.ds_kv_workspace_bytes.restype = SZ
        L.kv_evict_topk.argtypes = [ctypes.POINTER(KvShape), P, P, P, P, P, I32, I32, I32, I32, I32, I32, P,
                                    ctypes.POINTER(I32), P, SZ, P]
        L.kv_evict_topk.restype = I32
        L.ds_kv_device_status.argtypes = [P]
        L.ds_kv_device_status.restype = P
        L.ds_kv_indexed_workspace_bytes.argtypes = [I32]
        L.ds_kv_indexed_workspace_bytes.restype = SZ
        L.kv_evict_topk_indexed.argtypes = [I32, P, P, P, P, I32, I32, I32, I32, I32, I32, P, P,
                                            ctypes.POINTER(I32), P, SZ, P]
        L.kv_evict_topk_indexed.restype = I32
        L.kv_evict_topk_indexed_noalloc.argtypes = [I32, P, P, P, P, I32, I32, I32, I32, I32, I32, P, P, P,
                                                    ctypes.POINTER(I32), P]
        L.kv_evict_topk_indexed_noalloc.restype = I32
        L.kv_append_indexed.argtypes = [P, P, I32, I32, I32, P, I32, P, I32, P, I32, I32, I32, I32, P, P, P, P]
        L.kv_append_indexed.restype = I32
        _lib = L
    return _lib


def _check(status):
    if status != DS_OK:
        L = lib()
        raise DeltasError(status, L.ds_status_string(status).decode() + ": " + L.ds_last_error().decode())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def frames_of_length(n: int, frame_len: int) -> int:
    if n <= 0:
        return 0
    if frame_len <= 0:
        return 1
    return (n + frame_len - 1) // frame_len


def gdn_shape(lengths, H_k, H_v, d, frame_len, drift_per_slice=False):
    """ds_gdn_shape for streams of the given (host-known) lengths."""
    lengths = [int(x) for x in lengths]
    return GdnShape(len(lengths), sum(lengths), H_k, H_v, d, d, frame_len,
                    sum(frames_of_length(n, frame_len) for n in lengths), int(bool(drift_per_slice)))


def gdn_workspace_bytes(shape: GdnShape, write_signal: bool = False) -> int:
    """Workspace bytes of gdn_chunk_fwd for this shape (with write_partials if write_signal)."""
    L = lib()
    q = L.ds_gdn_write_workspace_bytes if write_signal else L.ds_gdn_workspace_bytes
    return int(q(ctypes.byref(shape)))


def gdn_chunk_fwd(q, k, v, g, beta, lengths, frame_len, cu_seqlens=None, state_in=None, state_out=None,
                  o=None, o_dtype=torch.float32, scale=1.0, drift_partials=True, write_partials=False,
                  snapshots=False, workspace=None, stream=None, drift_per_slice=False):
    """One gated-delta-rule layer over packed streams (see gdn_chunk_fwd in deltas.h).

    q, k: bf16 [T][H_k][d]; v: bf16 [T][H_v][d]; g, beta: fp32 [T][H_v];
    lengths: host list of stream lengths; cu_seqlens: device int32 [B+1]
    (built from lengths when None).  Returns a dict with o, state,
    drift_partials [F][H_v][2] ([F][H_v * d / 16][2] with drift_per_slice;
    or None), write_partials [F][H_v][2] (the beta ||e|| sums and token
    counts, or None) and snapshots (or None).  Each output argument may be
    True (allocate), False (skip) or a tensor.
    """
    T, H_k, d = q.shape
    H_v = v.shape[1]
    shape = gdn_shape(lengths, H_k, H_v, d, frame_len, drift_per_slice)
    dev = q.device
    if cu_seqlens is None and shape.B > 1:
        cu = [0]
        for n in lengths:
            cu.append(cu[-1] + int(n))
        cu_seqlens = torch.tensor(cu, dtype=torch.int32, device=dev)
    if state_out is None:
        state_out = torch.empty((shape.B, H_v, d, d), dtype=torch.float32, device=dev)
    if o is None:
        o = torch.empty((T, H_v, d), dtype=o_dtype, device=dev)
    od = DS_BF16 if o.dtype == torch.bfloat16 else DS_F32
    pairs = H_v * (d // 16) if drift_per_slice else H_v
    dp = torch.empty((shape.n_frames, pairs, 2), dtype=torch.float32, device=dev) if drift_partials is True \
        else drift_partials if drift_partials is not False else None
    wp = torch.empty((shape.n_frames, H_v, 2), dtype=torch.float32, device=dev) if write_partials is True \
        else write_partials if write_partials is not False else None
    sn = torch.empty((shape.n_frames, H_v, d, d), dtype=torch.float32, device=dev) if snapshots is True \
        else snapshots if snapshots is not False else None
    need = gdn_workspace_bytes(shape, wp is not None)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    _check(lib().gdn_chunk_fwd(ctypes.byref(shape), _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta),
                               _ptr(cu_seqlens), _ptr(state_in), _ptr(state_out), _ptr(o), od, float(scale),
                               _ptr(dp), _ptr(wp), _ptr(sn), _ptr(workspace), workspace.numel(), _stream(stream)))
    return dict(o=o, state=state_out, drift_partials=dp, write_partials=wp, snapshots=sn, workspace=workspace)


def deltas_drift(partials, mode=LAYER_FROB, scores=None, stream=None):
    """Per-frame drift from [L][F][H_v][2] sums (see deltas_drift in deltas.h)."""
    L, F, H, _ = partials.shape
    if scores is None:
        shape = (L, F, H) if mode == PER_HEAD else (F,)
        scores = torch.empty(shape, dtype=torch.float32, device=partials.device)
    _check(lib().deltas_drift(_ptr(partials), L, F, H, mode, _ptr(scores), _stream(stream)))
    return scores


def deltas_drift_states(S_before, S_after, partials=None, stream=None):
    """Drift sums (||S_after - S_before||^2, ||S_before||^2) per state head from two
    fp32 tensors [L][B][H_v][d_v][d_k] (see deltas_drift_states in deltas.h).
    Returns partials [L][B][H_v][2]."""
    if S_before.shape != S_after.shape or S_before.dim() != 5:
        raise ValueError("S_before and S_after must both be [L][B][H_v][d_v][d_k]")
    L, B, H, dv, dk = S_before.shape
    if partials is None:
        partials = torch.empty((L, B, H, 2), dtype=torch.float32, device=S_before.device)
    _check(lib().deltas_drift_states(_ptr(S_before), _ptr(S_after), L, B, H, dv, dk, _ptr(partials), _stream(stream)))
    return partials


def gdn_decode_step(q, k, v, g, beta, state_in=None, state_out=None, o=None, o_dtype=torch.float32, scale=1.0,
                    stream=None):
    """One token per stream (see gdn_decode_step in deltas.h).

    q, k: bf16 [B][H_k][d]; v: bf16 [B][H_v][d]; g, beta: fp32 [B][H_v];
    state_in / state_out: fp32 [B][H_v][d][d] (state_out may be state_in).
    Returns dict(o, state).
    """
    B, H_k, d = q.shape
    H_v = v.shape[1]
    if k.shape != q.shape or v.shape != (B, H_v, d) or g.shape != (B, H_v) or beta.shape != (B, H_v):
        raise ValueError("shape mismatch")
    for t in (q, k, v):
        if t.dtype != torch.bfloat16 or not t.is_contiguous():
            raise ValueError("q, k, v must be contiguous bf16")
    for t in (g, beta):
        if t.dtype != torch.float32 or not t.is_contiguous():
            raise ValueError("g, beta must be contiguous fp32")
    dev = q.device
    if state_out is None:
        state_out = torch.empty((B, H_v, d, d), dtype=torch.float32, device=dev)
    for t in (state_in, state_out):
        if t is not None and (t.dtype != torch.float32 or t.shape != (B, H_v, d, d) or not t.is_contiguous()):
            raise ValueError("states must be contiguous fp32 [B][H_v][d][d]")
    if o is None:
        o = torch.empty((B, H_v, d), dtype=o_dtype, device=dev)
    od = DS_BF16 if o.dtype == torch.bfloat16 else DS_F32
    if o.shape != (B, H_v, d) or not o.is_contiguous() or o.dtype not in (torch.bfloat16, torch.float32):
        raise ValueError("o must be contiguous bf16 or fp32 [B][H_v][d]")
    _check(lib().gdn_decode_step(B, H_k, H_v, d, d, _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta),
                                 _ptr(state_in), _ptr(state_out), _ptr(o), od, float(scale), _stream(stream)))
    return dict(o=o, state=state_out)


def kv_workspace_bytes(n_layers, row_bytes, capacity) -> int:
    return int(lib().ds_kv_workspace_bytes(ctypes.byref(KvShape(n_layers, row_bytes, capacity))))


def kv_evict_topk(k_layers, v_layers, pos, chunk_id, chunk_scores, length, M, n_sink, n_window, n_buckets,
                  keep_out=None, workspace=None, stream=None):
    """One eviction step (see kv_evict_topk in deltas.h).

    k_layers / v_layers: lists of device tensors [capacity][row elems] (any
    dtype, rows of row_bytes bytes).  Returns (new_len, workspace).
    """
    L = len(k_layers)
    capacity = k_layers[0].shape[0]
    row_bytes = k_layers[0][0].numel() * k_layers[0].element_size()
    shape = KvShape(L, row_bytes, capacity)
    need = int(lib().ds_kv_workspace_bytes(ctypes.byref(shape)))
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=pos.device)
    kp = (ctypes.c_void_p * L)(*[t.data_ptr() for t in k_layers])
    vp = (ctypes.c_void_p * L)(*[t.data_ptr() for t in v_layers])
    new_len = ctypes.c_int32(0)
    _check(lib().kv_evict_topk(ctypes.byref(shape), kp, vp, _ptr(pos), _ptr(chunk_id), _ptr(chunk_scores),
                               int(chunk_scores.numel()), int(length), int(M), int(n_sink), int(n_window),
                               int(n_buckets), _ptr(keep_out), ctypes.byref(new_len), _ptr(workspace),
                               workspace.numel(), _stream(stream)))
    return int(new_len.value), workspace


def kv_indexed_workspace_bytes(capacity) -> int:
    return int(lib().ds_kv_indexed_workspace_bytes(int(capacity)))


def kv_evict_topk_indexed(pos, chunk_id, slot, chunk_scores, length, M, n_sink, n_window, n_buckets,
                          keep_out=None, free_out=None, workspace=None, stream=None):
    """One eviction step over a slot-indexed cache (see kv_evict_topk_indexed
    in deltas.h): pos, chunk_id and slot (int32 [capacity]) are compacted in
    place; the K/V rows are not touched.  Returns (new_len, workspace,
    free_out) where free_out[:length - M] lists the freed physical rows.
    """
    capacity = slot.numel()
    for t in (pos, chunk_id, slot):
        if t.dtype != torch.int32 or t.numel() != capacity:
            raise ValueError("pos, chunk_id and slot must be int32 tensors of the same length")
    if free_out is not None and int(length) > int(M) and free_out.numel() < int(length) - int(M):
        raise ValueError(f"free_out holds {free_out.numel()} entries, {int(length) - int(M)} needed")
    if keep_out is not None and keep_out.numel() < int(M):
        raise ValueError(f"keep_out holds {keep_out.numel()} entries, {int(M)} needed")
    need = int(lib().ds_kv_indexed_workspace_bytes(capacity))
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=pos.device)
    if free_out is None:
        free_out = torch.empty(max(int(length) - int(M), 1), dtype=torch.int32, device=pos.device)
    new_len = ctypes.c_int32(0)
    _check(lib().kv_evict_topk_indexed(capacity, _ptr(pos), _ptr(chunk_id), _ptr(slot), _ptr(chunk_scores),
                                       int(chunk_scores.numel()), int(length), int(M), int(n_sink), int(n_window),
                                       int(n_buckets), _ptr(keep_out), _ptr(free_out), ctypes.byref(new_len),
                                       _ptr(workspace), workspace.numel(), _stream(stream)))
    return int(new_len.value), workspace, free_out


def kv_evict_topk_indexed_noalloc(pos, chunk_id, slot, chunk_scores, length, M, n_sink, n_window, n_buckets,
                                  keep_out=None, free_out=None, outcome=None, stream=None):
    """kv_evict_topk_indexed with the library's fixed scratch instead of a
    workspace (see kv_evict_topk_indexed_noalloc in deltas.h); every output
    buffer is the caller's.  Returns new_len."""
    capacity = slot.numel()
    for t in (pos, chunk_id, slot):
        if t.dtype != torch.int32 or t.numel() != capacity:
            raise ValueError("pos, chunk_id and slot must be int32 tensors of the same length")
    if int(length) > int(M) and (free_out is None or free_out.numel() < int(length) - int(M)):
        raise ValueError(f"free_out must hold {int(length) - int(M)} entries")
    if keep_out is not None and keep_out.numel() < int(M):
        raise ValueError(f"keep_out holds {keep_out.numel()} entries, {int(M)} needed")
    if outcome is not None and (outcome.dtype != torch.int32 or outcome.numel() < 1):
        raise ValueError("outcome must be an int32 tensor of at least one element")
    new_len = ctypes.c_int32(0)
    _check(lib().kv_evict_topk_indexed_noalloc(capacity, _ptr(pos), _ptr(chunk_id), _ptr(slot), _ptr(chunk_scores),
                                               int(chunk_scores.numel()), int(length), int(M), int(n_sink),
                                               int(n_window), int(n_buckets), _ptr(keep_out), _ptr(free_out),
                                               _ptr(outcome), ctypes.byref(new_len), _stream(stream)))
    return int(new_len.value)


def kv_device_status(workspace):
    """(outcome, moves-stopped flag, wait-timeout flag) left by the last eviction
    that ran on this workspace (synchronises).  Outcome: 0 ok, 1 cache
    invariants broken, 2 keep count wrong, 3 gather wait timed out."""
    return workspace[:12].view(torch.int32).cpu().tolist()


def kv_outcome_word(workspace):
    """The outcome word of the last eviction on this workspace as a device
    int32 tensor of one element (a view: no synchronisation)."""
    return workspace[:4].view(torch.int32)


def kv_append_indexed(k_planes, v_planes, k_new, v_new, free_a, na, free_b, nb, free_rest, T, n, pos0, chunk, pos,
                      chunk_id, slot, stream=None):
    """A chunk's rows into a slot-indexed cache (see kv_append_indexed in
    deltas.h): k_planes and v_planes [L][capacity][row] (2-byte elements),
    k_new and v_new [L][>= T][row] with contiguous rows; tokens n .. n + T - 1
    take the first T rows of free_a[:na] ++ free_b[:nb], the rest of that list
    goes to free_rest.  pos, chunk_id, slot: int32 [capacity]."""
    L, capacity, row = k_planes.shape
    if v_planes.shape != k_planes.shape or k_new.shape[0] != L or v_new.shape[0] != L:
        raise ValueError("K/V planes and new rows must have matching layer counts and shapes")
    for t in (k_new, v_new):
        if t.shape[-1] != row or t.stride(-1) != 1 or t.stride(-2) != row or t.shape[1] < int(T):
            raise ValueError("new rows must be [L][>= T][row] with contiguous rows")
    for t in (k_planes, v_planes):
        if not t.is_contiguous():
            raise ValueError("K/V planes must be contiguous")
    for t in (pos, chunk_id, slot):
        if t.dtype != torch.int32 or t.numel() != capacity:
            raise ValueError("pos, chunk_id and slot must be int32 tensors of the cache capacity")
    row_bytes = row * k_planes.element_size()
    planes = (ctypes.c_void_p * (2 * L))(*[k_planes[l].data_ptr() for l in range(L)],
                                         *[v_planes[l].data_ptr() for l in range(L)])
    rows = (ctypes.c_void_p * (2 * L))(*[k_new[l].data_ptr() for l in range(L)],
                                       *[v_new[l].data_ptr() for l in range(L)])
    _check(lib().kv_append_indexed(planes, rows, 2 * L, row_bytes, capacity, _ptr(free_a), int(na), _ptr(free_b),
                                   int(nb), _ptr(free_rest), int(T), int(n), int(pos0), int(chunk), _ptr(pos),
                                   _ptr(chunk_id), _ptr(slot), _stream(stream)))
