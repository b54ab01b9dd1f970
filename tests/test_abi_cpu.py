"""The C ABI on a machine without a GPU: the library loads, exports every
symbol the header declares, and rejects bad arguments on the host before any
launch (so these calls never touch a device)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "deltas.h")


@pytest.fixture(scope="module")
def ds():
    import paper_2609_27470_amd as ds
    if not ds.LIB_PATH.exists():
        from paper_2609_27470_amd import build
        build.build()
    return ds


def _declared():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b([a-z_][a-z0-9_]*)\s*\(", txt)) - {"if", "sizeof"})


def test_header_declares_the_entry_points():
    names = _declared()
    for n in ["gdn_chunk_fwd", "deltas_drift", "deltas_drift_states", "kv_evict_topk", "ds_gdn_workspace_bytes",
              "ds_gdn_write_workspace_bytes",
              "ds_kv_workspace_bytes", "ds_status_string", "ds_last_error", "ds_kv_device_status",
              "kv_evict_topk_indexed", "ds_kv_indexed_workspace_bytes"]:
        assert n in names


def test_library_exports_every_declared_symbol(ds):
    L = ds.lib()
    for n in _declared():
        assert hasattr(L, n), n
    assert sorted(ds.EXPORTED) == sorted(_declared())


def test_status_strings(ds):
    L = ds.lib()
    assert L.ds_status_string(0) == b"ok"
    assert L.ds_status_string(5) == b"unsupported configuration"


def test_gdn_workspace_size(ds):
    s = ds.gdn_shape([32768], 16, 32, 128, 1024)
    assert s.n_frames == 32
    nb = ds.gdn_workspace_bytes(s)
    nw = ds.gdn_workspace_bytes(s, write_signal=True)
    tiles = 512
    per = 2 * 6 * 64 * 8 * 2 + 128 * 4     # T and P fragments (fp16) + decay factors per (tile, v-head)
    wr = 32768 * 32 * 8 * 4                # per-token write norms per 16-row slice
    qh = tiles * 16 * 64 * 128 * 2         # q tiles in fp16 per qk-head
    assert nb >= tiles * 32 * per + qh
    assert nb <= tiles * 32 * per + qh + 32 * 32 * 8 * 2 * 4 + 4096   # + drift sums per slice
    assert nw - nb >= wr and nw - nb <= wr + 256          # the norm area only when the signal is asked for
    # 256 (stream, v-head) pairs run whole-head: no fp16 q tiles, a frame-start state per head instead
    sw = ds.gdn_shape([4096] * 8, 16, 32, 128, 1024)
    tw = (8 * 4096 + 63 * 8) // 64   # tiles_max: room for one ragged tile per stream
    nbw = ds.gdn_workspace_bytes(sw)
    assert nbw >= tw * 32 * per + 8 * 32 * 128 * 128 * 4
    assert nbw <= tw * 32 * per + 8 * 32 * 128 * 128 * 4 + 4 * 32 * 8 * 8 * 2 * 4 + 8192
    bad = ds.gdn_shape([64], 1, 1, 96, 64)
    assert ds.gdn_workspace_bytes(bad) == 0


def _call_gdn(ds, shape, **kw):
    L = ds.lib()
    P = ctypes.c_void_p
    fake = P(1 << 20)      # never dereferenced: validation fails first
    args = dict(q=fake, k=fake, v=fake, g=fake, beta=fake, cu=None, sin=None, sout=fake, o=fake,
                od=ds.DS_F32, scale=1.0, dp=None, wp=None, sn=None, ws=fake, wsb=1 << 40)
    args.update(kw)
    return L.gdn_chunk_fwd(ctypes.byref(shape), args["q"], args["k"], args["v"], args["g"], args["beta"],
                           args["cu"], args["sin"], args["sout"], args["o"], args["od"], args["scale"],
                           args["dp"], args["wp"], args["sn"], args["ws"], args["wsb"], None)


def test_gdn_rejects_bad_arguments(ds):
    P = ctypes.c_void_p
    good = ds.gdn_shape([1024], 2, 4, 64, 256)
    assert _call_gdn(ds, ds.gdn_shape([64], 1, 1, 96, 64)) == 5            # head dim
    assert _call_gdn(ds, ds.gdn_shape([64], 3, 4, 64, 64)) == 2            # GQA ratio
    assert _call_gdn(ds, ds.gdn_shape([64], 1, 1, 64, 100)) == 5           # frame length
    assert _call_gdn(ds, good, q=None) == 1
    assert _call_gdn(ds, good, sout=None) == 1
    assert _call_gdn(ds, good, od=7) == 3
    assert _call_gdn(ds, good, v=P((1 << 20) + 4)) == 4                    # alignment
    assert _call_gdn(ds, good, wsb=16) == 8                                # workspace
    assert b"workspace" in ds.lib().ds_last_error()
    bad_slices = ds.gdn_shape([1024], 2, 4, 64, 256)
    bad_slices.drift_per_slice = 2
    assert _call_gdn(ds, bad_slices) == 6
    assert _call_gdn(ds, ds.gdn_shape([10, 20], 1, 1, 64, 64), cu=None) == 1
    assert b"cu_seqlens" in ds.lib().ds_last_error()


def test_drift_rejects_bad_arguments(ds):
    L = ds.lib()
    assert L.deltas_drift(None, 1, 1, 1, 9, None, None) == 6
    assert L.deltas_drift(None, 1, 1, 0, 0, None, None) == 2
    assert L.deltas_drift(None, 1, 4, 2, 0, None, None) == 1
    assert L.deltas_drift(None, 0, 4, 2, 0, None, None) == 0               # nothing to do


def test_drift_states_rejects_bad_arguments(ds):
    L = ds.lib()
    assert L.deltas_drift_states(None, None, 1, 1, 0, 8, 8, None, None) == 2   # H_v < 1
    assert L.deltas_drift_states(None, None, 1, 1, 1, 3, 3, None, None) == 5   # d_v d_k % 4
    assert L.deltas_drift_states(None, None, 1, 1, 1, 8, 8, None, None) == 1   # NULL
    assert L.deltas_drift_states(None, None, 0, 1, 1, 8, 8, None, None) == 0   # nothing to do
    assert L.deltas_drift_states(8, 16, 1, 1, 1, 8, 8, 32, None) == 4          # misaligned


def test_kv_rejects_bad_arguments_and_noop(ds):
    L = ds.lib()
    shp = ds.KvShape(8, 4096, 17408)
    assert ds.kv_workspace_bytes(8, 4096, 17408) > 17408 * 4 * 5
    assert ds.kv_workspace_bytes(8, 4008, 17408) == 0
    nl = ctypes.c_int32(-1)
    P = ctypes.c_void_p
    f = P(1 << 20)

    layers = (P * 8)(*([1 << 20] * 8))   # host arrays of (never dereferenced) device pointers

    def call(length, M, ns, nw, nb, shape=shp, ws=f, wsb=1 << 40):
        return L.kv_evict_topk(ctypes.byref(shape), layers, layers, f, f, f, 1024, length, M, ns, nw, nb,
                               None, ctypes.byref(nl), ws, wsb, None)

    assert call(100, 200, 4, 8, 4) == 0 and nl.value == 100                 # under budget: no-op
    assert call(20000, 16384, 0, 0, 1) == 2                                 # len > capacity
    assert call(17408, 16, 10, 10, 1) == 6                                  # reserved > M
    assert call(17408, 16384, 0, 0, 65) == 6                                # too many spans
    assert call(17408, 16384, 0, 0, 1, wsb=8) == 8                          # workspace
    assert call(17408, 16384, 0, 0, 1, shape=ds.KvShape(40, 4096, 17408)) == 5


def test_kv_indexed_rejects_bad_arguments_and_noop(ds):
    L = ds.lib()
    P = ctypes.c_void_p
    f = P(1 << 20)
    nl = ctypes.c_int32(-1)
    assert ds.kv_indexed_workspace_bytes(17408) > 17408 * 4 * 5
    assert ds.kv_indexed_workspace_bytes(0) == 0
    # no gather flags: far smaller than the gather variant's workspace
    assert ds.kv_indexed_workspace_bytes(17408) < ds.kv_workspace_bytes(8, 4096, 17408)

    def call(length, M, ns, nw, nb, cap=17408, slot=f, free=f, ws=f, wsb=1 << 40):
        return L.kv_evict_topk_indexed(cap, f, f, slot, f, 1024, length, M, ns, nw, nb, None, free,
                                       ctypes.byref(nl), ws, wsb, None)

    assert call(100, 200, 4, 8, 4, slot=None, free=None) == 0 and nl.value == 100   # under budget: no-op
    assert call(20000, 16384, 0, 0, 1) == 2                                 # len > capacity
    assert call(17408, 16, 10, 10, 1) == 6                                  # reserved > M
    assert call(17408, 16384, 0, 0, 65) == 6                                # too many spans
    assert call(17408, 16384, 0, 0, 1, slot=None) == 1                      # slot table required
    assert call(17408, 16384, 0, 0, 1, free=None) == 1                      # free list required
    assert call(17408, 16384, 0, 0, 1, free=P((1 << 20) + 4)) == 4          # alignment
    assert call(17408, 16384, 0, 0, 1, wsb=8) == 8                          # workspace
    assert L.kv_evict_topk_indexed(17408, f, f, f, f, 1024, 17408, 16384, 0, 0, 1, None, f, None, f,
                                   1 << 40, None) == 1                      # new_len required


def test_decode_rejects_bad_arguments(ds):
    L = ds.lib()
    P = ctypes.c_void_p
    f = P(1 << 20)

    def call(B=4, H_k=2, H_v=4, dk=128, dv=128, q=f, st_in=None, st_out=P(1 << 30), od=ds.DS_F32):
        return L.gdn_decode_step(B, H_k, H_v, dk, dv, q, f, f, f, f, st_in, st_out, f, od, 1.0, None)

    assert call(B=-1) == 2
    assert call(H_k=3) == 2                         # H_v not a multiple of H_k
    assert call(dk=96, dv=96) == 5
    assert call(dk=64, dv=128) == 5
    assert call(od=7) == 3
    assert call(B=0, q=None) == 0                   # nothing to do
    assert call(q=None) == 1
    assert call(q=P((1 << 20) + 8)) == 4
    assert call(st_in=P(1 << 30), st_out=P((1 << 30) + 4096)) == 6   # overlapping states
    assert b"overlap" in L.ds_last_error()


def test_streaming_session_validates_on_host(ds):
    """The streaming session's argument checks run before any device work."""
    from paper_2609_27470_amd.streaming import DeltaSStream
    with pytest.raises(ValueError):
        DeltaSStream(2, 2, 4, 64, 1, 64, 100, 132, 8, n_sink=50, n_window=60, device="cpu")
    s = DeltaSStream(2, 2, 4, 64, 1, 64, 600, 132, 8, n_sink=4, n_window=256, device="cpu")
    assert s.capacity == 600 + 132 and s.state.shape == (2, 1, 4, 64, 64)
    import torch
    bad = [(torch.zeros((140, 2, 64), dtype=torch.bfloat16),) * 5] * 2
    with pytest.raises(ValueError):
        s.step(bad, None, None)                       # chunk longer than max_chunk


def test_noalloc_eviction_host_checks(ds):
    """kv_evict_topk_indexed_noalloc: capacities beyond its fixed scratch are
    refused before anything runs; a call that does not evict touches nothing;
    the indexed workspace of the largest accepted capacity fits the 4 MiB
    scratch."""
    L = ds.lib()
    n = ctypes.c_int32(-1)
    P = ctypes.c_void_p
    cap = ds.NOALLOC_MAX_CAPACITY
    assert L.kv_evict_topk_indexed_noalloc(cap + 1, None, None, None, None, 1, 10, 5, 0, 0, 1, None, None, None,
                                           ctypes.byref(n), None) == 5
    assert b"fixed scratch" in L.ds_last_error()
    assert L.kv_evict_topk_indexed_noalloc(cap, None, None, None, None, 1, 100, 200, 0, 0, 1, None, None, None,
                                           ctypes.byref(n), None) == 0
    assert n.value == 100
    assert L.kv_evict_topk_indexed_noalloc(cap, None, None, None, None, 1, 300, 200, 0, 0, 1, None, None, None,
                                           None, None) == 1
    assert L.ds_kv_indexed_workspace_bytes(cap) <= 4 << 20


def test_append_host_checks(ds):
    """kv_append_indexed refuses, before any launch, plane counts outside
    1..64, rows that are not whole 16-byte units, a chunk past the capacity, a
    free list shorter than the chunk or longer than the cache, NULL and
    misaligned pointers; an empty chunk with an empty list does nothing."""
    L = ds.lib()
    P = ctypes.c_void_p
    fake = 1 << 20                                   # never dereferenced: every call below fails on the host
    planes = (P * 2)(fake, fake)
    rows = (P * 2)(fake, fake)
    ok = dict(planes=planes, rows=rows, n_planes=2, row_bytes=64, capacity=100, fa=fake, na=50, fb=None, nb=0,
              rest=fake, T=10, n=40, pos0=0, chunk=0, pos=fake, cid=fake, slot=fake)

    def call(**kw):
        a = dict(ok, **kw)
        return L.kv_append_indexed(a["planes"], a["rows"], a["n_planes"], a["row_bytes"], a["capacity"], a["fa"],
                                   a["na"], a["fb"], a["nb"], a["rest"], a["T"], a["n"], a["pos0"], a["chunk"],
                                   a["pos"], a["cid"], a["slot"], None)

    assert call(n_planes=0) == 5 and call(n_planes=65) == 5
    assert call(row_bytes=24) == 2 and call(row_bytes=65552) == 5
    assert call(n=95) == 2                           # n + T > capacity
    assert call(na=5) == 6                           # free list shorter than the chunk
    assert call(na=60, nb=60) == 6                   # free list longer than the cache
    assert call(pos=None) == 1 and call(fa=None) == 1
    assert call(planes=(P * 2)(fake, fake + 8)) == 4
    assert call(slot=fake + 2) == 4
    assert b"int32 pointer" in L.ds_last_error()
    assert call(T=0, na=0, planes=None, rows=None) == 0
