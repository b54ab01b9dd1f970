"""Streaming DeltaS over a hybrid model's layers, chunk by chunk (Section 3.3,
Algorithm 1), with question-time save and restore of the memory.

One `DeltaSStream` holds, on the device, everything the retention policy
carries from chunk to chunk: the fp32 state of every linear-attention layer,
the full-attention layers' K/V cache with each slot's position and chunk id,
and the drift score of every chunk seen so far.  `step` consumes one chunk of
any length (a chunk of the paper is one second of video -- two frames at
2 fps -- of 118 to 132 tokens): each linear-attention layer runs `gdn_chunk_fwd` over the chunk as
one frame (so its drift sums cover exactly the chunk), `deltas_drift` turns
the per-layer sums into the chunk's score (Eq. 3, mean over layers), the
chunk's K/V rows are appended, and `kv_evict_topk` cuts the cache back to the
budget when it overflows.  `save` and `restore` copy that memory aside and
back, so a question can be answered (more tokens, decode steps) and the
stream then resumes exactly where it was.

Only argument marshalling and buffer bookkeeping happen here; every step of
the computation runs in the HIP kernels behind the C ABI.  The snapshot
copies are plain device copies.

A chunk is a tiny call per layer (about 125 tokens), so launching the layers
one by one from the host costs more than the kernels themselves.
`capture_graph` records all layers and the score of one chunk in a HIP graph
over fixed input buffers (`inputs`); the chunk's length is read on the
device, so a graph serves every chunk length up to the capacity it was
recorded for.  Two are recorded: one for chunks of at most two tiles
(SMALL_CHUNK tokens), whose layer calls take the library's one-launch path,
and one for max_chunk.  The
append and the eviction stay outside the graph: the cache length they work
from is host state.

By default (`indexed=True`) the cache is addressed through a slot table
(logical token i lives in physical row slot[i]): eviction is
`kv_evict_topk_indexed`, which keeps exactly the same tokens and moves no K/V
byte, and a chunk's rows are written into the rows the last eviction freed
(`kv_append_indexed`: rows and table entries in one launch).
The logical view (rows slot[0..length)) equals the order-preserving cache
that `indexed=False` keeps with `kv_evict_topk` (rows compacted in place).

Every eviction's outcome word (0 = ok) is folded into a device-side maximum
without a host synchronisation; `check()` reads it and raises if any
eviction since the session began reported a failure, and `save`, `restore`
and `logical_rows` call it.
"""
from __future__ import annotations

import contextlib
from dataclasses import dataclass

import torch

from . import (LAYER_FROB, deltas_drift, gdn_chunk_fwd, gdn_shape, gdn_workspace_bytes, kv_append_indexed,
               kv_evict_topk, kv_evict_topk_indexed, kv_indexed_workspace_bytes, kv_outcome_word, kv_workspace_bytes)

# the longest chunk whose layer calls fit two 64-token tiles
SMALL_CHUNK = 128


class EvictionFailed(RuntimeError):
    """An eviction reported a failure on the device (see ds_kv_device_status)."""


def _on(stream):
    return torch.cuda.stream(stream) if stream is not None else contextlib.nullcontext()


@dataclass
class Snapshot:
    """Device copies of a stream's memory at one point (see DeltaSStream.save)."""
    state: torch.Tensor
    k: torch.Tensor
    v: torch.Tensor
    pos: torch.Tensor
    chunk_id: torch.Tensor
    scores: torch.Tensor
    slot: object
    free: object
    length: int
    n_chunks: int
    next_pos: int


class DeltaSStream:
    """Memory of one video stream under the DeltaS retention policy.

    n_layers linear-attention layers of (H_k, H_v, d) heads; kv_layers
    full-attention layers whose K and V rows are row_elems bf16 values per
    token; budget M tokens, cache capacity M + max_chunk; the policy's sink,
    window and span counts (the paper uses 4, 1024 and 4).  `o` holds every
    linear-attention layer's output of the latest chunk ([layer][token]
    [H_v][d] in o_dtype).
    """

    def __init__(self, n_layers, H_k, H_v, d, kv_layers, row_elems, M, max_chunk, max_chunks,
                 n_sink=4, n_window=1024, n_buckets=4, score_mode=LAYER_FROB, device="cuda", indexed=True,
                 o_dtype=torch.bfloat16):
        if n_sink + n_window > M:
            raise ValueError("sink + window exceed the budget")
        dev = torch.device(device)
        self.dev = dev
        self.L, self.H_k, self.H_v, self.d = n_layers, H_k, H_v, d
        self.M, self.max_chunk = M, max_chunk
        self.policy = (n_sink, n_window, n_buckets)
        self.score_mode = score_mode
        self.capacity = M + max_chunk
        self.state = torch.zeros((n_layers, 1, H_v, d, d), dtype=torch.float32, device=dev)
        # Eq. 3 pools a layer's heads, so for it the drift pairs are taken per
        # 16-row slice of the state (no exchange between a head's workgroups)
        self.per_slice = score_mode == LAYER_FROB
        pairs = H_v * (d // 16) if self.per_slice else H_v
        self.partials = torch.zeros((n_layers, 1, pairs, 2), dtype=torch.float32, device=dev)
        self.o = torch.empty((n_layers, max_chunk, H_v, d), dtype=o_dtype, device=dev)
        self.k = torch.zeros((kv_layers, self.capacity, row_elems), dtype=torch.int16, device=dev)
        self.v = torch.zeros((kv_layers, self.capacity, row_elems), dtype=torch.int16, device=dev)
        self.pos = torch.zeros(self.capacity, dtype=torch.int32, device=dev)
        self.chunk_id = torch.zeros(self.capacity, dtype=torch.int32, device=dev)
        self.scores = torch.zeros(max_chunks, dtype=torch.float32, device=dev)
        shape = gdn_shape([max_chunk], H_k, H_v, d, 0)
        self.gdn_ws = torch.empty(max(gdn_workspace_bytes(shape), 1), dtype=torch.uint8, device=dev)
        self.indexed = indexed
        if indexed:
            self.slot = torch.zeros(self.capacity, dtype=torch.int32, device=dev)
            # rows not in use: self._free_bufs[self._fa][:self._na] followed by
            # self.freed[:self._nb] (the rows the last eviction freed); the
            # append takes the first T and writes the rest into the other buffer
            self._free_bufs = [torch.arange(self.capacity, dtype=torch.int32, device=dev),
                               torch.empty(self.capacity, dtype=torch.int32, device=dev)]
            self._fa, self._na, self._nb = 0, self.capacity, 0
            self.freed = torch.empty(self.capacity, dtype=torch.int32, device=dev)
            self.kv_ws = torch.empty(max(kv_indexed_workspace_bytes(self.capacity), 1), dtype=torch.uint8, device=dev)
        else:
            self.slot = None
            self.kv_ws = torch.empty(max(kv_workspace_bytes(kv_layers, row_elems * 2, self.capacity), 1),
                                     dtype=torch.uint8, device=dev)
        self.kv_fail = torch.zeros(1, dtype=torch.int32, device=dev)   # max outcome word of every eviction
        self.graph = None
        self.length = 0      # tokens in the cache
        self.n_chunks = 0    # chunks seen (the next chunk's id)
        self.next_pos = 0    # position of the next token

    @property
    def free(self):
        """The physical rows not in use, in the order the next chunk takes them
        (a new device tensor; None for the contiguous cache)."""
        if not self.indexed:
            return None
        return torch.cat([self._free_bufs[self._fa][:self._na], self.freed[:self._nb]])

    @free.setter
    def free(self, rows):
        if not self.indexed:
            raise ValueError("the contiguous cache has no free list")
        rows = rows.to(device=self.dev, dtype=torch.int32).reshape(-1)
        if rows.numel() > self.capacity:
            raise ValueError("free list longer than the cache")
        self._free_bufs[0][:rows.numel()].copy_(rows)
        self._fa, self._na, self._nb = 0, rows.numel(), 0

    def step(self, layer_inputs, k_rows, v_rows, stream=None):
        """Consume one chunk.

        layer_inputs: per linear-attention layer a tuple (q, k, v, g, beta) of
        the chunk's T tokens (bf16 [T][H_k][d], bf16 [T][H_k][d], bf16
        [T][H_v][d], fp32 [T][H_v] twice); k_rows, v_rows: the chunk's cache
        rows, int16 (bf16 bits) [kv_layers][T][row_elems].  Returns the number
        of tokens kept in the cache.
        """
        T = layer_inputs[0][0].shape[0]
        if not 0 < T <= self.max_chunk:
            raise ValueError(f"chunk of {T} tokens (1..{self.max_chunk})")
        if len(layer_inputs) != self.L:
            raise ValueError("one input tuple per linear-attention layer")
        c = self.n_chunks
        if c >= self.scores.numel():
            raise ValueError("score table full")
        # every launch and copy of the step on one stream (the caller's, else the current one)
        with _on(stream):
            for l, (q, k, v, g, beta) in enumerate(layer_inputs):
                st = self.state[l]
                gdn_chunk_fwd(q, k, v, g, beta, [T], 0, state_in=st, state_out=st, o=self.o[l, :T],
                              drift_partials=self.partials[l], workspace=self.gdn_ws, drift_per_slice=self.per_slice)
            deltas_drift(self.partials, self.score_mode, scores=self.scores[c:c + 1])
            return self._append_and_evict(T, k_rows, v_rows)

    def check(self):
        """Raise EvictionFailed if any eviction of this session reported a
        failure on the device (synchronises with the current stream)."""
        code = int(self.kv_fail.item())
        if code != 0:
            raise EvictionFailed(f"an eviction reported outcome {code} (1: cache invariants broken, "
                                 "2: keep count wrong, 3: gather wait timed out)")

    def _append_and_evict(self, T, k_rows, v_rows):
        c = self.n_chunks
        n = self.length
        if self.indexed:   # rows, positions, chunk ids and slots in one launch
            rest = self._free_bufs[1 - self._fa]
            kv_append_indexed(self.k, self.v, k_rows, v_rows, self._free_bufs[self._fa], self._na, self.freed,
                              self._nb, rest, T, n, self.next_pos, c, self.pos, self.chunk_id, self.slot)
            self._fa, self._na, self._nb = 1 - self._fa, self._na + self._nb - T, 0
        else:
            self.k[:, n:n + T].copy_(k_rows)
            self.v[:, n:n + T].copy_(v_rows)
            self.pos[n:n + T] = torch.arange(self.next_pos, self.next_pos + T, dtype=torch.int32, device=self.dev)
            self.chunk_id[n:n + T] = c
        self.next_pos += T
        self.n_chunks = c + 1
        n += T
        ns, nw, nb = self.policy
        if self.indexed:
            new_len, _, _ = kv_evict_topk_indexed(self.pos, self.chunk_id, self.slot, self.scores[:self.n_chunks],
                                                  n, self.M, ns, nw, nb, free_out=self.freed, workspace=self.kv_ws)
            self._nb = max(n - self.M, 0)
            self.length = new_len
        else:
            self.length, _ = kv_evict_topk(list(self.k), list(self.v), self.pos, self.chunk_id,
                                           self.scores[:self.n_chunks], n, self.M, ns, nw, nb,
                                           workspace=self.kv_ws)
        if n > self.M:   # the call evicted: fold its outcome word in (device side, no sync)
            torch.maximum(self.kv_fail, kv_outcome_word(self.kv_ws), out=self.kv_fail)
        return self.length

    def logical_rows(self):
        """(K, V) rows of the cached tokens in logical (arrival) order, [kv_layers][length][row]."""
        self.check()
        n = self.length
        if not self.indexed:
            return self.k[:, :n], self.v[:, :n]
        idx = self.slot[:n].to(torch.int64)
        return self.k[:, idx], self.v[:, idx]

    def capture_graph(self):
        """Allocate the fixed input buffers and record one chunk's linear-attention
        work (every layer, then the chunk score) as a HIP graph; see step_inputs."""
        L, Tm, H_k, H_v, d, dev = self.L, self.max_chunk, self.H_k, self.H_v, self.d, self.dev
        self.inputs = (torch.zeros((L, Tm, H_k, d), dtype=torch.bfloat16, device=dev),
                       torch.zeros((L, Tm, H_k, d), dtype=torch.bfloat16, device=dev),
                       torch.zeros((L, Tm, H_v, d), dtype=torch.bfloat16, device=dev),
                       torch.zeros((L, Tm, H_v), dtype=torch.float32, device=dev),
                       torch.zeros((L, Tm, H_v), dtype=torch.float32, device=dev))
        self.cu = torch.tensor([0, Tm], dtype=torch.int32, device=dev)
        self.score_buf = torch.zeros(1, dtype=torch.float32, device=dev)
        self.graphs = {}
        for cap in sorted({min(Tm, SMALL_CHUNK), Tm}):
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                self._layers_fixed(cap)
            torch.cuda.synchronize()
            self.graphs[cap] = g
        self.graph = self.graphs[Tm]

    def _layers_fixed(self, cap):
        q, k, v, g, b = self.inputs
        for l in range(self.L):
            st = self.state[l]
            gdn_chunk_fwd(q[l], k[l], v[l], g[l], b[l], [cap], 0, cu_seqlens=self.cu, state_in=st,
                          state_out=st, o=self.o[l], drift_partials=self.partials[l], workspace=self.gdn_ws,
                          drift_per_slice=self.per_slice)
        deltas_drift(self.partials, self.score_mode, scores=self.score_buf)

    def step_inputs(self, T, k_rows, v_rows):
        """Consume one chunk of T tokens whose layer inputs the caller has written
        into self.inputs (q, k, v, g, beta, each [layer][token]...) rows [0, T);
        replays the captured graph.  Same results as step, bit for bit."""
        if self.graph is None:
            raise RuntimeError("capture_graph() first")
        if not 0 < T <= self.max_chunk:
            raise ValueError(f"chunk of {T} tokens (1..{self.max_chunk})")
        c = self.n_chunks
        if c >= self.scores.numel():
            raise ValueError("score table full")
        self.cu[1:2].fill_(T)
        self.graphs[min(self.graphs) if T <= min(self.graphs) else self.max_chunk].replay()
        self.scores[c:c + 1].copy_(self.score_buf)
        return self._append_and_evict(T, k_rows, v_rows)

    def save(self) -> Snapshot:
        """Copy the memory aside (question time)."""
        self.check()
        n = self.length
        if self.indexed:   # rows stay where they are: keep the physical planes and the tables
            return Snapshot(self.state.clone(), self.k.clone(), self.v.clone(), self.pos[:n].clone(),
                            self.chunk_id[:n].clone(), self.scores[:self.n_chunks].clone(), self.slot[:n].clone(),
                            self.free, n, self.n_chunks, self.next_pos)
        return Snapshot(self.state.clone(), self.k[:, :n].clone(), self.v[:, :n].clone(), self.pos[:n].clone(),
                        self.chunk_id[:n].clone(), self.scores[:self.n_chunks].clone(), None, None, n, self.n_chunks,
                        self.next_pos)

    def restore(self, s: Snapshot):
        """Put a saved memory back; the stream continues as if nothing had run since."""
        self.check()
        n = s.length
        self.state.copy_(s.state)
        if self.indexed:
            self.k.copy_(s.k)
            self.v.copy_(s.v)
            self.slot[:n].copy_(s.slot)
            self.free = s.free
        else:
            self.k[:, :n].copy_(s.k)
            self.v[:, :n].copy_(s.v)
        self.pos[:n].copy_(s.pos)
        self.chunk_id[:n].copy_(s.chunk_id)
        self.scores[:s.n_chunks].copy_(s.scores)
        self.length, self.n_chunks, self.next_pos = n, s.n_chunks, s.next_pos
