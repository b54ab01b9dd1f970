/*
 * deltas.h -- C ABI of the DeltaS hot path on MI355X (gfx950).
 *
 * The operations, following the paper (DeltaS: reading the gated
 * linear-attention state for KV-cache eviction in streaming video):
 *
 *   gdn_chunk_fwd   gated-delta-rule forward of one linear-attention layer
 *                   (Section 3.2, Eq. 1 / Eq. 2) over packed streams, with
 *                   the per-frame state-drift sums of Eq. 3 fused in;
 *   gdn_decode_step one token per stream of the same recurrence, batched
 *                   over streams (the step that follows a state restore);
 *   deltas_drift    per-frame drift scores from those sums (Eq. 3 and
 *                   Algorithm 1's mean over layers);
 *   kv_evict_topk   one eviction step of Algorithm 1 / Section 3.3:
 *                   sink + recent window + N temporal spans with per-span
 *                   top-k and fill, then an order-preserving in-place gather
 *                   of every full-attention layer's K and V rows.
 *   kv_evict_topk_indexed
 *                   the same step over a slot-indexed cache: identical
 *                   selection, the K and V rows stay where they are.
 *   kv_append_indexed
 *                   a chunk's K and V rows and table entries into such a
 *                   cache, in one launch.
 *
 * Conventions shared by every entry point
 *   - Pointers are DEVICE pointers unless marked "host".  The caller owns
 *     every buffer; the library never allocates device memory.  Calls that
 *     need scratch memory take a caller-provided workspace whose size comes
 *     from the matching *_workspace_bytes query.
 *   - Every call is asynchronous on `stream` (a hipStream_t passed as void*;
 *     NULL is the default stream) and never synchronises the host.
 *   - Arguments are validated on the host before any launch; on failure the
 *     call returns a non-zero status and writes nothing.  Launch failures
 *     return DS_E_HIP.  Faults inside a kernel surface at the caller's next
 *     synchronisation.  Nothing aborts or throws across this boundary.
 *   - Device pointers must be 16-byte aligned.
 *   - The library keeps no state between calls except a thread-local string
 *     describing the last error (ds_last_error).
 */
#ifndef DELTAS_H
#define DELTAS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t ds_status;
enum {
    DS_OK = 0,
    DS_E_NULL = 1,        /* a required pointer is NULL */
    DS_E_SHAPE = 2,       /* inconsistent sizes */
    DS_E_DTYPE = 3,       /* unknown dtype code */
    DS_E_ALIGN = 4,       /* pointer not 16-byte aligned */
    DS_E_UNSUPPORTED = 5, /* valid but not implemented (e.g. head dim) */
    DS_E_ARG = 6,         /* other invalid argument */
    DS_E_HIP = 7,         /* a HIP runtime call failed */
    DS_E_WORKSPACE = 8    /* workspace NULL or smaller than required */
};

enum { DS_BF16 = 0, DS_F32 = 1 };

enum {
    DS_DRIFT_LAYER_FROB = 0, /* Eq. 3: per layer ||dS||_F / ||S_before||_F over all its heads, mean over layers */
    DS_DRIFT_HEAD_MEAN = 1,  /* mean over layers and heads of the per-head ratio */
    DS_DRIFT_PER_HEAD = 2,   /* the per-(layer, frame, head) ratios */
    DS_WRITE_MEAN = 3        /* write_partials of gdn_chunk_fwd: mean over layers, heads and the
                                frame's tokens of beta ||e|| (the beta ||e|| signal) */
};

/* Static description of a status code. */
const char *ds_status_string(ds_status s);
/* Detail of the last failing call on this host thread ("" if none). */
const char *ds_last_error(void);

/* ------------------------------------------------------------------------
 * gdn_chunk_fwd -- one gated-delta-rule layer over packed streams
 * ------------------------------------------------------------------------
 * Computes, for every stream b and v-head j (reading qk-head
 * h = j * H_k / H_v), token by token (Section 3.2, Eq. 2):
 *     alpha_t = exp(g_t);  e_t = beta_t (v_t - alpha_t S_{t-1} k_t)
 *     S_t = alpha_t S_{t-1} + e_t k_t^T;   o_t = scale * S_t q_t
 * where S (d_v x d_k, fp32) starts from state_in.  The kernels evaluate it
 * tile by tile (64 tokens) in an equivalent closed form; results match the
 * recurrence up to rounding.
 *
 * Frames: every frame_len tokens from each stream's first token, plus the
 * stream's ragged tail, is one frame (frame_len = 0: the whole stream is one
 * frame).  At the end of frame f the call writes, per v-head, the two sums
 * behind the state drift of Eq. 3:
 *     drift_partials[f][j][0] = ||S_end - S_start||_F^2
 *     drift_partials[f][j][1] = ||S_start||_F^2
 * (S_start = the state when the frame began, held on chip -- the temporary
 * copy of the previous state of Section 3.2), and optionally the state
 * itself into snapshots[f][j].  Frames are numbered stream by stream.
 * With shape->drift_per_slice = 1 the pairs are written per slice of 16
 * state rows instead: drift_partials[f][j][s] (s < d_v / 16) covers rows
 * 16 s .. 16 s + 15 of S, and the per-head pair is their sum.  Eq. 3 pools
 * all heads of a layer, so deltas_drift's DS_DRIFT_LAYER_FROB over these
 * pairs (passed as H_v * d_v / 16 "heads") is the same score; the kernels
 * then need no exchange between the workgroups of a head, which saves about
 * a microsecond per call (a few percent of a 1024-token call).
 * Optionally also the write-magnitude signal compared with the drift in the
 * appendix on retention signals (row beta ||e||):
 *     write_partials[f][j][0] = sum over the frame's tokens of beta_t ||e_t||_2
 *     write_partials[f][j][1] = number of tokens in the frame
 * with e_t = v_t - alpha_t S_{t-1} k_t; beta_t ||e_t|| is the Frobenius norm of
 * the token's rank-one write for unit keys.  The writes enter this sum in
 * fp16, so it carries a relative error of about 1e-3.
 *
 * Shapes and layouts (row-major, innermost last):
 *   q, k        bf16 [T_total][H_k][d_k]  (k expected L2-normalised per row)
 *   v           bf16 [T_total][H_v][d_v]
 *   g, beta     fp32 [T_total][H_v]       (g <= 0 is the log decay)
 *   cu_seqlens  int32 [B+1], stream b = tokens [cu[b], cu[b+1]);
 *               nondecreasing, cu[0] = 0, cu[B] <= T_total.  The lengths
 *               are read on the device, so T_total may be an upper bound
 *               (it sizes the workspace and the grids): one captured graph
 *               then serves chunks of any length up to it.  May be NULL
 *               when B == 1 (the stream is [0, T_total)); required when
 *               B > 1.  (Out-of-range values are clamped so that no access
 *               leaves the buffers; results are then unspecified.)
 *   state_in    fp32 [B][H_v][d_v][d_k] or NULL (zeros)
 *   state_out   fp32 [B][H_v][d_v][d_k]; may alias state_in
 *   o           [T_total][H_v][d_v] of dtype o_dtype (DS_BF16 or DS_F32)
 *   drift_partials fp32 [n_frames][H_v][2] (drift_per_slice = 1:
 *               [n_frames][H_v][d_v / 16][2]) or NULL
 *   write_partials fp32 [n_frames][H_v][2] or NULL
 *   snapshots   fp32 [n_frames][H_v][d_v][d_k] or NULL
 * Supported: d_k = d_v in {64, 128}; H_v a multiple of H_k; frame_len a
 * multiple of 64 or 0.  bf16 inputs and the state enter the matrix cores as
 * fp16 (fp32 accumulation), so |q|, |k|, |v| and the state's entries must
 * stay below 65504.
 * n_frames is the number of frames of all streams at the lengths the host
 * knows (frame_len = 0: B); for frames that the device lengths do not
 * reach, the drift and write sums are zero and no snapshot is written.
 */
typedef struct {
    int32_t B;         /* number of streams (>= 1) */
    int32_t T_total;   /* tokens over all streams (>= 0) */
    int32_t H_k;       /* query/key heads */
    int32_t H_v;       /* value heads (state heads) */
    int32_t d_k;       /* key head dim */
    int32_t d_v;       /* value head dim */
    int32_t frame_len; /* tokens per frame (multiple of 64) or 0 */
    int32_t n_frames;  /* frames over all streams */
    int32_t drift_per_slice; /* 0: drift_partials [n_frames][H_v][2]; 1: [n_frames][H_v][d_v / 16][2] */
} ds_gdn_shape;

/* Workspace bytes gdn_chunk_fwd needs for this shape when write_partials is
 * NULL (0 on a bad shape). */
size_t ds_gdn_workspace_bytes(const ds_gdn_shape *shape);
/* Workspace bytes gdn_chunk_fwd needs for this shape when write_partials is
 * given: the above plus 4 * T_total * H_v * d_v / 16 bytes of per-token norm
 * slices (0 on a bad shape). */
size_t ds_gdn_write_workspace_bytes(const ds_gdn_shape *shape);

ds_status gdn_chunk_fwd(const ds_gdn_shape *shape, const void *q, const void *k, const void *v,
                        const float *g, const float *beta, const int32_t *cu_seqlens,
                        const float *state_in, float *state_out, void *o, int32_t o_dtype,
                        float scale, float *drift_partials, float *write_partials, float *snapshots,
                        void *workspace, size_t workspace_bytes, void *stream);

/* ------------------------------------------------------------------------
 * gdn_decode_step -- one token of Eq. 2 for each of B streams
 * ------------------------------------------------------------------------
 * For every stream b and v-head j (reading qk-head j * H_k / H_v), with
 * alpha = exp(g[b][j]) and S = state_in[b][j] (zeros if state_in is NULL):
 *     e = beta (v - alpha S k),  S' = alpha S + e k^T,  o = scale S' q
 * (Section 3.2, Eq. 2; o read after the update as in gdn_chunk_fwd).
 * Layouts: q, k bf16 [B][H_k][d_k]; v bf16 [B][H_v][d_v]; g, beta fp32
 * [B][H_v]; state_in, state_out fp32 [B][H_v][d_v][d_k]; o [B][H_v][d_v]
 * in o_dtype (DS_BF16 or DS_F32).  state_out may equal state_in (in-place
 * update) but must not otherwise overlap it.  Arithmetic is fp32 (no
 * matrix cores); row sums use a fixed order, so results are reproducible.
 * No drift sums (a decode step is not a frame).  Requires d_k = d_v in
 * {64, 128}, H_v a multiple of H_k; B = 0 does nothing.  No workspace.
 */
ds_status gdn_decode_step(int32_t B, int32_t H_k, int32_t H_v, int32_t d_k, int32_t d_v, const void *q,
                          const void *k, const void *v, const float *g, const float *beta,
                          const float *state_in, float *state_out, void *o, int32_t o_dtype, float scale,
                          void *stream);

/* ------------------------------------------------------------------------
 * deltas_drift -- state drift per frame (Section 3.2, Eq. 3)
 * ------------------------------------------------------------------------
 * partials: fp32 [L][F][H_v][2] (num, den) as written by gdn_chunk_fwd for
 * L layers (layer l's F frames at offset l * F * H_v * 2).  Pairs written
 * per slice of the state (drift_per_slice = 1) are read as H_v * d_v / 16
 * heads: DS_DRIFT_LAYER_FROB is then the same score, while HEAD_MEAN and
 * PER_HEAD become per-slice ratios.
 *   DS_DRIFT_LAYER_FROB: scores[f] = mean_l sqrt(sum_h num / sum_h den)
 *   DS_DRIFT_HEAD_MEAN:  scores[f] = mean_{l,h} sqrt(num / den)
 *   DS_DRIFT_PER_HEAD:   scores[l][f][h] = sqrt(num / den)
 *   DS_WRITE_MEAN:       with write_partials (sum, count) in place of (num, den):
 *                        scores[f] = mean_{l,h} sum / count (0 where count = 0)
 * den = 0 gives +inf when num > 0 and 0 otherwise; a mean containing +inf
 * is +inf.  scores: fp32 [F] (or [L][F][H_v] for PER_HEAD).  partials must
 * be 8-byte aligned (each pair is read as one 8-byte word).
 */
ds_status deltas_drift(const float *partials, int32_t L, int32_t F, int32_t H_v, int32_t mode,
                       float *scores, void *stream);

/* ------------------------------------------------------------------------
 * deltas_drift_states -- drift sums from two copies of the state
 * ------------------------------------------------------------------------
 * The unfused form of the sums behind Eq. 3 (Section 3.2): the way the paper
 * measures the signal, by keeping a copy of every layer's state before a
 * frame and taking two norms after it.  For every (l, b, j):
 *     partials[l][b][j][0] = ||S_after - S_before||_F^2
 *     partials[l][b][j][1] = ||S_before||_F^2
 * S_before, S_after: fp32 [L][B][H_v][d_v][d_k], 16-byte aligned, d_v d_k a
 * multiple of 4.  partials: fp32 [L][B][H_v][2] (the layout deltas_drift
 * reads with F = B).  Each sum is accumulated in fp32 per thread and combined
 * in a fixed order in fp64.  Provided as the cost reference for the fused sums
 * of gdn_chunk_fwd.
 */
ds_status deltas_drift_states(const float *S_before, const float *S_after, int32_t L, int32_t B, int32_t H_v,
                              int32_t d_v, int32_t d_k, float *partials, void *stream);

/* ------------------------------------------------------------------------
 * kv_evict_topk -- one eviction step of Algorithm 1 (Section 3.3)
 * ------------------------------------------------------------------------
 * The cache holds `len` tokens (host-known) in slots [0, len) of every
 * layer; slot i carries its original position pos[i] and the index of the
 * chunk (frame) it arrived with, chunk_id[i].  A token's score is
 * chunk_scores[chunk_id[i]].  If len <= M the call does nothing and sets
 * *new_len = len.  Otherwise it keeps exactly M slots:
 *   - the first n_sink and the last n_window slots;
 *   - the candidates in between are split into N = max(n_buckets, 1) spans
 *     of chunk arrival time, span(a) = floor(N (a - a_min) / (a_max - a_min + 1));
 *     each span keeps its best floor((M - n_sink - n_window) / N)
 *     candidates, and the leftover slots go to the best candidates not yet
 *     kept.  "Best" orders by (score desc, chunk_id desc, pos desc): ties go
 *     to newer tokens.
 * The kept slots are compacted in place, in ascending slot order, in every
 * layer's K and V rows and in pos and chunk_id (positions are moved, never
 * rewritten).  Rows in [M, len) are unspecified afterwards.
 *
 * Layouts: k_layers / v_layers are HOST arrays of n_layers device pointers,
 * each to [capacity][row_bytes] bytes (row_bytes a multiple of 16);
 * pos, chunk_id: int32 [capacity]; chunk_scores fp32 [num_chunks], no NaN;
 * keep_out: int32 [M] (the kept slot indices) or NULL; new_len: host int32.
 * Cache invariants (as produced by appending chunks in arrival order and
 * compacting in order): chunk_id nondecreasing and pos strictly increasing
 * over [0, len), 0 <= chunk_id < num_chunks.  If the device finds them
 * broken it leaves the cache untouched; that and any other failure on the
 * device is recorded in the workspace's outcome word (ds_kv_device_status).
 * Requires 0 <= n_sink, 0 <= n_window, n_sink + n_window <= M, row_bytes <= 65536,
 * len <= capacity, n_buckets <= 64.
 */
typedef struct {
    int32_t n_layers;  /* full-attention layers sharing the ranking */
    int32_t row_bytes; /* bytes of one token's K (or V) row in one layer */
    int32_t capacity;  /* slots allocated per layer */
} ds_kv_shape;

size_t ds_kv_workspace_bytes(const ds_kv_shape *shape);

ds_status kv_evict_topk(const ds_kv_shape *shape, void *const *k_layers, void *const *v_layers,
                        int32_t *pos, int32_t *chunk_id, const float *chunk_scores,
                        int32_t num_chunks, int32_t len, int32_t M, int32_t n_sink,
                        int32_t n_window, int32_t n_buckets, int32_t *keep_out, int32_t *new_len,
                        void *workspace, size_t workspace_bytes, void *stream);

/* Device address of the int32 outcome word that kv_evict_topk and
 * kv_evict_topk_indexed leave in their workspace.  Every call that evicts
 * (len > M) overwrites it once its kernels have run:
 *   0  ok;
 *   1  the cache invariants were found broken: nothing was moved or rewritten;
 *   2  the kept count differed from M (an internal check): nothing was moved;
 *   3  kv_evict_topk only: a bounded wait of the in-place gather timed out;
 *      every move stopped at once, so K/V rows, pos and chunk_id in [0, M)
 *      are partially compacted and unspecified.
 * The calls return DS_OK before their kernels run, so a failure shows only
 * here: read the word after synchronising, or fold it into a device-side
 * maximum after each call to check many events with one read.  The two
 * int32 words after it are internal flags. */
int32_t *ds_kv_device_status(void *workspace);

/* ------------------------------------------------------------------------
 * kv_evict_topk_indexed -- the eviction step of Algorithm 1 (Section 3.3)
 * without moving K/V data
 * ------------------------------------------------------------------------
 * The cache is addressed through a slot table: logical token i (i < len, in
 * arrival order) lives in physical row slot[i] of every full-attention
 * layer's K and V; a consumer reads token i's rows at slot[i].  pos,
 * chunk_id and slot are indexed by logical token and carry the invariants
 * of kv_evict_topk (chunk_id nondecreasing, pos strictly increasing over
 * [0, len)); slot holds distinct rows in [0, capacity).
 * The kept set is exactly kv_evict_topk's (same arguments, same keep_out).
 * Only the three int32 arrays are compacted, in place and in ascending
 * logical order: slot'[d] = slot[keep[d]], pos'[d] = pos[keep[d]],
 * chunk_id'[d] = chunk_id[keep[d]] for d < M, so the logical order still
 * equals position order (positions are moved, never rewritten).  The
 * physical rows of the len - M evicted tokens are written to
 * free_out[0, len - M), in ascending logical order of the evicted tokens;
 * a caller appends its next tokens into those rows.  No K/V byte is read or
 * written.  Entries [M, len) of pos, chunk_id and slot are unspecified
 * afterwards.  If len <= M the call does nothing and sets *new_len = len.
 *
 * Layouts: pos, chunk_id, slot: int32 [capacity]; chunk_scores fp32
 * [num_chunks], no NaN; keep_out int32 [M] (logical indices kept) or NULL;
 * free_out int32 [len - M] (required); new_len: host int32.  The workspace
 * (ds_kv_indexed_workspace_bytes) holds the same status word as
 * kv_evict_topk's (ds_kv_device_status): if the device finds the invariants
 * broken it writes nothing else.
 * Requires 0 <= n_sink, 0 <= n_window, n_sink + n_window <= M,
 * len <= capacity, n_buckets <= 64.
 */
size_t ds_kv_indexed_workspace_bytes(int32_t capacity);

ds_status kv_evict_topk_indexed(int32_t capacity, int32_t *pos, int32_t *chunk_id, int32_t *slot,
                                const float *chunk_scores, int32_t num_chunks, int32_t len, int32_t M,
                                int32_t n_sink, int32_t n_window, int32_t n_buckets, int32_t *keep_out,
                                int32_t *free_out, int32_t *new_len, void *workspace,
                                size_t workspace_bytes, void *stream);

/* ------------------------------------------------------------------------
 * kv_append_indexed -- a chunk's K/V rows into the slot-indexed cache
 * ------------------------------------------------------------------------
 * The cache update of the streaming procedure (Section 3.3): before each
 * eviction step the new chunk's tokens join the cache.  With the cache
 * addressed through a slot table (kv_evict_topk_indexed), tokens
 * n .. n + T - 1 take the first T rows of the free list free_a[0, na)
 * followed by free_b[0, nb) (say, the rows the last eviction freed); for
 * t < T, with s_t that row:
 *     row s_t of plane p  =  new_rows[p][t]          (every plane)
 *     pos[n + t] = pos0 + t,  chunk_id[n + t] = chunk,  slot[n + t] = s_t,
 * and the remaining na + nb - T entries of the list go, in order, to
 * free_rest[0, na + nb - T).  One launch on `stream`; the caller keeps n and
 * the list lengths on the host.
 * Layouts: planes: n_planes device pointers, each [capacity][row_bytes]
 * (the K planes of the layers, then the V planes, as the caller likes);
 * new_rows: n_planes device pointers, each [T][row_bytes]; free_a, free_b,
 * free_rest: int32 (4-byte aligned; free_rest may not overlap the others);
 * pos, chunk_id, slot: int32 [capacity].
 * Requires 1 <= n_planes <= 64, row_bytes a multiple of 16, plane and row
 * pointers 16-byte aligned, T <= na + nb <= capacity and n + T <= capacity;
 * the call is rejected (nothing written) otherwise.  A free-list entry
 * outside [0, capacity) is skipped on the device (its token's rows and
 * table entries are not written).
 */
ds_status kv_append_indexed(void *const *planes, const void *const *new_rows, int32_t n_planes,
                            int32_t row_bytes, int32_t capacity, const int32_t *free_a, int32_t na,
                            const int32_t *free_b, int32_t nb, int32_t *free_rest, int32_t T, int32_t n,
                            int32_t pos0, int32_t chunk, int32_t *pos, int32_t *chunk_id, int32_t *slot,
                            void *stream);

/* ------------------------------------------------------------------------
 * kv_evict_topk_indexed_noalloc -- kv_evict_topk_indexed without a workspace
 * ------------------------------------------------------------------------
 * For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  The same
 * eviction step as kv_evict_topk_indexed (same arguments, same results, bit
 * for bit), with its scratch in a fixed device array of the library instead
 * of a workspace: 4 MiB per GPU, set up on the first call that evicts on that
 * GPU and held until the process ends.  The call allocates nothing and
 * calls no allocating routine.
 *   capacity  at most DS_KV_NOALLOC_MAX_CAPACITY slots; a larger capacity is
 *             rejected with DS_E_UNSUPPORTED before anything runs;
 *   outcome   device int32 [1] (4-byte aligned) or NULL: receives the
 *             outcome word of the call (0 ok, 1 cache invariants broken,
 *             2 keep count wrong; see ds_kv_device_status) when the call
 *             evicts.
 * Every call on one GPU shares that GPU's array: calls that overlap in time
 * on one GPU (two streams, two host threads) race and must be serialised by
 * the caller.  The array keeps the last call's contents; nothing in it has
 * to start at zero (each call writes every entry it reads).
 */
#define DS_KV_NOALLOC_MAX_CAPACITY 65536
ds_status kv_evict_topk_indexed_noalloc(int32_t capacity, int32_t *pos, int32_t *chunk_id, int32_t *slot,
                                        const float *chunk_scores, int32_t num_chunks, int32_t len, int32_t M,
                                        int32_t n_sink, int32_t n_window, int32_t n_buckets, int32_t *keep_out,
                                        int32_t *free_out, int32_t *outcome, int32_t *new_len, void *stream);

#ifdef __cplusplus
}
#endif
#endif /* DELTAS_H */
