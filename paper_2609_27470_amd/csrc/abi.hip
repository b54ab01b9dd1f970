// C ABI of libdeltas: argument validation, workspace sizing, launches.
// Every check runs on the host before the first launch; a rejected call
// writes nothing.  Nothing here throws or aborts.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include "deltas.h"
#include "kernels.h"

namespace {

thread_local char g_last_error[512] = "";

ds_status fail(ds_status s, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
    va_end(ap);
    return s;
}

ds_status hip_fail(hipError_t e, const char *where) {
    return fail(DS_E_HIP, "%s: %s", where, hipGetErrorString(e));
}

bool misaligned(const void *p) { return p && (((uintptr_t)p) & 15u) != 0; }

ds_status check_gdn_shape(const ds_gdn_shape *s) {
    if (!s) return fail(DS_E_NULL, "shape is NULL");
    if (s->B < 1 || s->T_total < 0 || s->H_k < 1 || s->H_v < 1 || s->n_frames < 0)
        return fail(DS_E_SHAPE, "bad sizes (B=%d T_total=%d H_k=%d H_v=%d n_frames=%d)", s->B, s->T_total,
                    s->H_k, s->H_v, s->n_frames);
    if (s->H_v % s->H_k != 0) return fail(DS_E_SHAPE, "H_v=%d is not a multiple of H_k=%d", s->H_v, s->H_k);
    if (s->d_k != s->d_v || (s->d_k != 64 && s->d_k != 128))
        return fail(DS_E_UNSUPPORTED, "head dims d_k=%d d_v=%d (supported: d_k = d_v in {64, 128})", s->d_k,
                    s->d_v);
    if (s->frame_len < 0 || s->frame_len % 64 != 0)
        return fail(DS_E_UNSUPPORTED, "frame_len=%d must be 0 or a multiple of 64", s->frame_len);
    if (s->drift_per_slice != 0 && s->drift_per_slice != 1)
        return fail(DS_E_ARG, "drift_per_slice=%d (0 or 1)", s->drift_per_slice);
    // keep every index of the kernels inside 32-bit ranges where they use them
    if ((long long)s->T_total * s->H_v > (1LL << 31) / 2 || (long long)s->B * s->H_v * (s->d_v / 16) > (1LL << 30))
        return fail(DS_E_UNSUPPORTED, "problem too large for one call");
    return DS_OK;
}

}  // namespace

extern "C" {

const char *ds_status_string(ds_status s) {
    switch (s) {
    case DS_OK: return "ok";
    case DS_E_NULL: return "required pointer is NULL";
    case DS_E_SHAPE: return "inconsistent sizes";
    case DS_E_DTYPE: return "unknown dtype";
    case DS_E_ALIGN: return "pointer not 16-byte aligned";
    case DS_E_UNSUPPORTED: return "unsupported configuration";
    case DS_E_ARG: return "invalid argument";
    case DS_E_HIP: return "HIP runtime error";
    case DS_E_WORKSPACE: return "workspace missing or too small";
    default: return "unknown status";
    }
}

const char *ds_last_error(void) { return g_last_error; }

size_t ds_gdn_workspace_bytes(const ds_gdn_shape *shape) {
    if (check_gdn_shape(shape) != DS_OK) return 0;
    return ds::gdn_workspace_layout(shape->B, shape->T_total, shape->H_k, shape->H_v, shape->d_v, shape->n_frames, false)
        .total;
}

size_t ds_gdn_write_workspace_bytes(const ds_gdn_shape *shape) {
    if (check_gdn_shape(shape) != DS_OK) return 0;
    return ds::gdn_workspace_layout(shape->B, shape->T_total, shape->H_k, shape->H_v, shape->d_v, shape->n_frames, true)
        .total;
}

ds_status gdn_chunk_fwd(const ds_gdn_shape *shape, const void *q, const void *k, const void *v, const float *g,
                        const float *beta, const int32_t *cu_seqlens, const float *state_in, float *state_out,
                        void *o, int32_t o_dtype, float scale, float *drift_partials, float *write_partials,
                        float *snapshots,
                        void *workspace, size_t workspace_bytes, void *stream) {
    g_last_error[0] = 0;
    ds_status st = check_gdn_shape(shape);
    if (st != DS_OK) return st;
    const ds_gdn_shape &s = *shape;
    if (s.T_total > 0 && (!q || !k || !v || !g || !beta || !o))
        return fail(DS_E_NULL, "q, k, v, g, beta and o are required");
    if (!state_out) return fail(DS_E_NULL, "state_out is required");
    if (s.B > 1 && !cu_seqlens) return fail(DS_E_NULL, "cu_seqlens is required when B > 1");
    if (o_dtype != DS_BF16 && o_dtype != DS_F32) return fail(DS_E_DTYPE, "o_dtype=%d", o_dtype);
    const void *ptrs[] = {q, k, v, g, beta, cu_seqlens, state_in, state_out, o, drift_partials, write_partials,
                          snapshots, workspace};
    for (const void *p : ptrs)
        if (misaligned(p)) return fail(DS_E_ALIGN, "a pointer is not 16-byte aligned");
    const ds::GdnWorkspace lay =
        ds::gdn_workspace_layout(s.B, s.T_total, s.H_k, s.H_v, s.d_v, s.n_frames, write_partials != nullptr);
    if (!workspace || workspace_bytes < lay.total)
        return fail(DS_E_WORKSPACE, "workspace needs %zu bytes, got %zu", lay.total, workspace_bytes);
    if (s.n_frames > 0 && s.frame_len == 0 && s.n_frames > s.B)
        return fail(DS_E_SHAPE, "n_frames=%d exceeds B=%d with frame_len=0", s.n_frames, s.B);
    if (s.frame_len > 0 && (long long)s.n_frames > (long long)s.T_total / s.frame_len + s.B)
        return fail(DS_E_SHAPE, "n_frames=%d is more than the streams can hold", s.n_frames);

    ds::GdnLaunch p;
    p.q = (const uint16_t *)q;
    p.k = (const uint16_t *)k;
    p.v = (const uint16_t *)v;
    p.g = g;
    p.beta = beta;
    p.cu_seqlens = cu_seqlens;
    p.B = s.B;
    p.T_total = s.T_total;
    p.H_k = s.H_k;
    p.H_v = s.H_v;
    p.d = s.d_k;
    p.frame_len = s.frame_len;
    p.n_frames = s.n_frames;
    p.state_in = state_in;
    p.state_out = state_out;
    p.o = o;
    p.o_bf16 = (o_dtype == DS_BF16);
    p.scale = scale;
    p.drift_partials = drift_partials;
    p.drift_slices = s.drift_per_slice;
    p.write_partials = write_partials;
    p.snapshots = snapshots;
    char *ws = (char *)workspace;
    p.wsT = (_Float16 *)(ws + lay.offT);
    p.wsP = (_Float16 *)(ws + lay.offP);
    p.wsQ = (_Float16 *)(ws + lay.offQ);
    p.wsGam = (float *)(ws + lay.offGam);
    p.wsDrift = (float *)(ws + lay.offDrift);
    p.wsCnt = (unsigned *)(ws + lay.offCnt);
    p.wsWrite = (float *)(ws + lay.offWrite);
    p.wsStart = (float *)(ws + lay.offStart);
    p.tiles_max = lay.tiles_max;
    p.n_split = lay.n_split;
    hipError_t e = ds::launch_gdn(p, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "gdn_chunk_fwd launch");
    return DS_OK;
}

ds_status deltas_drift(const float *partials, int32_t L, int32_t F, int32_t H_v, int32_t mode, float *scores,
                       void *stream) {
    g_last_error[0] = 0;
    if (L < 0 || F < 0 || H_v < 1) return fail(DS_E_SHAPE, "L=%d F=%d H_v=%d", L, F, H_v);
    if (mode < DS_DRIFT_LAYER_FROB || mode > DS_WRITE_MEAN) return fail(DS_E_ARG, "mode=%d", mode);
    if ((long long)L * F * H_v == 0) return DS_OK;
    if (!partials || !scores) return fail(DS_E_NULL, "partials and scores are required");
    if (((uintptr_t)partials) & 7u) return fail(DS_E_ALIGN, "partials must be 8-byte aligned");
    if ((long long)L * F * H_v * 2 > (1LL << 31)) return fail(DS_E_UNSUPPORTED, "too many partials");
    hipError_t e = ds::launch_drift(partials, L, F, H_v, mode, scores, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "deltas_drift launch");
    return DS_OK;
}

ds_status deltas_drift_states(const float *S_before, const float *S_after, int32_t L, int32_t B, int32_t H_v,
                              int32_t d_v, int32_t d_k, float *partials, void *stream) {
    g_last_error[0] = 0;
    if (L < 0 || B < 0 || H_v < 1 || d_v < 1 || d_k < 1)
        return fail(DS_E_SHAPE, "L=%d B=%d H_v=%d d_v=%d d_k=%d", L, B, H_v, d_v, d_k);
    if (((long long)d_v * d_k) % 4 != 0) return fail(DS_E_UNSUPPORTED, "d_v * d_k = %d is not a multiple of 4", d_v * d_k);
    const long long heads = (long long)L * B * H_v;
    if (heads == 0) return DS_OK;
    if (!S_before || !S_after || !partials) return fail(DS_E_NULL, "S_before, S_after and partials are required");
    if (heads > (1LL << 30) || (long long)d_v * d_k > (1LL << 30)) return fail(DS_E_UNSUPPORTED, "too many states");
    if (misaligned(S_before) || misaligned(S_after)) return fail(DS_E_ALIGN, "states must be 16-byte aligned");
    hipError_t e = ds::launch_drift_states(S_before, S_after, (int)heads, d_v * d_k, partials, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "deltas_drift_states launch");
    return DS_OK;
}

ds_status gdn_decode_step(int32_t B, int32_t H_k, int32_t H_v, int32_t d_k, int32_t d_v, const void *q,
                          const void *k, const void *v, const float *g, const float *beta, const float *state_in,
                          float *state_out, void *o, int32_t o_dtype, float scale, void *stream) {
    g_last_error[0] = 0;
    if (B < 0 || H_k < 1 || H_v < 1) return fail(DS_E_SHAPE, "B=%d H_k=%d H_v=%d", B, H_k, H_v);
    if (H_v % H_k != 0) return fail(DS_E_SHAPE, "H_v=%d is not a multiple of H_k=%d", H_v, H_k);
    if (d_k != d_v || (d_k != 64 && d_k != 128))
        return fail(DS_E_UNSUPPORTED, "head dims d_k=%d d_v=%d (supported: d_k = d_v in {64, 128})", d_k, d_v);
    if (o_dtype != DS_BF16 && o_dtype != DS_F32) return fail(DS_E_DTYPE, "o_dtype=%d", o_dtype);
    if ((long long)B * H_v * (d_v * d_k / 2048) > (1LL << 31) - 1) return fail(DS_E_UNSUPPORTED, "too many heads");
    if (B == 0) return DS_OK;
    if (!q || !k || !v || !g || !beta || !state_out || !o)
        return fail(DS_E_NULL, "q, k, v, g, beta, state_out and o are required");
    const void *ptrs[] = {q, k, v, state_in, state_out, o};
    for (const void *p : ptrs)
        if (misaligned(p)) return fail(DS_E_ALIGN, "a pointer is not 16-byte aligned");
    if (state_in && state_in != state_out) {
        const char *a0 = (const char *)state_in, *b0 = (const char *)state_out;
        const size_t n = (size_t)B * H_v * d_v * d_k * sizeof(float);
        if (a0 < b0 + n && b0 < a0 + n) return fail(DS_E_ARG, "state_in and state_out overlap without being equal");
    }
    ds::DecodeArgs a;
    a.q = (const uint16_t *)q;
    a.k = (const uint16_t *)k;
    a.v = (const uint16_t *)v;
    a.g = g;
    a.beta = beta;
    a.state_in = state_in;
    a.state_out = state_out;
    a.o = o;
    a.scale = scale;
    a.B = B;
    a.H_k = H_k;
    a.H_v = H_v;
    a.group = H_v / H_k;
    hipError_t e = ds::launch_gdn_decode(a, d_k, o_dtype == DS_BF16, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "gdn_decode_step launch");
    return DS_OK;
}

size_t ds_kv_workspace_bytes(const ds_kv_shape *shape) {
    if (!shape || shape->n_layers < 1 || shape->row_bytes < 16 || shape->row_bytes % 16 || shape->row_bytes > 65536 ||
        shape->capacity < 1 || 2 * shape->n_layers > ds::KV_MAX_PLANES)
        return 0;
    return ds::kv_workspace_layout(shape->n_layers, shape->row_bytes, shape->capacity).total;
}

int32_t *ds_kv_device_status(void *workspace) { return (int32_t *)workspace; }

ds_status kv_evict_topk(const ds_kv_shape *shape, void *const *k_layers, void *const *v_layers, int32_t *pos,
                        int32_t *chunk_id, const float *chunk_scores, int32_t num_chunks, int32_t len, int32_t M,
                        int32_t n_sink, int32_t n_window, int32_t n_buckets, int32_t *keep_out, int32_t *new_len,
                        void *workspace, size_t workspace_bytes, void *stream) {
    g_last_error[0] = 0;
    if (!shape || !new_len) return fail(DS_E_NULL, "shape and new_len are required");
    const ds_kv_shape &s = *shape;
    if (s.n_layers < 1 || 2 * s.n_layers > ds::KV_MAX_PLANES)
        return fail(DS_E_UNSUPPORTED, "n_layers=%d (1..%d)", s.n_layers, ds::KV_MAX_PLANES / 2);
    if (s.row_bytes < 16 || s.row_bytes % 16) return fail(DS_E_SHAPE, "row_bytes=%d must be a positive multiple of 16", s.row_bytes);
    if (s.row_bytes > 65536) return fail(DS_E_UNSUPPORTED, "row_bytes=%d (at most 65536)", s.row_bytes);
    if (s.capacity < 1) return fail(DS_E_SHAPE, "capacity=%d", s.capacity);
    if (len < 0 || len > s.capacity) return fail(DS_E_SHAPE, "len=%d outside [0, capacity=%d]", len, s.capacity);
    if (M < 0 || n_sink < 0 || n_window < 0 || (long long)n_sink + n_window > M)
        return fail(DS_E_ARG, "need 0 <= n_sink, 0 <= n_window, n_sink + n_window <= M (got %d, %d, %d)", n_sink,
                    n_window, M);
    if (n_buckets < 0 || n_buckets > 64) return fail(DS_E_ARG, "n_buckets=%d (0..64)", n_buckets);
    if (num_chunks < 1) return fail(DS_E_ARG, "num_chunks=%d", num_chunks);
    if ((long long)s.capacity * s.row_bytes > (1LL << 40) || 2LL * s.n_layers * s.row_bytes >= (1LL << 31))
        return fail(DS_E_UNSUPPORTED, "cache too large");
    if (len <= M) {
        *new_len = len;
        return DS_OK;
    }
    if (!k_layers || !v_layers || !pos || !chunk_id || !chunk_scores)
        return fail(DS_E_NULL, "cache pointers, pos, chunk_id and chunk_scores are required");
    ds::KvLaunch p;
    p.n_planes = 2 * s.n_layers;
    for (int l = 0; l < s.n_layers; ++l) {
        if (!k_layers[l] || !v_layers[l]) return fail(DS_E_NULL, "layer %d has a NULL K or V pointer", l);
        if (misaligned(k_layers[l]) || misaligned(v_layers[l]))
            return fail(DS_E_ALIGN, "layer %d K/V not 16-byte aligned", l);
        p.planes[l] = (char *)k_layers[l];
        p.planes[s.n_layers + l] = (char *)v_layers[l];
    }
    const void *ptrs[] = {pos, chunk_id, chunk_scores, keep_out, workspace};
    for (const void *q : ptrs)
        if (misaligned(q)) return fail(DS_E_ALIGN, "a pointer is not 16-byte aligned");
    const ds::KvWorkspace lay = ds::kv_workspace_layout(s.n_layers, s.row_bytes, s.capacity);
    if (!workspace || workspace_bytes < lay.total)
        return fail(DS_E_WORKSPACE, "workspace needs %zu bytes, got %zu", lay.total, workspace_bytes);
    p.row_bytes = s.row_bytes;
    p.capacity = s.capacity;
    p.pos = pos;
    p.chunk_id = chunk_id;
    p.chunk_scores = chunk_scores;
    p.num_chunks = num_chunks;
    p.len = len;
    p.M = M;
    p.n_sink = n_sink;
    p.n_window = n_window;
    p.n_buckets = n_buckets;
    p.keep_out = keep_out;
    p.slot = nullptr;
    p.free_out = nullptr;
    p.outcome_out = nullptr;
    p.ws = (char *)workspace;
    p.lay = lay;
    hipError_t e = ds::launch_kv_evict(p, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "kv_evict_topk launch");
    *new_len = M;
    return DS_OK;
}

ds_status kv_append_indexed(void *const *planes, const void *const *new_rows, int32_t n_planes,
                            int32_t row_bytes, int32_t capacity, const int32_t *free_a, int32_t na,
                            const int32_t *free_b, int32_t nb, int32_t *free_rest, int32_t T, int32_t n,
                            int32_t pos0, int32_t chunk, int32_t *pos, int32_t *chunk_id, int32_t *slot,
                            void *stream) {
    g_last_error[0] = 0;
    if (n_planes < 1 || n_planes > ds::KV_MAX_PLANES)
        return fail(DS_E_UNSUPPORTED, "n_planes=%d (1..%d)", n_planes, ds::KV_MAX_PLANES);
    if (row_bytes < 16 || row_bytes % 16) return fail(DS_E_SHAPE, "row_bytes=%d must be a positive multiple of 16", row_bytes);
    if (row_bytes > 65536) return fail(DS_E_UNSUPPORTED, "row_bytes=%d (at most 65536)", row_bytes);
    if (capacity < 1) return fail(DS_E_SHAPE, "capacity=%d", capacity);
    if (T < 0 || n < 0 || (long long)n + T > capacity)
        return fail(DS_E_SHAPE, "n=%d + T=%d outside [0, capacity=%d]", n, T, capacity);
    if (na < 0 || nb < 0 || (long long)na + nb < T)
        return fail(DS_E_ARG, "the free list (%d + %d rows) is shorter than T=%d", na, nb, T);
    if ((long long)na + nb > capacity) return fail(DS_E_ARG, "the free list (%d + %d rows) exceeds capacity", na, nb);
    if ((long long)capacity * row_bytes > (1LL << 40)) return fail(DS_E_UNSUPPORTED, "cache too large");
    if (T == 0 && na + nb == 0) return DS_OK;
    if (!planes || !new_rows || !pos || !chunk_id || !slot || (na > 0 && !free_a) || (nb > 0 && !free_b) ||
        (na + nb > T && !free_rest))
        return fail(DS_E_NULL, "planes, new_rows, pos, chunk_id, slot and the free lists are required");
    ds::KvAppendLaunch p;
    p.n_planes = n_planes;
    for (int i = 0; i < n_planes; ++i) {
        if (!planes[i] || !new_rows[i]) return fail(DS_E_NULL, "plane %d has a NULL pointer", i);
        if (misaligned(planes[i]) || misaligned(new_rows[i])) return fail(DS_E_ALIGN, "plane %d not 16-byte aligned", i);
        p.planes[i] = (char *)planes[i];
        p.new_rows[i] = (const char *)new_rows[i];
    }
    const void *ip[] = {free_a, free_b, free_rest, pos, chunk_id, slot};
    for (const void *q : ip)
        if (q && (((uintptr_t)q) & 3u)) return fail(DS_E_ALIGN, "an int32 pointer is not 4-byte aligned");
    p.row_bytes = row_bytes;
    p.capacity = capacity;
    p.free_a = free_a;
    p.free_b = free_b;
    p.na = na;
    p.nb = nb;
    p.free_rest = free_rest;
    p.T = T;
    p.n = n;
    p.pos0 = pos0;
    p.chunk = chunk;
    p.pos = pos;
    p.chunk_id = chunk_id;
    p.slot = slot;
    hipError_t e = ds::launch_kv_append(p, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "kv_append_indexed launch");
    return DS_OK;
}

size_t ds_kv_indexed_workspace_bytes(int32_t capacity) {
    if (capacity < 1) return 0;
    return ds::kv_workspace_layout(0, 16, capacity).total;
}

}  // extern "C"

namespace {

// Checks and launch shared by kv_evict_topk_indexed and its variant without a
// workspace: ws / ws_bytes is the scratch (caller's workspace or the
// library's own array), outcome a device copy of the outcome word or NULL.
ds_status evict_indexed(const char *who, int32_t capacity, int32_t *pos, int32_t *chunk_id, int32_t *slot,
                        const float *chunk_scores, int32_t num_chunks, int32_t len, int32_t M, int32_t n_sink,
                        int32_t n_window, int32_t n_buckets, int32_t *keep_out, int32_t *free_out, int32_t *outcome,
                        int32_t *new_len, char *ws, size_t ws_bytes, bool own_scratch, void *stream) {
    if (!new_len) return fail(DS_E_NULL, "new_len is required");
    if (capacity < 1) return fail(DS_E_SHAPE, "capacity=%d", capacity);
    if (own_scratch && capacity > ds::KV_NOALLOC_MAX_CAPACITY)
        return fail(DS_E_UNSUPPORTED, "capacity=%d exceeds the %d slots the library's fixed scratch holds", capacity,
                    ds::KV_NOALLOC_MAX_CAPACITY);
    if (len < 0 || len > capacity) return fail(DS_E_SHAPE, "len=%d outside [0, capacity=%d]", len, capacity);
    if (M < 0 || n_sink < 0 || n_window < 0 || (long long)n_sink + n_window > M)
        return fail(DS_E_ARG, "need 0 <= n_sink, 0 <= n_window, n_sink + n_window <= M (got %d, %d, %d)", n_sink,
                    n_window, M);
    if (n_buckets < 0 || n_buckets > 64) return fail(DS_E_ARG, "n_buckets=%d (0..64)", n_buckets);
    if (num_chunks < 1) return fail(DS_E_ARG, "num_chunks=%d", num_chunks);
    if (len <= M) {
        *new_len = len;
        return DS_OK;
    }
    if (!pos || !chunk_id || !slot || !chunk_scores || !free_out)
        return fail(DS_E_NULL, "pos, chunk_id, slot, chunk_scores and free_out are required");
    const void *ptrs[] = {pos, chunk_id, slot, chunk_scores, keep_out, free_out, ws};
    for (const void *q : ptrs)
        if (misaligned(q)) return fail(DS_E_ALIGN, "a pointer is not 16-byte aligned");
    if (outcome && (((uintptr_t)outcome) & 3u)) return fail(DS_E_ALIGN, "outcome is not 4-byte aligned");
    if (own_scratch) {  // every host check passed: the library's array on the current device
        hipError_t e = ds::kv_noalloc_scratch(&ws);
        if (e != hipSuccess) return hip_fail(e, "scratch address");
        ws_bytes = ds::KV_NOALLOC_SCRATCH_BYTES;
    }
    const ds::KvWorkspace lay = ds::kv_workspace_layout(0, 16, capacity);
    if (!ws || ws_bytes < lay.total)
        return fail(DS_E_WORKSPACE, "workspace needs %zu bytes, got %zu", lay.total, ws_bytes);
    ds::KvLaunch p{};
    p.n_planes = 0;
    p.row_bytes = 16;
    p.capacity = capacity;
    p.pos = pos;
    p.chunk_id = chunk_id;
    p.chunk_scores = chunk_scores;
    p.num_chunks = num_chunks;
    p.len = len;
    p.M = M;
    p.n_sink = n_sink;
    p.n_window = n_window;
    p.n_buckets = n_buckets;
    p.keep_out = keep_out;
    p.slot = slot;
    p.free_out = free_out;
    p.outcome_out = outcome;
    p.ws = ws;
    p.lay = lay;
    hipError_t e = ds::launch_kv_evict(p, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, who);
    *new_len = M;
    return DS_OK;
}

}  // namespace

extern "C" {

ds_status kv_evict_topk_indexed(int32_t capacity, int32_t *pos, int32_t *chunk_id, int32_t *slot,
                                const float *chunk_scores, int32_t num_chunks, int32_t len, int32_t M, int32_t n_sink,
                                int32_t n_window, int32_t n_buckets, int32_t *keep_out, int32_t *free_out,
                                int32_t *new_len, void *workspace, size_t workspace_bytes, void *stream) {
    g_last_error[0] = 0;
    return evict_indexed("kv_evict_topk_indexed launch", capacity, pos, chunk_id, slot, chunk_scores, num_chunks,
                         len, M, n_sink, n_window, n_buckets, keep_out, free_out, nullptr, new_len, (char *)workspace,
                         workspace_bytes, false, stream);
}

ds_status kv_evict_topk_indexed_noalloc(int32_t capacity, int32_t *pos, int32_t *chunk_id, int32_t *slot,
                                        const float *chunk_scores, int32_t num_chunks, int32_t len, int32_t M,
                                        int32_t n_sink, int32_t n_window, int32_t n_buckets, int32_t *keep_out,
                                        int32_t *free_out, int32_t *outcome, int32_t *new_len, void *stream) {
    g_last_error[0] = 0;
    return evict_indexed("kv_evict_topk_indexed_noalloc launch", capacity, pos, chunk_id, slot, chunk_scores,
                         num_chunks, len, M, n_sink, n_window, n_buckets, keep_out, free_out, outcome, new_len,
                         nullptr, 0, true, stream);
}

}  // extern "C"
