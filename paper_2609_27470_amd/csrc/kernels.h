// Internal launch interface between the C ABI (abi.hip) and the kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ds {

// ---------------------------------------------------------------- GDN forward
struct GdnLaunch {
    const uint16_t *q, *k, *v;
    const float *g, *beta;
    const int32_t *cu_seqlens;
    int B, T_total, H_k, H_v, d;  // d = d_k = d_v
    int frame_len, n_frames;
    const float *state_in;
    float *state_out;
    void *o;
    int o_bf16;
    float scale;
    float *drift_partials;  // [n_frames][H_v][2] (or [n_frames][H_v][n_split][2] with drift_slices) or null
    int drift_slices;       // drift pairs per 16-row slice of the state instead of per v-head
    float *write_partials;  // [n_frames][H_v][2] or null
    float *snapshots;       // [n_frames][H_v][d][d] or null
    // workspace pieces
    _Float16 *wsT;      // [tiles_max][H_v][6][64][8]  T diag(beta), fp16 A-fragments
    _Float16 *wsP;      // [tiles_max][H_v][6][64][8]  D (.) tril(Q K^T), fp16 A-fragments
    _Float16 *wsQ;      // [tiles_max][H_k][4][d/32][64][8] q in fp16, A-fragment order, for the per-slice kernel only
    float *wsGam;       // [tiles_max][H_v][2][64]   Gamma_r = exp(gamma_r), D_last,r = exp(gamma_last - gamma_r)
    float *wsDrift;     // [n_frames][H_v][n_split][2] (one pair per slice)
    float *wsWrite;     // [H_v][n_split][T_total] per-token ||E row||^2 over each slice's columns
    unsigned *wsCnt;    // [B][H_v] slices whose drift sums are written (drift reduction in the sequential kernel)
    float *wsStart;     // [B][H_v][d][d] frame-start state of the whole-head sequential kernel
    int tiles_max;
    int n_split;        // d_v slices of 16 per (stream, v-head)
};

// Workspace layout shared by the size query and the launcher.
struct GdnWorkspace {
    size_t offT, offP, offQ, offGam, offDrift, offWrite, offCnt, offStart, total;
    int tiles_max, n_split;
};
// with_write: also the per-token norm area of the write signal (write_partials != NULL)
GdnWorkspace gdn_workspace_layout(int B, int T_total, int H_k, int H_v, int d, int n_frames, bool with_write);
hipError_t launch_gdn(const GdnLaunch &p, hipStream_t stream);

// ---------------------------------------------------------------- decode step
struct DecodeArgs {
    const uint16_t *q, *k, *v;  // [B][H_k][d], [B][H_k][d], [B][H_v][d] bf16
    const float *g, *beta;      // [B][H_v]
    const float *state_in;      // [B][H_v][d][d] or null (zeros)
    float *state_out;           // [B][H_v][d][d] (may be state_in)
    void *o;                    // [B][H_v][d] bf16 or fp32
    float scale;
    int B, H_k, H_v, group;
};
hipError_t launch_gdn_decode(const DecodeArgs &a, int d, bool o_bf16, hipStream_t stream);

// ---------------------------------------------------------------- drift reduce
// n_heads heads of n_elem fp32 entries each (n_elem a multiple of 4)
hipError_t launch_drift_states(const float *before, const float *after, int n_heads, int n_elem, float *partials,
                               hipStream_t stream);
hipError_t launch_drift(const float *partials, int L, int F, int H_v, int mode, float *scores,
                        hipStream_t stream);

// ---------------------------------------------------------------- KV eviction
constexpr int KV_MAX_PLANES = 64;  // 2 * n_layers

struct KvWorkspace {
    size_t offStatus, offPlanes, offKeep, offInv, offThRun, offRunStart, offRunKey, offRunBkt, offRunTake,
        offRunFrom, offFlags, offStage, offStageMeta, total;
    int n_chunks;    // 64 KiB pieces of one token's rows over all layers
    int stage_rows;  // destinations per staged block
};
// n_layers = 0: the indexed variant's workspace (no gather flags)
KvWorkspace kv_workspace_layout(int n_layers, int row_bytes, int capacity);

struct KvLaunch {
    char *planes[KV_MAX_PLANES];  // K of layer 0..L-1, then V of layer 0..L-1
    int n_planes, row_bytes, capacity;
    int32_t *pos, *chunk_id;
    const float *chunk_scores;
    int num_chunks, len, M, n_sink, n_window, n_buckets;
    int32_t *keep_out;
    int32_t *slot, *free_out;  // indexed variant (slot != NULL): no K/V planes, no gather
    int32_t *outcome_out;      // indexed variant: device copy of the outcome word, or NULL
    char *ws;
    KvWorkspace lay;
};
hipError_t launch_kv_evict(const KvLaunch &p, hipStream_t stream);

// A chunk's rows into a slot-indexed cache (kv_append_indexed).
struct KvAppendLaunch {
    char *planes[KV_MAX_PLANES];          // [capacity][row_bytes] each
    const char *new_rows[KV_MAX_PLANES];  // [T][row_bytes] each
    int n_planes, row_bytes, capacity;
    const int32_t *free_a, *free_b;
    int na, nb;
    int32_t *free_rest;
    int T, n, pos0, chunk;
    int32_t *pos, *chunk_id, *slot;
};
hipError_t launch_kv_append(const KvAppendLaunch &p, hipStream_t stream);

// The library's own scratch for the indexed eviction without a workspace: a
// fixed device array per GPU (4 MiB) and the largest capacity whose layout
// fits in it.  kv_noalloc_scratch returns the array's address on the current
// device (looked up once per device).
constexpr size_t KV_NOALLOC_SCRATCH_BYTES = 4u << 20;
constexpr int KV_NOALLOC_MAX_CAPACITY = 65536;
hipError_t kv_noalloc_scratch(char **out);

}  // namespace ds
