// Device-side pieces shared by the GDN forward kernels (gdn_fwd.hip: the
// prep pass and the per-slice sequential kernel; gdn_wide.hip: the
// sequential kernel that owns whole heads): tile constants, the fragment
// layout of the prep pass's workspace, the kernel arguments and small helpers.
#pragma once
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace ds {

constexpr int TILE = 64;

// T diag(beta) and P are stored per (tile, v-head) as the six non-zero
// 16 x 32 A-fragments of v_mfma_f32_16x16x32_f16 (row block w = 0..3,
// k-step ks <= w / 2), 64 lanes x 8 halves each: lane l holds row
// 16 w + l % 16, and its half i the column kappa(ks, l / 16, i) =
// 32 ks + 16 (i / 4) + 4 (l / 16) + i % 4 -- the order in which the
// sequential kernel's B operands (tiles of R and E) hold the tokens.
constexpr int FRAG_HALVES = 64 * 8;
constexpr int TP_HALVES = 6 * FRAG_HALVES;
__host__ __device__ constexpr int frag_index(int w, int ks) { return w < 2 ? w : 2 + 2 * (w - 2) + ks; }

struct GdnArgs {
    const uint16_t *q, *k, *v;
    const float *g, *beta;
    Streams st;
    int H_k, H_v, group;
    int frame_len, n_frames;
    const float *state_in;
    float *state_out;
    void *o;
    float scale;
    float *snapshots;
    _Float16 *wsT, *wsP;
    _Float16 *wsQ;  // fp16 q fragments for the per-slice kernel (null for the whole-head kernel)
    float *wsGam, *wsDrift;
    float *wsWrite;  // per-token sums of squares of E over the slice's columns, or null
    float *wsStart;  // [B][H_v][d][d] state at the current frame's start (whole-head kernel)
    int n_split;
    // drift sums reduced inside the sequential kernel (null: a separate pass does it)
    float *drift_out;       // [n_frames][H_v][2]
    unsigned *drift_cnt;    // [B][H_v] slices done, zeroed by the prep kernel
    // drift pairs of frames past the real count, zeroed by the prep kernel
    float *drift_zero;      // the caller's drift_partials (either layout) or null
    int drift_zero_per_frame;  // pairs per frame in it: H_v, or H_v * n_split for per-slice pairs
    int prep_per_vhead;     // prep grid (tiles, H_v) instead of (tiles, H_k)
    // whole-head kernel: 0 one launch; 1, 2 the whole-head and the half-head
    // launch of a call split at a frame boundary (from which at most
    // wide_tail_streams streams have tiles left)
    int wide_phase, wide_tail_streams;
};

// Global tile index -> (stream, first token, valid tokens).  Tiles are
// numbered stream by stream; a stream of n tokens has ceil(n / 64) tiles.
__device__ bool locate_tile(const Streams &s, int ti, int &t0, int &n) {
    int base = 0;
    bool found = false;
    for_streams(s, [&](int, int st, int en) {
        const int nt = (en - st + TILE - 1) / TILE;
        if (ti < base + nt) {
            t0 = st + TILE * (ti - base);
            n = min(TILE, en - t0);
            found = true;
            return true;
        }
        base += nt;
        return false;
    });
    return found;
}

// Inclusive prefix sum over the 64 lanes of a wave on data-parallel
// primitives (no LDS round trip): Hillis-Steele inside each row of 16 lanes
// (row shifts by 1, 2, 4, 8, lanes shifted in from outside the row read 0),
// then the total of row 0 added to row 1 and of row 2 to row 3 (broadcast of
// lane 15 of the row before), then the total of rows 0 - 1 to rows 2 - 3
// (broadcast of lane 31).
template <int CTRL, int ROWS>
__device__ __forceinline__ float dpp_f32(float x) {  // lanes not written or shifted in from outside a row: 0
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, ROWS, 0xF, true));
}
__device__ __forceinline__ float wave_prefix_sum(float v) {
    v += dpp_f32<0x111, 0xF>(v);  // row_shr:1
    v += dpp_f32<0x112, 0xF>(v);  // row_shr:2
    v += dpp_f32<0x114, 0xF>(v);  // row_shr:4
    v += dpp_f32<0x118, 0xF>(v);  // row_shr:8
    v += dpp_f32<0x142, 0xA>(v);  // row_bcast:15 into rows 1 and 3
    v += dpp_f32<0x143, 0xC>(v);  // row_bcast:31 into rows 2 and 3
    return v;
}

__device__ __forceinline__ f32x4 mfma_f32_16x16x4(float a, float b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;

// L2 prefetch of 64 16-byte chunks (one per lane; 4 bytes of each are
// loaded).  The value is only handed to an empty asm statement two tiles
// later (see LoadSet::pf), so the load is kept and its wait comes late.
__device__ __forceinline__ uint32_t l2_prefetch(const void *chunk) { return *(const uint32_t *)chunk; }
__device__ __forceinline__ void l2_retire(uint32_t v) { asm volatile("" ::"v"(v)); }

// Transposed 16-bit fragment read: within each group of 16 lanes, lane l
// receives element (l % 4) of the 4 elements addressed by lane l/4 + 4 e.
__device__ __forceinline__ v4i16 ds_read_tr16(const void *p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16 *)p);
}
__device__ __forceinline__ u32x4 cat_u32x4(v4i16 a, v4i16 b) {
    return __builtin_bit_cast(u32x4, __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7));
}

// Workgroup barrier that orders LDS only.  The waves of both kernels exchange
// data through LDS alone, so their barriers need not wait for global loads in
// flight or for global stores to be acknowledged (a full __syncthreads waits
// for both, which drains every prefetch and costs a round trip to memory per
// barrier after a store).
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// K tile staged row-major in LDS (D bf16 per row) with the 16-byte chunks of
// a row permuted by an XOR with swz(row).  A bank group (4 banks, one chunk)
// is the chunk index mod 8, and a row starts on bank 0 (D = 64, 128), so:
// 8 consecutive rows read at one logical chunk (16-byte row reads, 8 lanes a
// cycle) see swz = a permutation of 0..7 and hit 8 distinct groups; the row
// writes cover a row's chunks; and a transposing read (4 rows 4 q .. 4 q + 3
// x 4 chunks 4 c .. 4 c + 3, 16 lanes of 8 bytes) sees swz in {0, 4, 1, 5} or
// {2, 6, 3, 7} and so touches each bank group twice, the least 16 such reads
// of one half-chunk can.
template <int D>
__device__ __forceinline__ int swz(int row) {
    static_assert(D == 64 || D == 128, "head dim");
    return ((row & 1) << 2) | ((row >> 1) & 3);
}

// Four consecutive fp32 output values of one lane to o at byte offset off of
// the buffer resource rs (one 16-byte store).
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ void store_o4_f32(const f32x4 &v, __amdgpu_buffer_rsrc_t rs, uint32_t off) {
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), rs, off, 0, 0);
}

// Two C blocks -> one fp16 operand (8 values per lane).
__device__ __forceinline__ half8 to_half8(const f32x4 &a, const f32x4 &b) {
    half8 r;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        r[e] = (_Float16)a[e];
        r[4 + e] = (_Float16)b[e];
    }
    return r;
}

// Slice drift pairs cross workgroups (and XCDs) through agent-scope atomic
// accesses, which the compiler emits as stores written through to, and loads
// served from, the GPU-wide point of coherence.  The handoff below then needs
// no agent-scope fence: such a fence writes back (release) or invalidates
// (acquire) a whole XCD's L2, and at the end of every workgroup of a short
// call that cost 18 % of a 1024-token layer call.  Ordering comes from the
// store acknowledgements: a writer's pairs are complete before its count
// increment is issued, and the last workgroup issues its loads only after
// its own increment has returned.
__device__ __forceinline__ void store_pair_coherent(float *p, float a, float b) {
    const unsigned long long bits =
        (unsigned long long)__float_as_uint(a) | ((unsigned long long)__float_as_uint(b) << 32);
    __hip_atomic_store((unsigned long long *)p, bits, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 load_pair_coherent(const float *p) {
    const unsigned long long bits =
        __hip_atomic_load((const unsigned long long *)p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return float2{__uint_as_float((unsigned)bits), __uint_as_float((unsigned)(bits >> 32))};
}
// Wait until every vector memory operation of this wave has completed (its
// stores acknowledged), with the compiler kept from moving memory accesses
// across the wait.
__device__ __forceinline__ void wait_vmem_all() {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0), expcnt and lgkmcnt not waited for
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// Sum of squares over the 16 columns of an E k-step held as a B operand (lane
// (ln, lg) element i is token kappa(ks, lg, i), column ln), reduced over the
// 16 lanes of each row by a transposing butterfly: afterwards lane ln holds
// the sum of element ln / 2 (lanes ln and ln ^ 1 agree).
__device__ __forceinline__ float row_sq_sum16(half8 ef, int ln) {
    float x[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = (float)ef[i] * (float)ef[i];
    const bool b3 = (ln >> 3) & 1, b2 = (ln >> 2) & 1, b1 = (ln >> 1) & 1;
    float y[4], z[2];
#pragma unroll
    for (int q = 0; q < 4; ++q) {  // partner ln ^ 8 (rotate the row of 16 by 8)
        const float send = b3 ? x[q] : x[4 + q];
        const float recv = __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, send), 0x128,
                                                                                  0xF, 0xF, false));
        y[q] = (b3 ? x[4 + q] : x[q]) + recv;
    }
#pragma unroll
    for (int q = 0; q < 2; ++q) {  // partner ln ^ 4 (swizzle with xor mask 4)
        const float send = b2 ? y[q] : y[2 + q];
        const float recv = __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, send), 0x101F));
        z[q] = (b2 ? y[2 + q] : y[q]) + recv;
    }
    // partner ln ^ 2, then ln ^ 1 (quad permutations)
    const float send = b1 ? z[0] : z[1];
    const float recv =
        __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, send), 0x4E, 0xF, 0xF, false));
    float w = (b1 ? z[1] : z[0]) + recv;
    w += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, w), 0xB1, 0xF, 0xF, false));
    return w;
}

// Sequential kernel owning all d_v rows of a (stream, v-head) per workgroup
// (gdn_wide.hip); returns the launch error.
hipError_t launch_gdn_wide(const GdnArgs &a, int n_heads, int tail_streams, bool o_bf16, bool drift,
                           hipStream_t stream);

}  // namespace ds
