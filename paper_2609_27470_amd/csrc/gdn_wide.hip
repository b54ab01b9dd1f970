// Sequential part of the chunkwise gated-delta-rule forward (Section 3.2,
// Eq. 2) with one workgroup per (stream, v-head): all 128 rows of the state
// of a head live in one workgroup.
//
// The per-slice kernel (gdn_fwd.hip) splits a head over 8 workgroups of 16
// state rows so that a single stream fills the GPU, but each of them pulls
// the whole tile (K, q, T diag(beta), P: about 46 KiB) from L2 for its 16
// rows.  With B * H_v heads enough to fill the GPU (several streams, the
// varlen batch), this kernel loads each tile once per head:
//   waves 0-3 (compute): wave w carries rows 32 w .. 32 w + 31 of S (two
//       16-row slices) in fp32 registers and does the whole tile for them:
//       K S0^T and S0 Q^T against the fp16 copy of its own rows (no exchange
//       between waves), R = V - diag(Gamma) K S0^T, E = T diag(beta) R,
//       O^T = scale diag(Gamma) S0 Q^T + (P E)^T (P carries the scale), and
//       the update S = Gamma_last S0 + (D_last E)^T K.  Every fragment read
//       from LDS (rows of K, Q, T, P, K^T) feeds both slices.
//   waves 4-7 (loaders): load the tile two tiles ahead and stage it in LDS
//       one tile ahead (K and q rows converted to fp16, the T fragments of the
//       prep pass, v rows, gamma in base 2 and D_last); form P = scale D (.)
//       tril(Q K^T) of the staged tile from its K and q on fp16 matrix cores,
//       so that the prep pass reads no q and writes no P; and store the
//       previous tile's bf16 o, which the compute waves left in LDS, as whole
//       rows.  Loader 3 also adds the frame-end drift sums of the 8 slices
//       (fixed order) and writes them, per slice or per head, with no exchange
//       between workgroups.
// Two barriers per tile (LDS-only): the tile's start, and one after the first
// two products, before which the loaders stage the next tile's rows (P is
// formed from them during the rest of the tile).  The state at a frame's
// start, needed for ||S_end - S_start||^2, is kept in a scratch area of the
// workspace (64 KiB per head) rather than in registers, and read back at the
// frame's end.
//
// A call of streams of unequal length leaves most CUs idle once the shorter
// streams end, and the per-tile time of the heads still running is then set
// by one workgroup's chain.  When its frames are whole tiles, the call runs as
// two launches: whole heads up to the cut (the first frame boundary from
// which at most as many streams are left as fill the GPU with two
// workgroups per head), then half heads (NSL = 1: 64 rows per workgroup, one
// 16-row slice per compute wave) from the states the first launch wrote.  A
// half head's drift sums go out per slice; with per-head pairs the second of
// a head's two workgroups to finish adds the 8 slices in order.
#include <type_traits>

#include "gdn_common.h"

namespace ds {

constexpr int WIDE_VLD = 128 + 16;  // halves per LDS row of the v tile (288 B: the 4 rows of a transposing
                                    // read start 8 banks apart, so its 16 lanes cover all 32 banks)

// A bf16 o tile is staged in the v buffer of its tile once the v rows are
// consumed: a compute wave writes the output dims of its own state rows (32 of
// a whole head, 16 of a half head) for every token, exactly the band of
// columns of v that it alone read, so no wave overwrites
// v that another still reads.  Inside the band the 8-byte pieces (4 dims) are
// permuted by an XOR with (row / 4) % 4, so that the 16 rows of one 8-byte
// write hit distinct banks.  Returns the halves offset of dims d .. d + 3
// (d % 4 == 0) of token row r.
__device__ __forceinline__ int o_stage_at(int r, int d) {
    return r * WIDE_VLD + 32 * (d >> 5) + 4 * (((d >> 2) & 7) ^ ((r >> 2) & 3));
}

// instruction classes of __builtin_amdgcn_sched_group_barrier
constexpr int SG_VALU = 0x2, SG_MFMA = 0x8, SG_DSR = 0x100;
#define WIDE_SG(mask, n) __builtin_amdgcn_sched_group_barrier((mask), (n), 0)

struct WideShared {
    uint16_t K[2][64 * 128];  // K tile (fp16), row-major, 16-byte chunks XOR-swizzled by row (swz)
    uint16_t Q[2][64 * 128];  // q tile (fp16), laid out like K
    u32x4 T[2][6][64];        // T diag(beta) A-fragments
    u32x4 P[2][6][64];        // P A-fragments
    uint16_t V[2][64 * WIDE_VLD];  // v rows (bf16)
    float G[2][2][64];        // Gamma_r, D_last,r
    float Gs[2][64];          // gamma_r in base-2 units (the gates of P)
    float2 DR[2][4][2][64];   // frame-end drift sums per [frame % 2][compute wave][slice][lane]
};

// One loader's share of a tile: K, q and v rows 16 X .. 16 X + 15, T
// fragments {2 X, 2 X + 1} (X < 2) or {4 + X - 2}; loader 0 also gamma (base
// 2), loader 1 D_last.
struct WideLoad {
    u32x4 k[4], q[4], v[4], t[2];
    float g;
};

// The tile index from which at most a.wide_tail_streams streams have tiles
// left, rounded up to a frame boundary (every workgroup computes the same
// value from the device lengths): the cut between the whole-head launch
// and the half-head launch of a split call.
__device__ int wide_cut(const GdnArgs &a) {
    constexpr int MAXS = 16;
    int top[MAXS + 1];  // the largest tile counts, descending
    const int S = min(a.wide_tail_streams, MAXS);
    for (int i = 0; i <= S; ++i) top[i] = 0;
    for_streams(a.st, [&](int, int s0, int e0) {
        int v = (e0 - s0 + TILE - 1) / TILE;
        for (int i = 0; i <= S; ++i) {  // insert, keeping the S + 1 largest
            if (v > top[i]) {
                const int t = top[i];
                top[i] = v;
                v = t;
            }
        }
        return false;
    });
    const int ft = a.frame_len / TILE;
    return (top[S] + ft - 1) / ft * ft;
}

// NSL = 2: one workgroup per (stream, v-head), compute wave w carrying rows
// 32 w .. 32 w + 31; NSL = 1: two workgroups per (stream, v-head), each with
// 64 rows (compute wave w: rows 64 h + 16 w .. + 15), for the tail of a split
// call, where few streams are left and half heads put more CUs to work.
template <bool OUT_BF16, bool DRIFT, int NSL>
__global__ __launch_bounds__(512, 1) void gdn_wide_kernel(GdnArgs a) {
    constexpr int D = 128, KS = D / 32, NKB = D / 16;
    constexpr int HW = 2 / NSL;  // workgroups per head
    __shared__ __align__(16) WideShared sh;
    const int tid = threadIdx.x, lane = tid & 63, ln = lane & 15, lg = lane >> 4;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);

    // ---- workgroup -> (stream, v-head, half); the workgroups of one qk-head of
    // one stream sit on one XCD (dispatch deals workgroups to the 8 XCDs in
    // turn), so its K and q tiles are fetched into that XCD's L2 once
    const int n_groups = a.st.B * a.H_k;
    const int gsz = a.group * HW;
    const int bid = blockIdx.x;
    int gidx, mem;
    if (n_groups % 8 == 0) {
        const int xcd = bid & 7, slot = bid >> 3;
        gidx = xcd + 8 * (slot / gsz);
        mem = slot % gsz;
    } else {
        gidx = bid / gsz;
        mem = bid % gsz;
    }
    const int b = gidx / a.H_k, qh = gidx % a.H_k;
    const int j = qh * a.group + mem / HW;
    const int r0 = 64 * (mem % HW);  // first state row of this workgroup
    const int sl0 = r0 / 16;          // its first 16-row slice

    int st = 0, en = 0, tile_base = 0, frame_base = 0;
    for_streams(a.st, [&](int bb, int s0, int e0) {
        if (bb == b) {
            st = s0;
            en = e0;
            return true;
        }
        tile_base += (e0 - s0 + TILE - 1) / TILE;
        frame_base += frames_in(e0 - s0, a.frame_len);
        return false;
    });
    const int len = en - st;
    const int n_tiles = (len + TILE - 1) / TILE;
    // the tiles of this launch: all of them, or those before (wide_phase 1) or
    // from (wide_phase 2) the cut, a frame boundary
    int lt0 = 0, lt1 = n_tiles;
    if (a.wide_phase != 0) {
        const int c = wide_cut(a);
        if (a.wide_phase == 1)
            lt1 = min(n_tiles, c);
        else
            lt0 = min(n_tiles, c);
    }
    const int nt = lt1 - lt0;
    if (a.wide_phase == 2 && nt == 0) return;  // the stream ended in the first launch
    const int tok0 = TILE * lt0;

    if (w < 4) {
        // ============================================================ compute
        // S^T block kb of slice sl, lane (ln, lg), element e =
        //   S[r0 + 16 NSL w + 16 sl + ln][sigma(kb, 4 lg + e)]
        const int wr0 = r0 + 16 * NSL * w;  // the wave's first row
        const size_t hbase = ((size_t)b * a.H_v + j) * D * D;
        // 16-byte pieces of the head's state rows go through buffer resources
        // (a uniform base in scalar registers, 32-bit lane offsets): S[sl][kb]
        // holds 4 consecutive columns of row wr0 + 16 sl + ln
        // byte offset of S[sl][kb]'s 4 columns = a per-lane base + a constant (passed
        // as the scalar offset, so that no per-(sl, kb) offset register stays live)
        const uint32_t lane_row = (uint32_t)((wr0 + ln) * D + 8 * lg) * 4u;
        auto sconst = [&](int sl, int kb) { return (int)((16 * sl * D + 32 * (kb >> 1) + 4 * (kb & 1)) * 4); };
        constexpr int RSRC_FLAGS = 0x00020000;
        f32x4 S[NSL][NKB];
        if (a.state_in) {
            const __amdgpu_buffer_rsrc_t rin =
                __builtin_amdgcn_make_buffer_rsrc((void *)(a.state_in + hbase), (short)0, D * D * 4, RSRC_FLAGS);
#pragma unroll
            for (int sl = 0; sl < NSL; ++sl)
#pragma unroll
                for (int kb = 0; kb < NKB; ++kb)
                    S[sl][kb] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rin, lane_row, sconst(sl, kb), 0));
        } else {
#pragma unroll
            for (int sl = 0; sl < NSL; ++sl)
#pragma unroll
                for (int kb = 0; kb < NKB; ++kb) S[sl][kb] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
        // the state at the start of the current frame, in this wave's own
        // register order (16-byte pieces, lane-contiguous)
        const __amdgpu_buffer_rsrc_t rstart = __builtin_amdgcn_make_buffer_rsrc(
            (void *)(a.wsStart + (((size_t)b * a.H_v + j) * 8 + wr0 / 16) * NKB * 64 * 4), (short)0, NSL * NKB * 64 * 16,
            RSRC_FLAGS);
        const uint32_t lane16 = (uint32_t)lane * 16u;
        auto start_const = [&](int sl, int kb) { return (sl * NKB + kb) * 64 * 16; };
        auto save_start = [&]() __attribute__((always_inline)) {
#pragma unroll
            for (int sl = 0; sl < NSL; ++sl)
#pragma unroll
                for (int kb = 0; kb < NKB; ++kb)
                    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, S[sl][kb]), rstart, lane16, start_const(sl, kb), 0);
        };
        if (DRIFT) save_start();
        int frame = frame_base + (a.frame_len > 0 ? tok0 / a.frame_len : 0);
        int frame_end = a.frame_len > 0 ? min(tok0 + a.frame_len, len) : len;  // tokens done at the next frame end

        // The tile runs as software-pipelined regions: every LDS operand is read
        // one step before its products, and scheduling groups interleave the
        // matrix-core products with the vector work that does not depend on them
        // (a compute wave is alone on its SIMD apart from a loader, so its own
        // instruction order has to hide the latencies).
        auto tile = [&](int lt, auto bufc) __attribute__((always_inline)) {
            constexpr int buf = decltype(bufc)::value;  // == (lt - lt0) % 2
            const int t0 = st + TILE * lt, n = min(TILE, en - t0);
            lds_barrier();
            const float gl = sh.G[buf][0][63];

            auto kread = [&](int ks, half8(&ka)[4]) __attribute__((always_inline)) {
#pragma unroll
                for (int rb = 0; rb < 4; ++rb) {
                    const int row = 16 * rb + ln;
                    ka[rb] = as_half8(*(const u32x4 *)(&sh.K[buf][row * D + 8 * ((4 * ks + lg) ^ swz<D>(row))]));
                }
            };
            auto qread = [&](int ks, half8(&qa)[4]) __attribute__((always_inline)) {
#pragma unroll
                for (int rb = 0; rb < 4; ++rb) {
                    const int row = 16 * rb + ln;
                    qa[rb] = as_half8(*(const u32x4 *)(&sh.Q[buf][row * D + 8 * ((4 * ks + lg) ^ swz<D>(row))]));
                }
            };
            // K^T fragments of state block kb by transposing reads (each used by both
            // slices): source lane (ln, lg) addresses token 32 ks + 16 r + 4 lg + ln / 4
            // and dims 32 (kb / 2) + 8 (ln % 4) + 4 (kb % 2) .. + 3
            auto ktread = [&](int kb, half8(&kt)[2]) __attribute__((always_inline)) {
#pragma unroll
                for (int ks = 0; ks < 2; ++ks) {
                    const int r0 = 32 * ks + 4 * lg + (ln >> 2), r1 = r0 + 16;
                    const int ch = 4 * (kb >> 1) + (ln & 3), hf = 4 * (kb & 1);
                    kt[ks] = __builtin_bit_cast(half8, cat_u32x4(ds_read_tr16(&sh.K[buf][r0 * D + 8 * (ch ^ swz<D>(r0)) + hf]),
                                                                 ds_read_tr16(&sh.K[buf][r1 * D + 8 * (ch ^ swz<D>(r1)) + hf])));
                }
            };

            // ---- (1) K S0^T (token rows 16 rb + 4 lg + e, state row wr0 + 16 sl + ln)
            // from the fp16 copy of S0 (k-step ks pairs state blocks 2 ks, 2 ks + 1).
            // Under it: the fp16 copy of the next k-step, and S <- Gamma_last S in place
            // for the blocks already copied (from here on the fp32 S is only the
            // update's accumulator).
            half8 s16[NSL][KS];
            f32x4 ks0[4][NSL];
            half8 ka[2][4];
#pragma unroll
            for (int rb = 0; rb < 4; ++rb)
#pragma unroll
                for (int sl = 0; sl < NSL; ++sl) ks0[rb][sl] = f32x4{0.f, 0.f, 0.f, 0.f};
            kread(0, ka[0]);
#pragma unroll
            for (int sl = 0; sl < NSL; ++sl) s16[sl][0] = to_half8(S[sl][0], S[sl][1]);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                if (ks + 1 < KS) {
                    kread(ks + 1, ka[(ks + 1) & 1]);
#pragma unroll
                    for (int sl = 0; sl < NSL; ++sl) s16[sl][ks + 1] = to_half8(S[sl][2 * ks + 2], S[sl][2 * ks + 3]);
                }
#pragma unroll
                for (int rb = 0; rb < 4; ++rb)
#pragma unroll
                    for (int sl = 0; sl < NSL; ++sl) ks0[rb][sl] = mfma_f16(ka[ks & 1][rb], s16[sl][ks], ks0[rb][sl]);
#pragma unroll
                for (int sl = 0; sl < NSL; ++sl)
#pragma unroll
                    for (int c = 0; c < 2; ++c)
#pragma unroll
                        for (int e = 0; e < 4; ++e) S[sl][2 * ks + c][e] *= gl;
                if (ks + 1 < KS) WIDE_SG(SG_DSR, 4);
#pragma unroll
                for (int i = 0; i < 4 * NSL; ++i) {
                    WIDE_SG(SG_MFMA, 1);
                    WIDE_SG(SG_VALU, 3);
                }
            }
            // operands of (2): q of the first k-step, Gamma, and v (transposed) of
            // the first quarter of R
            half8 qa[2][4];
            v4i16 vv[2][2];
            float4 g4[4];
            // v[16 rb + 4 lg + e][wr0 + 16 sl + ln], rb = 2 pr + h, for quarter (sl, pr)
            auto vread = [&](int sl, int pr, v4i16(&vq)[2]) __attribute__((always_inline)) {
#pragma unroll
                for (int h = 0; h < 2; ++h)
                    vq[h] = ds_read_tr16(&sh.V[buf][(16 * (2 * pr + h) + 4 * lg + (ln >> 2)) * WIDE_VLD + wr0 + 16 * sl + 4 * (ln & 3)]);
            };
            qread(0, qa[0]);
#pragma unroll
            for (int rb = 0; rb < 4; ++rb) g4[rb] = *(const float4 *)(&sh.G[buf][0][16 * rb + 4 * lg]);
            vread(0, 0, vv[0]);
            __builtin_amdgcn_sched_barrier(0);

            // ---- (2) O^T = S0 Q^T, S0 as the A operand and q as the B operand: lane
            // (ln, lg) holds state rows wr0 + 16 sl + 4 lg + e of token 16 rb + ln.
            // Under it, a quarter of R = V - diag(Gamma) K S0^T in each of the first
            // 2 NSL k-steps (slice ks / 2, row blocks 2 (ks % 2), 2 (ks % 2) + 1),
            // straight to fp16.
            constexpr int NQ = 2 * NSL;  // quarters of R
            f32x4 oacc[4][NSL];
            half8 rf[NSL][2];
#pragma unroll
            for (int rb = 0; rb < 4; ++rb)
#pragma unroll
                for (int sl = 0; sl < NSL; ++sl) oacc[rb][sl] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                if (ks + 1 < KS) qread(ks + 1, qa[(ks + 1) & 1]);
                if (ks + 1 < NQ) vread((ks + 1) >> 1, (ks + 1) & 1, vv[(ks + 1) & 1]);
#pragma unroll
                for (int rb = 0; rb < 4; ++rb)
#pragma unroll
                    for (int sl = 0; sl < NSL; ++sl) oacc[rb][sl] = mfma_f16(s16[sl][ks], qa[ks & 1][rb], oacc[rb][sl]);
                if (ks < NQ) {
                    const int sl = ks >> 1, pr = ks & 1;
                    f32x4 R[2];
#pragma unroll
                    for (int h = 0; h < 2; ++h) {
                        const int rb = 2 * pr + h;
                        const v4i16 v = vv[ks & 1][h];
                        R[h][0] = bf16_to_f32((uint16_t)v[0]) - g4[rb].x * ks0[rb][sl][0];
                        R[h][1] = bf16_to_f32((uint16_t)v[1]) - g4[rb].y * ks0[rb][sl][1];
                        R[h][2] = bf16_to_f32((uint16_t)v[2]) - g4[rb].z * ks0[rb][sl][2];
                        R[h][3] = bf16_to_f32((uint16_t)v[3]) - g4[rb].w * ks0[rb][sl][3];
                    }
                    rf[sl][pr] = to_half8(R[0], R[1]);
                }
                // (scheduling-group arguments have to be literal constants)
                if (ks + 1 < NQ) {
                    WIDE_SG(SG_DSR, 6);
                } else if (ks + 1 < KS) {
                    WIDE_SG(SG_DSR, 4);
                }
#pragma unroll
                for (int i = 0; i < 4 * NSL; ++i) {
                    WIDE_SG(SG_MFMA, 1);
                    if (ks < NQ) {
                        WIDE_SG(SG_VALU, 3);
                    } else {
                        WIDE_SG(SG_VALU, 1);
                    }
                }
            }
            // second barrier: the loaders have staged the next tile and form its P
            // from it during (3) - (5) (P of the first tile is in LDS from here on)
            lds_barrier();
            // operands of (3) - (5): T diag(beta) and P fragments, D_last, the
            // scale Gamma of each token, the first K^T fragments
            half8 tf[6], pf[6], kt[2][2];
            float4 d4[4];
            float gs[4];
#pragma unroll
            for (int f = 0; f < 6; ++f) tf[f] = as_half8(sh.T[buf][f][lane]);
#pragma unroll
            for (int rb = 0; rb < 4; ++rb) {
                d4[rb] = *(const float4 *)(&sh.G[buf][1][16 * rb + 4 * lg]);
                gs[rb] = a.scale * sh.G[buf][0][16 * rb + ln];
            }
#pragma unroll
            for (int f = 0; f < 6; ++f) pf[f] = as_half8(sh.P[buf][f][lane]);
            ktread(0, kt[0]);
            __builtin_amdgcn_sched_barrier(0);

            // ---- (3) E = T diag(beta) R and D_last E (fp16 B operands) per slice,
            // under them the scale Gamma of each token on (2)
            half8 e16[NSL][2], d16[NSL][2];
#pragma unroll
            for (int sl = 0; sl < NSL; ++sl) {
                f32x4 E[4];
#pragma unroll
                for (int rb = 0; rb < 4; ++rb) E[rb] = mfma_f16(tf[frag_index(rb, 0)], rf[sl][0], f32x4{0.f, 0.f, 0.f, 0.f});
#pragma unroll
                for (int rb = 2; rb < 4; ++rb) E[rb] = mfma_f16(tf[frag_index(rb, 1)], rf[sl][1], E[rb]);
#pragma unroll
                for (int rb = 0; rb < 4; ++rb)
#pragma unroll
                    for (int e = 0; e < 4; ++e) oacc[rb][sl][e] *= gs[rb];
                e16[sl][0] = to_half8(E[0], E[1]);
                e16[sl][1] = to_half8(E[2], E[3]);
#pragma unroll
                for (int rb = 0; rb < 4; ++rb) {
                    E[rb][0] *= d4[rb].x;
                    E[rb][1] *= d4[rb].y;
                    E[rb][2] *= d4[rb].z;
                    E[rb][3] *= d4[rb].w;
                }
                d16[sl][0] = to_half8(E[0], E[1]);
                d16[sl][1] = to_half8(E[2], E[3]);
            }
#pragma unroll
            for (int i = 0; i < 6 * NSL; ++i) {
                WIDE_SG(SG_MFMA, 1);
                WIDE_SG(SG_VALU, 4);
            }
            __builtin_amdgcn_sched_barrier(0);

            // ---- (4) + (5): O^T += (P E)^T = E^T P^T (E's B operand read as the A
            // operand, P's A fragments as B operands; P carries the scale),
            // interleaved with the update S = Gamma_last S0 + (D_last E)^T K.  A bf16
            // o goes to LDS, four consecutive dims per lane (the loaders store it a
            // tile later as whole rows: global stores from these waves would queue
            // behind the loaders' tile loads in the CU's vector-memory path); an fp32
            // o is stored at once through a buffer resource covering the tile's n
            // valid rows.
            constexpr int ES = OUT_BF16 ? 2 : 4;
            const uint32_t row_bytes = (uint32_t)a.H_v * D * ES;
            const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
                (char *)a.o + (size_t)t0 * row_bytes, (short)0, (int)(row_bytes * (uint32_t)n), 0x00020000);
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb) {
                if (kb + 1 < NKB) ktread(kb + 1, kt[(kb + 1) & 1]);
#pragma unroll
                for (int sl = 0; sl < NSL; ++sl) {
                    S[sl][kb] = mfma_f16(kt[kb & 1][0], d16[sl][0], S[sl][kb]);
                    S[sl][kb] = mfma_f16(kt[kb & 1][1], d16[sl][1], S[sl][kb]);
                }
                if (kb < 4) {
                    const int rb = kb;
#pragma unroll
                    for (int sl = 0; sl < NSL; ++sl) {
                        oacc[rb][sl] = mfma_f16(e16[sl][0], pf[frag_index(rb, 0)], oacc[rb][sl]);
                        if (rb >= 2) oacc[rb][sl] = mfma_f16(e16[sl][1], pf[frag_index(rb, 1)], oacc[rb][sl]);
                    }
#pragma unroll
                    for (int sl = 0; sl < NSL; ++sl) {
                        if constexpr (OUT_BF16) {
                            // into this wave's band of the v tile (o_stage_at), for the
                            // loaders to store as whole rows
                            const int r = 16 * rb + ln;
                            *(u32x2 *)(&sh.V[buf][o_stage_at(r, wr0 + 16 * sl + 4 * lg)]) =
                                __builtin_bit_cast(u32x2, __builtin_convertvector(oacc[rb][sl], bf16x4));
                        } else {
                            const uint32_t off = (uint32_t)(16 * rb + ln) * row_bytes + (uint32_t)(j * D + wr0 + 16 * sl + 4 * lg) * ES;
                            store_o4_f32(oacc[rb][sl], rs, off);
                        }
                    }
                }
                if (kb + 1 < NKB) WIDE_SG(SG_DSR, 4);
                const int nm = 2 * NSL + (kb < 2 ? NSL : kb < 4 ? 2 * NSL : 0);
                for (int i = 0; i < nm; ++i) {
                    WIDE_SG(SG_MFMA, 1);
                    WIDE_SG(SG_VALU, 2);
                }
            }
            __builtin_amdgcn_sched_barrier(0);

            // write signal: ||E row||^2 over each slice's 16 columns per token
            if (a.wsWrite) {
#pragma unroll
                for (int sl = 0; sl < NSL; ++sl) {
                    float *wb = a.wsWrite + ((size_t)j * a.n_split + wr0 / 16 + sl) * a.st.T + t0;
#pragma unroll
                    for (int ks = 0; ks < 2; ++ks) {
                        const float wsum = row_sq_sum16(e16[sl][ks], ln);
                        const int i = ln >> 1, tok = 32 * ks + 16 * (i >> 2) + 4 * lg + (i & 3);
                        if ((ln & 1) == 0 && tok < n) wb[tok] = wsum;
                    }
                }
            }

            // frame end: per-lane drift sums of the wave's slices against the state the
            // frame started from (read back from the scratch area), snapshot
            if (DRIFT && TILE * lt + n == frame_end) {
#pragma unroll
                for (int sl = 0; sl < NSL; ++sl) {
                    float num = 0.f, den = 0.f;
#pragma unroll
                    for (int kb = 0; kb < NKB; ++kb) {
                        const f32x4 s0 = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rstart, lane16, start_const(sl, kb), 0));
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const float dl = S[sl][kb][e] - s0[e];
                            num += dl * dl;
                            den += s0[e] * s0[e];
                        }
                    }
                    sh.DR[frame & 1][w][sl][lane] = float2{num, den};
                }
                if (a.snapshots && frame < a.n_frames) {
                    const __amdgpu_buffer_rsrc_t rsn = __builtin_amdgcn_make_buffer_rsrc(
                        (void *)(a.snapshots + ((size_t)frame * a.H_v + j) * D * D), (short)0, D * D * 4, RSRC_FLAGS);
#pragma unroll
                    for (int sl = 0; sl < NSL; ++sl)
#pragma unroll
                        for (int kb = 0; kb < NKB; ++kb)
                            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, S[sl][kb]), rsn, lane_row, sconst(sl, kb), 0);
                }
                save_start();
                ++frame;
                frame_end = min(frame_end + a.frame_len, len);
            }
        };
        for (int i = 0; i < nt; i += 2) {
            tile(lt0 + i, std::integral_constant<int, 0>());
            if (i + 1 < nt) tile(lt0 + i + 1, std::integral_constant<int, 1>());
        }
        if (nt > 0) lds_barrier();  // loader 3 reduces the last frame after it
        const __amdgpu_buffer_rsrc_t rout =
            __builtin_amdgcn_make_buffer_rsrc((void *)(a.state_out + hbase), (short)0, D * D * 4, RSRC_FLAGS);
#pragma unroll
        for (int sl = 0; sl < NSL; ++sl)
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb)
                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, S[sl][kb]), rout, lane_row, sconst(sl, kb), 0);
    } else {
        // ============================================================ loaders
        auto run = [&](auto xc) __attribute__((always_inline)) {
            constexpr int X = decltype(xc)::value;
            constexpr int NT = X < 2 ? 2 : 1;  // T and P fragments
            constexpr int F_FIRST = X < 2 ? 2 * X : 4 + (X - 2);
            constexpr int CH = D / 8, RPI = 64 / CH;  // 16-byte chunks per row, rows per 64-lane load
            // the workgroup's band of v and o columns (r0 .. r0 + 64 NSL - 1)
            constexpr int VCH = 8 * NSL, VRPI = 64 / VCH, NV = 16 / VRPI;  // chunks per row, rows per load, loads
            // it_: the tile's place in this launch (tile lt0 + it_)
            auto load = [&](WideLoad &s, int it_) __attribute__((always_inline)) {
                const int lt = lt0 + min(it_, nt - 1);  // clamped: every call issues the same loads
                const int t0 = st + TILE * lt, n = min(TILE, en - t0);
                const size_t tv = (size_t)(tile_base + lt) * a.H_v + j;
                const uint16_t *kb = a.k + (size_t)t0 * a.H_k * D + (size_t)qh * D + 8 * (lane % CH);
                const uint16_t *qb = a.q + (size_t)t0 * a.H_k * D + (size_t)qh * D + 8 * (lane % CH);
                const uint16_t *vb = a.v + ((size_t)t0 * a.H_v + j) * D + r0 + 8 * (lane % VCH);
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const uint32_t r = (uint32_t)min(16 * X + RPI * c + lane / CH, n - 1);
                    s.k[c] = *(const u32x4 *)(kb + r * (uint32_t)a.H_k * D);
                    s.q[c] = *(const u32x4 *)(qb + r * (uint32_t)a.H_k * D);
                }
#pragma unroll
                for (int c = 0; c < NV; ++c) {
                    const uint32_t r = (uint32_t)min(16 * X + VRPI * c + lane / VCH, n - 1);
                    s.v[c] = *(const u32x4 *)(vb + r * (uint32_t)a.H_v * D);
                }
                const u32x4 *tb = (const u32x4 *)(a.wsT + tv * TP_HALVES);
#pragma unroll
                for (int c = 0; c < NT; ++c) s.t[c] = tb[(F_FIRST + c) * 64 + lane];
                if (X < 2) s.g = a.wsGam[tv * 128 + 64 * X + lane];
            };
            auto stage = [&](const WideLoad &s, auto bufc) __attribute__((always_inline)) {
                constexpr int buf = decltype(bufc)::value;
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const int row = 16 * X + RPI * c + lane / CH, ch = lane % CH;
                    *(u32x4 *)(&sh.K[buf][row * D + 8 * (ch ^ swz<D>(row))]) = __builtin_bit_cast(u32x4, bf16x8_to_f16(s.k[c]));
                    *(u32x4 *)(&sh.Q[buf][row * D + 8 * (ch ^ swz<D>(row))]) = __builtin_bit_cast(u32x4, bf16x8_to_f16(s.q[c]));
                }
#pragma unroll
                for (int c = 0; c < NV; ++c) {
                    const int row = 16 * X + VRPI * c + lane / VCH;
                    *(u32x4 *)(&sh.V[buf][row * WIDE_VLD + r0 + 8 * (lane % VCH)]) = s.v[c];
                }
#pragma unroll
                for (int c = 0; c < NT; ++c) sh.T[buf][F_FIRST + c][lane] = s.t[c];
                if (X == 0) {
                    sh.G[buf][0][lane] = __builtin_amdgcn_exp2f(s.g);
                    sh.Gs[buf][lane] = s.g;
                } else if (X == 1) {
                    sh.G[buf][1][lane] = s.g;
                }
            };
            // P of the tile in LDS buffer buf, query rows 16 X .. 16 X + 15:
            // (K Q^T) blocks (nb, X) for key blocks nb <= X on fp16 matrix cores (lane
            // (ln, lg) holds keys 16 nb + 4 lg + e of query 16 X + ln: half of an A
            // fragment of P in the token order of E), gated by 2^(gamma_i - gamma_j)
            // and the output scale, zero above the diagonal.  Rows past a ragged
            // tile's end hold copies of its last row: they only reach o rows that
            // are not stored, since P is lower triangular
            auto form_p = [&](auto bufc) __attribute__((always_inline)) {
                constexpr int buf = decltype(bufc)::value;
                f32x4 gq[X + 1];
#pragma unroll
                for (int nb = 0; nb <= X; ++nb) gq[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < D / 32; ++ks) {
                    const int rq = 16 * X + ln;
                    const half8 bq = as_half8(*(const u32x4 *)(&sh.Q[buf][rq * D + 8 * ((4 * ks + lg) ^ swz<D>(rq))]));
#pragma unroll
                    for (int nb = 0; nb <= X; ++nb) {
                        const int rk = 16 * nb + ln;
                        const half8 ak = as_half8(*(const u32x4 *)(&sh.K[buf][rk * D + 8 * ((4 * ks + lg) ^ swz<D>(rk))]));
                        gq[nb] = mfma_f16(ak, bq, gq[nb]);
                    }
                }
                const float gi = sh.Gs[buf][16 * X + ln];
                auto pblock = [&](int nb) __attribute__((always_inline)) {
                    f32x4 pk = {0.f, 0.f, 0.f, 0.f};
                    if (nb <= X) {
                        const float4 gj = *(const float4 *)(&sh.Gs[buf][16 * nb + 4 * lg]);
                        const float gjv[4] = {gj.x, gj.y, gj.z, gj.w};
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            pk[e] = (nb < X || 4 * lg + e <= ln) ? __builtin_amdgcn_exp2f(gi - gjv[e]) * (a.scale * gq[nb][e]) : 0.f;
                    }
                    return pk;
                };
                sh.P[buf][frag_index(X, 0)][lane] = __builtin_bit_cast(u32x4, to_half8(pblock(0), pblock(1)));
                if (X >= 2) sh.P[buf][frag_index(X, 1)][lane] = __builtin_bit_cast(u32x4, to_half8(pblock(2), pblock(3)));
            };
            // bf16 o of tile lt from the v buffer it was staged in (rows 16 X .. 16 X +
            // 15, the rows this loader restages next): 16-byte pieces read back in
            // order, stored as whole rows of the workgroup's band; stores past a
            // ragged tile's end fall outside the buffer resource and are dropped
            // (read_o into registers before the rows are restaged, store_o later)
            auto read_o = [&](u32x4(&ov)[4], auto bufc) __attribute__((always_inline)) {
                constexpr int buf = decltype(bufc)::value;  // == (lt - lt0) % 2
#pragma unroll
                for (int c = 0; c < NV; ++c) {
                    const int r = 16 * X + VRPI * c + lane / VCH, ch = r0 / 8 + lane % VCH;
                    // dims 8 ch .. 8 ch + 7 = two 4-dim pieces, kept adjacent by the permutation
                    // and swapped when (r / 4) % 2 == 1
                    ov[c] = *(const u32x4 *)(&sh.V[buf][o_stage_at(r, 8 * ch) & ~7]);
                }
            };
            auto store_o = [&](int lt, const u32x4(&ov)[4]) __attribute__((always_inline)) {
                const int t0 = st + TILE * lt, n = min(TILE, en - t0);
                const uint32_t row_bytes = (uint32_t)a.H_v * D * 2;
                const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
                    (char *)a.o + (size_t)t0 * row_bytes, (short)0, (int)(row_bytes * (uint32_t)n), 0x00020000);
#pragma unroll
                for (int c = 0; c < NV; ++c) {
                    const int r = 16 * X + VRPI * c + lane / VCH, ch = r0 / 8 + lane % VCH;
                    const u32x4 v = ((r >> 2) & 1) ? u32x4{ov[c][2], ov[c][3], ov[c][0], ov[c][1]} : ov[c];
                    __builtin_amdgcn_raw_buffer_store_b128(v, rs, (uint32_t)r * row_bytes + (uint32_t)(j * D + 8 * ch) * 2, 0, 0);
                }
            };
            // drift: loader 3 adds the slices' sums of a frame that ended in the
            // previous tile and writes them: a whole head's 8 slices in order as
            // one pair, or per slice (a half head's 4 slices always per slice; the
            // head's pair is then added after both halves are done)
            const int fr0 = frame_base + (a.frame_len > 0 ? tok0 / a.frame_len : 0);
            int frame = fr0;
            int frame_end = a.frame_len > 0 ? min(tok0 + a.frame_len, len) : len;
            auto drift_reduce = [&](int it) __attribute__((always_inline)) {
                if (!DRIFT || X != 3 || it < 1) return;
                const int lt = lt0 + it - 1;
                if (TILE * lt + min(TILE, len - TILE * lt) != frame_end) return;
                if (a.wsDrift && frame < a.n_frames) {
                    constexpr int NS = 4 * NSL;  // this workgroup's slices sl0 .. sl0 + NS - 1
                    float2 pr[NS];
#pragma unroll
                    for (int s = 0; s < NS; ++s) {
                        const float2 p = sh.DR[frame & 1][s / NSL][s % NSL][lane];
                        pr[s] = float2{wave_sum(p.x), wave_sum(p.y)};
                    }
                    const size_t fj = (size_t)frame * a.H_v + j;
                    if (NSL == 2 && a.drift_out) {  // per-head pair: the slices in order
                        float num = 0.f, den = 0.f;
#pragma unroll
                        for (int s = 0; s < NS; ++s) {
                            num += pr[s].x;
                            den += pr[s].y;
                        }
                        if (lane == 0) *(float2 *)(a.drift_out + fj * 2) = float2{num, den};
                    } else if (lane < NS) {  // per-slice pairs
                        float2 mine = pr[0];
#pragma unroll
                        for (int s = 1; s < NS; ++s)
                            if (lane == s) mine = pr[s];
                        float *dst = a.wsDrift + (fj * a.n_split + sl0 + lane) * 2;
                        if (a.drift_out)  // read by the other half's workgroup
                            store_pair_coherent(dst, mine.x, mine.y);
                        else
                            *(float2 *)dst = mine;
                    }
                }
                ++frame;
                frame_end = min(frame_end + a.frame_len, len);
            };
            if (nt > 0) {
                WideLoad s0, s1;
                load(s0, 0);
                load(s1, 1);
                stage(s0, std::integral_constant<int, 0>());
                load(s0, 2);
                // P of tile it + 1 is formed during tile it, after the tile's second
                // barrier, from the K and q rows all four loaders staged before it, and
                // handed to the compute waves at the next tile's first barrier (P of
                // tile 0 before the first tile's second barrier).  Before the second
                // barrier a loader does LDS work only (the compute waves wait there for
                // the last loader; the o rows are read back before they are restaged);
                // its global stores and loads follow it
                auto step = [&](int it, WideLoad &s, auto bufc) __attribute__((always_inline)) {
                    lds_barrier();
                    if (it == 0) form_p(std::integral_constant<int, 0>());
                    u32x4 ov[4];
                    if (OUT_BF16 && it >= 1) read_o(ov, bufc);
                    if (it + 1 < nt) stage(s, bufc);
                    if (it < nt) lds_barrier();
                    if (OUT_BF16 && it >= 1) store_o(lt0 + it - 1, ov);
                    if (it + 1 < nt) form_p(bufc);
                    load(s, it + 3);
                    drift_reduce(it);
                };
                // tile lt0 + t lives in register set t % 2 and LDS buffer t % 2;
                // iteration it stages tile it + 1 and then loads tile it + 3 into the set
                // just freed
                for (int it = 0; it <= nt; it += 2) {
                    step(it, s1, std::integral_constant<int, 1>());
                    if (it + 1 <= nt) step(it + 1, s0, std::integral_constant<int, 0>());
                }
            }
            // half heads with per-head pairs: the second of the head's two
            // workgroups to finish adds the 8 slices of this launch's frames in
            // order (the counters were cleared by the prep pass)
            if (NSL == 1 && DRIFT && X == 3 && a.drift_out && a.wsDrift) {
                wait_vmem_all();  // this wave's pairs are coherent before the count
                unsigned prev = 0;
                if (lane == 0)
                    prev = __hip_atomic_fetch_add(&a.drift_cnt[b * a.H_v + j], 1u, __ATOMIC_RELAXED,
                                                  __HIP_MEMORY_SCOPE_AGENT);
                prev = __builtin_amdgcn_readfirstlane(prev);
                if (prev == (unsigned)HW - 1u) {
                    const int fr1 = min(frame_base + frames_in(len, a.frame_len), a.n_frames);
                    for (int f = fr0 + lane; f < fr1; f += 64) {
                        const size_t fj = (size_t)f * a.H_v + j;
                        float2 pr[8];
#pragma unroll
                        for (int s8 = 0; s8 < 8; ++s8) pr[s8] = load_pair_coherent(a.wsDrift + (fj * a.n_split + s8) * 2);
                        float num = 0.f, den = 0.f;
#pragma unroll
                        for (int s8 = 0; s8 < 8; ++s8) {
                            num += pr[s8].x;
                            den += pr[s8].y;
                        }
                        *(float2 *)(a.drift_out + fj * 2) = float2{num, den};
                    }
                }
            }
        };
        if (w == 4)
            run(std::integral_constant<int, 0>());
        else if (w == 5)
            run(std::integral_constant<int, 1>());
        else if (w == 6)
            run(std::integral_constant<int, 2>());
        else
            run(std::integral_constant<int, 3>());
    }
}

template <int NSL>
static hipError_t launch_wide_nsl(const GdnArgs &a, int n_wg, bool o_bf16, bool drift, hipStream_t stream) {
    if (o_bf16) {
        if (drift)
            hipLaunchKernelGGL((gdn_wide_kernel<true, true, NSL>), dim3(n_wg), dim3(512), 0, stream, a);
        else
            hipLaunchKernelGGL((gdn_wide_kernel<true, false, NSL>), dim3(n_wg), dim3(512), 0, stream, a);
    } else {
        if (drift)
            hipLaunchKernelGGL((gdn_wide_kernel<false, true, NSL>), dim3(n_wg), dim3(512), 0, stream, a);
        else
            hipLaunchKernelGGL((gdn_wide_kernel<false, false, NSL>), dim3(n_wg), dim3(512), 0, stream, a);
    }
    return hipGetLastError();
}

// One launch of whole heads, or, for calls whose frames are whole tiles and
// when at most tail_streams streams fit the GPU as half heads, whole heads up
// to the cut (the tile from which at most tail_streams streams are left,
// on a frame boundary) and half heads from it, the second launch starting
// from the states the first one wrote.
hipError_t launch_gdn_wide(const GdnArgs &a0, int n_heads, int tail_streams, bool o_bf16, bool drift,
                           hipStream_t stream) {
    GdnArgs a = a0;
    const bool split = tail_streams >= 1 && a.frame_len > 0 && a.frame_len % TILE == 0;
    a.wide_tail_streams = tail_streams;
    a.wide_phase = split ? 1 : 0;
    hipError_t e = launch_wide_nsl<2>(a, n_heads, o_bf16, drift, stream);
    if (e != hipSuccess || !split) return e;
    a.wide_phase = 2;
    a.state_in = a.state_out;
    return launch_wide_nsl<1>(a, 2 * n_heads, o_bf16, drift, stream);
}

}  // namespace ds
