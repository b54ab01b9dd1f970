// Chunkwise gated-delta-rule forward with fused frame drift (gfx950).
//
// The token recurrence of Section 3.2 (Eq. 2) is evaluated over tiles of 64
// tokens.  Inside a tile with entry state S0 (d_v x d_k), with
// gamma_r = sum_{j<=r} g_j, Gamma_r = exp(gamma_r), D_ri = exp(gamma_r - gamma_i),
// unrolling Eq. 2 gives the writes e_r as the solution of a unit
// lower-triangular system:
//     (I + A) E = diag(beta) (V - diag(Gamma) K S0^T),
//     A_ri = beta_r D_ri (k_r . k_i)  for i < r,
// and then
//     O    = diag(Gamma) Q S0^T + (D (.) Q K^T)_{i<=r} E
//     S_64 = Gamma_last S0 + E^T diag(D_last,.) K.
// Two kernels share the work:
//   gdn_prep  (all tiles in parallel): the state-independent part -- K K^T,
//             Q K^T on bf16 matrix cores, T = (I + A)^{-1} in fp32, written
//             as fp16 T diag(beta) and P = D (.) tril(Q K^T), plus the decay factors
//             exp(gamma_r) and exp(gamma_last - gamma_r);
//   gdn_seq   (one workgroup per (stream, v-head, 16 rows of S)): walks the
//             tiles in order, keeps its rows of S in fp32 registers, does the
//             state-dependent products on fp16 matrix cores, writes o, and at
//             every frame end the drift sums of Eq. 3 for its rows.
//   The drift sums of the slices are added in a fixed order by the last
//   workgroup of each (stream, v-head) to finish (gdn_drift_finalize only
//   for a call without tokens).
#include <type_traits>

#include "gdn_common.h"

namespace ds {

// ============================================================================
// The prep pass (prep_tile), per tile and qk-head.  The K and Q rows of the tile
// are loaded once as whole 16-byte chunks and staged in LDS; the Gram blocks
// K K^T and (K Q^T) run on bf16 matrix cores (exact bf16 inputs, fp32
// accumulation) and stay in registers.  Then, for every v-head of the group
// (its own gates): P is gated, multiplied by the output scale and written
// straight from the K Q^T registers (their layout is already P's fragment
// layout), and the inverse of the unit
// lower-triangular I + A is blocked in 16 x 16 blocks: the diagonal blocks by
// forward substitution, then the off-diagonal ones on fp32 matrix cores
// in two levels of the 2 x 2 block inverse
// [[T11, 0], [T21, T22]] with T21 = -T22 A21 T11: first the 32 x 32 halves,
// then the lower-left quarter.
// 39 KiB of LDS and at most 128 VGPRs, so that four workgroups share a CU.
// ============================================================================
template <int D>
struct PrepLds {
    static constexpr int ALD = 68;  // floats per LDS row of A and T (bank-conflict-free writes)
    static constexpr int RB = (64 * D * 2 > 64 * ALD * 4) ? 64 * D * 2 : 64 * ALD * 4;
    // K and Q tiles while the Gram blocks are formed, then A and T (39.4 KiB
    // in all for d = 128: four workgroups fit in a CU's LDS)
    __align__(16) char reg_k[RB];
    __align__(16) char reg_q[RB];
    float Ys[4][256];
    __align__(16) float gam_s[2][64];   // log2 Gamma and beta of up to two v-heads
    __align__(16) float beta_s[2][64];
};

// Set-up for the sequential kernel's drift output by threads tid (of nt):
// slice counters of the in-kernel reduction to zero (with the per-head sums),
// the pairs of frames past the real count to zero.
__device__ __forceinline__ void drift_setup(const GdnArgs &a, int tid, int nt) {
    if (a.drift_out)
        for (int i = tid; i < a.st.B * a.H_v; i += nt) a.drift_cnt[i] = 0u;
    int real = 0;
    for_streams(a.st, [&](int, int s0, int e0) {
        real += frames_in(e0 - s0, a.frame_len);
        return false;
    });
    const int per = a.drift_zero_per_frame;
    for (int i = min(real, a.n_frames) * per + tid; i < a.n_frames * per; i += nt)
        *(float2 *)(a.drift_zero + 2 * (size_t)i) = float2{0.f, 0.f};
}

// The prep of tile ti (tokens t0 .. t0 + n - 1 of the packed sequence) for
// qk-head h and the v-heads jbase .. jbase + gcount - 1 of its group, by four
// waves w = 0 .. 3 with the LDS block L.  Every call passes the same barriers
// (lds_barrier, workgroup-wide), so that two groups of four waves of one
// workgroup can each run a tile side by side.  write_q: this call writes the
// tile's fp16 q fragments (when the workspace has them).  WP = false (the
// whole-head sequential kernel, which forms P itself from the K and q tiles it
// stages): no q rows, no K Q^T and no P, and the first decay slot holds
// gamma_r in base-2 units instead of Gamma_r.
template <int D, bool WP = true>
__device__ __forceinline__ void prep_tile(const GdnArgs &a, int ti, int t0, int n, int h, int jbase, int gcount,
                                          PrepLds<D> &L, int w, int lane, bool write_q) {
    constexpr int KS = D / 32;   // 32-wide k-steps over the head dim
    constexpr int CH = D / 8;    // 16-byte chunks per K or Q row
    constexpr int RPI = 64 / CH;  // rows per 64-lane row load
    constexpr int NI = 16 / RPI;  // row loads per wave (16 rows each)
    constexpr int ALD = PrepLds<D>::ALD;
    uint16_t *Kl = (uint16_t *)L.reg_k, *Ql = (uint16_t *)L.reg_q;
    float *As = (float *)L.reg_k, *Ts = (float *)L.reg_q;
    float(&Ys)[4][256] = L.Ys;
    float(&gam_s)[2][64] = L.gam_s;
    float(&beta_s)[2][64] = L.beta_s;
    const int tid = 64 * w + lane, ln = lane & 15, lg = lane >> 4;

    constexpr int MAXG = 2;  // v-heads per qk-head whose gates are loaded with K and Q (more: loaded in turn)

    // ---- K and Q rows 16 w .. 16 w + 15: whole 16-byte chunks, RPI rows per
    // load; rows past a ragged tile's end are loaded clamped and zeroed here
    {
        u32x4 kv[NI], qv[NI];
        const uint16_t *kb = a.k + (size_t)t0 * a.H_k * D + (size_t)h * D;
        const uint16_t *qb = a.q + (size_t)t0 * a.H_k * D + (size_t)h * D;
#pragma unroll
        for (int c = 0; c < NI; ++c) {
            const int row = 16 * w + RPI * c + lane / CH, ch = lane % CH;
            const uint32_t off = (uint32_t)min(row, n - 1) * (uint32_t)a.H_k * D + 8 * ch;
            kv[c] = *(const u32x4 *)(kb + off);
            if (WP) qv[c] = *(const u32x4 *)(qb + off);
        }
        // gates of the group's first v-heads (wave 0, lane = token), issued after
        // K and Q so that waiting for K and Q does not wait for them; raw g and
        // beta go to the gate slots of LDS, where the gate phase picks them up
        float gpre[MAXG], bpre[MAXG];
        if (w == 0) {
            const uint32_t r = (uint32_t)min(lane, n - 1);
#pragma unroll
            for (int jj = 0; jj < MAXG; ++jj) {
                const int j = jbase + min(jj, gcount - 1);
                gpre[jj] = a.g[(size_t)(t0 + r) * a.H_v + j];
                bpre[jj] = a.beta[(size_t)(t0 + r) * a.H_v + j];
            }
        }
#pragma unroll
        for (int c = 0; c < NI; ++c) {
            const int row = 16 * w + RPI * c + lane / CH, ch = lane % CH;
            const u32x4 z = {0u, 0u, 0u, 0u};
            *(u32x4 *)(&Kl[row * D + 8 * (ch ^ swz<D>(row))]) = row < n ? kv[c] : z;
            if (!WP) continue;
            const u32x4 q = row < n ? qv[c] : z;
            *(u32x4 *)(&Ql[row * D + 8 * (ch ^ swz<D>(row))]) = q;
            // q in fp16 for the output waves of the per-slice sequential kernel, in
            // A-fragment order: row block row / 16, k-step ch / 4, lane (ch % 4) * 16 +
            // row % 16 (the whole-head kernel converts q rows itself).  Like the T and
            // P fragments it is stored nontemporally: the fragments outgrow the
            // caches before the sequential kernel reads them
            const size_t fq = ((size_t)(row >> 4) * KS + (ch >> 2)) * 64 + (ch & 3) * 16 + (row & 15);
            if (a.wsQ && write_q)
                __builtin_nontemporal_store(__builtin_bit_cast(u32x4, bf16x8_to_f16(q)), (u32x4 *)(a.wsQ + ((size_t)ti * a.H_k + h) * 64 * D + fq * 8));
        }
        if (w == 0) {
#pragma unroll
            for (int jj = 0; jj < MAXG; ++jj) {
                gam_s[jj][lane] = gpre[jj];
                beta_s[jj][lane] = bpre[jj];
            }
        }
    }
    lds_barrier();

    // ---- Gram blocks of row block w, fragments straight from LDS (a B fragment
    // of K^T is an A fragment of K): K K^T blocks (w, nb) and the transposed
    // blocks (K Q^T)(nb, w) for nb <= w.  Lane (ln, lg) of the latter holds keys
    // 16 nb + 4 lg + e of query 16 w + ln, which is half of an A fragment of P
    // in the token order of E: P is written from the registers.
    f32x4 gk[4], gq[4];
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
        gk[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
        gq[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        const int ra = 16 * w + ln, ca = 8 * ((4 * ks + lg) ^ swz<D>(ra));
        const bf16x8 ak = as_bf16x8(*(const u32x4 *)(&Kl[ra * D + ca]));
        const bf16x8 aq = WP ? as_bf16x8(*(const u32x4 *)(&Ql[ra * D + ca])) : ak;
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) {
            if (nb <= w) {
                const int rb = 16 * nb + ln;
                const bf16x8 bk = as_bf16x8(*(const u32x4 *)(&Kl[rb * D + 8 * ((4 * ks + lg) ^ swz<D>(rb))]));
                gk[nb] = mfma_bf16(ak, bk, gk[nb]);
                if (WP) gq[nb] = mfma_bf16(bk, aq, gq[nb]);
            }
        }
    }
    lds_barrier();  // K and Q tiles are dead from here on (A and T reuse them)

    // ---- per v-head of the qk-head's group: gates (wave 0), P from the Gram
    // registers, then A and its inverse.  Groups of one or two v-heads (gates
    // prefetched above) run as straight-line code: inside a loop with a
    // data-dependent trip count the compiler cannot count the memory operations
    // in flight and would wait for every earlier store before reading the
    // prefetched gates.  For two v-heads both gate sets and both P are formed
    // first, so that the Q K^T registers are free during the inversions.
    // gates: gamma = inclusive prefix sum of g in base-2 units, and beta, into
    // LDS slot `slot`; Gamma and D_last to the workspace
    auto gates = [&](int jj, int slot) __attribute__((always_inline)) {
        const int j = jbase + jj;
        const size_t tv = (size_t)ti * a.H_v + j;
        if (w == 0) {
            float gv = 0.f, bv = 0.f;
            if (jj < MAXG) {  // loaded with K and Q (slot == jj)
                gv = gam_s[jj][lane];
                bv = beta_s[jj][lane];
            } else {
                gv = a.g[(size_t)(t0 + min(lane, n - 1)) * a.H_v + j];
                bv = a.beta[(size_t)(t0 + min(lane, n - 1)) * a.H_v + j];
            }
            if (lane >= n) gv = bv = 0.f;
            float s = wave_prefix_sum(gv);
            s *= 1.4426950408889634f;  // exp(gamma) = exp2(s)
            gam_s[slot][lane] = s;
            beta_s[slot][lane] = bv;
            // padding rows have g = 0, so row 63 carries the tile's last gamma
            const float s_last = __shfl(s, 63, 64);
            a.wsGam[tv * 128 + lane] = WP ? __builtin_amdgcn_exp2f(s) : s;
            a.wsGam[tv * 128 + 64 + lane] = __builtin_amdgcn_exp2f(s_last - s);
        }
    };
    // P (lower incl. diagonal) of query block w, scale Gamma_i / Gamma_j (q_i . k_j)
    // for keys j <= i (the output scale rides on P: o = scale diag(Gamma) Q S0^T + P E), as the A fragments (w, ks) of P E (k-step ks pairs key
    // blocks 2 ks, 2 ks + 1); block (nb, w): key 16 nb + 4 lg + e, query 16 w + ln
    auto pfrags = [&](int jj, int slot) __attribute__((always_inline)) {
        if (!WP) return;
        const size_t tv = (size_t)ti * a.H_v + jbase + jj;
        // the gates first (one LDS round trip), then every product, masked by a
        // select: a lane-dependent condition around the products would compile
        // to a branch that waits for its own LDS reads
        const float gq_i = gam_s[slot][16 * w + ln];  // query 16 w + ln
        float4 gj[4];
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) gj[nb] = *(const float4 *)(&gam_s[slot][16 * nb + 4 * lg]);
        auto pblock = [&](int nb) __attribute__((always_inline)) {
            f32x4 pk = {0.f, 0.f, 0.f, 0.f};
            if (nb <= w) {  // wave-uniform
                const float gjv[4] = {gj[nb].x, gj[nb].y, gj[nb].z, gj[nb].w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float pv = __builtin_amdgcn_exp2f(gq_i - gjv[e]) * (a.scale * gq[nb][e]);
                    pk[e] = (nb < w || 4 * lg + e <= ln) ? pv : 0.f;
                }
            }
            return pk;
        };
        _Float16 *pw = a.wsP + tv * TP_HALVES + lane * 8;
        __builtin_nontemporal_store(__builtin_bit_cast(u32x4, to_half8(pblock(0), pblock(1))), (u32x4 *)(pw + frag_index(w, 0) * FRAG_HALVES));
        if (w >= 2) __builtin_nontemporal_store(__builtin_bit_cast(u32x4, to_half8(pblock(2), pblock(3))), (u32x4 *)(pw + frag_index(w, 1) * FRAG_HALVES));
    };
    auto invert = [&](int jj, int slot) __attribute__((always_inline)) {
        const size_t tv = (size_t)ti * a.H_v + jbase + jj;
        // A (strictly lower), rows of block w
        {
            const float4 gr = *(const float4 *)(&gam_s[slot][16 * w + 4 * lg]);
            const float4 br = *(const float4 *)(&beta_s[slot][16 * w + 4 * lg]);
            const float grv[4] = {gr.x, gr.y, gr.z, gr.w}, brv[4] = {br.x, br.y, br.z, br.w};
            float gi[4];
#pragma unroll
            for (int nb = 0; nb < 4; ++nb) gi[nb] = gam_s[slot][16 * nb + ln];
#pragma unroll
            for (int nb = 0; nb < 4; ++nb) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int r = 16 * w + 4 * lg + e, i = 16 * nb + ln;
                    float av = 0.f;
                    if (nb <= w) {  // wave-uniform; the lane condition is a select (see pfrags)
                        const float v = brv[e] * __builtin_amdgcn_exp2f(grv[e] - gi[nb]) * gk[nb][e];
                        av = i < r ? v : 0.f;
                    }
                    As[r * ALD + i] = av;
                }
            }
        }
        lds_barrier();

        // 16x16 block products on fp32 matrix cores from LDS (row-major blocks,
        // leading dimension ld): acc += X Y.  16x16x4 fragments: A lane = [ln][lg],
        // B lane = [lg][ln], C lane = [4 lg + e][ln].
        auto bmm = [&](f32x4 acc, const float *X, int ldx, const float *Y, int ldy) __attribute__((always_inline)) {
#pragma unroll
            for (int s4 = 0; s4 < 4; ++s4) acc = mfma_f32_16x16x4(X[ln * ldx + 4 * s4 + lg], Y[(4 * s4 + lg) * ldy + ln], acc);
            return acc;
        };
        auto blk = [&](float *M, int bi, int bj) __attribute__((always_inline)) { return M + 16 * bi * ALD + 16 * bj; };

        // (1) diagonal blocks: wave w inverts block w by forward substitution,
        // lane 4 c + p taking column c of the inverse and the terms i = p mod 4
        // of every row's dot product (its four partial sums are added across
        // the lane quad), so that a lane reads at most four A values per row
        // and the dependent chain per row is one product and two adds.  Lane p
        // keeps x_i for the rows i = p mod 4 (zero until they are formed; A is
        // zero on and above the diagonal).
        {
            const int o = 16 * w, c = lane >> 2, p = lane & 3;
            // all 36 A values of the lane read first (they do not depend on x;
            // left to the scheduler, each row's reads were waited for in turn)
            float am[16][4];
#pragma unroll
            for (int r = 1; r < 16; ++r)
#pragma unroll
                for (int m = 0; m < (r + 3) / 4; ++m) am[r][m] = As[(o + r) * ALD + o + 4 * m + p];
            __builtin_amdgcn_sched_barrier(0);
            float xp[4] = {0.f, 0.f, 0.f, 0.f};  // x_{4 m + p}
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                float ps = 0.f;
#pragma unroll
                for (int m = 0; m < (r + 3) / 4; ++m) ps += am[r][m] * xp[m];
                ps += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, ps), 0xB1, 0xF, 0xF, true));  // quad lanes p ^ 1
                ps += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, ps), 0x4E, 0xF, 0xF, true));  // quad lanes p ^ 2
                const float xr = ((r == c) ? 1.f : 0.f) - ps;
                if (p == (r & 3)) xp[r >> 2] = xr;
            }
#pragma unroll
            for (int m = 0; m < 4; ++m) Ts[(o + 4 * m + p) * ALD + o + c] = xp[m];
        }
        lds_barrier();

        // first level of the blocked inverse, waves 0 and 1:
        // T_{2u+1,2u} = -T_{2u+1,2u+1} (A_{2u+1,2u} T_{2u,2u})
        if (w < 2) {
            float *yw = Ys[w];
            const int bi = 2 * w + 1, bj = 2 * w;
            const f32x4 y = bmm(f32x4{0.f, 0.f, 0.f, 0.f}, blk(As, bi, bj), ALD, blk(Ts, bj, bj), ALD);
#pragma unroll
            for (int e = 0; e < 4; ++e) yw[(4 * lg + e) * 16 + ln] = y[e];
            __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's Y is in LDS
            const f32x4 t = bmm(f32x4{0.f, 0.f, 0.f, 0.f}, blk(Ts, bi, bi), ALD, yw, 16);
#pragma unroll
            for (int e = 0; e < 4; ++e) Ts[(16 * bi + 4 * lg + e) * ALD + 16 * bj + ln] = -t[e];
        }
        lds_barrier();

        // (2) second level: the lower-left 32x32 quarter
        //   T_[23][01] = -T_[23][23] (A_[23][01] T_[01][01]),
        // wave w forming block (i, j) = (2 + w / 2, w % 2) of each product
        {
            const int i = 2 + (w >> 1), j = w & 1;
            f32x4 y = bmm(f32x4{0.f, 0.f, 0.f, 0.f}, blk(As, i, j), ALD, blk(Ts, j, j), ALD);
            if (j == 0) y = bmm(y, blk(As, i, 1), ALD, blk(Ts, 1, 0), ALD);
            float *yw = Ys[w];
#pragma unroll
            for (int e = 0; e < 4; ++e) yw[(4 * lg + e) * 16 + ln] = y[e];
            lds_barrier();
            // Y_{m j} of wave 2 (m - 2) + j
            f32x4 t = bmm(f32x4{0.f, 0.f, 0.f, 0.f}, blk(Ts, i, 2), ALD, Ys[j], 16);
            if (i == 3) t = bmm(t, blk(Ts, 3, 3), ALD, Ys[2 + j], 16);
#pragma unroll
            for (int e = 0; e < 4; ++e) Ts[(16 * i + 4 * lg + e) * ALD + 16 * j + ln] = -t[e];
        }
        lds_barrier();

        // T diag(beta) (fp16, zero above the diagonal) in fragment order
        for (int c = tid; c < 6 * 64; c += 256) {
            const int f = c >> 6, l = c & 63;
            const int fw = f < 2 ? f : 2 + ((f - 2) >> 1), fks = f < 2 ? 0 : ((f - 2) & 1);
            const int r = 16 * fw + (l & 15), c4 = 32 * fks + 4 * (l >> 4);
            // columns c4 .. c4 + 3 and c4 + 16 .. c4 + 19 of row r, as two 16-byte reads each
            const float4 ta = *(const float4 *)(&Ts[r * ALD + c4]), tb = *(const float4 *)(&Ts[r * ALD + c4 + 16]);
            const float4 ba = *(const float4 *)(&beta_s[slot][c4]), bb = *(const float4 *)(&beta_s[slot][c4 + 16]);
            const float tx[8] = {ta.x * ba.x, ta.y * ba.y, ta.z * ba.z, ta.w * ba.w,
                                 tb.x * bb.x, tb.y * bb.y, tb.z * bb.z, tb.w * bb.w};
            half8 tv8;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int i = c4 + 16 * (e >> 2) + (e & 3);
                tv8[e] = (_Float16)((i <= r) ? tx[e] : 0.f);
            }
            __builtin_nontemporal_store(__builtin_bit_cast(u32x4, tv8), (u32x4 *)(a.wsT + tv * TP_HALVES + f * FRAG_HALVES + l * 8));
        }
        lds_barrier();  // before the next v-head reuses A, T and the gate slot
    };
    if (gcount == 1) {
        gates(0, 0);
        lds_barrier();
        pfrags(0, 0);
        invert(0, 0);
    } else if (gcount == 2) {
        gates(0, 0);
        gates(1, 1);
        lds_barrier();
        pfrags(0, 0);
        pfrags(1, 1);
        invert(0, 0);
        invert(1, 1);
    } else {
        for (int jj = 0; jj < gcount; ++jj) {
            gates(jj, 0);
            lds_barrier();
            pfrags(jj, 0);
            invert(jj, 0);
        }
    }
}

// ============================================================================
// gdn_prep: one workgroup per (tile, qk-head), or per (tile, v-head) for small
// launches; the work of a tile is prep_tile.
// ============================================================================
template <int D, bool WP>
__global__ __launch_bounds__(256, 4) void gdn_prep_kernel(GdnArgs a) {
    __shared__ __align__(16) PrepLds<D> L;
    // The grid is one-dimensional and tile-major per XCD (dispatch deals
    // workgroups to the 8 XCDs in turn): the workgroups of every head of one
    // tile run on one XCD one after another, so the gate rows of a token
    // (all v-heads in one line) are fetched into one L2 once.
    const int nhy = a.prep_per_vhead ? a.H_v : a.H_k;
    const int bid = blockIdx.x, slot = bid >> 3;
    const int ti = (slot / nhy) * 8 + (bid & 7), hy = slot % nhy;
    const int h = a.prep_per_vhead ? hy / a.group : hy;
    const int jbase = a.prep_per_vhead ? hy : h * a.group;
    const int gcount = a.prep_per_vhead ? 1 : a.group;
    if (ti == 0 && hy == 0 && a.drift_zero) drift_setup(a, threadIdx.x, 256);
    int t0 = 0, n = 0;
    if (!locate_tile(a.st, ti, t0, n)) return;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    // one writer of the q fragments per qk-head
    prep_tile<D, WP>(a, ti, t0, n, h, jbase, gcount, L, w, threadIdx.x & 63, jbase == h * a.group);
}

// ============================================================================
// gdn_seq: one workgroup of 8 waves per (stream, v-head, 16 consecutive rows
// of S):
//   waves 0 and 1, state:  carry the recurrence for the 16 rows of S in fp32
//                    registers, wave h owning the state columns (dims of k)
//                    of its half.  Per tile: both compute all of K S0^T from
//                    the fp16 copy of S0 that the two waves left in LDS at the
//                    end of the previous tile (identical sums in both, no
//                    handshake inside the tile), both form
//                    R = V - diag(Gamma) K S0^T and E = T diag(beta) R, and each
//                    updates its half, S = Gamma_last S0 + (D_last E)^T K, and
//                    writes the half's fp16 copy for the next tile.
//                    Every product's result becomes the next product's B
//                    operand inside the registers.  S0 and E are published in
//                    LDS for the output waves; at a frame end each lane
//                    leaves its share of the drift sums in LDS.
//   waves 2 and 3, output:  one tile behind, O = scale diag(Gamma) Q S0^T + P E
//                    (the prep pass folded the scale into P) for row blocks
//                    {0, 1} and {2, 3}; they load q (the fp16 fragments
//                    of the prep pass) and P themselves.
//   waves 4 - 7, loaders: each loads a quarter of the K rows, T diag(beta),
//                    v rows and the decay factors of a tile three tiles ahead
//                    and stages it in LDS one tile ahead.  The state waves read
//                    K as rows (A operand of K S0^T) and, by transposing reads,
//                    as K^T (A operand of the state update).  Loader 3 also
//                    reduces the frame-end drift sums over the lanes, one tile
//                    later, off the state waves' chain.
// All eight waves meet at one barrier per tile.  A single wave moves data
// from L2 and from LDS at a limited rate, which is why the chain is shared by
// two waves, every tile is loaded by four waves, and operands move as whole
// 16-byte pieces.
//
// Fragment bookkeeping.  The C layout of v_mfma_f32_16x16x32 (lane (ln, lg)
// holds rows 4 lg + e of column ln) of two row blocks 2 s and 2 s + 1 is,
// read as 8 values per lane, exactly a B operand (rows 8 lg .. 8 lg + 7 of a
// 32-row k-step) once the k-step's 32 rows are relabelled; the A operand that
// meets it is loaded with the same relabelling.  Two relabellings are used:
//   state rows  (k, the columns of S):  block kb, C row m  <->  k = sigma(kb, m)
//       sigma(kb, m) = 32 (kb / 2) + 8 (m / 4) + 4 (kb % 2) + m % 4,
//     so that S0 as a B operand runs over k = 32 ks + 8 lg + i in order and K
//     and Q are read as plain 16-byte rows;
//   token rows  (R, E, O):  C rows stay in order (row block rb, row 4 lg + e
//     is token 16 rb + 4 lg + e), so as a B operand element i of k-step ks
//     is token kappa(ks, lg, i) = 32 ks + 16 (i / 4) + 4 lg + i % 4; the
//     prep kernel writes T diag(beta) and P with their token columns in that
//     order, and the K^T fragments are read from LDS in it.
//
// Precision: the state stays fp32 in registers; as a matrix-core operand it
// is rounded to fp16 (relative error 2^-11, the same as R and E), and k and q
// meet it as fp16 (exact conversions of the bf16 inputs in fp16's normal
// range).  D_last E enters the state update as fp16; R, E, T diag(beta) and
// P are fp16.  All accumulation is fp32.
// ============================================================================

template <int D>
struct SeqShared {
    static constexpr int KS = D / 32, NKB = D / 16;
    uint16_t K[2][64 * D];     // K tile (fp16), row-major, 16-byte chunks XOR-swizzled by row (swz)
    u32x4 T[2][6][64];         // T diag(beta) A-fragments
    uint16_t V[2][64 * 16];    // v[token][v0 .. v0 + 15] (bf16, read transposed)
    float G[3][2][64];         // Gamma_r and D_last,r of tile t in G[t % 3] (the output waves read it a tile later)
    u32x4 S16[3][KS][64];      // S0 of tile t as fp16 B operand in S16[t % 3]: each state wave
                               // writes its half at the end of tile t - 1, both state waves
                               // read all of it in tile t, the output waves a tile later
    u32x4 E[2][2][64];         // E as B operand (fp16)
    float2 DR[2][2][64];       // per-lane drift sums of a frame end: [frame % 2][state wave][lane]
};

// One loader's share of a tile: K rows 16 x .. 16 x + 15 (whole 16-byte
// chunks, 64 / (D / 8) rows per load), T diag(beta) fragments {2 x, 2 x + 1}
// for x < 2 and {4 + x - 2} otherwise; loaders 0 and 1 also v rows
// 32 x .. 32 x + 31 and Gamma (x = 0) or D_last (x = 1).
template <int D>
struct LoadSet {
    static constexpr int NK = D / 32;  // row loads of K per loader
    u32x4 k[NK];
    u32x4 t[2];
    u32x4 v;        // loaders 0, 1: v[32 x + lane / 2][v0 + 8 (lane % 2) .. + 7]
    float g;        // loaders 0, 1: Gamma (x = 0) or D_last (x = 1) of token lane
    uint32_t pf[2]; // L2 prefetches issued with this set, retired when it is loaded again
};

// Output-wave registers for one tile (two row blocks).
template <int D>
struct OutSet {
    u32x4 q[2][D / 32];  // q rows 16 rb + ln (fp16), dims 32 ks + 8 lg .. + 7
    u32x4 p[4];          // P fragments of the two row blocks (2 or 4 used)
};

template <int D, bool OUT_BF16, bool DRIFT, bool FUSED>
__global__ __launch_bounds__(512, 1) void gdn_seq_kernel(GdnArgs a) {
    constexpr int KS = D / 32;   // k-steps over the head dim
    constexpr int NKB = D / 16;  // 16-row blocks of S^T
    constexpr int HKS = KS / 2, HKB = NKB / 2;  // per state wave
    using SH = SeqShared<D>;
    // FUSED (calls of at most two tiles): the prep of the workgroup's own tiles
    // runs first, in two LDS blocks that alias the sequential kernel's
    constexpr int NPG = 2;  // groups of four waves forming one tile's prep each
    constexpr size_t SMEM = !FUSED ? sizeof(SH)
                            : (sizeof(SH) > NPG * sizeof(PrepLds<D>) ? sizeof(SH) : NPG * sizeof(PrepLds<D>));
    __shared__ __align__(16) char smem[SMEM];
    SH &sh = *reinterpret_cast<SH *>(smem);

    // the wave index in a scalar register: branches on it are then plain jumps
    // rather than masked code (matrix-core ops ignore the execution mask)
    const int tid = threadIdx.x, lane = tid & 63, ln = lane & 15, lg = lane >> 4;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);

    // ---- workgroup -> (stream, v-head, slice).  All workgroups that read one
    // qk-head of one stream land on the same XCD (dispatch is round-robin
    // over the 8 XCDs) so its tiles are shared through that XCD's L2.
    const int gsz = a.group * a.n_split;
    const int n_groups = a.st.B * a.H_k;
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
    const int j = qh * a.group + mem / a.n_split, sl = mem % a.n_split;
    const int v0 = 16 * sl;

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

    if constexpr (FUSED) {
        // Small call, one launch: waves 4 g .. 4 g + 3 form the prep of tile g of
        // this v-head (the same barriers in both groups; with one tile the
        // second group takes it again) and write it to the workspace as the
        // prep pass would.  Every workgroup of the v-head (and, for q, of the
        // qk-head) writes the same bytes, so it may read its own copy whoever
        // wrote last.  A workgroup-scope release / acquire then orders those
        // stores before the loads below.
        if (blockIdx.x == 0 && a.drift_zero) drift_setup(a, tid, 64 * 4 * NPG);
        PrepLds<D> *pl = reinterpret_cast<PrepLds<D> *>(smem);
        const int grp = w >> 2;
        if (n_tiles > 0) {
            const int lt = min(grp, n_tiles - 1);
            const int t0 = st + TILE * lt;
            prep_tile<D>(a, tile_base + lt, t0, min(TILE, en - t0), qh, j, 1, pl[grp], w & 3, lane, true);
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
    }

    if (w < 2) {
        // ================================================================ state
        const int hh = w;  // half of the state columns: blocks kb in [hh HKB, (hh + 1) HKB)
        // S^T block kb, lane (ln, lg), element e  =  S[v0 + ln][sigma(kb, 4 lg + e)]
        auto scol = [&](int kb, int e) { return 32 * (kb >> 1) + 8 * lg + 4 * (kb & 1) + e; };
        const size_t sbase = ((size_t)b * a.H_v + j) * D * D + (size_t)(v0 + ln) * D;
        f32x4 S[HKB], S0f[HKB];
#pragma unroll
        for (int c = 0; c < HKB; ++c) {
            const int kb = hh * HKB + c;
#pragma unroll
            for (int e = 0; e < 4; ++e) S[c][e] = a.state_in ? a.state_in[sbase + scol(kb, e)] : 0.f;
            S0f[c] = S[c];
        }
        // own half of S0 as fp16 B operand for the first tile
        auto publish = [&](int s3) __attribute__((always_inline)) {
#pragma unroll
            for (int c = 0; c < HKS; ++c)
                sh.S16[s3][hh * HKS + c][lane] = __builtin_bit_cast(u32x4, to_half8(S[2 * c], S[2 * c + 1]));
        };
        publish(0);
        int frame = frame_base;
        int frame_end = a.frame_len > 0 ? min(a.frame_len, len) : len;  // tokens done at the next frame end

        auto tile = [&](int lt, auto bufc) __attribute__((always_inline)) {
            constexpr int buf = decltype(bufc)::value;  // == lt % 2
            const int n = min(TILE, len - TILE * lt);
            lds_barrier();

            // Gamma_last S0 first: the split below may then consume S0's registers
            const int g3 = lt % 3;
            const float gl = sh.G[g3][0][63];
            f32x4 Sn[HKB];
#pragma unroll
            for (int c = 0; c < HKB; ++c)
#pragma unroll
                for (int e = 0; e < 4; ++e) Sn[c][e] = gl * S[c][e];

            // S0 as fp16 B operand, both halves (written before the barrier)
            half8 s16[KS];
#pragma unroll
            for (int c = 0; c < KS; ++c) s16[c] = as_half8(sh.S16[g3][c][lane]);

            // every operand of the tile read now, so that the reads overlap the work below
            half8 ktf[2][HKB];
            half8 tf[6];
            float4 gam4[4], dl4[4];
            v4i16 vv4[4];
            // K^T fragments by transposing reads: source lane (ln, lg) addresses token
            // 32 ks + 16 r + 4 lg + ln / 4 and dims 32 (kb / 2) + 8 (ln % 4) + 4 (kb % 2) .. + 3
#pragma unroll
            for (int ks = 0; ks < 2; ++ks)
#pragma unroll
                for (int c = 0; c < HKB; ++c) {
                    const int kb = hh * HKB + c;
                    const int r0 = 32 * ks + 4 * lg + (ln >> 2), r1 = r0 + 16;
                    const int ch = 4 * (kb >> 1) + (ln & 3), half = 4 * (kb & 1);
                    ktf[ks][c] = __builtin_bit_cast(half8, cat_u32x4(ds_read_tr16(&sh.K[buf][r0 * D + 8 * (ch ^ swz<D>(r0)) + half]),
                                                                     ds_read_tr16(&sh.K[buf][r1 * D + 8 * (ch ^ swz<D>(r1)) + half])));
                }
#pragma unroll
            for (int f = 0; f < 6; ++f) tf[f] = as_half8(sh.T[buf][f][lane]);
#pragma unroll
            for (int rb = 0; rb < 4; ++rb) {
                gam4[rb] = *(const float4 *)(&sh.G[g3][0][16 * rb + 4 * lg]);
                dl4[rb] = *(const float4 *)(&sh.G[g3][1][16 * rb + 4 * lg]);
                // v[16 rb + 4 lg + e][ln], e = 0..3, by a transposing read
                vv4[rb] = ds_read_tr16(&sh.V[buf][(16 * rb + 4 * lg + (ln >> 2)) * 16 + 4 * (ln & 3)]);
            }

            // K S0^T over all of d_k in both state waves (token rows 16 rb + 4 lg + e,
            // column v0 + ln): the same sums in the same order, so both waves hold the
            // same E, and no exchange between them inside the tile
            f32x4 ks0[4];
#pragma unroll
            for (int rb = 0; rb < 4; ++rb) ks0[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int c = 0; c < KS; ++c) {
                half8 ka[4];
#pragma unroll
                for (int rb = 0; rb < 4; ++rb) {
                    const int row = 16 * rb + ln;
                    ka[rb] = as_half8(*(const u32x4 *)(&sh.K[buf][row * D + 8 * ((4 * c + lg) ^ swz<D>(row))]));
                }
#pragma unroll
                for (int rb = 0; rb < 4; ++rb) ks0[rb] = mfma_f16(ka[rb], s16[c], ks0[rb]);
            }

            // R = V - diag(Gamma) K S0^T
            f32x4 R[4];
#pragma unroll
            for (int rb = 0; rb < 4; ++rb) {
                const float4 g4 = gam4[rb];
                R[rb][0] = bf16_to_f32((uint16_t)vv4[rb][0]) - g4.x * ks0[rb][0];
                R[rb][1] = bf16_to_f32((uint16_t)vv4[rb][1]) - g4.y * ks0[rb][1];
                R[rb][2] = bf16_to_f32((uint16_t)vv4[rb][2]) - g4.z * ks0[rb][2];
                R[rb][3] = bf16_to_f32((uint16_t)vv4[rb][3]) - g4.w * ks0[rb][3];
            }

            // E = T diag(beta) R
            const half8 rf0 = to_half8(R[0], R[1]), rf1 = to_half8(R[2], R[3]);
            f32x4 E[4];
#pragma unroll
            for (int rb = 0; rb < 4; ++rb) E[rb] = mfma_f16(tf[frag_index(rb, 0)], rf0, f32x4{0.f, 0.f, 0.f, 0.f});
#pragma unroll
            for (int rb = 2; rb < 4; ++rb) E[rb] = mfma_f16(tf[frag_index(rb, 1)], rf1, E[rb]);
            if (hh == 0) {
                sh.E[buf][0][lane] = __builtin_bit_cast(u32x4, to_half8(E[0], E[1]));
                sh.E[buf][1][lane] = __builtin_bit_cast(u32x4, to_half8(E[2], E[3]));
            }

            // D_last E as fp16 B operand
            f32x4 DE[4];
#pragma unroll
            for (int rb = 0; rb < 4; ++rb) {
                const float4 d4 = dl4[rb];
                DE[rb][0] = E[rb][0] * d4.x;
                DE[rb][1] = E[rb][1] * d4.y;
                DE[rb][2] = E[rb][2] * d4.z;
                DE[rb][3] = E[rb][3] * d4.w;
            }
            const half8 d16[2] = {to_half8(DE[0], DE[1]), to_half8(DE[2], DE[3])};

            // own half of S = Gamma_last S0 + (D_last E)^T K
#pragma unroll
            for (int ks = 0; ks < 2; ++ks)
#pragma unroll
                for (int c = 0; c < HKB; ++c) Sn[c] = mfma_f16(ktf[ks][c], d16[ks], Sn[c]);
#pragma unroll
            for (int c = 0; c < HKB; ++c) S[c] = Sn[c];
            publish((lt + 1) % 3);  // S0 of the next tile

            // frame end: per-lane drift sums of this half of the slice (a
            // loader wave reduces them over the lanes), optional snapshot
            if (DRIFT && TILE * lt + n == frame_end) {
                float num = 0.f, den = 0.f;
#pragma unroll
                for (int c = 0; c < HKB; ++c)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float dl = S[c][e] - S0f[c][e];
                        num += dl * dl;
                        den += S0f[c][e] * S0f[c][e];
                    }
                sh.DR[frame & 1][hh][lane] = float2{num, den};
                if (a.snapshots && frame < a.n_frames) {
                    float *snap = a.snapshots + ((size_t)frame * a.H_v + j) * D * D + (size_t)(v0 + ln) * D;
#pragma unroll
                    for (int c = 0; c < HKB; ++c)
#pragma unroll
                        for (int e = 0; e < 4; ++e) snap[scol(hh * HKB + c, e)] = S[c][e];
                }
#pragma unroll
                for (int c = 0; c < HKB; ++c) S0f[c] = S[c];
                ++frame;
                frame_end = min(frame_end + a.frame_len, len);
            }
        };
        for (int lt = 0; lt < n_tiles; lt += 2) {
            tile(lt, std::integral_constant<int, 0>());
            if (lt + 1 < n_tiles) tile(lt + 1, std::integral_constant<int, 1>());
        }
        if (n_tiles > 0) lds_barrier();  // the output waves' last tile
#pragma unroll
        for (int c = 0; c < HKB; ++c)
#pragma unroll
            for (int e = 0; e < 4; ++e) a.state_out[sbase + scol(hh * HKB + c, e)] = S[c][e];
    } else if (w < 4) {
        // =============================================================== output
        // O = scale diag(Gamma) Q S0^T + P E (P carries the scale) for row blocks
        // {2 PR, 2 PR + 1}, one tile behind the state waves (Gamma from the
        // loaders' LDS copy)
        auto run = [&](auto prc) __attribute__((always_inline)) {
            constexpr int PR = decltype(prc)::value;
            constexpr int NP = PR == 0 ? 2 : 4;  // P fragments of the two row blocks
            // (tiles past the end are clamped to the last one so that every
            // iteration issues the same memory operations)
            auto load = [&](OutSet<D> &s, int lt_) __attribute__((always_inline)) {
                const int lt = min(lt_, n_tiles - 1);
                const size_t tv = (size_t)(tile_base + lt) * a.H_v + j;
                // q in A-fragment order: one contiguous 1 KiB per (row block, k-step)
                const u32x4 *qb = (const u32x4 *)(a.wsQ + ((size_t)(tile_base + lt) * a.H_k + qh) * 64 * D);
#pragma unroll
                for (int r = 0; r < 2; ++r)
#pragma unroll
                    for (int ks = 0; ks < KS; ++ks) s.q[r][ks] = qb[((2 * PR + r) * KS + ks) * 64 + lane];
                const u32x4 *pb = (const u32x4 *)(a.wsP + tv * TP_HALVES);
                // fragments {0, 1} (row blocks 0, 1) or {2, 3, 4, 5} (row blocks 2, 3)
#pragma unroll
                for (int f = 0; f < NP; ++f) s.p[f] = pb[(PR == 0 ? f : 2 + f) * 64 + lane];
            };
            auto compute = [&](const OutSet<D> &s, int lt, auto bufc) __attribute__((always_inline)) {
                constexpr int buf = decltype(bufc)::value;  // == lt % 2
                const int t0 = st + TILE * lt, n = min(TILE, en - t0);
                f32x4 acc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    const half8 bs = as_half8(sh.S16[lt % 3][ks][lane]);
#pragma unroll
                    for (int r = 0; r < 2; ++r) acc[r] = mfma_f16(as_half8(s.q[r][ks]), bs, acc[r]);
                }
                // scale Gamma of each token (P carries the scale already)
#pragma unroll
                for (int r = 0; r < 2; ++r) {
                    const float4 g4 = *(const float4 *)(&sh.G[lt % 3][0][16 * (2 * PR + r) + 4 * lg]);
                    acc[r][0] *= a.scale * g4.x;
                    acc[r][1] *= a.scale * g4.y;
                    acc[r][2] *= a.scale * g4.z;
                    acc[r][3] *= a.scale * g4.w;
                }
                const half8 ef0 = as_half8(sh.E[buf][0][lane]);
                if (PR == 0) {
                    acc[0] = mfma_f16(as_half8(s.p[0]), ef0, acc[0]);
                    acc[1] = mfma_f16(as_half8(s.p[1]), ef0, acc[1]);
                } else {
                    const half8 ef1 = as_half8(sh.E[buf][1][lane]);
                    acc[0] = mfma_f16(as_half8(s.p[0]), ef0, acc[0]);
                    acc[1] = mfma_f16(as_half8(s.p[2]), ef0, acc[1]);
                    acc[0] = mfma_f16(as_half8(s.p[1]), ef1, acc[0]);
                    acc[1] = mfma_f16(as_half8(s.p[3]), ef1, acc[1]);
                }
                // o straight from the accumulators (lane (ln, lg): rows 16 r + 4 lg + e
                // of the wave's 32, column v0 + ln: the 16 lanes of a row write 32
                // contiguous bytes), through a buffer resource covering the tile's n
                // valid rows: stores past a ragged tile's end fall outside it and are
                // dropped
                constexpr int ES = OUT_BF16 ? 2 : 4;
                const uint32_t row_bytes = (uint32_t)a.H_v * D * ES;
                const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
                    (char *)a.o + (size_t)t0 * row_bytes, (short)0, (int)(row_bytes * (uint32_t)n), 0x00020000);
                const uint32_t col = (uint32_t)(j * D + v0 + ln) * ES;
#pragma unroll
                for (int r = 0; r < 2; ++r)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const uint32_t off = (uint32_t)(32 * PR + 16 * r + 4 * lg + e) * row_bytes + col;
                        if (OUT_BF16)
                            __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(unsigned short, (__bf16)acc[r][e]), rs, off, 0, 0);
                        else
                            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc[r][e]), rs, off, 0, 0);  // (a bit cast of the vector element itself compiles to element 0)
                    }
            };
            // iteration it computes tile it - 1 and then loads tile it + 1 into the
            // same register set (set (it + 1) % 2)
            auto step = [&](int it, OutSet<D> &s, auto bufc) __attribute__((always_inline)) {
                lds_barrier();
                if (it >= 1) compute(s, it - 1, bufc);
                load(s, it + 1);
            };
            if (n_tiles > 0) {
                OutSet<D> sa, sb;
                load(sa, 0);
                for (int it = 0; it <= n_tiles; it += 2) {
                    step(it, sb, std::integral_constant<int, 1>());
                    if (it + 1 <= n_tiles) step(it + 1, sa, std::integral_constant<int, 0>());
                }
            }
        };
        if (w == 2)
            run(std::integral_constant<int, 0>());
        else
            run(std::integral_constant<int, 1>());
    } else {
        // ============================================================== loaders
        // Loader X takes K rows 16 X .. 16 X + 15 of every tile; loaders 0 and 1
        // also take two T diag(beta) fragments each, 32 v rows each and Gamma /
        // D_last; loaders 2 and 3 one T fragment each.  Each role is compiled on
        // its own so that every load is issued unconditionally.
        auto run = [&](auto xc) __attribute__((always_inline)) {
            constexpr int X = decltype(xc)::value;
            constexpr int NK = LoadSet<D>::NK;
            constexpr int NT = X < 2 ? 2 : 1;                    // T diag(beta) fragments
            constexpr int T_FIRST = X < 2 ? 2 * X : 4 + (X - 2);
            // the workgroups that share a tile run in step: each starts its K rows
            // and T fragments at a different piece, so that at any moment they ask
            // L2 for different lines
            const int krot = mem % NK, trot = sl % NT;
            auto load = [&](LoadSet<D> &s, int lt_) __attribute__((always_inline)) {
                if (X < 3 && lt_ >= 2) {  // the prefetches issued with this set two tiles ago
                    l2_retire(s.pf[0]);
                    l2_retire(s.pf[1]);
                }
                const int lt = min(lt_, n_tiles - 1);  // clamped: every call issues the same loads
                const int t0 = st + TILE * lt, n = min(TILE, en - t0);
                const size_t tv = (size_t)(tile_base + lt) * a.H_v + j;
                constexpr int CH = D / 8, RPI = 64 / CH;
                const uint16_t *kb = a.k + (size_t)t0 * a.H_k * D + (size_t)qh * D + 8 * (lane % CH);
#pragma unroll
                for (int c = 0; c < NK; ++c) {
                    const uint32_t r = (uint32_t)min(16 * X + RPI * ((c + krot) % NK) + lane / CH, n - 1);
                    s.k[c] = *(const u32x4 *)(kb + r * (uint32_t)a.H_k * D);
                }
                const u32x4 *tb = (const u32x4 *)(a.wsT + tv * TP_HALVES);
#pragma unroll
                for (int c = 0; c < NT; ++c) s.t[c] = tb[(T_FIRST + (c + trot) % NT) * 64 + lane];
                if (X < 2) {
                    // v rows 32 X + lane / 2, columns v0 + 8 (lane % 2) .. + 7
                    const uint16_t *vb = a.v + ((size_t)t0 * a.H_v + j) * D + v0 + 8 * (lane & 1);
                    s.v = *(const u32x4 *)(vb + (uint32_t)min(32 * X + (lane >> 1), n - 1) * (uint32_t)a.H_v * D);
                    s.g = a.wsGam[tv * 128 + 64 * X + lane];
                }
                // L2 prefetch of tile lt_ + 2 (five tiles ahead of the state
                // waves): the workgroups that share a tile run in step, so
                // without it all of them wait on the first one's miss to HBM.
                // Each takes a 1 KiB piece: of the qk-head's K rows and q tile
                // (piece mem), of its v-head's T and P fragments (piece sl) and
                // v rows (pieces 2 sl, 2 sl + 1).  (A direct-to-LDS load would
                // need no register, but the compiler then waits for it before
                // every LDS access.)
                if (X < 3) {
                    constexpr int CHP = D / 8;  // 16-byte chunks per row
                    const int lp = min(lt_ + 2, n_tiles - 1);
                    const int tp0 = st + TILE * lp, np = min(TILE, en - tp0);
                    const size_t tvp = (size_t)(tile_base + lp) * a.H_v + j;
                    // (unconditional, with clamped pieces: a load issued on some
                    // paths only makes the compiler wait for every load later)
                    if (X == 0) {
                        const int idx = 64 * (mem % CHP) + lane, r = min(idx / CHP, np - 1);
                        s.pf[0] = l2_prefetch(a.k + ((size_t)(tp0 + r) * a.H_k + qh) * D + 8 * (idx % CHP));
                        s.pf[1] = l2_prefetch(a.wsQ + ((size_t)(tile_base + lp) * a.H_k + qh) * 64 * D + 8 * idx);
                    }
                    if (X == 1) {
                        s.pf[0] = l2_prefetch(a.wsT + tvp * TP_HALVES + 8 * (64 * min(sl, 5) + lane));
                        s.pf[1] = l2_prefetch(a.wsP + tvp * TP_HALVES + 8 * (64 * min(sl, 5) + lane));
                    }
                    if (X == 2) {
#pragma unroll
                        for (int i = 0; i < 2; ++i) {
                            const int idx = 64 * (2 * sl + i) + lane, r = min(idx / CHP, np - 1);
                            s.pf[i] = l2_prefetch(a.v + ((size_t)(tp0 + r) * a.H_v + j) * D + 8 * (idx % CHP));
                        }
                    }
                }
            };
            auto stage = [&](const LoadSet<D> &s, auto bufc, int g3) __attribute__((always_inline)) {
                constexpr int buf = decltype(bufc)::value;
                constexpr int CH = D / 8, RPI = 64 / CH;
#pragma unroll
                for (int c = 0; c < NK; ++c) {
                    const int row = 16 * X + RPI * ((c + krot) % NK) + lane / CH, ch = lane % CH;
                    *(u32x4 *)(&sh.K[buf][row * D + 8 * (ch ^ swz<D>(row))]) = __builtin_bit_cast(u32x4, bf16x8_to_f16(s.k[c]));
                }
#pragma unroll
                for (int c = 0; c < NT; ++c) sh.T[buf][T_FIRST + (c + trot) % NT][lane] = s.t[c];
                if constexpr (X < 2) {
                    *(u32x4 *)(&sh.V[buf][(32 * X + (lane >> 1)) * 16 + 8 * (lane & 1)]) = s.v;
                    sh.G[g3][X][lane] = s.g;
                }
            };
            // drift sums: the state waves leave per-lane sums of a frame ending in
            // tile t in LDS; loader 3 reduces them after the next barrier (the
            // buffer of that frame's parity is written again two frames later,
            // after a barrier this wave only reaches once it is done reading)
            int frame = frame_base;
            int frame_end = a.frame_len > 0 ? min(a.frame_len, len) : len;
            auto drift_reduce = [&](int it) __attribute__((always_inline)) {
                if (!DRIFT || X != 3 || it < 1) return;
                const int lt = it - 1;
                if (TILE * lt + min(TILE, len - TILE * lt) != frame_end) return;
                if (a.wsDrift && frame < a.n_frames) {
                    const float2 p0 = sh.DR[frame & 1][0][lane], p1 = sh.DR[frame & 1][1][lane];
                    const float num = wave_sum(p0.x + p1.x), den = wave_sum(p0.y + p1.y);
                    if (lane == 0) store_pair_coherent(a.wsDrift + (((size_t)frame * a.H_v + j) * a.n_split + sl) * 2, num, den);
                }
                ++frame;
                frame_end = min(frame_end + a.frame_len, len);
            };
            // write signal: ||E row||^2 over the slice's 16 columns for every token
            // of tile it - 1, from the E the state waves left in LDS (valid until
            // they write that buffer again in tile it + 1): loader 2 takes the
            // tokens of k-step 0, loader 3 those of k-step 1 (loaders have slack at
            // the barrier; on the output waves this cost every tile of the chain)
            auto write_norms = [&](int it) __attribute__((always_inline)) {
                if (X < 2 || it < 1 || !a.wsWrite) return;
                constexpr int ks = X - 2;
                const int lt = it - 1;
                const int t0 = st + TILE * lt, n = min(TILE, en - t0);
                float *wb = a.wsWrite + ((size_t)j * a.n_split + sl) * a.st.T + t0;
                const float wsum = row_sq_sum16(as_half8(sh.E[lt & 1][ks][lane]), ln);
                const int i = ln >> 1, tok = 32 * ks + 16 * (i >> 2) + 4 * lg + (i & 3);
                if ((ln & 1) == 0 && tok < n) wb[tok] = wsum;
            };
            // tile t lives in register set t % 2 and LDS buffer t % 2.  Iteration it
            // stages tile it + 1 and then loads tile it + 3 into the set just freed.
            if (n_tiles > 0) {
                LoadSet<D> s0, s1;
                load(s0, 0);
                load(s1, 1);
                stage(s0, std::integral_constant<int, 0>(), 0);
                load(s0, 2);
                auto step = [&](int it, LoadSet<D> &s, auto bufc) __attribute__((always_inline)) {
                    lds_barrier();
                    if (it + 1 < n_tiles) stage(s, bufc, (it + 1) % 3);
                    load(s, it + 3);
                    drift_reduce(it);
                    write_norms(it);
                };
                for (int it = 0; it <= n_tiles; it += 2) {
                    step(it, s1, std::integral_constant<int, 1>());
                    if (it + 1 <= n_tiles) step(it + 1, s0, std::integral_constant<int, 0>());
                }
            }
            // the last of the stream's n_split workgroups of v-head j to finish
            // sums the slices of every frame of the stream (fixed order)
            if (DRIFT && X == 3 && a.drift_out) {
                wait_vmem_all();  // this wave's pairs (the only ones of the workgroup) are coherent before the count
                unsigned prev = 0;
                if (lane == 0)
                    prev = __hip_atomic_fetch_add(&a.drift_cnt[b * a.H_v + j], 1u, __ATOMIC_RELAXED,
                                                  __HIP_MEMORY_SCOPE_AGENT);
                prev = __builtin_amdgcn_readfirstlane(prev);
                if (prev == (unsigned)a.n_split - 1u) {
                    // the count has returned: every slice's pairs are readable at the point of coherence
                    const int nf = min(frames_in(len, a.frame_len), a.n_frames - frame_base);
                    for (int f = lane; f < nf; f += 64) {
                        const size_t fj = (size_t)(frame_base + f) * a.H_v + j;
                        // every slice's pair loaded before the sum (n_split <= 8):
                        // one round trip to memory instead of n_split
                        float2 pr[8];
#pragma unroll
                        for (int s = 0; s < 8; ++s)
                            pr[s] = s < a.n_split ? load_pair_coherent(a.wsDrift + (fj * a.n_split + s) * 2) : float2{0.f, 0.f};
                        float num = 0.f, den = 0.f;
#pragma unroll
                        for (int s = 0; s < 8; ++s) {
                            num += pr[s].x;
                            den += pr[s].y;
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

// Sum of the drift sums of every slice (fixed order) -> [n_frames][H_v][2].
// Entries past the real frame count are zeroed.
__global__ __launch_bounds__(256) void gdn_drift_finalize_kernel(const float *ws, float *out, int n_frames,
                                                                  int H_v, int n_split, Streams st,
                                                                  int frame_len) {
    const int idx = blockIdx.x * 256 + threadIdx.x;
    if (idx >= n_frames * H_v) return;
    int real = 0;
    for_streams(st, [&](int, int s0, int e0) {
        real += frames_in(e0 - s0, frame_len);
        return false;
    });
    const int f = idx / H_v;
    float num = 0.f, den = 0.f;
    if (f < real) {
        for (int s = 0; s < n_split; ++s) {
            num += ws[((size_t)idx * n_split + s) * 2];
            den += ws[((size_t)idx * n_split + s) * 2 + 1];
        }
    }
    out[(size_t)idx * 2] = num;
    out[(size_t)idx * 2 + 1] = den;
}

// Write-magnitude signal per (frame, v-head): the sum over the frame's tokens
// of sqrt(sum over slices of ||E row||^2) and the token count -> [n_frames][H_v][2].
// One workgroup per (frame, v-head); thread i takes tokens i, i + 256, ... of
// the frame (the slices of one token sit T_total apart, so adjacent lanes read
// adjacent words), then a fixed-order tree over the threads.  Frames past the
// real count are zeroed.
__global__ __launch_bounds__(256) void gdn_write_finalize_kernel(const float *ws, float *out, int n_frames, int H_v,
                                                                  int n_split, Streams st, int frame_len) {
    const int f = blockIdx.x, j = blockIdx.y, tid = threadIdx.x;
    int base = 0, tb = 0, te = 0;
    for_streams(st, [&](int, int s0, int e0) {
        const int nf = frames_in(e0 - s0, frame_len);
        if (f < base + nf) {
            const int lf = f - base;
            tb = s0 + (frame_len > 0 ? lf * frame_len : 0);
            te = frame_len > 0 ? min(tb + frame_len, e0) : e0;
            return true;
        }
        base += nf;
        return false;
    });
    // fp32 throughout (a frame's sum of at most a few thousand norms); the
    // slices of a token are loaded together (n_split <= 8 for d <= 128)
    float acc = 0.f;
    const float *wj = ws + (size_t)j * n_split * st.T;
    for (int t = tb + tid; t < te; t += 256) {
        float v[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) v[q] = q < n_split ? wj[(size_t)q * st.T + t] : 0.f;
        float s = 0.f;
#pragma unroll
        for (int q = 0; q < 8; ++q) s += v[q];
        acc += __builtin_sqrtf(s);
    }
    __shared__ float red[256];
    red[tid] = acc;
    __syncthreads();
    for (int off = 128; off > 0; off >>= 1) {
        if (tid < off) red[tid] += red[tid + off];
        __syncthreads();
    }
    if (tid == 0) {
        out[((size_t)f * H_v + j) * 2] = red[0];
        out[((size_t)f * H_v + j) * 2 + 1] = (float)(te - tb);
    }
}

// ============================================================================
// host side
// ============================================================================
static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// The sequential part runs one workgroup per (stream, v-head) (gdn_wide.hip)
// when there are enough heads to fill the GPU that way; otherwise one
// workgroup per 16-row slice of a head (8 per head at d = 128), which is what
// fills it for a single stream.
constexpr int WIDE_MIN_HEADS = 256;
static bool use_wide(int B, int H_v, int d) { return d == 128 && (long long)B * H_v >= WIDE_MIN_HEADS; }

// compute units of the current device (looked up once per device)
static int device_cus() {
    static int cus[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
    if (cus[dev] == 0) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
        cus[dev] = n;
    }
    return cus[dev];
}

GdnWorkspace gdn_workspace_layout(int B, int T_total, int H_k, int H_v, int d, int n_frames, bool with_write) {
    GdnWorkspace w{};
    w.tiles_max = (int)(((long long)T_total + 63LL * B) / 64);
    w.n_split = d / 16;
    size_t off = 0;
    w.offT = off;
    off = align256(off + (size_t)w.tiles_max * H_v * TP_HALVES * sizeof(_Float16));
    w.offP = off;
    off = align256(off + (size_t)w.tiles_max * H_v * TP_HALVES * sizeof(_Float16));
    w.offQ = off;  // fp16 q fragments, only for the per-slice kernel
    if (!use_wide(B, H_v, d)) off = align256(off + (size_t)w.tiles_max * H_k * 64 * d * sizeof(_Float16));
    w.offGam = off;
    off = align256(off + (size_t)w.tiles_max * H_v * 128 * sizeof(float));
    w.offDrift = off;
    off = align256(off + (size_t)n_frames * H_v * w.n_split * 2 * sizeof(float));
    w.offWrite = off;  // per-token norm slices, reserved only for calls that ask for the write signal
    if (with_write) off = align256(off + (size_t)T_total * H_v * w.n_split * sizeof(float));
    w.offCnt = off;
    off = align256(off + (size_t)B * H_v * sizeof(unsigned));
    w.offStart = off;  // frame-start states of the whole-head kernel
    if (use_wide(B, H_v, d)) off = align256(off + (size_t)B * H_v * d * d * sizeof(float));
    w.total = off;
    return w;
}

template <int D>
static hipError_t launch_d(const GdnLaunch &p, hipStream_t stream) {
    GdnArgs a;
    a.q = p.q;
    a.k = p.k;
    a.v = p.v;
    a.g = p.g;
    a.beta = p.beta;
    a.st = Streams{p.cu_seqlens, p.B, p.T_total};
    a.H_k = p.H_k;
    a.H_v = p.H_v;
    a.group = p.H_v / p.H_k;
    a.frame_len = p.frame_len;
    a.n_frames = p.n_frames;
    a.state_in = p.state_in;
    a.state_out = p.state_out;
    a.o = p.o;
    a.scale = p.scale;
    a.snapshots = p.snapshots;
    a.wsT = p.wsT;
    a.wsP = p.wsP;
    a.wsQ = use_wide(p.B, p.H_v, D) ? nullptr : p.wsQ;
    a.wsGam = p.wsGam;
    a.wsWrite = p.write_partials ? p.wsWrite : nullptr;
    a.wsStart = p.wsStart;
    a.n_split = p.n_split;
    // Per-slice pairs go straight to the caller's buffer.  Per-head pairs are
    // the sums of the slices, added by the sequential kernel itself (the last
    // workgroup of each stream and v-head to finish), so the drift costs no
    // launch of its own; only a call without tokens (no prep pass clears the
    // counters) leaves the zeros to the finalize pass
    const bool fused_drift = p.drift_partials && !p.drift_slices && p.n_frames > 0 && p.tiles_max > 0;
    a.wsDrift = !p.drift_partials ? nullptr : p.drift_slices ? p.drift_partials : p.wsDrift;
    a.drift_out = fused_drift ? p.drift_partials : nullptr;
    a.drift_cnt = p.wsCnt;
    a.drift_zero = p.n_frames > 0 ? p.drift_partials : nullptr;
    a.drift_zero_per_frame = p.drift_slices ? p.H_v * p.n_split : p.H_v;

    // one prep workgroup per (tile, v-head) whenever all of them are resident at
    // once (four per CU): a workgroup then inverts one v-head's system instead
    // of the group's in turn, at the price of a second Gram product per tile
    // (1024-token calls: 13.4 -> see the kernel trace; one streamed chunk:
    // 11.2 -> 8.6 us).  Longer calls share the Gram products of a qk-head.
    a.prep_per_vhead = a.group > 1 && (long long)p.tiles_max * p.H_v <= 1024;
    // calls of at most two tiles on the per-slice kernel (most streamed chunks)
    // form their prep inside it: one launch per layer, 16.1 instead of 18.4 us
    // a layer at 24 layers x 128 tokens.  (With three tiles a second prep round,
    // or a third group of waves, costs what the launch saves.)  Not with the
    // per-head drift sums, whose slice counters the prep pass clears before any
    // sequential workgroup runs.
    const bool one_launch = !use_wide(p.B, p.H_v, D) && p.tiles_max > 0 && p.tiles_max <= 2 && !fused_drift;
    if (p.tiles_max > 0 && !one_launch) {
        // tiles rounded up to a multiple of 8 (workgroups past the last tile exit)
        const long long n_prep = (long long)((p.tiles_max + 7) / 8) * 8 * (a.prep_per_vhead ? p.H_v : p.H_k);
        // the whole-head kernel forms P itself (prep without q, K Q^T and P)
        if (D == 128 && use_wide(p.B, p.H_v, D))
            hipLaunchKernelGGL((gdn_prep_kernel<D, false>), dim3((unsigned)n_prep), dim3(256), 0, stream, a);
        else
            hipLaunchKernelGGL((gdn_prep_kernel<D, true>), dim3((unsigned)n_prep), dim3(256), 0, stream, a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    // the frame-end work is compiled out when neither drift sums nor snapshots are asked for
    const bool drift = p.drift_partials || p.snapshots;
    if (D == 128 && use_wide(p.B, p.H_v, D)) {
        // whole heads: per-head drift pairs are added by the workgroup itself
        // the tail of the longest streams as half heads when at most as many
        // streams as fill the GPU that way are left
        hipError_t e = launch_gdn_wide(a, p.B * p.H_v, device_cus() / (2 * p.H_v), p.o_bf16, drift, stream);
        if (e != hipSuccess) return e;
        if (p.write_partials && p.n_frames > 0) {
            hipLaunchKernelGGL(gdn_write_finalize_kernel, dim3(p.n_frames, p.H_v), dim3(256), 0, stream, p.wsWrite,
                               p.write_partials, p.n_frames, p.H_v, p.n_split, a.st, p.frame_len);
            e = hipGetLastError();
        }
        return e;
    }
    const int n_wg = p.B * p.H_v * p.n_split;
    auto seq = [&](auto fc) {
        constexpr bool F = decltype(fc)::value;
        const int nt = 512;
        if (p.o_bf16) {
            if (drift)
                hipLaunchKernelGGL((gdn_seq_kernel<D, true, true, F>), dim3(n_wg), dim3(nt), 0, stream, a);
            else
                hipLaunchKernelGGL((gdn_seq_kernel<D, true, false, F>), dim3(n_wg), dim3(nt), 0, stream, a);
        } else {
            if (drift)
                hipLaunchKernelGGL((gdn_seq_kernel<D, false, true, F>), dim3(n_wg), dim3(nt), 0, stream, a);
            else
                hipLaunchKernelGGL((gdn_seq_kernel<D, false, false, F>), dim3(n_wg), dim3(nt), 0, stream, a);
        }
    };
    if (one_launch)
        seq(std::true_type());
    else
        seq(std::false_type());
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (p.drift_partials && p.n_frames > 0 && p.tiles_max == 0) {
        // no tokens: every frame's pairs are zero (the pass reads nothing when
        // no frame is real; per-slice pairs are passed as n_split-times more
        // heads of one slice each)
        const int heads = p.drift_slices ? p.H_v * p.n_split : p.H_v;
        const int n = p.n_frames * heads;
        hipLaunchKernelGGL(gdn_drift_finalize_kernel, dim3((n + 255) / 256), dim3(256), 0, stream, p.wsDrift,
                           p.drift_partials, p.n_frames, heads, 1, a.st, p.frame_len);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (p.write_partials && p.n_frames > 0) {
        hipLaunchKernelGGL(gdn_write_finalize_kernel, dim3(p.n_frames, p.H_v), dim3(256), 0, stream, p.wsWrite,
                           p.write_partials, p.n_frames, p.H_v, p.n_split, a.st, p.frame_len);
        e = hipGetLastError();
    }
    return e;
}

hipError_t launch_gdn(const GdnLaunch &p, hipStream_t stream) {
    if (p.d == 128) return launch_d<128>(p, stream);
    return launch_d<64>(p, stream);
}

}  // namespace ds
