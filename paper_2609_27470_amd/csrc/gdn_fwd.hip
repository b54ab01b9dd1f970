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
//             as fp16 T diag(beta) and P = D (.) tril(Q K^T), plus gamma;
//   gdn_seq   (one workgroup per (stream, v-head, 16 rows of S)): walks the
//             tiles in order, keeps its rows of S in fp32 registers, does the
//             state-dependent products on fp16 matrix cores, writes o, and at
//             every frame end the drift sums of Eq. 3 for its rows.
//   gdn_drift_finalize sums the partial drift sums in a fixed order.
#include "common.h"
#include "kernels.h"

namespace ds {

constexpr int TILE = 64;

// T diag(beta) and P are stored per (tile, v-head) as the six non-zero
// 16 x 32 A-fragments of v_mfma_f32_16x16x32_f16 (row block w = 0..3,
// k-step ks <= w / 2), 64 lanes x 8 halves each, lane l holding row
// 16 w + l % 16, columns 32 ks + 8 (l / 16) .. + 7.
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
    float *wsGam, *wsDrift;
    int n_split;
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

// ============================================================================
// gdn_prep: one workgroup per (tile, v-head).  Every global load is issued
// up front; K K^T and Q K^T run on bf16 matrix cores (fragments straight from
// global memory, exact bf16 inputs, fp32 accumulation); the inverse of the
// unit lower-triangular I + A is blocked in 16 x 16 blocks: the diagonal
// blocks by forward substitution, the off-diagonal ones on fp32 matrix cores,
// T_ij = -T_ii sum_{k=j}^{i-1} A_ik T_kj, by distance from the diagonal.
// ============================================================================
__device__ __forceinline__ f32x4 mfma_f32_16x16x4(float a, float b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

template <int D>
__global__ __launch_bounds__(256) void gdn_prep_kernel(GdnArgs a) {
    constexpr int KS = D / 32;   // 32-wide k-steps over the head dim
    constexpr int ALD = 65;      // floats per LDS row of A and T
    constexpr int PLD = 72;      // halves per LDS row of P
    __shared__ float As[64 * ALD];
    __shared__ float Ts[64 * ALD];
    __shared__ float Ys[4][256];
    __shared__ __align__(16) _Float16 Ps[64 * PLD];
    __shared__ float gam_s[64], beta_s[64];

    const int ti = blockIdx.x, j = blockIdx.y;
    const int h = j / a.group;
    int t0 = 0, n = 0;
    if (!locate_tile(a.st, ti, t0, n)) return;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, ln = lane & 15, lg = lane >> 4;
    const size_t tv = (size_t)ti * a.H_v + j;
    const uint4 zero4 = make_uint4(0, 0, 0, 0);

    // ---- loads: k rows of every 16-row block up to w, q rows of block w, gates
    uint4 kf[4][KS], ka[KS], qa[KS];
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
        const int r = 16 * nb + ln;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            kf[nb][ks] = zero4;
            if (nb <= w && r < n) kf[nb][ks] = *(const uint4 *)(a.k + ((size_t)(t0 + r) * a.H_k + h) * D + 32 * ks + 8 * lg);
        }
    }
    {
        const int r = 16 * w + ln;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const size_t off = ((size_t)(t0 + r) * a.H_k + h) * D + 32 * ks + 8 * lg;
            qa[ks] = (r < n) ? *(const uint4 *)(a.q + off) : zero4;
            ka[ks] = (r < n) ? *(const uint4 *)(a.k + off) : zero4;
        }
    }
    float gv = 0.f, bv = 0.f;
    if (w == 0 && lane < n) {
        gv = a.g[(size_t)(t0 + lane) * a.H_v + j];
        bv = a.beta[(size_t)(t0 + lane) * a.H_v + j];
    }

    // ---- gamma = inclusive prefix sum of g, in base-2 units
    if (w == 0) {
        float s = gv;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const float y = __shfl_up(s, off, 64);
            if (lane >= off) s += y;
        }
        s *= 1.4426950408889634f;  // exp(gamma) = exp2(s)
        gam_s[lane] = s;
        beta_s[lane] = bv;
        a.wsGam[tv * 64 + lane] = s;
    }

    // ---- Gram blocks of row block w: K K^T and Q K^T for column blocks nb <= w
    f32x4 gk[4], gq[4];
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
        gk[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
        gq[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (nb <= w) {
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                gk[nb] = mfma_bf16(as_bf16x8(ka[ks]), as_bf16x8(kf[nb][ks]), gk[nb]);
                gq[nb] = mfma_bf16(as_bf16x8(qa[ks]), as_bf16x8(kf[nb][ks]), gq[nb]);
            }
        }
    }
    __syncthreads();

    // ---- A (strictly lower) and P (lower incl. diagonal), rows of block w
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int r = 16 * w + 4 * lg + e, i = 16 * nb + ln;
            float av = 0.f, pv = 0.f;
            if (nb <= w && i <= r) {
                const float dri = exp2f(gam_s[r] - gam_s[i]);
                pv = dri * gq[nb][e];
                if (i < r) av = beta_s[r] * dri * gk[nb][e];
            }
            As[r * ALD + i] = av;
            Ps[r * PLD + i] = (_Float16)pv;
        }
    }
    __syncthreads();

    // ---- diagonal blocks (lane = 16 * block + column)
    if (w == 0) {
        const int o = 16 * (lane >> 4), c = lane & 15;
        float x[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            float s = (r == c) ? 1.f : 0.f;
#pragma unroll
            for (int i = 0; i < r; ++i) s -= As[(o + r) * ALD + o + i] * x[i];
            x[r] = s;
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) Ts[(o + r) * ALD + o + c] = x[r];
    } else {
        // P (fp16) -> workspace in fragment order, 16 B per lane
        for (int c = tid - 64; c < 6 * 64; c += 192) {
            const int f = c >> 6, l = c & 63;
            const int fw = f < 2 ? f : 2 + ((f - 2) >> 1), fks = f < 2 ? 0 : ((f - 2) & 1);
            const int r = 16 * fw + (l & 15), c8 = 32 * fks + 8 * (l >> 4);
            *(uint4 *)(a.wsP + tv * TP_HALVES + f * FRAG_HALVES + l * 8) = *(const uint4 *)(&Ps[r * PLD + c8]);
        }
    }
    __syncthreads();

    // ---- off-diagonal blocks.  16x16x4 fp32 fragments: A lane = [ln][lg],
    // B lane = [lg][ln], C lane = [4 lg + e][ln].
    for (int d = 1; d <= 3; ++d) {
        const int p = w;  // pair handled by this wave: block row bi = p + d, column bj = p
        if (p + d <= 3) {
            const int bi = p + d, bj = p;
            f32x4 y = {0.f, 0.f, 0.f, 0.f};
            for (int kb = bj; kb < bi; ++kb) {
#pragma unroll
                for (int s = 0; s < 4; ++s) {
                    const float av = As[(16 * bi + ln) * ALD + 16 * kb + 4 * s + lg];
                    const float tb = Ts[(16 * kb + 4 * s + lg) * ALD + 16 * bj + ln];
                    y = mfma_f32_16x16x4(av, tb, y);
                }
            }
            float *yw = Ys[w];
#pragma unroll
            for (int e = 0; e < 4; ++e) yw[(4 * lg + e) * 16 + ln] = y[e];
            __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's Y is in LDS
            f32x4 t = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const float ta = Ts[(16 * bi + ln) * ALD + 16 * bi + 4 * s + lg];
                const float yb = yw[(4 * s + lg) * 16 + ln];
                t = mfma_f32_16x16x4(ta, yb, t);
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) Ts[(16 * bi + 4 * lg + e) * ALD + 16 * bj + ln] = -t[e];
        }
        __syncthreads();
    }

    // ---- T diag(beta) (fp16, zero above the diagonal) in fragment order
    for (int c = tid; c < 6 * 64; c += 256) {
        const int f = c >> 6, l = c & 63;
        const int fw = f < 2 ? f : 2 + ((f - 2) >> 1), fks = f < 2 ? 0 : ((f - 2) & 1);
        const int r = 16 * fw + (l & 15), c8 = 32 * fks + 8 * (l >> 4);
        half8 tv8;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int i = c8 + e;
            tv8[e] = (_Float16)((i <= r) ? Ts[r * ALD + i] * beta_s[i] : 0.f);
        }
        *(uint4 *)(a.wsT + tv * TP_HALVES + f * FRAG_HALVES + l * 8) = as_uint4(tv8);
    }
}

// ============================================================================
// gdn_seq: one workgroup of 8 waves per (stream, v-head, 16 consecutive rows
// of S).  Waves 0-3 ("state waves") carry the recurrence: wave w owns state
// columns [w D/4, (w+1) D/4) of the 16 rows and, per tile, computes the rows
// 16 w .. 16 w + 15 of K S0^T, the residual and the writes E, and its block
// of the state update.  Waves 4-7 ("helper waves", helper h = w - 4 shares a
// SIMD with state wave h) do everything off that chain: they load the
// operands two tiles ahead, stage K, T diag(beta), v and gamma of the next
// tile in LDS, compute Q S0^T and the outputs O = diag(Gamma) Q S0^T + P E,
// and store o.  All 8 waves meet at the same 3 barriers per tile.
//
// Precision: k and q stay bf16 (as given) and meet the fp32 state through
// bf16 matrix-core products against a two-term bf16 split of the state
// (S ~ S_hi + S_lo, relative error ~2^-17); the writes D_last E enter the
// state update the same way.  The tile-local operands (R, E, T diag(beta),
// P) are fp16.  All accumulation is fp32.  K and the state are staged
// row-major and read as transposed fragments with ds_read_b64_tr_b16.
// ============================================================================
template <int D>
struct SeqTile {
    u32x4 k[D / 32], q[D / 32];  // bf16 rows 16 h + ln of k and q (8 dims per k-step)
    u32x4 t[2], p[2];            // fp16 T diag(beta), P fragments of rows 16 h + ln
    float4 gam;                  // gamma (base-2 units) of rows 16 h + 4 lg + e
    float gam_last;
    uint32_t v[4];               // bf16 v of rows 16 h + 4 lg + e, column v0 + ln
};

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;

// Transposed 16-bit fragment read: within each group of 16 lanes, lane l
// receives element (l % 4) of the 4 elements addressed by lanes l/4 + 4 e.
__device__ __forceinline__ v4i16 ds_read_tr16(const void *p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16 *)p);
}
__device__ __forceinline__ bf16x8 cat_bf16(v4i16 a, v4i16 b) {
    return __builtin_bit_cast(bf16x8, __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7));
}

// Operands of one tile for row block h (rows 16 h ..).  Rows past the end of
// a ragged tile are clamped to its last row: their products only meet zero
// entries of T diag(beta) and P (beta = 0 and k = 0 there in the prep kernel)
// and their outputs are never stored.
template <int D>
__device__ __forceinline__ void seq_load(const GdnArgs &a, SeqTile<D> &s, int t0, int n, size_t tv, int qh,
                                         int j, int v0, int h, int ln, int lg) {
    const uint16_t *kb = a.k + (size_t)t0 * a.H_k * D;
    const uint16_t *qb = a.q + (size_t)t0 * a.H_k * D;
    const uint32_t ra = (uint32_t)min(16 * h + ln, n - 1);
    const uint32_t off = (ra * (uint32_t)a.H_k + (uint32_t)qh) * D + 8 * lg;
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
        s.k[ks] = *(const u32x4 *)(kb + off + 32 * ks);
        s.q[ks] = *(const u32x4 *)(qb + off + 32 * ks);
    }
    const uint16_t *vb = a.v + (size_t)t0 * a.H_v * D + (size_t)j * D + v0 + ln;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const uint32_t r = (uint32_t)min(16 * h + 4 * lg + e, n - 1);
        s.v[e] = vb[r * (uint32_t)a.H_v * D];
    }
    const float *gb = a.wsGam + tv * 64;
    s.gam = *(const float4 *)(gb + 16 * h + 4 * lg);
    s.gam_last = gb[63];
    const _Float16 *tb = a.wsT + tv * TP_HALVES, *pb = a.wsP + tv * TP_HALVES;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
        // row blocks 0 and 1 have a single k-step; their second load repeats the first
        const int f = frag_index(h, (h >= 2) ? ks : 0);
        s.t[ks] = *(const u32x4 *)(tb + f * FRAG_HALVES + 8 * (ln + 16 * lg));
        s.p[ks] = *(const u32x4 *)(pb + f * FRAG_HALVES + 8 * (ln + 16 * lg));
    }
}

// fp32 pair -> bf16 pair (round to nearest even), packed in one dword
__device__ __forceinline__ uint32_t bf16_pack(float x, float y) {
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    bf16x2 r = {(__bf16)x, (__bf16)y};
    return __builtin_bit_cast(uint32_t, r);
}
__device__ __forceinline__ float bf16_lo_f(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi_f(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Inclusive prefix sum within each row of 16 lanes (DPP row shifts); lane 15
// of a row ends with the row's total.
__device__ __forceinline__ float row16_sum(float x) {
    x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x111, 0xF, 0xF, true));
    x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x112, 0xF, 0xF, true));
    x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x114, 0xF, 0xF, true));
    x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x118, 0xF, 0xF, true));
    return x;
}

template <int D>
struct SeqShared {
    static constexpr int KLD = D + 8;  // bf16 per LDS row of the K tile
    static constexpr int SLD = 20;     // bf16 per LDS row of S^T (16 rows of S + pad)
    static constexpr int TLD = 72;     // 16-bit elements per LDS row of R^T, E^T, (D E)^T
    uint16_t Ks[2][64 * KLD];          // K tile of the tile (row-major, bf16)
    u32x4 Tst[2][4][2][64];            // T diag(beta) fragments per state wave and lane
    uint2 Vst[2][4][64];               // v (4 bf16) per state wave and lane
    float4 Gst[2][4][64];              // gamma of the lane's 4 rows
    float Glast[2];                    // gamma of the tile's last row
    uint16_t SThi[2][D * SLD];         // S^T, high bf16 term
    uint16_t STlo[2][D * SLD];         // S^T, low bf16 term
    _Float16 RT[2][16 * TLD];          // R^T
    _Float16 ET[2][16 * TLD];          // E^T
    uint16_t DThi[2][16 * TLD];        // (D_last E)^T, high bf16 term
    uint16_t DTlo[2][16 * TLD];        // (D_last E)^T, low bf16 term
};

template <int D, bool OUT_BF16, bool DRIFT>
__global__ __launch_bounds__(512, 1) void gdn_seq_kernel(GdnArgs a) {
    constexpr int KS = D / 32;
    constexpr int NB = D / 64;  // 16-column state blocks per state wave
    using SH = SeqShared<D>;
    constexpr int KLD = SH::KLD, SLD = SH::SLD, TLD = SH::TLD;
    __shared__ __align__(16) SH sh;

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, ln = lane & 15, lg = lane >> 4;
    const bool state_wave = w < 4;
    const int h = w & 3;  // row block (and state column block) of this wave

    // ---- workgroup -> (stream, v-head, slice).  All workgroups that read one
    // qk-head of one stream land on the same XCD (dispatch is round-robin
    // over the 8 XCDs) so its q/k tiles are shared through that XCD's L2.
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
    const int trow = ln >> 2, tcol = 4 * (ln & 3);  // source element of a transposed read

    // ---- state (state waves): rows v0 + 4 lg + e, columns h D/4 + 16 nb + ln
    const size_t sbase = ((size_t)b * a.H_v + j) * D * D;
    f32x4 S[NB], S_start[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int vr = v0 + 4 * lg + e, c = h * (D / 4) + 16 * nb + ln;
            S[nb][e] = (state_wave && a.state_in) ? a.state_in[sbase + (size_t)vr * D + c] : 0.f;
        }
        S_start[nb] = S[nb];
    }
    int frame = frame_base;

    // S split in two bf16 terms -> S^T buffer `buf`
    auto write_state = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            const uint32_t h01 = bf16_pack(S[nb][0], S[nb][1]), h23 = bf16_pack(S[nb][2], S[nb][3]);
            const uint32_t l01 = bf16_pack(S[nb][0] - bf16_lo_f(h01), S[nb][1] - bf16_hi_f(h01));
            const uint32_t l23 = bf16_pack(S[nb][2] - bf16_lo_f(h23), S[nb][3] - bf16_hi_f(h23));
            const int off = (h * (D / 4) + 16 * nb + ln) * SLD + 4 * lg;
            *(uint2 *)(&sh.SThi[buf][off]) = make_uint2(h01, h23);
            *(uint2 *)(&sh.STlo[buf][off]) = make_uint2(l01, l23);
        }
    };
    // helper: stage tile data of row block h into buffer `buf`
    auto stage = [&](const SeqTile<D> &s, int buf) __attribute__((always_inline)) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) *(u32x4 *)(&sh.Ks[buf][(16 * h + ln) * KLD + 32 * ks + 8 * lg]) = s.k[ks];
        sh.Tst[buf][h][0][lane] = s.t[0];
        sh.Tst[buf][h][1][lane] = s.t[1];
        sh.Vst[buf][h][lane] = make_uint2(s.v[0] | (s.v[1] << 16), s.v[2] | (s.v[3] << 16));
        sh.Gst[buf][h][lane] = s.gam;
        if (h == 0 && lane == 0) sh.Glast[buf] = s.gam_last;
    };
    auto load_tile = [&](SeqTile<D> &s, int lt) __attribute__((always_inline)) {
        const int lc = min(lt, n_tiles - 1), t0 = st + TILE * lc;
        seq_load<D>(a, s, t0, min(TILE, en - t0), (size_t)(tile_base + lc) * a.H_v + j, qh, j, v0, h, ln, lg);
    };

    // ---- state waves: the recurrence, 3 barriers per tile
    auto state_step = [&](int lt) __attribute__((always_inline)) {
        const int t0 = st + TILE * lt, n = min(TILE, en - t0);
        const int buf = lt & 1;
        __syncthreads();  // ---- A: tile lt staged, S^T of tile lt written
        {
            // K S0^T for rows 16 h .. 16 h + 15, then R = V - diag(Gamma) K S0^T
            f32x4 xk0 = {0.f, 0.f, 0.f, 0.f}, xk1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const int r0 = (32 * ks + 8 * lg + trow) * SLD + tcol;
                const bf16x8 bh = cat_bf16(ds_read_tr16(&sh.SThi[buf][r0]), ds_read_tr16(&sh.SThi[buf][r0 + 4 * SLD]));
                const bf16x8 bl = cat_bf16(ds_read_tr16(&sh.STlo[buf][r0]), ds_read_tr16(&sh.STlo[buf][r0 + 4 * SLD]));
                const bf16x8 ka = as_bf16x8(*(const u32x4 *)(&sh.Ks[buf][(16 * h + ln) * KLD + 32 * ks + 8 * lg]));
                xk0 = mfma_bf16(ka, bh, xk0);
                xk1 = mfma_bf16(ka, bl, xk1);
            }
            const uint2 vv = sh.Vst[buf][h][lane];
            const float4 g4 = sh.Gst[buf][h][lane];
            const float gam[4] = {g4.x, g4.y, g4.z, g4.w};
            const float vr[4] = {__uint_as_float(vv.x << 16), __uint_as_float(vv.x & 0xffff0000u),
                                 __uint_as_float(vv.y << 16), __uint_as_float(vv.y & 0xffff0000u)};
            _Float16 rr[4] __attribute__((aligned(8)));
#pragma unroll
            for (int e = 0; e < 4; ++e)
                rr[e] = (_Float16)(vr[e] - __builtin_amdgcn_exp2f(gam[e]) * (xk0[e] + xk1[e]));
            *(uint2 *)(&sh.RT[buf][ln * TLD + 16 * h + 4 * lg]) = *(const uint2 *)rr;
        }
        __syncthreads();  // ---- B: R^T complete
        {
            // writes E = T diag(beta) R; D_last E split in two bf16 terms
            f32x4 E = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                if (ks <= (h >> 1)) {
                    const half8 br = *(const half8 *)(&sh.RT[buf][ln * TLD + 32 * ks + 8 * lg]);
                    E = mfma_f16(as_half8(sh.Tst[buf][h][ks][lane]), br, E);
                }
            }
            const float4 g4 = sh.Gst[buf][h][lane];
            const float gam[4] = {g4.x, g4.y, g4.z, g4.w};
            const float glast = sh.Glast[buf];
            _Float16 ee[4] __attribute__((aligned(8)));
            float de[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                ee[e] = (_Float16)E[e];
                de[e] = E[e] * __builtin_amdgcn_exp2f(glast - gam[e]);
            }
            const uint32_t h01 = bf16_pack(de[0], de[1]), h23 = bf16_pack(de[2], de[3]);
            const uint32_t l01 = bf16_pack(de[0] - bf16_lo_f(h01), de[1] - bf16_hi_f(h01));
            const uint32_t l23 = bf16_pack(de[2] - bf16_lo_f(h23), de[3] - bf16_hi_f(h23));
            const int off = ln * TLD + 16 * h + 4 * lg;
            *(uint2 *)(&sh.ET[buf][off]) = *(const uint2 *)ee;
            *(uint2 *)(&sh.DThi[buf][off]) = make_uint2(h01, h23);
            *(uint2 *)(&sh.DTlo[buf][off]) = make_uint2(l01, l23);
        }
        __syncthreads();  // ---- C: E^T and (D_last E)^T complete
        {
            // S = Gamma_last S0 + (D_last E)^T K
            const float gl = __builtin_amdgcn_exp2f(sh.Glast[buf]);
            f32x4 Sl[NB];
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
                for (int e = 0; e < 4; ++e) S[nb][e] *= gl;
                Sl[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
            }
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                const bf16x8 ah = as_bf16x8(*(const u32x4 *)(&sh.DThi[buf][ln * TLD + 32 * ks + 8 * lg]));
                const bf16x8 al = as_bf16x8(*(const u32x4 *)(&sh.DTlo[buf][ln * TLD + 32 * ks + 8 * lg]));
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) {
                    const int r0 = (32 * ks + 8 * lg + trow) * KLD + h * (D / 4) + 16 * nb + tcol;
                    const bf16x8 bk = cat_bf16(ds_read_tr16(&sh.Ks[buf][r0]), ds_read_tr16(&sh.Ks[buf][r0 + 4 * KLD]));
                    S[nb] = mfma_bf16(ah, bk, S[nb]);
                    Sl[nb] = mfma_bf16(al, bk, Sl[nb]);
                }
            }
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) S[nb] += Sl[nb];

            // frame end: drift sums of this slice (one pair per row of 16
            // lanes, reduced later in a fixed order), optional snapshot
            const int done = TILE * lt + n;
            if (DRIFT && ((a.frame_len > 0 && done % a.frame_len == 0) || done == len)) {
                float num = 0.f, den = 0.f;
#pragma unroll
                for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float dl = S[nb][e] - S_start[nb][e];
                        num += dl * dl;
                        den += S_start[nb][e] * S_start[nb][e];
                    }
                num = row16_sum(num);
                den = row16_sum(den);
                if (ln == 15 && a.wsDrift && frame < a.n_frames) {
                    float *dst = a.wsDrift + ((((size_t)frame * a.H_v + j) * a.n_split + sl) * 16 + 4 * h + lg) * 2;
                    dst[0] = num;
                    dst[1] = den;
                }
                if (a.snapshots && frame < a.n_frames) {
                    const size_t fb = ((size_t)frame * a.H_v + j) * D * D;
#pragma unroll
                    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            a.snapshots[fb + (size_t)(v0 + 4 * lg + e) * D + h * (D / 4) + 16 * nb + ln] = S[nb][e];
                }
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) S_start[nb] = S[nb];
                ++frame;
            }
            if (lt + 1 < n_tiles) write_state(buf ^ 1);
        }
    };

    // ---- helper waves: three register sets -- cur (tile lt), nxt (tile
    // lt + 1, loaded one tile ago, staged at the end of this tile) and nn
    // (tile lt + 2, loaded now)
    auto helper_step = [&](int lt, SeqTile<D> &cur, SeqTile<D> &nxt, SeqTile<D> &nn) __attribute__((always_inline)) {
        if (lt >= n_tiles) return;  // uniform over the workgroup
        const int t0 = st + TILE * lt, n = min(TILE, en - t0);
        const int buf = lt & 1;
        __syncthreads();  // ---- A
        // Q S0^T for rows 16 h .. 16 h + 15 (kept for the outputs)
        f32x4 xq = {0.f, 0.f, 0.f, 0.f}, xq1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const int r0 = (32 * ks + 8 * lg + trow) * SLD + tcol;
            const bf16x8 bh = cat_bf16(ds_read_tr16(&sh.SThi[buf][r0]), ds_read_tr16(&sh.SThi[buf][r0 + 4 * SLD]));
            const bf16x8 bl = cat_bf16(ds_read_tr16(&sh.STlo[buf][r0]), ds_read_tr16(&sh.STlo[buf][r0 + 4 * SLD]));
            const bf16x8 qa = as_bf16x8(cur.q[ks]);
            xq = mfma_bf16(qa, bh, xq);
            xq1 = mfma_bf16(qa, bl, xq1);
        }
        xq += xq1;
        load_tile(nn, lt + 2);
        __syncthreads();  // ---- B
        __syncthreads();  // ---- C
        // outputs O = diag(Gamma) Q S0^T + P E for rows 16 h .. 16 h + 15
        const float gam[4] = {cur.gam.x, cur.gam.y, cur.gam.z, cur.gam.w};
        f32x4 oacc;
#pragma unroll
        for (int e = 0; e < 4; ++e) oacc[e] = __builtin_amdgcn_exp2f(gam[e]) * xq[e];
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            if (ks <= (h >> 1)) {
                const half8 be = *(const half8 *)(&sh.ET[buf][ln * TLD + 32 * ks + 8 * lg]);
                oacc = mfma_f16(as_half8(cur.p[ks]), be, oacc);
            }
        }
        if (OUT_BF16) {
            uint16_t *ob = (uint16_t *)a.o + (size_t)t0 * a.H_v * D + (size_t)j * D + v0 + ln;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int r = 16 * h + 4 * lg + e;
                if (r < n) ob[(uint32_t)r * a.H_v * D] = __builtin_bit_cast(uint16_t, (__bf16)(a.scale * oacc[e]));
            }
        } else {
            float *ob = (float *)a.o + (size_t)t0 * a.H_v * D + (size_t)j * D + v0 + ln;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int r = 16 * h + 4 * lg + e;
                if (r < n) ob[(uint32_t)r * a.H_v * D] = a.scale * oacc[e];
            }
        }
        if (lt + 1 < n_tiles) stage(nxt, buf ^ 1);
    };

    if (n_tiles > 0) {
        if (state_wave) {
            write_state(0);
            for (int lt = 0; lt < n_tiles; ++lt) state_step(lt);
        } else {
            SeqTile<D> ta, tb, tc;
            load_tile(ta, 0);
            load_tile(tb, 1);
            stage(ta, 0);
            for (int lt = 0; lt < n_tiles; lt += 3) {
                helper_step(lt, ta, tb, tc);
                helper_step(lt + 1, tb, tc, ta);
                helper_step(lt + 2, tc, ta, tb);
            }
        }
    }

    if (state_wave) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int vr = v0 + 4 * lg + e, c = h * (D / 4) + 16 * nb + ln;
                a.state_out[sbase + (size_t)vr * D + c] = S[nb][e];
            }
    }
}

// Sum of the per-row drift sums of every slice (fixed order) -> [n_frames][H_v][2].
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
        for (int s = 0; s < n_split * 16; ++s) {
            num += ws[((size_t)idx * n_split * 16 + s) * 2];
            den += ws[((size_t)idx * n_split * 16 + s) * 2 + 1];
        }
    }
    out[(size_t)idx * 2] = num;
    out[(size_t)idx * 2 + 1] = den;
}

// ============================================================================
// host side
// ============================================================================
static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

GdnWorkspace gdn_workspace_layout(int B, int T_total, int H_v, int d, int n_frames) {
    GdnWorkspace w{};
    w.tiles_max = (int)(((long long)T_total + 63LL * B) / 64);
    w.n_split = d / 16;
    size_t off = 0;
    w.offT = off;
    off = align256(off + (size_t)w.tiles_max * H_v * TP_HALVES * sizeof(_Float16));
    w.offP = off;
    off = align256(off + (size_t)w.tiles_max * H_v * TP_HALVES * sizeof(_Float16));
    w.offGam = off;
    off = align256(off + (size_t)w.tiles_max * H_v * 64 * sizeof(float));
    w.offDrift = off;
    off = align256(off + (size_t)n_frames * H_v * w.n_split * 16 * 2 * sizeof(float));
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
    a.wsGam = p.wsGam;
    a.wsDrift = p.drift_partials ? p.wsDrift : nullptr;
    a.n_split = p.n_split;

    if (p.tiles_max > 0) {
        hipLaunchKernelGGL(gdn_prep_kernel<D>, dim3(p.tiles_max, p.H_v), dim3(256), 0, stream, a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const int n_wg = p.B * p.H_v * p.n_split;
    // the frame-end work is compiled out when neither drift sums nor snapshots are asked for
    const bool drift = p.drift_partials || p.snapshots;
    if (p.o_bf16) {
        if (drift)
            hipLaunchKernelGGL((gdn_seq_kernel<D, true, true>), dim3(n_wg), dim3(512), 0, stream, a);
        else
            hipLaunchKernelGGL((gdn_seq_kernel<D, true, false>), dim3(n_wg), dim3(512), 0, stream, a);
    } else {
        if (drift)
            hipLaunchKernelGGL((gdn_seq_kernel<D, false, true>), dim3(n_wg), dim3(512), 0, stream, a);
        else
            hipLaunchKernelGGL((gdn_seq_kernel<D, false, false>), dim3(n_wg), dim3(512), 0, stream, a);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (p.drift_partials && p.n_frames > 0) {
        const int n = p.n_frames * p.H_v;
        hipLaunchKernelGGL(gdn_drift_finalize_kernel, dim3((n + 255) / 256), dim3(256), 0, stream, p.wsDrift,
                           p.drift_partials, p.n_frames, p.H_v, p.n_split, a.st, p.frame_len);
        e = hipGetLastError();
    }
    return e;
}

hipError_t launch_gdn(const GdnLaunch &p, hipStream_t stream) {
    if (p.d == 128) return launch_d<128>(p, stream);
    return launch_d<64>(p, stream);
}

}  // namespace ds
