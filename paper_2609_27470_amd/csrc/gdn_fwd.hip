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
//   gdn_drift_finalize sums the per-slice drift sums in a fixed order.
#include "common.h"
#include "kernels.h"

namespace ds {

constexpr int TILE = 64;

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
// gdn_prep: one workgroup per (tile, qk-head); loops over the v-heads that
// read this qk-head.
// ============================================================================
template <int D>
__global__ __launch_bounds__(256) void gdn_prep_kernel(GdnArgs a) {
    constexpr int KS = D / 32;   // 32-wide k-steps over the head dim
    constexpr int KLD = D + 8;   // halves per LDS row of the K tile
    constexpr int ALD = 65;      // floats per LDS row of A and T
    constexpr int PLD = 72;      // halves per LDS row of P
    __shared__ __align__(16) uint16_t Ks[64 * KLD];
    __shared__ float As[64 * ALD];
    __shared__ float Ts[64 * ALD];
    __shared__ float Ys[3 * 256];
    __shared__ __align__(16) _Float16 Ps[64 * PLD];
    __shared__ float gam_s[64], beta_s[64];

    const int ti = blockIdx.x, h = blockIdx.y;
    int t0 = 0, n = 0;
    if (!locate_tile(a.st, ti, t0, n)) return;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, ln = lane & 15, lg = lane >> 4;
    const uint4 zero4 = make_uint4(0, 0, 0, 0);

    // ---- K tile -> LDS (bf16, rows past the stream end are zero)
    constexpr int CPR = D / 8;
    for (int c = tid; c < 64 * CPR; c += 256) {
        const int r = c / CPR, cc = c % CPR;
        uint4 val = zero4;
        if (r < n) val = *(const uint4 *)(a.k + ((size_t)(t0 + r) * a.H_k + h) * D + cc * 8);
        *(uint4 *)(&Ks[r * KLD + cc * 8]) = val;
    }
    uint4 qa[KS];
    {
        const int r = 16 * w + ln;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
            qa[ks] = (r < n) ? *(const uint4 *)(a.q + ((size_t)(t0 + r) * a.H_k + h) * D + 32 * ks + 8 * lg)
                             : zero4;
    }
    __syncthreads();

    // ---- Gram blocks of row block w: KK^T and QK^T for column blocks nb <= w
    f32x4 gk[4], gq[4];
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
        gk[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
        gq[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    {
        uint4 ka[KS];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) ka[ks] = *(const uint4 *)(&Ks[(16 * w + ln) * KLD + 32 * ks + 8 * lg]);
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) {
            if (nb <= w) {
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    const uint4 kb = *(const uint4 *)(&Ks[(16 * nb + ln) * KLD + 32 * ks + 8 * lg]);
                    gk[nb] = mfma_bf16(as_bf16x8(ka[ks]), as_bf16x8(kb), gk[nb]);
                    gq[nb] = mfma_bf16(as_bf16x8(qa[ks]), as_bf16x8(kb), gq[nb]);
                }
            }
        }
    }

    for (int jj = 0; jj < a.group; ++jj) {
        const int j = h * a.group + jj;
        const size_t tv = (size_t)ti * a.H_v + j;
        // ---- gates of this v-head; gamma = inclusive prefix sum of g
        if (w == 0) {
            float gv = 0.f, bv = 0.f;
            if (lane < n) {
                gv = a.g[(size_t)(t0 + lane) * a.H_v + j];
                bv = a.beta[(size_t)(t0 + lane) * a.H_v + j];
            }
            float s = gv;
#pragma unroll
            for (int off = 1; off < 64; off <<= 1) {
                const float y = __shfl_up(s, off, 64);
                if (lane >= off) s += y;
            }
            gam_s[lane] = s;
            beta_s[lane] = bv;
            a.wsGam[tv * 64 + lane] = s;
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
                    const float dri = expf(gam_s[r] - gam_s[i]);
                    pv = dri * gq[nb][e];
                    if (i < r) av = beta_s[r] * dri * gk[nb][e];
                }
                As[r * ALD + i] = av;
                Ps[r * PLD + i] = (_Float16)pv;
            }
        }
        __syncthreads();

        // ---- T = (I + A)^{-1}.  Diagonal 16x16 blocks by forward substitution
        // (lane = 16 * block + column), then the off-diagonal blocks by
        // distance from the diagonal: T_ij = -T_ii sum_{k=j}^{i-1} A_ik T_kj.
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
        }
        __syncthreads();
        {
            const int row = tid >> 4, col = tid & 15;
            for (int d = 1; d <= 3; ++d) {
                for (int p = 0; p + d <= 3; ++p) {
                    const int bi = p + d, bj = p;
                    float y = 0.f;
                    for (int kb = bj; kb < bi; ++kb) {
#pragma unroll
                        for (int m = 0; m < 16; ++m)
                            y += As[(16 * bi + row) * ALD + 16 * kb + m] * Ts[(16 * kb + m) * ALD + 16 * bj + col];
                    }
                    Ys[p * 256 + row * 16 + col] = y;
                }
                __syncthreads();
                for (int p = 0; p + d <= 3; ++p) {
                    const int bi = p + d, bj = p;
                    float t = 0.f;
#pragma unroll
                    for (int m = 0; m < 16; ++m) t -= Ts[(16 * bi + row) * ALD + 16 * bi + m] * Ys[p * 256 + m * 16 + col];
                    Ts[(16 * bi + row) * ALD + 16 * bj + col] = t;
                }
                __syncthreads();
            }
        }

        // ---- write T diag(beta) and P (fp16, row-major 64 x 64, zero above the diagonal)
        {
            const int r = tid >> 2, c0 = (tid & 3) * 16;
            half8 t_lo, t_hi;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int i0 = c0 + e, i1 = c0 + 8 + e;
                t_lo[e] = (_Float16)((i0 <= r) ? Ts[r * ALD + i0] * beta_s[i0] : 0.f);
                t_hi[e] = (_Float16)((i1 <= r) ? Ts[r * ALD + i1] * beta_s[i1] : 0.f);
            }
            _Float16 *dstT = a.wsT + tv * 4096 + r * 64 + c0;
            *(uint4 *)dstT = as_uint4(t_lo);
            *(uint4 *)(dstT + 8) = as_uint4(t_hi);
            _Float16 *dstP = a.wsP + tv * 4096 + r * 64 + c0;
            *(uint4 *)dstP = *(const uint4 *)(&Ps[r * PLD + c0]);
            *(uint4 *)(dstP + 8) = *(const uint4 *)(&Ps[r * PLD + c0 + 8]);
        }
        __syncthreads();
    }
}

// ============================================================================
// gdn_seq: one workgroup per (stream, v-head, 16 consecutive rows of S).
// Wave w owns state columns [w D/4, (w+1) D/4) of those 16 rows.
// ============================================================================
template <int D, bool OUT_BF16, bool DRIFT>
__global__ __launch_bounds__(256) void gdn_seq_kernel(GdnArgs a) {
    constexpr int KS = D / 32;
    constexpr int NB = D / 64;    // 16-column state blocks per wave
    constexpr int TLD = 72;       // halves per LDS row of K^T, R^T, E^T
    constexpr int SLD = D + 8;    // halves per LDS row of S0
    __shared__ __align__(16) _Float16 KT[D * TLD];
    __shared__ __align__(16) _Float16 S0h[16 * SLD];
    __shared__ __align__(16) _Float16 RT[16 * TLD];
    __shared__ __align__(16) _Float16 ET[16 * TLD];
    __shared__ __align__(16) _Float16 DET[16 * TLD];
    __shared__ float red[8];

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, ln = lane & 15, lg = lane >> 4;

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

    // ---- state rows v0 + 4 lg + e, columns w D/4 + 16 nb + ln
    const size_t sbase = ((size_t)b * a.H_v + j) * D * D;
    f32x4 S[NB], S_start[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int vr = v0 + 4 * lg + e, c = w * (D / 4) + 16 * nb + ln;
            S[nb][e] = a.state_in ? a.state_in[sbase + (size_t)vr * D + c] : 0.f;
        }
        S_start[nb] = S[nb];
    }

    const uint4 zero4 = make_uint4(0, 0, 0, 0);
    const int n_tiles = (len + TILE - 1) / TILE;
    int frame = frame_base;
    for (int lt = 0; lt < n_tiles; ++lt) {
        const int t0 = st + TILE * lt, n = min(TILE, en - t0);
        const size_t tv = (size_t)(tile_base + lt) * a.H_v + j;

        // ---- loads: k, q fragments of rows 16 w + ln; per-row v and gamma
        half8 kh[KS], qf[KS];
        {
            const int r = 16 * w + ln;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                uint4 kr = zero4, qr = zero4;
                if (r < n) {
                    const size_t off = ((size_t)(t0 + r) * a.H_k + qh) * D + 32 * ks + 8 * lg;
                    kr = *(const uint4 *)(a.k + off);
                    qr = *(const uint4 *)(a.q + off);
                }
                kh[ks] = bf16x8_to_f16(kr);
                qf[ks] = bf16x8_to_f16(qr);
            }
        }
        float vrow[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int r = 16 * w + 4 * lg + e;
            vrow[e] = (r < n) ? bf16_to_f32(a.v[((size_t)(t0 + r) * a.H_v + j) * D + v0 + ln]) : 0.f;
        }
        const float4 g4 = *(const float4 *)(a.wsGam + tv * 64 + 16 * w + 4 * lg);
        const float gam[4] = {g4.x, g4.y, g4.z, g4.w};
        const float gam_last = a.wsGam[tv * 64 + 63];
        uint4 ta[2], pa[2];
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            ta[ks] = zero4;
            pa[ks] = zero4;
            if (ks <= (w >> 1)) {
                const size_t off = tv * 4096 + (size_t)(16 * w + ln) * 64 + 32 * ks + 8 * lg;
                ta[ks] = *(const uint4 *)(a.wsT + off);
                pa[ks] = *(const uint4 *)(a.wsP + off);
            }
        }

        // ---- K^T and the entry state (fp16) into LDS
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
            for (int e = 0; e < 8; ++e) KT[(32 * ks + 8 * lg + e) * TLD + 16 * w + ln] = kh[ks][e];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int e = 0; e < 4; ++e) S0h[(4 * lg + e) * SLD + w * (D / 4) + 16 * nb + ln] = (_Float16)S[nb][e];
        __syncthreads();

        // ---- K S0^T and Q S0^T for rows 16 w .. 16 w + 15
        f32x4 xk = {0.f, 0.f, 0.f, 0.f}, xq = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const half8 bs = *(const half8 *)(&S0h[ln * SLD + 32 * ks + 8 * lg]);
            xk = mfma_f16(kh[ks], bs, xk);
            xq = mfma_f16(qf[ks], bs, xq);
        }
        // ---- residual R = V - diag(Gamma) K S0^T  -> R^T in LDS
        float Gam[4];
        {
            _Float16 rr[4] __attribute__((aligned(8)));
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                Gam[e] = expf(gam[e]);
                rr[e] = (_Float16)(vrow[e] - Gam[e] * xk[e]);
            }
            *(uint2 *)(&RT[ln * TLD + 16 * w + 4 * lg]) = *(const uint2 *)rr;
        }
        __syncthreads();

        // ---- writes E = T diag(beta) R
        f32x4 E = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            if (ks <= (w >> 1)) {
                const half8 br = *(const half8 *)(&RT[ln * TLD + 32 * ks + 8 * lg]);
                E = mfma_f16(as_half8(ta[ks]), br, E);
            }
        }
        {
            _Float16 ee[4] __attribute__((aligned(8))), de[4] __attribute__((aligned(8)));
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                ee[e] = (_Float16)E[e];
                de[e] = (_Float16)(E[e] * expf(gam_last - gam[e]));
            }
            *(uint2 *)(&ET[ln * TLD + 16 * w + 4 * lg]) = *(const uint2 *)ee;
            *(uint2 *)(&DET[ln * TLD + 16 * w + 4 * lg]) = *(const uint2 *)de;
        }
        __syncthreads();

        // ---- outputs O = diag(Gamma) Q S0^T + P E
        {
            f32x4 oacc;
#pragma unroll
            for (int e = 0; e < 4; ++e) oacc[e] = Gam[e] * xq[e];
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                if (ks <= (w >> 1)) {
                    const half8 be = *(const half8 *)(&ET[ln * TLD + 32 * ks + 8 * lg]);
                    oacc = mfma_f16(as_half8(pa[ks]), be, oacc);
                }
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int r = 16 * w + 4 * lg + e;
                if (r < n) {
                    const size_t off = ((size_t)(t0 + r) * a.H_v + j) * D + v0 + ln;
                    const float val = a.scale * oacc[e];
                    if (OUT_BF16)
                        ((uint16_t *)a.o)[off] = f32_to_bf16(val);
                    else
                        ((float *)a.o)[off] = val;
                }
            }
        }

        // ---- state update S = Gamma_last S0 + (D_last E)^T K
        {
            const float gl = expf(gam_last);
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                for (int e = 0; e < 4; ++e) S[nb][e] *= gl;
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                const half8 ad = *(const half8 *)(&DET[ln * TLD + 32 * ks + 8 * lg]);
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) {
                    const half8 bk = *(const half8 *)(&KT[(w * (D / 4) + 16 * nb + ln) * TLD + 32 * ks + 8 * lg]);
                    S[nb] = mfma_f16(ad, bk, S[nb]);
                }
            }
        }

        // ---- frame end: drift sums of this slice, optional snapshot
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
            num = wave_sum(num);
            den = wave_sum(den);
            if (lane == 0) {
                red[w] = num;
                red[4 + w] = den;
            }
            if (a.snapshots && frame < a.n_frames) {
                const size_t fb = ((size_t)frame * a.H_v + j) * D * D;
#pragma unroll
                for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        a.snapshots[fb + (size_t)(v0 + 4 * lg + e) * D + w * (D / 4) + 16 * nb + ln] = S[nb][e];
            }
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) S_start[nb] = S[nb];
            __syncthreads();
            if (tid == 0 && a.wsDrift && frame < a.n_frames) {
                float *dst = a.wsDrift + (((size_t)frame * a.H_v + j) * a.n_split + sl) * 2;
                dst[0] = (red[0] + red[1]) + (red[2] + red[3]);
                dst[1] = (red[4] + red[5]) + (red[6] + red[7]);
            }
            ++frame;
        }
        __syncthreads();
    }

#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int vr = v0 + 4 * lg + e, c = w * (D / 4) + 16 * nb + ln;
            a.state_out[sbase + (size_t)vr * D + c] = S[nb][e];
        }
}

// Sum of the per-slice drift sums (fixed order) -> [n_frames][H_v][2].
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
    off = align256(off + (size_t)w.tiles_max * H_v * 4096 * sizeof(_Float16));
    w.offP = off;
    off = align256(off + (size_t)w.tiles_max * H_v * 4096 * sizeof(_Float16));
    w.offGam = off;
    off = align256(off + (size_t)w.tiles_max * H_v * 64 * sizeof(float));
    w.offDrift = off;
    off = align256(off + (size_t)n_frames * H_v * w.n_split * 2 * sizeof(float));
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
        hipLaunchKernelGGL(gdn_prep_kernel<D>, dim3(p.tiles_max, p.H_k), dim3(256), 0, stream, a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const int n_wg = p.B * p.H_v * p.n_split;
    // the frame-end work is compiled out when neither drift sums nor snapshots are asked for
    const bool drift = p.drift_partials || p.snapshots;
    if (p.o_bf16) {
        if (drift)
            hipLaunchKernelGGL((gdn_seq_kernel<D, true, true>), dim3(n_wg), dim3(256), 0, stream, a);
        else
            hipLaunchKernelGGL((gdn_seq_kernel<D, true, false>), dim3(n_wg), dim3(256), 0, stream, a);
    } else {
        if (drift)
            hipLaunchKernelGGL((gdn_seq_kernel<D, false, true>), dim3(n_wg), dim3(256), 0, stream, a);
        else
            hipLaunchKernelGGL((gdn_seq_kernel<D, false, false>), dim3(n_wg), dim3(256), 0, stream, a);
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
