/*
 * fp64 oracle for the gated-delta-rule forward with frame drift partials.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, obviously correct CPU
 * reference that the HIP path is checked against.  Only the test suite, the
 * smoke check and the benchmark's CPU-baseline leg may build, load or call
 * it; the product library never does, and the two share no code.
 *
 * What it computes (paper, Section 3.2):
 *   for every stream b and v-head j (qk-head h = j * H_k / H_v), token by
 *   token, in the residual form of the gated delta rule (Eq. 2):
 *       alpha_t = exp(g_t)
 *       e_t     = beta_t * (v_t - alpha_t * S_{t-1} k_t)
 *       S_t     = alpha_t * S_{t-1} + e_t k_t^T          (S is d_v x d_k)
 *       o_t     = scale * S_t q_t                        (read after the update)
 *   and at the end of every frame (every frame_len tokens from the stream's
 *   first token, and at the stream's last token) the two sums behind the
 *   state drift of Eq. 3:
 *       num = ||S_end - S_start||_F^2,  den = ||S_start||_F^2
 *   after which S_start <- S_end.  S_start of the first frame is the entry
 *   state (the copy of the previous state kept for the score, Section 3.2).
 *   Also per frame the write-magnitude signal of the appendix on retention
 *   signals (the beta ||e|| row): the sum over the frame's tokens of
 *   ||e_t||_2 (e_t above already carries beta_t, so this is the Frobenius norm
 *   of the rank-one write for unit keys) and the number of tokens.
 *
 * Inputs are taken exactly as the GPU consumes them: bf16 bit patterns for
 * q, k, v and fp32 for g, beta, widened to fp64 without rounding.
 * Everything else is fp64.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static double bf16_to_f64(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* Frames of a stream of n tokens: one every frame_len tokens plus a ragged
 * tail; frame_len <= 0 makes the whole stream a single frame. */
static int64_t frames_of(int64_t n, int64_t frame_len)
{
    if (n <= 0) return 0;
    if (frame_len <= 0) return 1;
    return (n + frame_len - 1) / frame_len;
}

/*
 * B streams packed along the token axis; cu_seqlens[B+1] are their offsets.
 * q, k: [T][H_k][d_k]; v: [T][H_v][d_v]; g, beta: [T][H_v].
 * S0: [B][H_v][d_v][d_k] or NULL (zeros).
 * o: [T][H_v][d_v]; S_out: [B][H_v][d_v][d_k];
 * partials: [F_total][H_v][2] (num, den) or NULL;
 * writes: [F_total][H_v][2] (sum over the frame of ||e_t||_2, token count) or NULL;
 * snapshots: [F_total][H_v][d_v][d_k] (state at each frame end) or NULL.
 * Returns 0, or -1 on a bad argument.
 */
int ref_gdn_forward(int B, const int32_t *cu_seqlens, int H_k, int H_v, int d_k, int d_v,
                    int frame_len, const uint16_t *q, const uint16_t *k, const uint16_t *v,
                    const float *g, const float *beta, const double *S0, double scale,
                    double *o, double *S_out, double *partials, double *writes, double *snapshots,
                    int n_threads)
{
    if (B < 0 || H_k <= 0 || H_v <= 0 || d_k <= 0 || d_v <= 0 || H_v % H_k != 0) return -1;
    int64_t *frame_base = (int64_t *)malloc(sizeof(int64_t) * (size_t)(B + 1));
    if (!frame_base) return -1;
    frame_base[0] = 0;
    for (int b = 0; b < B; ++b)
        frame_base[b + 1] = frame_base[b] + frames_of(cu_seqlens[b + 1] - cu_seqlens[b], frame_len);

#ifdef _OPENMP
    if (n_threads > 0) omp_set_num_threads(n_threads);
#else
    (void)n_threads;
#endif
    const int64_t units = (int64_t)B * H_v;
    const int group = H_v / H_k;

#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t u = 0; u < units; ++u) {
        const int b = (int)(u / H_v);
        const int j = (int)(u % H_v);
        const int h = j / group;
        const int64_t t0 = cu_seqlens[b], t1 = cu_seqlens[b + 1];
        const size_t ss = (size_t)d_v * d_k;
        double *S = (double *)malloc(sizeof(double) * ss);
        double *S_start = (double *)malloc(sizeof(double) * ss);
        double *kt = (double *)malloc(sizeof(double) * d_k);
        double *qt = (double *)malloc(sizeof(double) * d_k);
        double *e = (double *)malloc(sizeof(double) * d_v);
        if (S0) {
            memcpy(S, S0 + ((size_t)b * H_v + j) * ss, sizeof(double) * ss);
        } else {
            memset(S, 0, sizeof(double) * ss);
        }
        memcpy(S_start, S, sizeof(double) * ss);
        int64_t frame = frame_base[b];
        double wsum = 0.0;
        int64_t wcount = 0;

        for (int64_t t = t0; t < t1; ++t) {
            const uint16_t *kp = k + ((size_t)t * H_k + h) * d_k;
            const uint16_t *qp = q + ((size_t)t * H_k + h) * d_k;
            const uint16_t *vp = v + ((size_t)t * H_v + j) * d_v;
            const double alpha = exp((double)g[(size_t)t * H_v + j]);
            const double bt = (double)beta[(size_t)t * H_v + j];
            for (int c = 0; c < d_k; ++c) {
                kt[c] = bf16_to_f64(kp[c]);
                qt[c] = bf16_to_f64(qp[c]);
            }
            /* e = beta * (v - alpha * S k) */
            for (int r = 0; r < d_v; ++r) {
                const double *Sr = S + (size_t)r * d_k;
                double sk = 0.0;
                for (int c = 0; c < d_k; ++c) sk += Sr[c] * kt[c];
                e[r] = bt * (bf16_to_f64(vp[r]) - alpha * sk);
            }
            {
                double ee = 0.0;
                for (int r = 0; r < d_v; ++r) ee += e[r] * e[r];
                wsum += sqrt(ee);
                ++wcount;
            }
            /* S = alpha * S + e k^T ; o = scale * S q */
            double *op = o + ((size_t)t * H_v + j) * d_v;
            for (int r = 0; r < d_v; ++r) {
                double *Sr = S + (size_t)r * d_k;
                double sq = 0.0;
                for (int c = 0; c < d_k; ++c) {
                    Sr[c] = alpha * Sr[c] + e[r] * kt[c];
                    sq += Sr[c] * qt[c];
                }
                op[r] = scale * sq;
            }
            const int64_t local = t - t0 + 1;
            const int frame_end = (t == t1 - 1) || (frame_len > 0 && local % frame_len == 0);
            if (frame_end) {
                double num = 0.0, den = 0.0;
                for (size_t x = 0; x < ss; ++x) {
                    const double dlt = S[x] - S_start[x];
                    num += dlt * dlt;
                    den += S_start[x] * S_start[x];
                }
                if (partials) {
                    partials[((size_t)frame * H_v + j) * 2 + 0] = num;
                    partials[((size_t)frame * H_v + j) * 2 + 1] = den;
                }
                if (writes) {
                    writes[((size_t)frame * H_v + j) * 2 + 0] = wsum;
                    writes[((size_t)frame * H_v + j) * 2 + 1] = (double)wcount;
                }
                wsum = 0.0;
                wcount = 0;
                if (snapshots) memcpy(snapshots + ((size_t)frame * H_v + j) * ss, S, sizeof(double) * ss);
                memcpy(S_start, S, sizeof(double) * ss);
                ++frame;
            }
        }
        memcpy(S_out + ((size_t)b * H_v + j) * ss, S, sizeof(double) * ss);
        free(S);
        free(S_start);
        free(kt);
        free(qt);
        free(e);
    }
    free(frame_base);
    return 0;
}

/* Number of OpenMP threads a parallel region would use (for reporting). */
int ref_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
