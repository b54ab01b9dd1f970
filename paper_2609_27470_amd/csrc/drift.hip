// State drift per frame from per-(layer, frame, head) sums (Section 3.2, Eq. 3).
//
// partials[l][f][h] = (num, den) with num = ||S_end - S_start||_F^2 and
// den = ||S_start||_F^2 of one head.  Eq. 3 takes the Frobenius norm over the
// whole state of a layer, i.e. over all its heads, and averages the ratio
// over layers.  Sums are accumulated in fp64 in a fixed order, so the result
// does not depend on scheduling.
#include "common.h"
#include "kernels.h"

namespace ds {

__device__ __forceinline__ double drift_ratio(double num, double den) {
    if (den > 0.0) return sqrt(num / den);
    return num > 0.0 ? __builtin_huge_val() : 0.0;
}

__device__ __forceinline__ double wave_sum_d(double x) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off, 64);
    return x;
}

// One workgroup (16 waves) per frame.  Wave w takes layers w, w + 16, ...;
// its lanes take the heads of a layer (lane, lane + 64, ...).  A wave loads
// the (num, den) pairs of up to DRIFT_LPW of its layers, up to 256 heads (or
// 16-row slices of 32 heads) each, before it reduces any of them, so a frame
// costs one memory round trip rather than one per layer;
// lanes sum in order, the lanes of a wave meet in a butterfly, and the waves'
// totals are added in wave order.  Every sum has a fixed order, so the result
// does not depend on scheduling.
constexpr int DRIFT_WAVES = 16, DRIFT_LPW = 4, DRIFT_HPL = 4;  // waves, layers per wave per round, heads per lane
__global__ __launch_bounds__(64 * DRIFT_WAVES) void drift_frame_kernel(const float *p, int L, int F, int H, int mode,
                                                                        float *scores) {
    const int f = blockIdx.x, lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    double acc = 0.0;  // same value in every lane of the wave
    bool inf = false;
    for (int l0 = w; l0 < L; l0 += DRIFT_WAVES * DRIFT_LPW) {
        // the pairs of this round's layers (heads lane, lane + 64 in registers;
        // more heads per layer are read in the loop below)
        float2 pr[DRIFT_LPW][DRIFT_HPL];
#pragma unroll
        for (int i = 0; i < DRIFT_LPW; ++i) {
            const int l = l0 + DRIFT_WAVES * i;
#pragma unroll
            for (int c = 0; c < DRIFT_HPL; ++c) {
                const int h = lane + 64 * c;
                pr[i][c] = (l < L && h < H) ? *(const float2 *)(p + (((size_t)l * F + f) * H + h) * 2) : float2{0.f, 0.f};
            }
        }
#pragma unroll
        for (int i = 0; i < DRIFT_LPW; ++i) {
            const int l = l0 + DRIFT_WAVES * i;
            if (l >= L) break;
            const float *row = p + ((size_t)l * F + f) * H * 2;
            if (mode == 0) {
                double num = 0.0, den = 0.0;
#pragma unroll
                for (int c = 0; c < DRIFT_HPL; ++c) {
                    num += (double)pr[i][c].x;
                    den += (double)pr[i][c].y;
                }
                for (int h = lane + 64 * DRIFT_HPL; h < H; h += 64) {
                    num += (double)row[2 * h];
                    den += (double)row[2 * h + 1];
                }
                const double r = drift_ratio(wave_sum_d(num), wave_sum_d(den));
                if (isinf(r)) inf = true; else acc += r;
            } else {
                double x = 0.0;
                bool xi = false;
                auto add = [&](float2 v, bool valid) {
                    if (!valid) return;
                    if (mode == 3) {
                        x += v.y > 0.f ? (double)v.x / (double)v.y : 0.0;
                    } else {
                        const double r = drift_ratio((double)v.x, (double)v.y);
                        if (isinf(r)) xi = true; else x += r;
                    }
                };
#pragma unroll
                for (int c = 0; c < DRIFT_HPL; ++c) add(pr[i][c], lane + 64 * c < H);
                for (int h = lane + 64 * DRIFT_HPL; h < H; h += 64) add(*(const float2 *)(row + 2 * h), true);
                acc += wave_sum_d(x);
                if (__any(xi)) inf = true;
            }
        }
    }
    __shared__ double s_acc[DRIFT_WAVES];
    __shared__ int s_inf[DRIFT_WAVES];
    if (lane == 0) {
        s_acc[w] = acc;
        s_inf[w] = inf;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double tot = 0.0;
        bool any_inf = false;
        for (int i = 0; i < DRIFT_WAVES; ++i) {
            tot += s_acc[i];
            any_inf |= s_inf[i] != 0;
        }
        const long long cnt = mode == 0 ? (long long)L : (long long)L * H;
        scores[f] = any_inf ? __builtin_huge_valf() : (cnt ? (float)(tot / (double)cnt) : 0.f);
    }
}

__global__ __launch_bounds__(256) void drift_head_kernel(const float *p, int n, float *scores) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    scores[i] = (float)drift_ratio((double)p[2 * (size_t)i], (double)p[2 * (size_t)i + 1]);
}

// Drift sums from two copies of the state (the unfused way: keep a copy of
// the state before a frame, then two norms after it).  One workgroup per
// (layer, stream, head); each thread sums a strided part of the d_v x d_k
// entries in fp32, the partial sums are combined in a fixed order in fp64.
__global__ __launch_bounds__(256) void drift_states_kernel(const float *before, const float *after, int n_elem,
                                                            float *partials) {
    const size_t base = (size_t)blockIdx.x * n_elem;
    const float4 *b4 = (const float4 *)(before + base), *a4 = (const float4 *)(after + base);
    float num = 0.f, den = 0.f;
    for (int i = threadIdx.x; i < n_elem / 4; i += 256) {
        const float4 b = b4[i], a = a4[i];
        const float d0 = a.x - b.x, d1 = a.y - b.y, d2 = a.z - b.z, d3 = a.w - b.w;
        num += d0 * d0 + d1 * d1 + d2 * d2 + d3 * d3;
        den += b.x * b.x + b.y * b.y + b.z * b.z + b.w * b.w;
    }
    __shared__ double sn[256], sd[256];
    sn[threadIdx.x] = num;
    sd[threadIdx.x] = den;
    __syncthreads();
    for (int off = 128; off > 0; off >>= 1) {
        if ((int)threadIdx.x < off) {
            sn[threadIdx.x] += sn[threadIdx.x + off];
            sd[threadIdx.x] += sd[threadIdx.x + off];
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        partials[2 * (size_t)blockIdx.x] = (float)sn[0];
        partials[2 * (size_t)blockIdx.x + 1] = (float)sd[0];
    }
}

hipError_t launch_drift_states(const float *before, const float *after, int n_heads, int n_elem, float *partials,
                               hipStream_t stream) {
    if (n_heads == 0) return hipSuccess;
    hipLaunchKernelGGL(drift_states_kernel, dim3(n_heads), dim3(256), 0, stream, before, after, n_elem, partials);
    return hipGetLastError();
}

hipError_t launch_drift(const float *partials, int L, int F, int H_v, int mode, float *scores,
                        hipStream_t stream) {
    if (mode == 2) {
        const int n = L * F * H_v;
        if (n == 0) return hipSuccess;
        hipLaunchKernelGGL(drift_head_kernel, dim3((n + 255) / 256), dim3(256), 0, stream, partials, n, scores);
    } else {
        if (F == 0) return hipSuccess;
        hipLaunchKernelGGL(drift_frame_kernel, dim3(F), dim3(64 * DRIFT_WAVES), 0, stream, partials, L, F, H_v, mode,
                           scores);
    }
    return hipGetLastError();
}

}  // namespace ds
