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

__global__ __launch_bounds__(256) void drift_frame_kernel(const float *p, int L, int F, int H, int mode,
                                                           float *scores) {
    const int f = blockIdx.x * 256 + threadIdx.x;
    if (f >= F) return;
    double acc = 0.0;
    bool inf = false;
    int cnt = 0;
    for (int l = 0; l < L; ++l) {
        const float *row = p + ((size_t)l * F + f) * H * 2;
        if (mode == 3) {
            // (sum, count) pairs: mean over heads of sum / count
            for (int h = 0; h < H; ++h) {
                const double c = (double)row[2 * h + 1];
                acc += c > 0.0 ? (double)row[2 * h] / c : 0.0;
                ++cnt;
            }
        } else if (mode == 0) {
            double num = 0.0, den = 0.0;
            for (int h = 0; h < H; ++h) {
                num += (double)row[2 * h];
                den += (double)row[2 * h + 1];
            }
            const double r = drift_ratio(num, den);
            if (isinf(r)) inf = true; else acc += r;
            ++cnt;
        } else {
            for (int h = 0; h < H; ++h) {
                const double r = drift_ratio((double)row[2 * h], (double)row[2 * h + 1]);
                if (isinf(r)) inf = true; else acc += r;
                ++cnt;
            }
        }
    }
    scores[f] = inf ? __builtin_huge_valf() : (cnt ? (float)(acc / cnt) : 0.f);
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
        hipLaunchKernelGGL(drift_frame_kernel, dim3((F + 255) / 256), dim3(256), 0, stream, partials, L, F, H_v,
                           mode, scores);
    }
    return hipGetLastError();
}

}  // namespace ds
