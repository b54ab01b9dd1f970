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
        if (mode == 0) {
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
