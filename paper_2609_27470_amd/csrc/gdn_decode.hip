// One decode step of the gated delta rule (Section 3.2, Eq. 2) for a batch of
// streams, one new token per stream: what answering a question after a state
// restore runs token by token.
//
// Per (stream, v-head) with state S (d_v x d_k, fp32), alpha = exp(g):
//     e      = beta (v - alpha S k)
//     S'     = alpha S + e k^T
//     o      = scale S' q = scale (alpha (S q) + e (k . q))
// Row r of S' depends only on row r of S (through (S k)_r), so the step is one
// pass over the state: each row is read once, its two dot products with k and
// q are formed, and the updated row is written back.  The pass is bound by HBM
// (the state is read and written once, 2 d_v d_k 4 bytes per head), so it runs
// on the vector units: D/8 lanes per row, 8 consecutive columns per lane
// (two 16-byte loads), row sums by an XOR butterfly over those lanes (every
// lane ends with the same bits), workgroups of 256 threads covering 256/(D/8)
// rows of one head.
#include "common.h"
#include "kernels.h"

namespace ds {

template <int D, bool OUT_BF16>
__global__ __launch_bounds__(256) void gdn_decode_kernel(DecodeArgs a) {
    constexpr int LPR = D / 8;          // lanes per row
    constexpr int ROWS = 256 / LPR;     // rows per workgroup
    constexpr int WPH = D / ROWS;       // workgroups per head
    const int head = blockIdx.x / WPH;  // b * H_v + j
    const int b = head / a.H_v, j = head % a.H_v, h = j / a.group;
    const int tid = threadIdx.x, sub = tid % LPR;
    const int r = (blockIdx.x % WPH) * ROWS + tid / LPR;
    const int c0 = 8 * sub;

    const size_t qk = ((size_t)b * a.H_k + h) * D + c0;
    const uint4 kr = *(const uint4 *)(a.k + qk), qr = *(const uint4 *)(a.q + qk);
    const float kf[8] = {bf16_lo(kr.x), bf16_hi(kr.x), bf16_lo(kr.y), bf16_hi(kr.y),
                         bf16_lo(kr.z), bf16_hi(kr.z), bf16_lo(kr.w), bf16_hi(kr.w)};
    const float qf[8] = {bf16_lo(qr.x), bf16_hi(qr.x), bf16_lo(qr.y), bf16_hi(qr.y),
                         bf16_lo(qr.z), bf16_hi(qr.z), bf16_lo(qr.w), bf16_hi(qr.w)};
    const size_t so = ((size_t)head * D + r) * D + c0;
    float s[8];
    if (a.state_in) {
        const float4 x = *(const float4 *)(a.state_in + so), y = *(const float4 *)(a.state_in + so + 4);
        s[0] = x.x; s[1] = x.y; s[2] = x.z; s[3] = x.w;
        s[4] = y.x; s[5] = y.y; s[6] = y.z; s[7] = y.w;
    } else {
#pragma unroll
        for (int c = 0; c < 8; ++c) s[c] = 0.f;
    }
    const float vr = bf16_to_f32(a.v[(size_t)head * D + r]);
    const float alpha = expf(a.g[head]), beta = a.beta[head];

    float sk = 0.f, sq = 0.f, kq = 0.f;
#pragma unroll
    for (int c = 0; c < 8; ++c) {
        sk += s[c] * kf[c];
        sq += s[c] * qf[c];
        kq += kf[c] * qf[c];
    }
#pragma unroll
    for (int off = 1; off < LPR; off <<= 1) {
        sk += __shfl_xor(sk, off, 64);
        sq += __shfl_xor(sq, off, 64);
        kq += __shfl_xor(kq, off, 64);
    }
    const float e = beta * (vr - alpha * sk);
    float n[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) n[c] = alpha * s[c] + e * kf[c];
    *(float4 *)(a.state_out + so) = float4{n[0], n[1], n[2], n[3]};
    *(float4 *)(a.state_out + so + 4) = float4{n[4], n[5], n[6], n[7]};
    if (sub == 0) {
        const float o = a.scale * (alpha * sq + e * kq);
        if (OUT_BF16)
            ((uint16_t *)a.o)[(size_t)head * D + r] = f32_to_bf16(o);
        else
            ((float *)a.o)[(size_t)head * D + r] = o;
    }
}

hipError_t launch_gdn_decode(const DecodeArgs &a, int d, bool o_bf16, hipStream_t stream) {
    const long long heads = (long long)a.B * a.H_v;
    if (heads == 0) return hipSuccess;
    // workgroups per head: d / (256 / (d / 8)) = d^2 / 2048
    const dim3 grid((unsigned)(heads * ((long long)d * d / 2048))), blk(256);
    if (d == 128) {
        if (o_bf16)
            hipLaunchKernelGGL((gdn_decode_kernel<128, true>), grid, blk, 0, stream, a);
        else
            hipLaunchKernelGGL((gdn_decode_kernel<128, false>), grid, blk, 0, stream, a);
    } else {
        if (o_bf16)
            hipLaunchKernelGGL((gdn_decode_kernel<64, true>), grid, blk, 0, stream, a);
        else
            hipLaunchKernelGGL((gdn_decode_kernel<64, false>), grid, blk, 0, stream, a);
    }
    return hipGetLastError();
}

}  // namespace ds
