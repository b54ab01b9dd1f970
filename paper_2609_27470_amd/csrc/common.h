// Device-side helpers shared by the HIP kernels of libdeltas (gfx950 only).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ds {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Matrix-core fragment layouts of v_mfma_f32_16x16x32_{f16,bf16} on a wave of
// 64 lanes, with ln = lane % 16 and lg = lane / 16:
//   A (16 x 32): lane holds A[ln][8*lg .. 8*lg+7]
//   B (32 x 16): lane holds B[8*lg .. 8*lg+7][ln]
//   C (16 x 16, fp32): lane holds C[4*lg + e][ln], e = 0..3
__device__ __forceinline__ f32x4 mfma_f16(half8 a, half8 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma_bf16(bf16x8 a, bf16x8 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// Round-to-nearest-even fp32 -> bf16 bit pattern (finite inputs).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u) return (uint16_t)((u >> 16) | ((u & 0xffff) ? 0x40 : 0));
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// 8 bf16 (one 16-byte load) -> 8 fp16 (exact for |x| in fp16's normal range).
__device__ __forceinline__ half8 bf16x8_to_f16(uint4 r) {
    half8 o;
    o[0] = (_Float16)bf16_lo(r.x); o[1] = (_Float16)bf16_hi(r.x);
    o[2] = (_Float16)bf16_lo(r.y); o[3] = (_Float16)bf16_hi(r.y);
    o[4] = (_Float16)bf16_lo(r.z); o[5] = (_Float16)bf16_hi(r.z);
    o[6] = (_Float16)bf16_lo(r.w); o[7] = (_Float16)bf16_hi(r.w);
    return o;
}

__device__ __forceinline__ half8 bf16x8_to_f16(u32x4 r) { return bf16x8_to_f16(uint4{r[0], r[1], r[2], r[3]}); }

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 r) { return __builtin_bit_cast(bf16x8, r); }
__device__ __forceinline__ half8 as_half8(uint4 r) { return __builtin_bit_cast(half8, r); }
__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 r) { return __builtin_bit_cast(bf16x8, r); }
__device__ __forceinline__ half8 as_half8(u32x4 r) { return __builtin_bit_cast(half8, r); }
__device__ __forceinline__ uint4 as_uint4(half8 h) { return __builtin_bit_cast(uint4, h); }

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off, 64);
    return x;
}

// Sanitised stream ranges: stream b covers [start, end) with streams ordered,
// disjoint and inside [0, T_total) whatever cu_seqlens holds.
struct Streams {
    const int32_t *cu;
    int B;
    int T;
};

// Walks streams in order; calls f(b, start, end) until it returns true.
template <typename F>
__device__ __forceinline__ void for_streams(const Streams &s, F f) {
    int prev_end = 0;
    for (int b = 0; b < s.B; ++b) {
        int st, en;
        if (s.cu) {
            st = min(max(s.cu[b], prev_end), s.T);
            en = min(max(s.cu[b + 1], st), s.T);
        } else {
            st = 0;
            en = s.T;
        }
        prev_end = en;
        if (f(b, st, en)) return;
    }
}

__device__ __forceinline__ int frames_in(int len, int frame_len) {
    if (len <= 0) return 0;
    if (frame_len <= 0) return 1;
    return (len + frame_len - 1) / frame_len;
}

}  // namespace ds
