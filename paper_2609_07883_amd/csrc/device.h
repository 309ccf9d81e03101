// Device-side types and helpers shared by the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace slw {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

__device__ __forceinline__ float bf2f(bf16 v) { return static_cast<float>(v); }
__device__ __forceinline__ bf16 f2bf(float v) { return static_cast<bf16>(v); }  // RNE

// 16x16x32 bf16 MFMA, fp32 accumulate.  Lane l supplies row (A) / column (B)
// l % 16 and the eight k values of group l / 16; the result holds, in lane l,
// element i: row 4 * (l / 16) + i, column l % 16.
__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// 32x32x16 bf16 MFMA.  Lane l supplies row / column l % 32 and the eight k
// values of group l / 32; element i of the result in lane l is
// row 8 * (i / 4) + 4 * (l / 32) + i % 4, column l % 32.
__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Work-groups of a launch are dispatched round-robin to the 8 XCDs (linear id
// % 8), each with its own L2.  Position in a work order of linear block id
// `pid` out of `total` such that every XCD takes a contiguous range of the
// order: work that shares operands, placed next to each other in the order,
// then runs on one XCD and shares its L2.
__device__ __forceinline__ int xcd_order(int pid, int total) {
    constexpr int kXcd = 8;
    const int q = total / kXcd, r = total % kXcd;
    const int xcd = pid % kXcd, local = pid / kXcd;
    return xcd < r ? xcd * (q + 1) + local : r * (q + 1) + (xcd - r) * q + local;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
    return v;
}

}  // namespace slw
