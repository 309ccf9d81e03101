// Small bandwidth-bound kernels: RMSNorm, the per-iteration set-up (metadata
// copy, RoPE table), the cache sweep, the seeded normal fill.
#include <math.h>

#include "device.h"
#include "kernels.h"

namespace slw {
namespace {

constexpr int kNormThreads = 256;

template <typename T>
struct Vec8;
template <>
struct Vec8<bf16> {
    bf16x8 v;
    __device__ void load(const bf16* p) { v = *reinterpret_cast<const bf16x8*>(p); }
    __device__ float operator[](int e) const { return bf2f(v[e]); }
};
template <>
struct Vec8<float> {
    f32x4 a, b;
    __device__ void load(const float* p) {
        a = *reinterpret_cast<const f32x4*>(p);
        b = *reinterpret_cast<const f32x4*>(p + 4);
    }
    __device__ float operator[](int e) const { return e < 4 ? a[e] : b[e - 4]; }
};

// One work-group per row, 8 values per access, fp32 arithmetic; d <= 8192.
template <typename T>
__global__ __launch_bounds__(kNormThreads) void rmsnorm_kernel(const T* __restrict__ x,
                                                               const bf16* __restrict__ g,
                                                               bf16* __restrict__ y, int d, float eps) {
    const int row = blockIdx.x;
    const T* xr = x + static_cast<size_t>(row) * d;
    const bf16x8* gv = reinterpret_cast<const bf16x8*>(g);
    bf16x8* yr = reinterpret_cast<bf16x8*>(y + static_cast<size_t>(row) * d);
    const int nvec = d / 8;
    Vec8<T> v[4];
    float ss = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int i = threadIdx.x + j * kNormThreads;
        if (i < nvec) {
            v[j].load(xr + i * 8);
#pragma unroll
            for (int e = 0; e < 8; ++e) ss += v[j][e] * v[j][e];
        }
    }
    __shared__ float red[kNormThreads / kWave];
    ss = wave_sum(ss);
    if ((threadIdx.x & (kWave - 1)) == 0) red[threadIdx.x / kWave] = ss;
    __syncthreads();
    float tot = 0.f;
#pragma unroll
    for (int w = 0; w < kNormThreads / kWave; ++w) tot += red[w];
    const float inv = 1.0f / sqrtf(tot / static_cast<float>(d) + eps);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int i = threadIdx.x + j * kNormThreads;
        if (i < nvec) {
            const bf16x8 gg = gv[i];
            bf16x8 o;
#pragma unroll
            for (int e = 0; e < 8; ++e) o[e] = f2bf(v[j][e] * inv * bf2f(gg[e]));
            yr[i] = o;
        }
    }
}

// One thread per (row, frequency): cos and sin of position pos[r] times
// theta^(-i/half), formed in fp64 so that large positions keep their accuracy.
__device__ __forceinline__ void rope_entry(const int32_t* pos, float2* cs, int idx, int half, double theta) {
    const int r = idx / half, i = idx % half;
    const double ang = static_cast<double>(pos[r]) * pow(theta, -static_cast<double>(i) / half);
    double s, c;
    sincos(ang, &s, &c);
    cs[idx] = make_float2(static_cast<float>(c), static_cast<float>(s));
}

// Reads the whole buffer so that it displaces whatever the caches hold, and
// leaves no dirty lines behind (a write sweep would make the next kernel pay
// for their write-back).  The store below keeps the loads alive; it fires
// only in the unlikely case that a thread's xor equals `key`.
__global__ void sweep_kernel(uint32_t* p, size_t n4, uint32_t key) {
    size_t i = blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x;
    const size_t stride = static_cast<size_t>(gridDim.x) * blockDim.x;
    const u32x4* q = reinterpret_cast<const u32x4*>(p);
    u32x4 acc = {0u, 0u, 0u, 0u};
    for (; i < n4; i += stride) acc ^= q[i];
    const uint32_t x = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
    if (x == key) p[0] = x;
}

// First kernel of an iteration.  Blocks [0, copy_blocks) copy n words of
// metadata from coherent host memory mapped into the device's address space
// (one 16-byte read per thread over the bus, then a tail of single words);
// done by a kernel rather than the copy engine, the copy is ordered with the
// kernels around it on the stream without a hand-off between engines.  The
// other blocks fill the RoPE table, reading the positions from the host copy
// (the device copy is not complete while this kernel runs).
__global__ void iteration_setup_kernel(uint32_t* __restrict__ dst, const uint32_t* __restrict__ src, size_t n,
                                       unsigned copy_blocks, const int32_t* __restrict__ pos_host,
                                       float2* __restrict__ cs, int rows, int half, double theta) {
    if (blockIdx.x < copy_blocks) {
        const size_t i = blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x;
        const size_t n4 = n / 4;
        if (i < n4) {
            reinterpret_cast<u32x4*>(dst)[i] = reinterpret_cast<const u32x4*>(src)[i];
        } else if (i < n4 + (n & 3)) {
            const size_t w = 4 * n4 + (i - n4);
            dst[w] = src[w];
        }
        return;
    }
    const int idx = static_cast<int>(blockIdx.x - copy_blocks) * blockDim.x + threadIdx.x;
    if (idx < rows * half) rope_entry(pos_host, cs, idx, half, theta);
}

// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC 2011): a counter-based
// generator, ten rounds of two 32x32->64-bit multiplies with a Weyl-sequence
// key schedule.
__device__ __forceinline__ u32x4 philox4x32_10(u32x4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        if (r) {
            k0 += 0x9E3779B9u;
            k1 += 0xBB67AE85u;
        }
        const uint64_t p0 = static_cast<uint64_t>(0xD2511F53u) * c[0];
        const uint64_t p1 = static_cast<uint64_t>(0xCD9E8D57u) * c[2];
        c = u32x4{static_cast<uint32_t>(p1 >> 32) ^ c[1] ^ k0, static_cast<uint32_t>(p1),
                  static_cast<uint32_t>(p0 >> 32) ^ c[3] ^ k1, static_cast<uint32_t>(p0)};
    }
    return c;
}

// Element i of the stream: draw t = i / 4 gives four normals by Box-Muller
// on the uniforms of its two word pairs (24-bit, exact in fp32):
//   u = (w0 >> 8 + 1/2) 2^-24,  v = (w1 >> 8) 2^-24,
//   z0 = sqrt(-2 ln u) cos(2 pi v),  z1 = sqrt(-2 ln u) sin(2 pi v).
__global__ void fill_normal_kernel(bf16* __restrict__ dst, size_t n, uint32_t k0, uint32_t k1, float mean,
                                   float std) {
    const size_t t = blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x;
    if (4 * t >= n) return;
    const u32x4 w = philox4x32_10(u32x4{static_cast<uint32_t>(t), static_cast<uint32_t>(t >> 32), 0u, 0u}, k0, k1);
    float z[4];
#pragma unroll
    for (int p = 0; p < 2; ++p) {
        const float u = (static_cast<float>(w[2 * p] >> 8) + 0.5f) * 0x1p-24f;
        const float v = static_cast<float>(w[2 * p + 1] >> 8) * 0x1p-24f;
        const float r = sqrtf(-2.0f * logf(u));
        float sn, cs;
        sincosf(6.2831853071795864f * v, &sn, &cs);
        z[2 * p] = r * cs;
        z[2 * p + 1] = r * sn;
    }
#pragma unroll
    for (int e = 0; e < 4; ++e)
        if (4 * t + e < n) dst[4 * t + e] = f2bf(mean + std * z[e]);
}

}  // namespace

void launch_fill_normal(void* dst, size_t n, uint64_t seed, float mean, float std, hipStream_t s) {
    const size_t draws = (n + 3) / 4;
    if (draws == 0) return;
    fill_normal_kernel<<<static_cast<unsigned>((draws + 255) / 256), 256, 0, s>>>(
        static_cast<bf16*>(dst), n, static_cast<uint32_t>(seed), static_cast<uint32_t>(seed >> 32), mean, std);
}

void launch_iteration_setup(void* dst, const void* src, size_t words, const int32_t* pos_host, float2* cs,
                            int rows, int hd, double theta, hipStream_t s) {
    const size_t copy_threads = words / 4 + (words & 3);
    const unsigned copy_blocks = static_cast<unsigned>((copy_threads + 255) / 256);
    const int half = hd / 2;
    const unsigned rope_blocks = static_cast<unsigned>((static_cast<size_t>(rows) * half + 255) / 256);
    if (copy_blocks + rope_blocks == 0) return;
    iteration_setup_kernel<<<copy_blocks + rope_blocks, 256, 0, s>>>(
        static_cast<uint32_t*>(dst), static_cast<const uint32_t*>(src), words, copy_blocks, pos_host, cs, rows,
        half, theta);
}

void launch_rmsnorm(const void* x, bool x_f32, const void* g, void* y, int rows, int d, float eps,
                    hipStream_t s) {
    if (rows <= 0) return;
    if (x_f32)
        rmsnorm_kernel<float><<<rows, kNormThreads, 0, s>>>(static_cast<const float*>(x),
                                                            static_cast<const bf16*>(g),
                                                            static_cast<bf16*>(y), d, eps);
    else
        rmsnorm_kernel<bf16><<<rows, kNormThreads, 0, s>>>(static_cast<const bf16*>(x),
                                                           static_cast<const bf16*>(g),
                                                           static_cast<bf16*>(y), d, eps);
}

void launch_cache_sweep(void* p, size_t bytes, uint32_t key, hipStream_t s) {
    const size_t n4 = bytes / 16;
    if (n4 == 0) return;
    sweep_kernel<<<2048, 256, 0, s>>>(static_cast<uint32_t*>(p), n4, key);
}

}  // namespace slw
