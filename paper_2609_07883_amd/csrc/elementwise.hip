// Bandwidth-bound per-row kernels: RMSNorm, RoPE with paged KV append, fill.
#include <math.h>

#include "device.h"
#include "kernels.h"

namespace slw {
namespace {

constexpr int kNormThreads = 256;

// One work-group per row; 8 bf16 per vector access, fp32 arithmetic.
__global__ __launch_bounds__(kNormThreads) void rmsnorm_kernel(const bf16* __restrict__ x,
                                                               const bf16* __restrict__ g,
                                                               bf16* __restrict__ y, int d,
                                                               float eps) {
    const int row = blockIdx.x;
    const bf16x8* xr = reinterpret_cast<const bf16x8*>(x + static_cast<size_t>(row) * d);
    const bf16x8* gv = reinterpret_cast<const bf16x8*>(g);
    bf16x8* yr = reinterpret_cast<bf16x8*>(y + static_cast<size_t>(row) * d);
    const int nvec = d / 8;
    // d <= 8 * 4 * kNormThreads (= 8192) keeps the row in registers.
    bf16x8 v[4];
    float ss = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        int i = threadIdx.x + j * kNormThreads;
        if (i < nvec) {
            v[j] = xr[i];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                float f = bf2f(v[j][e]);
                ss += f * f;
            }
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
        int i = threadIdx.x + j * kNormThreads;
        if (i < nvec) {
            bf16x8 gg = gv[i], o;
#pragma unroll
            for (int e = 0; e < 8; ++e) o[e] = f2bf(bf2f(v[j][e]) * inv * bf2f(gg[e]));
            yr[i] = o;
        }
    }
}

constexpr int kRopeThreads = 256;

// One work-group per row.  The angles p * theta^(-2i/hd) are formed and
// reduced in double precision, so large positions keep full accuracy.
// K page element (t, d): (d/32)*512 + t*32 + d%32; V page element: d*16 + t.
__global__ __launch_bounds__(kRopeThreads) void rope_append_kernel(RopeAppendArgs a) {
    const int row = blockIdx.x;
    const int hd = a.hd, half = hd / 2;
    const int width = (a.hq + 2 * a.hkv) * hd;
    bf16* r = reinterpret_cast<bf16*>(a.qkv) + static_cast<size_t>(row) * width;
    __shared__ float cs[64], sn[64];
    const int p = a.pos[row];
    if (threadIdx.x < half) {
        const int i = threadIdx.x;
        double ang = static_cast<double>(p) * pow(a.theta, -2.0 * i / hd);
        double c, s;
        sincos(ang, &s, &c);
        cs[i] = static_cast<float>(c);
        sn[i] = static_cast<float>(s);
    }
    __syncthreads();
    const int slot = a.slot[row];
    const size_t blk = slot >> 4, t = slot & 15;
    bf16* kp = reinterpret_cast<bf16*>(a.k_pool);
    bf16* vp = reinterpret_cast<bf16*>(a.v_pool);
    const size_t page = static_cast<size_t>(hd) * 16;
    // rotate q and k (heads 0 .. hq + hkv - 1 of the row), pair (i, i + half)
    const int pairs = (a.hq + a.hkv) * half;
    for (int w = threadIdx.x; w < pairs; w += kRopeThreads) {
        const int h = w / half, i = w % half;
        bf16* base = r + h * hd;
        float x1 = bf2f(base[i]), x2 = bf2f(base[i + half]);
        float y1 = x1 * cs[i] - x2 * sn[i];
        float y2 = x2 * cs[i] + x1 * sn[i];
        bf16 b1 = f2bf(y1), b2 = f2bf(y2);
        base[i] = b1;
        base[i + half] = b2;
        if (h >= a.hq) {
            const int kh = h - a.hq;
            bf16* pg = kp + (blk * a.hkv + kh) * page;
            const int d1 = i, d2 = i + half;
            pg[(d1 >> 5) * 512 + t * 32 + (d1 & 31)] = b1;
            pg[(d2 >> 5) * 512 + t * 32 + (d2 & 31)] = b2;
        }
    }
    // append v
    const bf16* vrow = r + (a.hq + a.hkv) * hd;
    for (int w = threadIdx.x; w < a.hkv * hd; w += kRopeThreads) {
        const int kh = w / hd, dd = w % hd;
        vp[(blk * a.hkv + kh) * page + dd * 16 + t] = vrow[w];
    }
}

__global__ void fill_kernel(uint32_t* p, size_t n, uint32_t v) {
    size_t i = blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x;
    size_t stride = static_cast<size_t>(gridDim.x) * blockDim.x;
    for (; i < n; i += stride) p[i] = v + static_cast<uint32_t>(i);
}

}  // namespace

void launch_rmsnorm(const void* x, const void* g, void* y, int rows, int d, float eps,
                    hipStream_t s) {
    if (rows <= 0) return;
    rmsnorm_kernel<<<rows, kNormThreads, 0, s>>>(static_cast<const bf16*>(x),
                                                 static_cast<const bf16*>(g), static_cast<bf16*>(y),
                                                 d, eps);
}

void launch_rope_append(const RopeAppendArgs& a, hipStream_t s) {
    if (a.rows <= 0) return;
    rope_append_kernel<<<a.rows, kRopeThreads, 0, s>>>(a);
}

void launch_fill(void* p, size_t bytes, uint32_t pattern, hipStream_t s) {
    size_t n = bytes / 4;
    if (n == 0) return;
    fill_kernel<<<2048, 256, 0, s>>>(static_cast<uint32_t*>(p), n, pattern);
}

}  // namespace slw
