// bf16 GEMM out = A W^T on gfx950 matrix cores (v_mfma_f32_32x32x16_bf16).
//
// A [m][k] and W [n][k] are both k-contiguous.  A work-group of four waves
// computes a BM x BN tile; k advances in steps of 64 through a double-buffered
// LDS tile (one barrier per step, next tile prefetched into registers while
// the current one feeds the matrix cores).  LDS rows are 128 bytes; the
// 16-byte chunk c of row r is stored at c ^ ((r >> 1) & 7) so that the rows
// read by one MFMA operand load hit distinct banks.
//
// Each wave's 64 columns are two 32-column MFMA tiles whose accumulators sit
// in the same lanes at the same element index.  Two epilogues use that by
// choosing which W rows feed the two tiles:
//   SwiGLU: tile 0 takes gate rows, tile 1 the matching up rows, so a lane
//           holds gate and up of one output and writes silu(gate) * up;
//   QKV:    within each head, tile 0 takes dims i and tile 1 dims i + hd/2,
//           so a lane holds both halves of a RoPE pair, rotates them, and
//           writes q, or writes k and v straight into their KV pages.
// Small problems split k across work-groups; fp32 partial sums are then
// reduced by a second kernel that applies the same epilogue.
#include <math.h>

#include <algorithm>

#include "device.h"
#include "kernels.h"

namespace slw {
namespace {

constexpr int BK_MAX = 64;  // k-steps per LDS stage are 32 or 64 wide

__device__ __forceinline__ float silu(float g) { return g / (1.0f + __expf(-g)); }

// Head-local order of 32-dim blocks for hd = 128: B blocks 0,1,2,3 hold dims
// blocks 0,2,1,3 (the map is its own inverse).  hd = 64 needs no reordering.
__device__ __forceinline__ int qkv_dim(int cw, int hd) {
    if (hd != 128) return cw;
    const int b = cw >> 5;
    return ((((b & 1) << 1) | (b >> 1)) << 5) | (cw & 31);
}

// W row feeding B column c (c = n0 + tile row).
template <int EPI>
__device__ __forceinline__ int w_row(const GemmArgs& g, int c) {
    if (EPI == EPI_SWIGLU) {
        const int sub = c >> 5, f = g.n >> 1;
        const int col = (sub >> 1) * 32 + (c & 31);
        return (sub & 1) ? f + col : col;
    }
    if (EPI == EPI_QKV) {
        const int cw = c % g.hd;
        return c - cw + qkv_dim(cw, g.hd);
    }
    return c;
}

// Rotate (x0, x1) = dims (d0, d0 + hd/2) of head hg of row `row` by
// cs = (cos, sin) (q and k heads; v heads are not rotated) and store; k and v
// also go to their KV page at slot[row].
__device__ __forceinline__ void qkv_store_cs(const GemmArgs& g, int row, int hg, int d0, float x0, float x1,
                                             float2 cs, int slot) {
    const int d1 = d0 + g.hd / 2;
    bf16* out = static_cast<bf16*>(g.out) + static_cast<size_t>(row) * g.ldo + hg * g.hd;
    if (hg < g.hq + g.hkv) {
        const float y0 = x0 * cs.x - x1 * cs.y;
        const float y1 = x1 * cs.x + x0 * cs.y;
        x0 = y0;
        x1 = y1;
    }
    const bf16 b0 = f2bf(x0), b1 = f2bf(x1);
    out[d0] = b0;
    out[d1] = b1;
    if (hg < g.hq) return;
    const size_t blk = slot >> 4, t = slot & 15;
    if (hg < g.hq + g.hkv) {
        bf16* pg = static_cast<bf16*>(g.k_pool) + (blk * g.hkv + (hg - g.hq)) * g.hd * 16;
        pg[(d0 >> 5) * 512 + t * 32 + (d0 & 31)] = b0;
        pg[(d1 >> 5) * 512 + t * 32 + (d1 & 31)] = b1;
    } else {
        bf16* pg = static_cast<bf16*>(g.v_pool) + (blk * g.hkv + (hg - g.hq - g.hkv)) * g.hd * 16;
        pg[d0 * 16 + t] = b0;
        pg[d1 * 16 + t] = b1;
    }
}

// The same with the rotation and the slot read from the iteration's tables.
__device__ __forceinline__ void qkv_store(const GemmArgs& g, int row, int hg, int d0, float x0, float x1) {
    const float2 cs = hg < g.hq + g.hkv ? g.rope_cs[row * (g.hd / 2) + d0] : make_float2(1.f, 0.f);
    qkv_store_cs(g, row, hg, d0, x0, x1, cs, hg < g.hq ? 0 : g.slot[row]);
}

// LDS rows hold BK bf16 (BK/8 chunks of 16 bytes).  Chunk c of row r is
// stored at c ^ ((r / (16 / CPR)) % CPR): the rows read by one MFMA operand
// load land on distinct banks for both 128-byte (BK 64) and 64-byte (BK 32)
// rows.
template <int BK>
__device__ __forceinline__ int swz(int row, int chunk) {
    constexpr int CPR = BK / 8;
    return chunk ^ ((row / (16 / CPR)) & (CPR - 1));
}

// Tile (tm, tn) at position t of the grouped tile order: group_m tile rows
// at a time, column by column within a group, so that tiles that run
// together share A rows and B columns.  With at most 16 tile rows a group
// spans them all: each weight panel is then streamed into an L2 once for
// every row tile.
__device__ __forceinline__ void tile_coords(int t, int nt_m, int nt_n, int& tm, int& tn) {
    const int GROUP_M = nt_m <= 16 ? nt_m : 8;
    const int per_group = GROUP_M * nt_n;
    const int first_m = (t / per_group) * GROUP_M;
    const int gsize = min(nt_m - first_m, GROUP_M);
    const int in_group = t % per_group;
    tm = first_m + in_group % gsize;
    tn = in_group / gsize;
}

__device__ __forceinline__ void tile_of(int pid, int nt_m, int nt_n, int& tm, int& tn) {
    tile_coords(xcd_order(pid, nt_m * nt_n), nt_m, nt_n, tm, tn);
}

// Wait until at most n vector-memory operations of this wave are
// outstanding (gfx9 s_waitcnt encoding, other counters left alone).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Direct global->LDS load of 16 bytes per lane: lane l's bytes land at
// lds + 16 l (lds is wave-uniform).  Issued as assembly so that the compiler,
// which cannot tell which LDS buffer such a load writes, does not make every
// later LDS read wait for all of them; the main loop waits for them itself.
// M0 is a reserved register that the compiler sets right before each
// instruction that reads it; no compiler-generated code in these kernels
// uses it, so the value left there is never relied on.
__device__ __forceinline__ void load_lds16(const void* src, void* lds) {
    const uint32_t dst = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(reinterpret_cast<uintptr_t>(lds)));
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "s"(dst) : "memory");
}

// Workgroup barrier with no memory fence: the asm statement's memory clobber
// keeps the compiler from moving LDS or global accesses across it, and the
// waits it needs are issued explicitly before it.
__device__ __forceinline__ void barrier_only() { asm volatile("s_barrier" ::: "memory"); }

// Main loops:
//   RING == 0:   registers prefetch the next k step while the current one
//                feeds the matrix cores, then write it to the second of two
//                LDS buffers (one barrier per step).  The k-32 tiles of this
//                kind ask for two waves per SIMD so that two work-groups fit
//                on a CU.
//   RING = 2..4: a ring of RING LDS buffers filled by direct global->LDS
//                loads (16 bytes per lane) issued RING - 1 steps ahead; no
//                staging registers.  Each lane loads the 16-byte chunk that
//                belongs at its LDS slot, so the XOR layout is kept.  A counted
//                wait for the wave's own loads of the step plus a bare barrier
//                make every wave's loads visible; the same barrier proves that
//                the buffer refilled next was finished by all waves.
// Main loop of one tile: acc = A rows [m0, m0 + BM) times W rows
// [n0, n0 + BN) over k steps [kb, kb + nk BK).  The register-staged loop ends
// on a barrier; after a ring loop, callers that reuse the LDS buffers first
// wait for every wave.
template <int BM, int BN, int WAVES_M, int WAVES_N, int BK, int RING, int EPI>
__device__ __forceinline__ void tile_mainloop(const GemmArgs& g, int m0, int n0, int kb, int nk,
                                              bf16 (*As)[BM * BK], bf16 (*Bs)[BN * BK],
                                              f32x16 (&acc)[BM / WAVES_M / 32][BN / WAVES_N / 32]) {
    constexpr int THREADS = WAVES_M * WAVES_N * 64;
    constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
    constexpr int TM = WM / 32, TN = WN / 32;
    constexpr int CPR = BK / 8;  // 16-byte chunks per LDS row
    constexpr int A_LOADS = BM * CPR / THREADS;
    constexpr int B_LOADS = BN * CPR / THREADS;
    static_assert(A_LOADS >= 1 && B_LOADS >= 1, "tile too small");
    static_assert(WN % 64 == 0, "paired epilogues need whole 64-column pairs per wave");

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;

    // Wave-uniform bases plus 32-bit per-lane element offsets (operands are
    // below 2^31 elements).  Rows past m read row m-1 instead: they only feed
    // output rows that are never stored, and an unconditional load keeps the
    // prefetch asynchronous.
    const bf16* A = static_cast<const bf16*>(g.a) + kb;
    const bf16* W = static_cast<const bf16*>(g.w) + kb;

#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f32x16{};

    int a_row[TM], b_row[TN];
#pragma unroll
    for (int i = 0; i < TM; ++i) a_row[i] = wm * WM + i * 32 + (lane & 31);
#pragma unroll
    for (int j = 0; j < TN; ++j) b_row[j] = wn * WN + j * 32 + (lane & 31);
    const int kg = lane >> 5;

    // Fragments of k-step s+1 are read from LDS while the MFMAs of step s run.
    auto compute = [&](int buf) {
        bf16x8 fa[2][TM], fb[2][TN];
        auto read_frags = [&](int s, bf16x8* a, bf16x8* b) {
#pragma unroll
            for (int i = 0; i < TM; ++i)
                a[i] = *reinterpret_cast<const bf16x8*>(&As[buf][a_row[i] * BK + swz<BK>(a_row[i], 2 * s + kg) * 8]);
#pragma unroll
            for (int j = 0; j < TN; ++j)
                b[j] = *reinterpret_cast<const bf16x8*>(&Bs[buf][b_row[j] * BK + swz<BK>(b_row[j], 2 * s + kg) * 8]);
        };
        read_frags(0, fa[0], fb[0]);
#pragma unroll
        for (int s = 0; s < BK / 16; ++s) {
            const int c = s & 1;
            if (s + 1 < BK / 16) read_frags(s + 1, fa[c ^ 1], fb[c ^ 1]);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) acc[i][j] = mfma32(fa[c][i], fb[c][j], acc[i][j]);
        }
        // Instruction order for the scheduler: the first slice's reads, then
        // per slice one next-slice read after each of the first TM + TN
        // MFMAs.  Left alone, the compiler issues each slice's reads right
        // before the MFMAs that use them and waits for them there (gate/up
        // and down +4-5% with the interleave).
        constexpr int NR = TM + TN, NM = TM * TN;
        if constexpr (NM >= NR) {
            __builtin_amdgcn_sched_group_barrier(0x100, NR, 0);  // 0x100: LDS reads
#pragma unroll
            for (int s = 0; s < BK / 16; ++s) {
                if (s + 1 < BK / 16) {
#pragma unroll
                    for (int r = 0; r < NR; ++r) {
                        __builtin_amdgcn_sched_group_barrier(0x8, 1, 0);  // 0x8: MFMA
                        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                    }
                    if constexpr (NM > NR) __builtin_amdgcn_sched_group_barrier(0x8, NM - NR, 0);
                } else {
                    __builtin_amdgcn_sched_group_barrier(0x8, NM, 0);
                }
            }
        }
    };

    if constexpr (RING == 0) {
        int a_off[A_LOADS], a_lds[A_LOADS];
#pragma unroll
        for (int i = 0; i < A_LOADS; ++i) {
            const int idx = tid + i * THREADS, row = idx / CPR, ch = idx % CPR;
            a_off[i] = min(m0 + row, g.m - 1) * g.lda + ch * 8;
            a_lds[i] = row * BK + swz<BK>(row, ch) * 8;
        }
        int b_off[B_LOADS], b_lds[B_LOADS];
#pragma unroll
        for (int i = 0; i < B_LOADS; ++i) {
            const int idx = tid + i * THREADS, row = idx / CPR, ch = idx % CPR;
            b_off[i] = w_row<EPI>(g, n0 + row) * g.k + ch * 8;
            b_lds[i] = row * BK + swz<BK>(row, ch) * 8;
        }
        bf16x8 ra[A_LOADS], rb[B_LOADS];
        auto load_tile = [&](int kt) {
            const bf16* Ak = A + kt * BK;
            const bf16* Wk = W + kt * BK;
#pragma unroll
            for (int i = 0; i < A_LOADS; ++i) ra[i] = *reinterpret_cast<const bf16x8*>(Ak + a_off[i]);
#pragma unroll
            for (int i = 0; i < B_LOADS; ++i) rb[i] = *reinterpret_cast<const bf16x8*>(Wk + b_off[i]);
        };
        auto store_tile = [&](int buf) {
#pragma unroll
            for (int i = 0; i < A_LOADS; ++i) *reinterpret_cast<bf16x8*>(&As[buf][a_lds[i]]) = ra[i];
#pragma unroll
            for (int i = 0; i < B_LOADS; ++i) *reinterpret_cast<bf16x8*>(&Bs[buf][b_lds[i]]) = rb[i];
        };
        load_tile(0);
        store_tile(0);
        __syncthreads();
        for (int kt = 0; kt < nk; ++kt) {
            const int buf = kt & 1;
            if (kt + 1 < nk) load_tile(kt + 1);
            compute(buf);
            if (kt + 1 < nk) store_tile(buf ^ 1);
            __syncthreads();
        }
    } else {
        // One direct load fills 1 KB of LDS: RPI rows of BK values.  Wave w
        // issues A loads w, w + NW, ... and B loads likewise.
        constexpr int NW = WAVES_M * WAVES_N;
        constexpr int RPI = 64 / CPR;
        constexpr int A_INS = BM / RPI / NW, B_INS = BN / RPI / NW;
        constexpr int PER_STEP = A_INS + B_INS;
        static_assert(BM % (RPI * NW) == 0 && BN % (RPI * NW) == 0, "direct loads must split evenly");
        static_assert(RING >= 2 && RING <= 4, "the counted waits cover rings of two to four buffers");
        const int r_in = lane / CPR, stored = lane % CPR;
        const bf16* a_src[A_INS];
        int a_dst[A_INS];
#pragma unroll
        for (int i = 0; i < A_INS; ++i) {
            const int row = (wave + i * NW) * RPI + r_in;
            const int ch = stored ^ ((row / (16 / CPR)) & (CPR - 1));  // logical chunk stored at this slot
            a_src[i] = A + static_cast<size_t>(min(m0 + row, g.m - 1)) * g.lda + ch * 8;
            a_dst[i] = (wave + i * NW) * RPI * BK;
        }
        const bf16* b_src[B_INS];
        int b_dst[B_INS];
#pragma unroll
        for (int i = 0; i < B_INS; ++i) {
            const int row = (wave + i * NW) * RPI + r_in;
            const int ch = stored ^ ((row / (16 / CPR)) & (CPR - 1));
            b_src[i] = W + static_cast<size_t>(w_row<EPI>(g, n0 + row)) * g.k + ch * 8;
            b_dst[i] = (wave + i * NW) * RPI * BK;
        }
        auto issue = [&](int kt) {
            const int buf = kt % RING;
#pragma unroll
            for (int i = 0; i < A_INS; ++i)
                load_lds16(a_src[i] + kt * BK, &As[buf][a_dst[i]]);
#pragma unroll
            for (int i = 0; i < B_INS; ++i)
                load_lds16(b_src[i] + kt * BK, &Bs[buf][b_dst[i]]);
        };
#pragma unroll
        for (int s = 0; s < RING - 1; ++s)
            if (s < nk) issue(s);
        for (int kt = 0; kt < nk; ++kt) {
            // this wave's loads of step kt are done once at most the younger
            // steps' loads (up to RING - 2 of them) are outstanding
            const int younger = min(nk - 1 - kt, RING - 2);
            if (RING >= 4 && younger >= 2) wait_vmcnt<2 * PER_STEP>();
            else if (RING >= 3 && younger >= 1) wait_vmcnt<PER_STEP>();
            else wait_vmcnt<0>();
            barrier_only();
            if (kt + RING - 1 < nk) issue(kt + RING - 1);
            compute(kt % RING);
        }
    }
}

// Fused epilogue of one tile: element e of MFMA tile (i, j) of a wave is row
// m0 + wm WM + 32 i + 8 (e / 4) + 4 (lane / 32) + e % 4, B column
// n0 + wn WN + 32 j + lane % 32.  The epilogue's inputs (RoPE table,
// residual) are read for a whole block of rows before any of its stores:
// the compiler cannot tell that the stores do not alias them, so reads and
// stores interleaved per element would each wait out a memory round trip.
// Reads of rows past m are clamped to row m - 1 and their stores skipped.
template <int BM, int BN, int WAVES_M, int WAVES_N, int EPI>
__device__ __forceinline__ void tile_store(const GemmArgs& g, int m0, int n0,
                                           const f32x16 (&acc)[BM / WAVES_M / 32][BN / WAVES_N / 32]) {
    constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
    constexpr int TM = WM / 32, TN = WN / 32;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    const int rbase = m0 + wm * WM + 4 * (lane >> 5);
    const int cbase = n0 + wn * WN + (lane & 31);
    if (EPI == EPI_SWIGLU || EPI == EPI_QKV) {
        bf16* out = static_cast<bf16*>(g.out);
#pragma unroll
        for (int pr = 0; pr < TN / 2; ++pr) {
            const int c0 = n0 + wn * WN + pr * 64;  // first B column of the pair (tile 2pr)
            int hg = 0, d0 = 0, fcol = 0;
            if (EPI == EPI_QKV) {
                hg = c0 / g.hd;
                d0 = ((c0 % g.hd) / 64) * 32 + (lane & 31);
            } else {
                fcol = (c0 >> 1) + (lane & 31);
            }
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                float2 cs[16];
                int sl[16];
                if (EPI == EPI_QKV) {
                    const bool rot = hg < g.hq + g.hkv, paged = hg >= g.hq;
#pragma unroll
                    for (int e = 0; e < 16; ++e) {
                        const int row = min(rbase + i * 32 + 8 * (e >> 2) + (e & 3), g.m - 1);
                        cs[e] = rot ? g.rope_cs[row * (g.hd / 2) + d0] : make_float2(1.f, 0.f);
                        sl[e] = paged ? g.slot[row] : 0;
                    }
                }
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int row = rbase + i * 32 + 8 * (e >> 2) + (e & 3);
                    if (row >= g.m) continue;
                    const float x0 = acc[i][2 * pr][e], x1 = acc[i][2 * pr + 1][e];
                    if (EPI == EPI_QKV) qkv_store_cs(g, row, hg, d0, x0, x1, cs[e], sl[e]);
                    else out[static_cast<size_t>(row) * g.ldo + fcol] = f2bf(silu(x0) * x1);
                }
            }
        }
        return;
    }
#pragma unroll
    for (int i = 0; i < TM; ++i) {
        float r[TN][16];
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int row = min(rbase + i * 32 + 8 * (e >> 2) + (e & 3), g.m - 1);
                const size_t o = static_cast<size_t>(row) * g.ldo + cbase + j * 32;
                r[j][e] = EPI == EPI_RESID_F32OUT ? bf2f(static_cast<const bf16*>(g.resid)[o])
                                                  : static_cast<const float*>(g.resid)[o];
            }
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int row = rbase + i * 32 + 8 * (e >> 2) + (e & 3);
                if (row >= g.m) continue;
                const size_t o = static_cast<size_t>(row) * g.ldo + cbase + j * 32;
                if (EPI == EPI_RESID_F32OUT)
                    static_cast<float*>(g.out)[o] = acc[i][j][e] + r[j][e];
                else
                    static_cast<bf16*>(g.out)[o] = f2bf(acc[i][j][e] + r[j][e]);
            }
    }
}

// Split-K partial of one tile into P [m][n] (B column order).
template <int BM, int BN, int WAVES_M, int WAVES_N, int EPI>
__device__ __forceinline__ void tile_store_split(const GemmArgs& g, int m0, int n0, float* __restrict__ P,
                                       const f32x16 (&acc)[BM / WAVES_M / 32][BN / WAVES_N / 32]) {
    constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
    constexpr int TM = WM / 32, TN = WN / 32;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    const int rbase = m0 + wm * WM + 4 * (lane >> 5);
    const int cbase = n0 + wn * WN + (lane & 31);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int row = rbase + i * 32 + 8 * (e >> 2) + (e & 3);
                if (row < g.m) P[static_cast<size_t>(row) * g.n + cbase + j * 32] = acc[i][j][e];
            }
}

// Stream-K partial of one tile into P [BM][BN] (tile rows, B column order).
template <int BM, int BN, int WAVES_M, int WAVES_N>
__device__ __forceinline__ void tile_store_partial(float* __restrict__ P,
                                                   const f32x16 (&acc)[BM / WAVES_M / 32][BN / WAVES_N / 32]) {
    constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
    constexpr int TM = WM / 32, TN = WN / 32;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    const int rbase = wm * WM + 4 * (lane >> 5);
    const int cbase = wn * WN + (lane & 31);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e)
                P[(rbase + i * 32 + 8 * (e >> 2) + (e & 3)) * BN + cbase + j * 32] = acc[i][j][e];
}

template <int BM, int BN, int WAVES_M, int WAVES_N, int BK, int RING, int EPI, bool SPLIT>
__global__ __launch_bounds__(WAVES_M * WAVES_N * 64, (BK == 32 && RING == 0) ? 2 : 1) void gemm_kernel(
    GemmArgs g, float* __restrict__ partial, int k_per_split) {
    constexpr int NBUF = RING == 0 ? 2 : RING;
    __shared__ __attribute__((aligned(16))) bf16 As[NBUF][BM * BK];
    __shared__ __attribute__((aligned(16))) bf16 Bs[NBUF][BN * BK];
    int tm, tn;
    tile_of(blockIdx.x, (g.m + BM - 1) / BM, g.n / BN, tm, tn);
    f32x16 acc[BM / WAVES_M / 32][BN / WAVES_N / 32];
    tile_mainloop<BM, BN, WAVES_M, WAVES_N, BK, RING, EPI>(g, tm * BM, tn * BN, blockIdx.y * k_per_split,
                                                          k_per_split / BK, As, Bs, acc);
    if (SPLIT)
        tile_store_split<BM, BN, WAVES_M, WAVES_N, EPI>(
            g, tm * BM, tn * BN, partial + static_cast<size_t>(blockIdx.y) * g.m * g.n, acc);
    else
        tile_store<BM, BN, WAVES_M, WAVES_N, EPI>(g, tm * BM, tn * BN, acc);
}

// Stream-K schedule: whole tiles first, then equal shares of k steps.
// Blocks [0, dp_tiles) each run one whole tile of the first dp_tiles of the
// tile order.  The k steps of the remaining tiles, laid end to end (`iters`
// of them), are cut into `workers` equal ranges, worker w taking
// [w iters / workers, (w + 1) iters / workers).  A range covers the tail of
// one tile, whole tiles and the head of another; whole tiles get the fused
// epilogue, pieces are stored as partials in slot 2w (the range's first
// piece) or 2w + 1 (its last) and summed by sk_fixup_kernel.  No block waits
// for another.
__device__ __forceinline__ int64_t sk_range_start(int w, int64_t iters, int workers) {
    return static_cast<int64_t>(w) * iters / workers;
}
// Worker whose range holds step x: the largest w with w iters / workers <= x.
__device__ __forceinline__ int sk_worker_of(int64_t x, int64_t iters, int workers) {
    return static_cast<int>(((x + 1) * workers - 1) / iters);
}

// One piece of a stream-K range: k steps [k0, k1) of tile t, stored whole or
// as the partial in `slot`.  Kept out of line: inlined into the loop over a
// range's pieces, the tile code spills its accumulators.
template <int BM, int BN, int WAVES_M, int WAVES_N, int BK, int RING, int EPI>
__device__ __noinline__ void sk_piece(const GemmArgs& g, float* __restrict__ partial, int t, int k0, int k1, int slot) {
    constexpr int NBUF = RING == 0 ? 2 : RING;
    __shared__ __attribute__((aligned(16))) bf16 As[NBUF][BM * BK];
    __shared__ __attribute__((aligned(16))) bf16 Bs[NBUF][BN * BK];
    const int nt_m = (g.m + BM - 1) / BM, nt_n = g.n / BN;
    const int nk = g.k / BK;
    f32x16 acc[BM / WAVES_M / 32][BN / WAVES_N / 32];
    int tm, tn;
    tile_coords(t, nt_m, nt_n, tm, tn);
    tile_mainloop<BM, BN, WAVES_M, WAVES_N, BK, RING, EPI>(g, tm * BM, tn * BN, k0 * BK, k1 - k0, As, Bs, acc);
    if (k0 == 0 && k1 == nk)
        tile_store<BM, BN, WAVES_M, WAVES_N, EPI>(g, tm * BM, tn * BN, acc);
    else
        tile_store_partial<BM, BN, WAVES_M, WAVES_N>(partial + static_cast<size_t>(slot) * BM * BN, acc);
}

template <int BM, int BN, int WAVES_M, int WAVES_N, int BK, int RING, int EPI>
__global__ __launch_bounds__(WAVES_M * WAVES_N * 64, (BK == 32 && RING == 0) ? 2 : 1) void gemm_sk_kernel(
    GemmArgs g, float* __restrict__ partial, int dp_tiles, int workers) {
    const int nt_m = (g.m + BM - 1) / BM, nt_n = g.n / BN;
    const int nk = g.k / BK;
    // Steps of all tiles in one space, the whole tiles first: a whole-tile
    // block's range is its tile, worker w's range follows dp_tiles * nk.
    const int bid = blockIdx.x;
    const int64_t iters = static_cast<int64_t>(nt_m * nt_n - dp_tiles) * nk;
    int w = 0;
    int64_t lo, hi;
    if (bid < dp_tiles) {
        lo = static_cast<int64_t>(xcd_order(bid, dp_tiles)) * nk;
        hi = lo + nk;
    } else {
        // workers on one XCD take consecutive ranges (dp_tiles is a multiple of 8)
        w = xcd_order(bid - dp_tiles, workers);
        lo = static_cast<int64_t>(dp_tiles) * nk + sk_range_start(w, iters, workers);
        hi = static_cast<int64_t>(dp_tiles) * nk + sk_range_start(w + 1, iters, workers);
    }
    for (int64_t it = lo; it < hi;) {
        const int t = static_cast<int>(it / nk);
        const int k0 = static_cast<int>(it - static_cast<int64_t>(t) * nk);
        const int k1 = static_cast<int>(min<int64_t>(nk, k0 + (hi - it)));
        if (it != lo) __syncthreads();  // every wave is done with the previous piece's LDS buffers
        sk_piece<BM, BN, WAVES_M, WAVES_N, BK, RING, EPI>(g, partial, t, k0, k1, 2 * w + (it == lo ? 0 : 1));
        it += k1 - k0;
    }
}

// Sum the partial pieces of each stream-K tile that several workers shared
// and apply the epilogue.  Block (x, y): tile dp_tiles + x of the order,
// y-th group of 256 output units (a RoPE pair, or four outputs).
template <int BM, int BN, int BK, int EPI>
__global__ __launch_bounds__(256) void sk_fixup_kernel(GemmArgs g, const float* __restrict__ partial, int dp_tiles,
                                                       int workers) {
    const int nt_m = (g.m + BM - 1) / BM, nt_n = g.n / BN;
    const int nk = g.k / BK;
    const int64_t iters = static_cast<int64_t>(nt_m * nt_n - dp_tiles) * nk;
    const int t = blockIdx.x;
    const int64_t t0 = static_cast<int64_t>(t) * nk;
    const int wa = sk_worker_of(t0, iters, workers), wb = sk_worker_of(t0 + nk - 1, iters, workers);
    if (wa == wb) return;  // one worker ran the whole tile and stored it
    int tm, tn;
    tile_coords(dp_tiles + t, nt_m, nt_n, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;
    // slot of worker w's piece of this tile: its first piece unless its range starts before the tile
    auto slot_of = [&](int w) { return 2 * w + (sk_range_start(w, iters, workers) < t0 ? 1 : 0); };
    const int u = blockIdx.y * 256 + threadIdx.x;
    if (EPI == EPI_QKV) {  // one unit per RoPE pair
        const int half = g.hd / 2, pairs = BN / 2;
        if (u >= BM * pairs) return;
        const int r = u / pairs, j = u % pairs;
        if (m0 + r >= g.m) return;
        const int hl = j / half, d0 = j % half;
        const int c0 = hl * g.hd + qkv_dim(d0, g.hd), c1 = hl * g.hd + qkv_dim(d0 + half, g.hd);
        float x0 = 0.f, x1 = 0.f;
        for (int w = wa; w <= wb; ++w) {
            const float* P = partial + static_cast<size_t>(slot_of(w)) * BM * BN + r * BN;
            x0 += P[c0];
            x1 += P[c1];
        }
        qkv_store(g, m0 + r, n0 / g.hd + hl, d0, x0, x1);
        return;
    }
    const int n_out = EPI == EPI_SWIGLU ? BN / 2 : BN;
    const int per_row = n_out / 4;
    if (u >= BM * per_row) return;
    const int r = u / per_row, c4 = (u % per_row) * 4;
    if (m0 + r >= g.m) return;
    if (EPI == EPI_SWIGLU) {
        const int gc = (c4 >> 5) * 64 + (c4 & 31);  // gate column in B order; up is +32
        f32x4 gs = {}, us = {};
        for (int w = wa; w <= wb; ++w) {
            const float* P = partial + static_cast<size_t>(slot_of(w)) * BM * BN + r * BN + gc;
            gs += *reinterpret_cast<const f32x4*>(P);
            us += *reinterpret_cast<const f32x4*>(P + 32);
        }
        bf16* out = static_cast<bf16*>(g.out) + static_cast<size_t>(m0 + r) * g.ldo + n0 / 2 + c4;
#pragma unroll
        for (int e = 0; e < 4; ++e) out[e] = f2bf(silu(gs[e]) * us[e]);
        return;
    }
    f32x4 sum = {};
    for (int w = wa; w <= wb; ++w)
        sum += *reinterpret_cast<const f32x4*>(partial + static_cast<size_t>(slot_of(w)) * BM * BN + r * BN + c4);
    const size_t o = static_cast<size_t>(m0 + r) * g.ldo + n0 + c4;
    if (EPI == EPI_RESID_F32OUT) {
        const bf16* rs = static_cast<const bf16*>(g.resid) + o;
#pragma unroll
        for (int e = 0; e < 4; ++e) sum[e] += bf2f(rs[e]);
        *reinterpret_cast<f32x4*>(static_cast<float*>(g.out) + o) = sum;
    } else {
        sum += *reinterpret_cast<const f32x4*>(static_cast<const float*>(g.resid) + o);
        bf16* out = static_cast<bf16*>(g.out) + o;
#pragma unroll
        for (int e = 0; e < 4; ++e) out[e] = f2bf(sum[e]);
    }
}

// Sum split-K partials [splits][m][n] (B column order) and apply the epilogue.
template <int EPI>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(GemmArgs g, const float* __restrict__ part,
                                                            int splits) {
    const size_t slab = static_cast<size_t>(g.m) * g.n;
    const size_t idx = blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x;
    if (EPI == EPI_QKV) {  // one thread per RoPE pair
        const int pairs = g.n / 2, half = g.hd / 2;
        if (idx >= static_cast<size_t>(g.m) * pairs) return;
        const int row = static_cast<int>(idx / pairs), j = static_cast<int>(idx % pairs);
        const int hg = j / half, d0 = j % half;
        const size_t c0 = static_cast<size_t>(hg) * g.hd + qkv_dim(d0, g.hd);
        const size_t c1 = static_cast<size_t>(hg) * g.hd + qkv_dim(d0 + half, g.hd);
        float x0 = 0.f, x1 = 0.f;
        for (int z = 0; z < splits; ++z) {
            const float* p = part + z * slab + static_cast<size_t>(row) * g.n;
            x0 += p[c0];
            x1 += p[c1];
        }
        qkv_store(g, row, hg, d0, x0, x1);
        return;
    }
    const int n_out = (EPI == EPI_SWIGLU) ? g.n / 2 : g.n;
    const int per_row = n_out / 4;
    if (idx >= static_cast<size_t>(g.m) * per_row) return;
    const int row = static_cast<int>(idx / per_row);
    const int c4 = static_cast<int>(idx % per_row) * 4;
    const size_t o = static_cast<size_t>(row) * g.ldo + c4;
    if (EPI == EPI_SWIGLU) {
        const int gc = (c4 >> 5) * 64 + (c4 & 31);  // gate column in B order; up is +32
        f32x4 gs = {}, us = {};
        for (int z = 0; z < splits; ++z) {
            const float* p = part + z * slab + static_cast<size_t>(row) * g.n + gc;
            gs += *reinterpret_cast<const f32x4*>(p);
            us += *reinterpret_cast<const f32x4*>(p + 32);
        }
        bf16* out = static_cast<bf16*>(g.out) + o;
#pragma unroll
        for (int e = 0; e < 4; ++e) out[e] = f2bf(silu(gs[e]) * us[e]);
        return;
    }
    f32x4 s = {};
    for (int z = 0; z < splits; ++z)
        s += *reinterpret_cast<const f32x4*>(part + z * slab + static_cast<size_t>(row) * g.n + c4);
    if (EPI == EPI_RESID_F32OUT) {
        const bf16* r = static_cast<const bf16*>(g.resid) + o;
#pragma unroll
        for (int e = 0; e < 4; ++e) s[e] += bf2f(r[e]);
        *reinterpret_cast<f32x4*>(static_cast<float*>(g.out) + o) = s;
    } else {
        s += *reinterpret_cast<const f32x4*>(static_cast<const float*>(g.resid) + o);
        bf16* out = static_cast<bf16*>(g.out) + o;
#pragma unroll
        for (int e = 0; e < 4; ++e) out[e] = f2bf(s[e]);
    }
}

// Weight-streaming GEMM for small m (at most 32 T rows).  W is read once,
// straight from memory into MFMA operand registers with no LDS staging, so
// the bytes in flight per CU are bounded only by registers and occupancy.
// A work-group has KS waves that split its k range; every wave computes the
// same 64 B columns (two 32-column groups that pair like the tile kernel's
// epilogue tiles) for all tokens over its k slice, and the slices are summed
// through LDS before the epilogue.  Work-groups are small so that several
// share a CU and the whole grid runs in one round.
// In a 64-wide k step a lane reads 64 contiguous bytes of its row (lanes
// 0-31 the first 32 k, lanes 32-63 the next 32); the step's four MFMAs take
// its 16-byte quarters.  Both operands use this same order of k inside the
// step, so every dot product is unchanged.  MFMA rows are W rows and columns
// are tokens: element e of lane l is W row 8(e/4) + 4(l/32) + e%4 of its
// column group, token 32 t + l%32.
template <int T, int EPI, bool SPLIT>
__global__ __launch_bounds__(256) void skinny_kernel(GemmArgs g, float* __restrict__ partial, int k_per_split,
                                                     int ks_count) {
    constexpr int NA = 2 * T;  // accumulator tiles: 2 column groups x T token groups
    __shared__ float red[2][NA * 16][64];  // ks_count / 2 <= 2 slots

    const int lane = threadIdx.x & 63, ks = threadIdx.x >> 6;
    const int r = lane & 31, h = lane >> 5;
    const int c0 = blockIdx.x * 64;
    const int k_wave = k_per_split / ks_count;
    const int kbeg = blockIdx.y * k_per_split + ks * k_wave + 32 * h;
    const int nkb = k_wave / 64;

    const bf16* W = static_cast<const bf16*>(g.w);
    const bf16* A = static_cast<const bf16*>(g.a);
    const bf16* wp[2];
    wp[0] = W + static_cast<size_t>(w_row<EPI>(g, c0 + r)) * g.k + kbeg;
    wp[1] = W + static_cast<size_t>(w_row<EPI>(g, c0 + 32 + r)) * g.k + kbeg;
    const bf16* ap[T];
#pragma unroll
    for (int t = 0; t < T; ++t)  // rows past m read row m-1; their results are never stored
        ap[t] = A + static_cast<size_t>(min(t * 32 + r, g.m - 1)) * g.lda + kbeg;

    bf16x8 wf[2][2][4], af[2][T][4];
    auto load = [&](int kb, int b) {
        const int off = kb * 64;
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
            for (int j = 0; j < 4; ++j) wf[b][c][j] = *reinterpret_cast<const bf16x8*>(wp[c] + off + 8 * j);
#pragma unroll
        for (int t = 0; t < T; ++t)
#pragma unroll
            for (int j = 0; j < 4; ++j) af[b][t][j] = *reinterpret_cast<const bf16x8*>(ap[t] + off + 8 * j);
    };
    f32x16 acc[2][T];
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int t = 0; t < T; ++t) acc[c][t] = f32x16{};
    auto compute = [&](int b) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int c = 0; c < 2; ++c)
#pragma unroll
                for (int t = 0; t < T; ++t) acc[c][t] = mfma32(wf[b][c][j], af[b][t][j], acc[c][t]);
    };

    load(0, 0);
    for (int kb = 0; kb < nkb; kb += 2) {
        if (kb + 1 < nkb) load(kb + 1, 1);
        compute(0);
        if (kb + 1 >= nkb) break;
        if (kb + 2 < nkb) load(kb + 2, 0);
        compute(1);
    }

    // Sum the k slices: halve the active slices per round.
    for (int half = ks_count / 2; half >= 1; half /= 2) {
        if (ks >= half && ks < 2 * half) {
#pragma unroll
            for (int c = 0; c < 2; ++c)
#pragma unroll
                for (int t = 0; t < T; ++t)
#pragma unroll
                    for (int e = 0; e < 16; ++e) red[ks - half][(c * T + t) * 16 + e][lane] = acc[c][t][e];
        }
        __syncthreads();
        if (ks < half) {
#pragma unroll
            for (int c = 0; c < 2; ++c)
#pragma unroll
                for (int t = 0; t < T; ++t)
#pragma unroll
                    for (int e = 0; e < 16; ++e) acc[c][t][e] += red[ks][(c * T + t) * 16 + e][lane];
        }
        __syncthreads();
    }
    if (ks != 0) return;

#pragma unroll
    for (int t = 0; t < T; ++t) {
        const int row = t * 32 + r;
        if (row >= g.m) continue;
#pragma unroll
        for (int e4 = 0; e4 < 4; ++e4) {
            const int i0 = 8 * e4 + 4 * h;  // W row of element 4 e4 within its column group
            if (SPLIT) {
                float* P = partial + (static_cast<size_t>(blockIdx.y) * g.m + row) * g.n + c0 + i0;
#pragma unroll
                for (int c = 0; c < 2; ++c)
                    *reinterpret_cast<f32x4*>(P + 32 * c) =
                        f32x4{acc[c][t][4 * e4], acc[c][t][4 * e4 + 1], acc[c][t][4 * e4 + 2], acc[c][t][4 * e4 + 3]};
                continue;
            }
            if (EPI == EPI_QKV) {
                // rotations (and the KV slot) read before any store, which the
                // compiler cannot tell apart from the tables
                const int hg = c0 / g.hd, d0 = ((c0 % g.hd) / 64) * 32 + i0;
                const bool rot = hg < g.hq + g.hkv;
                float2 cs[4];
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    cs[q] = rot ? g.rope_cs[row * (g.hd / 2) + d0 + q] : make_float2(1.f, 0.f);
                const int slot = hg < g.hq ? 0 : g.slot[row];
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    qkv_store_cs(g, row, hg, d0 + q, acc[0][t][4 * e4 + q], acc[1][t][4 * e4 + q], cs[q], slot);
            } else if (EPI == EPI_SWIGLU) {
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    static_cast<bf16*>(g.out)[static_cast<size_t>(row) * g.ldo + (c0 >> 1) + i0 + q] =
                        f2bf(silu(acc[0][t][4 * e4 + q]) * acc[1][t][4 * e4 + q]);
            } else {
                // four consecutive output columns per lane: one vector read of
                // the residual and one vector store for each 32-column group
                f32x4 rv[2];
#pragma unroll
                for (int c = 0; c < 2; ++c) {
                    const size_t o = static_cast<size_t>(row) * g.ldo + c0 + 32 * c + i0;
                    if (EPI == EPI_RESID_F32OUT) {
                        const bf16x4 rb = *reinterpret_cast<const bf16x4*>(static_cast<const bf16*>(g.resid) + o);
                        rv[c] = f32x4{bf2f(rb[0]), bf2f(rb[1]), bf2f(rb[2]), bf2f(rb[3])};
                    } else {
                        rv[c] = *reinterpret_cast<const f32x4*>(static_cast<const float*>(g.resid) + o);
                    }
                }
#pragma unroll
                for (int c = 0; c < 2; ++c) {
                    const size_t o = static_cast<size_t>(row) * g.ldo + c0 + 32 * c + i0;
                    const f32x4 v = f32x4{acc[c][t][4 * e4], acc[c][t][4 * e4 + 1], acc[c][t][4 * e4 + 2],
                                          acc[c][t][4 * e4 + 3]} + rv[c];
                    if (EPI == EPI_RESID_F32OUT) {
                        *reinterpret_cast<f32x4*>(static_cast<float*>(g.out) + o) = v;
                    } else {
                        const bf16x4 ob = {f2bf(v[0]), f2bf(v[1]), f2bf(v[2]), f2bf(v[3])};
                        *reinterpret_cast<bf16x4*>(static_cast<bf16*>(g.out) + o) = ob;
                    }
                }
            }
        }
    }
}

// Narrow GEMM for m <= 32 rows (decode-sized batches): a work-group of KS
// waves owns 16 output columns (CG == 1) or a RoPE / SwiGLU pair of 16-column
// groups 32 apart (CG == 2) and all m rows; each wave takes K / KS of the k
// range, so every weight byte is read once, and the waves' sums are added in
// LDS before the fused epilogue: no split of k across work-groups, no second
// kernel.  16 x 16 x 32 MFMAs with the weights as the A operand: a 64-lane
// operand load reads 64 contiguous bytes of each of 16 weight rows (16 cache
// lines, against 32 for a 32-row operand).  Four k slices of 32 are kept in
// flight per wave in a ring of registers.
constexpr int kNarrowMaxWaves = 8;
template <int T, int CG, int EPI>
__global__ __launch_bounds__(64 * kNarrowMaxWaves) void narrow_kernel(GemmArgs g, int ks_count) {
    constexpr int R = 4;  // slices in flight
    __shared__ f32x4 red[kNarrowMaxWaves][CG * T][64];
    const int lane = threadIdx.x & 63, ks = threadIdx.x >> 6;
    const int j = lane & 15, grp = lane >> 4;
    // first column of each group: CG == 2 takes 16 columns of a 64-column
    // tile and their partners 32 further on
    int col0[CG];
    if constexpr (CG == 2) {
        const int tile64 = (blockIdx.x >> 1) * 64, half = (blockIdx.x & 1) * 16;
        col0[0] = tile64 + half;
        col0[1] = tile64 + 32 + half;
    } else {
        col0[0] = blockIdx.x * 16;
    }
    const int k_wave = g.k / ks_count;
    const int kbeg = ks * k_wave + 8 * grp;
    const int nslice = k_wave / 32;
    const bf16* W = static_cast<const bf16*>(g.w);
    const bf16* A = static_cast<const bf16*>(g.a);
    const bf16* wp[CG];
#pragma unroll
    for (int c = 0; c < CG; ++c) wp[c] = W + static_cast<size_t>(w_row<EPI>(g, col0[c] + j)) * g.k + kbeg;
    const bf16* ap[T];
#pragma unroll
    for (int t = 0; t < T; ++t)  // rows past m read row m - 1; their results are never stored
        ap[t] = A + static_cast<size_t>(min(t * 16 + j, g.m - 1)) * g.lda + kbeg;

    bf16x8 wf[R][CG], af[R][T];
    auto load = [&](int sl, int b) {
#pragma unroll
        for (int c = 0; c < CG; ++c) wf[b][c] = *reinterpret_cast<const bf16x8*>(wp[c] + 32 * sl);
#pragma unroll
        for (int t = 0; t < T; ++t) af[b][t] = *reinterpret_cast<const bf16x8*>(ap[t] + 32 * sl);
    };
    f32x4 acc[CG][T];
#pragma unroll
    for (int c = 0; c < CG; ++c)
#pragma unroll
        for (int t = 0; t < T; ++t) acc[c][t] = f32x4{};
#pragma unroll
    for (int b = 0; b < R; ++b)
        if (b < nslice) load(b, b);
    for (int s0 = 0; s0 < nslice; s0 += R) {
#pragma unroll
        for (int b = 0; b < R; ++b) {
            if (s0 + b < nslice) {
#pragma unroll
                for (int c = 0; c < CG; ++c)
#pragma unroll
                    for (int t = 0; t < T; ++t) acc[c][t] = mfma16(wf[b][c], af[b][t], acc[c][t]);
                if (s0 + b + R < nslice) load(s0 + b + R, b);
            }
        }
    }

    // Sum over the waves; wave t then stores token group t.
#pragma unroll
    for (int c = 0; c < CG; ++c)
#pragma unroll
        for (int t = 0; t < T; ++t) red[ks][c * T + t][lane] = acc[c][t];
    __syncthreads();
    if (ks >= T) return;
    const int t = ks;
    f32x4 v[CG];
#pragma unroll
    for (int c = 0; c < CG; ++c) {
        v[c] = red[0][c * T + t][lane];
        for (int w = 1; w < ks_count; ++w) v[c] += red[w][c * T + t][lane];
    }
    const int row = t * 16 + j;
    if (row >= g.m) return;
    // element e of a lane: column col0[c] + 4 grp + e of row `row`
    if constexpr (EPI == EPI_QKV) {
        const int tile64 = col0[0] - (blockIdx.x & 1) * 16;
        const int hg = tile64 / g.hd, d0 = ((tile64 % g.hd) / 64) * 32 + (col0[0] - tile64) + 4 * grp;
#pragma unroll
        for (int e = 0; e < 4; ++e) qkv_store(g, row, hg, d0 + e, v[0][e], v[CG - 1][e]);
    } else if constexpr (EPI == EPI_SWIGLU) {
        const int tile64 = col0[0] - (blockIdx.x & 1) * 16;
        bf16* out = static_cast<bf16*>(g.out) + static_cast<size_t>(row) * g.ldo + (tile64 >> 1) +
                    (col0[0] - tile64) + 4 * grp;
        bf16x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = f2bf(silu(v[0][e]) * v[CG - 1][e]);
        *reinterpret_cast<bf16x4*>(out) = o;
    } else {
        const size_t o = static_cast<size_t>(row) * g.ldo + col0[0] + 4 * grp;
        if constexpr (EPI == EPI_RESID_F32OUT) {
            const bf16x4 rb = *reinterpret_cast<const bf16x4*>(static_cast<const bf16*>(g.resid) + o);
            *reinterpret_cast<f32x4*>(static_cast<float*>(g.out) + o) =
                v[0] + f32x4{bf2f(rb[0]), bf2f(rb[1]), bf2f(rb[2]), bf2f(rb[3])};
        } else {
            const f32x4 r = *reinterpret_cast<const f32x4*>(static_cast<const float*>(g.resid) + o) + v[0];
            *reinterpret_cast<bf16x4*>(static_cast<bf16*>(g.out) + o) = bf16x4{f2bf(r[0]), f2bf(r[1]), f2bf(r[2]), f2bf(r[3])};
        }
    }
}

struct TileCfg {
    int bm, bn, waves_m, waves_n, bk, ring;  // ring 0: register-staged double buffer
};
// BM x BN / waves (per-wave tile), k depth per stage, main loop, LDS:
// 0: 128x128 / 4 (64x64), k 64, register-staged (64 KB: two work-groups per CU)
// 1: 64x128 / 4 (32x64), k 64, register-staged (the fallback when n is not a
//    multiple of 256)
// 2: 256x128 / 4 (128x64), k 32, register-staged (48 KB: two per CU)
// 3: 256x256 / 8 (128x64), k 64, 2-buffer direct-load ring (128 KB)
// 4: 192x256 / 8 (96x64), k 64, 2-buffer ring (112 KB): less row padding
//    than 256 where m is just past a multiple of 256
// 5: 128x128 / 4 (64x64), k 64, 2-buffer ring (64 KB: two per CU)
// 6: 96x256 / 4 (96x64), k 64, 3-buffer ring (132 KB): a single row tile
//    for m up to 96, three stages of weights in flight
// 7: 160x256 / 4 (160x64), k 64, 2-buffer ring (104 KB)
// 8: 128x128 / 4 (64x64), k 64, 4-buffer ring (128 KB)
// 9: 64x256 / 4 (64x64), k 64, 3-buffer ring (120 KB)
// 10: 128x128 / 4 (64x64), k 64, 3-buffer ring (96 KB)
// The deep rings of the small-m tiles keep more weight bytes in flight per
// CU, which is what the weight-streaming shapes are short of.
constexpr TileCfg kCfgs[] = {{128, 128, 2, 2, 64, 0}, {64, 128, 2, 2, 64, 0}, {256, 128, 2, 2, 32, 0},
                             {256, 256, 2, 4, 64, 2}, {192, 256, 2, 4, 64, 2}, {128, 128, 2, 2, 64, 2},
                             {96, 256, 1, 4, 64, 3},  {160, 256, 1, 4, 64, 2}, {128, 128, 2, 2, 64, 4},
                             {64, 256, 1, 4, 64, 3},  {128, 128, 2, 2, 64, 3}};
constexpr int kNumCfgs = sizeof(kCfgs) / sizeof(kCfgs[0]);

template <int EPI>
void launch_reduce(const GemmArgs& g, const float* part, int splits, hipStream_t s) {
    size_t work;
    if (EPI == EPI_QKV) work = static_cast<size_t>(g.m) * (g.n / 2);
    else if (EPI == EPI_SWIGLU) work = static_cast<size_t>(g.m) * (g.n / 8);
    else work = static_cast<size_t>(g.m) * (g.n / 4);
    splitk_reduce_kernel<EPI><<<static_cast<unsigned>((work + 255) / 256), 256, 0, s>>>(g, part, splits);
}

template <int BM, int BN, int WAVES_M, int WAVES_N, int BK, int ST, int EPI>
void launch_epi(const GemmArgs& g, const GemmPlan& p, float* part, hipStream_t s) {
    constexpr int THREADS = WAVES_M * WAVES_N * 64;
    const int tiles = ((g.m + BM - 1) / BM) * (g.n / BN);
    if (p.sk_workers > 0) {
        gemm_sk_kernel<BM, BN, WAVES_M, WAVES_N, BK, ST, EPI>
            <<<p.dp_tiles + p.sk_workers, THREADS, 0, s>>>(g, part, p.dp_tiles, p.sk_workers);
        const int units = EPI == EPI_QKV ? BM * BN / 2 : EPI == EPI_SWIGLU ? BM * BN / 8 : BM * BN / 4;
        sk_fixup_kernel<BM, BN, BK, EPI>
            <<<dim3(tiles - p.dp_tiles, (units + 255) / 256), 256, 0, s>>>(g, part, p.dp_tiles, p.sk_workers);
        return;
    }
    dim3 grid(tiles, p.splits);
    const int kps = g.k / p.splits;
    if (p.splits == 1) {
        gemm_kernel<BM, BN, WAVES_M, WAVES_N, BK, ST, EPI, false><<<grid, THREADS, 0, s>>>(g, nullptr, kps);
        return;
    }
    gemm_kernel<BM, BN, WAVES_M, WAVES_N, BK, ST, EPI, true><<<grid, THREADS, 0, s>>>(g, part, kps);
    launch_reduce<EPI>(g, part, p.splits, s);
}

template <int T, int EPI>
void launch_skinny_epi(const GemmArgs& g, const GemmPlan& p, float* part, hipStream_t s) {
    dim3 grid(g.n / 64, p.splits);
    const int threads = 64 * p.ks;
    const int kps = g.k / p.splits;
    if (p.splits == 1) {
        skinny_kernel<T, EPI, false><<<grid, threads, 0, s>>>(g, nullptr, kps, p.ks);
        return;
    }
    skinny_kernel<T, EPI, true><<<grid, threads, 0, s>>>(g, part, kps, p.ks);
    launch_reduce<EPI>(g, part, p.splits, s);
}

template <int T>
void launch_skinny(const GemmArgs& g, const GemmPlan& p, void* partial, hipStream_t s) {
    float* part = static_cast<float*>(partial);
    switch (g.epi) {
        case EPI_RESID_F32OUT: launch_skinny_epi<T, EPI_RESID_F32OUT>(g, p, part, s); break;
        case EPI_RESID_F32IN: launch_skinny_epi<T, EPI_RESID_F32IN>(g, p, part, s); break;
        case EPI_SWIGLU: launch_skinny_epi<T, EPI_SWIGLU>(g, p, part, s); break;
        default: launch_skinny_epi<T, EPI_QKV>(g, p, part, s); break;
    }
}

template <int T, int CG, int EPI>
void launch_narrow_epi(const GemmArgs& g, const GemmPlan& p, hipStream_t s) {
    narrow_kernel<T, CG, EPI><<<g.n / (16 * CG), 64 * p.ks, 0, s>>>(g, p.ks);
}

template <int T>
void launch_narrow(const GemmArgs& g, const GemmPlan& p, hipStream_t s) {
    switch (g.epi) {
        case EPI_RESID_F32OUT: launch_narrow_epi<T, 1, EPI_RESID_F32OUT>(g, p, s); break;
        case EPI_RESID_F32IN: launch_narrow_epi<T, 1, EPI_RESID_F32IN>(g, p, s); break;
        case EPI_SWIGLU: launch_narrow_epi<T, 2, EPI_SWIGLU>(g, p, s); break;
        default: launch_narrow_epi<T, 2, EPI_QKV>(g, p, s); break;
    }
}

template <int BM, int BN, int WAVES_M, int WAVES_N, int BK, int ST>
void launch_cfg(const GemmArgs& g, const GemmPlan& p, void* partial, hipStream_t s) {
    float* part = static_cast<float*>(partial);
    switch (g.epi) {
        case EPI_RESID_F32OUT: launch_epi<BM, BN, WAVES_M, WAVES_N, BK, ST, EPI_RESID_F32OUT>(g, p, part, s); break;
        case EPI_RESID_F32IN: launch_epi<BM, BN, WAVES_M, WAVES_N, BK, ST, EPI_RESID_F32IN>(g, p, part, s); break;
        case EPI_SWIGLU: launch_epi<BM, BN, WAVES_M, WAVES_N, BK, ST, EPI_SWIGLU>(g, p, part, s); break;
        default: launch_epi<BM, BN, WAVES_M, WAVES_N, BK, ST, EPI_QKV>(g, p, part, s); break;
    }
}

}  // namespace

// Tile and split choice per projection shape, from one sweep that timed
// every configuration plainly, with k split two ways and with the stream-K
// schedule at m = 64 .. 4104 (21 points) on the 8B-layer shapes, each run
// after a read sweep of the caches.  Band i covers m in (m_hi[i - 1], m_hi[i]]
// and takes the fastest entry measured at its upper end (the previous
// choice where it was within 1.5%); neighbouring bands with the same choice
// are merged.  The bands are not monotone in m: what pays is how m fills
// whole row tiles and rounds of the CUs.  splits: 0 the default rule of
// plan_with_cfg, 2 a forced two-way split, -1 the stream-K schedule.
struct Band {
    int m_hi;
    int8_t cfg, splits;
};
constexpr Band kBandsQkv[] = {{64, 9, 0},     {96, 6, 0},     {128, 0, 0},    {160, 4, 0},
                              {192, 10, 2},   {224, 8, 2},    {288, 9, 2},    {480, 6, 2},
                              {544, 5, 0},    {928, 4, 2},    {1056, 5, 0},   {1312, 4, -1},
                              {1568, 4, 2},   {2592, 5, 0},   {3104, 4, 0},   {4104, 3, 0}};
constexpr Band kBandsO[] = {{128, 10, 0},  {192, 6, 0},   {224, 5, 0},   {352, 10, 2},  {480, 8, 2},
                            {672, 6, 2},   {800, 5, 0},   {928, 8, -1},  {1312, 4, 2},  {1568, 0, 0},
                            {2080, 3, -1}, {2592, 4, 0},  {3104, 5, 0},  {4104, 4, 0}};
constexpr Band kBandsGateUp[] = {{64, 9, 2},   {96, 6, 2},   {128, 0, 0},  {192, 4, 2},  {224, 3, 2},
                                 {352, 4, 0},  {416, 3, 0},  {480, 2, 0},  {544, 7, 0},  {672, 4, 0},
                                 {928, 3, 0},  {1056, 4, 0}, {1312, 3, 0}, {1568, 4, 0}, {4104, 3, 0}};
constexpr Band kBandsDown[] = {{128, 10, 0},  {192, 6, 0},   {224, 5, 0},   {288, 7, 0},
                               {352, 4, 0},   {480, 3, 0},   {544, 7, -1},  {672, 4, -1},
                               {928, 3, -1},  {1056, 4, -1}, {1312, 4, 2},  {1568, 3, 2},
                               {2080, 3, -1}, {2592, 4, -1}, {3104, 3, -1}, {4104, 4, 0}};

template <size_t N>
const Band& band_of(const Band (&t)[N], int m) {
    for (const Band& b : t)
        if (m <= b.m_hi) return b;
    return t[N - 1];
}

// The narrow kernel takes qkv, the output and the down projection up to 8
// rows and the output projection up to 24 (8B layer, against the kernels
// below: output -34% at 1 row, -18% at 16, -7% at 24; down -22% at 1 row,
// -13% at 8; qkv -12% at 1 row; it loses on gate/up and beyond those row
// counts, where every work-group re-reads all the activation rows; 64-column
// work-groups, which re-read them a quarter as often, measured 1.5-3x slower
// for want of work-groups).  The weight-streaming
// kernel takes the other narrow projections up to 32 rows and gate/up up to
// 16 (it won there by 10-20%; on qkv the tile kernels measured faster).
// Shapes outside the 8B layer take the band of their projection class; n must
// be a multiple of 128 and k of 64.
GemmPlan plan_gemm(int m, int n, int k) {
    const bool wide = n >= 16384, qkv_like = n >= 6144 && !wide;
    if (n % 64 == 0 && k % 32 == 0 && !wide && (m <= 8 || (m <= 24 && !qkv_like && k < 8192)))
        return plan_with_cfg(kNarrowCfg, m, n, k);
    if (n % 64 == 0 && (wide ? m <= 16 : m <= 32 && !qkv_like)) return plan_with_cfg(kSkinnyCfg, m, n, k);
    const Band& b = k >= 8192 ? band_of(kBandsDown, m)
                    : wide    ? band_of(kBandsGateUp, m)
                    : qkv_like ? band_of(kBandsQkv, m)
                               : band_of(kBandsO, m);
    if (n % kCfgs[b.cfg].bn) return plan_with_cfg(n % 128 ? 1 : 0, m, n, k);
    if (b.splits < 0) return plan_stream_k(b.cfg, m, n, k);
    GemmPlan p = plan_with_cfg(b.cfg, m, n, k);
    if (b.splits > 0 && k % (b.splits * BK_MAX) == 0) {
        p.splits = b.splits;
        p.partial_bytes = b.splits > 1 ? static_cast<size_t>(b.splits) * m * n * sizeof(float) : 0;
    }
    return p;
}

GemmPlan plan_with_cfg(int cfg, int m, int n, int k) {
    GemmPlan p{};
    p.cfg = cfg;
    if (cfg == kNarrowCfg) {
        // waves per work-group: each takes a whole number of 32-wide k slices
        int ks = 8;
        while (ks > 1 && k % (32 * ks)) ks /= 2;
        p.ks = ks;
        p.bm = m <= 16 ? 16 : 32;
        p.bn = 16;
        p.splits = 1;
        return p;
    }
    if (cfg == kSkinnyCfg) {
        // Four waves slice k inside a work-group (fewer when k is short); k is
        // also split across work-groups until there are 384 of them (three
        // share a CU), keeping whole 64-wide steps per wave.
        p.bn = 64;
        p.bm = 32;
        int ks = 4;
        while (ks > 1 && k % (64 * ks)) ks /= 2;
        p.ks = ks;
        int splits = 1;
        while (splits < 8 && (n / 64) * splits < 384 && k % (2 * 64 * ks * splits) == 0) splits *= 2;
        p.splits = splits;
        p.partial_bytes = splits > 1 ? static_cast<size_t>(splits) * m * n * sizeof(float) : 0;
        return p;
    }
    p.bm = kCfgs[cfg].bm;
    p.bn = kCfgs[cfg].bn;
    const long tiles = static_cast<long>(n / p.bn) * ((m + p.bm - 1) / p.bm);
    int splits = 1;
    // Too few tiles to fill 256 compute units: split k (each split >= 512 deep).
    while (splits < 8 && tiles * splits < 384 && k % (2 * splits * BK_MAX) == 0 && k / (2 * splits) >= 512)
        splits *= 2;
    p.splits = splits;
    p.partial_bytes = splits > 1 ? static_cast<size_t>(splits) * m * n * sizeof(float) : 0;
    return p;
}

GemmPlan plan_stream_k(int cfg, int m, int n, int k) {
    GemmPlan p = plan_with_cfg(cfg, m, n, k);
    if (cfg == kSkinnyCfg || cfg == kNarrowCfg) return p;
    const TileCfg& t = kCfgs[cfg];
    // work-groups a CU holds at once: one for eight waves or more than 80 KB of LDS
    const int lds = (t.ring == 0 ? 2 : t.ring) * (t.bm + t.bn) * t.bk * 2;
    const int slots = kStreamKCus * ((t.waves_m * t.waves_n >= 8 || lds > 80 * 1024) ? 1 : 2);
    const int tiles = ((m + t.bm - 1) / t.bm) * (n / t.bn);
    p.splits = 1;
    p.partial_bytes = 0;
    if (tiles % slots == 0) return p;  // whole rounds: plain tiles
    const int q = tiles / slots, r = tiles % slots;
    p.dp_tiles = q >= 1 ? (q - 1) * slots : 0;  // the last full round joins the stream-K part
    const long iters = static_cast<long>(tiles - p.dp_tiles) * (k / t.bk);
    p.sk_workers = static_cast<int>(std::min<long>(slots, iters));
    (void)r;
    p.partial_bytes = static_cast<size_t>(2) * p.sk_workers * t.bm * t.bn * sizeof(float);
    return p;
}

bool gemm_shape_ok(const GemmPlan& p, int n, int k) {
    if (p.cfg == kNarrowCfg)  // m <= 32 is the caller's part; paired epilogues need 64-column tiles
        return n % 64 == 0 && p.ks >= 1 && p.ks <= 8 && k % (32 * p.ks) == 0;
    if (p.cfg == kSkinnyCfg)  // m <= 32 is the caller's part (plan_gemm)
        return n % 64 == 0 && p.ks >= 1 && p.ks <= 4 && k % (64 * p.ks * p.splits) == 0;
    return p.cfg >= 0 && p.cfg < kNumCfgs && n % p.bn == 0 && k % (p.splits * BK_MAX) == 0;
}

void launch_gemm(const GemmArgs& g, const GemmPlan& p, void* partial, hipStream_t s) {
    if (g.m <= 0) return;
    if (p.cfg == kNarrowCfg) {  // plans cover m <= 32
        if (g.m <= 16) launch_narrow<1>(g, p, s);
        else launch_narrow<2>(g, p, s);
        return;
    }
    if (p.cfg == kSkinnyCfg) {
        launch_skinny<1>(g, p, partial, s);  // plans cover m <= 32
        return;
    }
    switch (p.cfg) {
        case 0: launch_cfg<128, 128, 2, 2, 64, 0>(g, p, partial, s); break;
        case 1: launch_cfg<64, 128, 2, 2, 64, 0>(g, p, partial, s); break;
        case 2: launch_cfg<256, 128, 2, 2, 32, 0>(g, p, partial, s); break;
        case 3: launch_cfg<256, 256, 2, 4, 64, 2>(g, p, partial, s); break;
        case 4: launch_cfg<192, 256, 2, 4, 64, 2>(g, p, partial, s); break;
        case 5: launch_cfg<128, 128, 2, 2, 64, 2>(g, p, partial, s); break;
        case 6: launch_cfg<96, 256, 1, 4, 64, 3>(g, p, partial, s); break;
        case 7: launch_cfg<160, 256, 1, 4, 64, 2>(g, p, partial, s); break;
        case 8: launch_cfg<128, 128, 2, 2, 64, 4>(g, p, partial, s); break;
        case 9: launch_cfg<64, 256, 1, 4, 64, 3>(g, p, partial, s); break;
        default: launch_cfg<128, 128, 2, 2, 64, 3>(g, p, partial, s); break;
    }
}

}  // namespace slw
