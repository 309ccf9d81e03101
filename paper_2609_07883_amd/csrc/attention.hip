// Paged attention on gfx950 matrix cores (v_mfma_f32_16x16x32_bf16).
//
// Both kernels compute transposed scores S^T = K Q^T: 16 keys are the A
// operand and Q^T the B operand, so lane l holds, for query (or head)
// l % 16, the scores of rows 4 (l / 16) .. 4 (l / 16) + 3 of the key tile.
// Two such tiles over a pair of pages take their keys in an order that
// leaves lane group g with keys 8 g .. 8 g + 7 of the pair (pair_key below):
// exactly the eight k-values lane l must supply as the A operand (P) of the
// P V product, whose k index runs over the same keys, and eight consecutive
// tokens of one page, so the V operand is one 16-byte piece of the
// dim-major V page.  The softmax is online (running max and sum per query,
// base-2 exponentials) in fp32.
//
// Page layouts (one (layer, block, kv head) page of 16 tokens):
//   K: [hd/32][16][32]  element (t, d) at (d/32)*512 + t*32 + d%32
//   V: [hd][16]         element (t, d) at d*16 + t
#include <math.h>

#include "device.h"
#include "kernels.h"

namespace slw {
namespace {

constexpr float kLog2e = 1.4426950408889634f;
// LDS tiles in the chunk-attention ring: two (64 KB) measured slightly ahead
// of three or four (96 or 128 KB) on the long-context and layer-sweep shapes.
// The kernel's registers (about 200 per lane) allow one work-group per CU.
constexpr int kChunkStages = 2;

// 2^x straight on the transcendental unit (v_exp_f32).  Results below
// 2^-126 may flush to zero, which softmax weights taken relative to a running
// maximum can afford; the library exp2f adds range scaling around the same
// instruction, five more VALU operations per call.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Block tables read through the scalar cache: a wave-uniform index into
// constant-address-space memory.
typedef const int32_t __attribute__((address_space(4))) const_i32;

// Max and sum over lanes l, l ^ 16, l ^ 32 and l ^ 48 (the four 16-lane rows
// of a wave), with the gfx950 row-swap instructions instead of LDS permutes:
// a swap of a register with itself leaves, in every lane, its own value in
// one result and its partner's in the other.
__device__ __forceinline__ float rows4_max(float x) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float rows4_sum(float x) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

__device__ __forceinline__ bf16x8 to_bf16x8(f32x4 lo, f32x4 hi) {
    bf16x8 r;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        r[e] = f2bf(lo[e]);
        r[4 + e] = f2bf(hi[e]);
    }
    return r;
}

// ---------------------------------------------------------------------------
// Chunk attention: C queries at positions P..P+C-1 of one sequence attend to
// its keys 0..P+C-1 under the causal mask.
//
// A work-group owns one kv head and 256 rows = (position, q head) pairs of
// that head's group; each of its eight waves owns 32 rows, the two 16-column
// Q^T tiles of its MFMAs, so one K or V fragment read from LDS feeds two
// MFMAs and two waves share each SIMD, overlapping one wave's softmax with
// the other's matrix work.  Keys advance 64 at a time (four pages) through a
// ring of ST LDS tiles shared by the eight waves, filled by direct
// global->LDS loads issued ST - 1 tiles ahead (each lane fetches the 16-byte
// chunk that belongs at its swizzled LDS slot; every wave issues the same
// number of loads per tile, so a counted wait for its own loads plus a bare
// barrier publishes a tile).  Within a tile the LDS reads run one step ahead
// of the MFMAs: the next score tile's K fragments and the next group's V
// fragments are read while the current ones are multiplied.  On an item's
// last tile the V values of keys past the range end are zeroed in LDS once,
// so the P V loop carries no masking.  The row sums of the probabilities come
// from the matrix cores (P times a column of ones, two MFMAs per page pair),
// so they add the same bf16 values the P V product does and take no VALU
// additions.  A work item covers one key range of one query
// tile, and a work-group runs the items its slot lists one after the other
// (the host gives each work-group whole query tiles when they balance, and
// otherwise cuts the keys of all query tiles into equal runs).
// A query tile covered by one item is normalised and stored directly; the
// items of a query tile split over several write fp32 partials (running max,
// sum, unnormalised output) that attn_merge_kernel combines.
// ---------------------------------------------------------------------------

// Keys of the two score tiles of a pair of pages (32 keys): row r of tile
// tau holds key 16 (r / 8) + 8 ((r / 4) % 2) + 4 tau + r % 4, so that lane
// group g (rows 4 g .. 4 g + 3 of both tiles) ends up with keys 8 g .. 8 g + 7:
// the eight consecutive tokens of one page that the P V product's k slice g
// covers, and one 16-byte chunk of a dim-major V page.
__device__ __forceinline__ int pair_key(int r, int tau) { return 16 * (r >> 3) + 8 * ((r >> 2) & 1) + 4 * tau + (r & 3); }

// LDS swizzles of 16-byte chunks: K rows (64 B = four chunks of 8 dims) and
// V rows (32 B = two chunks of 8 tokens).  An operand read serves eight lanes
// per pass: for K the rows of tokens {0..3, 8..11} or {4..7, 12..15} of a
// page, for V eight consecutive dims; both swizzles put those on distinct
// banks.
__device__ __forceinline__ int kswz(int t, int sub) { return sub ^ (((t >> 1) & 1) | (((t >> 3) & 1) << 1)); }
__device__ __forceinline__ int vswz(int d, int h) { return h ^ ((d >> 2) & 1); }

// Direct global->LDS load of 16 bytes per lane: lane l's bytes land at
// lds + 16 l (lds is wave-uniform).  Issued as assembly so that the compiler,
// which cannot tell which LDS buffer such a load writes, does not make every
// later LDS read wait for all of them; the kernel waits for them itself.
// M0 is a reserved register that the compiler sets right before each
// instruction that reads it; no compiler-generated code in these kernels
// uses it, so the value left there is never relied on.
__device__ __forceinline__ void load_lds16(const void* src, void* lds) {
    const uint32_t dst = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(reinterpret_cast<uintptr_t>(lds)));
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "s"(dst) : "memory");
}

// Wait until at most N vector-memory operations of this wave are outstanding.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Wait until this wave's LDS operations are complete (vector memory
// operations may stay outstanding).
__device__ __forceinline__ void wait_lgkmcnt0() { __builtin_amdgcn_s_waitcnt(0xC07F); }

// Workgroup barrier with no memory fence (the memory clobber keeps the
// compiler from moving LDS or global accesses across it).
__device__ __forceinline__ void barrier_only() { asm volatile("s_barrier" ::: "memory"); }

template <int HD>
__device__ __forceinline__ void decode_attn_wave(const DecodeAttnArgs& a, int slot, int kvh, int lane);

// With DECODE, the launch also runs decode attention: work-groups past the
// n_slots * hkv chunk work-groups hold eight decode waves each (wave v of
// that part takes slot v % n_slots of kv head v / n_slots).  They start as
// chunk work-groups leave CUs free, so the decodes fill the chunk part's
// tail and any CUs a short chunk leaves idle, with no second stream to fork
// and join.  The decode wave's index is read as wave-uniform, so that its
// work list and block-table entries come through the scalar cache as in the
// decode kernel.  Decode waves need no barrier; the chunk part's barriers see all
// eight waves of its work-groups, which come first in the grid, so the
// hardware's round-robin over the XCDs sees them in order.  (The chunk code
// stays in the kernel itself: compiled as a separate function and inlined,
// it came out with different branch conversion and ran up to 4% slower.)
template <int HD, int GROUP, int ST, bool DECODE>
__global__ __launch_bounds__(512) void chunk_attn_kernel(ChunkAttnArgs a, DecodeAttnArgs da) {
    if constexpr (DECODE) {
        const int n_chunk = a.n_slots * a.hkv;
        if (static_cast<int>(blockIdx.x) >= n_chunk) {
            const int v = (static_cast<int>(blockIdx.x) - n_chunk) * 8 +
                          __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x >> 6));
            if (v < da.n_slots * da.hkv) decode_attn_wave<HD>(da, v % da.n_slots, v / da.n_slots, threadIdx.x & 63);
            return;
        }
    }
    constexpr int KK = HD / 32, NT = HD / 16, PAGE = HD * 16;
    constexpr int SLABS = 2 * 4 * PAGE / 512;  // 1 KB direct loads per tile (K and V of four pages)
    constexpr int PER_WAVE = SLABS / 8;        // loads each wave issues per tile
    static_assert(SLABS % 8 == 0, "tile loads must split evenly over the waves");
    static_assert(ST >= 2 && ST <= 4, "ring of two to four tiles");
    static_assert(NT % 4 == 0, "V fragments are read four at a time");
    constexpr int CT = 2;                 // 16-row column tiles per wave (32 rows)
    constexpr int PW = 32 / GROUP;        // positions per wave (eight waves: a tile of 8 PW positions)
    // Lazy rescaling: a row keeps its running max until a tile exceeds it by
    // 2^kSlack, so probabilities stay <= 2^kSlack and most tiles skip the
    // rescale of the output accumulators.
    constexpr float kSlack = 8.0f;
    __shared__ __attribute__((aligned(16))) bf16 Ks[ST][4 * PAGE];
    __shared__ __attribute__((aligned(16))) bf16 Vs[ST][4 * PAGE];

    // The wave index goes through readfirstlane so that the compiler knows it
    // is wave-uniform: the per-wave tests of the tile loop (live rows, masked
    // tile) then become scalar branches, where a per-lane reading put every
    // score of every tile under an exec-mask branch of its own.
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int grp = lane >> 4, col = lane & 15;
    // Work order: kv-head major, the runs of one head in key order.  All
    // runs of a head read that head's keys and values, and runs that start
    // together read the same pages together: with the order spread over the
    // XCDs in contiguous ranges, they share one L2.
    const int pos = xcd_order(blockIdx.x, a.n_slots * a.hkv);
    const int kvh = pos / a.n_slots, slot = pos % a.n_slots;
    const float sl2 = kLog2e / sqrtf(static_cast<float>(HD));
    const bf16* kpool = static_cast<const bf16*>(a.k_pool);
    const bf16* vpool = static_cast<const bf16*>(a.v_pool);
    bf16x8 ones;  // the B operand of the row-sum MFMAs
#pragma unroll
    for (int e = 0; e < 8; ++e) ones[e] = bf16(1.0f);

    // Load j of a tile (j = wave + 8 i): 0 .. 4 KK - 1 are K slabs (page j / KK,
    // dims 32 (j % KK) ..), the rest V slabs (page, 32 dims of 16 tokens).
    // Pages past the key range load the range's last page instead (their
    // scores are masked and their values zeroed in LDS on the item's last
    // tile), so every wave issues PER_WAVE loads.
    int l_page[PER_WAVE], l_elem[PER_WAVE], l_dst[PER_WAVE];
    bool l_isv[PER_WAVE];
#pragma unroll
    for (int i = 0; i < PER_WAVE; ++i) {
        const int j = wave + 8 * i;
        const bool is_v = j >= 4 * KK;
        const int jj = is_v ? j - 4 * KK : j;
        const int p = jj / KK, slab = jj % KK;
        l_isv[i] = is_v;
        l_page[i] = p;
        if (!is_v) {  // lane: token t, stored chunk lane % 4 holds dims chunk kswz(t, .)
            const int t = lane >> 2, sub = kswz(t, lane & 3);
            l_elem[i] = slab * 512 + t * 32 + sub * 8;
        } else {      // lane: dim d, stored chunk lane % 2 holds tokens 8 vswz(d, .)
            const int d = slab * 32 + (lane >> 1), h = (lane & 1) ^ ((d >> 2) & 1);
            l_elem[i] = d * 16 + h * 8;
        }
        l_dst[i] = p * PAGE + slab * 512;
    }
    // Block-table entries are read through the scalar cache (a uniform index
    // into constant memory): a vector load here would make the compiler wait
    // for every direct load in flight before using its result.
    const int i0 = a.slot_off[slot], i1 = a.slot_off[slot + 1];
    for (int k = i0; k < i1; ++k) {
        const int item = a.slot_items[k];
        const int qt = a.item_qt[item], kb = a.item_kb[item], ke = a.item_ke[item];
        // the query tile: rows row0 .. row0 + nrows - 1 at positions pos0 .. of one sequence
        const int row0 = a.qt_row0[qt], nrows = a.qt_rows[qt], pos0 = a.qt_pos0[qt];
        const const_i32* bt_s = (const const_i32*)(a.bt + a.qt_bt[qt]);
        const int j0 = wave * PW;            // first tile position of this wave
        const int n_tiles = (ke - kb + 63) / 64;
        const int wave_qpos_lo = pos0 + j0, wave_qpos_hi = pos0 + j0 + PW - 1;
        const bool wave_live = j0 < nrows;
        // a query tile covered by one item is written here, else as a partial
        const bool whole = a.qt_off[qt + 1] - a.qt_off[qt] == 1;

        // Q^T operand: row r = ct*16 + col is tile position j0 + r / GROUP, head kvh*GROUP + r % GROUP
        bf16x8 qf[CT][KK];
        const bf16* qkv = static_cast<const bf16*>(a.qkv);
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
            const int r = ct * 16 + col, j = j0 + r / GROUP, h = kvh * GROUP + r % GROUP;
#pragma unroll
            for (int kk = 0; kk < KK; ++kk)
                qf[ct][kk] = j < nrows ? *reinterpret_cast<const bf16x8*>(
                                             qkv + static_cast<size_t>(row0 + j) * a.ld_qkv + h * HD + kk * 32 + grp * 8)
                                       : bf16x8{};
        }

        const int last_page = (ke - 1) >> 4;
        // Block ids of the pages the wave's loads of a tile read, fetched
        // through the scalar cache one tile before the loads that use them:
        // the wait for a scalar load then costs nothing where the loads are
        // issued (read there, it stalled every wave of the CU once per page).
        int blk_next[PER_WAVE];
        auto fetch = [&](int t) {
#pragma unroll
            for (int i = 0; i < PER_WAVE; ++i)
                blk_next[i] = bt_s[__builtin_amdgcn_readfirstlane(min((kb >> 4) + 4 * t + l_page[i], last_page))];
        };
        auto issue = [&](int t) {
            const int buf = t % ST;
#pragma unroll
            for (int i = 0; i < PER_WAVE; ++i) {
                const size_t blk = blk_next[i];
                const bf16* src = (l_isv[i] ? vpool : kpool) + (blk * a.hkv + kvh) * PAGE + l_elem[i];
                load_lds16(src, l_isv[i] ? &Vs[buf][l_dst[i]] : &Ks[buf][l_dst[i]]);
            }
        };

        f32x4 o[CT][NT];
#pragma unroll
        for (int ct = 0; ct < CT; ++ct)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) o[ct][nt] = f32x4{};
        float m_run[CT];
        // Row sums of P on the matrix cores (P times a column of ones): lane
        // (grp, col) holds the sums of rows 4 grp .. 4 grp + 3 of column tile ct.
        f32x4 l_acc[CT];
        int qpos_col[CT];  // query position of row ct*16 + col
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
            m_run[ct] = -INFINITY;
            l_acc[ct] = f32x4{};
            qpos_col[ct] = wave_qpos_lo + (ct * 16 + col) / GROUP;
        }

        // Q fragments land before the ring starts; the compiler then has no
        // loads of its own pending inside the loop, so it adds no waits there.
        wait_vmcnt<0>();
        // every wave is past the previous item's last tile before its buffers refill
        if (k != i0) barrier_only();
#pragma unroll
        for (int t = 0; t < ST - 1; ++t)
            if (t < n_tiles) {
                fetch(t);
                issue(t);
            }
        if (ST - 1 < n_tiles) fetch(ST - 1);
        for (int t = 0; t < n_tiles; ++t) {
            const int buf = t % ST;
            // this wave's loads of tile t are done once at most the loads of the
            // younger tiles in flight (up to ST - 2 of them) are outstanding
            const int younger = min(n_tiles - 1 - t, ST - 2);
            if (ST >= 4 && younger >= 2) wait_vmcnt<2 * PER_WAVE>();
            else if (ST >= 3 && younger >= 1) wait_vmcnt<PER_WAVE>();
            else wait_vmcnt<0>();
            barrier_only();
            if (t + ST - 1 < n_tiles) issue(t + ST - 1);
            const int key0 = kb + t * 64;
            // The item's last tile: keys at or past ke (unwritten slots of the
            // last page, stand-in pages) get probability 0, and their V values
            // are zeroed here once for all waves, so that whatever the pool
            // holds there cannot turn 0 into NaN in the P V product.
            if (key0 + 63 >= ke) {
                for (int r = tid; r < 4 * HD; r += 512) {  // row r: page r / HD, dim r % HD
                    const int pg = r / HD, d = r % HD;
#pragma unroll
                    for (int tt = 0; tt < 16; ++tt)
                        if (key0 + 16 * pg + tt >= ke)
                            Vs[buf][pg * PAGE + d * 16 + vswz(d, tt >> 3) * 8 + (tt & 7)] = bf16(0.0f);
                }
                wait_lgkmcnt0();
                barrier_only();
            }
            if (wave_live && key0 <= wave_qpos_hi) {
                f32x4 sc[4][CT];  // [2 pair + tile][ct]
#pragma unroll
                for (int p = 0; p < 4; ++p)
#pragma unroll
                    for (int ct = 0; ct < CT; ++ct) sc[p][ct] = f32x4{};
                // K fragments of score tile p + 1 are read while tile p's
                // MFMAs run (two register sets); the scheduling groups below
                // keep that order, which the compiler otherwise undoes by
                // reading each fragment right before its MFMAs and waiting there.
                bf16x8 kf[2][KK];
                auto kread = [&](int p, bf16x8(&k)[KK]) {
                    const int key = pair_key(col, p & 1), tok = key & 15;
                    const int base = (2 * (p >> 1) + (key >> 4)) * PAGE + tok * 32 + kswz(tok, grp) * 8;
#pragma unroll
                    for (int kk = 0; kk < KK; ++kk) k[kk] = *reinterpret_cast<const bf16x8*>(&Ks[buf][base + kk * 512]);
                };
                kread(0, kf[0]);
#pragma unroll
                for (int p = 0; p < 4; ++p) {
                    if (p + 1 < 4) kread(p + 1, kf[(p + 1) & 1]);
#pragma unroll
                    for (int kk = 0; kk < KK; ++kk)
#pragma unroll
                        for (int ct = 0; ct < CT; ++ct) sc[p][ct] = mfma16(kf[p & 1][kk], qf[ct][kk], sc[p][ct]);
                }
                // V fragments in groups of four: group g covers page pair
                // g / (NT / 4) (k slice grp = tokens 8 (grp % 2) .. + 7 of page
                // 2 j + grp / 2) and output dims 16 n0 .. 16 n0 + 63,
                // n0 = 4 (g % (NT / 4)).  The first group is read during the
                // last score tile's MFMAs, each next one during the current
                // one's P V MFMAs.
                constexpr int VG = 2 * NT / 4;
                bf16x8 vf[2][4];
                auto vread = [&](int g, bf16x8(&v)[4]) {
                    const int j = g / (NT / 4), n0 = (g % (NT / 4)) * 4;
                    const int v_base = (2 * j + (grp >> 1)) * PAGE;
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int d = (n0 + i) * 16 + col;
                        v[i] = *reinterpret_cast<const bf16x8*>(&Vs[buf][v_base + d * 16 + vswz(d, grp & 1) * 8]);
                    }
                };
                vread(0, vf[0]);
                __builtin_amdgcn_sched_group_barrier(0x100, KK, 0);  // 0x100: LDS reads
#pragma unroll
                for (int p = 0; p < 3; ++p) {  // next score tile's K reads
#pragma unroll
                    for (int r = 0; r < KK; ++r) {
                        __builtin_amdgcn_sched_group_barrier(0x8, 1, 0);  // 0x8: MFMA
                        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                    }
                    if constexpr (KK * CT > KK) __builtin_amdgcn_sched_group_barrier(0x8, KK * CT - KK, 0);
                }
#pragma unroll
                for (int r = 0; r < 4; ++r) {  // the last score tile: V group 0's reads
                    __builtin_amdgcn_sched_group_barrier(0x8, 1, 0);
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                }
                if constexpr (KK * CT > 4) __builtin_amdgcn_sched_group_barrier(0x8, KK * CT - 4, 0);
                // Only tiles that reach the wave's diagonal or the range end
                // are masked: one wave-uniform branch around the whole mask.
                if (key0 + 63 > wave_qpos_lo || key0 + 63 >= ke) {
#pragma unroll
                    for (int p = 0; p < 4; ++p)
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const int kpos = key0 + 32 * (p >> 1) + pair_key(4 * grp + e, p & 1);
#pragma unroll
                            for (int ct = 0; ct < CT; ++ct)
                                sc[p][ct][e] = (kpos <= qpos_col[ct] && kpos < ke) ? sc[p][ct][e] : -INFINITY;
                        }
                }
                float mx[CT];
                bool grow = false;
#pragma unroll
                for (int ct = 0; ct < CT; ++ct) {
                    float m = -INFINITY;
#pragma unroll
                    for (int p = 0; p < 4; ++p)
#pragma unroll
                        for (int e = 0; e < 4; ++e) m = fmaxf(m, sc[p][ct][e]);
                    m = rows4_max(m);
                    mx[ct] = m * sl2;
                    grow |= mx[ct] > m_run[ct] + kSlack;
                }
                if (__any(grow)) {  // wave-uniform: move every row's max up to its tile max
#pragma unroll
                    for (int ct = 0; ct < CT; ++ct) {
                        const float m_new = fmaxf(m_run[ct], mx[ct]);
                        const float alpha = m_new == -INFINITY ? 1.f : fast_exp2(m_run[ct] - m_new);
                        m_run[ct] = m_new;
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const float ae = __shfl(alpha, grp * 4 + e, 64);
                            l_acc[ct][e] *= ae;
#pragma unroll
                            for (int nt = 0; nt < NT; ++nt) o[ct][nt][e] *= ae;
                        }
                    }
                }
#pragma unroll
                for (int ct = 0; ct < CT; ++ct) {
                    const float m_use = m_run[ct] == -INFINITY ? 0.f : m_run[ct];
#pragma unroll
                    for (int p = 0; p < 4; ++p)
#pragma unroll
                        for (int e = 0; e < 4; ++e) sc[p][ct][e] = fast_exp2(fmaf(sc[p][ct][e], sl2, -m_use));
                }
                // P in bf16, the A operand of the P V MFMAs (keys 8 grp .. 8 grp + 7
                // of page pair j in lane group grp)
                bf16x8 pf[2][CT];
#pragma unroll
                for (int j = 0; j < 2; ++j)
#pragma unroll
                    for (int ct = 0; ct < CT; ++ct) pf[j][ct] = to_bf16x8(sc[2 * j][ct], sc[2 * j + 1][ct]);
#pragma unroll
                for (int g = 0; g < VG; ++g) {
                    const int j = g / (NT / 4), n0 = (g % (NT / 4)) * 4;
                    if (g + 1 < VG) vread(g + 1, vf[(g + 1) & 1]);
#pragma unroll
                    for (int i = 0; i < 4; ++i)
#pragma unroll
                        for (int ct = 0; ct < CT; ++ct) o[ct][n0 + i] = mfma16(pf[j][ct], vf[g & 1][i], o[ct][n0 + i]);
                    if (n0 == 0) {
#pragma unroll
                        for (int ct = 0; ct < CT; ++ct) l_acc[ct] = mfma16(pf[j][ct], ones, l_acc[ct]);
                    }
                }
#pragma unroll
                for (int g = 0; g < VG; ++g) {
                    if (g + 1 < VG) {
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            __builtin_amdgcn_sched_group_barrier(0x8, 1, 0);
                            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                        }
                        if (g % (NT / 4) == 0) __builtin_amdgcn_sched_group_barrier(0x8, 5 * CT - 4, 0);
                        else __builtin_amdgcn_sched_group_barrier(0x8, 4 * CT - 4, 0);
                    } else {
                        if (g % (NT / 4) == 0) __builtin_amdgcn_sched_group_barrier(0x8, 5 * CT, 0);
                        else __builtin_amdgcn_sched_group_barrier(0x8, 4 * CT, 0);
                    }
                }
            }
            // after the tile's last LDS read: scalar loads return out of
            // order, so one in flight makes every wait for an LDS read a
            // wait for it too
            if (t + ST < n_tiles) fetch(t + ST);
        }
        if (!wave_live) continue;

#pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
            if (!whole) {
                const size_t rbase = (static_cast<size_t>(item) * a.hkv + kvh) * 256 + wave * 32 + ct * 16;
                if (grp == 0) a.part_ml[(rbase + col) * 2 + 0] = m_run[ct];
                if (col == 0) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) a.part_ml[(rbase + grp * 4 + e) * 2 + 1] = l_acc[ct][e];
                }
#pragma unroll
                for (int e = 0; e < 4; ++e)
#pragma unroll
                    for (int nt = 0; nt < NT; ++nt)
                        a.part_o[(rbase + grp * 4 + e) * HD + nt * 16 + col] = o[ct][nt][e];
            } else {
                bf16* out = static_cast<bf16*>(a.out);
                const int ldo = a.hq * HD;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int r = ct * 16 + grp * 4 + e;
                    const int j = j0 + r / GROUP, h = kvh * GROUP + r % GROUP;
                    const float inv = 1.0f / l_acc[ct][e];
                    if (j < nrows) {
#pragma unroll
                        for (int nt = 0; nt < NT; ++nt)
                            out[static_cast<size_t>(row0 + j) * ldo + h * HD + nt * 16 + col] =
                                f2bf(o[ct][nt][e] * inv);
                    }
                }
            }
        }
    }  // items of this work-group
}

// Combine n partials (running max, sum and unnormalised output) of one
// row and write it normalised; 64 threads, HD / 64 dims each.  Partial w
// sits at row r0 + w * stride of ml [.][2] and po [.][HD]; a max of -inf
// means every key of that range was masked for the row.
template <int HD>
__device__ __forceinline__ void merge_row(const float* __restrict__ ml, const float* __restrict__ po, size_t r0,
                                          size_t stride, int n, bf16* __restrict__ out) {
    constexpr int CH = 8, PER = HD / 64;
    const int lane = threadIdx.x & 63;
    // One pass with a running maximum: each group of CH partials is loaded
    // at once, the sums so far are rescaled to the group's new maximum and
    // the group is added, so a list of up to CH partials costs one memory
    // round trip.
    float mmax = -INFINITY, lsum = 0.f;
    float acc[PER] = {};
    for (int c = 0; c < n; c += CH) {
        float m[CH], l[CH], v[CH][PER];
#pragma unroll
        for (int j = 0; j < CH; ++j) {
            const bool ok = c + j < n;
            const size_t r = r0 + (c + j) * stride;
            m[j] = ok ? ml[r * 2] : -INFINITY;
            l[j] = ok ? ml[r * 2 + 1] : 0.f;
#pragma unroll
            for (int p = 0; p < PER; ++p) v[j][p] = ok ? po[r * HD + lane + 64 * p] : 0.f;
        }
        float mc = -INFINITY;
#pragma unroll
        for (int j = 0; j < CH; ++j) mc = fmaxf(mc, m[j]);
        if (mc == -INFINITY) continue;  // every key of these ranges masked
        const float mn = fmaxf(mmax, mc);
        const float rs = fast_exp2(mmax - mn);  // 0 while nothing has been added
        lsum *= rs;
#pragma unroll
        for (int p = 0; p < PER; ++p) acc[p] *= rs;
#pragma unroll
        for (int j = 0; j < CH; ++j) {
            if (m[j] == -INFINITY) continue;
            const float sc = fast_exp2(m[j] - mn);
            lsum += sc * l[j];
#pragma unroll
            for (int p = 0; p < PER; ++p) acc[p] += sc * v[j][p];
        }
        mmax = mn;
    }
    const float inv = 1.0f / lsum;
#pragma unroll
    for (int p = 0; p < PER; ++p) out[lane + 64 * p] = f2bf(acc[p] * inv);
}

// Combine the key-range partials of one (tile position, q head): position x
// of the flattened tiles is position x % PWG of query tile x / PWG.
template <int HD, int GROUP>
__device__ __forceinline__ void chunk_merge_row(const ChunkAttnArgs& a, int x, int h) {
    constexpr int PWG = 256 / GROUP;
    const int kvh = h / GROUP;
    const int qt = x / PWG, j = x % PWG;
    if (j >= a.qt_rows[qt]) return;  // past the tile's last row
    const int row = j * GROUP + h % GROUP;
    const int w0 = a.qt_off[qt], w1 = a.qt_off[qt + 1];
    if (w1 - w0 == 1) return;  // written by the attention kernel
    merge_row<HD>(a.part_ml, a.part_o, (static_cast<size_t>(w0) * a.hkv + kvh) * 256 + row,
                  static_cast<size_t>(a.hkv) * 256, w1 - w0,
                  static_cast<bf16*>(a.out) + static_cast<size_t>(a.qt_row0[qt] + j) * a.hq * HD + h * HD);
}

// ---------------------------------------------------------------------------
// Decode attention, split over the key axis: one wave per (slot, kv head).
// The host lays the keys of all decodes end to end and cuts them into equal
// runs, one per slot; a slot's run is a list of work items (a key range of
// one decode, starting on a multiple of 64), which the wave takes one after
// the other, each leaving a partial for the merge.  Equal runs make every
// wave of the launch finish together, where one wave per fixed-size split
// left a ragged last round.  All q heads of the kv head's group (<= 16) are the columns of Q^T.  Keys are
// taken 32 at a time (two pages) straight from the pages into MFMA operand
// registers, with the next step's pages requested before the current step is
// multiplied (two register sets), so every wave keeps 16 KB of loads in
// flight while it computes.  The two score tiles of a step take their keys
// in the pair_key order of chunk attention: lane group g then holds the
// scores of keys 8 g .. 8 g + 7, eight consecutive tokens of one page, and
// its V operand of the P V product is one 16-byte piece of the dim-major V
// page.
// ---------------------------------------------------------------------------
template <int HD>
struct DecodeStep {
    bf16x8 k[2][HD / 32];  // [score tile][32-dim slab]
    bf16x8 v[HD / 16];     // [16-dim output tile]
};

// The loads of one step.  The two block-table entries of the pair come
// through the scalar cache (bt_s is wave-uniform): a vector load there would
// make the wave wait for every load in flight, the previous step's prefetch
// included, before it could address the next pages.  Pages past the item's
// last page load that page instead, so every load is unconditional and the
// waits can count; keys at or past tok1 are masked (scores) and zeroed (V)
// by the caller.

template <int HD>
__device__ __forceinline__ void decode_load(DecodeStep<HD>& st, const bf16* kpool, const bf16* vpool,
                                            const const_i32* bt_s, int c0, int last_pg, int hkv, int kvh, int col,
                                            int grp) {
    constexpr int KK = HD / 32, NT = HD / 16, PAGE = HD * 16;
    const int pg0 = c0 >> 4;
    const int b0 = bt_s[min(pg0, last_pg)], b1 = bt_s[min(pg0 + 1, last_pg)];
    // K: row `col` of score tile tau is key pair_key(col, tau) of the 32-key pair
    const size_t kpage = (static_cast<size_t>((col >> 3) ? b1 : b0) * hkv + kvh) * PAGE;
#pragma unroll
    for (int tau = 0; tau < 2; ++tau) {
        const int tok = pair_key(col, tau) & 15;
#pragma unroll
        for (int kk = 0; kk < KK; ++kk)
            st.k[tau][kk] = *reinterpret_cast<const bf16x8*>(kpool + kpage + kk * 512 + tok * 32 + grp * 8);
    }
    // V: lane group grp covers keys 8 grp .. 8 grp + 7 of the pair, tokens
    // 8 (grp % 2) .. + 7 of page grp / 2, for dim nt * 16 + col
    const size_t vpage = (static_cast<size_t>((grp >> 1) ? b1 : b0) * hkv + kvh) * PAGE;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
        st.v[nt] = *reinterpret_cast<const bf16x8*>(vpool + vpage + (nt * 16 + col) * 16 + 8 * (grp & 1));
}

// One decode-attention wave: the items of `slot` for kv head kvh.
template <int HD>
__device__ __forceinline__ void decode_attn_wave(const DecodeAttnArgs& a, int slot, int kvh, int lane) {
    constexpr int KK = HD / 32, NT = HD / 16;
    constexpr float kSlack = 8.0f;  // lazy rescaling threshold (log2 units)
    const int grp = lane >> 4, col = lane & 15;
    const int group = a.hq / a.hkv;
    const float sl2 = kLog2e / sqrtf(static_cast<float>(HD));
    const bf16* kpool = static_cast<const bf16*>(a.k_pool);
    const bf16* vpool = static_cast<const bf16*>(a.v_pool);

    // The wave's items one after the other: keys [tok0, tok1) of decode b,
    // each leaving its partial (running max, sum, unnormalised output).
    const int i0 = a.slot_off[slot], i1 = a.slot_off[slot + 1];
    for (int w = i0; w < i1; ++w) {
        const int b = a.work_b[w], tok0 = a.work_kb[w], tok1 = a.work_ke[w];
        const int last_pg = (tok1 - 1) >> 4;
        const const_i32* bt_s = (const const_i32*)(a.bt + a.bt_off[b]);

        bf16x8 qf[KK];
        {
            const bf16* q = static_cast<const bf16*>(a.q) + static_cast<size_t>(b) * a.ld_q;
            const int h = kvh * group + col;
#pragma unroll
            for (int kk = 0; kk < KK; ++kk)
                qf[kk] = col < group ? *reinterpret_cast<const bf16x8*>(q + h * HD + kk * 32 + grp * 8)
                                     : bf16x8{};
        }

        f32x4 o[NT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) o[nt] = f32x4{};
        float m_run = -INFINITY, l_run = 0.f;

        // lane (grp, col): element e of score tile tau is key 8 grp + 4 tau + e of
        // the step.  Keys at or past tok1 (the item's end; stand-in pages and
        // unwritten slots lie there) get score -inf and V 0, without branches: a
        // branch that rewrites loaded registers makes the compiler's wait counts
        // conservative and stalls on the prefetch in flight.
        auto compute = [&](DecodeStep<HD>& st, int c0) {
            const int nv = min(max(tok1 - c0 - 8 * grp, 0), 8);  // valid keys of this lane group
            u32x4 vmask;
#pragma unroll
            for (int j = 0; j < 4; ++j)
                vmask[j] = (2 * j < nv ? 0x0000FFFFu : 0u) | (2 * j + 1 < nv ? 0xFFFF0000u : 0u);
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                u32x4 bits = __builtin_bit_cast(u32x4, st.v[nt]) & vmask;
                st.v[nt] = __builtin_bit_cast(bf16x8, bits);
            }
            f32x4 s[2];
#pragma unroll
            for (int tau = 0; tau < 2; ++tau) {
                s[tau] = f32x4{};
#pragma unroll
                for (int kk = 0; kk < KK; ++kk) s[tau] = mfma16(st.k[tau][kk], qf[kk], s[tau]);
            }
            float mx = -INFINITY;
#pragma unroll
            for (int tau = 0; tau < 2; ++tau)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float x = 4 * tau + e < nv ? s[tau][e] : -INFINITY;
                    s[tau][e] = x;
                    mx = fmaxf(mx, x);
                }
            mx = rows4_max(mx);
            mx *= sl2;
            if (__any(mx > m_run + kSlack)) {
                const float m_new = fmaxf(m_run, mx);
                const float alpha = m_new == -INFINITY ? 1.f : fast_exp2(m_run - m_new);
                l_run *= alpha;
                m_run = m_new;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float ae = __shfl(alpha, grp * 4 + e, 64);
#pragma unroll
                    for (int nt = 0; nt < NT; ++nt) o[nt][e] *= ae;
                }
            }
            const float m_use = m_run == -INFINITY ? 0.f : m_run;
            float ls = 0.f;
#pragma unroll
            for (int tau = 0; tau < 2; ++tau)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float v = fast_exp2(fmaf(s[tau][e], sl2, -m_use));
                    s[tau][e] = v;
                    ls += v;
                }
            l_run += ls;
            const bf16x8 pf = to_bf16x8(s[0], s[1]);  // keys 8 grp .. 8 grp + 7 in order
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) o[nt] = mfma16(pf, st.v[nt], o[nt]);
        };

        // The next step's loads are issued before every step's compute, also
        // past the item's end (they then re-read its last page, still in L2):
        // no branch skips a load, so the compiler's counted waits leave the
        // prefetched step in flight while the current one is multiplied.
        DecodeStep<HD> sa, sb;
        decode_load<HD>(sa, kpool, vpool, bt_s, tok0, last_pg, a.hkv, kvh, col, grp);
        for (int c0 = tok0;; c0 += 64) {
            decode_load<HD>(sb, kpool, vpool, bt_s, c0 + 32, last_pg, a.hkv, kvh, col, grp);
            compute(sa, c0);
            if (c0 + 32 >= tok1) break;
            decode_load<HD>(sa, kpool, vpool, bt_s, c0 + 64, last_pg, a.hkv, kvh, col, grp);
            compute(sb, c0 + 32);
            if (c0 + 64 >= tok1) break;
        }

        float l = l_run;
        l = rows4_sum(l);
        const size_t hbase = static_cast<size_t>(w) * a.hq + kvh * group;
        if (grp == 0 && col < group) {
            a.part_ml[(hbase + col) * 2 + 0] = m_run;
            a.part_ml[(hbase + col) * 2 + 1] = l;
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int h = grp * 4 + e;
            if (h < group) {
#pragma unroll
                for (int nt = 0; nt < NT; ++nt) a.part_o[(hbase + h) * HD + nt * 16 + col] = o[nt][e];
            }
        }
    }
}

template <int HD>
__global__ __launch_bounds__(64, 2) void decode_attn_kernel(DecodeAttnArgs a) {
    decode_attn_wave<HD>(a, blockIdx.x, blockIdx.y, threadIdx.x);
}

// Merge the items of one (decode, q head): weights 2^(m_s - max m).
template <int HD>
__device__ __forceinline__ void decode_merge_row(const DecodeAttnArgs& a, int b, int h) {
    const int w0 = a.work_off[b], w1 = a.work_off[b + 1];
    merge_row<HD>(a.part_ml, a.part_o, static_cast<size_t>(w0) * a.hq + h, a.hq, w1 - w0,
                  static_cast<bf16*>(a.out) + static_cast<size_t>(b) * a.hq * HD + h * HD);
}

// One launch for both merges of a layer: blocks x < chunk_rows combine the
// partials of position x of the flattened query tiles (tiles split over
// several items), the rest those of decode x - chunk_rows; wave w of block
// (x, y) takes q head y * WAVES + w.
template <int HD, int GROUP, int WAVES>
__global__ __launch_bounds__(64 * WAVES) void attn_merge_kernel(ChunkAttnArgs ca, DecodeAttnArgs da,
                                                                int chunk_rows) {
    const int x = blockIdx.x, h = blockIdx.y * WAVES + (threadIdx.x >> 6);
    if (x < chunk_rows) chunk_merge_row<HD, GROUP>(ca, x, h);
    else decode_merge_row<HD>(da, x - chunk_rows, h);
}

template <int HD, int GROUP>
void launch_chunk_g(const ChunkAttnArgs& a, hipStream_t s) {
    chunk_attn_kernel<HD, GROUP, kChunkStages, false><<<a.n_slots * a.hkv, 512, 0, s>>>(a, DecodeAttnArgs{});
}

template <int HD, int GROUP>
void launch_both_g(const ChunkAttnArgs& ca, const DecodeAttnArgs& da, hipStream_t s) {
    const int blocks = ca.n_slots * ca.hkv + (da.n_slots * da.hkv + 7) / 8;
    chunk_attn_kernel<HD, GROUP, kChunkStages, true><<<blocks, 512, 0, s>>>(ca, da);
}

template <int HD, int GROUP>
void launch_merge_g(const ChunkAttnArgs& ca, const DecodeAttnArgs& da, int chunk_rows, int hq, hipStream_t s) {
    // four heads per work-group where they divide evenly: a quarter of the
    // (tiny) work-groups to dispatch
    if (hq % 4 == 0)
        attn_merge_kernel<HD, GROUP, 4><<<dim3(chunk_rows + da.b, hq / 4), 256, 0, s>>>(ca, da, chunk_rows);
    else
        attn_merge_kernel<HD, GROUP, 1><<<dim3(chunk_rows + da.b, hq), 64, 0, s>>>(ca, da, chunk_rows);
}

template <int HD>
void launch_merge_hd(const ChunkAttnArgs& ca, const DecodeAttnArgs& da, int chunk_rows, int group, int hq,
                     hipStream_t s) {
    switch (group) {
        case 1: launch_merge_g<HD, 1>(ca, da, chunk_rows, hq, s); break;
        case 2: launch_merge_g<HD, 2>(ca, da, chunk_rows, hq, s); break;
        case 4: launch_merge_g<HD, 4>(ca, da, chunk_rows, hq, s); break;
        case 8: launch_merge_g<HD, 8>(ca, da, chunk_rows, hq, s); break;
        default: launch_merge_g<HD, 16>(ca, da, chunk_rows, hq, s); break;
    }
}

template <int HD>
void launch_chunk_hd(const ChunkAttnArgs& a, hipStream_t s) {
    switch (a.hq / a.hkv) {
        case 1: launch_chunk_g<HD, 1>(a, s); break;
        case 2: launch_chunk_g<HD, 2>(a, s); break;
        case 4: launch_chunk_g<HD, 4>(a, s); break;
        case 8: launch_chunk_g<HD, 8>(a, s); break;
        default: launch_chunk_g<HD, 16>(a, s); break;
    }
}

template <int HD>
void launch_both_hd(const ChunkAttnArgs& ca, const DecodeAttnArgs& da, hipStream_t s) {
    switch (ca.hq / ca.hkv) {
        case 1: launch_both_g<HD, 1>(ca, da, s); break;
        case 2: launch_both_g<HD, 2>(ca, da, s); break;
        case 4: launch_both_g<HD, 4>(ca, da, s); break;
        case 8: launch_both_g<HD, 8>(ca, da, s); break;
        default: launch_both_g<HD, 16>(ca, da, s); break;
    }
}

}  // namespace

void launch_attention(const ChunkAttnArgs& ca, const DecodeAttnArgs& da, hipStream_t s) {
    if (ca.c <= 0 || ca.n_items <= 0) {
        launch_decode_attention_split(da, s);
        return;
    }
    if (da.b <= 0) {
        launch_chunk_attention(ca, s);
        return;
    }
    if (ca.hd == 128) launch_both_hd<128>(ca, da, s);
    else launch_both_hd<64>(ca, da, s);
}

void launch_chunk_attention(const ChunkAttnArgs& a, hipStream_t s) {
    if (a.c <= 0 || a.n_items <= 0) return;
    if (a.hd == 128) launch_chunk_hd<128>(a, s);
    else launch_chunk_hd<64>(a, s);
}

void launch_decode_attention_split(const DecodeAttnArgs& a, hipStream_t s) {
    if (a.b <= 0) return;
    dim3 grid(a.n_slots, a.hkv);
    if (a.hd == 128) decode_attn_kernel<128><<<grid, 64, 0, s>>>(a);
    else decode_attn_kernel<64><<<grid, 64, 0, s>>>(a);
}

void launch_attention_merge(const ChunkAttnArgs* ca, const DecodeAttnArgs* da, hipStream_t s) {
    // every position of every query tile (positions past a tile's rows return at once)
    const int chunk_rows = ca && ca->c > 0 && ca->split ? ca->n_qt * chunk_tile_positions(ca->hq / ca->hkv) : 0;
    DecodeAttnArgs dd{};
    if (da && da->b > 0) dd = *da;
    if (chunk_rows + dd.b == 0) return;
    ChunkAttnArgs cc{};
    if (ca) cc = *ca;
    const int hq = chunk_rows ? cc.hq : dd.hq, hkv = chunk_rows ? cc.hkv : dd.hkv, hd = chunk_rows ? cc.hd : dd.hd;
    if (hd == 128) launch_merge_hd<128>(cc, dd, chunk_rows, hq / hkv, hq, s);
    else launch_merge_hd<64>(cc, dd, chunk_rows, hq / hkv, hq, s);
}

}  // namespace slw
