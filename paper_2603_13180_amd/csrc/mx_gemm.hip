// MX matrix product H = dec(A) dec(B)^T on the gfx950 block-scaled matrix
// cores (Sec. 3.7 eq. (mx-matmul): the product MXNormLinear takes of MXNorm's
// output and the gain-folded weight cast; the implementation appendix's
// mx_norm_linear_forward ends in this product).
//
// A [M, K] (activations, MXNorm codes) and B [N, K] (weights) are both blocked
// along K with one E8M0 scale per 32 elements; elements are E4M3 (one byte)
// or E2M1 (two per byte, element 2j in the low nibble).  The hardware
// instruction v_mfma_scale_f32_16x16x128_f8f6f4 multiplies a 16x128 tile of
// each operand with one scale byte per row and 32-element block applied
// exactly, accumulating in fp32.
//
// Tiling: a workgroup of 8 waves (two per SIMD) computes a 256 (M) x 256 (N)
// output tile; wave w owns the 128 x 64 quarter-column (w & 1, w >> 1) as
// 8 x 4 matrix-core tiles of 16 x 16, 128 accumulator registers.  Two waves
// per SIMD are what lets the matrix core run while the other wave waits on
// LDS or a barrier: with one wave per SIMD the E2M1 instruction issues at
// about half its rate.  The K loop moves 128 bytes of every row per step
// (128 E4M3 or 256 E2M1 elements) from global memory straight into LDS
// (16-byte global_load_lds, no staging registers) into two stages of 66 KB;
// each step reads its four B fragments into registers and streams the eight
// A fragments two ahead of the matrix core.  In LDS, 16-byte chunk c of row r
// lives at chunk c ^ (r & 7) of the row, so the fragment reads of 8
// consecutive rows hit distinct banks.
//
// What bounds it: at 256 x 256 the operand stream is 64 KB per K step per
// workgroup, about 10 TB/s of L2 requests at half the fp8 peak.  Two stages
// fill LDS, so the DMA runs one step ahead of the products and each step
// waits for it; the tile's stores slow the operand stream (the non-temporal
// policy below halves that); and after each step's barrier every wave reads
// fragments before its first product.  The eight waves' accumulators fill
// half the register file, which leaves no room for a third stage in
// registers.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>
#include <type_traits>

#include "mxnorm.h"
#include "status.h"

namespace mxg {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
#define LDS_AS __attribute__((address_space(3)))

constexpr int BM = 256;    // tile rows of A (M)
constexpr int BN = 256;    // tile rows of B (N)
constexpr int KB = 128;    // bytes of each row per K step
constexpr int NT = 512;    // threads: 8 waves, two per SIMD
constexpr int WTM = 128;   // wave tile along M
constexpr int WTN = 64;    // wave tile along N
constexpr int FM = WTM / 16, FN = WTN / 16;
constexpr int GROUP_M = 4; // tile rows per group in the visiting order
constexpr int NXCD = 8;

// scale bytes per row and K step: 4 blocks of 32 (E4M3), 8 blocks (E2M1)
template <int ELEM> struct Op {
    static constexpr int SB = ELEM == MX_ELEM_E2M1 ? 8 : 4;
    static constexpr int STAGE = (BM + BN) * KB + (BM + BN) * SB;
};

struct Args {
    const uint8_t *a, *as, *b, *bs;
    const uint16_t *bgain; // bf16 [N] or NULL
    void *out;
    int64_t M, N;
    int64_t rb;   // code bytes per row
    int64_t rs;   // scale bytes per row
    int steps;    // K steps of KB bytes
    int tiles_m, tiles_n;
    int xcd_ranges; // 1: each XCD runs a contiguous range of tiles; 0: round robin
    int grid_max;   // workgroups resident at once: one per compute unit
};

// Global -> LDS DMA loads: lane i of the wave reads gbase + off_i (gbase
// wave-uniform, in SGPRs; off_i a 32-bit lane offset) and writes the bytes at
// LDS address lds_base + bytes * i (lds_base wave-uniform, passed in M0).
// Written as inline asm rather than with the compiler builtin: for the builtin
// the compiler cannot tell that the LDS reads of one stage do not alias the
// DMA into the other, and would wait for the prefetch before every read.  The
// waits are explicit (wait_vmcnt) instead.  An LDS DMA needs one wait state
// after the scalar write of M0 that the compiler places just before the asm:
// hence the s_nop.
__device__ __forceinline__ void lds_load16(const void *gbase, uint32_t off, uint32_t lds_base)
{
    asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(gbase),
                 "{m0}"(lds_base)
                 : "memory");
}

__device__ __forceinline__ void lds_load4(const void *gbase, uint32_t off, uint32_t lds_base)
{
    asm volatile("s_nop 0\n\tglobal_load_lds_dword %0, %1" ::"v"(off), "s"(gbase),
                 "{m0}"(lds_base)
                 : "memory");
}

// Wait until at most N_ of this wave's vector memory operations (loads and
// stores, which complete in issue order) are outstanding.
template <int N_> __device__ __forceinline__ void wait_vmcnt()
{
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N_) : "memory");
}

// Workgroup barrier without the memory fence of __syncthreads(): the fence
// would wait for every outstanding load, including the DMA of the next step.
// LDS written by the DMA is covered by the vmcnt wait each wave makes before
// arriving; the lgkmcnt(0) completes this wave's own LDS reads, so that a
// stage read before the barrier can be refilled after it.  The "memory"
// clobber keeps the compiler from moving LDS accesses across it.
__device__ __forceinline__ void barrier()
{
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Per-lane part of the DMA addresses, fixed for the whole K loop: byte
// offsets, relative to the tile's first row, of the rows this lane moves.
// Wave w moves code rows 32w .. 32w+31 of both tiles (4 instructions of
// 8 rows x 128 bytes each: lane l fills LDS slot l % 8 of row l / 8 of its
// group, which holds source chunk (l % 8) ^ (l / 8)); waves 0-3 move the
// scale bytes of A's rows 64w .. 64w+63, waves 4-7 those of B's rows
// 64(w-4) .. 64(w-4)+63 (lane i of scale instruction u moves dword
// i % (SB/4) of row u (64 / (SB/4)) + i / (SB/4)).  Rows past M or N read
// row M-1 or N-1: their results are never stored.
template <int ELEM> struct Rows {
    uint32_t a[4], b[4];
    uint32_t s[Op<ELEM>::SB / 4];
};

template <int ELEM>
__device__ __forceinline__ Rows<ELEM> lane_rows(const Args &A, int64_t m0, int64_t n0, int w,
                                                int l)
{
    constexpr int DW = Op<ELEM>::SB / 4;
    Rows<ELEM> R;
    const int rr = l >> 3;       // row within the 8-row group
    const int ch = (l & 7) ^ rr; // source chunk for this LDS slot (the swizzle)
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        const int r = 32 * w + 8 * t + rr;
        R.a[t] = (uint32_t)((min(m0 + r, A.M - 1) - m0) * A.rb) + 16 * ch;
        R.b[t] = (uint32_t)((min(n0 + r, A.N - 1) - n0) * A.rb) + 16 * ch;
    }
    const bool on_a = w < 4;
    const int64_t base = on_a ? m0 : n0, lim = on_a ? A.M : A.N;
#pragma unroll
    for (int u = 0; u < DW; ++u) {
        const int r = 64 * (w & 3) + u * (64 / DW) + l / DW;
        R.s[u] = (uint32_t)((min(base + r, lim - 1) - base) * A.rs) + 4 * (l % DW);
    }
    return R;
}

// Issue this wave's loads of K step s into one LDS stage, laid out as
// [A codes 256 x 128][B codes 256 x 128][A scales 256 x SB][B scales 256 x SB].
template <int ELEM>
__device__ __forceinline__ void issue_step(const uint8_t *ta, const uint8_t *tb,
                                           const uint8_t *tsa, const uint8_t *tsb,
                                           const Rows<ELEM> &R, int s, uint32_t stage, int w)
{
    constexpr int SB = Op<ELEM>::SB;
    constexpr int DW = SB / 4;
    const uint32_t xa = stage;
    const uint32_t xb = stage + BM * KB;
    const uint32_t kc = (uint32_t)s * KB, ks = (uint32_t)s * SB;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        lds_load16(ta, R.a[t] + kc, xa + (32 * w + 8 * t) * KB);
        lds_load16(tb, R.b[t] + kc, xb + (32 * w + 8 * t) * KB);
    }
    const uint8_t *ts = w < 4 ? tsa : tsb;
    const uint32_t xs = stage + (BM + BN) * KB + (w < 4 ? 0 : BM * SB) + 64 * (w & 3) * SB;
#pragma unroll
    for (int u = 0; u < DW; ++u)
        lds_load4(ts, R.s[u] + ks, xs + u * (64 / DW) * SB);
}

__device__ __forceinline__ v8i join(u32x4 lo, u32x4 hi)
{
    return __builtin_bit_cast(v8i, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// two floats to bf16 (round to nearest even, on gfx950's conversion unit),
// the first in the low half
__device__ __forceinline__ uint32_t pack_bf16(float a, float b)
{
    const __bf16 x = (__bf16)a, y = (__bf16)b;
    return (uint32_t)__builtin_bit_cast(uint16_t, x) |
           ((uint32_t)__builtin_bit_cast(uint16_t, y) << 16);
}

// One operand fragment for a 16-row group and one K step: lane (g, q) holds
// the 16-byte chunks g and 4+g of row r (E4M3: k = 16g..16g+15 and
// 64+16g..64+16g+15 of the step, the matrix core's own k order for this
// operand size; E2M1: chunk g is the 32-element block g of the first
// instruction, chunk 4+g block g of the second) and the E8M0 scale bytes of
// the blocks it supplies (E4M3: block g; E2M1: blocks g and 4+g).
struct Frag {
    v8i v;
    int s0, s1;
};

// Lane-relative LDS offsets of one operand's fragments within a stage: the
// lane reads row r0 + qd (+16 j for fragment j) at chunks g and 4 + g,
// swizzled by (r0 + qd) & 7 = qd & 7 (r0 is a multiple of 16), and the
// scale bytes g (and 4 + g) of that row.
struct FragBase {
    uint32_t lo, hi, sc;
};

template <int ELEM>
__device__ __forceinline__ FragBase frag_base(uint32_t codes_off, uint32_t scales_off, int r0,
                                              int qd, int g)
{
    constexpr int SB = Op<ELEM>::SB;
    FragBase b;
    b.lo = codes_off + (r0 + qd) * KB + 16 * (g ^ (qd & 7));
    b.hi = codes_off + (r0 + qd) * KB + 16 * ((4 + g) ^ (qd & 7));
    b.sc = scales_off + (r0 + qd) * SB + g;
    return b;
}

// fragment J of an operand from the stage at st; the row offset J*16 rows is
// a compile-time constant that the LDS reads take as their immediate offset
template <int ELEM, int J>
__device__ __forceinline__ Frag read_frag(const LDS_AS uint8_t *st, const FragBase &b)
{
    constexpr int SB = Op<ELEM>::SB;
    Frag f;
    const u32x4 lo = *reinterpret_cast<const LDS_AS u32x4 *>(st + b.lo + J * 16 * KB);
    const u32x4 hi = *reinterpret_cast<const LDS_AS u32x4 *>(st + b.hi + J * 16 * KB);
    f.v = join(lo, hi);
    f.s0 = st[b.sc + J * 16 * SB];
    f.s1 = ELEM == MX_ELEM_E2M1 ? (int)st[b.sc + J * 16 * SB + 4] : 0;
    return f;
}

// acc += B-fragment x A-fragment over one E4M3 K step (B is the
// instruction's first operand: each lane's four results are then four
// consecutive columns of one row of H)
__device__ __forceinline__ void mma_e4m3(v4f &acc, const Frag &b, const Frag &a)
{
    acc = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(b.v, a.v, acc, 0, 0, 0, b.s0, 0, a.s0);
}

// The products of one K step from the stage at st: the step's four B
// fragments held in registers, the eight A fragments streamed, each requested
// two ahead of the products that use it.
template <int ELEM>
__device__ __forceinline__ void step_products(v4f (&acc)[FN][FM], const LDS_AS uint8_t *st,
                                              const FragBase &ba, const FragBase &bb)
{
    if constexpr (ELEM == MX_ELEM_E2M1) {
        // Whole fragments, read in the E4M3 order below (the lane's low and
        // high 16-byte chunks each feed one instruction: E2M1 blocks g and
        // 4 + g of the step).  Per column, the four tiles' products of the
        // low halves, then those of the high halves: an accumulator's two
        // instructions sit four apart, not back to back (where the second
        // waits for the first's result), in the same order of additions.
        // (Two passes over the 32 tiles, every low half and then every high
        // half from half-fragment reads, were 1.5-3% slower at the QKV and
        // gate+up shapes.)
        const v8i z = {0, 0, 0, 0, 0, 0, 0, 0};
        auto lo = [&](v4f &acc, const Frag &b, const Frag &a) {
            const v8i b0 = __builtin_shufflevector(b.v, z, 0, 1, 2, 3, 8, 8, 8, 8);
            const v8i a0 = __builtin_shufflevector(a.v, z, 0, 1, 2, 3, 8, 8, 8, 8);
            acc = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(b0, a0, acc, 4, 4, 0, b.s0, 0,
                                                                   a.s0);
        };
        auto hi = [&](v4f &acc, const Frag &b, const Frag &a) {
            const v8i b1 = __builtin_shufflevector(b.v, z, 4, 5, 6, 7, 8, 8, 8, 8);
            const v8i a1 = __builtin_shufflevector(a.v, z, 4, 5, 6, 7, 8, 8, 8, 8);
            acc = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(b1, a1, acc, 4, 4, 0, b.s1, 0,
                                                                   a.s1);
        };
        Frag fb[FN], fa[FM];
        fb[0] = read_frag<ELEM, 0>(st, bb);
        fb[1] = read_frag<ELEM, 1>(st, bb);
        fa[0] = read_frag<ELEM, 0>(st, ba);
        __builtin_amdgcn_sched_barrier(0);
        fb[2] = read_frag<ELEM, 2>(st, bb);
        fb[3] = read_frag<ELEM, 3>(st, bb);
        fa[1] = read_frag<ELEM, 1>(st, ba);
        __builtin_amdgcn_sched_barrier(0);
        auto column = [&](auto jc) {
            constexpr int j = decltype(jc)::value;
            if constexpr (j + 2 < FM)
                fa[j + 2] = read_frag<ELEM, j + 2>(st, ba);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int i = 0; i < FN; ++i)
                lo(acc[i][j], fb[i], fa[j]);
#pragma unroll
            for (int i = 0; i < FN; ++i)
                hi(acc[i][j], fb[i], fa[j]);
            __builtin_amdgcn_sched_barrier(0);
        };
        column(std::integral_constant<int, 0>{});
        column(std::integral_constant<int, 1>{});
        column(std::integral_constant<int, 2>{});
        column(std::integral_constant<int, 3>{});
        column(std::integral_constant<int, 4>{});
        column(std::integral_constant<int, 5>{});
        column(std::integral_constant<int, 6>{});
        column(std::integral_constant<int, 7>{});
        return;
    }
    // The step starts with every wave reading fragments after the barrier:
    // B0, B1 and A0 first, so that the first two products wait for three
    // fragments, not six (QKV shape: 1-3% faster).
    Frag fb[FN], fa[FM];
    fb[0] = read_frag<ELEM, 0>(st, bb);
    fb[1] = read_frag<ELEM, 1>(st, bb);
    fa[0] = read_frag<ELEM, 0>(st, ba);
    __builtin_amdgcn_sched_barrier(0);
    fb[2] = read_frag<ELEM, 2>(st, bb);
    fb[3] = read_frag<ELEM, 3>(st, bb);
    fa[1] = read_frag<ELEM, 1>(st, ba);
    __builtin_amdgcn_sched_barrier(0);
    fa[2] = read_frag<ELEM, 2>(st, ba);
    __builtin_amdgcn_sched_barrier(0);
    mma_e4m3(acc[0][0], fb[0], fa[0]);
    mma_e4m3(acc[1][0], fb[1], fa[0]);
    __builtin_amdgcn_sched_barrier(0);
    mma_e4m3(acc[2][0], fb[2], fa[0]);
    mma_e4m3(acc[3][0], fb[3], fa[0]);
    __builtin_amdgcn_sched_barrier(0);
    auto column = [&](auto jc) {
        constexpr int j = decltype(jc)::value;
        if constexpr (j + 2 < FM)
            fa[j + 2] = read_frag<ELEM, j + 2>(st, ba);
        // keep the read ahead of this fragment's products
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < FN; ++i)
            mma_e4m3(acc[i][j], fb[i], fa[j]);
        __builtin_amdgcn_sched_barrier(0);
    };
    column(std::integral_constant<int, 1>{});
    column(std::integral_constant<int, 2>{});
    column(std::integral_constant<int, 3>{});
    column(std::integral_constant<int, 4>{});
    column(std::integral_constant<int, 5>{});
    column(std::integral_constant<int, 6>{});
    column(std::integral_constant<int, 7>{});
}

// Output stores bypass the caches' normal allocation (cache policy sc0 sc1
// nt: system scope, non-temporal): H is written once and read by a later
// kernel, and with the default policy the stores slow the operand stream
// more (QKV shape, E4M3 -> bf16: 720 -> 673 us).
constexpr int kStorePolicy = 0x13;

// stores per wave and tile
template <int OUT> constexpr int kTileStores = OUT == MX_OUT_F32 ? FM * FN : FM * FN / 2;

// Store the workgroup's accumulators as H[m0 .., n0 ..] (f32 or bf16), times
// the column gain if there is one.  Every lane runs the same stores (exactly
// kTileStores of them when the tile lies inside H); lanes outside H are
// masked.
template <int OUT>
__device__ __forceinline__ void store_tile(const Args &A, const v4f (&acc)[FN][FM], int64_t m0,
                                           int64_t n0, int wm, int wn, int g, int qd)
{
    // lane (g, qd) of tile (i, j) holds H[m][n .. n+3] with
    // m = m0 + wm + 16 j + qd and n = n0 + wn + 16 i + 4 g.  N is a multiple
    // of 16, so a tile column base below N has its 16 columns inside H.
    // The gains of the lane's columns are loaded before any store.
    uint2 gw[FN];
    if (A.bgain) {
#pragma unroll
        for (int i = 0; i < FN; ++i) {
            const int64_t n = n0 + wn + 16 * i + 4 * g;
            gw[i] = *reinterpret_cast<const uint2 *>(A.bgain + (n < A.N ? n : 0));
        }
    }
    auto gained = [&](int i, int j) {
        v4f v = acc[i][j];
        if (A.bgain) {
            v[0] = v[0] * __uint_as_float(gw[i].x << 16);
            v[1] = v[1] * __uint_as_float(gw[i].x & 0xFFFF0000u);
            v[2] = v[2] * __uint_as_float(gw[i].y << 16);
            v[3] = v[3] * __uint_as_float(gw[i].y & 0xFFFF0000u);
        }
        return v;
    };
    constexpr int ES = OUT == MX_OUT_F32 ? 4 : 2; // bytes per element
#pragma unroll
    for (int j = 0; j < FM; ++j) {
        // buffer over the 16 rows of tile row j (byte offsets below 2^31:
        // the host limits N)
        const int64_t mr = m0 + wm + 16 * j;
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            static_cast<uint8_t *>(A.out) + mr * A.N * ES, 0, 0x7FFFFFFF, 0x00020000);
        const int64_t m = mr + qd;
        const uint32_t row = (uint32_t)(qd * A.N) * ES;
        if constexpr (OUT == MX_OUT_F32) {
#pragma unroll
            for (int i = 0; i < FN; ++i) {
                const int64_t n = n0 + wn + 16 * i + 4 * g;
                const v4f v = gained(i, j);
                if (m < A.M && n < A.N)
                    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), rs,
                                                           (int)(row + (uint32_t)n * 4), 0,
                                                           kStorePolicy);
            }
        } else {
            // bf16: tiles i and i+1 are stored together.  v_permlane16_swap
            // trades the odd lane rows (g = 1, 3) of tile i's values with the
            // even lane rows (g = 0, 2) of tile i+1's, after which lane row g
            // holds 8 adjacent columns, 16 bytes, of tile i + (g & 1) from
            // column 8 (g >> 1): one 16-byte store per lane and tile pair
            // instead of two 8-byte stores.  The swap runs on every lane; only
            // the stores are masked.
            static_assert(FN % 2 == 0, "tiles are stored in pairs");
#pragma unroll
            for (int i = 0; i < FN; i += 2) {
                uint32_t lo[2], hi[2];
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const v4f v = gained(i + h, j);
                    lo[h] = pack_bf16(v[0], v[1]);
                    hi[h] = pack_bf16(v[2], v[3]);
                }
                const auto sl = __builtin_amdgcn_permlane16_swap(lo[0], lo[1], false, false);
                const auto sh = __builtin_amdgcn_permlane16_swap(hi[0], hi[1], false, false);
                const int64_t n = n0 + wn + 16 * (i + (g & 1)) + 8 * (g >> 1);
                if (m < A.M && n < A.N)
                    __builtin_amdgcn_raw_buffer_store_b128(u32x4{sl[0], sh[0], sl[1], sh[1]}, rs,
                                                           (int)(row + (uint32_t)n * 2), 0,
                                                           kStorePolicy);
            }
        }
    }
}

template <int ELEM, int OUT>
__global__ void __launch_bounds__(NT) mx_gemm_kernel(Args A)
{
    constexpr int SB = Op<ELEM>::SB;
    constexpr int STAGE = Op<ELEM>::STAGE;
    __shared__ __attribute__((aligned(16))) uint8_t lds[2 * STAGE];

    // Tiles.  The grid is at most one workgroup per compute unit, and
    // workgroup b takes tiles v = b, b + grid, b + 2 grid, ...  Dispatch is
    // round robin over the XCDs (each with its own L2).  With xcd_ranges, v
    // is renumbered so that each XCD runs a contiguous range of tiles; either
    // way the tiles are visited in groups of GROUP_M tile rows that share
    // operand blocks.
    const int G = A.tiles_m * A.tiles_n;
    auto tile_of = [&](int v, int64_t &m0, int64_t &n0) {
        int pid = v;
        if (A.xcd_ranges) {
            const int xcd = v % NXCD, loc = v / NXCD;
            const int q = G / NXCD, rem = G % NXCD;
            pid = xcd < rem ? xcd * (q + 1) + loc : rem * (q + 1) + (xcd - rem) * q + loc;
        }
        const int in_group = GROUP_M * A.tiles_n;
        const int first_m = (pid / in_group) * GROUP_M;
        const int gsz = min(A.tiles_m - first_m, GROUP_M);
        m0 = (int64_t)(first_m + (pid % in_group) % gsz) * BM;
        n0 = (int64_t)((pid % in_group) / gsz) * BN;
    };

    const int tid = threadIdx.x;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6); // wave-uniform
    const int l = tid & 63;
    const int g = l >> 4, qd = l & 15; // lane group (K block / output row quad), row in fragment
    const int wm = (w & 1) * WTM, wn = (w >> 1) * WTN;

    LDS_AS uint8_t *st0 = (LDS_AS uint8_t *)lds;
    const uint32_t st0_addr = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)st0);
    const FragBase ba = frag_base<ELEM>(0, (BM + BN) * KB, wm, qd, g);
    const FragBase bb = frag_base<ELEM>(BM * KB, (BM + BN) * KB + BM * SB, wn, qd, g);

    int v = blockIdx.x;
    int64_t m0, n0;
    tile_of(v, m0, n0);
    Rows<ELEM> R = lane_rows<ELEM>(A, m0, n0, w, l);

    // Pipeline, one barrier per K step.  At the top of a step every wave has
    // its own DMA of the step landed (vmcnt) and, past the barrier, so has
    // every other wave, and no wave still reads the other stage (the previous
    // step): the DMA of the next step goes there, and after a tile's last
    // step the DMA of the next tile's first step, which then runs under that
    // last step's products and the tile's stores.
    issue_step<ELEM>(A.a + m0 * A.rb, A.b + n0 * A.rb, A.as + m0 * A.rs, A.bs + n0 * A.rs, R, 0,
                     st0_addr, w);
    bool prev_full = false; // the previous tile lies inside H (all its stores ran)
    for (int gs = 0;;) {
        v4f acc[FN][FM];
#pragma unroll
        for (int i = 0; i < FN; ++i)
#pragma unroll
            for (int j = 0; j < FM; ++j)
                acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};
        const int nv = v + (int)gridDim.x;
        int64_t m1 = 0, n1 = 0;
        for (int s = 0; s < A.steps; ++s, ++gs) {
            const int cur = gs & 1;
            // this step's DMA has landed.  In a tile's first step the
            // previous tile's stores, issued after this DMA, need not have
            // completed: operations complete in order, so at most that many
            // may remain (a partial tile ran fewer stores: wait for all).
            if (s == 0 && prev_full)
                wait_vmcnt<kTileStores<OUT>>();
            else
                wait_vmcnt<0>();
            barrier();
            const uint32_t nxt = st0_addr + (cur ^ 1) * STAGE;
            if (s + 1 < A.steps) {
                issue_step<ELEM>(A.a + m0 * A.rb, A.b + n0 * A.rb, A.as + m0 * A.rs,
                                 A.bs + n0 * A.rs, R, s + 1, nxt, w);
            } else if (nv < G) {
                tile_of(nv, m1, n1);
                R = lane_rows<ELEM>(A, m1, n1, w, l);
                issue_step<ELEM>(A.a + m1 * A.rb, A.b + n1 * A.rb, A.as + m1 * A.rs,
                                 A.bs + n1 * A.rs, R, 0, nxt, w);
            }
            step_products<ELEM>(acc, st0 + cur * STAGE, ba, bb);
        }
        store_tile<OUT>(A, acc, m0, n0, wm, wn, g, qd);
        prev_full = m0 + BM <= A.M && n0 + BN <= A.N;
        if (nv >= G)
            break;
        v = nv;
        m0 = m1;
        n0 = n1;
    }
}

template <int ELEM, int OUT>
hipError_t launch(const Args &A, hipStream_t stream)
{
    const int G = A.tiles_m * A.tiles_n;
    const int grid = G < A.grid_max ? G : A.grid_max;
    hipLaunchKernelGGL((mx_gemm_kernel<ELEM, OUT>), dim3((unsigned)grid), dim3(NT), 0, stream, A);
    return hipGetLastError();
}

} // namespace mxg

// host side -------------------------------------------------------------------

namespace {

bool aligned(const void *p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

// Compute units of the device `stream` runs on (the current device for the
// null stream), looked up once per device; 0 if unknown.
int compute_units(hipStream_t stream)
{
    static std::atomic<int> cache[64];
    int dev = -1;
    if (stream) {
        hipDevice_t hd;
        if (hipStreamGetDevice(static_cast<hipStream_t>(stream), &hd) != hipSuccess)
            return 0;
        dev = (int)hd;
    } else if (hipGetDevice(&dev) != hipSuccess) {
        return 0;
    }
    if (dev < 0 || dev >= 64)
        return 0;
    int n = cache[dev].load(std::memory_order_relaxed);
    if (n == 0) {
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            n <= 0)
            return 0;
        cache[dev].store(n, std::memory_order_relaxed);
    }
    return n;
}

} // namespace

extern "C" {

mx_status mx_matmul_fwd(const uint8_t *a_codes, const uint8_t *a_scales, const uint8_t *b_codes,
                        const uint8_t *b_scales, int64_t M, int64_t N, int64_t K, int block,
                        int elem, const void *b_gain, int out_dtype, void *out, hipStream_t stream)
{
    mxk::clear_error();
    if (M < 0 || N < 0 || K <= 0)
        return mxk::fail(MX_EINVAL, "M and N must be >= 0 and K > 0");
    if (elem != MX_ELEM_E4M3 && elem != MX_ELEM_E2M1)
        return mxk::fail(MX_EINVAL, "elem must be MX_ELEM_E4M3 or MX_ELEM_E2M1");
    if (out_dtype != MX_OUT_F32 && out_dtype != MX_OUT_BF16)
        return mxk::fail(MX_EINVAL, "out_dtype must be MX_OUT_F32 or MX_OUT_BF16");
    if (block != 32)
        return mxk::fail(MX_EUNSUPPORTED, "the matrix cores apply one scale per 32 elements: block must be 32");
    const int64_t kstep = elem == MX_ELEM_E2M1 ? 256 : 128;
    if (K % kstep != 0)
        return mxk::fail(MX_EUNSUPPORTED, "K must be a multiple of 128 (E4M3) or 256 (E2M1)");
    if (N % 16 != 0)
        return mxk::fail(MX_EUNSUPPORTED, "N must be a multiple of 16");
    if (K > MX_MATMUL_MAX_K)
        return mxk::fail(MX_EUNSUPPORTED, "K exceeds %d", MX_MATMUL_MAX_K);
    if (M == 0 || N == 0)
        return MX_OK;
    if (!a_codes || !a_scales || !b_codes || !b_scales || !out)
        return mxk::fail(MX_EINVAL, "NULL pointer");
    if (!aligned(a_codes, 16) || !aligned(b_codes, 16) || !aligned(a_scales, 4) ||
        !aligned(b_scales, 4) || !aligned(out, 16) ||
        (b_gain && !aligned(b_gain, 8)))
        return mxk::fail(MX_EINVAL, "codes and out must be 16-byte, scales 4-byte and b_gain "
                               "8-byte aligned");
    const int64_t tm = (M + mxg::BM - 1) / mxg::BM, tn = (N + mxg::BN - 1) / mxg::BN;
    if (tm * tn > INT32_MAX / 2 || M > INT32_MAX || N > MX_MATMUL_MAX_N)
        return mxk::fail(MX_EUNSUPPORTED, "problem too large (N at most %d)", MX_MATMUL_MAX_N);
    mxg::Args A;
    A.a = a_codes;
    A.as = a_scales;
    A.b = b_codes;
    A.bs = b_scales;
    A.bgain = static_cast<const uint16_t *>(b_gain);
    A.out = out;
    A.M = M;
    A.N = N;
    A.rb = elem == MX_ELEM_E2M1 ? K / 2 : K;
    A.rs = K / 32;
    A.steps = (int)(A.rb / mxg::KB);
    A.tiles_m = (int)tm;
    A.tiles_n = (int)tn;
    // Tile order: each XCD runs a contiguous range of tiles.  Measured at
    // d = 4096 on MI355X against plain round robin: the QKV shape 737 vs
    // 801 us; the gate+up shape (N = 28672) 1583 vs 1715 us at M = 16384 and
    // 3214 vs 3446 us at M = 32768 (E2M1: 958 vs 1019 us).  (Before the
    // output stores took their non-temporal policy, round robin was the
    // faster order from N = 16384 on.)
    A.xcd_ranges = 1;
    // one workgroup per compute unit (each holds 135-139 KB of LDS); with the
    // count unknown, one workgroup per tile
    const int cus = compute_units(stream);
    A.grid_max = cus > 0 ? cus : (int)(tm * tn);
    hipStream_t st = static_cast<hipStream_t>(stream);
    hipError_t e;
    if (elem == MX_ELEM_E4M3)
        e = out_dtype == MX_OUT_F32 ? mxg::launch<MX_ELEM_E4M3, MX_OUT_F32>(A, st)
                                         : mxg::launch<MX_ELEM_E4M3, MX_OUT_BF16>(A, st);
    else
        e = out_dtype == MX_OUT_F32 ? mxg::launch<MX_ELEM_E2M1, MX_OUT_F32>(A, st)
                                         : mxg::launch<MX_ELEM_E2M1, MX_OUT_BF16>(A, st);
    if (e != hipSuccess)
        return mxk::fail(MX_EHIP, "kernel launch failed: %s", hipGetErrorString(e));
    return MX_OK;
}

} // extern "C"
