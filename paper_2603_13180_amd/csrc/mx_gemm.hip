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
// Tiling: a workgroup of 4 waves computes a 256 (M) x 256 (N) tile; each wave
// a 128 x 128 quarter as 8 x 8 matrix-core tiles of 16 x 16, accumulated in
// the AGPRs.  The K loop moves 128 bytes of every row per step (128 E4M3 or
// 256 E2M1 elements) from global memory straight into LDS (16-byte
// global_load_lds, no staging registers), double-buffered, and reads the next
// step's fragments into registers while the current step's matrix-core work
// runs (see the pipeline note in the kernel).  In LDS, 16-byte chunk c of row r lives at chunk
// c ^ (r & 7) of the row, so the fragment reads of 8 consecutive rows hit
// distinct banks.  Workgroups are renumbered so that each XCD (each with its
// own L2) runs a contiguous range of tiles, visited in groups of tile rows
// that share operand blocks.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mxnorm.h"
#include "status.h"

namespace mxg {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
#define LDS_AS __attribute__((address_space(3)))

constexpr int BM = 256;    // tile rows of A (M)
constexpr int BN = 256;    // tile rows of B (N)
constexpr int KB = 128;    // bytes of each row per K step
constexpr int NT = 256;    // threads: 4 waves
constexpr int WTM = 128;   // wave tile along M
constexpr int WTN = 128;   // wave tile along N
constexpr int FM = WTM / 16, FN = WTN / 16;
constexpr int GROUP_M = 4; // tile rows per group in the visiting order
constexpr int NXCD = 8;

// scale bytes per row and K step: 4 blocks of 32 (E4M3), 8 blocks (E2M1)
template <int ELEM> struct Op {
    static constexpr int SB = ELEM == MX_ELEM_E2M1 ? 8 : 4;
    static constexpr int FMT = ELEM == MX_ELEM_E2M1 ? 4 : 0; // matrix-core operand format
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

// Wait until at most N of this wave's vector memory loads are outstanding
// (they complete in issue order).
template <int N> __device__ __forceinline__ void wait_vmcnt()
{
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Per-lane part of the DMA addresses, fixed for the whole K loop: byte
// offsets, relative to the tile's first row, of the rows this lane moves.
// Rows past M or N read row M-1 or N-1: their results are never stored.
template <int ELEM> struct Rows {
    uint32_t a[8], b[8];     // code rows 64w + 8t + l/8, times the row pitch, plus the chunk
    uint32_t sa[Op<ELEM>::SB / 4], sb[Op<ELEM>::SB / 4]; // scale rows, plus the dword
};

template <int ELEM>
__device__ __forceinline__ Rows<ELEM> lane_rows(const Args &A, int64_t m0, int64_t n0, int w,
                                                int l)
{
    constexpr int DW = Op<ELEM>::SB / 4;
    Rows<ELEM> R;
    const int rr = l >> 3;        // row within the 8-row group
    const int ch = (l & 7) ^ rr;  // source chunk for this LDS slot (the swizzle)
#pragma unroll
    for (int t = 0; t < 8; ++t) {
        const int r = 64 * w + 8 * t + rr;
        R.a[t] = (uint32_t)((min(m0 + r, A.M - 1) - m0) * A.rb) + 16 * ch;
        R.b[t] = (uint32_t)((min(n0 + r, A.N - 1) - n0) * A.rb) + 16 * ch;
    }
#pragma unroll
    for (int u = 0; u < DW; ++u) {
        const int r = 64 * w + u * (64 / DW) + l / DW;
        R.sa[u] = (uint32_t)((min(m0 + r, A.M - 1) - m0) * A.rs) + 4 * (l % DW);
        R.sb[u] = (uint32_t)((min(n0 + r, A.N - 1) - n0) * A.rs) + 4 * (l % DW);
    }
    return R;
}

// Issue the loads of K step s into one LDS stage.  Wave w moves rows
// 64w .. 64w+63 of both operand tiles (8 instructions of 8 rows x 128 bytes
// each; lane l fills LDS slot l of its group, which holds source chunk
// (l % 8) ^ (l / 8)) and their scale bytes, stored row-major [row][SB]
// (lane i of scale instruction u moves dword i % (SB/4) of row
// 64w + u (64 / (SB/4)) + i / (SB/4)).
template <int ELEM>
__device__ __forceinline__ void issue_step(const uint8_t *ta, const uint8_t *tb,
                                           const uint8_t *tsa, const uint8_t *tsb,
                                           const Rows<ELEM> &R, int s, uint32_t stage, int w)
{
    constexpr int SB = Op<ELEM>::SB;
    constexpr int DW = SB / 4;
    const uint32_t xa = stage;
    const uint32_t xb = stage + BM * KB;
    const uint32_t sa = stage + (BM + BN) * KB;
    const uint32_t sb = sa + BM * SB;
    const uint32_t kc = (uint32_t)s * KB, ks = (uint32_t)s * SB;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
        lds_load16(ta, R.a[t] + kc, xa + (64 * w + 8 * t) * KB);
        lds_load16(tb, R.b[t] + kc, xb + (64 * w + 8 * t) * KB);
    }
#pragma unroll
    for (int u = 0; u < DW; ++u) {
        lds_load4(tsa, R.sa[u] + ks, sa + (64 * w + u * (64 / DW)) * SB);
        lds_load4(tsb, R.sb[u] + ks, sb + (64 * w + u * (64 / DW)) * SB);
    }
}

// Workgroup barrier without the memory fence of __syncthreads(): the fence
// would wait for every outstanding load, including the prefetch of the next
// step.  LDS written by the DMA loads is covered by the explicit vmcnt waits
// each wave makes before arriving; the lgkmcnt(0) completes this wave's own
// LDS reads, so that a stage read before the barrier can be refilled after
// it.  The "memory" clobber keeps the compiler from moving LDS accesses
// across it.
__device__ __forceinline__ void barrier()
{
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// loads per lane in issue_step
template <int ELEM> constexpr int loads_per_step() { return 16 + 2 * (Op<ELEM>::SB / 4); }

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ u32x4 lds_chunk(const LDS_AS uint8_t *base, int row, int c)
{
    return *reinterpret_cast<const LDS_AS u32x4 *>(base + row * KB + 16 * (c ^ (row & 7)));
}

__device__ __forceinline__ v8i join(u32x4 lo, u32x4 hi)
{
    return __builtin_bit_cast(v8i, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f)
{
    const uint32_t u = __float_as_uint(f);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u)
        return (uint16_t)((u >> 16) | 0x40u); // quiet NaN, sign kept
    return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
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

template <int ELEM>
__device__ __forceinline__ Frag read_frag(const LDS_AS uint8_t *codes,
                                          const LDS_AS uint8_t *scales, int r, int g)
{
    Frag f;
    f.v = join(lds_chunk(codes, r, g), lds_chunk(codes, r, 4 + g));
    if constexpr (ELEM == MX_ELEM_E2M1) {
        typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
        const u32x2 d = *reinterpret_cast<const LDS_AS u32x2 *>(scales + r * 8);
        f.s0 = (int)((d.x >> (8 * g)) & 0xFFu);
        f.s1 = (int)((d.y >> (8 * g)) & 0xFFu);
    } else {
        const uint32_t d = *reinterpret_cast<const LDS_AS uint32_t *>(scales + r * 4);
        f.s0 = (int)((d >> (8 * g)) & 0xFFu);
        f.s1 = 0;
    }
    return f;
}

// acc += B-fragment x A-fragment over one K step (B is the instruction's
// first operand: each lane's four results are then four consecutive columns
// of one row of H)
template <int ELEM>
__device__ __forceinline__ void mma(v4f &acc, const Frag &b, const Frag &a)
{
    if constexpr (ELEM == MX_ELEM_E2M1) {
        const v8i z = {0, 0, 0, 0, 0, 0, 0, 0};
        const v8i b0 = __builtin_shufflevector(b.v, z, 0, 1, 2, 3, 8, 8, 8, 8);
        const v8i a0 = __builtin_shufflevector(a.v, z, 0, 1, 2, 3, 8, 8, 8, 8);
        const v8i b1 = __builtin_shufflevector(b.v, z, 4, 5, 6, 7, 8, 8, 8, 8);
        const v8i a1 = __builtin_shufflevector(a.v, z, 4, 5, 6, 7, 8, 8, 8, 8);
        acc = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(b0, a0, acc, 4, 4, 0, b.s0, 0, a.s0);
        acc = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(b1, a1, acc, 4, 4, 0, b.s1, 0, a.s1);
    } else {
        acc = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(b.v, a.v, acc, 0, 0, 0, b.s0, 0, a.s0);
    }
}

template <int ELEM, int OUT>
__global__ void __launch_bounds__(NT) mx_gemm_kernel(Args A)
{
    constexpr int SB = Op<ELEM>::SB;
    constexpr int STAGE = Op<ELEM>::STAGE;
    __shared__ __attribute__((aligned(16))) uint8_t lds[2 * STAGE];

    // tile of this workgroup: contiguous per XCD (dispatch is round-robin
    // over the XCDs), then grouped GROUP_M tile rows at a time
    const int G = A.tiles_m * A.tiles_n;
    const int wg = blockIdx.x;
    const int xcd = wg % NXCD, loc = wg / NXCD;
    const int q = G / NXCD, rem = G % NXCD;
    const int pid = xcd < rem ? xcd * (q + 1) + loc : rem * (q + 1) + (xcd - rem) * q + loc;
    const int in_group = GROUP_M * A.tiles_n;
    const int first_m = (pid / in_group) * GROUP_M;
    const int gsz = min(A.tiles_m - first_m, GROUP_M);
    const int tm = first_m + (pid % in_group) % gsz;
    const int tn = (pid % in_group) / gsz;
    const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;

    const int tid = threadIdx.x;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6); // wave-uniform
    const int l = tid & 63;
    const int g = l >> 4, qd = l & 15; // lane group (K block / output row quad), row in fragment
    const int wm = (w & 1) * WTM, wn = (w >> 1) * WTN;

    v4f acc[FN][FM];
#pragma unroll
    for (int i = 0; i < FN; ++i)
#pragma unroll
        for (int j = 0; j < FM; ++j)
            acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

    // Pipeline.  Registers hold every fragment of the current step.  Each
    // step is split at a barrier: the first half multiplies A fragments
    // 0..FM/2-1 with all B fragments; at the barrier the next step's data has
    // landed in the other stage and every wave has finished reading this
    // stage, so the DMA for two steps ahead can refill it; the second half
    // multiplies A fragments FM/2.. fragment by fragment of B, reloading each
    // B fragment (and the free A fragments) with the next step's data as soon
    // as it is used up.  A wave therefore never waits on LDS at a step start.
    constexpr int HJ = FM / 2;
    LDS_AS uint8_t *st0 = (LDS_AS uint8_t *)lds;
    const uint32_t st0_addr = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)st0);
    auto codes_a = [&](int stage) { return (const LDS_AS uint8_t *)(st0 + stage * STAGE); };
    auto codes_b = [&](int stage) { return (const LDS_AS uint8_t *)(st0 + stage * STAGE + BM * KB); };
    auto scales_a = [&](int stage) {
        return (const LDS_AS uint8_t *)(st0 + stage * STAGE + (BM + BN) * KB);
    };
    auto scales_b = [&](int stage) {
        return (const LDS_AS uint8_t *)(st0 + stage * STAGE + (BM + BN) * KB + BM * SB);
    };

    // tile bases (wave-uniform) and this lane's row offsets
    const uint8_t *ta = A.a + m0 * A.rb, *tb = A.b + n0 * A.rb;
    const uint8_t *tsa = A.as + m0 * A.rs, *tsb = A.bs + n0 * A.rs;
    const Rows<ELEM> R = lane_rows<ELEM>(A, m0, n0, w, l);

    issue_step<ELEM>(ta, tb, tsa, tsb, R, 0, st0_addr, w);
    if (A.steps > 1) {
        issue_step<ELEM>(ta, tb, tsa, tsb, R, 1, st0_addr + STAGE, w);
        wait_vmcnt<loads_per_step<ELEM>()>();
    } else {
        wait_vmcnt<0>();
    }
    barrier();

    Frag fb[FN], fa[FM];
#pragma unroll
    for (int i = 0; i < FN; ++i)
        fb[i] = read_frag<ELEM>(codes_b(0), scales_b(0), wn + 16 * i + qd, g);
#pragma unroll
    for (int j = 0; j < FM; ++j)
        fa[j] = read_frag<ELEM>(codes_a(0), scales_a(0), wm + 16 * j + qd, g);

    for (int s = 0; s < A.steps; ++s) {
        const int cur = s & 1, nxt = cur ^ 1;
        const bool more = s + 1 < A.steps;

        // every wave has read this step's fragments (during the previous
        // step): the stage can take the DMA for two steps ahead now
        barrier();
        if (s + 2 < A.steps)
            issue_step<ELEM>(ta, tb, tsa, tsb, R, s + 2, st0_addr + cur * STAGE, w);

#pragma unroll
        for (int j = 0; j < HJ; ++j)
#pragma unroll
            for (int i = 0; i < FN; ++i)
                mma<ELEM>(acc[i][j], fb[i], fa[j]);

        // the next step's data has landed (the step after it may still be
        // in flight)
        if (s + 2 < A.steps)
            wait_vmcnt<loads_per_step<ELEM>()>();
        else if (more)
            wait_vmcnt<0>();
        barrier();

        // (the reloads are unconditional: after the last step they read a
        // stale stage that nothing uses, which keeps the loop free of
        // branches that would hold old and new fragments live together)
#pragma unroll
        for (int j = 0; j < HJ; ++j)
            fa[j] = read_frag<ELEM>(codes_a(nxt), scales_a(nxt), wm + 16 * j + qd, g);
#pragma unroll
        for (int i = 0; i < FN; ++i) {
#pragma unroll
            for (int j = HJ; j < FM; ++j)
                mma<ELEM>(acc[i][j], fb[i], fa[j]);
            // keep the reload after the last use of fb[i] (its registers)
            __builtin_amdgcn_sched_barrier(0);
            fb[i] = read_frag<ELEM>(codes_b(nxt), scales_b(nxt), wn + 16 * i + qd, g);
        }
#pragma unroll
        for (int j = HJ; j < FM; ++j)
            fa[j] = read_frag<ELEM>(codes_a(nxt), scales_a(nxt), wm + 16 * j + qd, g);
    }

    // lane (g, qd) of tile (i, j) holds H[m][n .. n+3] with
    // m = m0 + wm + 16 j + qd and n = n0 + wn + 16 i + 4 g.  N is a multiple
    // of 16, so a tile column base below N has its 16 columns inside H.
    auto gained = [&](int i, int j) {
        v4f v = acc[i][j];
        if (A.bgain) {
            const int64_t n = n0 + wn + 16 * i + 4 * g;
            const uint2 gw = *reinterpret_cast<const uint2 *>(A.bgain + (n < A.N ? n : 0));
            v[0] = v[0] * __uint_as_float(gw.x << 16);
            v[1] = v[1] * __uint_as_float(gw.x & 0xFFFF0000u);
            v[2] = v[2] * __uint_as_float(gw.y << 16);
            v[3] = v[3] * __uint_as_float(gw.y & 0xFFFF0000u);
        }
        return v;
    };
    if constexpr (OUT == MX_OUT_F32) {
#pragma unroll
        for (int j = 0; j < FM; ++j) {
            const int64_t m = m0 + wm + 16 * j + qd;
#pragma unroll
            for (int i = 0; i < FN; ++i) {
                const int64_t n = n0 + wn + 16 * i + 4 * g;
                const v4f v = gained(i, j);
                if (m < A.M && n < A.N)
                    *reinterpret_cast<float4 *>(static_cast<float *>(A.out) + m * A.N + n) =
                        make_float4(v[0], v[1], v[2], v[3]);
            }
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
        typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
#pragma unroll
        for (int j = 0; j < FM; ++j) {
            const int64_t m = m0 + wm + 16 * j + qd;
#pragma unroll
            for (int i = 0; i < FN; i += 2) {
                uint32_t lo[2], hi[2];
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const v4f v = gained(i + h, j);
                    lo[h] = f32_to_bf16_rne(v[0]) | ((uint32_t)f32_to_bf16_rne(v[1]) << 16);
                    hi[h] = f32_to_bf16_rne(v[2]) | ((uint32_t)f32_to_bf16_rne(v[3]) << 16);
                }
                const auto sl = __builtin_amdgcn_permlane16_swap(lo[0], lo[1], false, false);
                const auto sh = __builtin_amdgcn_permlane16_swap(hi[0], hi[1], false, false);
                const int64_t n = n0 + wn + 16 * (i + (g & 1)) + 8 * (g >> 1);
                if (m < A.M && n < A.N)
                    *reinterpret_cast<u32x4v *>(static_cast<uint16_t *>(A.out) + m * A.N + n) =
                        u32x4v{sl[0], sh[0], sl[1], sh[1]};
            }
        }
    }
}

template <int ELEM, int OUT>
hipError_t launch(const Args &A, hipStream_t stream)
{
    const int G = A.tiles_m * A.tiles_n;
    hipLaunchKernelGGL((mx_gemm_kernel<ELEM, OUT>), dim3((unsigned)G), dim3(NT), 0, stream, A);
    return hipGetLastError();
}

} // namespace mxg

// host side -------------------------------------------------------------------

namespace {

bool aligned(const void *p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

} // namespace

extern "C" {

mx_status mx_matmul_fwd(const uint8_t *a_codes, const uint8_t *a_scales, const uint8_t *b_codes,
                        const uint8_t *b_scales, int64_t M, int64_t N, int64_t K, int block,
                        int elem, const void *b_gain, int out_dtype, void *out, void *stream)
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
    if (tm * tn > INT32_MAX / 2 || M > INT32_MAX || N > INT32_MAX)
        return mxk::fail(MX_EUNSUPPORTED, "problem too large");
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
