// backward.hip -- the MXNormLinear backward pieces for gfx950, behind the C
// ABI declared in include/mxnorm.h:
//
//  * mx_cast_t_fwd: the column-wise MX cast.  The weight gradient multiplies
//    MXCast(grad_H^T) by MXCast(rho~ . X), both blocked along the token
//    dimension (Sec. 3.7), while the forward quantises along rows; this cast
//    reads a row-major [R, C] matrix, optionally scales row r by rho[r]
//    ("in higher precision", float), and writes the MX encoding of its
//    transpose, blocks of 32 consecutive rows of one column.
//  * mxnorm_ste_bwd: the straight-through estimator (Sec. 3.7; the
//    RMSNorm-gradient appendix with S = 1/rho~): per row, with
//    dXb = grad_Z * gamma and u = sum_j dXb_j x_j,
//      grad_x_j = rho dXb_j - (1/d) rho^3 u x_j,
//    and grad_gamma_j = sum over rows of (rho x_j) grad_Z_j.
//
// Both are streaming kernels bound by HBM bandwidth.  Unlike the norm/cast
// kernel they use ordinary stores: non-temporal ones measured slower here
// (the column cast's 32-byte pieces of many rows rely on being merged in L2:
// 3.3x slower with the hint; the STE 6% slower).
#include <hip/hip_runtime.h>

#include <mutex>

#include <stdint.h>

#include <algorithm>

#include "mxnorm.h"
#include "norm_cast.h"
#include "status.h"

#pragma clang fp contract(off)

namespace mxb {

using namespace mxk;

// ---------------------------------------------------------- column cast --

constexpr int CT_ROWS = 128;  // tile rows (four 32-row blocks)

// Tile shape: 128 rows x COLS columns, staged by NTH threads.
template <int COLS, int NTH> struct CtShape {
    static constexpr int CPR = COLS / 8;          // 16-byte chunks per tile row
    static constexpr int RPP = NTH / CPR;         // tile rows per staging pass
    static constexpr int NLD = CT_ROWS / RPP;     // staging loads per thread
    static constexpr int PITCH = COLS * 2;        // bytes per staged row
    static constexpr int BLKB = 32 * PITCH + 32;  // bytes per staged 32-row block
    static __device__ __forceinline__ int off(int r) { return (r >> 5) * BLKB + (r & 31) * PITCH; }
};

struct CastTArgs {
    const uint16_t *x;
    const float *rho;
    uint8_t *codes;
    uint8_t *scales;
    int64_t R, C;
    int64_t tile_r0; // row tile of blockIdx.y == 0 (launches of at most 65535 row tiles)
    int mode;
    int order;       // tile visiting order, see cast_t_kernel
};

// Lane (cc, blk) of a cast pass: column cc of the staged tile over rows
// 32 blk .. 32 blk + 31 (one scale block, rows rb .. of x): reads its 32
// values down the column, scales them by rho, decides the E8M0 byte from
// their absmax and writes 32 codes (E4M3: 32 B; E2M1: 16 B) into row orow
// of the transposed output.  The four lanes of a column write 128 (E4M3)
// or 64 (E2M1) contiguous bytes, so a store instruction covers whole cache
// lines of 16 output rows.  With the padding, the 64 lanes of a read fall in
// distinct LDS banks (the blocks sit 8 banks apart).  Returns the scale
// byte.
template <bool FP4, int COLS>
__device__ __forceinline__ uint32_t cast_block(const CastTArgs &A, const uint8_t *tile,
                                               const float *rs, int cc, int blk, int64_t orow,
                                               int64_t rb)
{
    using S = CtShape<COLS, 256>; // PITCH and BLKB do not depend on the thread count
    constexpr int CT_PITCH = S::PITCH, CT_BLKB = S::BLKB;
    // the block's 32 scaled values, read once from LDS and kept in
    // registers; their absmax as the integer max of the magnitude
    // bits (NaN propagates)
    const uint8_t *col = tile + blk * CT_BLKB + 2 * cc;
    const float *rr = rs + 32 * blk;
    auto bits = [&](int i) {
        return (uint32_t)*reinterpret_cast<const uint16_t *>(col + i * CT_PITCH);
    };
    float tv[32];
    uint32_t m = 0;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        // four rho values per 16-byte read (the block's lanes share
        // it); without rho the staged values are 1 and t = RN(x * 1)
        // = x, so the reads need no branch
        const float4 r4 = reinterpret_cast<const float4 *>(rr)[k];
        const float rk[4] = {r4.x, r4.y, r4.z, r4.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float v = __uint_as_float(bits(4 * k + e) << 16);
            tv[4 * k + e] = v * rk[e];
            m = max(m, __float_as_uint(tv[4 * k + e]) & 0x7FFFFFFFu);
        }
    }
    auto value = [&](int i) { return tv[i]; };
    const float a = __uint_as_float(m);
    uint32_t byte;
    if constexpr (!FP4) {
        byte = e8m0_byte<false>(a, A.mode);
        if (A.mode == MX_SCALE_FLOOR) {
            // |t| <= 448 * 2^e: saturate before the conversion
            // (RCEIL never exceeds it)
            const float lim = __uint_as_float(((byte + 8u) << 23) | 0x600000u);
#pragma unroll
            for (int i = 0; i < 32; ++i)
                tv[i] = __builtin_amdgcn_fmed3f(tv[i], -lim, lim);
        }
        const float scale = __uint_as_float(byte << 23);
        uint32_t q[8];
#pragma unroll
        for (int k = 0; k < 8; ++k)
            q[k] = e4m3x4_hw(value(4 * k), value(4 * k + 1), value(4 * k + 2), value(4 * k + 3), scale);
        if (__builtin_amdgcn_ballot_w64(byte == 0xFFu)) { // rare: non-finite input
            if (byte == 0xFFu) { // input signs, all-ones magnitude
#pragma unroll
                for (int k = 0; k < 8; ++k) {
                    uint32_t r = 0x7F7F7F7Fu;
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        r |= (bits(4 * k + e) >> 15) << (8 * e + 7);
                    q[k] = r;
                }
            }
        }
        uint4 *dst = reinterpret_cast<uint4 *>(A.codes + orow * A.R + rb);
        dst[0] = make_uint4(q[0], q[1], q[2], q[3]);
        dst[1] = make_uint4(q[4], q[5], q[6], q[7]);
    } else {
        // the scaled fp4 conversion divides by the scale's power of
        // two, rounds to nearest even and saturates at 6
        byte = e8m0_byte<true>(a, A.mode);
        const float scale = __uint_as_float(byte << 23);
        uint32_t q[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            uint32_t p = 0;
            p = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p, value(8 * k), value(8 * k + 1), scale, 0);
            p = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p, value(8 * k + 2), value(8 * k + 3), scale, 1);
            p = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p, value(8 * k + 4), value(8 * k + 5), scale, 2);
            p = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p, value(8 * k + 6), value(8 * k + 7), scale, 3);
            q[k] = p;
        }
        if (__builtin_amdgcn_ballot_w64(byte == 0xFFu)) { // rare: non-finite input
            if (byte == 0xFFu) {
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    uint32_t p = 0x77777777u;
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        p |= (bits(8 * k + e) >> 15) << (4 * e + 3);
                    q[k] = p;
                }
            }
        }
        *reinterpret_cast<uint4 *>(A.codes + orow * (A.R / 2) + rb / 2) =
            make_uint4(q[0], q[1], q[2], q[3]);
    }
    return byte;
}

// Staging of one 128 x COLS tile of x (and its rho values) into registers:
// thread t moves 16-byte chunk t % CPR of tile rows t / CPR + RPP k, through
// a buffer resource over the tile's rows (chunks past C and rows past R read
// zeros; no per-lane branch, which would serialise the loads).  The tile's
// rho values travel with its rows (thread t < 128: row t), so that waiting
// for them is not a wait for every store in flight.
template <int COLS, int NTH> struct TileLoad {
    uint4 v[CtShape<COLS, NTH>::NLD];
    float rv;
};

template <int COLS, int NTH>
__device__ __forceinline__ void fetch_tile(const CastTArgs &A, int64_t r0, int64_t c0, int tid,
                                           TileLoad<COLS, NTH> &L)
{
    using S = CtShape<COLS, NTH>;
    const int ch = tid % S::CPR, rbase = tid / S::CPR;
    const uint32_t chunk_off = c0 + 8 * ch < A.C ? 16u * (uint32_t)ch : kOutside; // C % 8 == 0
    const uint32_t pitch = (uint32_t)A.C * 2u;
    const uint32_t rows = (uint32_t)max((int64_t)0, min((int64_t)CT_ROWS, A.R - r0));
    const __amdgpu_buffer_rsrc_t xr = buffer_rsrc(A.x + r0 * A.C + c0, rows * pitch);
#pragma unroll
    for (int k = 0; k < S::NLD; ++k) {
        const uint32_t r = (uint32_t)(rbase + S::RPP * k);
        const uint32_t off = chunk_off == kOutside ? kOutside : r * pitch + chunk_off;
        const u32x4_t t = __builtin_amdgcn_raw_buffer_load_b128(xr, (int)off, 0, kBufNT);
        L.v[k] = make_uint4(t.x, t.y, t.z, t.w);
    }
    if (A.rho) {
        const __amdgpu_buffer_rsrc_t rr = buffer_rsrc(A.rho + r0, rows * 4u);
        L.rv = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                             rr, (int)(tid < CT_ROWS ? 4u * (uint32_t)tid : kOutside), 0, 0));
    } else {
        L.rv = 1.0f;
    }
}

// The staged tile in LDS: as it is in x (2 COLS bytes per row), 32 bytes of
// padding after every 32 rows; rho of row t in rs[t].
template <int COLS, int NTH>
__device__ __forceinline__ void stage_tile(const TileLoad<COLS, NTH> &L, int tid, uint8_t *tile, float *rs)
{
    using S = CtShape<COLS, NTH>;
    const int ch = tid % S::CPR, rbase = tid / S::CPR;
#pragma unroll
    for (int k = 0; k < S::NLD; ++k)
        *reinterpret_cast<uint4 *>(&tile[S::off(rbase + S::RPP * k) + 16 * ch]) = L.v[k];
    if (tid < CT_ROWS)
        rs[tid] = L.rv;
}

// Workgroup (tile_c, y) casts the 128 x COLS tile of x at columns COLS
// tile_c and rows 128 (tile_r0 + y) (COLS = 256: 512-byte pieces of each x
// row, 128-byte output pieces).  A tile is staged in LDS, then cast in passes of
// 16 NW columns (NW waves): in pass h, lane 4 cc + b of wave w takes column
// 16 NW h + 16 w + cc over rows 32 b .. 32 b + 31 (cast_block).  A column's
// four scale bytes (blocks 0..3 of the tile) reach the quad's first lane
// through DPP and go out as one dword when the tile is whole and R a
// multiple of 128, else byte by byte.  One tile per workgroup with 512
// threads was the fastest of the shapes measured on MI355X: at [32768, 4096]
// 79 us against 83 (128-column tiles, 256 threads) and 89 (spans of four
// 128-column tiles per workgroup, the next tile prefetched in registers, the
// span's scale bytes gathered in LDS); at [32768, 28672] 626 against 632 us
// (spans of 256-column tiles).
template <bool FP4, int COLS, int NTH>
__global__ void __launch_bounds__(NTH) cast_t_kernel(CastTArgs A)
{
    using S = CtShape<COLS, NTH>;
    constexpr int NW = NTH / 64;
    static_assert(COLS % (16 * NW) == 0, "whole passes");
    __shared__ __attribute__((aligned(16))) uint8_t tile[4 * S::BLKB];
    __shared__ __attribute__((aligned(16))) float rs[CT_ROWS];
    const int tid = threadIdx.x;
    // Tile of this workgroup.  order 0: dispatch order, the column tiles of
    // one row band after another.  order 1 (wide matrices): workgroups are
    // dispatched round robin over the 8 XCDs; renumbered so that each XCD
    // runs a contiguous range of a sequence that takes groups of 64 row
    // tiles, column tile by column tile.  The 32 workgroups an XCD runs at
    // once then write 4 KB runs of 256 output rows, where the dispatch order
    // wrote 128-byte pieces of thousands (MI355X, [32768, 28672]: 623 ->
    // 544 us; [16384, 28672] 308 -> 272; [32768, 14336] 286 -> 278; at 8192
    // columns and fewer the dispatch order is faster).
    int64_t ct = blockIdx.x, rt = blockIdx.y;
    if (A.order) {
        constexpr int64_t GR = 64, NX = 8;
        const int64_t nc = gridDim.x, nr = gridDim.y, nt = nc * nr;
        const int64_t v = ct + rt * nc;
        const int64_t xcd = v % NX, loc = v / NX, q = nt / NX, rem = nt % NX;
        const int64_t p = xcd < rem ? xcd * (q + 1) + loc : rem * (q + 1) + (xcd - rem) * q + loc;
        const int64_t g = p / (GR * nc), in = p - g * GR * nc;
        const int64_t gsz = min(GR, nr - g * GR);
        rt = g * GR + in % gsz;
        ct = in / gsz;
    }
    const int64_t c0 = ct * COLS;
    const int w = tid >> 6, lane = tid & 63;
    const int blk = lane & 3; // 32-row block this lane casts
    const int64_t r0 = (A.tile_r0 + rt) * CT_ROWS;
    {
        TileLoad<COLS, NTH> L;
        fetch_tile<COLS, NTH>(A, r0, c0, tid, L);
        stage_tile<COLS, NTH>(L, tid, tile, rs);
    }
    lds_barrier();
    const int64_t rb = r0 + 32 * blk; // first row of this lane's block
    const bool whole = r0 + CT_ROWS <= A.R && (A.R & 127) == 0;
#pragma unroll
    for (int h = 0; h < COLS / (16 * NW); ++h) {
        const int cc = 16 * NW * h + 16 * w + (lane >> 2); // column in the tile
        const int64_t orow = c0 + cc;
        uint32_t byte = 0;
        if (rb < A.R && orow < A.C)
            byte = cast_block<FP4, COLS>(A, tile, rs, cc, blk, orow, rb);
        // every lane of the quad takes part: quad_perm broadcasts of lanes 1, 2, 3
        const uint32_t b1 = (uint32_t)__builtin_amdgcn_mov_dpp((int)byte, 0x55, 0xF, 0xF, false);
        const uint32_t b2 = (uint32_t)__builtin_amdgcn_mov_dpp((int)byte, 0xAA, 0xF, 0xF, false);
        const uint32_t b3 = (uint32_t)__builtin_amdgcn_mov_dpp((int)byte, 0xFF, 0xF, 0xF, false);
        if (blk == 0 && orow < A.C) {
            uint8_t *sdst = A.scales + orow * (A.R / 32) + r0 / 32;
            if (whole) {
                *reinterpret_cast<uint32_t *>(sdst) = byte | (b1 << 8) | (b2 << 16) | (b3 << 24);
            } else {
                const uint32_t bs[4] = {byte, b1, b2, b3};
#pragma unroll
                for (int k = 0; k < 4; ++k)
                    if (r0 + 32 * k < A.R)
                        sdst[k] = (uint8_t)bs[k];
            }
        }
    }
}

// ------------------------------------------------------------ STE rows --

// grad_x is written once and read by a later kernel: its stores take the
// sc0 sc1 nt cache policy (system scope, non-temporal).  At [32768, 4096]
// on MI355X the call ran 144.5 -> 135.5 us with it (137.0 with nt alone).
constexpr int kGradXPolicy = 0x13;

// rows per workgroup (each writes one partial row of grad_gamma): 4 .. 64,
// as many as keep about 512 workgroups, two per compute unit (at [32768,
// 4096] on MI355X, with the current row pipeline: 134-136 us for the call
// against 145 with 768 workgroups; before it, 1024 workgroups were 2% and
// 384 11% slower)
inline int ste_rpw(int64_t T)
{
    return (int)std::max<int64_t>(4, std::min<int64_t>(64, (T + 511) / 512));
}

struct SteArgs {
    const uint16_t *x, *gz, *gamma;
    const float *rho;
    void *gx;
    float *part; // [workgroups, d] grad_gamma partials, or NULL
    int64_t T;
    int rpw;     // rows per workgroup
    int d, nc; // columns, 8-column chunks
};

__device__ __forceinline__ uint16_t f32_to_bf16(float f)
{
    const uint32_t u = __float_as_uint(f);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u)
        return (uint16_t)((u >> 16) | 0x40u); // quiet NaN, sign kept
    return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

// The workgroup of NT threads is one team: thread l holds 8-column chunks
// j NT + l, j < CPL, of each row, and the workgroup's rows are done one
// after the other, each row's x and grad_Z loads issued while the rows before
// it are processed.  Per row: dXb = RN(gz gamma) (exact: a product of two
// bf16 values fits in float), u = sum dXb x accumulated in double (exact
// products), reduced in the wave by DPP and over the team through LDS; c =
// RN(rho^3 u / d) computed in double; grad_x = RN(RN(rho dXb) - RN(c x)).
// Each thread keeps sum over its rows of RN(rho x) gz for its columns (float)
// and stores it as this workgroup's partial row of grad_gamma.  Loads and
// grad_x stores go through buffer resources, so chunks past the row's end
// and rows past T read zeros and store nowhere
// without a per-lane branch (which would serialise the loads).  Loads and
// stores use one resource per row.
template <int NT, int CPL, int OUT, bool GAM, bool GG>
__global__ void __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(NT * CPL <= 512 ? 2 : 1)))
ste_bwd_kernel(SteArgs A)
{
    constexpr int NW = NT / 64;
    constexpr uint32_t OB = OUT == MX_OUT_F32 ? 4u : 2u; // grad_x bytes per element
    __shared__ double red[2][NW];
    const int tid = threadIdx.x;
    const int cpl = (A.nc + NT - 1) / NT; // chunks this row really has (uniform)

    // workgroup b takes rows b, b + G, b + 2G, ... (G workgroups, all
    // resident at once): the rows in flight across the chip at any moment
    // form one contiguous band of the tensors rather than G separate streams
    const int64_t G = gridDim.x;
    const int rows = (int)((A.T - (int64_t)blockIdx.x + G - 1) / G);
    const uint32_t rowb = (uint32_t)A.d * 2u; // bytes of a bf16 row
    auto row_of = [&](int k) { return (int64_t)blockIdx.x + (int64_t)k * G; };
    // byte offset of chunk j inside a bf16 row, or past every resource
    uint32_t coff[CPL];
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
        const int ch = j * NT + tid;
        coff[j] = ch < A.nc ? 16u * (uint32_t)ch : kOutside;
    }

    uint4 g[GAM ? CPL : 1];
    if constexpr (GAM) {
        const __amdgpu_buffer_rsrc_t gr = buffer_rsrc(A.gamma, rowb);
#pragma unroll
        for (int j = 0; j < CPL; ++j) {
            const u32x4_t t = __builtin_amdgcn_raw_buffer_load_b128(gr, (int)coff[j], 0, 0);
            g[j] = make_uint4(t.x, t.y, t.z, t.w);
        }
    }
    float gg[GG ? CPL : 1][8];
    if constexpr (GG) {
#pragma unroll
        for (int j = 0; j < CPL; ++j)
#pragma unroll
            for (int e = 0; e < 8; ++e)
                gg[j][e] = 0.0f;
    }

    // row k's x and grad_Z chunks and its rho (k >= rows: an empty resource,
    // which reads zeros and moves no data).  rho travels with the row: a load
    // issued later than the rows in flight would make its wait one for all
    // of them (the vector memory counter completes in order)
    auto load = [&](int k, uint4 (&xv)[CPL], uint4 (&zv)[CPL], float &rv) {
        const int64_t row = k < rows ? row_of(k) : 0;
        rv = k < rows ? A.rho[row] : 0.0f;
        const uint32_t n = k < rows ? rowb : 0u;
        const __amdgpu_buffer_rsrc_t xr = buffer_rsrc(A.x + row * A.d, n);
        const __amdgpu_buffer_rsrc_t zr = buffer_rsrc(A.gz + row * A.d, n);
#pragma unroll
        for (int j = 0; j < CPL; ++j) {
            const u32x4_t a = __builtin_amdgcn_raw_buffer_load_b128(xr, (int)coff[j], 0, kBufNT);
            const u32x4_t b = __builtin_amdgcn_raw_buffer_load_b128(zr, (int)coff[j], 0, kBufNT);
            xv[j] = make_uint4(a.x, a.y, a.z, a.w);
            zv[j] = make_uint4(b.x, b.y, b.z, b.w);
        }
    };

    // row k's partial sums of u: this wave's sum into LDS slot k & 1
    auto reduce = [&](int k, const uint4 (&xv)[CPL], const uint4 (&zv)[CPL]) {
        // u = sum dXb x over the row
        double s = 0.0;
#pragma unroll
        for (int j = 0; j < CPL; ++j) {
            if (j >= cpl)
                break;
            const uint32_t xw[4] = {xv[j].x, xv[j].y, xv[j].z, xv[j].w};
            const uint32_t zw[4] = {zv[j].x, zv[j].y, zv[j].z, zv[j].w};
            uint32_t gw[4] = {0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u}; // 1.0
            if constexpr (GAM) {
                gw[0] = g[j].x;
                gw[1] = g[j].y;
                gw[2] = g[j].z;
                gw[3] = g[j].w;
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float d0 = bf16_lo(zw[i]) * bf16_lo(gw[i]);
                const float d1 = bf16_hi(zw[i]) * bf16_hi(gw[i]);
                s = __builtin_fma((double)d0, (double)bf16_lo(xw[i]), s);
                s = __builtin_fma((double)d1, (double)bf16_hi(xw[i]), s);
            }
        }
        s = team_sum<64>(s, nullptr, tid); // the wave's sum, in every lane
        double *red_k = red[k & 1];        // two slots: one barrier per row suffices
        if ((tid & 63) == 0)
            red_k[tid >> 6] = s;
    };
    // u of row k, once the barrier after its reduce has passed
    auto finish = [&](int k) {
        const double *red_k = red[k & 1];
        double u = 0.0;
#pragma unroll
        for (int i = 0; i < NW; ++i)
            u += red_k[i];
        return u;
    };
    // grad_x of row k and its grad_gamma terms, given u
    auto output = [&](int k, const uint4 (&xv)[CPL], const uint4 (&zv)[CPL], const float rho,
                      const double u) {
        const int64_t row = row_of(k);
        const __amdgpu_buffer_rsrc_t outr =
            buffer_rsrc(static_cast<uint8_t *>(A.gx) + row * A.d * OB, (uint32_t)A.d * OB);
        const double rd = (double)rho;
        const float cf = (float)(rd * rd * rd * u / (double)A.d);

#pragma unroll
        for (int j = 0; j < CPL; ++j) {
            if (j >= cpl)
                break;
            const uint32_t xw[4] = {xv[j].x, xv[j].y, xv[j].z, xv[j].w};
            const uint32_t zw[4] = {zv[j].x, zv[j].y, zv[j].z, zv[j].w};
            uint32_t gw[4] = {0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u};
            if constexpr (GAM) {
                gw[0] = g[j].x;
                gw[1] = g[j].y;
                gw[2] = g[j].z;
                gw[3] = g[j].w;
            }
            float o[8];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float x0 = bf16_lo(xw[i]), x1 = bf16_hi(xw[i]);
                const float z0 = bf16_lo(zw[i]), z1 = bf16_hi(zw[i]);
                const float d0 = z0 * bf16_lo(gw[i]), d1 = z1 * bf16_hi(gw[i]);
                o[2 * i] = rho * d0 - cf * x0;
                o[2 * i + 1] = rho * d1 - cf * x1;
                if constexpr (GG) {
                    gg[j][2 * i] += (rho * x0) * z0;
                    gg[j][2 * i + 1] += (rho * x1) * z1;
                }
            }
            // grad_x of chunk j: OB * 8 bytes at OB/2 times the bf16 offset
            const uint32_t off = coff[j] == kOutside ? kOutside : coff[j] * (OB / 2u);
            if constexpr (OUT == MX_OUT_F32) {
                __builtin_amdgcn_raw_buffer_store_b128(
                    (u32x4_t){__float_as_uint(o[0]), __float_as_uint(o[1]), __float_as_uint(o[2]),
                              __float_as_uint(o[3])},
                    outr, (int)off, 0, kGradXPolicy);
                __builtin_amdgcn_raw_buffer_store_b128(
                    (u32x4_t){__float_as_uint(o[4]), __float_as_uint(o[5]), __float_as_uint(o[6]),
                              __float_as_uint(o[7])},
                    outr, (int)(off == kOutside ? kOutside : off + 16u), 0, kGradXPolicy);
            } else {
                uint32_t p[4];
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    p[i] = f32_to_bf16(o[2 * i]) | ((uint32_t)f32_to_bf16(o[2 * i + 1]) << 16);
                __builtin_amdgcn_raw_buffer_store_b128((u32x4_t){p[0], p[1], p[2], p[3]}, outr, (int)off,
                                                       0, kGradXPolicy);
            }
        }
    };

    // Up to 512 chunks per thread set (d <= 4096): three register sets and
    // a pipeline.  While row k is written, row k+1's sums go to LDS and row
    // k+2's loads are in flight; the barrier that completes row k+1's u then
    // comes after row k's output work instead of stalling every wave between
    // a row's sums and its output (5.7% faster at [32768, 4096]).  Wider
    // rows: two register sets (row k+1's loads in flight while row k is
    // summed and written), and one for the 1024-thread teams, which have
    // 128 registers per lane.  Every wave of the workgroup takes the same
    // barriers: rows is uniform.
    if constexpr (NT * CPL <= 512) {
        uint4 xa[CPL], za[CPL], xb[CPL], zb[CPL], xc[CPL], zc[CPL];
        float ra, rb, rc;
        load(0, xa, za, ra);
        load(1, xb, zb, rb);
        reduce(0, xa, za);
        lds_barrier();
        double u = finish(0);
        for (int k = 0; k < rows; k += 3) {
            load(k + 2, xc, zc, rc);
            reduce(k + 1, xb, zb);
            output(k, xa, za, ra, u);
            lds_barrier();
            u = finish(k + 1);
            if (k + 1 >= rows)
                break;
            load(k + 3, xa, za, ra);
            reduce(k + 2, xc, zc);
            output(k + 1, xb, zb, rb, u);
            lds_barrier();
            u = finish(k + 2);
            if (k + 2 >= rows)
                break;
            load(k + 4, xb, zb, rb);
            reduce(k + 3, xa, za);
            output(k + 2, xc, zc, rc, u);
            lds_barrier();
            u = finish(k + 3);
        }
    } else if constexpr (NT * CPL <= 2048) {
        uint4 xa[CPL], za[CPL], xb[CPL], zb[CPL];
        float ra, rb;
        load(0, xa, za, ra);
        for (int k = 0; k < rows; k += 2) {
            load(k + 1, xb, zb, rb);
            reduce(k, xa, za);
            lds_barrier();
            output(k, xa, za, ra, finish(k));
            if (k + 1 >= rows)
                break;
            load(k + 2, xa, za, ra);
            reduce(k + 1, xb, zb);
            lds_barrier();
            output(k + 1, xb, zb, rb, finish(k + 1));
        }
    } else {
        uint4 xa[CPL], za[CPL];
        float ra;
        for (int k = 0; k < rows; ++k) {
            load(k, xa, za, ra);
            reduce(k, xa, za);
            lds_barrier();
            output(k, xa, za, ra, finish(k));
        }
    }

    if constexpr (GG) {
        float *dst = A.part + (int64_t)blockIdx.x * A.d;
#pragma unroll
        for (int j = 0; j < CPL; ++j) {
            const int ch = j * NT + tid;
            if (j < cpl && ch < A.nc) {
                float4 *p = reinterpret_cast<float4 *>(dst) + 2 * ch;
                p[0] = make_float4(gg[j][0], gg[j][1], gg[j][2], gg[j][3]);
                p[1] = make_float4(gg[j][4], gg[j][5], gg[j][6], gg[j][7]);
            }
        }
    }
}

// grad_gamma[j] = RN(sum of the P partial rows, in double, in a fixed
// order), in one launch.  Block b (1024 threads) sums columns [64 b, +64):
// thread (g, q), g = 0 .. 63, q = 0 .. 15, adds rows g, g + 64, g + 128, ...
// of columns 64 b + 4 q .. +3 in order, 16 bytes per row, so every thread has
// several loads in flight; the 64 row groups' sums are then added in order
// of g.  Deterministic for a given P.  (Two launches, slices of rows then a
// sum of the slices, took about 10 us at [32768, 4096]; 256 threads with
// 4-byte loads per column were latency-bound.)
constexpr int GG_GROUPS = 64;
__global__ void __launch_bounds__(1024) ggamma_reduce_kernel(const float *part, int64_t P, int d,
                                                             float *out)
{
    __shared__ double red[GG_GROUPS][64];
    const int q = threadIdx.x & 15, g = threadIdx.x >> 4;
    const int j0 = blockIdx.x * 64 + 4 * q; // d % 8 == 0: j0 < d means j0 + 3 < d
    double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
    if (j0 < d) {
#pragma unroll 4
        for (int64_t p = g; p < P; p += GG_GROUPS) {
            const float4 v = *reinterpret_cast<const float4 *>(part + p * d + j0);
            s0 += (double)v.x;
            s1 += (double)v.y;
            s2 += (double)v.z;
            s3 += (double)v.w;
        }
    }
    red[g][4 * q] = s0;
    red[g][4 * q + 1] = s1;
    red[g][4 * q + 2] = s2;
    red[g][4 * q + 3] = s3;
    lds_barrier();
    const int c = threadIdx.x;
    if (c < 64 && blockIdx.x * 64 + c < d) {
        double t = 0.0;
        for (int i = 0; i < GG_GROUPS; ++i)
            t += red[i][c];
        out[blockIdx.x * 64 + c] = (float)t;
    }
}

template <int NT, int CPL, int OUT, bool GAM>
hipError_t launch_ste(const SteArgs &A, hipStream_t st)
{
    const unsigned blocks = (unsigned)((A.T + A.rpw - 1) / A.rpw);
    if (A.part)
        hipLaunchKernelGGL((ste_bwd_kernel<NT, CPL, OUT, GAM, true>), dim3(blocks), dim3(NT), 0,
                           st, A);
    else
        hipLaunchKernelGGL((ste_bwd_kernel<NT, CPL, OUT, GAM, false>), dim3(blocks), dim3(NT), 0,
                           st, A);
    return hipGetLastError();
}

template <int OUT, bool GAM>
hipError_t launch_ste_out(const SteArgs &A, hipStream_t st)
{
    // smallest chunk count per thread that covers the row: 256 threads up to
    // 8192 columns, then 1024 threads up to 32768
    if (A.nc <= 256)
        return launch_ste<256, 1, OUT, GAM>(A, st);
    if (A.nc <= 512)
        return launch_ste<256, 2, OUT, GAM>(A, st);
    if (A.nc <= 1024)
        return launch_ste<256, 4, OUT, GAM>(A, st);
    if (A.nc <= 2048)
        return launch_ste<1024, 2, OUT, GAM>(A, st);
    return launch_ste<1024, 4, OUT, GAM>(A, st);
}

} // namespace mxb

// host side -------------------------------------------------------------------

namespace {

bool aligned(const void *p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

int64_t ste_workgroups(int64_t T) { return (T + mxb::ste_rpw(T) - 1) / mxb::ste_rpw(T); }

// Device-resident workspace of mxnorm_ste_bwd_noalloc: the grad_gamma partial
// rows live here instead of in caller memory.  Each GPU the
// library runs on holds its own copy for the life of the process.  In host
// code `scratch` only names the symbol; its device address (one per GPU) is
// looked up once per device with hipGetSymbolAddress and kept in
// scratch_ptr.
constexpr size_t kScratchBytes = size_t(32) << 20;
constexpr int kMaxDevices = 64;
__device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex scratch_mu;
void *scratch_ptr[kMaxDevices];

// The scratch address on the device that `stream` belongs to (the current
// device for the null stream), or an error.
mx_status scratch_for(hipStream_t stream, void **out)
{
    int dev = -1;
    hipError_t e;
    if (stream) {
        hipDevice_t hd;
        e = hipStreamGetDevice(static_cast<hipStream_t>(stream), &hd);
        dev = (int)hd;
    } else {
        e = hipGetDevice(&dev);
    }
    if (e != hipSuccess)
        return mxk::fail(MX_EHIP, "cannot find the stream's device: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxDevices)
        return mxk::fail(MX_EUNSUPPORTED, "device %d is beyond the %d the library tracks", dev,
                         kMaxDevices);
    std::lock_guard<std::mutex> lock(scratch_mu);
    if (!scratch_ptr[dev]) {
        int cur = -1;
        if ((e = hipGetDevice(&cur)) != hipSuccess)
            return mxk::fail(MX_EHIP, "hipGetDevice failed: %s", hipGetErrorString(e));
        if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess)
            return mxk::fail(MX_EHIP, "hipSetDevice(%d) failed: %s", dev, hipGetErrorString(e));
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (cur != dev)
            (void)hipSetDevice(cur);
        if (e != hipSuccess || !p)
            return mxk::fail(MX_EHIP, "hipGetSymbolAddress(scratch) failed on device %d: %s", dev,
                             hipGetErrorString(e));
        scratch_ptr[dev] = p;
    }
    *out = scratch_ptr[dev];
    return MX_OK;
}

} // namespace

extern "C" {

mx_status mx_cast_t_fwd(const void *x, const float *rho, int64_t R, int64_t C, int block,
                        int elem, int scale_mode, uint8_t *codes, uint8_t *scales, hipStream_t stream)
{
    mxk::clear_error();
    if (R < 0 || C <= 0)
        return mxk::fail(MX_EINVAL, "R must be >= 0 and C > 0");
    if (elem != MX_ELEM_E4M3 && elem != MX_ELEM_E2M1)
        return mxk::fail(MX_EINVAL, "elem must be MX_ELEM_E4M3 or MX_ELEM_E2M1");
    if (scale_mode != MX_SCALE_RCEIL && scale_mode != MX_SCALE_FLOOR)
        return mxk::fail(MX_EINVAL, "unknown scale_mode %d", scale_mode);
    if (block != 32)
        return mxk::fail(MX_EUNSUPPORTED, "the column cast supports block = 32");
    if (R % 32 != 0)
        return mxk::fail(MX_EINVAL, "R must be a multiple of the block (32)");
    if (C % 8 != 0)
        return mxk::fail(MX_EINVAL, "C must be a multiple of 8");
    if (R > ((int64_t)1 << 31) || C > ((int64_t)1 << 23))
        return mxk::fail(MX_EUNSUPPORTED, "matrix too large (R <= 2^31, C <= 2^23)");
    if (R == 0)
        return MX_OK;
    if (!x || !codes || !scales)
        return mxk::fail(MX_EINVAL, "x, codes and scales must be non-NULL");
    if (!aligned(x, 16) || !aligned(codes, 16) || (rho && !aligned(rho, 4)))
        return mxk::fail(MX_EINVAL, "x and codes must be 16-byte, rho 4-byte aligned");
    mxb::CastTArgs A;
    A.x = static_cast<const uint16_t *>(x);
    A.rho = rho;
    A.codes = codes;
    A.scales = scales;
    A.R = R;
    A.C = C;
    A.mode = scale_mode;
    // one 128 x 256 tile per workgroup (see the kernel), at most 65535 row
    // tiles per launch
    constexpr int kCols = 256, kThreads = 512;
    constexpr int64_t kMaxRowTiles = 65535;
    const int64_t col_tiles = (C + kCols - 1) / kCols;
    const int64_t row_tiles = (R + mxb::CT_ROWS - 1) / mxb::CT_ROWS;
    A.order = col_tiles >= 48 ? 1 : 0; // from 12288 columns on (see the kernel)
    hipStream_t st = static_cast<hipStream_t>(stream);
    for (int64_t t0 = 0; t0 < row_tiles; t0 += kMaxRowTiles) {
        A.tile_r0 = t0;
        const dim3 grid((unsigned)col_tiles, (unsigned)std::min<int64_t>(row_tiles - t0, kMaxRowTiles));
        if (elem == MX_ELEM_E4M3)
            hipLaunchKernelGGL((mxb::cast_t_kernel<false, kCols, kThreads>), grid, dim3(kThreads), 0, st, A);
        else
            hipLaunchKernelGGL((mxb::cast_t_kernel<true, kCols, kThreads>), grid, dim3(kThreads), 0, st, A);
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return mxk::fail(MX_EHIP, "kernel launch failed: %s", hipGetErrorString(e));
    return MX_OK;
}

size_t mxnorm_ste_bwd_workspace_bytes(int64_t T, int64_t d)
{
    if (T <= 0 || d <= 0)
        return 0;
    // one float partial row of grad_gamma per workgroup
    return (size_t)ste_workgroups(T) * (size_t)d * sizeof(float);
}

mx_status mxnorm_ste_bwd(const void *x, const void *grad_z, const void *gamma, const float *rho,
                         int64_t T, int64_t d, int out_dtype, void *grad_x, float *grad_gamma,
                         void *workspace, size_t workspace_bytes, hipStream_t stream)
{
    mxk::clear_error();
    if (T < 0)
        return mxk::fail(MX_EINVAL, "T must be >= 0");
    if (d <= 0 || d % 8 != 0)
        return mxk::fail(MX_EINVAL, "d must be a positive multiple of 8");
    if (d > MXNORM_MAX_D)
        return mxk::fail(MX_EUNSUPPORTED, "d = %lld exceeds %d", (long long)d, MXNORM_MAX_D);
    if (out_dtype != MX_OUT_F32 && out_dtype != MX_OUT_BF16)
        return mxk::fail(MX_EINVAL, "out_dtype must be MX_OUT_F32 or MX_OUT_BF16");
    if (T == 0)
        return MX_OK;
    if (!x || !grad_z || !rho || !grad_x)
        return mxk::fail(MX_EINVAL, "x, grad_z, rho and grad_x must be non-NULL");
    if (!aligned(x, 16) || !aligned(grad_z, 16) || (gamma && !aligned(gamma, 16)) ||
        !aligned(grad_x, 16) || !aligned(rho, 4))
        return mxk::fail(MX_EINVAL, "x, grad_z, gamma and grad_x must be 16-byte, rho 4-byte "
                                    "aligned");
    if (grad_gamma) {
        if (!aligned(grad_gamma, 4))
            return mxk::fail(MX_EINVAL, "grad_gamma must be 4-byte aligned");
        if (!workspace || !aligned(workspace, 16) ||
            workspace_bytes < mxnorm_ste_bwd_workspace_bytes(T, d))
            return mxk::fail(MX_EINVAL, "grad_gamma needs a 16-byte aligned workspace of "
                                        "mxnorm_ste_bwd_workspace_bytes(T, d) = %zu bytes",
                             mxnorm_ste_bwd_workspace_bytes(T, d));
    }
    if (ste_workgroups(T) > INT32_MAX)
        return mxk::fail(MX_EUNSUPPORTED, "T too large");
    mxb::SteArgs A;
    A.x = static_cast<const uint16_t *>(x);
    A.gz = static_cast<const uint16_t *>(grad_z);
    A.gamma = static_cast<const uint16_t *>(gamma);
    A.rho = rho;
    A.gx = grad_x;
    A.part = grad_gamma ? static_cast<float *>(workspace) : nullptr;
    A.T = T;
    A.rpw = mxb::ste_rpw(T);
    A.d = (int)d;
    A.nc = (int)(d / 8);
    hipStream_t st = static_cast<hipStream_t>(stream);
    hipError_t e;
    if (out_dtype == MX_OUT_F32)
        e = gamma ? mxb::launch_ste_out<MX_OUT_F32, true>(A, st)
                  : mxb::launch_ste_out<MX_OUT_F32, false>(A, st);
    else
        e = gamma ? mxb::launch_ste_out<MX_OUT_BF16, true>(A, st)
                  : mxb::launch_ste_out<MX_OUT_BF16, false>(A, st);
    if (e == hipSuccess && grad_gamma) {
        hipLaunchKernelGGL(mxb::ggamma_reduce_kernel, dim3((unsigned)((d + 63) / 64)), dim3(1024), 0,
                           st, static_cast<const float *>(workspace), ste_workgroups(T), (int)d,
                           grad_gamma);
        e = hipGetLastError();
    }
    if (e != hipSuccess)
        return mxk::fail(MX_EHIP, "kernel launch failed: %s", hipGetErrorString(e));
    return MX_OK;
}

size_t mxnorm_ste_bwd_noalloc_max_workspace(void) { return kScratchBytes; }

mx_status mxnorm_ste_bwd_noalloc(const void *x, const void *grad_z, const void *gamma,
                                 const float *rho, int64_t T, int64_t d, int out_dtype,
                                 void *grad_x, float *grad_gamma, hipStream_t stream)
{
    mxk::clear_error();
    if (grad_gamma && T > 0 && d > 0 && mxnorm_ste_bwd_workspace_bytes(T, d) > kScratchBytes)
        return mxk::fail(MX_EUNSUPPORTED,
                         "grad_gamma at T = %lld, d = %lld needs %zu bytes of workspace, more "
                         "than the %zu the allocation-free entry point holds",
                         (long long)T, (long long)d, mxnorm_ste_bwd_workspace_bytes(T, d),
                         kScratchBytes);
    void *ws = nullptr;
    if (grad_gamma && T > 0) {
        const mx_status st = scratch_for(stream, &ws);
        if (st != MX_OK)
            return st;
    }
    // every partial row is written before it is read, so the scratch needs
    // no clearing between calls
    return mxnorm_ste_bwd(x, grad_z, gamma, rho, T, d, out_dtype, grad_x, grad_gamma, ws,
                          ws ? kScratchBytes : 0, stream);
}

} // extern "C"
