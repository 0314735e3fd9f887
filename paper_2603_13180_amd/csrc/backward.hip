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

#include <stdint.h>

#include <algorithm>

#include "mxnorm.h"
#include "norm_cast.h"
#include "status.h"

#pragma clang fp contract(off)

namespace mxb {

using namespace mxk;

// ---------------------------------------------------------- column cast --

constexpr int CT_ROWS = 128; // tile rows (4 waves x one 32-row block)
constexpr int CT_COLS = 64;  // tile columns (one per lane)
constexpr int CT_TILES = 16; // most tiles per workgroup (a span of up to 2048 rows)

struct CastTArgs {
    const uint16_t *x;
    const float *rho;
    uint8_t *codes;
    uint8_t *scales;
    int64_t R, C;
    int mode;
    int tiles; // tiles per span, 1 .. CT_TILES
};

// Workgroup (span, tile_c) casts columns [64 tile_c, +64) over a span of
// `tiles` x 128 rows, 128 rows at a time (the host sizes the span so that
// the grid still fills the chip).  Each 128 x 64 tile is staged in
// LDS as it is in x (128 bytes per row; the next tile's loads are already in
// flight in registers); wave w then casts rows 32w .. 32w+31 of it, lane c
// column c: it reads its 32 values down the column (the 64 lanes of a read
// on 128 consecutive bytes: no bank conflicts), scales them by rho, decides
// the E8M0 byte from their absmax and writes 32 codes (E4M3: 32 B; E2M1:
// 16 B) into row c0 + c of the transposed output.  The span's 64 scale bytes
// per column are gathered in LDS and written at the end, 64 contiguous
// bytes per output row, rather than one scattered byte per tile.
template <bool FP4>
__global__ void __launch_bounds__(256) cast_t_kernel(CastTArgs A)
{
    __shared__ __attribute__((aligned(16))) uint16_t tile[CT_ROWS * CT_COLS];
    __shared__ float rs[CT_ROWS];
    __shared__ __attribute__((aligned(16))) uint8_t sb[CT_COLS][CT_TILES * 4];

    const int tid = threadIdx.x;
    const int64_t span0 = (int64_t)blockIdx.y * CT_ROWS * A.tiles;
    const int64_t c0 = (int64_t)blockIdx.x * CT_COLS;
    const int ntiles = (int)min((int64_t)A.tiles, (A.R - span0 + CT_ROWS - 1) / CT_ROWS);
    const int w = tid >> 6, c = tid & 63;
    const int64_t orow = c0 + c;
    const bool col_ok = orow < A.C;

    // staging: thread t moves 16-byte chunk t % 8 of tile rows t / 8 + 32 k
    const int ch = tid & 7;
    const bool chunk_ok = c0 + 8 * ch < A.C; // C % 8 == 0: whole chunks
    auto fetch = [&](int64_t r0, uint4 v[4]) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int r = (tid >> 3) + 32 * k;
            v[k] = (chunk_ok && r0 + r < A.R)
                       ? load_stream(reinterpret_cast<const uint4 *>(A.x + (r0 + r) * A.C + c0) + ch)
                       : make_uint4(0u, 0u, 0u, 0u);
        }
    };
    uint4 nxt[4];
    fetch(span0, nxt);

    for (int t = 0; t < ntiles; ++t) {
        const int64_t r0 = span0 + (int64_t)t * CT_ROWS;
#pragma unroll
        for (int k = 0; k < 4; ++k)
            *reinterpret_cast<uint4 *>(&tile[((tid >> 3) + 32 * k) * CT_COLS + 8 * ch]) = nxt[k];
        if (tid < CT_ROWS)
            rs[tid] = (A.rho && r0 + tid < A.R) ? A.rho[r0 + tid] : 1.0f;
        __syncthreads();
        if (t + 1 < ntiles)
            fetch(r0 + CT_ROWS, nxt);

        const int64_t rb = r0 + 32 * w; // first row of this wave's block
        if (rb < A.R && col_ok) {
            // pass 1: the block absmax of the scaled values (integer max of
            // the magnitude bits: NaN propagates); pass 2 re-reads the column
            // from LDS and converts a few values at a time
            const uint16_t *col = tile + 32 * w * CT_COLS + c;
            const float *rr = rs + 32 * w;
            auto value = [&](int i) {
                const float v = __uint_as_float((uint32_t)col[i * CT_COLS] << 16);
                return A.rho ? v * rr[i] : v;
            };
            uint32_t m = 0;
#pragma unroll 8
            for (int i = 0; i < 32; ++i)
                m = max(m, __float_as_uint(value(i)) & 0x7FFFFFFFu);
            const float a = __uint_as_float(m);
            uint32_t byte;
            if constexpr (!FP4) {
                byte = e8m0_byte<false>(a, A.mode);
                // FLOOR: |t| <= 448 * 2^e, saturate before the conversion
                // (RCEIL never exceeds it)
                const float lim = A.mode == MX_SCALE_FLOOR
                                      ? __uint_as_float(((byte + 8u) << 23) | 0x600000u)
                                      : __builtin_inff();
                const float scale = __uint_as_float(byte << 23);
                uint32_t q[8];
#pragma unroll
                for (int k = 0; k < 8; ++k) {
                    float v[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        v[e] = __builtin_amdgcn_fmed3f(value(4 * k + e), -lim, lim);
                    q[k] = e4m3x4_hw(v[0], v[1], v[2], v[3], scale);
                    if (byte == 0xFFu) { // non-finite input: input signs, all-ones magnitude
                        uint32_t r = 0x7F7F7F7Fu;
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            r |= ((uint32_t)col[(4 * k + e) * CT_COLS] >> 15) << (8 * e + 7);
                        q[k] = r;
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
                    if (byte == 0xFFu) {
                        p = 0x77777777u;
#pragma unroll
                        for (int e = 0; e < 8; ++e)
                            p |= ((uint32_t)col[(8 * k + e) * CT_COLS] >> 15) << (4 * e + 3);
                    }
                    q[k] = p;
                }
                *reinterpret_cast<uint4 *>(A.codes + orow * (A.R / 2) + rb / 2) =
                    make_uint4(q[0], q[1], q[2], q[3]);
            }
            sb[c][4 * t + w] = (uint8_t)byte;
        }
        __syncthreads(); // the tile is overwritten next
    }

    // the span's scale bytes: column c has 4 per tile (fewer where R ends
    // inside the span), written by the 4 threads of its row as 16-byte pieces
    // when whole and aligned, else byte by byte
    const int64_t nblk = min((int64_t)ntiles * 4, (A.R - span0) / 32);
    const int cc = tid >> 2, part = tid & 3;
    const int64_t srow = c0 + cc;
    if (srow < A.C) {
        uint8_t *dst = A.scales + srow * (A.R / 32) + span0 / 32;
        const int lo = 16 * part;
        if (lo + 16 <= nblk && (((uintptr_t)(dst + lo)) & 15) == 0) {
            *reinterpret_cast<uint4 *>(dst + lo) = *reinterpret_cast<const uint4 *>(&sb[cc][lo]);
        } else {
            for (int k = lo; k < lo + 16 && k < nblk; ++k)
                dst[k] = sb[cc][k];
        }
    }
}

// ------------------------------------------------------------ STE rows --

// rows per workgroup (each writes one partial row of grad_gamma): 4 .. 32,
// as many as keep about 512 workgroups
inline int ste_rpw(int64_t T)
{
    return (int)std::max<int64_t>(4, std::min<int64_t>(32, (T + 511) / 512));
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
// j NT + l, j < CPL, of each row, and rows [rpw b, rpw b + rpw) are done one
// after the other.  Per row: dXb = RN(gz gamma) (exact: a product of two
// bf16 values fits in float), u = sum dXb x accumulated in double (exact
// products) and reduced over the team through LDS; c = RN(rho^3 u / d)
// computed in double; grad_x = RN(RN(rho dXb) - RN(c x)).  Each thread keeps
// sum over its rows of RN(rho x) gz for its columns (float) and stores it as
// this workgroup's partial row of grad_gamma.
template <int NT, int CPL, int OUT, bool GAM, bool GG>
__global__ void __launch_bounds__(NT) ste_bwd_kernel(SteArgs A)
{
    constexpr int NW = NT / 64;
    __shared__ double red[2][NW];
    const int tid = threadIdx.x;
    const int cpl = (A.nc + NT - 1) / NT; // chunks this row really has (uniform)

    uint4 g[GAM ? CPL : 1];
    if constexpr (GAM) {
#pragma unroll
        for (int j = 0; j < CPL; ++j) {
            const int ch = j * NT + tid;
            g[j] = (j < cpl && ch < A.nc) ? reinterpret_cast<const uint4 *>(A.gamma)[ch]
                                          : make_uint4(0u, 0u, 0u, 0u);
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

    const int64_t row0 = (int64_t)blockIdx.x * A.rpw;
    const int64_t rows = min((int64_t)A.rpw, A.T - row0);
    for (int64_t k = 0; k < rows; ++k) {
        const int64_t row = row0 + k;
        const uint4 *xr = reinterpret_cast<const uint4 *>(A.x + row * A.d);
        const uint4 *zr = reinterpret_cast<const uint4 *>(A.gz + row * A.d);
        uint4 xv[CPL], zv[CPL];
#pragma unroll
        for (int j = 0; j < CPL; ++j) {
            const int ch = j * NT + tid;
            const bool ok = j < cpl && ch < A.nc;
            xv[j] = ok ? load_stream(xr + ch) : make_uint4(0u, 0u, 0u, 0u);
            zv[j] = ok ? load_stream(zr + ch) : make_uint4(0u, 0u, 0u, 0u);
        }
        const float rho = A.rho[row];

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
#pragma unroll
        for (int off = 1; off < 64; off <<= 1)
            s += __shfl_xor(s, off, 64);
        double *rb = red[k & 1]; // two buffers: one barrier per row suffices
        if ((tid & 63) == 0)
            rb[tid >> 6] = s;
        __syncthreads();
        double u = 0.0;
#pragma unroll
        for (int i = 0; i < NW; ++i)
            u += rb[i];
        const double rd = (double)rho;
        const float cf = (float)(rd * rd * rd * u / (double)A.d);

#pragma unroll
        for (int j = 0; j < CPL; ++j) {
            if (j >= cpl)
                break;
            const int ch = j * NT + tid;
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
            if (ch < A.nc) {
                if constexpr (OUT == MX_OUT_F32) {
                    float4 *dst = reinterpret_cast<float4 *>(static_cast<float *>(A.gx) + row * A.d) +
                                  2 * ch;
                    dst[0] = make_float4(o[0], o[1], o[2], o[3]);
                    dst[1] = make_float4(o[4], o[5], o[6], o[7]);
                } else {
                    uint32_t p[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        p[i] = f32_to_bf16(o[2 * i]) | ((uint32_t)f32_to_bf16(o[2 * i + 1]) << 16);
                    reinterpret_cast<uint4 *>(static_cast<uint16_t *>(A.gx) + row * A.d)[ch] =
                        make_uint4(p[0], p[1], p[2], p[3]);
                }
            }
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

// grad_gamma[j] = sum of the P partial rows, in double, in a fixed order:
// block b sums columns [64 b, 64 b + 64); thread (g, c) adds rows g, g + 16,
// g + 32, ... of column c in order, then the 16 partial sums are added in
// order of g.  Deterministic, and 16 x 64 loads in flight per block.
constexpr int RG = 16;
__global__ void __launch_bounds__(1024) ggamma_reduce_kernel(const float *part, int64_t P, int d,
                                                             float *out)
{
    __shared__ double red[RG][64];
    const int c = threadIdx.x & 63, g = threadIdx.x >> 6;
    const int j = blockIdx.x * 64 + c;
    double s = 0.0;
    if (j < d)
#pragma unroll 4
        for (int64_t p = g; p < P; p += RG)
            s += (double)part[p * d + j];
    red[g][c] = s;
    __syncthreads();
    if (g == 0 && j < d) {
        double t = 0.0;
#pragma unroll
        for (int i = 0; i < RG; ++i)
            t += red[i][c];
        out[j] = (float)t;
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

} // namespace

extern "C" {

mx_status mx_cast_t_fwd(const void *x, const float *rho, int64_t R, int64_t C, int block,
                        int elem, int scale_mode, uint8_t *codes, uint8_t *scales, void *stream)
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
    if (R > ((int64_t)1 << 31) || C > ((int64_t)1 << 31))
        return mxk::fail(MX_EUNSUPPORTED, "matrix too large");
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
    // tiles per workgroup: as many as keep about 1024 workgroups (longer
    // spans write longer runs of scale bytes), at most CT_TILES
    const int64_t col_tiles = (C + mxb::CT_COLS - 1) / mxb::CT_COLS;
    const int64_t row_tiles = (R + mxb::CT_ROWS - 1) / mxb::CT_ROWS;
    A.tiles = (int)std::max<int64_t>(1, std::min<int64_t>(mxb::CT_TILES,
                                                          col_tiles * row_tiles / 1024));
    const int64_t span = (int64_t)mxb::CT_ROWS * A.tiles;
    const dim3 grid((unsigned)col_tiles, (unsigned)((R + span - 1) / span));
    if (grid.y > 65535u)
        return mxk::fail(MX_EUNSUPPORTED, "R too large for one launch");
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (elem == MX_ELEM_E4M3)
        hipLaunchKernelGGL(mxb::cast_t_kernel<false>, grid, dim3(256), 0, st, A);
    else
        hipLaunchKernelGGL(mxb::cast_t_kernel<true>, grid, dim3(256), 0, st, A);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return mxk::fail(MX_EHIP, "kernel launch failed: %s", hipGetErrorString(e));
    return MX_OK;
}

size_t mxnorm_ste_bwd_workspace_bytes(int64_t T, int64_t d)
{
    if (T <= 0 || d <= 0)
        return 0;
    return (size_t)ste_workgroups(T) * (size_t)d * sizeof(float);
}

mx_status mxnorm_ste_bwd(const void *x, const void *grad_z, const void *gamma, const float *rho,
                         int64_t T, int64_t d, int out_dtype, void *grad_x, float *grad_gamma,
                         void *workspace, size_t workspace_bytes, void *stream)
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
        hipLaunchKernelGGL(mxb::ggamma_reduce_kernel, dim3((unsigned)((d + 63) / 64)),
                           dim3(1024), 0, st, static_cast<const float *>(workspace),
                           ste_workgroups(T), (int)d, grad_gamma);
        e = hipGetLastError();
    }
    if (e != hipSuccess)
        return mxk::fail(MX_EHIP, "kernel launch failed: %s", hipGetErrorString(e));
    return MX_OK;
}

} // extern "C"
