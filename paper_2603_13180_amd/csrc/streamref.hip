// streamref.hip -- bandwidth reference with the MXNorm kernel's traffic and
// access pattern and no arithmetic (see include/streamref.h).
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "streamref.h"

namespace {

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint4 load_stream(const uint4 *p)
{
    const u32x4_t t = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(p));
    return make_uint4(t.x, t.y, t.z, t.w);
}

// One wave per row, rows of nc = d/8 16-byte chunks, nc in {64, 128, ..., 512}.
template <int MODE>
__global__ void __launch_bounds__(256) stream_kernel(const uint4 *x, int64_t T, int nc,
                                                     uint8_t *out, uint8_t *out_small)
{
    __shared__ __attribute__((aligned(16))) uint8_t sbuf[4 * 256];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int64_t row = (int64_t)blockIdx.x * 4 + wave;
    const bool row_ok = row < T;
    const int64_t rr = row_ok ? row : 0;
    const int cpl = nc / 64;
    // loads issued unconditionally from in-bounds addresses, zeros selected
    // afterwards (as the norm/cast kernel does): a load under a per-lane
    // condition waits for its own data and serialises the wave's loads
    uint4 v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        if (MODE == MX_STREAM_WRITE)
            v[j] = make_uint4((uint32_t)rr, (uint32_t)j, (uint32_t)lane, 1u);
        else
            v[j] = load_stream(x + rr * nc + (j < cpl ? j * 64 : 0) + lane);
    }
    if (MODE != MX_STREAM_WRITE) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const bool ok = row_ok && j < cpl;
            v[j].x = ok ? v[j].x : 0u;
            v[j].y = ok ? v[j].y : 0u;
            v[j].z = ok ? v[j].z : 0u;
            v[j].w = ok ? v[j].w : 0u;
        }
    }
    uint8_t *sb = sbuf + wave * 256;
    if (MODE == MX_STREAM_READ) {
        uint32_t acc = 0;
#pragma unroll
        for (int j = 0; j < 8; ++j)
            acc ^= v[j].x ^ v[j].y ^ v[j].z ^ v[j].w;
        for (int off = 1; off < 64; off <<= 1)
            acc ^= __shfl_xor(acc, off, 64);
        if (row_ok && lane == 0)
            *reinterpret_cast<uint4 *>(out_small + 16 * rr) = make_uint4(acc, 0u, 0u, 0u);
        return;
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        if (row_ok && j < cpl) {
            const int c = j * 64 + lane;
            if (MODE == MX_STREAM_NVFP4) {
                // 4 bytes of codes per 8 elements; one scale byte per 16
                const uint32_t o = ((v[j].x >> 8) ^ v[j].y) ^ ((v[j].z << 3) ^ v[j].w);
                __builtin_nontemporal_store(o, reinterpret_cast<uint32_t *>(
                                                   out + rr * nc * 4 + (int64_t)c * 4));
                if ((lane & 1) == 0)
                    sb[c >> 1] = (uint8_t)v[j].x;
            } else {
                const uint2 o = make_uint2((v[j].x >> 8) ^ v[j].y, (v[j].z >> 8) ^ v[j].w);
                __builtin_nontemporal_store(((unsigned long long)o.y << 32) | o.x,
                                            reinterpret_cast<unsigned long long *>(
                                                out + rr * nc * 8 + (int64_t)c * 8));
                if ((lane & 3) == 0)
                    sb[c >> 2] = (uint8_t)v[j].x;
            }
        }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const int K = MODE == MX_STREAM_NVFP4 ? nc / 2 : nc / 4;
    typedef unsigned int u32x4v __attribute__((ext_vector_type(4)));
    if (row_ok && lane < K / 16)
        __builtin_nontemporal_store(*reinterpret_cast<const u32x4v *>(sb + 16 * lane),
                                    reinterpret_cast<u32x4v *>(out_small + rr * K + 16 * lane));
}

// The straight-through estimator's traffic: per row, x and grad_z read and
// grad_x written, bf16 [T, d] each, one row per wave, 16-byte accesses, all
// loads of a row issued before its stores, which take the STE kernel's
// cache policy (sc0 sc1 nt).
__global__ void __launch_bounds__(256) ste_stream_kernel(const uint4 *x, const uint4 *gz, int64_t T,
                                                         int nc, uint4 *out)
{
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= T)
        return;
    const int cpl = nc / 64;
    uint4 a[8], b[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int64_t c = row * nc + (j < cpl ? j * 64 : 0) + lane;
        a[j] = load_stream(x + c);
        b[j] = load_stream(gz + c);
    }
    const __amdgpu_buffer_rsrc_t orr = __builtin_amdgcn_make_buffer_rsrc(
        out + row * nc, 0, nc * 16, 0x00020000);
#pragma unroll
    for (int j = 0; j < 8; ++j)
        if (j < cpl)
            __builtin_amdgcn_raw_buffer_store_b128(
                (u32x4_t){a[j].x ^ b[j].x, a[j].y ^ b[j].y, a[j].z ^ b[j].z, a[j].w ^ b[j].w}, orr,
                (j * 64 + lane) * 16, 0, 0x13);
}

// The column cast's traffic and access pattern (mx_cast_t_fwd): one 128-row
// x 256-column tile of x per workgroup of 512 threads, staged in LDS (32
// bytes of padding per 32-row block), 128 rho values per tile; lane 4 cc + b
// of wave w takes tile column 128 h + 16 w + cc over rows 32 b .. 32 b + 31
// and writes 32 bytes (the high bytes of its 32 values) as two 16-byte
// stores into that column's row of out [C, R]; a column's four block bytes
// (the first high byte of each block, xor the block's rho bits) go out as one
// dword of out_small [C, R/32].
constexpr int kTR = 128, kTC = 256, kTT = 512;
constexpr int kTPitch = 2 * kTC, kTBlk = 32 * kTPitch + 32;

__global__ void __launch_bounds__(kTT) transpose_stream_kernel(const uint16_t *x, const float *rho,
                                                               int64_t R, int64_t C,
                                                               uint8_t *out, uint8_t *out_small)
{
    __shared__ __attribute__((aligned(16))) uint8_t tile[4 * kTBlk];
    __shared__ float rs[kTR];
    const int tid = threadIdx.x;
    const int64_t c0 = (int64_t)blockIdx.x * kTC, r0 = (int64_t)blockIdx.y * kTR;
    constexpr int CPR = kTC / 8, RPP = kTT / CPR, NLD = kTR / RPP;
    const int ch = tid % CPR, rb = tid / CPR;
    uint4 v[NLD];
#pragma unroll
    for (int k = 0; k < NLD; ++k)
        v[k] = load_stream(reinterpret_cast<const uint4 *>(x + (r0 + rb + RPP * k) * C + c0) + ch);
    const float rv = tid < kTR ? rho[r0 + tid] : 0.f;
#pragma unroll
    for (int k = 0; k < NLD; ++k) {
        const int r = rb + RPP * k;
        *reinterpret_cast<uint4 *>(&tile[(r >> 5) * kTBlk + (r & 31) * kTPitch + 16 * ch]) = v[k];
    }
    if (tid < kTR)
        rs[tid] = rv;
    __syncthreads();
    const int w = tid >> 6, lane = tid & 63, b = lane & 3;
#pragma unroll
    for (int h = 0; h < kTC / 128; ++h) {
        const int cc = 128 * h + 16 * w + (lane >> 2);
        const uint8_t *col = tile + b * kTBlk + 2 * cc + 1;
        uint32_t q[8];
#pragma unroll
        for (int k = 0; k < 8; ++k)
            q[k] = (uint32_t)col[(4 * k) * kTPitch] | ((uint32_t)col[(4 * k + 1) * kTPitch] << 8) |
                   ((uint32_t)col[(4 * k + 2) * kTPitch] << 16) |
                   ((uint32_t)col[(4 * k + 3) * kTPitch] << 24);
        uint4 *dst = reinterpret_cast<uint4 *>(out + (c0 + cc) * R + r0 + 32 * b);
        dst[0] = make_uint4(q[0], q[1], q[2], q[3]);
        dst[1] = make_uint4(q[4], q[5], q[6], q[7]);
        const uint32_t byte = (q[0] ^ __float_as_uint(rs[32 * b])) & 0xFFu;
        const uint32_t b1 = (uint32_t)__builtin_amdgcn_mov_dpp((int)byte, 0x55, 0xF, 0xF, false);
        const uint32_t b2 = (uint32_t)__builtin_amdgcn_mov_dpp((int)byte, 0xAA, 0xF, 0xF, false);
        const uint32_t b3 = (uint32_t)__builtin_amdgcn_mov_dpp((int)byte, 0xFF, 0xF, 0xF, false);
        if (b == 0)
            *reinterpret_cast<uint32_t *>(out_small + (c0 + cc) * (R / 32) + r0 / 32) =
                byte | (b1 << 8) | (b2 << 16) | (b3 << 24);
    }
}

} // namespace

extern "C" int mx_stream_reference_transpose(const void *x, const float *rho, int64_t R, int64_t C,
                                             uint8_t *out, uint8_t *out_small, hipStream_t stream)
{
    if (R <= 0 || C <= 0 || R % kTR != 0 || C % kTC != 0 || R / kTR > 65535 || C / kTC > 65535)
        return R == 0 && C > 0 && C % kTC == 0 ? 0 : 1;
    if (!x || !rho || !out || !out_small || (uintptr_t)x % 16 || (uintptr_t)rho % 4 ||
        (uintptr_t)out % 16 || (uintptr_t)out_small % 4)
        return 1;
    hipLaunchKernelGGL(transpose_stream_kernel, dim3((unsigned)(C / kTC), (unsigned)(R / kTR)),
                       dim3(kTT), 0, (hipStream_t)stream, static_cast<const uint16_t *>(x), rho, R,
                       C, out, out_small);
    return hipGetLastError() == hipSuccess ? 0 : 3;
}

extern "C" int mx_stream_reference_ste(const void *x, const void *grad_z, int64_t T, int64_t d,
                                       void *out, hipStream_t stream)
{
    if (T < 0 || d <= 0 || d % 512 != 0 || d > 4096 || T > ((int64_t)1 << 34))
        return 1;
    if (T == 0)
        return 0;
    if (!x || !grad_z || !out || (uintptr_t)x % 16 || (uintptr_t)grad_z % 16 ||
        (uintptr_t)out % 16)
        return 1;
    hipLaunchKernelGGL(ste_stream_kernel, dim3((unsigned)((T + 3) / 4)), dim3(256), 0,
                       (hipStream_t)stream, static_cast<const uint4 *>(x),
                       static_cast<const uint4 *>(grad_z), T, (int)(d / 8), static_cast<uint4 *>(out));
    return hipGetLastError() == hipSuccess ? 0 : 3;
}

extern "C" int mx_stream_reference(const void *x, int64_t T, int64_t d, uint8_t *out,
                                   uint8_t *out_small, int mode, hipStream_t stream)
{
    if (T < 0 || d <= 0 || d % 512 != 0 || d > 4096 || T > ((int64_t)1 << 34))
        return 1;
    if (mode != MX_STREAM_MIXED && mode != MX_STREAM_READ && mode != MX_STREAM_WRITE &&
        mode != MX_STREAM_NVFP4)
        return 1;
    if (T == 0)
        return 0;
    if ((mode != MX_STREAM_WRITE && (!x || (uintptr_t)x % 16)) || !out_small ||
        (uintptr_t)out_small % 16 || (mode != MX_STREAM_READ && (!out || (uintptr_t)out % 16)))
        return 1;
    const dim3 grid((unsigned)((T + 3) / 4)), block(256);
    hipStream_t st = (hipStream_t)stream;
    const uint4 *xp = static_cast<const uint4 *>(x);
    const int nc = (int)(d / 8);
    if (mode == MX_STREAM_MIXED)
        hipLaunchKernelGGL(stream_kernel<MX_STREAM_MIXED>, grid, block, 0, st, xp, T, nc, out, out_small);
    else if (mode == MX_STREAM_READ)
        hipLaunchKernelGGL(stream_kernel<MX_STREAM_READ>, grid, block, 0, st, xp, T, nc, out, out_small);
    else if (mode == MX_STREAM_WRITE)
        hipLaunchKernelGGL(stream_kernel<MX_STREAM_WRITE>, grid, block, 0, st, xp, T, nc, out, out_small);
    else
        hipLaunchKernelGGL(stream_kernel<MX_STREAM_NVFP4>, grid, block, 0, st, xp, T, nc, out, out_small);
    return hipGetLastError() == hipSuccess ? 0 : 3;
}
