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
// loads of a row issued before its stores.
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
#pragma unroll
    for (int j = 0; j < 8; ++j)
        if (j < cpl)
            out[row * nc + j * 64 + lane] =
                make_uint4(a[j].x ^ b[j].x, a[j].y ^ b[j].y, a[j].z ^ b[j].z, a[j].w ^ b[j].w);
}

} // namespace

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
