// Test aid, not part of the library: gfx950's scaled conversion
// instructions applied element by element, so that a GPU test can hold them
// to a round-to-nearest-even definition over every fp32 input of a range.
// The norm/cast kernels rely on these instructions for their E4M3 and E2M1
// codes (v_cvt_scalef32_pk_fp8_f32 and v_cvt_scalef32_pk_fp4_f32: the value
// divided by 2^(exponent field of the scale operand - 127), rounded to
// nearest even), and the MX matmul's bf16 output on the float -> bf16
// conversion (v_cvt_pk_bf16_f32, what a __bf16 cast compiles to).
//
//   int hwc_e4m3(const float *in, uint8_t *out, int64_t n, uint32_t scale_byte, void *stream)
//   int hwc_e2m1(const float *in, uint8_t *out, int64_t n, uint32_t scale_byte, void *stream)
//   int hwc_bf16(const float *in, uint16_t *out, int64_t n, void *stream)
//
// in, out: device arrays of n elements (n even); out[i] is the code of
// in[i] (E2M1: a nibble in the low half of the byte; bf16: the 16 bits).  scale_byte: the E8M0
// byte whose power of two divides the values (127 = 1).  Returns 0, or -1
// for a bad argument (nothing launched), or the HIP error code.
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef short short2_t __attribute__((ext_vector_type(2)));

__global__ void __launch_bounds__(256) hwc_e4m3_kernel(const float *in, uint8_t *out, int64_t n,
                                                       float scale)
{
    const int64_t stride = (int64_t)gridDim.x * 256 * 2;
    for (int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 2; i < n; i += stride) {
        const short2_t r =
            __builtin_amdgcn_cvt_scalef32_pk_fp8_f32((short2_t){0, 0}, in[i], in[i + 1], scale, false);
        const uint32_t w = __builtin_bit_cast(uint32_t, r);
        out[i] = (uint8_t)(w & 0xFFu);
        out[i + 1] = (uint8_t)((w >> 8) & 0xFFu);
    }
}

__global__ void __launch_bounds__(256) hwc_e2m1_kernel(const float *in, uint8_t *out, int64_t n,
                                                       float scale)
{
    const int64_t stride = (int64_t)gridDim.x * 256 * 2;
    for (int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 2; i < n; i += stride) {
        const uint32_t w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, in[i], in[i + 1], scale, 0);
        out[i] = (uint8_t)(w & 0xFu);
        out[i + 1] = (uint8_t)((w >> 4) & 0xFu);
    }
}

__global__ void __launch_bounds__(256) hwc_bf16_kernel(const float *in, uint16_t *out, int64_t n)
{
    const int64_t stride = (int64_t)gridDim.x * 256 * 2;
    for (int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 2; i < n; i += stride) {
        const __bf16 a = (__bf16)in[i], b = (__bf16)in[i + 1];
        out[i] = __builtin_bit_cast(uint16_t, a);
        out[i + 1] = __builtin_bit_cast(uint16_t, b);
    }
}

static int launch(bool fp4, const float *in, uint8_t *out, int64_t n, uint32_t scale_byte,
                  void *stream)
{
    if (n < 0 || (n & 1) || scale_byte > 254u || (n && (!in || !out)))
        return -1;
    if (n == 0)
        return 0;
    const float scale = __builtin_bit_cast(float, scale_byte << 23);
    const int64_t pairs = n / 2;
    const unsigned blocks = (unsigned)(pairs < 256 * 8192 ? (pairs + 255) / 256 : 8192);
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (fp4)
        hipLaunchKernelGGL(hwc_e2m1_kernel, dim3(blocks), dim3(256), 0, st, in, out, n, scale);
    else
        hipLaunchKernelGGL(hwc_e4m3_kernel, dim3(blocks), dim3(256), 0, st, in, out, n, scale);
    const hipError_t e = hipGetLastError();
    return e == hipSuccess ? 0 : (int)e;
}

extern "C" int hwc_e4m3(const float *in, uint8_t *out, int64_t n, uint32_t scale_byte, void *stream)
{
    return launch(false, in, out, n, scale_byte, stream);
}

extern "C" int hwc_e2m1(const float *in, uint8_t *out, int64_t n, uint32_t scale_byte, void *stream)
{
    return launch(true, in, out, n, scale_byte, stream);
}

extern "C" int hwc_bf16(const float *in, uint16_t *out, int64_t n, void *stream)
{
    if (n < 0 || (n & 1) || (n && (!in || !out)))
        return -1;
    if (n == 0)
        return 0;
    const int64_t pairs = n / 2;
    const unsigned blocks = (unsigned)(pairs < 256 * 8192 ? (pairs + 255) / 256 : 8192);
    hipLaunchKernelGGL(hwc_bf16_kernel, dim3(blocks), dim3(256), 0,
                       static_cast<hipStream_t>(stream), in, out, n);
    const hipError_t e = hipGetLastError();
    return e == hipSuccess ? 0 : (int)e;
}
