/*
 * streamref.h -- C ABI of libstreamref.so: a bandwidth reference for the
 * MXNorm kernels on AMD Instinct MI355X (gfx950).
 *
 * mx_stream_reference moves the same HBM bytes with the same access pattern
 * as mxnorm_mxfp8_fwd (include/mxnorm.h) -- one row of x bf16 [T, d] per
 * wave, 16-byte loads, 8-byte code stores, one row of d/32 scale bytes staged
 * in LDS and written with 16-byte stores -- but computes nothing beyond a
 * byte extraction.  Its throughput is the practical ceiling for that traffic
 * mix on the device it runs on, the denominator against which the MXNorm
 * kernels' bandwidth can be judged besides the published HBM peak.
 *
 * mode: MX_STREAM_MIXED reads x and writes out [T, d] and out_small
 *       [T, d/32]; MX_STREAM_READ reads x and writes one 16-byte word per
 *       row to out_small (which must hold 16*T bytes); MX_STREAM_WRITE
 *       writes out and out_small without reading x; MX_STREAM_NVFP4 has
 *       the traffic and access pattern of mxnorm_nvfp4_fwd: it reads x,
 *       writes 4 bytes per 8 elements to out [T, d/2] and one byte per 16
 *       elements to out_small [T, d/16] (staged in LDS, 16-byte stores).
 * d must be a positive multiple of 512 and at most 4096; x, out and
 * out_small 16-byte aligned device pointers.  Asynchronous on `stream`.
 * Returns 0 on success, 1 for an invalid argument (nothing launched), 3 if
 * the launch failed.
 */
#ifndef STREAMREF_H
#define STREAMREF_H

#include <stdint.h>

#include <hip/hip_runtime_api.h> /* hipStream_t (host C code: -D__HIP_PLATFORM_AMD__) */

#ifdef __cplusplus
extern "C" {
#endif

#define MX_STREAM_MIXED 0
#define MX_STREAM_READ 1
#define MX_STREAM_WRITE 2
#define MX_STREAM_NVFP4 3

int mx_stream_reference(const void *x, int64_t T, int64_t d, uint8_t *out, uint8_t *out_small,
                        int mode, hipStream_t stream);

/*
 * mx_stream_reference_ste moves the bytes of mxnorm_ste_bwd with bf16
 * output: it reads x and grad_z, bf16 [T, d] each, and writes out, bf16
 * [T, d] (their bitwise xor), one row per wave with 16-byte accesses, the
 * stores with the STE kernel's cache policy (sc0 sc1 nt).  Same size and
 * alignment rules and return codes as mx_stream_reference.
 */
int mx_stream_reference_ste(const void *x, const void *grad_z, int64_t T, int64_t d, void *out,
                            hipStream_t stream);

/*
 * mx_stream_reference_transpose moves the bytes of mx_cast_t_fwd with E4M3
 * codes and rho given, with its tiling (one 128 x 256 tile per workgroup of
 * 512 threads, staged in LDS, 32-byte pieces per output row and lane, one
 * scale dword per column and tile) and no arithmetic: it reads x bf16
 * [R, C] and rho float [R], and writes out [C, R] (the high byte of each
 * element, transposed) and out_small [C, R/32].  R a positive multiple of
 * 128 and C of 256, each at most 65535 tiles (R == 0: nothing to do); x and
 * out 16-byte, rho and out_small 4-byte aligned device pointers.  Return
 * codes as mx_stream_reference.
 */
int mx_stream_reference_transpose(const void *x, const float *rho, int64_t R, int64_t C,
                                  uint8_t *out, uint8_t *out_small, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* STREAMREF_H */
