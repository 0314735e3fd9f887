/*
 * mxnorm.h -- C ABI of libmxnorm.so: MXNorm and RMSNorm + MX-cast forward
 * kernels for AMD Instinct MI355X (gfx950).
 *
 * Paper: "MXNorm: Reusing MXFP block scales for efficient tensor
 * normalisation" (McLean et al., arXiv 2603.13180).
 *
 * Common conventions for every compute entry point
 * ------------------------------------------------
 *  - x is a row-major bf16 matrix [T, d] (T tokens, hidden size d) given as
 *    a device pointer; gamma is a bf16 vector [d] (device) or NULL.
 *  - Outputs are device buffers owned by the caller, contiguous row-major:
 *      MXFP8: codes  uint8 [T, d]       E4M3 codes, one per element
 *             scales uint8 [T, d/32]    E8M0 scale bytes (value 2^(b-127),
 *                                       0xFF = NaN), block k = columns
 *                                       [32k, 32k+32)
 *      NVFP4: codes  uint8 [T, d/2]     E2M1 codes, two per byte, element 2j
 *                                       in the low nibble of byte j
 *             scales uint8 [T, d/16]    E4M3 block scales (0x7F = NaN)
 *      rho    float [T] or NULL         the per-row inverse RMS (estimate)
 *    Dequantised value: code * scale (MXFP8), code * scale * global_scale
 *    (NVFP4).
 *  - Alignment: x, gamma and codes must be 16-byte aligned; rho 4-byte.
 *    x must not overlap any output.
 *  - Every call is asynchronous on `stream` (a hipStream_t; NULL is the
 *    default stream).  Nothing is allocated, nothing synchronises.
 *  - Argument errors are detected on the host and returned before any launch;
 *    nothing is written then.  mx_last_error() gives a description.
 *  - T == 0 is a valid no-op (the pointers are not used and may be NULL).
 *  - d must be a multiple of the block size (32 for MXFP8, 16 for NVFP4, the
 *    chosen block for the general MX entry points) and at most MXNORM_MAX_D;
 *    larger d returns MX_EUNSUPPORTED.
 *
 * Semantics fixed where the paper leaves a choice (the same readings the
 * test oracle follows):
 *  - rho and the estimate rho~ are computed in double precision from double
 *    sums and rounded once to float; every quantity that decides a code is
 *    then computed in IEEE single precision: t = RN(x * rho~).
 *  - epsilon goes inside the square root: rho~ = (r^2 + eps)^(-1/2).  A zero
 *    radicand (all-zero row with eps = 0) gives rho~ = 0.
 *  - Element casts round to nearest-even and saturate (448 for E4M3, 6 for
 *    E2M1); signs are kept, also on zero.
 *  - A block whose scale is NaN (non-finite input) has every code equal to
 *    the input's sign bit with an all-ones magnitude.
 */
#ifndef MXNORM_H
#define MXNORM_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h> /* hipStream_t (host C code: -D__HIP_PLATFORM_AMD__) */

#ifdef __cplusplus
extern "C" {
#endif

#define MXNORM_ABI_VERSION 1
#define MXNORM_MAX_D 32768
#define MX_MATMUL_MAX_K (1 << 22)
#define MX_MATMUL_MAX_N (1 << 24)

typedef enum {
    MX_OK = 0,
    MX_EINVAL = 1,        /* a bad argument; nothing was launched */
    MX_EUNSUPPORTED = 2,  /* valid but outside what is implemented (d too large) */
    MX_EHIP = 3           /* the HIP runtime reported an error at launch */
} mx_status;

typedef enum {
    MX_SCALE_RCEIL = 0,   /* e = smallest integer with amax <= max * 2^e  */
    MX_SCALE_FLOOR = 1    /* e = floor(log2 amax) - log2(P); elements saturate */
} mx_scale_mode;
/* max = the element format's largest finite value (448 for E4M3, 6 for
 * E2M1); P = its largest power of two (256 for E4M3, 4 for E2M1). */

typedef enum {
    MX_ELEM_E4M3 = 0,     /* OCP FP8 E4M3, one code per byte            */
    MX_ELEM_E2M1 = 1      /* OCP FP4 E2M1, two codes per byte, element 2j
                             in the low nibble of byte j                */
} mx_elem;

/*
 * MXNorm, MXFP8 output (Algorithm 2; Sec. 3.4).
 * Per row t: m~_k = max over the 32 elements of block k of |x|;
 *   G = ((1/K) sum_k m~_k^p)^(1/p);  r = coef * G;  rho~ = (r^2 + eps)^(-1/2);
 *   a_k = RN(m~_k * rho~);  e_k from a_k by `scale_mode`, clamped to
 *   [-127, 127];  scales = e_k + 127;  codes = E4M3(RN(x * rho~) * 2^-e_k).
 * p: 1 or 2.  coef: the RMS/G ratio; a value <= 0 selects the paper's table
 * value for 32-element blocks (0.4261 for p = 1, 0.4185 for p = 2).
 * eps: >= 0, finite.  No gain: it is folded into the next layer's weight
 * (Sec. 3.7).
 */
mx_status mxnorm_mxfp8_fwd(const void *x, int64_t T, int64_t d, int p, float coef, float eps,
                           int scale_mode, uint8_t *codes, uint8_t *scales, float *rho,
                           hipStream_t stream);

/*
 * RMSNorm, optional gain, then the MXFP8 cast (Algorithm 1; Sec. 3.1 eq.
 * (rms) and eq. (gain); Sec. 3.2 eq. (blockscale) and eq. (blockvals)).
 * rho = ((1/d) sum x^2 + eps)^(-1/2);  y = RN(RN(x * rho) * gamma) (gamma
 * NULL: y = RN(x * rho));  m_k = max |y| over block k;  e_k from m_k;
 * codes = E4M3(y * 2^-e_k).
 */
mx_status rmsnorm_mxfp8_fwd(const void *x, const void *gamma, int64_t T, int64_t d, float eps,
                            int scale_mode, uint8_t *codes, uint8_t *scales, float *rho,
                            hipStream_t stream);

/*
 * MXNorm with NVFP4 output: 16-element blocks, E4M3 block scales, a float
 * tensor decode scale global_scale (s_g), E2M1 codes.  rho~ as for MXFP8 with
 * the 16-element-block coefficient (coef <= 0 selects 0.4814 for p = 1,
 * 0.4688 for p = 2).  Per block: a = RN(m~ * rho~);  q = a / RN(6 s_g);
 * S = E4M3(q);  den = RN(dec(S) * s_g);  codes = E2M1(RN(RN(x * rho~) / den)),
 * or signed zeros when den == 0.
 * global_scale: finite, >= FLT_MIN and <= FLT_MAX / 6.  The paper uses NVFP4
 * in its kernel and layer benchmarks (Sec. 4.4); the format's conventions
 * here are this library's.
 */
mx_status mxnorm_nvfp4_fwd(const void *x, int64_t T, int64_t d, int p, float coef, float eps,
                           float global_scale, uint8_t *codes, uint8_t *scales, float *rho,
                           hipStream_t stream);

/* RMSNorm (+ optional gain) then the NVFP4 cast, as above with y for t. */
mx_status rmsnorm_nvfp4_fwd(const void *x, const void *gamma, int64_t T, int64_t d, float eps,
                            float global_scale, uint8_t *codes, uint8_t *scales, float *rho,
                            hipStream_t stream);

/*
 * MXNorm with a general MX output: `block` in {16, 32, 64} elements per E8M0
 * scale and `elem` E4M3 or E2M1 codes (the block size and element dtype are
 * parameters of the paper's mx_norm, and its kernel benchmark sweeps both,
 * Sec. 4.4 and the performance appendix).  As mxnorm_mxfp8_fwd, with the
 * scale rule of mx_scale_mode for the element format and codes [T, d]
 * (E4M3) or [T, d/2] (E2M1); scales [T, d/block].  coef <= 0 selects the
 * table value for (block, p).  mxnorm_mx_fwd(.., 32, MX_ELEM_E4M3, ..) is
 * mxnorm_mxfp8_fwd.
 */
mx_status mxnorm_mx_fwd(const void *x, int64_t T, int64_t d, int block, int elem, int p,
                        float coef, float eps, int scale_mode, uint8_t *codes, uint8_t *scales,
                        float *rho, hipStream_t stream);

/*
 * Post-round MXNorm (the post-round appendix; an ablation the paper reports
 * unstable in training): the RMS is estimated from the block absmaxes
 * rounded down to powers of two, r(m~) = 2^floor(log2 m~) (0 for an
 * all-zero block), through the inverse of f(sigma) = E[max_i r(|X_i|)] for
 * `block` independent N(0, sigma^2) values:  Xbar = (1/K) sum_k r(m~_k);
 * sigma = f^-1(Xbar), read from a 65-point table on [1, 2] at x_i =
 * 2^(i/64) by linear interpolation in x, scaled by the power of two that
 * brings Xbar into [1, 2) (f(2 sigma) = 2 f(sigma));  rho~ = (sigma^2 +
 * eps)^(-1/2) (a zero radicand gives 0).  Then the cast of mxnorm_mx_fwd
 * (Algorithm 2).  The table is computed once per block size from the
 * appendix's series in double (sum over j = -64..64) by bisection, values
 * rounded to float; mxnorm_postround_table returns it.  Arguments as
 * mxnorm_mx_fwd without p and coef.
 */
mx_status mxnorm_postround_mx_fwd(const void *x, int64_t T, int64_t d, int block, int elem,
                                  float eps, int scale_mode, uint8_t *codes, uint8_t *scales,
                                  float *rho, hipStream_t stream);

/* The post-round table for `block` (16, 32, 64): x[i] = RN32(2^(i/64)),
 * v[i] = RN32(f^-1(x[i])), i = 0..64; host arrays of 65 floats. */
int mxnorm_postround_table(int block, float *x, float *v);

/* RMSNorm (+ optional gain) then the general MX cast (Algorithm 1). */
mx_status rmsnorm_mx_fwd(const void *x, const void *gamma, int64_t T, int64_t d, int block,
                         int elem, float eps, int scale_mode, uint8_t *codes, uint8_t *scales,
                         float *rho, hipStream_t stream);

/*
 * The plain MX cast of x, or of x * gamma (gamma NULL or bf16 [d]), with no
 * normalisation: y = RN(x * gamma), then E8M0 scales per `block` elements
 * and E4M3 or E2M1 codes exactly as in the entry points above.  With x = a
 * linear layer's weight W [N, d] (rows = output features) and gamma the norm
 * gain, this is MXCast(W gamma), the gain folded into the next weight that
 * the MXNormLinear forward multiplies MXNorm(X) with (Sec. 3.7 eq.
 * (mx-matmul); the implementation appendix's mx_norm_linear_forward).
 */
mx_status mx_cast_fwd(const void *x, const void *gamma, int64_t T, int64_t d, int block,
                      int elem, int scale_mode, uint8_t *codes, uint8_t *scales, hipStream_t stream);

typedef enum {
    MX_OUT_F32 = 0,       /* float32 output */
    MX_OUT_BF16 = 1       /* bfloat16 output, rounded to nearest even */
} mx_out_dtype;

/*
 * The MX matrix product of the MXNormLinear forward (Sec. 3.7 eq.
 * (mx-matmul)):  H = dec(A) dec(B)^T,  H[m][n] = sum_k A[m][k] B[n][k],
 * where A is an activation [M, K] (e.g. the output of mxnorm_mx_fwd) and B a
 * weight [N, K] (e.g. the output of mx_cast_fwd), both MX-encoded along K:
 * codes uint8 [rows, K] (E4M3) or [rows, K/2] (E2M1, two per byte, element
 * 2j in the low nibble) and E8M0 scales uint8 [rows, K/block], row-major,
 * device pointers.  out: device [M, N] row-major, float32 or bf16
 * (mx_out_dtype), written entirely; owned by the caller.
 * The product runs on the block-scaled matrix cores: each 32-element block's
 * scales are applied exactly, products of the elements are exact, and the
 * sum is accumulated in float32 with the matrix core's own rounding (within
 * one instruction, products far below the largest one can be dropped; the
 * total error stays within 2^-9 of sum_k |A[m][k] B[n][k]|).  A NaN scale or
 * code gives NaN; results beyond the float range are infinite.
 * block: 32 (other sizes: MX_EUNSUPPORTED).  elem: mx_elem.  Requirements:
 * K a multiple of 128 (E4M3) or 256 (E2M1) and at most MX_MATMUL_MAX_K, N a
 * multiple of 16 and at most MX_MATMUL_MAX_N (else MX_EUNSUPPORTED); codes
 * 16-byte, scales 4-byte and out
 * 16-byte aligned (else MX_EINVAL).  M == 0 or N == 0 is a no-op.  Asynchronous on
 * `stream`; nothing is allocated.
 */
mx_status mx_matmul_fwd(const uint8_t *a_codes, const uint8_t *a_scales, const uint8_t *b_codes,
                        const uint8_t *b_scales, int64_t M, int64_t N, int64_t K, int block,
                        int elem, const void *b_gain, int out_dtype, void *out, hipStream_t stream);
/* b_gain: bf16 [N] or NULL.  When given, H[m][n] = RN(acc * b_gain[n]) in
 * float: the gain applied after the product, as the weight gradient needs
 * (Sec. 3.7: grad W = MXCast(grad_H^T) MXCast(rho~ . X) . gamma); 8-byte
 * aligned. */

/*
 * Column-wise MX cast for the MXNormLinear backward (Sec. 3.7): y =
 * RN(x * rho[r]) in float (rho NULL: y = x), then the MX encoding of y^T,
 * blocked along the rows of x.  x: bf16 [R, C] row-major (device); rho: float
 * [R] or NULL; codes: [C, R] (E4M3) or [C, R/2] (E2M1, two per byte, element
 * 2j in the low nibble); scales: E8M0 [C, R/32].  Scale rule, rounding and
 * the NaN-block codes as in the forward entry points (signs from x).  With x
 * = X and rho = rho~ this is MXCast(rho~ . X) blocked along tokens; with rho
 * NULL it gives MXCast(grad_H^T) and the weight blocked along its output
 * dimension.  block: 32 (else MX_EUNSUPPORTED).  R a multiple of 32 and C of
 * 8 (else MX_EINVAL); R <= 2^31 and C <= 2^23 (else MX_EUNSUPPORTED); x and
 * codes 16-byte aligned, rho 4-byte.  R == 0 is a no-op.
 */
mx_status mx_cast_t_fwd(const void *x, const float *rho, int64_t R, int64_t C, int block,
                        int elem, int scale_mode, uint8_t *codes, uint8_t *scales, hipStream_t stream);

/*
 * The straight-through estimator of the MXNorm backward (Sec. 3.7: RMSNorm's
 * gradient used for MXNorm; the RMSNorm-gradient appendix with the RMS S
 * replaced by the estimate 1/rho~).  Per row t of x [T, d]:
 *   dXb = grad_z * gamma;  u = sum_j dXb_j x_j;
 *   grad_x_j = rho dXb_j - (1/d) rho^3 u x_j;
 *   grad_gamma_j = sum_t (rho_t x_tj) grad_z_tj.
 * x, grad_z: bf16 [T, d] (grad_z is the gradient at the norm's gained
 * output, grad_Y W); gamma: bf16 [d] or NULL (= 1); rho: float [T], the rho~
 * the forward returned.  grad_x: [T, d] float32 or bf16 (out_dtype).
 * Arithmetic: dXb exact in float, u summed in double, c = rho^3 u / d in
 * double rounded to float, grad_x = RN(RN(rho dXb) - RN(c x)); the
 * grad_gamma partial sums are float over the rows of one workgroup (at most
 * 64), then summed in double in a fixed order (deterministic for a given T).  grad_gamma: float [d] or NULL (not computed);
 * it needs `workspace`, caller-owned device memory of at least
 * mxnorm_ste_bwd_workspace_bytes(T, d) bytes (16-byte aligned), overwritten.
 * d a multiple of 8 and <= MXNORM_MAX_D; 16-byte alignment of x, grad_z,
 * gamma, grad_x; T == 0 is a no-op.
 */
size_t mxnorm_ste_bwd_workspace_bytes(int64_t T, int64_t d);
mx_status mxnorm_ste_bwd(const void *x, const void *grad_z, const void *gamma, const float *rho,
                         int64_t T, int64_t d, int out_dtype, void *grad_x, float *grad_gamma,
                         void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * mxnorm_ste_bwd without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same arguments, arithmetic, outputs and
 * errors as mxnorm_ste_bwd; the grad_gamma partial rows go to a
 * static device array of mxnorm_ste_bwd_noalloc_max_workspace() bytes
 * (32 MiB) that each GPU holds for the life of the process.  It calls no
 * hipMalloc, hipFree or allocating library routine.  Returns MX_EUNSUPPORTED,
 * before any launch, when grad_gamma is requested and
 * mxnorm_ste_bwd_workspace_bytes(T, d) exceeds that size (for example
 * T = 32768 fits up to d = 16384).  The device is the stream's (the current
 * device for the null stream); its array's address is looked up on the first
 * call on that device.  All calls on one GPU share its array: calls that
 * overlap in time on one GPU (on different streams, or from several host
 * threads) race and give wrong grad_gamma.  Every byte a call reads from the
 * array is written earlier in the same call, so nothing needs clearing.
 */
size_t mxnorm_ste_bwd_noalloc_max_workspace(void);
mx_status mxnorm_ste_bwd_noalloc(const void *x, const void *grad_z, const void *gamma,
                                 const float *rho, int64_t T, int64_t d, int out_dtype,
                                 void *grad_x, float *grad_gamma, hipStream_t stream);

/*
 * Default NVFP4 tensor decode scales: an output bound divided by 6 * 448, so
 * the bound maps to the largest E2M1 x E4M3 magnitude.  MXNorm: Lemma 2's
 * bound K^(1/p) / coef (K = d / block; coef <= 0 selects the table value);
 * RMSNorm: Lemma 1's bound sqrt(d), times max |gamma|.  Sec. 3.5.
 * Return NaN for invalid arguments.
 */
float mxnorm_default_global_scale(int64_t d, int block, int p, float coef);
float rmsnorm_default_global_scale(int64_t d, float gamma_absmax);

/* The paper's absmax_scale_factor table (implementation appendix): block in
 * {16, 32, 64}, p in {1, 2}; NaN otherwise. */
float mxnorm_coef(int block, int p);

/* Static description of a status code. */
const char *mx_status_str(mx_status s);

/* Description of the last non-OK status returned on the calling thread
 * ("" if none).  The pointer stays valid until the next call on the thread. */
const char *mx_last_error(void);

/* MXNORM_ABI_VERSION of the built library. */
int mxnorm_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* MXNORM_H */
