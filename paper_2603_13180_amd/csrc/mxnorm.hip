// mxnorm.hip -- MXNorm and RMSNorm + MX-cast forward kernels for gfx950
// (AMD Instinct MI355X), behind the C ABI declared in include/mxnorm.h.
//
// Paper: "MXNorm: Reusing MXFP block scales for efficient tensor
// normalisation" (McLean et al., arXiv 2603.13180): Algorithm 1 (RMSNorm +
// MXCast), Algorithm 2 (MXNorm), Sec. 3.1-3.4.
//
// Kernel design (one launch = one pass over the activations):
//  * A row of d bf16 values is split into 16-byte chunks (8 elements).  A
//    "team" of TL lanes owns a row; lane l holds chunks j*TL + l, j < CPL, so
//    every wave-wide load and store is fully coalesced and the whole row stays
//    in registers between the statistics pass and the cast.  TL is 16, 32 or
//    64 lanes inside one wave, or 2/4/8 waves (LDS joins their partial sums).
//  * A scale block (32 elements for MXFP8, 16 for NVFP4) is 4 (2) consecutive
//    lanes' chunks, so its absmax is a lane-local max plus 2 (1) DPP
//    quad-permute steps.  MXNorm takes the absmax on the raw bf16 bits (an
//    unsigned 16-bit max of the magnitudes); the RMSNorm baseline has to form
//    y = x * rho first and take the absmax of y.
//  * The row statistic (sum of squared block absmaxes for MXNorm: K terms;
//    sum of squared elements for RMSNorm: d terms) is accumulated in double
//    and reduced across the team; rho is computed once per row in double and
//    rounded to float.  Everything that decides a code is single precision.
//  * No MFMA: the work is a streaming reduction plus an element-wise cast,
//    bound by HBM bandwidth.
#include <hip/hip_runtime.h>

#include <float.h>
#include <math.h>
#include <stdarg.h>
#include <stdint.h>
#include <stdio.h>

#include "mxnorm.h"
#include "norm_cast.h"
#include "status.h"

#include <cmath>
#include <mutex>

namespace mxk {

hipError_t launch_norm_cast_MX8_B16(const Args &A, int kind, int TL, int CPL, hipStream_t stream);
hipError_t launch_norm_cast_MX8_B32(const Args &A, int kind, int TL, int CPL, hipStream_t stream);
hipError_t launch_norm_cast_MX8_B64(const Args &A, int kind, int TL, int CPL, hipStream_t stream);
hipError_t launch_norm_cast_MX4_B16(const Args &A, int kind, int TL, int CPL, hipStream_t stream);
hipError_t launch_norm_cast_MX4_B32(const Args &A, int kind, int TL, int CPL, hipStream_t stream);
hipError_t launch_norm_cast_MX4_B64(const Args &A, int kind, int TL, int CPL, hipStream_t stream);
hipError_t launch_norm_cast_NV4_B16(const Args &A, int kind, int TL, int CPL, hipStream_t stream);

hipError_t launch_norm_cast(int fmt, const Args &A, int kind, int TL, int CPL, hipStream_t stream)
{
    switch (fmt) {
    case MX8_B16: return launch_norm_cast_MX8_B16(A, kind, TL, CPL, stream);
    case MX8_B32: return launch_norm_cast_MX8_B32(A, kind, TL, CPL, stream);
    case MX8_B64: return launch_norm_cast_MX8_B64(A, kind, TL, CPL, stream);
    case MX4_B16: return launch_norm_cast_MX4_B16(A, kind, TL, CPL, stream);
    case MX4_B32: return launch_norm_cast_MX4_B32(A, kind, TL, CPL, stream);
    case MX4_B64: return launch_norm_cast_MX4_B64(A, kind, TL, CPL, stream);
    case NV4_B16: return launch_norm_cast_NV4_B16(A, kind, TL, CPL, stream);
    default: return hipErrorInvalidValue;
    }
}

thread_local char g_err[256] = "";

mx_status fail(mx_status st, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return st;
}

void clear_error() { g_err[0] = '\0'; }

const char *last_error() { return g_err; }

} // namespace mxk

namespace {

using namespace mxk;

// ------------------------------------------------------------ host side --

bool aligned(const void *p, uintptr_t n) { return ((uintptr_t)p % n) == 0; }

float table_coef(int block, int p)
{
    if (p != 1 && p != 2)
        return NAN;
    switch (block) {
    case 16: return p == 1 ? 0.4814f : 0.4688f;
    case 32: return p == 1 ? 0.4261f : 0.4185f;
    case 64: return p == 1 ? 0.3852f : 0.3803f;
    default: return NAN;
    }
}

// Team size (lanes per row, 16 .. 512) and register chunks per lane (4 or 8).
// The smallest team that holds the row in at most 8 chunks per lane gives the
// most independent loads per lane; when that leaves fewer than kMinWaves
// waves in the launch (too few rows to cover 256 compute units several times
// over), wider teams with fewer chunks per lane are taken, up to 64 lanes.
constexpr int64_t kMinWaves = 4096;

void pick_team(int64_t T, int nc, int &TL, int &CPL)
{
    static const int sizes[] = {16, 32, 64, 128, 256, 512};
    TL = 0;
    CPL = 0;
    for (int s : sizes) {
        if (nc <= 8 * s) {
            TL = s;
            break;
        }
    }
    if (TL == 0)
        return;
    // widen short-of-waves launches while every lane keeps at least one chunk
    while (TL < 64 && T * TL / 64 < kMinWaves && nc >= 2 * TL)
        TL *= 2;
    CPL = (nc + TL - 1) / TL <= 4 ? 4 : 8;
}

mx_status check_common(const void *x, const void *gamma, int64_t T, int64_t d, int block,
                       float eps, const uint8_t *codes, const uint8_t *scales, const float *rho)
{
    if (T < 0)
        return fail(MX_EINVAL, "T must be >= 0 (got %lld)", (long long)T);
    if (T > 0 && (!x || !codes || !scales))
        return fail(MX_EINVAL, "x, codes and scales must be non-NULL");
    if (d <= 0 || d % block != 0)
        return fail(MX_EINVAL, "d must be a positive multiple of %d (got %lld)", block,
                    (long long)d);
    if (d > MXNORM_MAX_D)
        return fail(MX_EUNSUPPORTED, "d = %lld exceeds the supported maximum %d", (long long)d,
                    MXNORM_MAX_D);
    if (!(eps >= 0.0f) || !(eps <= FLT_MAX))
        return fail(MX_EINVAL, "eps must be finite and >= 0");
    if (!aligned(x, 16) || !aligned(codes, 16) || (gamma && !aligned(gamma, 16)))
        return fail(MX_EINVAL, "x, gamma and codes must be 16-byte aligned");
    if (rho && !aligned(rho, 4))
        return fail(MX_EINVAL, "rho must be 4-byte aligned");
    if (T > (int64_t)(INT64_MAX / d) || T / 16 > (int64_t)0x7FFFFFFF)
        return fail(MX_EUNSUPPORTED, "T = %lld is too large", (long long)T);
    return MX_OK;
}

mx_status check_global_scale(float s_g)
{
    if (!(s_g >= FLT_MIN) || !(s_g <= FLT_MAX / 6.0f))
        return fail(MX_EINVAL, "global_scale must be finite, >= FLT_MIN and <= FLT_MAX/6");
    return MX_OK;
}

mx_status run(Args A, int fmt, int kind, hipStream_t stream)
{
    int TL, CPL;
    pick_team(A.T, A.nc, TL, CPL);
    if (TL == 0)
        return fail(MX_EUNSUPPORTED, "no launch configuration for d = %d", A.d);
    if (A.T == 0)
        return MX_OK;
    // widest scale store that K and the buffer's alignment allow (K <= 4*TL,
    // so 16-byte stores need at most one per lane)
    const uintptr_t sa = (uintptr_t)A.scales;
    A.sw = (A.K % 16 == 0 && sa % 16 == 0) ? 16 : (A.K % 4 == 0 && sa % 4 == 0) ? 4 : 1;
    hipStream_t st = (hipStream_t)stream;
    hipError_t e;
    if (fmt < MX8_B16 || fmt > NV4_B16)
        return fail(MX_EINVAL, "unknown output format");
    e = launch_norm_cast(fmt, A, kind, TL, CPL, st);
    if (e != hipSuccess)
        return fail(MX_EHIP, "kernel launch failed: %s", hipGetErrorString(e));
    return MX_OK;
}

// ----------------------------------------------------- post-round table --
//
// Post-round MXNorm estimates the RMS as f^-1(Xbar), Xbar the mean of the
// block absmaxes rounded down to powers of two and f(sigma) = E[r(M)], with
// M the largest of B independent |N(0, sigma^2)| values and r(m) =
// 2^floor(log2 m) (the post-round appendix).  Because f(2 sigma) = 2
// f(sigma) the inverse is tabulated on [1, 2] at x_i = 2^(i/64) (values
// rounded to float) and scaled by powers of two in the kernel.
//
// The library evaluates f through the layer-cake identity rather than the
// appendix's sum over the events {r(M) = 2^j}: r(m) = sum over j with
// 2^j <= m of 2^(j-1), so
//     f(sigma) = sum_j 2^(j-1) P(M >= 2^j) = sum_j 2^(j-1) (1 - F_j^B),
// F_j = erf(2^j / (sigma sqrt 2)).  1 - F^B is formed from erfc so that the
// upper terms keep their relative precision.  For the sigmas the table
// needs (about 0.3 .. 3) every term below j = kLow has F_j^B < 2^-600, so it
// equals 2^(j-1) in double and their sum is the closed form 2^(kLow-1);
// above j = kHigh the terms are zero.  The root of f(sigma) = x is then found by
// Newton's method on the analytic derivative
//     f'(sigma) = sum_j 2^(j-1) B F_j^(B-1) (2/sqrt(pi)) e^(-u_j^2) u_j / sigma,
// u_j = 2^j / (sigma sqrt 2), kept inside a bracket that halving the step
// falls back to.

constexpr int kLow = -40, kHigh = 40;

// P(M >= 2^j) = 1 - erf(u)^B, u = 2^j / (sigma sqrt 2)
double tail_prob(double u, int B)
{
    const double q = std::erfc(u);
    if (q < 0.5)
        return -std::expm1((double)B * std::log1p(-q));
    return 1.0 - std::pow(std::erf(u), (double)B);
}

// f(sigma) and f'(sigma) together
void layer_cake_f(double sigma, int B, double &f, double &df)
{
    const double inv_s2 = 1.0 / (sigma * std::sqrt(2.0));
    const double c = 2.0 / std::sqrt(M_PI);
    f = std::ldexp(1.0, kLow - 1); // the terms j < kLow, each 2^(j-1) exactly
    df = 0.0;
    for (int j = kLow; j <= kHigh; ++j) {
        const double w = std::ldexp(1.0, j - 1);
        const double u = std::ldexp(inv_s2, j);
        f += w * tail_prob(u, B);
        const double g = std::erf(u);
        if (g > 0.0)
            df += w * (double)B * std::pow(g, (double)(B - 1)) * c * std::exp(-u * u) * u / sigma;
    }
}

// f^-1(x) for x > 0: bracket by powers of two (f(2 s) = 2 f(s)), then
// Newton steps, replaced by the bracket's midpoint whenever a step would
// leave the bracket; stop when a step no longer changes sigma by more than
// a few units in the last place.
double layer_cake_inverse(double x, int B)
{
    double f, df;
    double lo = x, hi = x;
    for (layer_cake_f(lo, B, f, df); f > x; layer_cake_f(lo, B, f, df))
        lo *= 0.5;
    for (layer_cake_f(hi, B, f, df); f < x; layer_cake_f(hi, B, f, df))
        hi *= 2.0;
    double s = 0.5 * (lo + hi);
    for (int it = 0; it < 100; ++it) {
        layer_cake_f(s, B, f, df);
        const double r = f - x;
        if (r == 0.0)
            return s;
        (r < 0.0 ? lo : hi) = s;
        double next = df > 0.0 ? s - r / df : 0.5 * (lo + hi);
        if (!(next > lo && next < hi))
            next = 0.5 * (lo + hi);
        const bool done = std::fabs(next - s) <= 4.0 * DBL_EPSILON * s;
        s = next;
        if (done)
            break;
    }
    return s;
}

struct PostTable {
    float x[65], v[65];
};

// The table for block size B (16, 32 or 64), computed once per process.
const PostTable &post_table(int B)
{
    static std::once_flag once[3];
    static PostTable tab[3];
    const int k = B == 16 ? 0 : B == 32 ? 1 : 2;
    std::call_once(once[k], [&] {
        for (int i = 0; i <= 64; ++i) {
            tab[k].x[i] = (float)std::pow(2.0, (double)i / 64.0);
            tab[k].v[i] = (float)layer_cake_inverse((double)tab[k].x[i], B);
        }
    });
    return tab[k];
}

// The MX format for a block size and element format, or -1.
int mx_format(int block, int elem)
{
    if (elem != MX_ELEM_E4M3 && elem != MX_ELEM_E2M1)
        return -1;
    const int base = elem == MX_ELEM_E4M3 ? MX8_B16 : MX4_B16;
    switch (block) {
    case 16: return base;
    case 32: return base + 1;
    case 64: return base + 2;
    default: return -1;
    }
}

Args make_args(const void *x, const void *gamma, int64_t T, int64_t d, int block, int p,
               float coef, float eps, int mode, float s_g, uint8_t *codes, uint8_t *scales,
               float *rho)
{
    Args A;
    A.x = static_cast<const uint16_t *>(x);
    A.gamma = static_cast<const uint16_t *>(gamma);
    A.codes = codes;
    A.scales = scales;
    A.rho = rho;
    A.T = T;
    A.d = (int)d;
    A.nc = (int)(d / 8);
    A.K = (int)(d / block);
    A.p = p;
    A.coef = coef;
    A.eps = eps;
    A.mode = mode;
    A.s_g = s_g;
    // NVFP4: the scale quotient's divisor 6 s_g and its reciprocal, each one
    // IEEE float rounding, once per launch rather than once per row
    A.six_sg = 6.0f * s_g;
    A.rcp_six_sg = A.six_sg > 0.0f ? 1.0f / A.six_sg : 0.0f;
    return A;
}

mx_status check_p_coef(int p, float &coef, int block)
{
    if (p != 1 && p != 2)
        return fail(MX_EINVAL, "p must be 1 or 2 (got %d)", p);
    if (isnan(coef) || isinf(coef))
        return fail(MX_EINVAL, "coef must be finite");
    if (coef <= 0.0f)
        coef = table_coef(block, p);
    return MX_OK;
}

} // namespace

extern "C" {

mx_status mxnorm_mxfp8_fwd(const void *x, int64_t T, int64_t d, int p, float coef, float eps,
                           int scale_mode, uint8_t *codes, uint8_t *scales, float *rho,
                           hipStream_t stream)
{
    clear_error();
    mx_status st = check_common(x, nullptr, T, d, 32, eps, codes, scales, rho);
    if (st != MX_OK)
        return st;
    if ((st = check_p_coef(p, coef, 32)) != MX_OK)
        return st;
    if (scale_mode != MX_SCALE_RCEIL && scale_mode != MX_SCALE_FLOOR)
        return fail(MX_EINVAL, "unknown scale_mode %d", scale_mode);
    return run(make_args(x, nullptr, T, d, 32, p, coef, eps, scale_mode, 1.0f, codes, scales,
                         rho),
               MX8_B32, K_MXN, stream);
}

mx_status rmsnorm_mxfp8_fwd(const void *x, const void *gamma, int64_t T, int64_t d, float eps,
                            int scale_mode, uint8_t *codes, uint8_t *scales, float *rho,
                            hipStream_t stream)
{
    clear_error();
    mx_status st = check_common(x, gamma, T, d, 32, eps, codes, scales, rho);
    if (st != MX_OK)
        return st;
    if (scale_mode != MX_SCALE_RCEIL && scale_mode != MX_SCALE_FLOOR)
        return fail(MX_EINVAL, "unknown scale_mode %d", scale_mode);
    return run(make_args(x, gamma, T, d, 32, 2, 1.0f, eps, scale_mode, 1.0f, codes, scales,
                         rho),
               MX8_B32, K_RMS, stream);
}

mx_status mxnorm_nvfp4_fwd(const void *x, int64_t T, int64_t d, int p, float coef, float eps,
                           float global_scale, uint8_t *codes, uint8_t *scales, float *rho,
                           hipStream_t stream)
{
    clear_error();
    mx_status st = check_common(x, nullptr, T, d, 16, eps, codes, scales, rho);
    if (st != MX_OK)
        return st;
    if ((st = check_p_coef(p, coef, 16)) != MX_OK)
        return st;
    if ((st = check_global_scale(global_scale)) != MX_OK)
        return st;
    return run(make_args(x, nullptr, T, d, 16, p, coef, eps, MX_SCALE_RCEIL, global_scale,
                         codes, scales, rho),
               NV4_B16, K_MXN, stream);
}

mx_status rmsnorm_nvfp4_fwd(const void *x, const void *gamma, int64_t T, int64_t d, float eps,
                            float global_scale, uint8_t *codes, uint8_t *scales, float *rho,
                            hipStream_t stream)
{
    clear_error();
    mx_status st = check_common(x, gamma, T, d, 16, eps, codes, scales, rho);
    if (st != MX_OK)
        return st;
    if ((st = check_global_scale(global_scale)) != MX_OK)
        return st;
    return run(make_args(x, gamma, T, d, 16, 2, 1.0f, eps, MX_SCALE_RCEIL, global_scale, codes,
                         scales, rho),
               NV4_B16, K_RMS, stream);
}

mx_status mxnorm_mx_fwd(const void *x, int64_t T, int64_t d, int block, int elem, int p,
                        float coef, float eps, int scale_mode, uint8_t *codes, uint8_t *scales,
                        float *rho, hipStream_t stream)
{
    clear_error();
    const int fmt = mx_format(block, elem);
    if (fmt < 0)
        return fail(MX_EINVAL, "block must be 16, 32 or 64 and elem E4M3 or E2M1");
    mx_status st = check_common(x, nullptr, T, d, block, eps, codes, scales, rho);
    if (st != MX_OK)
        return st;
    if ((st = check_p_coef(p, coef, block)) != MX_OK)
        return st;
    if (scale_mode != MX_SCALE_RCEIL && scale_mode != MX_SCALE_FLOOR)
        return fail(MX_EINVAL, "unknown scale_mode %d", scale_mode);
    return run(make_args(x, nullptr, T, d, block, p, coef, eps, scale_mode, 1.0f, codes, scales,
                         rho),
               fmt, K_MXN, stream);
}

mx_status mxnorm_postround_mx_fwd(const void *x, int64_t T, int64_t d, int block, int elem,
                                  float eps, int scale_mode, uint8_t *codes, uint8_t *scales,
                                  float *rho, hipStream_t stream)
{
    clear_error();
    const int fmt = mx_format(block, elem);
    if (fmt < 0)
        return fail(MX_EINVAL, "block must be 16, 32 or 64 and elem E4M3 or E2M1");
    mx_status st = check_common(x, nullptr, T, d, block, eps, codes, scales, rho);
    if (st != MX_OK)
        return st;
    if (scale_mode != MX_SCALE_RCEIL && scale_mode != MX_SCALE_FLOOR)
        return fail(MX_EINVAL, "unknown scale_mode %d", scale_mode);
    Args A = make_args(x, nullptr, T, d, block, 1, 1.0f, eps, scale_mode, 1.0f, codes, scales,
                       rho);
    const PostTable &tab = post_table(block);
    for (int i = 0; i <= 64; ++i) {
        A.pr_x[i] = tab.x[i];
        A.pr_v[i] = tab.v[i];
    }
    return run(A, fmt, K_MXN_POST, stream);
}

int mxnorm_postround_table(int block, float *x, float *v)
{
    clear_error();
    if (block != 16 && block != 32 && block != 64)
        return fail(MX_EINVAL, "block must be 16, 32 or 64");
    if (!x || !v)
        return fail(MX_EINVAL, "x and v must be non-NULL");
    const PostTable &tab = post_table(block);
    for (int i = 0; i <= 64; ++i) {
        x[i] = tab.x[i];
        v[i] = tab.v[i];
    }
    return MX_OK;
}

mx_status rmsnorm_mx_fwd(const void *x, const void *gamma, int64_t T, int64_t d, int block,
                         int elem, float eps, int scale_mode, uint8_t *codes, uint8_t *scales,
                         float *rho, hipStream_t stream)
{
    clear_error();
    const int fmt = mx_format(block, elem);
    if (fmt < 0)
        return fail(MX_EINVAL, "block must be 16, 32 or 64 and elem E4M3 or E2M1");
    mx_status st = check_common(x, gamma, T, d, block, eps, codes, scales, rho);
    if (st != MX_OK)
        return st;
    if (scale_mode != MX_SCALE_RCEIL && scale_mode != MX_SCALE_FLOOR)
        return fail(MX_EINVAL, "unknown scale_mode %d", scale_mode);
    return run(make_args(x, gamma, T, d, block, 2, 1.0f, eps, scale_mode, 1.0f, codes, scales,
                         rho),
               fmt, K_RMS, stream);
}

mx_status mx_cast_fwd(const void *x, const void *gamma, int64_t T, int64_t d, int block,
                      int elem, int scale_mode, uint8_t *codes, uint8_t *scales, hipStream_t stream)
{
    clear_error();
    const int fmt = mx_format(block, elem);
    if (fmt < 0)
        return fail(MX_EINVAL, "block must be 16, 32 or 64 and elem E4M3 or E2M1");
    mx_status st = check_common(x, gamma, T, d, block, 0.0f, codes, scales, nullptr);
    if (st != MX_OK)
        return st;
    if (scale_mode != MX_SCALE_RCEIL && scale_mode != MX_SCALE_FLOOR)
        return fail(MX_EINVAL, "unknown scale_mode %d", scale_mode);
    return run(make_args(x, gamma, T, d, block, 2, 1.0f, 0.0f, scale_mode, 1.0f, codes, scales,
                         nullptr),
               fmt, K_CAST, stream);
}

float mxnorm_default_global_scale(int64_t d, int block, int p, float coef)
{
    if (d <= 0 || (block != 16 && block != 32 && block != 64) || d % block || (p != 1 && p != 2))
        return NAN;
    if (!(coef > 0.0f))
        coef = table_coef(block, p);
    const double K = (double)(d / block);
    const double bound = (p == 1 ? K : sqrt(K)) / (double)coef;
    return (float)(bound / (6.0 * 448.0));
}

float rmsnorm_default_global_scale(int64_t d, float gamma_absmax)
{
    if (d <= 0 || !(gamma_absmax > 0.0f) || !(gamma_absmax <= FLT_MAX))
        return NAN;
    return (float)(sqrt((double)d) * (double)gamma_absmax / (6.0 * 448.0));
}

float mxnorm_coef(int block, int p) { return table_coef(block, p); }

const char *mx_status_str(mx_status s)
{
    switch (s) {
    case MX_OK: return "MX_OK";
    case MX_EINVAL: return "MX_EINVAL: invalid argument";
    case MX_EUNSUPPORTED: return "MX_EUNSUPPORTED: unsupported size";
    case MX_EHIP: return "MX_EHIP: HIP runtime error";
    }
    return "unknown mx_status";
}

const char *mx_last_error(void) { return mxk::last_error(); }

int mxnorm_abi_version(void) { return MXNORM_ABI_VERSION; }

} // extern "C"
