// norm_cast.h -- the fused norm + MX-cast kernel template shared by the
// per-format translation units (norm_cast_f*.hip) of libmxnorm.so.  See
// mxnorm.hip for the design notes and include/mxnorm.h for the ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <float.h>
#include <math.h>
#include <stdint.h>

#include "mxnorm.h"

#pragma clang fp contract(off)

namespace mxk {


struct Args {
    const uint16_t *x;
    const uint16_t *gamma;
    uint8_t *codes;
    uint8_t *scales;
    float *rho;
    int64_t T;
    int d;      // hidden size
    int nc;     // 16-byte chunks per row (d / 8)
    int K;      // scale blocks per row
    int p;      // p-mean exponent (1 or 2)
    float coef; // RMS / G_p ratio
    float eps;
    int mode;   // MX_SCALE_RCEIL or MX_SCALE_FLOOR
    float s_g;  // NVFP4 tensor decode scale
    float six_sg, rcp_six_sg; // RN(6 s_g) and RN(1 / RN(6 s_g))
    int sw;     // bytes per scale store: 16, 4 or 1 (set from K and alignment)
    // post-round MXNorm: the inverse of f on [1, 2] at x_i = 2^(i/64)
    float pr_x[65], pr_v[65];
};

// ---------------------------------------------------------------- helpers --

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

// Streaming 16-byte load: each input byte is read exactly once, so mark it
// non-temporal.
__device__ __forceinline__ uint4 load_stream(const uint4 *p)
{
    const u32x4_t t = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(p));
    return make_uint4(t.x, t.y, t.z, t.w);
}

// Largest of v over the BL lanes (2, 4 or 8 consecutive, aligned) of a scale
// block: quad permutes for lane i^1 and i^2, then the DPP row-half-mirror
// (lane i <-> 7 - i inside each group of 8) to join two quads.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_mov(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}

template <int BL>
__device__ __forceinline__ uint32_t block_max(uint32_t m)
{
    m = max(m, dpp_mov<0xB1>(m));
    if constexpr (BL >= 4)
        m = max(m, dpp_mov<0x4E>(m));
    if constexpr (BL >= 8)
        m = max(m, dpp_mov<0x141>(m));
    return m;
}

typedef unsigned short ushort2_t __attribute__((ext_vector_type(2)));

// Largest |x| of 8 bf16 values as the 15-bit magnitude pattern.  Unsigned
// order of bf16 magnitudes is numeric order, with NaN above Inf, so a NaN
// input propagates.
__device__ __forceinline__ uint32_t chunk_absmax_bits(uint4 v)
{
    const uint32_t m = 0x7FFF7FFFu;
    ushort2_t a = __builtin_bit_cast(ushort2_t, v.x & m);
    ushort2_t b = __builtin_bit_cast(ushort2_t, v.y & m);
    ushort2_t c = __builtin_bit_cast(ushort2_t, v.z & m);
    ushort2_t d = __builtin_bit_cast(ushort2_t, v.w & m);
    ushort2_t r = __builtin_elementwise_max(__builtin_elementwise_max(a, b),
                                            __builtin_elementwise_max(c, d));
    return r.x > r.y ? (uint32_t)r.x : (uint32_t)r.y;
}

// E8M0 scale byte of a block whose largest |value| is a (>= +0 or NaN): e + 127,
// or 0xFF when a is not finite.  With E the biased fp32 exponent of a, m its
// 23-bit significand field, and the element format's largest finite value
// 1.75 * 2^8 (E4M3) or 1.5 * 2^2 (E2M1): RCEIL (the smallest e with
// a <= max * 2^e) is e + 127 = E - P + [m > 0x600000] (E4M3, P = 8) or
// E - P + [m > 0x400000] (E2M1, P = 2), i.e. ((a + 0x1FFFFF) >> 23) - 8 and
// ((a + 0x3FFFFF) >> 23) - 2 on the bit pattern; FLOOR (e = floor(log2 a) -
// P, P the log2 of the format's largest power of two) is (a >> 23) - P.
// Both are clamped below at byte 0 (e = -127), which also covers zero and
// fp32 subnormals; the largest finite a stays below byte 254.
template <bool FP4>
__device__ __forceinline__ uint32_t e8m0_byte(float a, int mode)
{
    constexpr uint32_t P = FP4 ? 2u : 8u;
    constexpr uint32_t ROUND = FP4 ? 0x3FFFFFu : 0x1FFFFFu;
    const uint32_t ab = __float_as_uint(a); // sign bit clear unless a is NaN
    const uint32_t round = (mode == MX_SCALE_RCEIL) ? ROUND : 0u;
    const uint32_t biased = (ab + round) >> 23;
    const uint32_t byte = max(biased, P) - P;
    return (ab >= 0x7F800000u) ? 0xFFu : byte;
}

typedef short short2_t __attribute__((ext_vector_type(2)));

// Four E4M3 codes (one dword, element 0 in the low byte) of t0..t3 / 2^e.
// v_cvt_scalef32_pk_fp8_f32 divides by 2^(exponent field of the scale
// operand - 127) and rounds to nearest even; the E8M0 byte shifted into the
// fp32 exponent field is therefore the scale operand (byte 0 reads as
// 2^-127).  The instruction returns NaN above 464 instead of saturating, so
// callers keep |t / 2^e| <= 448: RCEIL guarantees it, FLOOR clamps first.
// Before use it was checked on the device, on all 2^32 fp32 inputs and for
// scale exponents -127, -7, 5 and 120, against an integer-rounding E4M3
// encoder (fp32 significand rounded to 3 bits, ties to even, exponent
// rebiased; n * 2^-9 with n = rint(|v| * 512) below 2^-6); the GPU parity
// tests hold it to the oracle.
__device__ __forceinline__ uint32_t e4m3x4_hw(float t0, float t1, float t2, float t3,
                                              float scale)
{
    short2_t r = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32((short2_t){0, 0}, t0, t1, scale, false);
    r = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(r, t2, t3, scale, true);
    return __builtin_bit_cast(uint32_t, r);
}

// E2M1 code (low nibble) of |v| with the sign bit of `sign_src`, nearest
// even, saturating at 6 (a NaN magnitude, which only an overflowed quotient
// produces here, saturates too).  [1, 6): round the significand to 1 bit and
// rebias (127 -> 1); below 1 the value is n * 0.5 with n = rint(2 |v|).
__device__ __forceinline__ uint32_t e2m1_code(float v, float sign_src)
{
    const uint32_t s = (__float_as_uint(sign_src) >> 28) & 0x8u;
    const uint32_t a = __float_as_uint(v) & 0x7FFFFFFFu;
    uint32_t r;
    if (a >= 0x40C00000u)
        r = 7u;
    else if (a >= 0x3F800000u)
        r = ((a + 0x1FFFFFu + ((a >> 22) & 1u)) >> 22) - 0xFCu;
    else
        r = (uint32_t)__builtin_rintf(__uint_as_float(a) * 2.0f);
    return s | r;
}

// Value of a non-negative finite E4M3 code.
__device__ __forceinline__ float e4m3_value(uint32_t S)
{
    const uint32_t E = S >> 3, M = S & 7u;
    return E ? __uint_as_float(((E + 120u) << 23) | (M << 20)) : (float)M * 0x1p-9f;
}

// Correctly rounded t / den from the correctly rounded reciprocal r = 1/den:
// one product and one fused correction (Markstein).  Exact for den >= 2^-90
// whenever |t / den| >= 2^-20; smaller quotients are below every E2M1 and
// E4M3 rounding threshold, so the code is unaffected.
__device__ __forceinline__ float div_by_recip(float t, float den, float r)
{
    const float q0 = t * r;
    const float rem = __builtin_fmaf(-q0, den, t);
    return __builtin_fmaf(rem, r, q0);
}

// -(t / den) from r = 1/den as div_by_recip computes it, with the
// correction applied as -rem * r + (-q0): for a nonzero quotient the single
// rounding gives exactly the negated value, and a zero or underflowing
// quotient comes out with the sign opposite to t's (q0 and rem carry the
// sign of t), where rem * r + q0 would round an exact zero to +0.  Encoding
// the negated quotients and flipping every code's sign bit afterwards keeps
// the sign of t on zeros at one operation per eight codes.
__device__ __forceinline__ float neg_div_by_recip(float t, float den, float r)
{
    const float q0 = t * r;
    const float rem = __builtin_fmaf(-q0, den, t);
    return __builtin_fmaf(-rem, r, -q0);
}

// Codes of a NaN block: each element's bf16 sign bit with an all-ones
// magnitude.  w0, w1 hold four bf16 values (elements 0..3).
__device__ __forceinline__ uint32_t nan_codes_e4m3(uint32_t w0, uint32_t w1)
{
    return 0x7F7F7F7Fu | ((w0 >> 8) & 0x80u) | ((w0 >> 16) & 0x8000u) |
           ((w1 << 8) & 0x800000u) | (w1 & 0x80000000u);
}

__device__ __forceinline__ uint32_t sign_nibbles(uint4 v)
{
    // bit 15 of bf16 element k -> bit 4k+3
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    uint32_t r = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        r |= ((w[i] >> 15) & 1u) << (8 * i + 3);
        r |= ((w[i] >> 31) & 1u) << (8 * i + 7);
    }
    return r;
}

// rho~ = (r^2 + eps)^(-1/2), r = coef * G_p, G_p from the sum S of m~^p over
// K blocks (Alg. 2; Sec. 3.4).  Double precision, rounded once to float.
__device__ __forceinline__ float rho_estimate(double S, int K, int p, float coef, float eps)
{
    // S / K; for a power-of-two K the scaling is exact, so it equals the
    // correctly rounded quotient without the division's latency
    const double mean = (K & (K - 1)) == 0 ? ldexp(S, -__builtin_ctz((unsigned)K)) : S / (double)K;
    const double G = (p == 1) ? mean : sqrt(mean);
    const double r = (double)coef * G;
    const double u = r * r + (double)eps;
    return (u == 0.0) ? 0.0f : (float)(1.0 / sqrt(u));
}

// rho = ((1/d) sum x^2 + eps)^(-1/2) (Sec. 3.1 eq. (rms)).
__device__ __forceinline__ float rho_rms(double S, int d, float eps)
{
    const double mean = (d & (d - 1)) == 0 ? ldexp(S, -__builtin_ctz((unsigned)d)) : S / (double)d;
    const double u = mean + (double)eps;
    return (u == 0.0) ? 0.0f : (float)(1.0 / sqrt(u));
}

// r(m~) = 2^floor(log2 m~) of a bf16 block absmax given as its 16-bit
// magnitude pattern, as float bits: the exponent field alone for normal
// values, the highest set significand bit for subnormals; 0 stays 0 and
// Inf/NaN pass through.
__device__ __forceinline__ uint32_t pow2_floor_bits(uint32_t m)
{
    const uint32_t u = m << 16;
    if (u >= 0x7F800000u)
        return u;
    if (u & 0x7F800000u)
        return u & 0x7F800000u;
    return u ? (0x80000000u >> __builtin_clz(u)) : 0u;
}

// Post-round MXNorm's rho~ from Xbar, the mean of r(m~) over the row's
// blocks (the post-round appendix): sigma = f^-1(Xbar) with Xbar = y 2^k,
// y in [1, 2), f^-1(y) interpolated linearly between the table points that
// bracket y, times 2^k; rho~ = (sigma^2 + eps)^(-1/2) in double, rounded to
// float (a zero radicand gives 0).
__device__ __forceinline__ float rho_postround(double X, const float *px, const float *pv, float eps)
{
    double sigma = X;
    if (X != 0.0 && X <= DBL_MAX) {
        int e;
        const double y = 2.0 * frexp(X, &e);
        // the segment: the largest i with x_i <= y.  Start from the estimate
        // 64 log2(y) and correct it exactly against the table, which lands on
        // the same i as a scan from 0 at a few steps' cost
        int i = min(max((int)(64.0f * __log2f((float)y)), 0), 63);
        while (i > 0 && (double)px[i] > y)
            --i;
        while (i + 1 < 64 && (double)px[i + 1] <= y)
            ++i;
        const double t = (y - (double)px[i]) / ((double)px[i + 1] - (double)px[i]);
        sigma = ldexp((double)pv[i] + t * ((double)pv[i + 1] - (double)pv[i]), e - 1);
    }
    const double u = sigma * sigma + (double)eps;
    return (u == 0.0) ? 0.0f : (float)(1.0 / sqrt(u));
}

// v from another lane by the DPP control CTRL, on both 32-bit halves; lanes
// outside ROW_MASK's rows (or with no source lane) read 0.0.
template <int CTRL, int ROW_MASK = 0xF>
__device__ __forceinline__ double dpp_f64(double v)
{
    const unsigned long long b = __builtin_bit_cast(unsigned long long, v);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)b, CTRL, ROW_MASK, 0xF, false);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(b >> 32), CTRL, ROW_MASK, 0xF, false);
    return __builtin_bit_cast(double, ((unsigned long long)hi << 32) | lo);
}

__device__ __forceinline__ double readlane_f64(double v, int lane)
{
    const unsigned long long b = __builtin_bit_cast(unsigned long long, v);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)b, lane);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(b >> 32), lane);
    return __builtin_bit_cast(double, ((unsigned long long)hi << 32) | lo);
}

// Workgroup barrier that orders LDS accesses only.  The threads of these
// kernels share data through LDS alone, and __syncthreads()' fence would also
// wait for every global load and store in flight, including loads issued
// ahead for later rows and the stores of the row just finished.
__device__ __forceinline__ void lds_barrier()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Sum of one double per lane over a team of TL lanes; every lane of the team
// gets the same bits.  Inside a 16-lane row: DPP quad permutes (lane i^1,
// i^2) and the half-row and row mirrors, each step adding the same two values
// on both lanes.  Across rows: row 15 broadcasts (rows 1 and 3 add row 0's and
// row 2's sum, then rows 2 and 3 add lane 31's) and a read of the total's
// lane.  Multi-wave teams join the per-wave sums through LDS.  No LDS round
// trips inside a wave: the row statistic's latency is part of every row's
// time.
template <int TL>
__device__ __forceinline__ double team_sum(double s, double *red, int tid)
{
    s += dpp_f64<0xB1>(s);  // quad_perm [1,0,3,2]
    s += dpp_f64<0x4E>(s);  // quad_perm [2,3,0,1]
    s += dpp_f64<0x141>(s); // row_half_mirror
    s += dpp_f64<0x140>(s); // row_mirror
    if constexpr (TL >= 32) {
        s += dpp_f64<0x142, 0xA>(s); // row_bcast:15 into rows 1 and 3
        if constexpr (TL == 32) {
            // two teams per wave: rows 0-1 (total in lane 31), rows 2-3 (lane 63)
            const double t0 = readlane_f64(s, 31), t1 = readlane_f64(s, 63);
            s = (tid & 32) ? t1 : t0;
        } else {
            s += dpp_f64<0x143, 0xC>(s); // row_bcast:31 into rows 2 and 3
            s = readlane_f64(s, 63);
        }
    }
    if constexpr (TL > 64) {
        constexpr int NW = TL / 64;
        const int wave = tid >> 6;
        if ((tid & 63) == 0)
            red[wave] = s;
        lds_barrier();
        const int first = (wave / NW) * NW;
        double t = 0.0;
#pragma unroll
        for (int i = 0; i < NW; ++i)
            t += red[first + i];
        s = t;
    }
    return s;
}

// ------------------------------------------------------------------ kernel --

template <int TL>
struct Team {
    static constexpr int BLOCK = TL > 256 ? TL : 256;
    static constexpr int TEAMS = BLOCK / TL; // rows per workgroup
};

// NV: NVFP4 output (else MXFP8).  MXN: MXNorm (else RMSNorm).  GAM: apply
// gamma (RMSNorm only).
// Output formats.  MX*: one E8M0 scale per B-element block and E4M3 (8-bit)
// or E2M1 (4-bit, two per byte) codes; NV4: NVFP4 (16-element blocks, E4M3
// scales times a tensor scale, E2M1 codes).
enum OutFmt : int { MX8_B16, MX8_B32, MX8_B64, MX4_B16, MX4_B32, MX4_B64, NV4_B16 };

template <int F>
struct Fmt {
    static constexpr int B =
        (F == MX8_B16 || F == MX4_B16 || F == NV4_B16) ? 16 : (F == MX8_B32 || F == MX4_B32) ? 32 : 64;
    static constexpr bool NV = F == NV4_B16;
    static constexpr bool FP4 = F >= MX4_B16; // 4-bit codes
    static constexpr int BL = B / 8;          // lanes (16-byte chunks) per block
};

// Buffer resources.  A raw buffer access whose offset is at or past the
// resource's byte count reads zeros (loads) or is dropped (stores) in the
// hardware, so rows past T and chunks past the end of a row need no branch:
// their offsets point past the end.  Each workgroup builds its resources
// over its own rows, which keeps every offset far below 2^31.
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
constexpr uint32_t kOutside = 0x80000000u; // an offset past every resource
// Cache policy of the streaming accesses: each input byte is read once and
// each output byte written once, never read back by the kernel, so both are
// non-temporal; the hint keeps the outputs from displacing the input stream
// in the caches (on MI355X: +8% for the MXFP8 kernels, +1..5% for MXFP4).
constexpr int kBufNT = 2;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void *base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, (int)bytes, 0x00020000);
}

// Chunks j*TL + l (j < CPL) of the team's row into v, zeros outside the
// tensor.  All CPL loads issue back to back: a load under a per-lane branch
// would end its branch with a wait for its own data and leave the wave one
// 16-byte load in flight at a time (measured on MI355X: 5.8 against 6.5 TB/s
// for the same traffic).
template <int TL, int CPL>
__device__ __forceinline__ void load_row(__amdgpu_buffer_rsrc_t xr, uint32_t row_off, int nc, int l,
                                         uint4 (&v)[CPL])
{
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
        const int c = j * TL + l;
        const uint32_t off = c < nc ? row_off + 16u * (uint32_t)c : kOutside;
        const u32x4_t t = __builtin_amdgcn_raw_buffer_load_b128(xr, (int)off, 0, kBufNT);
        v[j] = make_uint4(t.x, t.y, t.z, t.w);
    }
}

// What a kernel computes before the cast: RMSNorm (Alg. 1), MXNorm (Alg. 2),
// or nothing (the plain MX cast of x, or of x * gamma -- the gain-folded weight
// cast MXCast(W gamma) of the MXNormLinear forward, Sec. 3.7).
enum Kind : int { K_RMS = 0, K_MXN = 1, K_CAST = 2, K_MXN_POST = 3 };

// Waves per SIMD the register allocation must allow.  A kernel that keeps
// the row in registers and waits for it once per row hides that wait with
// other waves: 7 per SIMD (72 VGPRs) hold the E8M0 kernels with the row's
// block maxima kept from the statistics pass (at 8 per SIMD those spill; at
// 8 without them, recomputing the maxima in the cast pass, the kernel was 1%
// slower on MI355X); the gain, NVFP4 and multi-wave-team kernels need more
// registers and take what they get.
template <int TL, int F, bool GAM>
constexpr int min_waves()
{
    return (GAM || Fmt<F>::NV || TL > 64) ? 1 : 7;
}

// F: output format.  KIND: see Kind.  GAM: apply gamma (RMSNorm and cast).  Workgroup b handles rows b*TEAMS .. b*TEAMS+TEAMS-1, one per team.
// (A persistent variant that prefetches each team's next row during the
// current one needs about twice the registers; at the resulting occupancy it
// was slower for five of the six MXFP8/NVFP4 kernels on MI355X.)
template <int TL, int CPL, int F, int KIND, bool GAM>
__global__ void __launch_bounds__(Team<TL>::BLOCK) __attribute__((amdgpu_waves_per_eu(min_waves<TL, F, GAM>())))
norm_cast_kernel(Args A)
{
    constexpr bool POST = KIND == K_MXN_POST;
    constexpr bool MXN = KIND == K_MXN || POST; // statistic from the block absmaxes
    constexpr bool CAST = KIND == K_CAST;
    constexpr int BLOCK = Team<TL>::BLOCK;
    constexpr int TEAMS = Team<TL>::TEAMS;
    constexpr bool NV = Fmt<F>::NV;
    constexpr bool FP4 = Fmt<F>::FP4;
    constexpr int BL = Fmt<F>::BL; // lanes (chunks) per scale block
    __shared__ double red[TL > 64 ? BLOCK / 64 : 1];
    // the scale bytes of each row, gathered here and written with wide stores
    constexpr int KMAX = TL * CPL / BL;
    __shared__ __attribute__((aligned(16))) uint8_t sbuf[TEAMS * KMAX];
    // NVFP4: for every finite E4M3 block scale S, den = RN(dec(S) s_g) and
    // its correctly rounded reciprocal -- one IEEE division per entry per
    // workgroup instead of one per block.  A zero reciprocal marks the scales
    // whose blocks take the exact slow path (den = 0 or den < 2^-90).
    __shared__ float2 den_tab[NV ? 128 : 1];
    float six_sg = 0.0f, rcp_six_sg = 0.0f;
    bool six_sg_ok = false;
    if constexpr (NV) {
        if (threadIdx.x < 127) {
            const float den = e4m3_value(threadIdx.x) * A.s_g;
            den_tab[threadIdx.x] = make_float2(den, den >= 0x1p-90f ? 1.0f / den : 0.0f);
        }
        six_sg = A.six_sg;
        rcp_six_sg = A.rcp_six_sg;
        six_sg_ok = six_sg >= 0x1p-90f;
        lds_barrier();
    }

    const int tid = threadIdx.x;
    const int team = tid / TL;
    const int l = tid - team * TL;
    uint8_t *sb = sbuf + team * KMAX;

    uint4 g[GAM ? CPL : 1]; // gamma chunks: the same columns for every row
    if constexpr (GAM) {
        const __amdgpu_buffer_rsrc_t gr = buffer_rsrc(A.gamma, (uint32_t)A.d * 2u);
#pragma unroll
        for (int j = 0; j < CPL; ++j) {
            const int c = j * TL + l;
            const uint32_t off = c < A.nc ? 16u * (uint32_t)c : kOutside;
            const u32x4_t t = __builtin_amdgcn_raw_buffer_load_b128(gr, (int)off, 0, 0);
            g[j] = make_uint4(t.x, t.y, t.z, t.w);
        }
    }

    // chunks per lane this row actually has: the same for every lane, so the
    // loops below skip the unused tail of the register array uniformly
    const int cpl = (A.nc + TL - 1) / TL;
    uint4 v[CPL];
    {
        const int64_t row0 = (int64_t)blockIdx.x * TEAMS; // the workgroup's first row
        const int64_t row = row0 + team;
        const bool row_ok = row < A.T;
        // rows of this workgroup inside the tensor, and the resources over them
        const uint32_t rows = (uint32_t)min((int64_t)TEAMS, A.T - row0);
        const uint32_t dcode = FP4 ? (uint32_t)A.d / 2u : (uint32_t)A.d; // code bytes per row
        const __amdgpu_buffer_rsrc_t xr = buffer_rsrc(A.x + row0 * A.d, rows * (uint32_t)A.d * 2u);
        const __amdgpu_buffer_rsrc_t cr = buffer_rsrc(A.codes + row0 * dcode, rows * dcode);
        load_row<TL, CPL>(xr, (uint32_t)team * (uint32_t)A.d * 2u, A.nc, l, v);
        // where this team's codes start in the store region; chunks past the
        // row's end store nowhere (the hardware drops the access)
        const uint32_t code_row = (uint32_t)team * dcode;

        // ---- pass 1: the row statistic ----
        double s = 0.0;
        uint32_t mb[MXN ? CPL : 1]; // the blocks' absmax patterns, for pass 2
        if constexpr (MXN) {
#pragma unroll
            for (int j = 0; j < CPL; ++j) {
                if (j >= cpl)
                    break;
                const uint32_t m = block_max<BL>(chunk_absmax_bits(v[j]));
                mb[j] = m;
                // every lane of the block adds its term: the sum is BL times
                // the block sum, removed exactly (BL is a power of two) below
                if constexpr (POST) {
                    s += (double)__uint_as_float(pow2_floor_bits(m)); // r(m~)
                } else {
                    const double md = (double)__uint_as_float(m << 16);
                    s += (A.p == 1) ? md : md * md;
                }
            }
        } else if constexpr (!CAST) {
#pragma unroll
            for (int j = 0; j < CPL; ++j) {
                if (j >= cpl)
                    break;
                const uint32_t w[4] = {v[j].x, v[j].y, v[j].z, v[j].w};
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const double a = (double)bf16_lo(w[i]);
                    const double b = (double)bf16_hi(w[i]);
                    s = __builtin_fma(a, a, s);
                    s = __builtin_fma(b, b, s);
                }
            }
        }


        // keep the row as raw bf16 between the passes rather than letting
        // values converted in pass 1 stay live
#pragma unroll
        for (int j = 0; j < CPL; ++j)
            asm volatile("" : "+v"(v[j].x), "+v"(v[j].y), "+v"(v[j].z), "+v"(v[j].w));
        float rho = 1.0f; // the plain cast: t = RN(x * 1) = x
        if constexpr (!CAST) {
            s = team_sum<TL>(s, red, tid);
            if constexpr (MXN)
                s *= 1.0 / BL;
            if constexpr (POST)
                rho = rho_postround((A.K & (A.K - 1)) == 0 ? ldexp(s, -__builtin_ctz((unsigned)A.K))
                                                           : s / (double)A.K,
                                    A.pr_x, A.pr_v, A.eps);
            else
                rho = MXN ? rho_estimate(s, A.K, A.p, A.coef, A.eps) : rho_rms(s, A.d, A.eps);
            if (row_ok && l == 0 && A.rho)
                A.rho[row] = rho;
        }

        // ---- pass 2: block scales and element codes ----
#pragma unroll
        for (int j = 0; j < CPL; ++j) {
            if (j >= cpl)
                break;
            const int c = j * TL + l;
            const uint32_t w[4] = {v[j].x, v[j].y, v[j].z, v[j].w};
            float t[8];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                t[2 * i] = bf16_lo(w[i]) * rho;
                t[2 * i + 1] = bf16_hi(w[i]) * rho;
            }
            if constexpr (GAM) {
                const uint32_t gw[4] = {g[j].x, g[j].y, g[j].z, g[j].w};
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    t[2 * i] = t[2 * i] * bf16_lo(gw[i]);
                    t[2 * i + 1] = t[2 * i + 1] * bf16_hi(gw[i]);
                }
            }
            // block maximum of |t|
            float a;
            if constexpr (MXN) {
                // = max |t| (RN is monotone), from the block maximum kept
                // from pass 1
                a = __uint_as_float(mb[j] << 16) * rho;
            } else {
                // integer max of the magnitude patterns: NaN propagates
                uint32_t m = 0;
#pragma unroll
                for (int k = 0; k < 8; ++k)
                    m = max(m, __float_as_uint(t[k]) & 0x7FFFFFFFu);
                a = __uint_as_float(block_max<BL>(m));
            }

            if constexpr (!NV && !FP4) {
                const uint32_t byte = e8m0_byte<false>(a, A.mode);
                if (A.mode == MX_SCALE_FLOOR) {
                    // |t| <= 448 * 2^e: saturate before the conversion
                    const float lim = __uint_as_float(((byte + 8u) << 23) | 0x600000u);
#pragma unroll
                    for (int k = 0; k < 8; ++k)
                        t[k] = __builtin_amdgcn_fmed3f(t[k], -lim, lim);
                }
                const float scale = __uint_as_float(byte << 23);
                uint32_t lo = e4m3x4_hw(t[0], t[1], t[2], t[3], scale);
                uint32_t hi = e4m3x4_hw(t[4], t[5], t[6], t[7], scale);
                if (__builtin_amdgcn_ballot_w64(byte == 0xFFu)) { // rare: non-finite input
                    if (byte == 0xFFu) {
                        lo = nan_codes_e4m3(w[0], w[1]);
                        hi = nan_codes_e4m3(w[2], w[3]);
                    }
                }
                __builtin_amdgcn_raw_buffer_store_b64(
                    (u32x2_t){lo, hi}, cr, (int)(c < A.nc ? code_row + 8u * (uint32_t)c : kOutside), 0,
                    kBufNT);
                if ((l % BL) == 0) // blocks past K are staged but never stored
                    sb[c / BL] = (uint8_t)byte;
            } else if constexpr (!NV) {
                // MXFP4: E2M1 codes of t / 2^e.  The scaled fp4 conversion
                // divides by the scale operand's power of two, rounds to
                // nearest even and saturates at 6 (checked on the device on all
                // fp32 inputs for scale exponents -127 .. 120), so FLOOR needs
                // no clamp.
                const uint32_t byte = e8m0_byte<true>(a, A.mode);
                const float scale = __uint_as_float(byte << 23);
                uint32_t packed = 0;
                packed = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(packed, t[0], t[1], scale, 0);
                packed = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(packed, t[2], t[3], scale, 1);
                packed = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(packed, t[4], t[5], scale, 2);
                packed = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(packed, t[6], t[7], scale, 3);
                if (__builtin_amdgcn_ballot_w64(byte == 0xFFu)) { // rare: non-finite input
                    if (byte == 0xFFu)
                        packed = 0x77777777u | sign_nibbles(v[j]);
                }
                __builtin_amdgcn_raw_buffer_store_b32(
                    packed, cr, (int)(c < A.nc ? code_row + 4u * (uint32_t)c : kOutside), 0, kBufNT);
                if ((l % BL) == 0)
                    sb[c / BL] = (uint8_t)byte;
            } else {
                uint32_t S, packed = 0;
                if (!(a <= FLT_MAX)) { // NaN or Inf block maximum
                    S = 0x7Fu;
                    packed = 0x77777777u | sign_nibbles(v[j]);
                } else {
                    float q = six_sg_ok ? div_by_recip(a, six_sg, rcp_six_sg) : a / six_sg;
                    if (q != q) // a is finite: a NaN here is an overflowed quotient
                        q = __builtin_inff();
                    // E4M3 code of q >= 0, nearest even, on the conversion
                    // unit; the instruction gives NaN above 464 instead of
                    // saturating, so clamp to 448 first
                    S = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(__builtin_fminf(q, 448.0f),
                                                                  0.0f, 0, false) & 0xFFu;
                    const float2 dr = den_tab[S];
                    const float den = dr.x, r = dr.y;
                    if (r > 0.0f && a * r <= 0x1p100f) {
                        // common case: every quotient is finite and the
                        // Markstein correction is exact.  The negated
                        // quotients are encoded and the sign bits flipped
                        // back, so zero and underflowing quotients keep the
                        // sign of t
                        float vq[8];
#pragma unroll
                        for (int k = 0; k < 8; ++k)
                            vq[k] = neg_div_by_recip(t[k], den, r);
                        packed = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(packed, vq[0], vq[1], 1.0f, 0);
                        packed = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(packed, vq[2], vq[3], 1.0f, 1);
                        packed = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(packed, vq[4], vq[5], 1.0f, 2);
                        packed = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(packed, vq[6], vq[7], 1.0f, 3);
                        packed ^= 0x88888888u;
                    } else if (den == 0.0f) {
#pragma unroll
                        for (int k = 0; k < 8; ++k)
                            packed |= ((__float_as_uint(t[k]) >> 31) << 3) << (4 * k);
                    } else {
#pragma unroll
                        for (int k = 0; k < 8; ++k)
                            packed |= e2m1_code(t[k] / den, t[k]) << (4 * k);
                    }
                }
                __builtin_amdgcn_raw_buffer_store_b32(
                    packed, cr, (int)(c < A.nc ? code_row + 4u * (uint32_t)c : kOutside), 0, kBufNT);
                if ((l & 1) == 0)
                    sb[c >> 1] = (uint8_t)S;
            }
        }

        // ---- the row's K scale bytes: LDS -> one wide store per lane ----
        if constexpr (TL > 64) {
            lds_barrier();
        } else {
            // the team lives in one wave: order its LDS writes before the reads
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        }
        if (A.sw == 16) {
            // K/16 lanes store 16 bytes each; rows past T store nowhere
            const __amdgpu_buffer_rsrc_t sr = buffer_rsrc(A.scales + row0 * A.K, rows * (uint32_t)A.K);
            const bool in = l < A.K / 16;
            const u32x4_t val = *reinterpret_cast<const u32x4_t *>(sb + 16 * (in ? l : 0));
            __builtin_amdgcn_raw_buffer_store_b128(
                val, sr, (int)(in ? (uint32_t)team * (uint32_t)A.K + 16u * (uint32_t)l : kOutside), 0,
                kBufNT);
        } else if (row_ok) {
            uint8_t *dst = A.scales + row * A.K;
            if (A.sw == 4) {
                for (int i = l; i < A.K / 4; i += TL)
                    *reinterpret_cast<uint32_t *>(dst + 4 * i) =
                        *reinterpret_cast<const uint32_t *>(sb + 4 * i);
            } else {
                for (int i = l; i < A.K; i += TL)
                    dst[i] = sb[i];
            }
        }
    }
}

// Workgroups per compute unit the gain-free kernels with one-wave teams run
// best at (each such workgroup puts one wave on each SIMD), per output
// format and kernel; 0 = as many as the registers allow.  Measured on
// MI355X at [32768, 4096]: the 4-bit formats write in small pieces and lose
// 2-5% when more rows are in flight (MXNorm E2M1 57.4 us at 8 per CU, 54.4
// at 4; MXNorm NVFP4 57.9 at 8, 56.6 at 5); E4M3 gains a little at 6 (MXNorm
// 64.3 -> 64.1 us, RMSNorm 65.1 -> 64.3).  RMSNorm NVFP4 runs best at the 7
// its registers allow (59.5 us; 60.1 at 5).  The gain kernels already run
// at 5 (their register count) and are left alone.
template <int F, int KIND>
constexpr int wg_per_cu()
{
    return Fmt<F>::NV ? (KIND == K_RMS ? 0 : 5) : Fmt<F>::FP4 ? 4 : 6;
}

// LDS bytes per compute unit of the current device (160 KiB on gfx950), or
// 0 if the runtime does not say
inline size_t lds_per_cu()
{
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev) !=
            hipSuccess || v <= 0)
        return 0;
    return (size_t)v;
}

// Dynamic LDS that caps the kernel at wg_per_cu<F, KIND>() workgroups per compute
// unit: the workgroup's total LDS is set between a (cap+1)-th and a cap-th of
// the unit's.  The memory is never touched; it only limits occupancy.
template <int TL, int CPL, int F, int KIND, bool GAM>
size_t occupancy_lds()
{
    if constexpr (GAM || TL > 64 || wg_per_cu<F, KIND>() == 0) {
        return 0;
    } else {
        static const size_t dyn = []() -> size_t {
            const size_t per_cu = lds_per_cu();
            hipFuncAttributes fa;
            if (per_cu == 0 ||
                hipFuncGetAttributes(&fa, reinterpret_cast<const void *>(
                                              &norm_cast_kernel<TL, CPL, F, KIND, GAM>)) != hipSuccess)
                return 0;
            const size_t cap = (size_t)wg_per_cu<F, KIND>();
            const size_t lo = per_cu / (cap + 1) + 1024, hi = per_cu / cap;
            const size_t total = (lo + hi) / 2 / 512 * 512;
            return total > fa.sharedSizeBytes && total <= 65536 ? total - fa.sharedSizeBytes : 0;
        }();
        return dyn;
    }
}

template <int TL, int CPL, int F, int KIND, bool GAM>
hipError_t launch_one(const Args &A, hipStream_t stream)
{
    const int64_t blocks = (A.T + Team<TL>::TEAMS - 1) / Team<TL>::TEAMS;
    const size_t dyn_lds = occupancy_lds<TL, CPL, F, KIND, GAM>();
    hipLaunchKernelGGL((norm_cast_kernel<TL, CPL, F, KIND, GAM>), dim3((unsigned)blocks),
                       dim3(Team<TL>::BLOCK), dyn_lds, stream, A);
    return hipGetLastError();
}

template <int F, int KIND, bool GAM>
hipError_t launch_kind(const Args &A, int TL, int CPL, hipStream_t stream)
{
#define MXN_CASE(tl)                                                                     \
    case tl:                                                                             \
        return CPL == 4 ? launch_one<tl, 4, F, KIND, GAM>(A, stream)                     \
                        : launch_one<tl, 8, F, KIND, GAM>(A, stream);
    switch (TL) {
        MXN_CASE(16)
        MXN_CASE(32)
        MXN_CASE(64)
        MXN_CASE(128)
        MXN_CASE(256)
        MXN_CASE(512)
    }
#undef MXN_CASE
    return hipErrorInvalidValue;
}

template <int F>
hipError_t launch_fmt(const Args &A, int kind, int TL, int CPL, hipStream_t stream)
{
    if (kind == K_MXN)
        return launch_kind<F, K_MXN, false>(A, TL, CPL, stream);
    if constexpr (!Fmt<F>::NV) {
        if (kind == K_MXN_POST)
            return launch_kind<F, K_MXN_POST, false>(A, TL, CPL, stream);
    }
    if (kind == K_CAST)
        return A.gamma ? launch_kind<F, K_CAST, true>(A, TL, CPL, stream)
                       : launch_kind<F, K_CAST, false>(A, TL, CPL, stream);
    return A.gamma ? launch_kind<F, K_RMS, true>(A, TL, CPL, stream)
                   : launch_kind<F, K_RMS, false>(A, TL, CPL, stream);
}


// One instantiation per output format, each in its own translation unit.
hipError_t launch_norm_cast(int fmt, const Args &A, int kind, int TL, int CPL, hipStream_t stream);

} // namespace mxk
