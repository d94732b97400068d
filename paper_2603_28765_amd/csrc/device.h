// device.h -- gfx950 device helpers for the adaptive block-scaled formats:
// format traits, E4M3 scale codec, element rounding, Philox4x32-10, the
// 16-point random Hadamard transform and the per-group quantizer.
//
// Every floating-point step is written out explicitly (the library is built
// with -ffp-contract=off, so no FMA appears unless __builtin_fmaf is
// called) because the codes must be bit-identical to the format's
// definition evaluated in binary32.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ifq.h"

namespace ifq {

constexpr int kGroup = 16;

// ------------------------------------------------------------ format traits
// EB/MB: exponent and mantissa widths of the FP element (ExMy, bias
// 2^(EB-1)-1, subnormals, no Inf/NaN).  INT elements are two's complement
// in [-IMAX, IMAX].  KIND says how a group's element type is chosen:
// FP only (NVFP4), adaptive FP/INT by squared error (IF formats, Fig. 3a),
// INT only (NVINT4, Sec. 2) or FP scaled to a maximum of 6 or 4 (4/6,
// Sec. 3).  M is the group target of Eq. 2 and A8 the E4M3 factor of Eq. 1
// (alpha = max|X| / (M * A8)).  c_up = fp32(IMAX / FP_MAX), k_dn =
// fp32(FP_MAX / IMAX) realise the 6/7 method (Sec. 3) and its IF3/IF6
// analogues (Sec. 5.1 footnote); NVINT4 scales straight to IMAX (both 1).
enum FmtKind { kKindFP = 0, kKindAdaptive = 1, kKindInt = 2, kKindFourSix = 3 };

template <int FMT> struct Fmt;
template <> struct Fmt<IFQ_FMT_IF4> {
    static constexpr int BITS = 4, EB = 2, MB = 1, IMAX = 7, KIND = kKindAdaptive, G = 16;
    static constexpr bool ADAPTIVE = true;
    static constexpr float FP_MAX = 6.0f, M = 6.0f, A8 = 448.0f;
};
template <> struct Fmt<IFQ_FMT_NVFP4> {
    static constexpr int BITS = 4, EB = 2, MB = 1, IMAX = 7, KIND = kKindFP, G = 16;
    static constexpr bool ADAPTIVE = false;
    static constexpr float FP_MAX = 6.0f, M = 6.0f, A8 = 448.0f;
};
template <> struct Fmt<IFQ_FMT_IF3> {
    static constexpr int BITS = 3, EB = 2, MB = 0, IMAX = 3, KIND = kKindAdaptive, G = 16;
    static constexpr bool ADAPTIVE = true;
    static constexpr float FP_MAX = 4.0f, M = 4.0f, A8 = 448.0f;
};
template <> struct Fmt<IFQ_FMT_IF6_E2M3> {
    static constexpr int BITS = 6, EB = 2, MB = 3, IMAX = 31, KIND = kKindAdaptive, G = 16;
    static constexpr bool ADAPTIVE = true;
    static constexpr float FP_MAX = 7.5f, M = 7.5f, A8 = 448.0f;
};
template <> struct Fmt<IFQ_FMT_IF6_E3M2> {
    static constexpr int BITS = 6, EB = 3, MB = 2, IMAX = 31, KIND = kKindAdaptive, G = 16;
    static constexpr bool ADAPTIVE = true;
    static constexpr float FP_MAX = 28.0f, M = 28.0f, A8 = 448.0f;
};
template <> struct Fmt<IFQ_FMT_NVINT4> {
    static constexpr int BITS = 4, EB = 2, MB = 1, IMAX = 7, KIND = kKindInt, G = 16;
    static constexpr bool ADAPTIVE = false;
    static constexpr float FP_MAX = 6.0f, M = 7.0f, A8 = 448.0f;
};
template <> struct Fmt<IFQ_FMT_NVFP4_46> {
    static constexpr int BITS = 4, EB = 2, MB = 1, IMAX = 7, KIND = kKindFourSix, G = 16;
    static constexpr bool ADAPTIVE = false;
    static constexpr float FP_MAX = 6.0f, M = 6.0f, A8 = 256.0f;
};

// Block size 8 (Sec. 5.1; Table 6, App. D): the same elements with one scale per 8
// values (G = 8).  A quantizer lane still owns 16 values -- two groups, two
// adjacent scale bytes -- and the code bit stream of 16 values is unchanged.
template <> struct Fmt<IFQ_FMT_IF4_BS8> : Fmt<IFQ_FMT_IF4> { static constexpr int G = 8; };
template <> struct Fmt<IFQ_FMT_IF3_BS8> : Fmt<IFQ_FMT_IF3> { static constexpr int G = 8; };
template <> struct Fmt<IFQ_FMT_NVFP4_BS8> : Fmt<IFQ_FMT_NVFP4> { static constexpr int G = 8; };

// The 16-value format whose element arithmetic a format uses (itself, or
// the block-16 counterpart of a block-8 format).
template <int FMT> struct Base { static constexpr int F = FMT; };
template <> struct Base<IFQ_FMT_IF4_BS8> { static constexpr int F = IFQ_FMT_IF4; };
template <> struct Base<IFQ_FMT_IF3_BS8> { static constexpr int F = IFQ_FMT_IF3; };
template <> struct Base<IFQ_FMT_NVFP4_BS8> { static constexpr int F = IFQ_FMT_NVFP4; };

template <int FMT> struct FmtDerived {
    using F = Fmt<FMT>;
    static constexpr int BIAS = (1 << (F::EB - 1)) - 1;
    static constexpr float C_UP = F::KIND == kKindInt ? 1.0f : (float)F::IMAX / F::FP_MAX;
    static constexpr float K_DN = F::KIND == kKindInt ? 1.0f : F::FP_MAX / (float)F::IMAX;
    static constexpr uint32_t CODE_MASK = (1u << F::BITS) - 1u;
    static constexpr uint32_t SIGN_BIT = 1u << (F::BITS - 1);
};

// Kernel-side quantizer options (the `qflags` argument of the quantize
// kernels): with SR, decide the type / scaling on round-to-nearest
// candidates; the 16/17 margin of Sec. 4.1 (needed for 4/6's second target).
constexpr int kQSrRtnType = 1, kQMargin = 2;
// 4 and 4 * 16/17 rounded once to fp32: the second target of 4/6.
constexpr float kFourTarget = 4.0f;
constexpr float kFourTargetMargin = (float)(4.0 * 16.0 / 17.0);

// ------------------------------------------------------------- bit helpers
__device__ __forceinline__ float bf16lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f)
{
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// ------------------------------------------------------------ E4M3 scales
// The encoder: nearest E4M3 code to x >= 0, ties to
// even, saturating at 448 (0x7E); a NaN quotient (0 / 0) also gives 0x7E.
// gfx950's fp32 -> OCP E4M3 conversion rounds to nearest even with
// subnormal codes (step 2^-9); an exhaustive comparison over every fp32 in
// [0, 464] found it equal to that rule, so after clamping to 448 it is the
// whole encoder.

__device__ __forceinline__ uint32_t e4m3_encode(float x)
{
    return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(fminf(x, 448.0f), 0.0f, 0, false) & 0xFFu;
}

// Value of E4M3 code c (bits 0-6; 0x7F never produced): the hardware decode,
// exact for every finite code.
__device__ __forceinline__ float e4m3_value(uint32_t c)
{
    return __builtin_amdgcn_cvt_f32_fp8((int)(c & 0x7Fu), 0);
}

// 1/s rounded to nearest for a normal s > 0: the hardware reciprocal
// estimate with one fma correction.  An exhaustive comparison over every
// normal fp32 found it equal to the correctly rounded quotient up to
// s = 2^126; above, where 1/s is subnormal, the correctly rounded division
// is used.  (Three operations instead of the division's nine.)
__device__ __forceinline__ float recip_rn_normal(float s)
{
    const float r0 = __builtin_amdgcn_rcpf(s);
    const float e = __builtin_fmaf(-s, r0, 1.0f);
    return __builtin_fmaf(e, r0, r0);
}

__device__ __forceinline__ float recip_rn(float s)
{
    if (s > 0x1p126f) return 1.0f / s;
    return recip_rn_normal(s);
}

// A divisor shared by a launch's groups -- denom = fp32(alpha * M) of Eq. 2
// -- with its correctly rounded reciprocal, so that a group's quotient
// amax / denom costs four operations instead of a division's eleven:
// q0 = amax * r, e = amax - denom * q0 (exact, one fma), q = q0 + e * r
// rounded once.  This is Markstein's correction, which gives the correctly
// rounded quotient when r = RN(1/denom), denom and r are normal and the
// residual e does not underflow -- guaranteed here by amax >= 2^-100 (the
// residual is then far above 2^-126); checked against the division for 1024
// divisor significands (all-ones tails, neighbours of powers of two,
// random) times every dividend significand.  A quotient that overflows
// becomes NaN or inf and one that underflows is below 2^-126; the E4M3
// encoder maps both as it maps the true quotient (to 0x7E after its clamp,
// and to code 0).  A wavefront uses the correction only when every lane
// qualifies, else the division: a wave-uniform branch (all lanes share
// alpha), which also keeps the compiler from interleaving the code before
// and after it and lowers register pressure.  `small_s`: every group scale
// s = alpha * Delta <= alpha * 448 is at most 2^126, so its reciprocal needs
// no range check.
struct Div {
    float d, r;
    bool fast, small_s;
};

__device__ __forceinline__ Div make_div(float alpha, float d)
{
    Div x;
    x.d = d;
    x.fast = d >= 0x1p-125f && d <= 0x1p125f;
    x.small_s = __all(alpha * 448.0f <= 0x1p126f);
    x.r = x.fast ? recip_rn_normal(d) : 0.0f;
    return x;
}

// min(a / x.d, 448): the encoder's clamp is applied on each path, where the
// compiler sees a canonical quotient and needs no NaN quieting before the
// minimum (the empty asm statements keep it from merging the two minima
// after the branch).
__device__ __forceinline__ float div_rn_clamp448(float a, const Div& x)
{
    float q;
    if (__builtin_expect(__all(x.fast && a >= 0x1p-100f), 1)) {
        const float q0 = a * x.r;
        const float e = __builtin_fmaf(-x.d, q0, a);
        q = fminf(__builtin_fmaf(e, x.r, q0), 448.0f);
        asm volatile("; markstein" : "+v"(q));
    } else {
        q = fminf(a / x.d, 448.0f);
        asm volatile("; division" : "+v"(q));
    }
    return q;
}

// 1 / s for a group scale s = alpha * Delta >= 2^-126.  MK: with the
// wave-uniform range test of x (see Div); else with the per-lane test.
template <bool MK>
__device__ __forceinline__ float recip_scale(float s, const Div& x)
{
    if constexpr (MK) {
        if (__builtin_expect(x.small_s, 1)) return recip_rn_normal(s);
    }
    return recip_rn(s);
}

// Group scale of Eq. 2: the E4M3 code of amax / denom and its value Delta.
// MK: the quotient by Markstein's correction (the stochastic-rounding
// quantizers, where the wave-uniform branch also lowers register pressure
// enough for a third wavefront per SIMD); else by the division.  In the
// first form the converter's second source (0) encodes to byte 0 and the
// untouched bytes are zero, so the code needs no mask.
template <bool MK>
__device__ __forceinline__ uint32_t group_scale(float amax, const Div& denom, float& delta)
{
    if constexpr (MK) {
        const uint32_t code =
            (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(div_rn_clamp448(amax, denom), 0.0f, 0, false);
        delta = __builtin_amdgcn_cvt_f32_fp8((int)code, 0);
        return code;
    } else {
        const uint32_t code = e4m3_encode(amax / denom.d);
        delta = e4m3_value(code);
        return code;
    }
}

// --------------------------------------------------------- Philox4x32-10
// Salmon et al., SC'11.
__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1)
{
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        if (r) {
            k0 += 0x9E3779B9u;
            k1 += 0xBB67AE85u;
        }
        // one 32 x 32 -> 64-bit product per multiplier (v_mad_u64_u32), and
        // each three-way exclusive or as one gfx950 v_bitop3 (truth table 0x96)
        const uint64_t p0 = (uint64_t)0xD2511F53u * c.x, p1 = (uint64_t)0xCD9E8D57u * c.z;
        c = make_uint4(__builtin_amdgcn_bitop3_b32((uint32_t)(p1 >> 32), c.y, k0, 0x96), (uint32_t)p1,
                       __builtin_amdgcn_bitop3_b32((uint32_t)(p0 >> 32), c.w, k1, 0x96), (uint32_t)p0);
    }
    return c;
}

// 8 words = 16 draws of 16 bits for group `gi`; draw j = half (j&1) of word j>>1.
__device__ __forceinline__ void sr_words(uint64_t seed, uint64_t gi, uint32_t (&w)[8])
{
    uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
    uint4 a = philox4x32_10(make_uint4((uint32_t)gi, (uint32_t)(gi >> 32), 0u, 0u), k0, k1);
    uint4 b = philox4x32_10(make_uint4((uint32_t)gi, (uint32_t)(gi >> 32), 1u, 0u), k0, k1);
    w[0] = a.x; w[1] = a.y; w[2] = a.z; w[3] = a.w;
    w[4] = b.x; w[5] = b.y; w[6] = b.z; w[7] = b.w;
}

// The first Philox block of group gi's counter (8 draws: a group of 8).
__device__ __forceinline__ void sr_words_first(uint64_t seed, uint64_t gi, uint32_t (&w)[8])
{
    uint4 a = philox4x32_10(make_uint4((uint32_t)gi, (uint32_t)(gi >> 32), 0u, 0u), (uint32_t)seed,
                            (uint32_t)(seed >> 32));
    w[0] = a.x; w[1] = a.y; w[2] = a.z; w[3] = a.w;
    w[4] = 0u; w[5] = 0u; w[6] = 0u; w[7] = 0u;
}

__device__ __forceinline__ float sr_uniform(const uint32_t (&w)[8], int j)
{
    uint32_t h = (w[j >> 1] >> (16 * (j & 1))) & 0xFFFFu;
    return (float)h * (1.0f / 65536.0f);
}

// Stochastic rounding of t >= 0 to an integer with the draw u = h / 2^16:
// floor(t) + 1 iff u < t - floor(t), which is ceil(t - u) of the exact
// values.  The subtraction is exact wherever the result depends on it: for
// t in [2^k, 2^(k+1)) with 0 <= k <= 7, t is a multiple of 2^(k-23) and u of
// 2^-16, so t - u is a multiple of 2^(k-23) below 2^(k+1) (24 bits); for
// t < 1, ceil is 0 or 1 and only the sign of t - u matters, which rounding
// keeps (t - u is a multiple of 2^-149 and above -1).  The result may be -0
// (t - u in (-1, 0)); callers use its magnitude.
__device__ __forceinline__ float sr_ceil(float t, float u)
{
    return __builtin_ceilf(t - u);
}

// The 16-bit draw h of element j as a float (exact), and sr_ceil with u =
// h * 2^-16 taken inside one fma: h * 2^-16 is exact, so the fma's single
// rounding of t - h * 2^-16 is the rounding of t - u that sr_ceil takes.
__device__ __forceinline__ float sr_draw(const uint32_t (&w)[8], int j)
{
    return (float)((w[j >> 1] >> (16 * (j & 1))) & 0xFFFFu);
}
__device__ __forceinline__ float sr_ceil_h(float t, float h)
{
    return __builtin_ceilf(__builtin_fmaf(h, -0x1p-16f, t));
}

// |m| with the sign of x (one bit-field insert)
__device__ __forceinline__ float with_sign_of(float m, float x)
{
    return __uint_as_float((__float_as_uint(m) & 0x7FFFFFFFu) | (__float_as_uint(x) & 0x80000000u));
}

// --------------------------------------------------------------- RHT-16
// The butterflies of the 16-point Hadamard transform, Sylvester order,
// strides 1, 2, 4, 8 (no signs, no scale).
__device__ __forceinline__ void hadamard16(float (&v)[kGroup])
{
#pragma unroll
    for (int h = 1; h < kGroup; h <<= 1) {
#pragma unroll
        for (int i = 0; i < kGroup; ++i) {
            if (i & h) continue;
            float a = v[i], b = v[i + h];
            v[i] = a + b;
            v[i + h] = a - b;
        }
    }
}

// v <- (1/4) H16 diag(s) v
__device__ __forceinline__ void rht16(float (&v)[kGroup], uint32_t signs)
{
#pragma unroll
    for (int j = 0; j < kGroup; ++j)
        v[j] = __uint_as_float(__float_as_uint(v[j]) ^ (((signs >> j) & 1u) << 31));
    hadamard16(v);
#pragma unroll
    for (int j = 0; j < kGroup; ++j) v[j] = v[j] * 0.25f;
}

// The signs of elements 2d and 2d + 1 as the sign bits (15, 31) of a dword
// holding them as a bf16 pair: one exclusive or flips both before unpacking.
__device__ __forceinline__ uint32_t rht_pair_mask(uint32_t signs, int d)
{
    return (((signs >> (2 * d)) & 1u) << 15) | (((signs >> (2 * d + 1)) & 1u) << 31);
}

// For bf16 inputs every value the butterflies produce is a multiple of 2^-133
// (the bf16 quantum; a rounded sum is a multiple of its ulp, which is at
// least 2^-133 wherever rounding happens), so H diag(s) v / 4 is exact: a
// maximum of |H diag(s) v| times 1/4 is the maximum of the transformed
// values.

// ---------------------------------------------------- FP element rounding
// Magnitude of non-negative FP code `idx` (both forms computed and selected:
// a branch here diverges per element).
template <int FMT> __device__ __forceinline__ float fp_magnitude(uint32_t idx)
{
    using F = Fmt<FMT>;
    constexpr int BIAS = FmtDerived<FMT>::BIAS;
    const uint32_t E = idx >> F::MB, M = idx & ((1u << F::MB) - 1u);
    const float sub = (float)M * __uint_as_float((uint32_t)(127 + 1 - BIAS - F::MB) << 23);
    const float nor = __uint_as_float(((E - BIAS + 127u) << 23) | (M << (23 - F::MB)));
    return E ? nor : sub;
}

// Nearest FP code index to m >= 0 (ties to the even code), saturating.
template <int FMT> __device__ __forceinline__ uint32_t fp_rtn_index(float m)
{
    using F = Fmt<FMT>;
    if constexpr (F::MB == 1 && F::EB == 2) {
        // E2M1 midpoints; ">=" where the upper neighbour has the even code
        return (uint32_t)(m > 0.25f) + (uint32_t)(m >= 0.75f) + (uint32_t)(m > 1.25f) +
               (uint32_t)(m >= 1.75f) + (uint32_t)(m > 2.5f) + (uint32_t)(m >= 3.5f) +
               (uint32_t)(m > 5.0f);
    } else if constexpr (F::MB == 0) {
        // E2M0 (0, 1, 2, 4): with no mantissa bit the even code decides ties
        return (uint32_t)(m > 0.5f) + (uint32_t)(m >= 1.5f) + (uint32_t)(m > 3.0f);
    } else {
        // ExMy with MB >= 1: round m to a multiple of the local quantum; the
        // parity of that multiple is the parity of the code.
        constexpr int BIAS = FmtDerived<FMT>::BIAS;
        m = fminf(m, F::FP_MAX);
        int e = (int)((__float_as_uint(m) >> 23) & 0xFFu) - 127;
        int ee = e > 1 - BIAS ? e : 1 - BIAS;
        float inv_u = __uint_as_float((uint32_t)(127 - (ee - F::MB)) << 23);
        float r = __builtin_rintf(m * inv_u);
        return (uint32_t)(((ee + BIAS) << F::MB) + (int)r - (1 << F::MB));
    }
}

// Stochastic rounding of m >= 0 between its grid neighbours lo <= m < hi:
// up iff u * (hi - lo) < m - lo.
template <int FMT> __device__ __forceinline__ uint32_t fp_sr_index(float m, float u)
{
    using F = Fmt<FMT>;
    constexpr int BIAS = FmtDerived<FMT>::BIAS;
    m = fminf(m, F::FP_MAX);
    int e = (int)((__float_as_uint(m) >> 23) & 0xFFu) - 127;
    int ee = e > 1 - BIAS ? e : 1 - BIAS;
    // m / q for the grid step q = 2^(ee - MB): exact, below 2^(MB + 1)
    float inv_q = __uint_as_float((uint32_t)(127 - (ee - F::MB)) << 23);
    int r = (int)sr_ceil(m * inv_q, u);
    return (uint32_t)(((ee + BIAS) << F::MB) + r - (1 << F::MB));
}

// ---------------------------------------------------- group quantizer
// One group of 16 (already transformed) values under tensor scale alpha.
// denom = fp32(alpha * M) with M = M_FP (or M_FP*16/17).  Writes the 16 codes
// (low bits of each byte) and returns the scale byte.  Fig. 3a: Delta, the FP
// candidate, the INT candidate scaled by c_up, and INT iff its error is
// strictly smaller.  Errors are sums of squares in x-bar units, accumulated
// in element order with fused multiply-adds.  RTN_TYPE (with SR): the type is
// decided on the round-to-nearest candidates' errors and the stored codes
// are the stochastic candidate of that type (the App. B alternative).
template <int FMT, bool SR, bool RTN_TYPE = false, int N = kGroup>
__device__ __forceinline__ uint32_t quantize_group(const float (&v)[N], float alpha,
                                                   const Div& denom, const uint32_t (&w)[8],
                                                   uint32_t (&code)[N])
{
    using F = Fmt<FMT>;
    using D = FmtDerived<FMT>;
    float amax = 0.0f;
#pragma unroll
    for (int j = 0; j < N; ++j) amax = fmaxf(amax, fabsf(v[j]));
    float delta;
    uint32_t dcode = group_scale<SR>(amax, denom, delta);
    float s = alpha * delta;
    if (!(s >= 1.17549435e-38f)) {
#pragma unroll
        for (int j = 0; j < N; ++j) code[j] = 0;
        return 0;
    }
    float inv = recip_scale<SR>(s, denom);

    float ef = 0.0f, ei = 0.0f;
    float rf = 0.0f, ri = 0.0f;  // RTN errors (RTN_TYPE only)
    uint32_t cf[N], ci[N];
#pragma unroll
    for (int j = 0; j < N; ++j) {
        float xb = v[j] * inv;
        if constexpr (SR && RTN_TYPE && F::ADAPTIVE) {
            const float m0 = fabsf(xb);
            const uint32_t n0 = __float_as_uint(xb) >> 31;
            const float q0 = __uint_as_float(__float_as_uint(fp_magnitude<FMT>(fp_rtn_index<FMT>(m0))) | (n0 << 31));
            const float d0 = q0 - xb;
            rf = __builtin_fmaf(d0, d0, rf);
            const float xc = __builtin_amdgcn_fmed3f(xb, -F::FP_MAX, F::FP_MAX);
            const float r0 = __builtin_fmaf(xc, D::C_UP, 12582912.0f) - 12582912.0f;
            const float e0 = __builtin_fmaf(r0, D::K_DN, -xb);
            ri = __builtin_fmaf(e0, e0, ri);
        }
        float m = fabsf(xb);
        uint32_t neg = __float_as_uint(xb) >> 31;
        // FP candidate
        uint32_t idx;
        if constexpr (SR)
            idx = fp_sr_index<FMT>(m, sr_uniform(w, j));
        else
            idx = fp_rtn_index<FMT>(m);
        cf[j] = (neg ? D::SIGN_BIT : 0u) | idx;
        float q = __uint_as_float(__float_as_uint(fp_magnitude<FMT>(idx)) | (neg << 31));
        float d = q - xb;
        ef = __builtin_fmaf(d, d, ef);
        if constexpr (F::ADAPTIVE) {
            // INT candidate
            float r;
            if constexpr (SR) {
                float y = xb * D::C_UP;
                r = with_sign_of(fminf(sr_ceil(fabsf(y), sr_uniform(w, j)), (float)F::IMAX), y);
            } else {
                float xc = __builtin_amdgcn_fmed3f(xb, -F::FP_MAX, F::FP_MAX);
                float t = __builtin_fmaf(xc, D::C_UP, 12582912.0f);  // rint(xc*c_up) + 1.5*2^23
                r = t - 12582912.0f;
            }
            ci[j] = (uint32_t)(int)r & D::CODE_MASK;
            float di = __builtin_fmaf(r, D::K_DN, -xb);
            ei = __builtin_fmaf(di, di, ei);
        }
    }
    bool use_int;
    if constexpr (SR && RTN_TYPE)
        use_int = F::ADAPTIVE && (ri < rf);
    else
        use_int = F::ADAPTIVE && (ei < ef);
#pragma unroll
    for (int j = 0; j < N; ++j) code[j] = use_int ? ci[j] : cf[j];
    return dcode | (use_int ? 0x80u : 0u);
}

// ------------------------------------------- fast E2M1 group quantizer
// The E2M1 round-to-nearest candidate of 16 scaled values through the
// gfx950 converter v_cvt_scalef32_pk_fp4_f32 (scale 1.0): round to nearest
// even onto E2M1, saturating at 6, sign kept (a negative value that rounds to
// zero gives code 0x8) -- identical to the nearest-even rule over every fp32
// input -- and v_cvt_scalef32_pk_f32_fp4 to read the candidate back.  The
// codes come out packed (element 2i in the low nibble of byte i); returns
// sum_j (q_j - x_j)^2 accumulated in element order with fused multiply-adds.
__device__ __forceinline__ float e2m1_candidate(const float (&xb)[kGroup], uint32_t& f0, uint32_t& f1)
{
    f0 = 0;
    f1 = 0;
    f0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(f0, xb[0], xb[1], 1.0f, 0);
    f0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(f0, xb[2], xb[3], 1.0f, 1);
    f0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(f0, xb[4], xb[5], 1.0f, 2);
    f0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(f0, xb[6], xb[7], 1.0f, 3);
    f1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(f1, xb[8], xb[9], 1.0f, 0);
    f1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(f1, xb[10], xb[11], 1.0f, 1);
    f1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(f1, xb[12], xb[13], 1.0f, 2);
    f1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(f1, xb[14], xb[15], 1.0f, 3);
    float q[kGroup];
    {
        typedef float f2 __attribute__((ext_vector_type(2)));
        f2 t;
        t = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(f0, 1.0f, 0); q[0] = t[0]; q[1] = t[1];
        t = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(f0, 1.0f, 1); q[2] = t[0]; q[3] = t[1];
        t = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(f0, 1.0f, 2); q[4] = t[0]; q[5] = t[1];
        t = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(f0, 1.0f, 3); q[6] = t[0]; q[7] = t[1];
        t = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(f1, 1.0f, 0); q[8] = t[0]; q[9] = t[1];
        t = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(f1, 1.0f, 1); q[10] = t[0]; q[11] = t[1];
        t = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(f1, 1.0f, 2); q[12] = t[0]; q[13] = t[1];
        t = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(f1, 1.0f, 3); q[14] = t[0]; q[15] = t[1];
    }
    float ef = 0.0f;
#pragma unroll
    for (int j = 0; j < kGroup; ++j) {
        const float d = q[j] - xb[j];
        ef = __builtin_fmaf(d, d, ef);
    }
    return ef;
}

// Packed INT4 codes from 16 floats t_j = r_j + 1.5 * 2^23 (r_j integral,
// |r_j| <= 8): the low nibble of t_j's bit pattern is r_j in two's
// complement.  Even elements -> low nibbles, odd -> high nibbles.
__device__ __forceinline__ void pack_int4_biased(const uint32_t (&tb)[kGroup], uint32_t& i0, uint32_t& i1)
{
    const uint32_t e0 = __builtin_amdgcn_perm(tb[2], tb[0], 0x0C0C0400u) |
                        __builtin_amdgcn_perm(tb[6], tb[4], 0x04000C0Cu);
    const uint32_t o0 = __builtin_amdgcn_perm(tb[3], tb[1], 0x0C0C0400u) |
                        __builtin_amdgcn_perm(tb[7], tb[5], 0x04000C0Cu);
    const uint32_t e1 = __builtin_amdgcn_perm(tb[10], tb[8], 0x0C0C0400u) |
                        __builtin_amdgcn_perm(tb[14], tb[12], 0x04000C0Cu);
    const uint32_t o1 = __builtin_amdgcn_perm(tb[11], tb[9], 0x0C0C0400u) |
                        __builtin_amdgcn_perm(tb[15], tb[13], 0x04000C0Cu);
    i0 = (e0 & 0x0F0F0F0Fu) | ((o0 << 4) & 0xF0F0F0F0u);
    i1 = (e1 & 0x0F0F0F0Fu) | ((o1 << 4) & 0xF0F0F0F0u);
}

__device__ __forceinline__ float group_amax(const float (&v)[kGroup])
{
    float amax = 0.0f;
#pragma unroll
    for (int j = 0; j < kGroup; ++j) amax = fmaxf(amax, fabsf(v[j]));
    return amax;
}

// IF4 / NVFP4 with round-to-nearest.  Same arithmetic as quantize_group,
// with the FP candidate from e2m1_candidate.
template <bool ADAPTIVE>
__device__ __forceinline__ uint32_t quantize_group_e2m1(const float (&v)[kGroup], float alpha,
                                                        const Div& denom, uint2& packed)
{
    constexpr float C_UP = 7.0f / 6.0f, K_DN = 6.0f / 7.0f;
    const float amax = group_amax(v);
    float delta;
    const uint32_t dcode = group_scale<false>(amax, denom, delta);
    const float s = alpha * delta;
    if (!(s >= 1.17549435e-38f)) {
        packed = make_uint2(0, 0);
        return 0;
    }
    const float inv = recip_scale<false>(s, denom);
    float xb[kGroup];
#pragma unroll
    for (int j = 0; j < kGroup; ++j) xb[j] = v[j] * inv;

    uint32_t f0, f1;
    const float ef = e2m1_candidate(xb, f0, f1);
    if constexpr (!ADAPTIVE) {
        packed = make_uint2(f0, f1);
        return dcode;
    }
    // INT candidate: rint(clamp(x, -6, 6) * 7/6) in one rounding (1.5 * 2^23
    // bias); the low nibble of the biased float is the two's-complement code.
    float ei = 0.0f;
    uint32_t tb[kGroup];
#pragma unroll
    for (int j = 0; j < kGroup; ++j) {
        const float xc = __builtin_amdgcn_fmed3f(xb[j], -6.0f, 6.0f);
        const float t = __builtin_fmaf(xc, C_UP, 12582912.0f);
        tb[j] = __float_as_uint(t);
        const float r = t - 12582912.0f;
        const float d = __builtin_fmaf(r, K_DN, -xb[j]);
        ei = __builtin_fmaf(d, d, ei);
    }
    uint32_t i0, i1;
    pack_int4_biased(tb, i0, i1);
    const bool use_int = ei < ef;
    packed = use_int ? make_uint2(i0, i1) : make_uint2(f0, f1);
    return dcode | (use_int ? 0x80u : 0u);
}

// Block size 8 (IF4-BS8, NVFP4-BS8) with round-to-nearest: the arithmetic
// of quantize_group over one block of 8 values with the candidates of
// quantize_group_e2m1 (FP from the E2M1 converter, INT by the biased
// rounding); returns the scale byte and the block's 8 codes in one word
// (code j in nibble j).
template <bool ADAPTIVE>
__device__ __forceinline__ uint32_t quantize_block8_e2m1(const float (&v)[8], float alpha, const Div& denom,
                                                         uint32_t& word)
{
    constexpr float C_UP = 7.0f / 6.0f, K_DN = 6.0f / 7.0f;
    float amax = 0.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j) amax = fmaxf(amax, fabsf(v[j]));
    float delta;
    const uint32_t dcode = group_scale<false>(amax, denom, delta);
    const float s = alpha * delta;
    if (!(s >= 1.17549435e-38f)) {
        word = 0;
        return 0;
    }
    const float inv = recip_scale<false>(s, denom);
    float xb[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) xb[j] = v[j] * inv;
    uint32_t f = 0;
    f = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(f, xb[0], xb[1], 1.0f, 0);
    f = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(f, xb[2], xb[3], 1.0f, 1);
    f = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(f, xb[4], xb[5], 1.0f, 2);
    f = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(f, xb[6], xb[7], 1.0f, 3);
    if constexpr (!ADAPTIVE) {
        word = f;
        return dcode;
    }
    float q[8];
    {
        typedef float f2 __attribute__((ext_vector_type(2)));
        f2 t;
        t = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(f, 1.0f, 0); q[0] = t[0]; q[1] = t[1];
        t = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(f, 1.0f, 1); q[2] = t[0]; q[3] = t[1];
        t = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(f, 1.0f, 2); q[4] = t[0]; q[5] = t[1];
        t = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(f, 1.0f, 3); q[6] = t[0]; q[7] = t[1];
    }
    float ef = 0.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const float d = q[j] - xb[j];
        ef = __builtin_fmaf(d, d, ef);
    }
    float ei = 0.0f;
    uint32_t tb[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const float xc = __builtin_amdgcn_fmed3f(xb[j], -6.0f, 6.0f);
        const float t = __builtin_fmaf(xc, C_UP, 12582912.0f);
        tb[j] = __float_as_uint(t);
        const float d = __builtin_fmaf(t - 12582912.0f, K_DN, -xb[j]);
        ei = __builtin_fmaf(d, d, ei);
    }
    const uint32_t e = __builtin_amdgcn_perm(tb[2], tb[0], 0x0C0C0400u) |
                       __builtin_amdgcn_perm(tb[6], tb[4], 0x04000C0Cu);
    const uint32_t o = __builtin_amdgcn_perm(tb[3], tb[1], 0x0C0C0400u) |
                       __builtin_amdgcn_perm(tb[7], tb[5], 0x04000C0Cu);
    const uint32_t ic = (e & 0x0F0F0F0Fu) | ((o << 4) & 0xF0F0F0F0u);
    const bool use_int = ei < ef;
    word = use_int ? ic : f;
    return dcode | (use_int ? 0x80u : 0u);
}

// IF3 (and IF3-BS8 per block of 8) with round-to-nearest: the arithmetic of
// quantize_group with fewer steps.  The E2M0 candidate comes straight from
// the three midpoint comparisons as its value q in {0, 1, 2, 4} (ties to the
// even code: 0.5 -> 0, 1.5 -> 2, 3 -> 2), its code index is the frexp
// exponent of q (0, 1, 2, 3), and its error uses q - |x-bar| (the signed
// difference negated exactly); the INT3 code is the low three bits of the
// biased float of the rounded value.  Codes come out one per element.
template <int N>
__device__ __forceinline__ uint32_t quantize_group_e2m0(const float (&v)[N], float alpha, const Div& denom,
                                                        uint32_t (&code)[N])
{
    constexpr float C_UP = 3.0f / 4.0f, K_DN = 4.0f / 3.0f;
    float amax = 0.0f;
#pragma unroll
    for (int j = 0; j < N; ++j) amax = fmaxf(amax, fabsf(v[j]));
    float delta;
    const uint32_t dcode = group_scale<false>(amax, denom, delta);
    const float s = alpha * delta;
    if (!(s >= 1.17549435e-38f)) {
#pragma unroll
        for (int j = 0; j < N; ++j) code[j] = 0;
        return 0;
    }
    const float inv = recip_scale<false>(s, denom);
    float ef = 0.0f, ei = 0.0f;
    uint32_t cf[N], ci[N];
#pragma unroll
    for (int j = 0; j < N; ++j) {
        const float xb = v[j] * inv;
        const float m = fabsf(xb);
        float q = m > 0.5f ? 1.0f : 0.0f;
        q = m >= 1.5f ? 2.0f : q;
        q = m > 3.0f ? 4.0f : q;
        cf[j] = ((__float_as_uint(xb) >> 29) & 4u) | (uint32_t)__builtin_amdgcn_frexp_expf(q);
        const float d = q - m;
        ef = __builtin_fmaf(d, d, ef);
        const float xc = __builtin_amdgcn_fmed3f(xb, -4.0f, 4.0f);
        const float t = __builtin_fmaf(xc, C_UP, 12582912.0f);  // rint(xc * 3/4) + 1.5 * 2^23
        ci[j] = __float_as_uint(t) & 7u;
        const float di = __builtin_fmaf(t - 12582912.0f, K_DN, -xb);
        ei = __builtin_fmaf(di, di, ei);
    }
    const bool use_int = ei < ef;
#pragma unroll
    for (int j = 0; j < N; ++j) code[j] = use_int ? ci[j] : cf[j];
    return dcode | (use_int ? 0x80u : 0u);
}

// ------------------------------------------------------------ NVINT4
// INT4 elements scaled straight to 7 (Sec. 2, Table 1): Delta =
// E4M3(max|X_g| / (alpha * 7)), q = the nearest integer to x-bar clamped to
// [-7, 7] (ties to even), or with SR up iff u < |x-bar| - floor(|x-bar|)
// (clamped to 7).  Scale bit 7 stays clear.  Codes come out packed.
template <bool SR>
__device__ __forceinline__ uint32_t quantize_group_int4(const float (&v)[kGroup], float alpha,
                                                        const Div& denom, const uint32_t (&w)[8],
                                                        uint2& packed)
{
    const float amax = group_amax(v);
    float delta;
    const uint32_t dcode = group_scale<SR>(amax, denom, delta);
    const float s = alpha * delta;
    if (!(s >= 1.17549435e-38f)) {
        packed = make_uint2(0, 0);
        return 0;
    }
    const float inv = recip_scale<SR>(s, denom);
    uint32_t tb[kGroup];
#pragma unroll
    for (int j = 0; j < kGroup; ++j) {
        const float xb = v[j] * inv;
        float t;
        if constexpr (SR) {
            const float rr = fminf(sr_ceil(fabsf(xb), sr_uniform(w, j)), 7.0f);
            t = with_sign_of(rr, xb) + 12582912.0f;  // exact: an integer
        } else {
            t = __builtin_amdgcn_fmed3f(xb, -7.0f, 7.0f) + 12582912.0f;  // rint, ties to even
        }
        tb[j] = __float_as_uint(t);
    }
    uint32_t i0, i1;
    pack_int4_biased(tb, i0, i1);
    packed = make_uint2(i0, i1);
    return dcode;
}

// ------------------------------------------------------------ 4/6
// NVFP4 with Four Over Six (Sec. 3): the group is scaled to a maximum of 6
// (denom6 = alpha * M) and of 4 (denom4 = alpha * 4, both with the 16/17
// margin when it is on), rounded onto E2M1 each time, and the scaling with
// the smaller Delta_t^2 * sum_j (q_j - x-bar_j)^2 (the dequantized squared
// error over alpha^2) is kept; ties keep 6.  Delta_4 >= Delta_6: when
// alpha * Delta_4 is below FLT_MIN the group stores zeros, when only
// alpha * Delta_6 is, the scaling to 4 is kept.
//
// FP candidate of one scaling with optional SR: codes and the error sum of
// the stored candidate, plus (RTN_ERR) the error of the round-to-nearest one.
template <bool SR, bool RTN_ERR>
__device__ __forceinline__ void e2m1_candidate_sr(const float (&v)[kGroup], float inv,
                                                  const uint32_t (&w)[8], uint32_t (&code)[kGroup],
                                                  float& err, float& err_rtn)
{
    err = 0.0f;
    err_rtn = 0.0f;
#pragma unroll
    for (int j = 0; j < kGroup; ++j) {
        const float xb = v[j] * inv;
        const float m = fabsf(xb);
        const uint32_t neg = __float_as_uint(xb) >> 31;
        uint32_t idx;
        if constexpr (SR)
            idx = fp_sr_index<IFQ_FMT_NVFP4>(m, sr_uniform(w, j));
        else
            idx = fp_rtn_index<IFQ_FMT_NVFP4>(m);
        code[j] = (neg << 3) | idx;
        const float q = __uint_as_float(__float_as_uint(fp_magnitude<IFQ_FMT_NVFP4>(idx)) | (neg << 31));
        const float d = q - xb;
        err = __builtin_fmaf(d, d, err);
        if constexpr (RTN_ERR) {
            const float q0 = __uint_as_float(
                __float_as_uint(fp_magnitude<IFQ_FMT_NVFP4>(fp_rtn_index<IFQ_FMT_NVFP4>(m))) | (neg << 31));
            const float d0 = q0 - xb;
            err_rtn = __builtin_fmaf(d0, d0, err_rtn);
        }
    }
}

// Round-to-nearest 4/6 with the converter path; codes packed.
__device__ __forceinline__ uint32_t quantize_group_46(const float (&v)[kGroup], float alpha,
                                                      const Div& denom6, const Div& denom4, uint2& packed)
{
    const float amax = group_amax(v);
    float d6, d4;
    const uint32_t dc6 = group_scale<false>(amax, denom6, d6), dc4 = group_scale<false>(amax, denom4, d4);
    const float s6 = alpha * d6, s4 = alpha * d4;
    if (!(s4 >= 1.17549435e-38f)) {
        packed = make_uint2(0, 0);
        return 0;
    }
    float xb[kGroup];
    const float inv4 = recip_scale<false>(s4, denom6);
#pragma unroll
    for (int j = 0; j < kGroup; ++j) xb[j] = v[j] * inv4;
    uint32_t b0, b1;
    const float e4 = (d4 * d4) * e2m1_candidate(xb, b0, b1);
    bool keep4 = true;
    uint32_t a0 = 0, a1 = 0;
    if (s6 >= 1.17549435e-38f) {
        const float inv6 = recip_scale<false>(s6, denom6);
#pragma unroll
        for (int j = 0; j < kGroup; ++j) xb[j] = v[j] * inv6;
        const float e6 = (d6 * d6) * e2m1_candidate(xb, a0, a1);
        keep4 = e4 < e6;
    }
    packed = keep4 ? make_uint2(b0, b1) : make_uint2(a0, a1);
    return keep4 ? dc4 : dc6;
}

// Stochastic 4/6: both scalings round with the same draws; RTN_TYPE compares
// the round-to-nearest candidates' errors instead (App. B).
template <bool RTN_TYPE>
__device__ __forceinline__ uint32_t quantize_group_46_sr(const float (&v)[kGroup], float alpha,
                                                         const Div& denom6, const Div& denom4,
                                                         const uint32_t (&w)[8], uint32_t (&code)[kGroup])
{
    const float amax = group_amax(v);
    float d6, d4;
    const uint32_t dc6 = group_scale<true>(amax, denom6, d6), dc4 = group_scale<true>(amax, denom4, d4);
    const float s6 = alpha * d6, s4 = alpha * d4;
    if (!(s4 >= 1.17549435e-38f)) {
#pragma unroll
        for (int j = 0; j < kGroup; ++j) code[j] = 0;
        return 0;
    }
    uint32_t c4[kGroup], c6[kGroup];
    float e4, r4, e6 = 0.0f, r6 = 0.0f;
    e2m1_candidate_sr<true, RTN_TYPE>(v, recip_scale<true>(s4, denom6), w, c4, e4, r4);
    bool keep4 = true;
    if (s6 >= 1.17549435e-38f) {
        e2m1_candidate_sr<true, RTN_TYPE>(v, recip_scale<true>(s6, denom6), w, c6, e6, r6);
        keep4 = RTN_TYPE ? ((d4 * d4) * r4 < (d6 * d6) * r6) : ((d4 * d4) * e4 < (d6 * d6) * e6);
    }
#pragma unroll
    for (int j = 0; j < kGroup; ++j) code[j] = keep4 ? c4[j] : c6[j];
    return keep4 ? dc4 : dc6;
}

// Dense little-endian bit stream of 16 codes of BITS bits: 2*BITS bytes,
// written as BITS/2 32-bit words for even BITS and as 3 16-bit halves for 3.
template <int BITS> struct Packed;
template <> struct Packed<4> { uint32_t w[2]; };
template <> struct Packed<6> { uint32_t w[3]; };
template <> struct Packed<3> { uint32_t w[2]; };  // 48 bits: w[0] full, w[1] low 16

template <int BITS> __device__ __forceinline__ Packed<BITS> pack16(const uint32_t (&c)[kGroup])
{
    Packed<BITS> p;
    if constexpr (BITS == 3) {
        // 32-bit shifts only (code 10 straddles the words)
        uint32_t w0 = c[0], w1 = c[10] >> 2;
#pragma unroll
        for (int j = 1; j < 11; ++j) w0 |= c[j] << (3 * j);
#pragma unroll
        for (int j = 11; j < kGroup; ++j) w1 |= c[j] << (3 * j - 32);
        p.w[0] = w0;
        p.w[1] = w1;
        return p;
    }
    uint64_t lo = 0, hi = 0;
#pragma unroll
    for (int j = 0; j < kGroup; ++j) {
        int bit = j * BITS;
        if (bit < 64) {
            lo |= (uint64_t)c[j] << bit;
            if (bit + BITS > 64) hi |= (uint64_t)c[j] >> (64 - bit);
        } else {
            hi |= (uint64_t)c[j] << (bit - 64);
        }
    }
    if constexpr (BITS == 4) {
        p.w[0] = (uint32_t)lo; p.w[1] = (uint32_t)(lo >> 32);
    } else if constexpr (BITS == 6) {
        p.w[0] = (uint32_t)lo; p.w[1] = (uint32_t)(lo >> 32); p.w[2] = (uint32_t)hi;
    } else {
        p.w[0] = (uint32_t)lo; p.w[1] = (uint32_t)(lo >> 32);
    }
    return p;
}

template <int BITS> __device__ __forceinline__ void store_packed(uint8_t* dst, const Packed<BITS>& p)
{
    if constexpr (BITS == 4) {
        *reinterpret_cast<uint2*>(dst) = make_uint2(p.w[0], p.w[1]);
    } else if constexpr (BITS == 6) {
        // 12 bytes at a 4-byte aligned address (group pitch 12)
        uint32_t* d = reinterpret_cast<uint32_t*>(dst);
        d[0] = p.w[0]; d[1] = p.w[1]; d[2] = p.w[2];
    } else {
        // 6 bytes at a 2-byte aligned address (group pitch 6)
        uint16_t* d = reinterpret_cast<uint16_t*>(dst);
        d[0] = (uint16_t)p.w[0]; d[1] = (uint16_t)(p.w[0] >> 16); d[2] = (uint16_t)p.w[1];
    }
}

template <int BITS> __device__ __forceinline__ void load_unpack16(const uint8_t* src, uint32_t (&c)[kGroup])
{
    uint64_t lo, hi = 0;
    if constexpr (BITS == 4) {
        uint2 t = *reinterpret_cast<const uint2*>(src);
        lo = (uint64_t)t.x | ((uint64_t)t.y << 32);
    } else if constexpr (BITS == 6) {
        const uint32_t* s = reinterpret_cast<const uint32_t*>(src);
        lo = (uint64_t)s[0] | ((uint64_t)s[1] << 32);
        hi = s[2];
    } else {
        const uint16_t* s = reinterpret_cast<const uint16_t*>(src);
        lo = (uint64_t)s[0] | ((uint64_t)s[1] << 16) | ((uint64_t)s[2] << 32);
    }
#pragma unroll
    for (int j = 0; j < kGroup; ++j) {
        int bit = j * BITS;
        uint64_t val;
        if (bit + BITS <= 64)
            val = lo >> bit;
        else if (bit >= 64)
            val = hi >> (bit - 64);
        else
            val = (lo >> bit) | (hi << (64 - bit));
        c[j] = (uint32_t)val & ((1u << BITS) - 1u);
    }
}

// IF4 / NVFP4 with stochastic rounding: the arithmetic of quantize_group
// with SR (FP: grid neighbours lo <= m < lo + q of the clamped magnitude m,
// up iff u q < m - lo; INT: y = x c_up, up iff u < |y| - floor|y|, clamped to
// 7), with fewer steps: the grid step q of m's binade (0.5 below 2, 1 below
// 4, 2 above) comes from m's exponent bits, both roundings are sr_ceil of the
// exact ratio (m / q, |y|), the candidate is the chosen grid value itself
// (lo or lo + q, exact) with x's sign instead of a rebuild from its code,
// and the codes come from the converters -- the E2M1 code of an
// exact grid value (round to nearest even leaves it in place, the sign and a
// signed zero kept) and, for INT, the low nibble of r + 1.5 * 2^23.  RTN_TYPE
// decides the type on the round-to-nearest candidates' errors (App. B).
template <bool ADAPTIVE, bool RTN_TYPE>
__device__ __forceinline__ uint32_t quantize_group_e2m1_sr(const float (&v)[kGroup], float alpha, const Div& denom,
                                                           const uint32_t (&w)[8], uint2& packed)
{
    constexpr float C_UP = 7.0f / 6.0f, K_DN = 6.0f / 7.0f;
    const float amax = group_amax(v);
    float delta;
    const uint32_t dcode = group_scale<true>(amax, denom, delta);
    const float s = alpha * delta;
    if (!(s >= 1.17549435e-38f)) {
        packed = make_uint2(0, 0);
        return 0;
    }
    const float inv = recip_scale<true>(s, denom);
    float xb[kGroup], qf[kGroup];
    uint32_t tb[kGroup];
    float ef = 0.0f, ei = 0.0f;
#pragma unroll
    for (int j = 0; j < kGroup; ++j) {
        xb[j] = v[j] * inv;
        const float h = sr_draw(w, j);
        const float m = fminf(fabsf(xb[j]), 6.0f);
        // 2^floor(log2 m) (0 for m below 2^-126), the step q and 1/q (powers of two)
        const float p2 = __uint_as_float(__float_as_uint(m) & 0x7F800000u);
        const float q = fmaxf(p2 * 0.5f, 0.5f);
        const float inv_q = __uint_as_float((254u << 23) - __float_as_uint(q));
        qf[j] = with_sign_of(sr_ceil_h(m * inv_q, h) * q, xb[j]);
        const float d = qf[j] - xb[j];
        ef = __builtin_fmaf(d, d, ef);
        if constexpr (ADAPTIVE) {
            const float y = xb[j] * C_UP;
            const float r = with_sign_of(fminf(sr_ceil_h(fabsf(y), h), 7.0f), y);
            tb[j] = __float_as_uint(r + 12582912.0f);
            const float di = __builtin_fmaf(r, K_DN, -xb[j]);
            ei = __builtin_fmaf(di, di, ei);
        }
    }
    uint32_t f0 = 0, f1 = 0;
    f0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(f0, qf[0], qf[1], 1.0f, 0);
    f0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(f0, qf[2], qf[3], 1.0f, 1);
    f0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(f0, qf[4], qf[5], 1.0f, 2);
    f0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(f0, qf[6], qf[7], 1.0f, 3);
    f1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(f1, qf[8], qf[9], 1.0f, 0);
    f1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(f1, qf[10], qf[11], 1.0f, 1);
    f1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(f1, qf[12], qf[13], 1.0f, 2);
    f1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(f1, qf[14], qf[15], 1.0f, 3);
    if constexpr (!ADAPTIVE) {
        packed = make_uint2(f0, f1);
        return dcode;
    }
    bool use_int;
    if constexpr (RTN_TYPE) {
        // the round-to-nearest candidates' errors decide the type
        uint32_t g0, g1;
        const float rf = e2m1_candidate(xb, g0, g1);
        float ri = 0.0f;
#pragma unroll
        for (int j = 0; j < kGroup; ++j) {
            const float xc = __builtin_amdgcn_fmed3f(xb[j], -6.0f, 6.0f);
            const float r0 = __builtin_fmaf(xc, C_UP, 12582912.0f) - 12582912.0f;
            const float e0 = __builtin_fmaf(r0, K_DN, -xb[j]);
            ri = __builtin_fmaf(e0, e0, ri);
        }
        use_int = ri < rf;
    } else {
        use_int = ei < ef;
    }
    uint32_t i0, i1;
    pack_int4_biased(tb, i0, i1);
    packed = use_int ? make_uint2(i0, i1) : make_uint2(f0, f1);
    return dcode | (use_int ? 0x80u : 0u);
}

// IF6 (E2M3 / E3M2) with round-to-nearest: the arithmetic of quantize_group
// with the FP candidate from gfx950's 32-value FP6 converters: fp32 -> FP6
// rounds to nearest even and saturates, keeping the sign (signed zero
// included), and writes 32 codes at bits 6j .. 6j + 5, code 2i from element
// i of its first source and 2i + 1 from element i of its second.  With the
// group's even elements in the first source and its odd ones in the second
// (zeros after them), the first three dwords are the group's FP codes in the
// packed layout of the format; FP6 -> fp32 reads them back in code order.
// An exhaustive comparison over every finite fp32 of both signs found the
// conversion equal to the nearest-even encoder of quantize_group, and the
// decode exact for all 64 codes of either format.
template <int FMT>
__device__ __forceinline__ uint32_t quantize_group_fp6(const float (&v)[kGroup], float alpha, const Div& denom,
                                                       Packed<6>& out)
{
    using F = Fmt<FMT>;
    using D = FmtDerived<FMT>;
    typedef float f16v __attribute__((ext_vector_type(16)));
    typedef float f32v __attribute__((ext_vector_type(32)));
    typedef uint32_t u6v __attribute__((ext_vector_type(6)));
    const float amax = group_amax(v);
    float delta;
    const uint32_t dcode = group_scale<false>(amax, denom, delta);
    const float s = alpha * delta;
    if (!(s >= 1.17549435e-38f)) {
        out.w[0] = out.w[1] = out.w[2] = 0;
        return 0;
    }
    const float inv = recip_scale<false>(s, denom);
    float xa[kGroup];
    f16v ev, od;
#pragma unroll
    for (int j = 0; j < kGroup; ++j) xa[j] = v[j] * inv;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        ev[i] = xa[2 * i];
        od[i] = xa[2 * i + 1];
        ev[8 + i] = 0.0f;
        od[8 + i] = 0.0f;
    }
    u6v fc;
    f32v q;
    if constexpr (F::EB == 2) {
        fc = __builtin_amdgcn_cvt_scalef32_2xpk16_fp6_f32(ev, od, 1.0f);
        q = __builtin_amdgcn_cvt_scalef32_pk32_f32_fp6(fc, 1.0f);
    } else {
        fc = __builtin_amdgcn_cvt_scalef32_2xpk16_bf6_f32(ev, od, 1.0f);
        q = __builtin_amdgcn_cvt_scalef32_pk32_f32_bf6(fc, 1.0f);
    }
    float ef = 0.0f, ei = 0.0f;
    uint32_t ci[kGroup];
#pragma unroll
    for (int j = 0; j < kGroup; ++j) {
        const float d = q[j] - xa[j];
        ef = __builtin_fmaf(d, d, ef);
        const float xc = __builtin_amdgcn_fmed3f(xa[j], -F::FP_MAX, F::FP_MAX);
        const float t = __builtin_fmaf(xc, D::C_UP, 12582912.0f);  // rint(xc*c_up) + 1.5*2^23
        ci[j] = __float_as_uint(t) & D::CODE_MASK;                   // two's complement, 6 bits
        const float di = __builtin_fmaf(t - 12582912.0f, D::K_DN, -xa[j]);
        ei = __builtin_fmaf(di, di, ei);
    }
    if (ei < ef) {
        out = pack16<6>(ci);
        return dcode | 0x80u;
    }
    out.w[0] = fc[0];
    out.w[1] = fc[1];
    out.w[2] = fc[2];
    return dcode;
}

// ------------------------------------------------------ group dispatcher
// Quantize one (already transformed) block of 16 values of any format:
// returns its scale byte (two, low byte first, for block size 8) and the
// packed codes.  denom = fp32(alpha * M) with M the format's
// group target (with the margin when it is on); gi is the group's index for
// the SR draws.
template <int FMT, bool SR>
__device__ __forceinline__ uint32_t quantize_any(const float (&v)[kGroup], float alpha, const Div& denom,
                                                 int qflags, uint64_t seed, int64_t gi,
                                                 Packed<Fmt<FMT>::BITS>& out)
{
    using F = Fmt<FMT>;
    constexpr int BITS = F::BITS;
    const bool rtn_type = (qflags & kQSrRtnType) != 0;
    if constexpr (F::G == 8 && BITS == 4 && !SR) {
        // two blocks of 8; returns both scale bytes, low byte first
        float v0[8], v1[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            v0[j] = v[j];
            v1[j] = v[8 + j];
        }
        const uint32_t b0 = quantize_block8_e2m1<F::ADAPTIVE>(v0, alpha, denom, out.w[0]);
        const uint32_t b1 = quantize_block8_e2m1<F::ADAPTIVE>(v1, alpha, denom, out.w[1]);
        return b0 | (b1 << 8);
    } else if constexpr (F::G == 8 && BITS == 3 && !SR) {
        float v0[8], v1[8];
        uint32_t c0[8], c1[8], c[kGroup];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            v0[j] = v[j];
            v1[j] = v[8 + j];
        }
        const uint32_t b0 = quantize_group_e2m0<8>(v0, alpha, denom, c0);
        const uint32_t b1 = quantize_group_e2m0<8>(v1, alpha, denom, c1);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            c[j] = c0[j];
            c[8 + j] = c1[j];
        }
        out = pack16<3>(c);
        return b0 | (b1 << 8);
    } else if constexpr (F::G == 8) {
        // two groups of 8 (scale bytes 2 gi and 2 gi + 1, which are also their
        // SR counters); returns both scale bytes, low byte first
        constexpr int B = Base<FMT>::F;
        uint32_t c[kGroup];
        uint32_t sb = 0;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            float vh[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) vh[j] = v[8 * h + j];
            uint32_t w[8] = {0, 0, 0, 0, 0, 0, 0, 0};
            if constexpr (SR) sr_words_first(seed, 2 * (uint64_t)gi + h, w);
            uint32_t ch[8];
            const uint32_t b = (SR && rtn_type) ? quantize_group<B, SR, true, 8>(vh, alpha, denom, w, ch)
                                                : quantize_group<B, SR, false, 8>(vh, alpha, denom, w, ch);
#pragma unroll
            for (int j = 0; j < 8; ++j) c[8 * h + j] = ch[j];
            sb |= b << (8 * h);
        }
        out = pack16<BITS>(c);
        return sb;
    }
    uint32_t w[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if constexpr (SR) sr_words(seed, (uint64_t)gi, w);
    if constexpr (F::KIND == kKindFourSix) {
        const Div denom4 = make_div(alpha, alpha * ((qflags & kQMargin) ? kFourTargetMargin : kFourTarget));
        if constexpr (SR) {
            uint32_t c[kGroup];
            const uint32_t sb = rtn_type ? quantize_group_46_sr<true>(v, alpha, denom, denom4, w, c)
                                         : quantize_group_46_sr<false>(v, alpha, denom, denom4, w, c);
            out = pack16<4>(c);
            return sb;
        } else {
            uint2 pk;
            const uint32_t sb = quantize_group_46(v, alpha, denom, denom4, pk);
            out.w[0] = pk.x;
            out.w[1] = pk.y;
            return sb;
        }
    } else if constexpr (F::KIND == kKindInt) {
        uint2 pk;
        const uint32_t sb = quantize_group_int4<SR>(v, alpha, denom, w, pk);
        out.w[0] = pk.x;
        out.w[1] = pk.y;
        return sb;
    } else if constexpr (BITS == 4 && !SR) {
        uint2 pk;
        const uint32_t sb = quantize_group_e2m1<F::ADAPTIVE>(v, alpha, denom, pk);
        out.w[0] = pk.x;
        out.w[1] = pk.y;
        return sb;
    } else if constexpr (BITS == 4) {
        uint2 pk;
        const uint32_t sb = rtn_type ? quantize_group_e2m1_sr<F::ADAPTIVE, true>(v, alpha, denom, w, pk)
                                     : quantize_group_e2m1_sr<F::ADAPTIVE, false>(v, alpha, denom, w, pk);
        out.w[0] = pk.x;
        out.w[1] = pk.y;
        return sb;
    } else if constexpr (BITS == 6 && !SR) {
        return quantize_group_fp6<FMT>(v, alpha, denom, out);
    } else if constexpr (BITS == 3 && !SR) {
        uint32_t c[kGroup];
        const uint32_t sb = quantize_group_e2m0<kGroup>(v, alpha, denom, c);
        out = pack16<3>(c);
        return sb;
    } else {
        uint32_t c[kGroup];
        const uint32_t sb = (SR && rtn_type) ? quantize_group<FMT, SR, true>(v, alpha, denom, w, c)
                                             : quantize_group<FMT, SR, false>(v, alpha, denom, w, c);
        out = pack16<BITS>(c);
        return sb;
    }
}

}  // namespace ifq
