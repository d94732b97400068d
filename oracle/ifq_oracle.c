/*
 * ifq_oracle.c -- plain, slow, scalar CPU oracle for the adaptive
 * block-scaled formats of "Adaptive Block-Scaled Data Types"
 * (IF3, IF4, IF6-E2M3, IF6-E3M2, and IF4 / IF3 with block size 8) and the
 * comparison formats NVFP4 (also with block size 8), NVINT4 and NVFP4 with
 * Four Over Six (4/6).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only tests/, the smoke check and the CPU-baseline leg of
 * bench.py do.  It shares no code, header, table or constant generator with
 * the HIP library.
 *
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fno-fast-math -shared -fPIC
 * (binary32 round-to-nearest-even everywhere, denormals kept, no FMA
 * contraction: every fmaf() below is written on purpose).
 *
 * Precision.  The paper fixes the tensor scale as FP32 (Sec. 3, Eq. 1) and
 * the group scale as FP8 E4M3 (Sec. 3, Eq. 2).  The remaining arithmetic
 * (scaled values, candidate errors) decides integer codes, so it is carried
 * out in binary32 in a fixed operation order that the GPU kernels follow
 * too.  Rounding onto a code grid is done by exhaustive nearest-point search
 * over the grid (ties to the even code), which is the definition of
 * round-to-nearest-even, not a bit trick.
 *
 * Parity pins (tests/test_oracle_*.py) fix this file against the paper:
 *   FP4 grid (Sec. 1), E4M3 max 448 (Sec. 3) and min 2^-9 (Table 1),
 *   the Fig. 3a worked example, brute force over tiny groups, the
 *   IF4 <= NVFP4 error invariant, Table 1 MSE values, exact round trips,
 *   RHT orthonormality, SR unbiasedness, and the Philox4x32-10 stream
 *   against an independent installed implementation.  NVINT4 and 4/6:
 *   Table 1 MSE and maxima, brute force in exact rationals (nearest codes,
 *   nearest E4M3 scales, the smaller-error scaling), agreement with the
 *   independent numpy implementation, round trips and the 4/6 tie rule.
 *   Block size 8 (IF4-BS8, IF3-BS8, NVFP4-BS8): Table 6's bits per
 *   parameter, reduction to the 16-value algorithm with zero padding, brute
 *   force over tiny groups, lower error than block size 16.
 * The fp32 operation order itself (reciprocal-multiply scaling, the error
 * accumulation order) is not fixed by the paper: parity unpinned beyond the
 * self-consistency of oracle and kernels, as recorded in the design notes.
 */
#include <float.h>
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* format ids: must match the numbering the tests use */
enum {
    FMT_IF4 = 0,
    FMT_NVFP4 = 1,
    FMT_IF3 = 2,
    FMT_IF6_E2M3 = 3,
    FMT_IF6_E3M2 = 4,
    FMT_NVINT4 = 5,
    FMT_NVFP4_46 = 6,
    FMT_IF4_BS8 = 7,
    FMT_IF3_BS8 = 8,
    FMT_NVFP4_BS8 = 9,
    FMT_COUNT = 10
};
/* element-type rule of a format */
enum {
    KIND_FP = 0,        /* FP elements only (NVFP4) */
    KIND_ADAPTIVE = 1,  /* per-group FP or INT by squared error (IF formats) */
    KIND_INT = 2,       /* INT elements only (NVINT4) */
    KIND_FOUR_SIX = 3   /* FP elements, group scaled to a maximum of 6 or 4 (4/6) */
};
/* flag bits */
enum { F_RHT = 1, F_SR = 2, F_MARGIN = 4, F_SCALE_IN = 8, F_STRIDED = 16, F_SR_RTN_TYPE = 32 };

#define GROUP 16 /* the largest group; also the RHT block and the K granularity */

typedef struct {
    int bits;          /* bits per stored code */
    int ebits, mbits;  /* FP element: exponent and mantissa field widths */
    int kind;          /* KIND_* */
    int gsize;         /* values per group (one scale each): 16, or 8 (Sec. 5.1) */
    int adaptive;      /* kind == KIND_ADAPTIVE */
    float m_scale;     /* M of Eq. 1-2: the element maximum a group is scaled to */
    float alpha_fp8;   /* the E4M3 factor of Eq. 1: 448, or 256 for 4/6 */
    int n_mag;         /* number of non-negative FP codes = 2^(bits-1) */
    double mag[32];    /* FP magnitude of each non-negative code (exact) */
    float fp_max;      /* M_FP: largest FP magnitude */
    int int_max;       /* M_I = 2^(bits-1) - 1 (INT code -2^(bits-1) unused) */
    float c_up;        /* fp32(M_I / M_FP): INT candidates are scaled up by this */
    float k_dn;        /* fp32(M_FP / M_I): INT codes are scaled down by this */
} fmt_desc;

static fmt_desc g_fmt[FMT_COUNT];
static int g_init = 0;

/* Magnitude of an ExMy code (no infinities, no NaN, subnormals at E = 0):
 * the usual IEEE-style value rule with bias 2^(e-1) - 1 (Sec. 5.1 names
 * the element types by their ExMy split; E2M1 gives the FP4 grid of Sec. 1). */
static double exmy_value(int ebits, int mbits, int code)
{
    int bias = (1 << (ebits - 1)) - 1;
    int E = code >> mbits, M = code & ((1 << mbits) - 1);
    if (E == 0) return ldexp((double)M, 1 - bias - mbits);
    return ldexp((double)((1 << mbits) + M), E - bias - mbits);
}

static void init_fmt(fmt_desc* f, int bits, int ebits, int mbits, int kind)
{
    f->bits = bits;
    f->ebits = ebits;
    f->mbits = mbits;
    f->kind = kind;
    f->gsize = GROUP;
    f->adaptive = kind == KIND_ADAPTIVE;
    f->n_mag = 1 << (bits - 1);
    for (int i = 0; i < f->n_mag; ++i) f->mag[i] = exmy_value(ebits, mbits, i);
    f->fp_max = (float)f->mag[f->n_mag - 1];
    f->int_max = (1 << (bits - 1)) - 1;
    /* Sec. 3 ("6/7 method") and the Sec. 5.1 footnote: INT groups are scaled
     * by M_I/M_FP before rounding and by M_FP/M_I after, so both element
     * types span [0, M_FP * Delta].  Each ratio is rounded once to fp32. */
    f->c_up = (float)f->int_max / f->fp_max;
    f->k_dn = f->fp_max / (float)f->int_max;
    f->m_scale = f->fp_max;
    f->alpha_fp8 = 448.0f;
    if (kind == KIND_INT) {
        /* NVINT4 (Sec. 2, Table 1): INT4 elements scaled straight to
         * M_I = 7, so neither range factor applies; max value 7 x 448. */
        f->m_scale = (float)f->int_max;
        f->c_up = 1.0f;
        f->k_dn = 1.0f;
    } else if (kind == KIND_FOUR_SIX) {
        /* 4/6 (Sec. 3 and Table 1): the tensor scale uses 6 x 256 so that
         * the group with the tensor maximum can still be scaled to 4. */
        f->alpha_fp8 = 256.0f;
    }
}

static void ensure_init(void)
{
    if (g_init) return;
    init_fmt(&g_fmt[FMT_IF4], 4, 2, 1, KIND_ADAPTIVE);       /* E2M1 / INT4, Sec. 3 */
    init_fmt(&g_fmt[FMT_NVFP4], 4, 2, 1, KIND_FP);           /* E2M1 only: Fig. 3a up to the FP candidate */
    init_fmt(&g_fmt[FMT_IF3], 3, 2, 0, KIND_ADAPTIVE);       /* E2M0 / INT3, Sec. 5.1 */
    init_fmt(&g_fmt[FMT_IF6_E2M3], 6, 2, 3, KIND_ADAPTIVE);  /* E2M3 / INT6, Table 6 */
    init_fmt(&g_fmt[FMT_IF6_E3M2], 6, 3, 2, KIND_ADAPTIVE);  /* E3M2 / INT6, Table 6 */
    init_fmt(&g_fmt[FMT_NVINT4], 4, 2, 1, KIND_INT);         /* INT4 only, Sec. 2 */
    init_fmt(&g_fmt[FMT_NVFP4_46], 4, 2, 1, KIND_FOUR_SIX);  /* E2M1, max 6 or 4, Sec. 3 */
    /* block size 8: one scale per 8 values (Sec. 5.1; Table 6, App. D) */
    init_fmt(&g_fmt[FMT_IF4_BS8], 4, 2, 1, KIND_ADAPTIVE);
    init_fmt(&g_fmt[FMT_IF3_BS8], 3, 2, 0, KIND_ADAPTIVE);
    init_fmt(&g_fmt[FMT_NVFP4_BS8], 4, 2, 1, KIND_FP);
    g_fmt[FMT_IF4_BS8].gsize = 8;
    g_fmt[FMT_IF3_BS8].gsize = 8;
    g_fmt[FMT_NVFP4_BS8].gsize = 8;
    g_init = 1;
}

/* ---------------------------------------------------------------- E4M3 -- */

/* Value of a non-negative finite E4M3 code (0..126); 127 is NaN. */
double oracle_e4m3_value(int code)
{
    code &= 0x7F;
    if (code == 0x7F) return NAN;
    return exmy_value(4, 3, code);
}

/* Nearest non-negative finite E4M3 value to x >= 0, ties to the even code.
 * Exhaustive search over the 127 finite codes, so values above the largest
 * (448, Sec. 3) saturate to it and values at or below 2^-10 round to zero. */
int oracle_e4m3_encode(float x)
{
    double xd = (double)x;
    /* at or beyond the largest finite value that value is the nearest one
     * (comparing distances in fp64 would lose it for huge x) */
    if (xd >= 448.0) return 0x7E;
    int best = 0;
    double best_err = fabs(xd);
    for (int c = 1; c < 127; ++c) {
        double err = fabs(oracle_e4m3_value(c) - xd);
        if (err < best_err || (err == best_err && (c & 1) == 0 && (best & 1) == 1)) {
            best = c;
            best_err = err;
        }
    }
    return best;
}

/* -------------------------------------------------------- FP grid (RTN) -- */

/* Index of the FP magnitude nearest to m >= 0, ties to the even index.
 * Saturates at M_FP because the search only sees grid points. */
static int fp_nearest_index(const fmt_desc* f, double m)
{
    if (m >= f->mag[f->n_mag - 1]) return f->n_mag - 1;
    int best = 0;
    double best_err = fabs(m);
    for (int i = 1; i < f->n_mag; ++i) {
        double err = fabs(f->mag[i] - m);
        if (err < best_err || (err == best_err && (i & 1) == 0 && (best & 1) == 1)) {
            best = i;
            best_err = err;
        }
    }
    return best;
}

int oracle_fp_round_index(int fmt, float m)
{
    ensure_init();
    return fp_nearest_index(&g_fmt[fmt], fabs((double)m));
}

double oracle_fp_magnitude(int fmt, int idx)
{
    ensure_init();
    return g_fmt[fmt].mag[idx];
}

int oracle_group_size(int fmt)
{
    ensure_init();
    return g_fmt[fmt].gsize;
}

void oracle_fmt_constants(int fmt, float* fp_max, int* int_max, float* c_up, float* k_dn, int* bits)
{
    ensure_init();
    const fmt_desc* f = &g_fmt[fmt];
    *fp_max = f->fp_max;
    *int_max = f->int_max;
    *c_up = f->c_up;
    *k_dn = f->k_dn;
    *bits = f->bits;
}

/* ------------------------------------------------------ Philox4x32-10 -- */
/* Counter-based generator of Salmon, Moraes, Dror and Shaw (SC'11): ten
 * rounds of two 32x32->64 multiplies with a Weyl-sequence key schedule. */
#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

void oracle_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4])
{
    uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
    uint32_t k0 = key_in[0], k1 = key_in[1];
    for (int r = 0; r < 10; ++r) {
        if (r > 0) {
            k0 += PHILOX_W0;
            k1 += PHILOX_W1;
        }
        uint64_t p0 = (uint64_t)PHILOX_M0 * c0;
        uint64_t p1 = (uint64_t)PHILOX_M1 * c2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        uint32_t n0 = hi1 ^ c1 ^ k0;
        uint32_t n1 = lo1;
        uint32_t n2 = hi0 ^ c3 ^ k1;
        uint32_t n3 = lo0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* The 16 uniform 16-bit draws of group number `group` (the linear index of
 * its scale byte): two Philox blocks with counter (group lo, group hi,
 * block, 0) and key = seed; element j takes half (j & 1) of word j >> 1. */
void oracle_sr_bits(uint64_t seed, uint64_t group, uint16_t h[GROUP])
{
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint32_t w[8];
    for (uint32_t blk = 0; blk < 2; ++blk) {
        uint32_t ctr[4] = {(uint32_t)group, (uint32_t)(group >> 32), blk, 0u};
        oracle_philox4x32_10(ctr, key, &w[4 * blk]);
    }
    for (int j = 0; j < GROUP; ++j) h[j] = (uint16_t)(w[j >> 1] >> (16 * (j & 1)));
}

/* ------------------------------------------------------------- RHT-16 -- */
/* 16-point random Hadamard transform (Sec. 1 and Sec. 4.1 apply it to the
 * weight-gradient inputs): v = (1/4) H16 diag(s) x with H16 the Sylvester
 * Hadamard matrix, H[i][j] = (-1)^popcount(i & j), and s_j = -1 where bit j
 * of `signs` is set.  H16 is evaluated with the fast butterfly (strides 1, 2,
 * 4, 8; pair (a, b) -> (a + b, a - b)), each add rounded to fp32, then the
 * exact scaling by 1/4. */
void oracle_rht16(const float x[GROUP], uint32_t signs, float v[GROUP])
{
    for (int j = 0; j < GROUP; ++j) v[j] = ((signs >> j) & 1u) ? -x[j] : x[j];
    for (int h = 1; h < GROUP; h <<= 1) {
        for (int i = 0; i < GROUP; ++i) {
            if (i & h) continue;
            float a = v[i], b = v[i + h];
            v[i] = a + b;
            v[i + h] = a - b;
        }
    }
    for (int j = 0; j < GROUP; ++j) v[j] = v[j] * 0.25f;
}

/* ------------------------------------------------------ scale factors -- */

/* A group target m (M_FP, M_I for NVINT4, 6 or 4 for 4/6), or m * 16/17
 * when the gradient margin of Sec. 4.1 is on. */
static float with_margin(float m, uint32_t flags)
{
    if (flags & F_MARGIN) return (float)((double)m * 16.0 / 17.0);
    return m;
}

static float scale_max(const fmt_desc* f, uint32_t flags) { return with_margin(f->m_scale, flags); }

/* Eq. (1): alpha = max|X| / (M * M_FP8) with M_FP8 = 448 (256 for 4/6). */
float oracle_tensor_scale(int fmt, float amax, uint32_t flags)
{
    ensure_init();
    const fmt_desc* f = &g_fmt[fmt];
    float denom = scale_max(f, flags) * f->alpha_fp8;
    return amax / denom;
}

/* ------------------------------------------------------ one group -- */

/* The two candidates of one group (Fig. 3a) for scaled values
 * xb: codes cf (FP) and ci (INT) and their squared errors, with
 * round-to-nearest-even or, with sr, stochastic rounding by h. */
static void candidates(const fmt_desc* f, const float xb[GROUP], int sr, const uint16_t h[GROUP],
                       uint8_t cf[GROUP], uint8_t ci[GROUP], float* e_fp, float* e_int)
{
    const int n = f->gsize;
    const int sign_bit = 1 << (f->bits - 1);
    const int code_mask = (1 << f->bits) - 1;
    /* FP candidate (Fig. 3a). */
    float ef = 0.0f;
    for (int j = 0; j < n; ++j) {
        double m = fabs((double)xb[j]);
        int idx;
        if (!sr) {
            idx = fp_nearest_index(f, m);
        } else {
            /* Stochastic rounding between the grid neighbours lo <= m < hi:
             * up with probability ~ (m - lo) / (hi - lo), using h_j. */
            float mf = fminf(fabsf(xb[j]), f->fp_max);
            idx = 0;
            while (idx + 1 < f->n_mag && f->mag[idx + 1] <= (double)mf) ++idx;
            if (idx + 1 < f->n_mag) {
                float lo = (float)f->mag[idx], hi = (float)f->mag[idx + 1];
                float u = (float)h[j] * (1.0f / 65536.0f);
                if (u * (hi - lo) < mf - lo) ++idx;
            }
        }
        int neg = signbit(xb[j]) != 0;
        cf[j] = (uint8_t)((neg ? sign_bit : 0) | idx);
        float q = (float)f->mag[idx];
        if (neg) q = -q;
        float d = q - xb[j];
        ef = fmaf(d, d, ef);
    }

    /* INT candidate (Fig. 3a): int(x-bar * M_I/M_FP), clamped to
     * +-M_I, reconstructed as code * M_FP/M_I. */
    float ei = 0.0f;
    for (int j = 0; j < n; ++j) {
        double r;
        if (!sr) {
            /* nearest integer to the exact product, ties to even */
            r = nearbyint((double)xb[j] * (double)f->c_up);
        } else {
            float y = xb[j] * f->c_up;
            float a = fabsf(y);
            float lo = floorf(a);
            float u = (float)h[j] * (1.0f / 65536.0f);
            float rr = (u < a - lo) ? lo + 1.0f : lo;
            r = (y < 0.0f) ? -(double)rr : (double)rr;
        }
        if (r > f->int_max) r = f->int_max;
        if (r < -f->int_max) r = -f->int_max;
        int ri = (int)r;
        ci[j] = (uint8_t)(ri & code_mask);
        float d = fmaf((float)ri, f->k_dn, -xb[j]);
        ei = fmaf(d, d, ei);
    }

    *e_fp = ef;
    *e_int = ei;
}

/* Quantize one group of 16 values v (already transformed when the RHT is
 * on) under tensor scale alpha; Fig. 3a with alpha restored
 * (Eq. 2 divides by alpha * M_FP).
 *   h      16-bit uniforms for stochastic rounding (ignored without F_SR)
 *   codes  out: 16 element codes (low `bits` bits used)
 *   scale  out: E4M3 code of Delta, bit 7 set when the group is INT
 *   e_fp, e_int  out: the two candidate errors (sum of squares, x-bar units)
 */
/* 4/6 (Sec. 3, following Four Over Six): the group is scaled twice, to a
 * maximum of 6 and to a maximum of 4 (Eq. 2 with M = 6 or 4), rounded onto
 * E2M1 each time, and the scaling whose dequantized values have the smaller
 * squared error is kept (ties keep 6).  With x-bar_t = X / (alpha Delta_t) the
 * squared error of scaling t divided by alpha^2 is
 * Delta_t^2 * sum_j (q_j - x-bar_j)^2; that product, rounded to fp32, is
 * what is compared.  Delta_4 >= Delta_6, so a scaling to 4 whose combined
 * scale is below FLT_MIN leaves none: the group stores zeros; when only the
 * scaling to 6 falls below FLT_MIN, 4 is kept.  With SR both scalings round
 * stochastically with the same draws; with F_SR_RTN_TYPE the comparison uses
 * their round-to-nearest candidates instead. */
static void four_six_group(const fmt_desc* f, const float v[GROUP], float alpha, uint32_t flags,
                           const uint16_t h[GROUP], uint8_t codes[GROUP], uint8_t* scale,
                           float* e6, float* e4)
{
    const int sr = (flags & F_SR) != 0;
    const int n = f->gsize;
    float amax_g = 0.0f;
    for (int j = 0; j < n; ++j) {
        float a = fabsf(v[j]);
        if (a > amax_g) amax_g = a;
    }
    const float target[2] = {scale_max(f, flags), with_margin(4.0f, flags)};
    uint8_t cand[2][GROUP];
    int dcode[2];
    float err[2] = {0.0f, 0.0f};
    int ok[2];
    for (int t = 0; t < 2; ++t) {
        float denom = alpha * target[t];
        dcode[t] = (denom > 0.0f) ? oracle_e4m3_encode(amax_g / denom) : 0;
        float delta = (float)oracle_e4m3_value(dcode[t]);
        float s = alpha * delta;
        ok[t] = s >= FLT_MIN;
        if (!ok[t]) continue;
        float inv = 1.0f / s;
        float xb[GROUP];
        for (int j = 0; j < n; ++j) xb[j] = v[j] * inv;
        uint8_t ci[GROUP];
        float ef, ei;
        candidates(f, xb, sr, h, cand[t], ci, &ef, &ei);
        if (sr && (flags & F_SR_RTN_TYPE)) {
            uint8_t rf[GROUP];
            candidates(f, xb, 0, h, rf, ci, &ef, &ei);
        }
        err[t] = (delta * delta) * ef;
    }
    *e6 = err[0];
    *e4 = err[1];
    if (!ok[1]) {
        memset(codes, 0, (size_t)n);
        *scale = 0;
        return;
    }
    int pick = (ok[0] && !(err[1] < err[0])) ? 0 : 1;
    memcpy(codes, cand[pick], (size_t)n);
    *scale = (uint8_t)dcode[pick];
}

/* One group of the format's size (v, h and codes hold that many; 16 or 8).
 * IF formats and NVFP4: Fig. 3a.  NVINT4: the INT candidate
 * alone, scaled to M_I (c_up = 1).  4/6: four_six_group, which reports the
 * two scalings' errors in e_fp (to 6) and e_int (to 4). */
void oracle_quantize_group(int fmt, const float v[GROUP], float alpha, uint32_t flags,
                           const uint16_t h[GROUP], uint8_t codes[GROUP], uint8_t* scale,
                           float* e_fp, float* e_int)
{
    ensure_init();
    const fmt_desc* f = &g_fmt[fmt];
    const int sr = (flags & F_SR) != 0;
    const int n = f->gsize;
    if (f->kind == KIND_FOUR_SIX) {
        four_six_group(f, v, alpha, flags, h, codes, scale, e_fp, e_int);
        return;
    }

    /* Fig. 3a, Eq. (2): Delta = max|X_g| / (alpha * M). */
    float amax_g = 0.0f;
    for (int j = 0; j < n; ++j) {
        float a = fabsf(v[j]);
        if (a > amax_g) amax_g = a;
    }
    float denom = alpha * scale_max(f, flags);
    float delta_raw = amax_g / denom;
    /* Fig. 3a: cast to E4M3 (round to nearest even, saturating). */
    int dcode = (denom > 0.0f) ? oracle_e4m3_encode(delta_raw) : 0;
    float delta = (float)oracle_e4m3_value(dcode);

    /* Scaled values x-bar = X / (alpha * Delta) (Fig. 3a, alpha from
     * Eq. 1), as a multiply by the rounded reciprocal.  A group whose
     * combined scale is zero or below the smallest normal fp32 stores zeros. */
    float s = alpha * delta;
    if (!(s >= FLT_MIN)) {
        memset(codes, 0, (size_t)n);
        *scale = 0;
        *e_fp = 0.0f;
        *e_int = 0.0f;
        return;
    }
    float inv = 1.0f / s;
    float xb[GROUP];
    for (int j = 0; j < n; ++j) xb[j] = v[j] * inv;

    uint8_t cf[GROUP], ci[GROUP];
    float ef, ei;
    candidates(f, xb, sr, h, cf, ci, &ef, &ei);
    /* App. B variant: the type is decided on the round-to-nearest candidates
     * (independent of the random draws), and the group is then rounded
     * stochastically in that type. */
    float sel_f = ef, sel_i = ei;
    if (sr && (flags & F_SR_RTN_TYPE)) {
        uint8_t rf[GROUP], ri[GROUP];
        candidates(f, xb, 0, h, rf, ri, &sel_f, &sel_i);
    }

    /* Fig. 3a (selection): INT only if strictly better; Sec. 3: the choice is
     * recorded in the scale's sign bit.  NVINT4 always stores INT codes and
     * its scale is a plain E4M3 value (bit 7 clear). */
    int use_int = f->adaptive && (sel_i < sel_f);
    if (f->kind == KIND_INT) {
        memcpy(codes, ci, (size_t)n);
        *scale = (uint8_t)dcode;
    } else {
        memcpy(codes, use_int ? ci : cf, (size_t)n);
        *scale = (uint8_t)(dcode | (use_int ? 0x80 : 0));
    }
    *e_fp = sel_f;
    *e_int = sel_i;
}

/* Dense little-endian bit stream: code j of a group at bits [j*b, j*b+b);
 * a group of n codes fills n*b/8 bytes. */
static void pack_group(int bits, int n, const uint8_t codes[GROUP], uint8_t* out)
{
    memset(out, 0, (size_t)(n * bits / 8));
    for (int j = 0; j < n; ++j) {
        for (int t = 0; t < bits; ++t) {
            int bit = j * bits + t;
            if ((codes[j] >> t) & 1) out[bit >> 3] |= (uint8_t)(1u << (bit & 7));
        }
    }
}

static void unpack_group(int bits, int n, const uint8_t* in, uint8_t codes[GROUP])
{
    for (int j = 0; j < n; ++j) {
        int c = 0;
        for (int t = 0; t < bits; ++t) {
            int bit = j * bits + t;
            c |= ((in[bit >> 3] >> (bit & 7)) & 1) << t;
        }
        codes[j] = (uint8_t)c;
    }
}

void oracle_pack_group(int fmt, const uint8_t codes[GROUP], uint8_t* out)
{
    ensure_init();
    pack_group(g_fmt[fmt].bits, g_fmt[fmt].gsize, codes, out);
}

void oracle_unpack_group(int fmt, const uint8_t* in, uint8_t codes[GROUP])
{
    ensure_init();
    unpack_group(g_fmt[fmt].bits, g_fmt[fmt].gsize, in, codes);
}

static float bf16_to_float(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

/* ------------------------------------------------------ whole tensor -- */

/* Quantize a bf16 matrix x (rows x cols, row stride ld_x elements).
 * Row-wise: groups of 16 run along cols; codes are [rows, cols*bits/8],
 * scales [rows, cols/16].  With F_STRIDED the groups run along rows and the
 * output describes the transposed matrix: codes [cols, rows*bits/8], scales
 * [cols, rows/16].  tensor_scale is written (or read with F_SCALE_IN).
 * Returns 0, or -1 on bad arguments.  Non-finite inputs are rejected. */
int oracle_quantize(int fmt, const uint16_t* x, int64_t rows, int64_t cols, int64_t ld_x,
                    uint32_t flags, uint32_t rht_signs, uint64_t seed, uint8_t* codes,
                    uint8_t* scales, float* tensor_scale)
{
    ensure_init();
    if (fmt < 0 || fmt >= FMT_COUNT) return -1;
    const fmt_desc* f = &g_fmt[fmt];
    const int n = f->gsize;
    const int strided = (flags & F_STRIDED) != 0;
    const int64_t out_rows = strided ? cols : rows;   /* logical rows of the output */
    const int64_t out_k = strided ? rows : cols;      /* grouped (K) dimension */
    if (out_k % GROUP) return -1;
    const int64_t bpr = out_k / GROUP;                /* 16-value blocks (RHT blocks) per row */
    const int64_t gpr = out_k / n;                    /* groups (scale bytes) per row */
    const int64_t ngroups = out_rows * gpr;
    const int64_t code_bytes_row = out_k * f->bits / 8;

    /* Gather each 16-value block (and transform it) into a dense fp32
     * buffer in output order. */
    float* vbuf = (float*)malloc((size_t)(out_rows * out_k > 0 ? out_rows * out_k : 1) * sizeof(float));
    if (!vbuf) return -1;
    float amax = 0.0f;
    for (int64_t o = 0; o < out_rows; ++o) {
        for (int64_t b = 0; b < bpr; ++b) {
            float xg[GROUP];
            for (int j = 0; j < GROUP; ++j) {
                int64_t k = b * GROUP + j;
                int64_t r = strided ? k : o, c = strided ? o : k;
                xg[j] = bf16_to_float(x[r * ld_x + c]);
                if (!isfinite(xg[j])) {
                    free(vbuf);
                    return -1;
                }
            }
            float* v = vbuf + o * out_k + b * GROUP;
            if (flags & F_RHT)
                oracle_rht16(xg, rht_signs, v);
            else
                memcpy(v, xg, sizeof(xg));
            for (int j = 0; j < GROUP; ++j) {
                float a = fabsf(v[j]);
                if (a > amax) amax = a;
            }
        }
    }

    /* Eq. (1), unless the caller supplies alpha. */
    float alpha = (flags & F_SCALE_IN) ? *tensor_scale : oracle_tensor_scale(fmt, amax, flags);
    if (!(flags & F_SCALE_IN)) *tensor_scale = alpha;

    /* Group gi (the index of its scale byte) draws its SR numbers from the
     * Philox blocks of counter gi; a group of 8 uses the first 8. */
    for (int64_t o = 0; o < out_rows; ++o) {
        for (int64_t g = 0; g < gpr; ++g) {
            int64_t gi = o * gpr + g;
            uint16_t h[GROUP];
            if (flags & F_SR)
                oracle_sr_bits(seed, (uint64_t)gi, h);
            else
                memset(h, 0, sizeof(h));
            uint8_t cg[GROUP], sb;
            float ef, ei;
            oracle_quantize_group(fmt, vbuf + o * out_k + g * n, alpha, flags, h, cg, &sb, &ef, &ei);
            scales[gi] = sb;
            pack_group(f->bits, n, cg, codes + o * code_bytes_row + g * n * f->bits / 8);
        }
    }
    (void)ngroups;
    free(vbuf);
    return 0;
}

/* Dequantized value of one element (Fig. 3a's dequantized values with alpha):
 * q * Delta, times M_FP/M_I for INT groups of the IF formats (1 for
 * NVINT4), times alpha, each step an fp32
 * multiply in that order (q * Delta is exact). */
static float dequant_element(const fmt_desc* f, uint8_t code, uint8_t sbyte, float alpha)
{
    float delta = (float)oracle_e4m3_value(sbyte & 0x7F);
    int is_int = f->kind == KIND_INT || (f->adaptive && (sbyte & 0x80));
    float q;
    if (is_int) {
        int c = code;
        if (c & (1 << (f->bits - 1))) c -= (1 << f->bits); /* two's complement */
        q = (float)c;
    } else {
        int idx = code & (f->n_mag - 1);
        q = (float)f->mag[idx];
        if (code & f->n_mag) q = -q;
    }
    float t = q * delta;
    if (is_int) t = t * f->k_dn;
    return t * alpha;
}

/* codes/scales as written by oracle_quantize (row-wise layout of the
 * logical [rows, cols] tensor); out is fp32 [rows, cols]. */
int oracle_dequantize(int fmt, const uint8_t* codes, const uint8_t* scales, float alpha,
                      int64_t rows, int64_t cols, float* out)
{
    ensure_init();
    if (fmt < 0 || fmt >= FMT_COUNT || cols % GROUP) return -1;
    const fmt_desc* f = &g_fmt[fmt];
    const int n = f->gsize;
    const int64_t gpr = cols / n;
    const int64_t code_bytes_row = cols * f->bits / 8;
    for (int64_t r = 0; r < rows; ++r) {
        for (int64_t g = 0; g < gpr; ++g) {
            uint8_t cg[GROUP];
            unpack_group(f->bits, n, codes + r * code_bytes_row + g * n * f->bits / 8, cg);
            uint8_t sb = scales[r * gpr + g];
            for (int j = 0; j < n; ++j)
                out[r * cols + g * n + j] = dequant_element(f, cg[j], sb, alpha);
        }
    }
    return 0;
}

/* Exact dequantized values in fp64: alpha * Delta * q * (M_FP/M_I for INT
 * groups), with M_FP/M_I as the fp64 nearest to the rational.  Used as the
 * operands of the fp64 GEMM reference. */
int oracle_dequantize_f64(int fmt, const uint8_t* codes, const uint8_t* scales, float alpha,
                          int64_t rows, int64_t cols, double* out)
{
    ensure_init();
    if (fmt < 0 || fmt >= FMT_COUNT || cols % GROUP) return -1;
    const fmt_desc* f = &g_fmt[fmt];
    const int n = f->gsize;
    const int64_t gpr = cols / n;
    const int64_t code_bytes_row = cols * f->bits / 8;
    const double kdn = f->kind == KIND_INT ? 1.0 : (double)f->fp_max / (double)f->int_max;
    for (int64_t r = 0; r < rows; ++r) {
        for (int64_t g = 0; g < gpr; ++g) {
            uint8_t cg[GROUP];
            unpack_group(f->bits, n, codes + r * code_bytes_row + g * n * f->bits / 8, cg);
            uint8_t sb = scales[r * gpr + g];
            double delta = oracle_e4m3_value(sb & 0x7F);
            int is_int = f->kind == KIND_INT || (f->adaptive && (sb & 0x80));
            for (int j = 0; j < n; ++j) {
                double q;
                if (is_int) {
                    int c = cg[j];
                    if (c & (1 << (f->bits - 1))) c -= (1 << f->bits);
                    q = (double)c * kdn;
                } else {
                    q = f->mag[cg[j] & (f->n_mag - 1)];
                    if (cg[j] & f->n_mag) q = -q;
                }
                out[r * cols + g * n + j] = (double)alpha * delta * q;
            }
        }
    }
    return 0;
}
