/* Arithmetic identities the quantizer kernels rely on, checked on the CPU
 * in IEEE binary32 (build with -ffp-contract=off; fmaf is the fused
 * multiply-add).  Test infrastructure: it restates the kernels' formulas
 * next to the straightforward ones and counts differences.
 *
 *   sr   : stochastic rounding with a 16-bit draw u = h / 2^16.
 *          Straightforward: lo = floor(t) (on the format's grid), up iff
 *          u * step < m - lo.  Kernel: ceil(t - u) with t = m / step.
 *          Grids: E2M1 (IF4/NVFP4 FP), E2M3 and E3M2 (IF6), E2M0 (IF3),
 *          and the INT candidates (|y| rounded, clamped to 7, 31, 3).
 *   div  : the scale quotient a / d by Markstein's correction
 *          q0 = a r, e = fma(-d, q0, a), q = fma(e, r, q0), r = RN(1/d),
 *          against the correctly rounded division (a >= 2^-100, d and 1/d
 *          normal): equal wherever the E4M3 encoder distinguishes values;
 *          where the true quotient exceeds 448 the clamped one is 448 (an
 *          overflow gives inf or NaN, both clamped to 448), and where it is
 *          below 2^-10 (code 0) so is the corrected one.
 *
 * usage: kernel_identities <sr|div> <stride>   (stride 1 = every value)
 * prints "checks N mismatches M" and exits 1 on any mismatch. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

static float f_of(uint32_t u) { float x; memcpy(&x, &u, 4); return x; }
static uint32_t u_of(float x) { uint32_t u; memcpy(&u, &x, 4); return u; }

/* grid of an ExMy format: MB mantissa bits, exponent bias BIAS, max FMAX */
typedef struct { int mb, bias; float fmax; } Grid;

static int sr_index_plain(float m, float u, Grid g)
{
    m = fminf(m, g.fmax);
    int e = (int)((u_of(m) >> 23) & 0xFF) - 127;
    int ee = e > 1 - g.bias ? e : 1 - g.bias;
    float q = f_of((uint32_t)(127 + ee - g.mb) << 23), inv_q = f_of((uint32_t)(127 - (ee - g.mb)) << 23);
    float lo_r = floorf(m * inv_q), lo = lo_r * q;
    int r = (int)lo_r + ((u * q < m - lo) ? 1 : 0);
    return ((ee + g.bias) << g.mb) + r - (1 << g.mb);
}

static int sr_index_ceil(float m, float u, Grid g)
{
    m = fminf(m, g.fmax);
    int e = (int)((u_of(m) >> 23) & 0xFF) - 127;
    int ee = e > 1 - g.bias ? e : 1 - g.bias;
    float inv_q = f_of((uint32_t)(127 - (ee - g.mb)) << 23);
    volatile float t = m * inv_q;
    volatile float d = t - u;
    return ((ee + g.bias) << g.mb) + (int)ceilf(d) - (1 << g.mb);
}

/* E2M1 magnitude as the IF4/NVFP4 SR kernel forms it (step from m's binade) */
static float e2m1_plain(float m, float u)
{
    m = fminf(m, 6.0f);
    float p2 = f_of(u_of(m) & 0x7F800000u), q = fmaxf(p2 * 0.5f, 0.5f);
    float inv_q = f_of((254u << 23) - u_of(q)), lo = floorf(m * inv_q) * q;
    return (u * q < m - lo) ? lo + q : lo;
}

static float e2m1_ceil(float m, float u)
{
    m = fminf(m, 6.0f);
    float p2 = f_of(u_of(m) & 0x7F800000u), q = fmaxf(p2 * 0.5f, 0.5f);
    float inv_q = f_of((254u << 23) - u_of(q));
    volatile float t = m * inv_q;
    volatile float d = t - u;
    volatile float c = ceilf(d);
    return fabsf(c * q);
}

static float int_plain(float a, float u, float imax)
{
    float il = floorf(a);
    return fminf((u < a - il) ? il + 1.0f : il, imax);
}

static float int_ceil(float a, float u, float imax)
{
    volatile float d = a - u;
    return fabsf(fminf(ceilf(d), imax));
}

static long checks, bad;

static void report(const char* what, double x, double u)
{
    if (bad < 5) printf("mismatch %s x=%a u=%a\n", what, x, u);
    ++bad;
}

/* draws at, just below and above the fraction of t, plus 0, the maximum and one more */
static int draws(double t, float* u)
{
    int h0 = (int)floor((t - floor(t)) * 65536.0), n = 0;
    int cand[6] = {0, 65535, h0 - 1, h0, h0 + 1, (h0 * 7919 + 12345) & 0xFFFF};
    for (int k = 0; k < 6; ++k)
        if (cand[k] >= 0 && cand[k] <= 65535) u[n++] = (float)cand[k] * (1.0f / 65536.0f);
    return n;
}

static void check_sr(uint32_t stride)
{
    const Grid grids[4] = {{1, 1, 6.0f}, {3, 1, 7.5f}, {2, 3, 28.0f}, {0, 1, 4.0f}};
    const float imaxes[4] = {7.0f, 31.0f, 31.0f, 3.0f};
    for (int gi = 0; gi < 4; ++gi) {
        const Grid g = grids[gi];
        const uint32_t top = u_of(g.fmax * 1.1f), itop = u_of(imaxes[gi] + 0.9f);
        for (uint32_t b = 0; b <= top; b += stride) {
            float m = f_of(b), u[6];
            float mm = fminf(m, g.fmax);
            int e = (int)((u_of(mm) >> 23) & 0xFF) - 127;
            int ee = e > 1 - g.bias ? e : 1 - g.bias;
            int n = draws(ldexp((double)mm, -(ee - g.mb)), u);
            for (int k = 0; k < n; ++k) {
                ++checks;
                if (sr_index_plain(m, u[k], g) != sr_index_ceil(m, u[k], g)) report("grid", m, u[k]);
                if (gi == 0) {
                    ++checks;
                    if (u_of(e2m1_plain(m, u[k])) != u_of(e2m1_ceil(m, u[k]))) report("e2m1", m, u[k]);
                }
            }
        }
        for (uint32_t b = 0; b <= itop; b += stride) {
            float a = f_of(b), u[6];
            int n = draws((double)a, u);
            for (int k = 0; k < n; ++k) {
                ++checks;
                if (u_of(int_plain(a, u[k], imaxes[gi])) != u_of(int_ceil(a, u[k], imaxes[gi])))
                    report("int", a, u[k]);
            }
        }
    }
}

static void check_div(uint32_t stride)
{
    /* divisor significands: all-ones tails, neighbours of powers of two, pseudo-random */
    uint32_t sig[160];
    int ns = 0;
    for (int k = 0; k < 24; ++k) {
        sig[ns++] = (1u << k) - 1u;
        sig[ns++] = 0x7FFFFFu & ~((1u << k) - 1u);
    }
    sig[ns++] = 1u;
    sig[ns++] = 0x7FFFFEu;
    uint32_t st = 12345u;
    while (ns < 160) {
        st = st * 1664525u + 1013904223u;
        sig[ns++] = st >> 9;
    }
    const int dexp[3] = {-100, 0, 100};   /* divisor exponents, normal reciprocals */
    const int aexp[4] = {-100, -1, 0, 60}; /* dividend exponents, a >= 2^-100 */
    for (int i = 0; i < ns; ++i)
        for (int de = 0; de < 3; ++de) {
            const float d = f_of(((uint32_t)(127 + dexp[de]) << 23) | sig[i]);
            const float r = 1.0f / d;
            for (uint32_t m = (uint32_t)i % stride; m < (1u << 23); m += stride)
                for (int ae = 0; ae < 4; ++ae) {
                    const float a = f_of(((uint32_t)(127 + aexp[ae]) << 23) | m);
                    const float q0 = a * r, e = fmaf(-d, q0, a), q = fmaf(e, r, q0);
                    const float t = a / d;
                    ++checks;
                    /* what the encoder consumes: min(q, 448) (NaN -> 448); below
                     * 2^-10 every value encodes to code 0 */
                    if (t > 448.0f ? fminf(q, 448.0f) != 448.0f
                                   : t < 0x1p-10f ? !(q < 0x1p-10f) : u_of(q) != u_of(t))
                        report("div", a, d);
                }
        }
}

int main(int argc, char** argv)
{
    if (argc < 3) return 2;
    const uint32_t stride = (uint32_t)strtoul(argv[2], 0, 10);
    if (!strcmp(argv[1], "sr")) check_sr(stride ? stride : 1);
    else if (!strcmp(argv[1], "div")) check_div(stride ? stride : 1);
    else return 2;
    printf("checks %ld mismatches %ld\n", checks, bad);
    return bad != 0;
}
