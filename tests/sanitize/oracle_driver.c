/* Sanitizer driver for the CPU oracle (test infrastructure): built with
 * -fsanitize=address,undefined and run by tests/test_sanitizers_cpu.py.  It
 * calls every exported oracle function over every format and flag set on
 * seeded inputs (ragged, strided, degenerate and tiny-valued tensors,
 * exact sizes for every buffer), so an out-of-bounds access or undefined
 * behaviour in the oracle stops the run with a report. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

double oracle_e4m3_value(int code);
int oracle_e4m3_encode(float x);
int oracle_fp_round_index(int fmt, float m);
double oracle_fp_magnitude(int fmt, int idx);
int oracle_group_size(int fmt);
void oracle_fmt_constants(int fmt, float* fp_max, int* int_max, float* c_up, float* k_dn, int* bits);
void oracle_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]);
void oracle_sr_bits(uint64_t seed, uint64_t group, uint16_t h[16]);
void oracle_rht16(const float x[16], uint32_t signs, float v[16]);
float oracle_tensor_scale(int fmt, float amax, uint32_t flags);
void oracle_quantize_group(int fmt, const float v[16], float alpha, uint32_t flags, const uint16_t h[16],
                           uint8_t codes[16], uint8_t* scale, float* ef, float* ei);
void oracle_pack_group(int fmt, const uint8_t codes[16], uint8_t* out);
void oracle_unpack_group(int fmt, const uint8_t* in, uint8_t codes[16]);
int oracle_quantize(int fmt, const uint16_t* x, int64_t rows, int64_t cols, int64_t ld_x, uint32_t flags,
                    uint32_t rht_signs, uint64_t seed, uint8_t* codes, uint8_t* scales, float* tensor_scale);
int oracle_dequantize(int fmt, const uint8_t* codes, const uint8_t* scales, float alpha, int64_t rows,
                      int64_t cols, float* out);
int oracle_dequantize_f64(int fmt, const uint8_t* codes, const uint8_t* scales, float alpha, int64_t rows,
                          int64_t cols, double* out);

enum { NFMT = 10 };
static const int kBits[NFMT] = {4, 4, 3, 6, 6, 4, 4, 4, 3, 4};

static uint64_t rng = 0x9E3779B97F4A7C15ull;
static uint32_t next32(void)
{
    rng ^= rng << 13; rng ^= rng >> 7; rng ^= rng << 17;
    return (uint32_t)(rng >> 16);
}

/* bf16 bits of a finite value: a random magnitude spread over many binades */
static uint16_t rand_bf16(int wide)
{
    float v = ((float)(next32() & 0xFFFFFF) / 16777216.0f - 0.5f) * 8.0f;
    if (wide) v = ldexpf(v, (int)(next32() % 60) - 30);
    uint32_t u;
    memcpy(&u, &v, 4);
    return (uint16_t)(u >> 16);
}

static int check_tensor(int fmt, int64_t rows, int64_t cols, uint32_t flags, int wide)
{
    const int strided = (flags & 16u) != 0;
    const int64_t R = strided ? cols : rows, K = strided ? rows : cols;
    const int g = oracle_group_size(fmt);
    uint16_t* x = malloc((size_t)(rows * cols > 0 ? rows * cols : 1) * 2);
    uint8_t* codes = malloc((size_t)(R * K * kBits[fmt] / 8 > 0 ? R * K * kBits[fmt] / 8 : 1));
    uint8_t* scales = malloc((size_t)(R * (K / g) > 0 ? R * (K / g) : 1));
    float* out = malloc((size_t)(R * K > 0 ? R * K : 1) * sizeof(float));
    double* out64 = malloc((size_t)(R * K > 0 ? R * K : 1) * sizeof(double));
    if (!x || !codes || !scales || !out || !out64) return 1;
    for (int64_t i = 0; i < rows * cols; ++i) x[i] = rand_bf16(wide);
    float ts = (flags & 8u) ? 0.0123f : 0.0f;
    int rc = oracle_quantize(fmt, x, rows, cols, cols, flags, 0xA5C3, 77, codes, scales, &ts);
    if (rc == 0) {
        rc |= oracle_dequantize(fmt, codes, scales, ts, R, K, out);
        rc |= oracle_dequantize_f64(fmt, codes, scales, ts, R, K, out64);
    }
    free(x); free(codes); free(scales); free(out); free(out64);
    return rc;
}

int main(void)
{
    int fails = 0;
    for (int c = 0; c < 128; ++c) (void)oracle_e4m3_value(c);
    for (int i = 0; i < 4096; ++i) {
        float v = (float)i * 0.125f;
        (void)oracle_e4m3_encode(v);
        (void)oracle_e4m3_encode(ldexpf(v, -20));
    }
    for (int fmt = 0; fmt < NFMT; ++fmt) {
        float fm, cu, kd;
        int im, b;
        oracle_fmt_constants(fmt, &fm, &im, &cu, &kd, &b);
        for (int i = 0; i < 64; ++i) (void)oracle_fp_round_index(fmt, (float)i * 0.25f);
        for (int i = 0; i < (1 << (kBits[fmt] - 1)); ++i) (void)oracle_fp_magnitude(fmt, i);
        for (uint32_t fl = 0; fl < 8; ++fl) (void)oracle_tensor_scale(fmt, 3.5f, fl);
        uint8_t cg[16], packed[16], back[16];
        for (int j = 0; j < 16; ++j) cg[j] = (uint8_t)(next32() & ((1u << kBits[fmt]) - 1));
        oracle_pack_group(fmt, cg, packed);
        oracle_unpack_group(fmt, packed, back);
        float v[16];
        uint16_t h[16];
        for (int j = 0; j < 16; ++j) { v[j] = (float)(int)(next32() % 200) - 100.0f; h[j] = (uint16_t)next32(); }
        for (uint32_t fl = 0; fl < 64; ++fl) {
            uint8_t sb;
            float ef, ei;
            oracle_quantize_group(fmt, v, 0.01f, fl & ~16u, h, cg, &sb, &ef, &ei);
        }
        /* every flag set, row-wise and strided, ragged and degenerate shapes */
        const int64_t shapes[][2] = {{16, 16}, {48, 32}, {3, 80}, {32, 48}, {0, 16}, {16, 0}, {1, 16}};
        for (uint32_t fl = 0; fl < 64; ++fl) {
            for (size_t si = 0; si < sizeof(shapes) / sizeof(shapes[0]); ++si) {
                int64_t r = shapes[si][0], cc = shapes[si][1];
                if ((fl & 16u) ? (r % 16) : (cc % 16)) continue;
                if (check_tensor(fmt, r, cc, fl, (int)(si & 1))) {
                    fprintf(stderr, "oracle rejected fmt %d flags %u shape %lldx%lld\n", fmt, fl,
                            (long long)r, (long long)cc);
                    ++fails;
                }
            }
        }
    }
    uint32_t ctr[4] = {1, 2, 3, 4}, key[2] = {5, 6}, out[4];
    oracle_philox4x32_10(ctr, key, out);
    uint16_t h[16];
    oracle_sr_bits(0xFFFFFFFFFFFFFFFFull, 0x123456789ull, h);
    float x[16], y[16];
    for (int j = 0; j < 16; ++j) x[j] = (float)j - 7.5f;
    oracle_rht16(x, 0xFFFF, y);
    /* rejected arguments: non-finite input, K not a multiple of 16 */
    uint16_t bad[32];
    for (int j = 0; j < 32; ++j) bad[j] = 0x3F80;
    bad[5] = 0x7FC0;
    uint8_t cb[32], sbuf[2];
    float ts = 0;
    if (oracle_quantize(0, bad, 1, 32, 32, 0, 0, 0, cb, sbuf, &ts) != -1) ++fails;
    if (oracle_quantize(0, bad, 1, 24, 24, 0, 0, 0, cb, sbuf, &ts) != -1) ++fails;
    printf("oracle driver: %d failures\n", fails);
    return fails != 0;
}
