/*
 * Host sanitizer driver for the C oracle (built by tests/test_sanitizers.py
 * with gcc -fsanitize=address,undefined and linked with oracle/q2d_oracle.c).
 *
 * Every output buffer is allocated at exactly the size its layout needs, so a
 * write one byte past a row, a scale grid or a 1D scale-word array is caught.
 * Inputs are seeded bf16 / fp32 matrices with boundary blocks, zero blocks,
 * subnormals and non-finite values, read both directly and through a
 * transposed strided view.  Beyond memory safety the driver checks that the
 * two stored orientations hold the same nibbles (the transposition
 * invariance of 2D blocks) and exits non-zero on any mismatch.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

void or_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]);
uint32_t or_sr_bits(int64_t idx, uint64_t seed, uint64_t offset);
int or_fp4_scale_exponent(double M);
int or_fp4_floor_exponent(double M);
int or_fp8_scale_exponent(double M);
unsigned or_fp4_code(double x, int e, int stochastic, uint32_t r16);
unsigned or_e4m3_code(double x, int e);
void or_quantize_fp4_2d(const void *x, int dtype, int64_t R, int64_t C, int64_t sr, int64_t sc,
                        int64_t idx0, int b, int mode, uint64_t seed, uint64_t offset,
                        uint8_t *codes, int64_t ldc, uint8_t *codes_t, int64_t ldt,
                        uint8_t *scales, int64_t lds, uint8_t *scales_t, int64_t ldst,
                        int nthreads);
void or_quantize_fp4_1d(const void *x, int dtype, int64_t R, int64_t C, int64_t sr, int64_t sc,
                        int mode, uint64_t seed, uint64_t offset,
                        uint8_t *codes, int64_t ldc, uint8_t *scales, int64_t lds,
                        uint8_t *codes_t, int64_t ldt, uint8_t *scales_t, int64_t ldst,
                        int nthreads);
void or_quantize_mxfp8(const void *x, int dtype, int64_t R, int64_t C, int64_t sr, int64_t sc,
                       uint8_t *codes, int64_t ldc, uint8_t *scales, int64_t lds,
                       uint8_t *codes_t, int64_t ldt, uint8_t *scales_t, int64_t ldst,
                       int nthreads);
void or_fp4_codes(const double *x, const int *e, const uint32_t *r16, int stochastic,
                  int64_t n, uint8_t *out);
void or_e4m3_codes(const double *x, const int *e, int64_t n, uint8_t *out);

static int failures = 0;
#define CHECK(cond, ...) do { if (!(cond)) { fprintf(stderr, __VA_ARGS__); fputc('\n', stderr); ++failures; } } while (0)

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static uint32_t rnd(void)      /* xorshift64*: input generation only */
{
    rng_state ^= rng_state >> 12; rng_state ^= rng_state << 25; rng_state ^= rng_state >> 27;
    return (uint32_t)((rng_state * 0x2545F4914F6CDD1Dull) >> 32);
}

static float sample(int64_t i)
{
    switch (rnd() % 16) {
    case 0: return 0.0f;
    case 1: return ldexpf((float)(rnd() % 1000), -140);          /* subnormal fp32 */
    case 2: return (i % 97 == 0) ? INFINITY : 1.0f;
    case 3: return (i % 89 == 0) ? NAN : -2.0f;
    default: return ldexpf((float)((int32_t)rnd()) / 2147483648.0f, (int)(rnd() % 40) - 20);
    }
}

static void *make_input(int dtype, int64_t n)
{
    if (dtype == 0) {
        float *x = malloc((size_t)n * 4);
        for (int64_t i = 0; i < n; ++i) x[i] = sample(i);
        return x;
    }
    uint16_t *x = malloc((size_t)n * 2);
    for (int64_t i = 0; i < n; ++i) {
        float f = sample(i);
        uint32_t b;
        memcpy(&b, &f, 4);
        x[i] = (uint16_t)(b >> 16);
    }
    return x;
}

static unsigned nib(const uint8_t *row, int64_t pos) { return (row[pos >> 1] >> (4 * (pos & 1))) & 15u; }

/* 2D FP4 (block b) of x read directly and of its stored transpose read through a view */
static void run_2d(int dtype, int64_t R, int64_t C, int b, int mode)
{
    const int64_t n = R * C, nbr = (R + b - 1) / b, nbc = (C + b - 1) / b;
    void *x = make_input(dtype, n);
    const int64_t ldc = (C + 1) / 2, ldt = (R + 1) / 2;
    uint8_t *codes = calloc((size_t)(R * ldc), 1), *codes_t = calloc((size_t)(C * ldt), 1);
    uint8_t *scales = calloc((size_t)(nbr * nbc), 1), *scales_t = calloc((size_t)(nbc * nbr), 1);
    or_quantize_fp4_2d(x, dtype, R, C, C, 1, 0, b, mode, 7, 3, codes, ldc, codes_t, ldt,
                       scales, nbc, scales_t, nbr, 2);
    for (int64_t r = 0; r < R; ++r)
        for (int64_t c = 0; c < C; ++c)
            CHECK(nib(codes + r * ldc, c) == nib(codes_t + c * ldt, r),
                  "2d dtype %d %lldx%lld b%d mode %d: orientations differ at (%lld, %lld)", dtype,
                  (long long)R, (long long)C, b, mode, (long long)r, (long long)c);
    for (int64_t I = 0; I < nbr; ++I)
        for (int64_t J = 0; J < nbc; ++J)
            CHECK(scales[I * nbc + J] == scales_t[J * nbr + I], "2d scales differ at block (%lld, %lld)",
                  (long long)I, (long long)J);
    /* the C x R transpose as a strided view of the same storage (the stochastic
       draws are keyed by storage index, which the view keeps) */
    uint8_t *vcodes = calloc((size_t)(C * ldt), 1), *vcodes_t = calloc((size_t)(R * ldc), 1);
    uint8_t *vscales = calloc((size_t)(nbc * nbr), 1), *vscales_t = calloc((size_t)(nbr * nbc), 1);
    or_quantize_fp4_2d(x, dtype, C, R, 1, C, 0, b, mode, 7, 3, vcodes, ldt, vcodes_t, ldc,
                       vscales, nbr, vscales_t, nbc, 2);
    CHECK(memcmp(vcodes, codes_t, (size_t)(C * ldt)) == 0 && memcmp(vcodes_t, codes, (size_t)(R * ldc)) == 0,
          "2d transposed view: layouts not swapped (dtype %d %lldx%lld b%d mode %d)", dtype,
          (long long)R, (long long)C, b, mode);
    CHECK(memcmp(vscales, scales_t, (size_t)(nbc * nbr)) == 0, "2d transposed view: scales");
    /* one orientation only (the other pointers NULL), as a grouped segment */
    memset(codes, 0, (size_t)(R * ldc));
    or_quantize_fp4_2d(x, dtype, R, C, C, 1, 12345, b, mode, 7, 3, codes, ldc, NULL, 0,
                       scales, nbc, NULL, 0, 1);
    free(vcodes); free(vcodes_t); free(vscales); free(vscales_t);
    free(codes); free(codes_t); free(scales); free(scales_t); free(x);
}

/* 1D FP4: scale words of K-tiles of 128, byte J % 4 of word (J / 4, r) */
static void run_1d(int dtype, int64_t R, int64_t C, int mode)
{
    void *x = make_input(dtype, R * C);
    const int64_t ldc = (C + 1) / 2, ldt = (R + 1) / 2;
    const int64_t wr = ((C + 31) / 32 + 3) / 4, wc = ((R + 31) / 32 + 3) / 4;   /* word rows */
    uint8_t *codes = calloc((size_t)(R * ldc), 1), *codes_t = calloc((size_t)(C * ldt), 1);
    uint8_t *scales = calloc((size_t)(wr * 4 * R), 1), *scales_t = calloc((size_t)(wc * 4 * C), 1);
    or_quantize_fp4_1d(x, dtype, R, C, C, 1, mode, 11, 5, codes, ldc, scales, 4 * R,
                       codes_t, ldt, scales_t, 4 * C, 2);
    free(codes); free(codes_t); free(scales); free(scales_t); free(x);
}

static void run_mxfp8(int dtype, int64_t R, int64_t C)
{
    void *x = make_input(dtype, R * C);
    const int64_t nbc = (C + 31) / 32, nbr = (R + 31) / 32;
    uint8_t *codes = calloc((size_t)(R * C), 1), *codes_t = calloc((size_t)(C * R), 1);
    uint8_t *scales = calloc((size_t)(R * nbc), 1), *scales_t = calloc((size_t)(C * nbr), 1);
    or_quantize_mxfp8(x, dtype, R, C, C, 1, codes, C, scales, nbc, codes_t, R, scales_t, nbr, 2);
    free(codes); free(codes_t); free(scales); free(scales_t); free(x);
}

int main(void)
{
    static const int64_t shapes[][2] = {{1, 1}, {1, 33}, {33, 1}, {31, 65}, {97, 130}, {64, 64}, {129, 257}};
    const int ns = (int)(sizeof(shapes) / sizeof(shapes[0]));
    for (int s = 0; s < ns; ++s)
        for (int dtype = 0; dtype < 2; ++dtype) {
            for (int mode = 0; mode < 4; ++mode) {
                run_2d(dtype, shapes[s][0], shapes[s][1], 32, mode);
                run_2d(dtype, shapes[s][0], shapes[s][1], 64, mode & 1);
            }
            run_1d(dtype, shapes[s][0], shapes[s][1], 0);
            run_1d(dtype, shapes[s][0], shapes[s][1], 1);
            run_mxfp8(dtype, shapes[s][0], shapes[s][1]);
        }
    /* scalar codecs over extreme exponents and arguments */
    static const double ms[] = {0.0, 4.9e-324, 1e-300, 1.5, 6.0, 6.000001, 1e30, 3.4e38, 1e300};
    for (int i = 0; i < (int)(sizeof(ms) / sizeof(ms[0])); ++i) {
        int e = or_fp4_scale_exponent(ms[i]), f = or_fp4_floor_exponent(ms[i]), g = or_fp8_scale_exponent(ms[i]);
        CHECK(e >= -127 && e <= 127 && f >= -127 && f <= 127 && g >= -127 && g <= 127, "exponent range");
        for (int k = -127; k <= 127; k += 127) {
            (void)or_fp4_code(ms[i], k, 0, 0);
            (void)or_fp4_code(-ms[i], k, 1, 0xFFFFu);
            (void)or_e4m3_code(ms[i], k);
        }
    }
    double xs[4] = {0.25, -7.0, 1e-40, 3.0};
    int es[4] = {-127, 0, 127, -1};
    uint32_t rs[4] = {0, 65535, 1, 32768};
    uint8_t out[4];
    or_fp4_codes(xs, es, rs, 1, 4, out);
    or_fp4_codes(xs, es, NULL, 0, 4, out);
    or_e4m3_codes(xs, es, 4, out);
    uint32_t ctr[4] = {0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu}, key[2] = {0xFFFFFFFFu, 0}, w[4];
    or_philox4x32_10(ctr, key, w);
    (void)or_sr_bits(INT64_MAX, UINT64_MAX, UINT64_MAX);
    if (failures) {
        fprintf(stderr, "%d check(s) failed\n", failures);
        return 1;
    }
    printf("sanitize_oracle: ok\n");
    return 0;
}
