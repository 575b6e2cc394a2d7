/*
 * CPU oracle for transposition-invariant 2D-block FP4 quantization and its
 * MXFP8 companion.  TEST INFRASTRUCTURE ONLY: it is called by the tests, by
 * the smoke check and by the benchmark's CPU-baseline leg, never by the
 * product path.  It shares no code, header or table with the HIP library.
 *
 * Everything here is written as the plain definition, in double precision,
 * one element at a time:
 *
 *   - Blocks: b x b squares B_ij = X[ib:(i+1)b, jb:(j+1)b]; boundary blocks
 *     use their valid entries only (App. D, "Boundary blocks").
 *   - Block maximum M_ij = max |x| over the block (App. D).
 *   - Truncation-free scale S = 2^ceil(log2(2M / (Qp - Qn))) with the E2M1
 *     bounds Qp = 6, Qn = -6 (Sec. 3.1; App. D), i.e. the smallest power of
 *     two with 6 * S >= M.  Stored as the E8M0 byte e + 127.
 *   - Quantized block S * round_FP4(B / S) (App. D) with round-to-nearest on
 *     forward operands and stochastic rounding with E[round(x)] = x on
 *     gradients (Sec. 3.1; App. E).
 *   - MXFP8 for the Q/K path (Sec. 3.2; App. C): 1x32 blocks, E4M3 elements,
 *     the same truncation-free rule with Qp = 448.
 *   - 1D FP4 for activations (Sec. 3; App. C): 1x32 and 32x1 blocks with the
 *     FP4 scale rule and codec.
 *
 * Readings of what the paper leaves open (each is listed in the design notes):
 *   - the FP4 grid is OCP E2M1, magnitudes {0, .5, 1, 1.5, 2, 3, 4, 6};
 *   - M = 0 gives e = -127 (byte 0x00); e is clamped to [-127, 127];
 *   - a block holding a NaN or an infinity gets scale byte 0xFF and all-zero codes;
 *   - round-to-nearest breaks ties to the even E2M1 code; the sign bit of the
 *     input is kept even when the magnitude rounds to zero;
 *   - stochastic rounding uses 16 random bits per element from Philox4x32-10:
 *     for storage index i (elements from the base pointer), counter
 *     (g lo, g hi, offset lo, offset hi) with g = i >> 3, key (seed lo, seed hi),
 *     r16 = 16-bit half (i & 1) of output word (i & 7) >> 1; the magnitude
 *     rounds up iff floor(2^16 * d / delta) + r16 >= 2^16 where d is the distance
 *     to the grid point below and delta the grid spacing.
 *
 * Philox4x32-10 follows its published definition (Salmon, Moraes, Dror, Shaw,
 * "Parallel random numbers: as easy as 1, 2, 3", SC 2011).
 *
 * Layouts (shared with the library's contract, not with its code):
 *   codes   [R][ldc]: byte (r, c/2), low nibble = even c; bytes up to
 *           roundup(C,128)/2 are written, padding nibbles are 0;
 *   codes_t [C][ldt]: byte (c, r/2), low nibble = even r;
 *   scales  [ceil(R/32)][lds] and scales_t [ceil(C/32)][ldst] (its transpose).
 * The caller zero-fills the buffers; this file only writes valid entries.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ---------------------------------------------------------------- Philox */

void or_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4])
{
    const uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;     /* round multipliers */
    const uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;     /* Weyl key increments */
    uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
    uint32_t k0 = key_in[0], k1 = key_in[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) { k0 += W0; k1 += W1; }
        uint64_t p0 = (uint64_t)M0 * c0;
        uint64_t p1 = (uint64_t)M1 * c2;
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

/* 16 random bits for the element at storage index idx. */
uint32_t or_sr_bits(int64_t idx, uint64_t seed, uint64_t offset)
{
    uint64_t g = (uint64_t)idx >> 3;
    int j = (int)(idx & 7);
    uint32_t ctr[4] = {(uint32_t)g, (uint32_t)(g >> 32), (uint32_t)offset, (uint32_t)(offset >> 32)};
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint32_t w[4];
    or_philox4x32_10(ctr, key, w);
    return (w[j >> 1] >> (16 * (j & 1))) & 0xFFFFu;
}

/* ---------------------------------------------------------------- scales */

/* Smallest integer e with qmax * 2^e >= M, searched upward from the clamp -127. */
static int tf_exponent(double M, double qmax)
{
    int e = -127;
    while (e < 127 && qmax * ldexp(1.0, e) < M) ++e;
    return e;
}

int or_fp4_scale_exponent(double M) { return tf_exponent(M, 6.0); }

/*
 * The scale rule that the truncation-free ablation goes back to (Sec. 4.2, the
 * ablation figure; App. G, "Truncation-free scaling"): the shared exponent of
 * the OCP microscaling formats, floor(log2 M) minus the largest E2M1 exponent
 * (2, as 6 = 1.5 * 2^2): the largest integer e with 4 * 2^e <= M, searched
 * upward from the clamp -127.  Elements above 6 * 2^e then saturate to +-6
 * (or_fp4_code never returns a magnitude above index 7).
 */
int or_fp4_floor_exponent(double M)
{
    int e = -127;
    while (e < 127 && 4.0 * ldexp(1.0, e + 1) <= M) ++e;
    return e;
}
int or_fp8_scale_exponent(double M) { return tf_exponent(M, 448.0); }

/* ---------------------------------------------------------------- FP4 element */

static const double E2M1[8] = {0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0};

/* 4-bit E2M1 code (sign << 3 | magnitude index) of x / 2^e. */
unsigned or_fp4_code(double x, int e, int stochastic, uint32_t r16)
{
    unsigned s = signbit(x) ? 1u : 0u;
    double v = fabs(x) * ldexp(1.0, -e);          /* exact: power-of-two scaling */
    int k = 0;
    while (k < 7 && E2M1[k + 1] <= v) ++k;         /* largest grid point <= v */
    unsigned mag = (unsigned)k;
    if (v != E2M1[k] && k < 7) {
        double d = v - E2M1[k];
        double delta = E2M1[k + 1] - E2M1[k];
        if (!stochastic) {
            if (d > 0.5 * delta || (d == 0.5 * delta && (k & 1))) mag = (unsigned)k + 1;
        } else {
            double F = floor(d / delta * 65536.0);
            if (F + (double)r16 >= 65536.0) mag = (unsigned)k + 1;
        }
    }
    return (s << 3) | mag;
}

/* ---------------------------------------------------------------- E4M3 element */

/* Value of the non-negative E4M3FN code b (0..126): bias 7, 3 mantissa bits. */
static double e4m3_value(int b)
{
    int E = b >> 3, m = b & 7;
    if (E == 0) return ldexp((double)m, -9);
    return ldexp(1.0 + m / 8.0, E - 7);
}

/* 8-bit E4M3FN code of x / 2^e, round to nearest, ties to even code. */
unsigned or_e4m3_code(double x, int e)
{
    unsigned s = signbit(x) ? 1u : 0u;
    double v = fabs(x) * ldexp(1.0, -e);
    int lo = 0, hi = 126;                           /* largest code with value <= v */
    while (lo < hi) {
        int mid = (lo + hi + 1) / 2;
        if (e4m3_value(mid) <= v) lo = mid; else hi = mid - 1;
    }
    int b = lo;
    if (b < 126 && e4m3_value(b) != v) {
        double d = v - e4m3_value(b);
        double gap = e4m3_value(b + 1) - e4m3_value(b);
        if (d > 0.5 * gap || (d == 0.5 * gap && (b & 1))) b += 1;
    }
    return (s << 7) | (unsigned)b;
}

/* ---------------------------------------------------------------- inputs */

static double load(const void *x, int dtype, int64_t idx)
{
    if (dtype == 0) return (double)((const float *)x)[idx];
    uint32_t bits = (uint32_t)((const uint16_t *)x)[idx] << 16;   /* bfloat16 */
    float f;
    memcpy(&f, &bits, 4);
    return (double)f;
}

static void put_nibble(uint8_t *row, int64_t pos, unsigned code)
{
    if (pos & 1) row[pos >> 1] = (uint8_t)((row[pos >> 1] & 0x0F) | (code << 4));
    else         row[pos >> 1] = (uint8_t)((row[pos >> 1] & 0xF0) | code);
}

/* ---------------------------------------------------------------- 2D FP4 */

/*
 * Quantize the R x C matrix x[r*sr + c*sc] (sr, sc in elements) into 2D-block
 * FP4.  idx0 is added to every storage index before it keys the random stream
 * (0 for a whole tensor; the segment's first storage index for a grouped one).
 * mode bit 0: stochastic rounding (else round to nearest); bit 1: the floor
 * scale rule of the truncation-free ablation (else the truncation-free rule).
 */
void or_quantize_fp4_2d(const void *x, int dtype, int64_t R, int64_t C, int64_t sr, int64_t sc,
                        int64_t idx0, int b, int mode, uint64_t seed, uint64_t offset,
                        uint8_t *codes, int64_t ldc, uint8_t *codes_t, int64_t ldt,
                        uint8_t *scales, int64_t lds, uint8_t *scales_t, int64_t ldst,
                        int nthreads)
{
    int64_t nbr = (R + b - 1) / b, nbc = (C + b - 1) / b;
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(dynamic)
#endif
    for (int64_t I = 0; I < nbr; ++I) {
        for (int64_t J = 0; J < nbc; ++J) {
            int64_t r1 = (I + 1) * b < R ? (I + 1) * b : R;
            int64_t c1 = (J + 1) * b < C ? (J + 1) * b : C;
            double M = 0.0;
            int finite = 1;
            for (int64_t r = I * b; r < r1; ++r)
                for (int64_t c = J * b; c < c1; ++c) {
                    double v = load(x, dtype, r * sr + c * sc);
                    if (!isfinite(v)) finite = 0;
                    else if (fabs(v) > M) M = fabs(v);
                }
            int e = (mode & 2) ? or_fp4_floor_exponent(M) : or_fp4_scale_exponent(M);
            uint8_t sbyte = finite ? (uint8_t)(e + 127) : 0xFF;
            if (scales) scales[I * lds + J] = sbyte;
            if (scales_t) scales_t[J * ldst + I] = sbyte;
            for (int64_t r = I * b; r < r1; ++r)
                for (int64_t c = J * b; c < c1; ++c) {
                    unsigned code = 0;
                    if (finite) {
                        int64_t idx = r * sr + c * sc;
                        uint32_t r16 = (mode & 1) ? or_sr_bits(idx0 + idx, seed, offset) : 0;
                        code = or_fp4_code(load(x, dtype, idx), e, mode & 1, r16);
                    }
                    if (codes) put_nibble(codes + r * ldc, c, code);
                    if (codes_t) put_nibble(codes_t + c * ldt, r, code);
                }
        }
    }
}

/* ---------------------------------------------------------------- 1D FP4 */

/*
 * One-dimensional FP4 for activations (Sec. 3, "Application to linear
 * layers": activations keep a 1D block layout; App. C, "Activations"; the
 * 1D-FP4 activation entry of the training configuration table).  The block is
 * a 1 x 32 run of one row for the copy the forward GEMM reads (K = columns),
 * and a 32 x 1 run of one column for the copy the weight-gradient GEMM reads
 * (K = rows) -- the forward/backward scale mismatch of 1D layouts that the
 * 2D blocks remove (Sec. 2, "Scale inconsistency under transposition").  Each
 * block gets the truncation-free E8M0 scale of the 2D method (Sec. 3.1) and its
 * elements the same E2M1 codec; a stochastic element uses its one storage-index
 * draw in both copies.
 *   rowwise: codes [R][ldc] (byte (r, c/2), low nibble = even c); scales as
 *            4-byte words, one per row and K-tile of 128 columns: the scale of
 *            block (r, J) is byte J % 4 of word (J / 4, r), at
 *            scales[(J / 4) * lds + 4 r + J % 4];
 *   colwise: codes_t [C][ldt] (byte (c, r/2), low nibble = even r); the scale
 *            of block (I, c) at scales_t[(I / 4) * ldst + 4 c + I % 4].
 * (The word layout is the library's storage contract: a GEMM K-tile reads the
 * words of consecutive rows from consecutive addresses.)
 */
void or_quantize_fp4_1d(const void *x, int dtype, int64_t R, int64_t C, int64_t sr, int64_t sc,
                        int mode, uint64_t seed, uint64_t offset,
                        uint8_t *codes, int64_t ldc, uint8_t *scales, int64_t lds,
                        uint8_t *codes_t, int64_t ldt, uint8_t *scales_t, int64_t ldst,
                        int nthreads)
{
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(static)
#endif
    for (int64_t r = 0; r < R; ++r) {                 /* rowwise: 1 x 32 blocks */
        if (!codes) continue;
        for (int64_t J = 0; J * 32 < C; ++J) {
            int64_t c1 = (J + 1) * 32 < C ? (J + 1) * 32 : C;
            double M = 0.0; int finite = 1;
            for (int64_t c = J * 32; c < c1; ++c) {
                double v = load(x, dtype, r * sr + c * sc);
                if (!isfinite(v)) finite = 0; else if (fabs(v) > M) M = fabs(v);
            }
            int e = or_fp4_scale_exponent(M);
            scales[(J / 4) * lds + 4 * r + J % 4] = finite ? (uint8_t)(e + 127) : 0xFF;
            for (int64_t c = J * 32; c < c1; ++c) {
                unsigned code = 0;
                if (finite) {
                    int64_t idx = r * sr + c * sc;
                    uint32_t r16 = mode ? or_sr_bits(idx, seed, offset) : 0;
                    code = or_fp4_code(load(x, dtype, idx), e, mode, r16);
                }
                put_nibble(codes + r * ldc, c, code);
            }
        }
    }
#ifdef _OPENMP
#pragma omp parallel for schedule(static)
#endif
    for (int64_t c = 0; c < C; ++c) {                 /* colwise: 32 x 1 blocks */
        if (!codes_t) continue;
        for (int64_t I = 0; I * 32 < R; ++I) {
            int64_t r1 = (I + 1) * 32 < R ? (I + 1) * 32 : R;
            double M = 0.0; int finite = 1;
            for (int64_t r = I * 32; r < r1; ++r) {
                double v = load(x, dtype, r * sr + c * sc);
                if (!isfinite(v)) finite = 0; else if (fabs(v) > M) M = fabs(v);
            }
            int e = or_fp4_scale_exponent(M);
            scales_t[(I / 4) * ldst + 4 * c + I % 4] = finite ? (uint8_t)(e + 127) : 0xFF;
            for (int64_t r = I * 32; r < r1; ++r) {
                unsigned code = 0;
                if (finite) {
                    int64_t idx = r * sr + c * sc;
                    uint32_t r16 = mode ? or_sr_bits(idx, seed, offset) : 0;
                    code = or_fp4_code(load(x, dtype, idx), e, mode, r16);
                }
                put_nibble(codes_t + c * ldt, r, code);
            }
        }
    }
}

/* ---------------------------------------------------------------- MXFP8 */

/*
 * Rowwise copy: 1x32 blocks along columns, codes [R][ldc] bytes, scales [R][lds].
 * Colwise copy: 32x1 blocks along rows, stored transposed: codes_t [C][ldt],
 * scales_t [C][ldst].  E4M3 round-to-nearest-even; truncation-free scale with 448.
 */
void or_quantize_mxfp8(const void *x, int dtype, int64_t R, int64_t C, int64_t sr, int64_t sc,
                       uint8_t *codes, int64_t ldc, uint8_t *scales, int64_t lds,
                       uint8_t *codes_t, int64_t ldt, uint8_t *scales_t, int64_t ldst,
                       int nthreads)
{
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(static)
#endif
    for (int64_t r = 0; r < R; ++r) {                 /* rowwise */
        if (!codes) continue;
        for (int64_t J = 0; J * 32 < C; ++J) {
            int64_t c1 = (J + 1) * 32 < C ? (J + 1) * 32 : C;
            double M = 0.0; int finite = 1;
            for (int64_t c = J * 32; c < c1; ++c) {
                double v = load(x, dtype, r * sr + c * sc);
                if (!isfinite(v)) finite = 0; else if (fabs(v) > M) M = fabs(v);
            }
            int e = or_fp8_scale_exponent(M);
            scales[r * lds + J] = finite ? (uint8_t)(e + 127) : 0xFF;
            for (int64_t c = J * 32; c < c1; ++c)
                codes[r * ldc + c] = finite ? (uint8_t)or_e4m3_code(load(x, dtype, r * sr + c * sc), e) : 0;
        }
    }
#ifdef _OPENMP
#pragma omp parallel for schedule(static)
#endif
    for (int64_t c = 0; c < C; ++c) {                 /* colwise */
        if (!codes_t) continue;
        for (int64_t I = 0; I * 32 < R; ++I) {
            int64_t r1 = (I + 1) * 32 < R ? (I + 1) * 32 : R;
            double M = 0.0; int finite = 1;
            for (int64_t r = I * 32; r < r1; ++r) {
                double v = load(x, dtype, r * sr + c * sc);
                if (!isfinite(v)) finite = 0; else if (fabs(v) > M) M = fabs(v);
            }
            int e = or_fp8_scale_exponent(M);
            scales_t[c * ldst + I] = finite ? (uint8_t)(e + 127) : 0xFF;
            for (int64_t r = I * 32; r < r1; ++r)
                codes_t[c * ldt + r] = finite ? (uint8_t)or_e4m3_code(load(x, dtype, r * sr + c * sc), e) : 0;
        }
    }
}

/* Element-wise forms of the two scalar codecs, for exhaustive checks. */
void or_fp4_codes(const double *x, const int *e, const uint32_t *r16, int stochastic,
                  int64_t n, uint8_t *out)
{
    for (int64_t i = 0; i < n; ++i)
        out[i] = (uint8_t)or_fp4_code(x[i], e[i], stochastic, r16 ? r16[i] : 0);
}

void or_e4m3_codes(const double *x, const int *e, int64_t n, uint8_t *out)
{
    for (int64_t i = 0; i < n; ++i) out[i] = (uint8_t)or_e4m3_code(x[i], e[i]);
}

int or_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
