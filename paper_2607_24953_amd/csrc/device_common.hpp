// Device-side helpers shared by the libq2d kernels (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace q2d {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v16f __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float bits_f(uint32_t u) { return __uint_as_float(u); }
__device__ __forceinline__ uint32_t f_bits(float f) { return __float_as_uint(f); }

// a ^ b ^ k in one v_bitop3_b32 (truth table 0x96, symmetric in its inputs);
// k is wave-uniform
__device__ __forceinline__ uint32_t xor3_uniform(uint32_t a, uint32_t b, uint32_t k)
{
    uint32_t r;
    asm("v_bitop3_b32 %0, %1, %2, %3 bitop3:0x96" : "=v"(r) : "v"(a), "v"(b), "s"(k));
    return r;
}

// Philox4x32 with 10 rounds (Salmon, Moraes, Dror, Shaw, SC 2011): two 32x32->64
// multiplies per round, key bumped by the Weyl constants between rounds.  The
// key is wave-uniform, so the bumps stay scalar.  Each product is formed as one
// 64-bit result (v_mad_u64_u32) rather than separate low and high multiplies:
// about a quarter fewer cycles per block on gfx950.
__device__ __forceinline__ void philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                              uint32_t k0, uint32_t k1, uint32_t out[4])
{
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        if (r) { k0 += 0x9E3779B9u; k1 += 0xBB67AE85u; }
        const uint64_t p0 = (uint64_t)0xD2511F53u * c0, p1 = (uint64_t)0xCD9E8D57u * c2;
        const uint32_t lo0 = (uint32_t)p0, hi0 = (uint32_t)(p0 >> 32);
        const uint32_t lo1 = (uint32_t)p1, hi1 = (uint32_t)(p1 >> 32);
        const uint32_t n0 = xor3_uniform(hi1, c1, k0);
        const uint32_t n2 = xor3_uniform(hi0, c3, k1);
        c0 = n0; c1 = lo1; c2 = n2; c3 = lo0;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

// The 16-bit stochastic-rounding draw of storage index idx: half (idx & 1) of
// word (idx & 7) >> 1 of the block for counter (idx >> 3, offset).
__device__ __forceinline__ uint32_t sr_draw(uint64_t idx, uint32_t k0, uint32_t k1,
                                            uint32_t off_lo, uint32_t off_hi)
{
    const uint64_t g = idx >> 3;
    uint32_t w[4];
    philox4x32_10((uint32_t)g, (uint32_t)(g >> 32), off_lo, off_hi, k0, k1, w);
    const uint32_t j = (uint32_t)idx & 7u;
    const uint32_t word = (j & 4u) ? ((j & 2u) ? w[3] : w[2]) : ((j & 2u) ? w[1] : w[0]);
    return (word >> ((j & 1u) * 16u)) & 0xFFFFu;
}

// Truncation-free E2M1 block exponent from the block maximum's float32 bit
// pattern (sign cleared): the smallest e with 6 * 2^e >= M.  For M = 1.f * 2^p
// that is p - 2, plus one when f > 1.5; subnormal and tiny maxima clamp to -127.
__device__ __forceinline__ int fp4_block_exponent(uint32_t amax_bits)
{
    const int eb = (int)(amax_bits >> 23);
    if (eb == 0) return -127;
    const int e = eb - 129 + ((amax_bits & 0x7FFFFFu) > 0x400000u ? 1 : 0);
    return e < -127 ? -127 : e;
}

// Scale rule of the truncation-free ablation (the shared-exponent rule of the
// OCP microscaling formats): e = floor(log2 M) - 2, the exponent of M's leading
// bit minus E2M1's largest exponent (6 = 1.5 * 2^2), clamped to -127.  Block
// maxima with a mantissa above 1.5 then exceed 6 * 2^e and saturate to +-6.
__device__ __forceinline__ int fp4_floor_exponent(uint32_t amax_bits)
{
    const int e = (int)(amax_bits >> 23) - 129;
    return e < -127 ? -127 : e;
}

// Same rule for E4M3 (largest magnitude 448 = 1.75 * 2^8): e = p - 8, plus one
// when f > 1.75.
__device__ __forceinline__ int fp8_block_exponent(uint32_t amax_bits)
{
    const int eb = (int)(amax_bits >> 23);
    if (eb == 0) return -127;
    const int e = eb - 135 + ((amax_bits & 0x7FFFFFu) > 0x600000u ? 1 : 0);
    return e < -127 ? -127 : e;
}

// 2^-e as a float for e in [-127, 126].
__device__ __forceinline__ float inv_pow2(int e) { return bits_f((uint32_t)(127 - e) << 23); }

// E4M3FN code magnitude of v in [0, 448], round to nearest even.  Below 2^-6
// the spacing is 2^-9 (subnormals); above it the 3-bit mantissa is rounded on
// the float32 bit pattern.
__device__ __forceinline__ uint32_t e4m3_rne(float v)
{
    if (v < 0.015625f) return (uint32_t)(int)__builtin_rintf(v * 512.0f);
    uint32_t b = f_bits(v);
    b += 0x7FFFFu + ((b >> 20) & 1u);
    return (b >> 20) - (120u << 3);
}

__device__ __forceinline__ float bf16_to_f(uint16_t h) { return bits_f((uint32_t)h << 16); }

__device__ __forceinline__ uint16_t f_to_bf16_rne(float f)
{
    uint32_t b = f_bits(f);
    if ((b & 0x7F800000u) == 0x7F800000u) return (uint16_t)((b >> 16) | ((b & 0xFFFFu) ? 0x40u : 0u));
    b += 0x7FFFu + ((b >> 16) & 1u);
    return (uint16_t)(b >> 16);
}

// ---- grouped (MoE) segment tables, built per workgroup in LDS

constexpr int kMaxSegs = 1024;

// Inclusive prefix over `n` values produced by f(i) (i < n), written to out[1..n]
// with out[0] = 0.  Run by one full wave; n <= kMaxSegs.
template <typename F>
__device__ __forceinline__ void wave_prefix(int n, F f, int32_t *out)
{
    const int lane = threadIdx.x & 63;
    int32_t carry = 0;
    if (lane == 0) out[0] = 0;
    for (int base = 0; base < n; base += 64) {
        const int i = base + lane;
        int32_t v = i < n ? f(i) : 0;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int32_t u = __shfl_up(v, d);
            if (lane >= d) v += u;
        }
        if (i < n) out[i + 1] = carry + v;
        carry += __shfl(v, 63);
    }
}

// Segment offsets as the kernels use them: out[i] = min(max(0, off[0], ..,
// off[i]), total) for i = 0 .. n.  A valid table (ascending from 0 to total) is
// unchanged; any other one becomes ascending and inside [0, total], so the
// segments stay inside the input rows and their padded sizes inside the
// grouped capacity.  Run by one full wave; n <= kMaxSegs.
__device__ __forceinline__ void wave_offsets(int n, const int64_t *off, int64_t total, int32_t *out)
{
    const int lane = threadIdx.x & 63;
    int32_t carry = 0;
    for (int base = 0; base <= n; base += 64) {
        const int i = base + lane;
        int64_t o = i <= n ? off[i] : 0;
        o = o < 0 ? 0 : (o > total ? total : o);
        int32_t v = (int32_t)o;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int32_t u = __shfl_up(v, d);
            if (lane >= d) v = max(v, u);
        }
        v = max(v, carry);
        if (i <= n) out[i] = v;
        carry = __shfl(v, 63);
    }
}

// Largest e < n with table[e] <= x (table ascending, table[0] = 0 <= x).
__device__ __forceinline__ int seg_search(const int32_t *table, int n, int32_t x)
{
    int lo = 0, hi = n - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (table[mid] <= x) lo = mid; else hi = mid - 1;
    }
    return lo;
}

}  // namespace q2d
