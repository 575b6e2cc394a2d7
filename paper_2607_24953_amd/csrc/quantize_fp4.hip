// Fused 2D-block FP4 quantizer (Sec. 3, Sec. 3.1; App. D, App. E).
//
// One pass over the input: block maximum, truncation-free E8M0 scale, round to
// nearest or Philox stochastic rounding, and both packed layouts (row-packed
// codes and column-packed codes_t) plus the scale grid and its transpose.
//
// Work split: a workgroup owns a 128-row tile of WC x 128 columns; each wave
// owns a 32 x 128 strip (four 32 x 32 blocks side by side).  Lane l owns an
// 8 x 8 sub-block: rows 8*(l/16) .. +7 and columns 8*(l%16) .. +7 of the strip.
// A row of the sub-block is one 16-byte load (bf16), so every load
// instruction of the wave reads four 256-byte row segments.  The 8 x 8
// sub-block makes the transposition local: each lane packs eight nibbles per
// row for codes and eight per column for codes_t without data exchange.  The
// block maximum is a max over the lane's 64 values followed by four cross-lane
// butterflies (the 16 lanes of a 32 x 32 block differ in lane bits 0, 1, 4, 5).
// bfloat16 rows stay packed two elements per register.
//
// The packed codes go through LDS and leave as 16-byte stores: full 128-byte
// lines of codes when the tile is 256 columns wide (WC = 2, round to nearest),
// 64-byte runs of codes_t.
//
// Round to nearest uses gfx950's v_cvt_scalef32_pk_fp4_{bf16,f32}: the E2M1
// code of x / S rounded to nearest even, two elements per instruction, which
// is the round-to-nearest definition exactly.
//
// Stochastic rounding uses v_cvt_scalef32_sr_pk_fp4_f32.  It converts a pair
// with one 32-bit seed: the first element adds seed >> 10 below its kept
// mantissa bit (after aligning subnormal E2M1 results) and truncates, the
// second element adds (seed << 1) >> 10.  A seed of r16 << 16 for the first
// element, or r16 << 15 for the second, therefore rounds the magnitude up
// exactly when floor(2^16 d / delta) + r16 >= 2^16 -- the rounding contract of
// this library.  Each element is converted in an instruction where it has its
// own draw; the other nibble of that result is dropped.  The parity tests
// compare every bfloat16 value under every scale, in both modes, bit for bit
// with the CPU definition.
//
// The same kernel emits 1D FP4 for activations (ONED; Sec. 3, "Application to
// linear layers"; App. C, "Activations"): 1 x 32 row blocks for the codes copy
// and 32 x 1 column blocks for the codes_t copy, each with its own
// truncation-free scale.  A row block spans the 4 lanes that differ in lane
// bits 0-1, a column block the 4 lanes that differ in bits 4-5; the codes are
// packed and stored exactly as for 2D blocks, and the scales (one byte per row
// and K-group) go through LDS and leave as 4-byte words in K-tile-major order.
#include "device_common.hpp"
#include "kernels.hpp"

namespace q2d {

namespace {

constexpr int kTile = 128;          // tile rows

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f2v __attribute__((ext_vector_type(2)));
typedef unsigned int u4v __attribute__((ext_vector_type(4)));

// 16-byte streaming load: the input is read once, so it should not displace
// cache lines that are reused
__device__ __forceinline__ uint4 load_stream16(const void *p)
{
    const u4v v = __builtin_nontemporal_load(reinterpret_cast<const u4v *>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

typedef uint16_t u16x2 __attribute__((ext_vector_type(2)));

template <typename T>
struct Elem;

template <>
struct Elem<float> {
    static __device__ __forceinline__ uint32_t bits(const float *p) { return f_bits(*p); }
};

template <>
struct Elem<uint16_t> {
    static __device__ __forceinline__ uint32_t bits(const uint16_t *p) { return (uint32_t)*p << 16; }
};

// Round-to-nearest E2M1 pair into byte SEL of `old`: f32 sources as two
// float32 bit patterns, bf16 sources as one packed register (low half first).
template <int SEL>
__device__ __forceinline__ uint32_t rtn_pair_f32(uint32_t old, uint32_t lo, uint32_t hi, float scale)
{
    return __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(old, bits_f(lo), bits_f(hi), scale, SEL);
}
template <int SEL>
__device__ __forceinline__ uint32_t rtn_pair_bf16(uint32_t old, uint32_t packed, float scale)
{
    return __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(old, __builtin_bit_cast(bf16x2, packed), scale, SEL);
}

// Stochastic E2M1 conversion of a pair into byte `sel`; the other bytes of the
// result are not defined and the caller masks them.
__device__ __forceinline__ uint32_t sr_pair(int sel, f2v v, uint32_t seed, float scale)
{
    switch (sel) {
    case 0: return __builtin_amdgcn_cvt_scalef32_sr_pk_fp4_f32(0u, v, seed, scale, 0);
    case 1: return __builtin_amdgcn_cvt_scalef32_sr_pk_fp4_f32(0u, v, seed, scale, 1);
    case 2: return __builtin_amdgcn_cvt_scalef32_sr_pk_fp4_f32(0u, v, seed, scale, 2);
    default: return __builtin_amdgcn_cvt_scalef32_sr_pk_fp4_f32(0u, v, seed, scale, 3);
    }
}

// Stochastic E2M1 conversion of the pair (columns 2k, 2k+1) of one sub-block
// row into byte `sel` (bf16 rows are one packed register, float32 rows two bit
// patterns).  Both go through the float32 conversion: the bf16-source form
// rounds differently near the carry boundary (its parity against the rounding
// contract fails), so bf16 pairs are widened first.  As for sr_pair, the other
// bytes of the result are not defined.
template <typename T>
__device__ __forceinline__ uint32_t sr_row_pair(int sel, const uint32_t *row, uint32_t seed, float scale)
{
    f2v p;
    if constexpr (sizeof(T) == 2) p = f2v{bits_f(row[sel] << 16), bits_f(row[sel] & 0xFFFF0000u)};
    else p = f2v{bits_f(row[2 * sel]), bits_f(row[2 * sel + 1])};
    return sr_pair(sel, p, seed, scale);
}

// 8 x 8 transpose of 4-bit elements: nibble j of in[i] becomes nibble i of
// out[j].  Three exchange stages of doubling width (nibbles within row pairs,
// bytes across distance 2, half-words across distance 4).
__device__ __forceinline__ void nibble_transpose8(const uint32_t in[8], uint32_t out[8])
{
    uint32_t m[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) m[i] = in[i];
#pragma unroll
    for (int p = 0; p < 8; p += 2) {
        const uint32_t t = ((m[p] >> 4) ^ m[p + 1]) & 0x0F0F0F0Fu;
        m[p + 1] ^= t;
        m[p] ^= t << 4;
    }
#pragma unroll
    for (int i = 0; i < 8; i += (i & 1) ? 3 : 1) {         // 0, 1, 4, 5
        const uint32_t x = m[i], y = m[i + 2];
        m[i] = __builtin_amdgcn_perm(y, x, 0x06020400u);     // bytes x0 y0 x2 y2
        m[i + 2] = __builtin_amdgcn_perm(y, x, 0x07030501u); // bytes x1 y1 x3 y3
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t x = m[i], y = m[i + 4];
        out[i] = __builtin_amdgcn_perm(y, x, 0x05040100u);       // x.lo, y.lo
        out[i + 4] = __builtin_amdgcn_perm(y, x, 0x07060302u);   // x.hi, y.hi
    }
}

// Philox4x32-10 block with one 32x32->64 multiply per product (v_mad_u64_u32)
// and one three-input xor per output word.
__device__ __forceinline__ void philox_block(uint64_t g, uint32_t o0, uint32_t o1, uint32_t k0, uint32_t k1,
                                             uint32_t w[4])
{
    uint32_t c0 = (uint32_t)g, c1 = (uint32_t)(g >> 32), c2 = o0, c3 = o1;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        if (r) { k0 += 0x9E3779B9u; k1 += 0xBB67AE85u; }
        const uint64_t p0 = (uint64_t)0xD2511F53u * c0;
        const uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
        const uint32_t n0 = xor3_uniform((uint32_t)(p1 >> 32), c1, k0);
        const uint32_t n2 = xor3_uniform((uint32_t)(p0 >> 32), c3, k1);
        c0 = n0; c1 = (uint32_t)p1; c2 = n2; c3 = (uint32_t)p0;
    }
    w[0] = c0; w[1] = c1; w[2] = c2; w[3] = c3;
}

// One 128-row tile (row tile tr, column tile tc) of the quantization described
// by `a` (for a grouped tensor, `a` is already narrowed to the tile's segment).
// VEC: rows are read as aligned 8-element vectors (stride_c == 1).
// SR: stochastic rounding.  ALIGNED8: every sub-block row starts at a storage
// index that is a multiple of 8, so one Philox block serves its 8 elements.
// GROUPED: the rows are expert segments (see QuantArgs).  WC: 128-column
// strips per tile (waves side by side).  ONED: 1 x 32 / 32 x 1 blocks.
template <typename T, bool VEC, bool SR, bool ALIGNED8, bool GROUPED, int WC, bool ONED>
__device__ __forceinline__ void quantize_tile(QuantArgs a, const int64_t tr, const int64_t tc)
{
    constexpr int kTC = 128 * WC;
    constexpr int kThreads = 256 * WC;
    constexpr bool PK = sizeof(T) == 2;     // bf16: two elements per register
    constexpr int NV = PK ? 4 : 8;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int wr = wave / WC, wc = wave % WC;
    const int64_t strip_r = tr * kTile + wr * 32;
    const int rg = lane >> 4, cc = lane & 15;
    const int64_t r0 = strip_r + 8 * rg;
    const int64_t c0 = tc * kTC + wc * 128 + 8 * cc;
    const T *x = reinterpret_cast<const T *>(a.x);

    // ---- load the 8 x 8 sub-block (0 outside R x C).  bf16: v[i][k] holds
    // columns 2k (low half) and 2k+1 (high half) of row i; fp32: bit patterns.
    uint32_t v[8][NV];
    if (PK) {
        if (VEC && c0 + 8 <= a.cols) {
            const T *xr = x + r0 * a.stride_r + c0;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                uint4 q = make_uint4(0u, 0u, 0u, 0u);
                if (r0 + i < a.rows) q = load_stream16(xr);
                v[i][0] = q.x; v[i][1] = q.y; v[i][2] = q.z; v[i][3] = q.w;
                xr += a.stride_r;
            }
        } else {
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int64_t r = r0 + i;
#pragma unroll
                for (int k = 0; k < NV; ++k) {
                    const int64_t c = c0 + 2 * k;
                    const uint32_t lo = (r < a.rows && c < a.cols) ? Elem<T>::bits(x + r * a.stride_r + c * a.stride_c) : 0u;
                    const uint32_t hi = (r < a.rows && c + 1 < a.cols) ? Elem<T>::bits(x + r * a.stride_r + (c + 1) * a.stride_c) : 0u;
                    v[i][k] = (lo >> 16) | hi;
                }
            }
        }
    } else if (VEC && c0 + 8 <= a.cols) {
        const T *xr = x + r0 * a.stride_r + c0;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            uint4 q0 = make_uint4(0u, 0u, 0u, 0u), q1 = q0;
            if (r0 + i < a.rows) {
                q0 = load_stream16(xr);
                q1 = load_stream16(xr + 4);
            }
            v[i][0] = q0.x; v[i][1] = q0.y; v[i][2] = q0.z; v[i][3] = q0.w;
            v[i][NV - 4] = q1.x; v[i][NV - 3] = q1.y; v[i][NV - 2] = q1.z; v[i][NV - 1] = q1.w;
            xr += a.stride_r;
        }
    } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int64_t r = r0 + i;
#pragma unroll
            for (int j = 0; j < NV; ++j) {
                const int64_t c = c0 + j;
                v[i][j] = (r < a.rows && c < a.cols) ? Elem<T>::bits(x + r * a.stride_r + c * a.stride_c) : 0u;
            }
        }
    }
    // float32 bit pattern of element (i, j)
    auto elem = [&](int i, int j) -> uint32_t {
        if (PK) return (j & 1) ? (v[i][j >> 1] & 0xFFFF0000u) : (v[i][j >> 1] << 16);
        return v[i][j];
    };

    // ---- block maximum on |bits| (NaN > inf > finite, as unsigned integers).
    // 2D: one per lane group of 16; 1D: one per row (rm) and per column (cm).
    uint32_t am = 0;
    uint32_t rm[8], cm[8];
    if (!ONED) {
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
            for (int k = 0; k < NV; ++k) {
                if (PK) {
                    const uint32_t w = v[i][k] & 0x7FFF7FFFu;
                    am = max(am, max(w & 0xFFFFu, w >> 16));
                } else {
                    am = max(am, v[i][k] & 0x7FFFFFFFu);
                }
            }
        if (PK) am <<= 16;
        am = max(am, (uint32_t)__shfl_xor((int)am, 1));
        am = max(am, (uint32_t)__shfl_xor((int)am, 2));
        am = max(am, (uint32_t)__shfl_xor((int)am, 16));
        am = max(am, (uint32_t)__shfl_xor((int)am, 32));
    } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) cm[j] = 0;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            uint32_t m = 0;
#pragma unroll
            for (int k = 0; k < NV; ++k) {
                if (PK) {
                    const uint32_t w = v[i][k] & 0x7FFF7FFFu;
                    m = max(m, max(w & 0xFFFFu, w >> 16));
                    cm[2 * k] = max(cm[2 * k], w & 0xFFFFu);
                    cm[2 * k + 1] = max(cm[2 * k + 1], w >> 16);
                } else {
                    const uint32_t w = v[i][k] & 0x7FFFFFFFu;
                    m = max(m, w);
                    cm[k] = max(cm[k], w);
                }
            }
            rm[i] = PK ? m << 16 : m;
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            rm[i] = max(rm[i], (uint32_t)__shfl_xor((int)rm[i], 1));
            rm[i] = max(rm[i], (uint32_t)__shfl_xor((int)rm[i], 2));
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            if (PK) cm[j] <<= 16;
            cm[j] = max(cm[j], (uint32_t)__shfl_xor((int)cm[j], 16));
            cm[j] = max(cm[j], (uint32_t)__shfl_xor((int)cm[j], 32));
        }
    }
    if (!ONED && !GROUPED && a.block == 64) {
        // 64 x 64 blocks: the 32 x 32 block beside it in this wave (lane bit 2), then
        // the 32-row strip of the paired wave through LDS
        __shared__ uint32_t am64[4][2 * WC];
        am = max(am, (uint32_t)__shfl_xor((int)am, 4));
        if (rg == 0 && (cc & 7) == 0) am64[wr][wc * 2 + (cc >> 3)] = am;
        __syncthreads();
        am = max(am, am64[wr ^ 1][wc * 2 + (cc >> 3)]);
    }
    const bool finite = am < 0x7F800000u;
    const bool floor_rule = !ONED && a.floor_scale;
    const int e = floor_rule ? fp4_floor_exponent(am) : fp4_block_exponent(am);
    const float scale = bits_f((uint32_t)(127 + e) << 23);       // 2^e
    if (floor_rule && finite) {
        // saturate magnitudes above 6 * 2^e (exact in bf16: 1.5 * 2^(e+2)): the
        // magnitude bits take their minimum with the limit's, the sign stays
        // (bf16: both halves of a word at once, in place)
        const uint32_t lim = ((uint32_t)(e + 129) << 23) | 0x400000u;
        const u16x2 l16 = {(uint16_t)(lim >> 16), (uint16_t)(lim >> 16)};
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
            for (int k = 0; k < NV; ++k) {
                if (PK) {
                    const u16x2 mag = __builtin_bit_cast(u16x2, v[i][k] & 0x7FFF7FFFu);
                    v[i][k] = (v[i][k] & 0x80008000u) | __builtin_bit_cast(uint32_t, __builtin_elementwise_min(mag, l16));
                } else {
                    v[i][k] = (v[i][k] & 0x80000000u) | min(v[i][k] & 0x7FFFFFFFu, lim);
                }
            }
    }
    // scale of row i / column j of the sub-block (the block scale for 2D)
    auto rscale = [&](int i) -> float {
        return ONED ? bits_f((uint32_t)(127 + fp4_block_exponent(rm[i])) << 23) : scale;
    };
    auto cscale = [&](int j) -> float {
        return ONED ? bits_f((uint32_t)(127 + fp4_block_exponent(cm[j])) << 23) : scale;
    };

    // ---- encode: rowp[i] = eight nibbles of row i, colp[j] = eight nibbles of column j
    uint32_t rowp[8], colp[8];
    if (!SR) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            uint32_t w = 0;
            const float sc = rscale(i);
            if (PK) {
                w = rtn_pair_bf16<0>(w, v[i][0], sc);
                w = rtn_pair_bf16<1>(w, v[i][1], sc);
                w = rtn_pair_bf16<2>(w, v[i][2], sc);
                w = rtn_pair_bf16<3>(w, v[i][3], sc);
            } else {
                w = rtn_pair_f32<0>(w, elem(i, 0), elem(i, 1), sc);
                w = rtn_pair_f32<1>(w, elem(i, 2), elem(i, 3), sc);
                w = rtn_pair_f32<2>(w, elem(i, 4), elem(i, 5), sc);
                w = rtn_pair_f32<3>(w, elem(i, 6), elem(i, 7), sc);
            }
            rowp[i] = w;
        }
        if constexpr (!ONED) {
            // 2D blocks: one scale for both layouts, so the column-packed words are
            // the nibble transpose of the row-packed ones (each element converted
            // once, and the inputs are dead after the row pass)
            nibble_transpose8(rowp, colp);
        } else {
            // 1D: every column has its own scale and is converted on its own
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                uint32_t w = 0;
                const float sc = cscale(j);
                if (PK) {
                    // rows (2m, 2m+1) of column j as one packed pair
                    const int k = j >> 1;
                    auto pr = [&](int m) -> uint32_t {
                        const uint32_t lo = v[2 * m][k], hi = v[2 * m + 1][k];
                        return (j & 1) ? ((lo >> 16) | (hi & 0xFFFF0000u)) : ((lo & 0xFFFFu) | (hi << 16));
                    };
                    w = rtn_pair_bf16<0>(w, pr(0), sc);
                    w = rtn_pair_bf16<1>(w, pr(1), sc);
                    w = rtn_pair_bf16<2>(w, pr(2), sc);
                    w = rtn_pair_bf16<3>(w, pr(3), sc);
                } else {
                    w = rtn_pair_f32<0>(w, elem(0, j), elem(1, j), sc);
                    w = rtn_pair_f32<1>(w, elem(2, j), elem(3, j), sc);
                    w = rtn_pair_f32<2>(w, elem(4, j), elem(5, j), sc);
                    w = rtn_pair_f32<3>(w, elem(6, j), elem(7, j), sc);
                }
                colp[j] = w;
            }
        }
    } else {
        const uint32_t k0 = (uint32_t)a.seed, k1 = (uint32_t)(a.seed >> 32);
        const uint32_t o0 = (uint32_t)a.offset, o1 = (uint32_t)(a.offset >> 32);
        // the draws of row i (storage index idx_row of its first element) as
        // seeds r16 << 16
        auto row_draws = [&](int i, int64_t idx_row, uint32_t s16[8]) __attribute__((always_inline)) {
            uint32_t w[4] = {0, 0, 0, 0}, w2[4] = {0, 0, 0, 0};
            if (VEC) {
                philox_block((uint64_t)idx_row >> 3, o0, o1, k0, k1, w);
                if (!ALIGNED8) philox_block(((uint64_t)idx_row >> 3) + 1, o0, o1, k0, k1, w2);
            }
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                uint32_t r;
                if (VEC) {
                    if (ALIGNED8) {
                        r = (j & 1) ? (w[j >> 1] & 0xFFFF0000u) : (w[j >> 1] << 16);
                    } else {
                        // the row's eight draws straddle two Philox blocks
                        const uint32_t q = (uint32_t)(idx_row & 7) + (uint32_t)j;     // 0..14
                        const uint32_t sq = q & 7u;
                        const uint32_t wa = (sq & 4u) ? ((sq & 2u) ? w[3] : w[2]) : ((sq & 2u) ? w[1] : w[0]);
                        const uint32_t wb = (sq & 4u) ? ((sq & 2u) ? w2[3] : w2[2]) : ((sq & 2u) ? w2[1] : w2[0]);
                        const uint32_t ww = q < 8u ? wa : wb;
                        r = (sq & 1u) ? (ww & 0xFFFF0000u) : (ww << 16);
                    }
                } else {
                    const uint64_t idx = (uint64_t)(a.index_base + (r0 + i) * a.stride_r + (c0 + j) * a.stride_c);
                    r = sr_draw(idx, k0, k1, o0, o1) << 16;
                }
                s16[j] = r;
            }
        };
        int64_t idx0 = a.index_base + r0 * a.stride_r + c0;
        if constexpr (!ONED) {
            // 2D blocks: both layouts share the block scale, so every element is
            // converted once, row by row; the column-packed words are the 8 x 8
            // nibble transpose of the row-packed ones
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                uint32_t s16[8];
                row_draws(i, idx0, s16);
                idx0 += a.stride_r;
                uint32_t w = 0;
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    // element 2k from a conversion with its draw, element 2k + 1 from
                    // one with its own (the second element reads seed << 1)
                    const uint32_t lo = sr_row_pair<T>(k, v[i], s16[2 * k], scale);
                    const uint32_t hi = sr_row_pair<T>(k, v[i], s16[2 * k + 1] >> 1, scale);
                    w |= ((lo & 0x0F0F0F0Fu) | (hi & 0xF0F0F0F0u)) & (0xFFu << (8 * k));
                }
                rowp[i] = w;
            }
            nibble_transpose8(rowp, colp);
        } else {
#pragma unroll
            for (int i = 0; i < 8; ++i) { rowp[i] = 0; colp[i] = 0; }
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                // draws of rows 2m and 2m+1 as seeds r16 << 16
                uint32_t s16[2][8];
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    row_draws(2 * m + h, idx0, s16[h]);
                    idx0 += a.stride_r;
                }
                // rows 2m and 2m+1: pairs (2k, 2k+1) into byte k
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int i = 2 * m + h;
                    const float sc = rscale(i);
                    uint32_t acc = 0;
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        const f2v pr = {bits_f(elem(i, 2 * k)), bits_f(elem(i, 2 * k + 1))};
                        const uint32_t lo = sr_pair(k, pr, s16[h][2 * k], sc);
                        const uint32_t hi = sr_pair(k, pr, s16[h][2 * k + 1] >> 1, sc);
                        acc |= (lo & (0x0Fu << (8 * k))) | (hi & (0xF0u << (8 * k)));
                    }
                    rowp[i] = acc;
                }
                // every column: rows (2m, 2m+1) into byte m, each with its column's scale
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const f2v pr = {bits_f(elem(2 * m, j)), bits_f(elem(2 * m + 1, j))};
                    const float sc = cscale(j);
                    const uint32_t lo = sr_pair(m, pr, s16[0][j], sc);
                    const uint32_t hi = sr_pair(m, pr, s16[1][j] >> 1, sc);
                    colp[j] |= (lo & (0x0Fu << (8 * m))) | (hi & (0xF0u << (8 * m)));
                }
            }
        }
    }
    if (!ONED && !finite) {
#pragma unroll
        for (int i = 0; i < 8; ++i) { rowp[i] = 0; colp[i] = 0; }
    }
    if (ONED) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            if (rm[i] >= 0x7F800000u) rowp[i] = 0;
            if (cm[i] >= 0x7F800000u) colp[i] = 0;
        }
    }

    // ---- stores through LDS: 16 bytes per lane, codes rows r < store_rows as
    // WC * 64-byte runs, codes_t rows c < C as 64-byte runs
    __shared__ uint32_t st_r[kTile][16 * WC + 1];
    __shared__ uint32_t st_c[kTC][17];
    __shared__ uint8_t st_rs[ONED ? kTile : 1][4 * WC];     // 1D: row scales of the tile
    __shared__ uint8_t st_cs[ONED ? kTC : 1][4];            // 1D: column scales of the tile
    {
        // the lane geometry again, from the thread index: cheaper than keeping it
        // live across the conversion (the opaque copy stops the compiler from
        // reusing the values computed at the top)
        int t = threadIdx.x;
        asm volatile("" : "+v"(t));
        const int wr = (t >> 6) / WC, wc = (t >> 6) % WC, rg = (t & 63) >> 4, cc = t & 15;
        const int rl = wr * 32 + 8 * rg;
#pragma unroll
        for (int i = 0; i < 8; ++i) st_r[rl + i][wc * 16 + cc] = rowp[i];
#pragma unroll
        for (int j = 0; j < 8; ++j) st_c[wc * 128 + 8 * cc + j][wr * 4 + rg] = colp[j];
        if (ONED) {
            auto sbyte = [](uint32_t m) -> uint8_t {
                return m < 0x7F800000u ? (uint8_t)(127 + fp4_block_exponent(m)) : (uint8_t)0xFF;
            };
            if ((cc & 3) == 0) {
#pragma unroll
                for (int i = 0; i < 8; ++i) st_rs[rl + i][wc * 4 + (cc >> 2)] = sbyte(rm[i]);
            }
            if (rg == 0) {
#pragma unroll
                for (int j = 0; j < 8; ++j) st_cs[wc * 128 + 8 * cc + j][wr] = sbyte(cm[j]);
            }
        }
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        const int item = threadIdx.x + kThreads * q;
        if (a.codes) {
            const int line = item / (4 * WC), part = item % (4 * WC);
            const int64_t r = tr * kTile + line;
            if (r < a.store_rows && tc * kTC + part * 32 < a.cols_pad) {
                const uint4 w = make_uint4(st_r[line][4 * part], st_r[line][4 * part + 1],
                                           st_r[line][4 * part + 2], st_r[line][4 * part + 3]);
                *reinterpret_cast<uint4 *>(a.codes + r * a.ld_codes + tc * (kTC / 2) + part * 16) = w;
            }
        }
        if (a.codes_t) {
            const int line = item >> 2, part = item & 3;
            const int64_t c = tc * kTC + line;
            if (c < a.cols) {
                const uint4 w = make_uint4(st_c[line][4 * part], st_c[line][4 * part + 1],
                                           st_c[line][4 * part + 2], st_c[line][4 * part + 3]);
                *reinterpret_cast<uint4 *>(a.codes_t + c * a.ld_codes_t + tr * (kTile / 2) + part * 16) = w;
            }
        }
    }
    if (ONED) {
        // scale words, K-tile major: row r's word of each 128-column strip k at
        // (k, r); column c's word of this 128-row tile at (tr, c)
        const int t = threadIdx.x;
        if (t < kTile) {
            const int64_t r = tr * kTile + t;
            if (a.scales && r < a.rows) {
#pragma unroll
                for (int w = 0; w < WC; ++w)
                    if (tc * kTC + w * 128 < a.cols_pad)
                        *reinterpret_cast<uint32_t *>(a.scales + ((tc * kTC + w * 128) / 128) * a.ld_scales + 4 * r) =
                            *reinterpret_cast<const uint32_t *>(&st_rs[t][4 * w]);
            }
        } else if (t >= kThreads - kTC) {
            const int cl = t - (kThreads - kTC);
            const int64_t c = tc * kTC + cl;
            if (a.scales_t && c < a.cols)
                *reinterpret_cast<uint32_t *>(a.scales_t + tr * a.ld_scales_t + 4 * c) =
                    *reinterpret_cast<const uint32_t *>(&st_cs[cl][0]);
        }
        return;
    }
    // the block's scale byte, from one lane per 32 x 32 block (lane geometry
    // recomputed, as above)
    int t = threadIdx.x;
    asm volatile("" : "+v"(t));
    const int tw = t >> 6, tl = t & 63;
    if (tc * kTC + (tw % WC) * 128 < a.cols_pad && (tl >> 4) == 0 && (tl & 3) == 0) {
        const uint8_t sbyte = finite ? (uint8_t)(e + 127) : (uint8_t)0xFF;
        const int64_t rb = (tr * kTile + (tw / WC) * 32) >> 5, cb = (tc * kTC + (tw % WC) * 128 + 8 * (tl & 15)) >> 5;
        if (a.scales && rb < a.nbr) a.scales[rb * a.ld_scales + cb] = sbyte;
        if (a.scales_t && cb < a.nbc) a.scales_t[cb * a.ld_scales_t + rb] = sbyte;
    }
}

// A lane holds its 8 x 8 sub-block (32 registers of bf16 pairs, 64 of float32)
// and converts each element once, so the bf16 vector-load variants take 91-115
// VGPRs with nothing spilled (four or five waves per SIMD).  Of the bounds below
// (at most 168 VGPRs for stochastic rounding, whose Philox latency needs three
// waves per SIMD; at most 128 for round to nearest) only the float32
// round-to-nearest variants reach theirs.
// Spilled registers cost HBM writes here, not only latency: every wave's spill
// lines end up evicted by the streaming traffic.
template <typename T, bool VEC, bool SR, bool ALIGNED8, bool GROUPED, int WC, bool ONED>
__global__ __launch_bounds__(256 * WC)
__attribute__((amdgpu_waves_per_eu(VEC && SR ? 3 : (VEC ? 4 : 1)))) void fp4_quantize_kernel(QuantArgs a)
{
    static_assert(!(ONED && GROUPED), "grouped tensors use 2D blocks");
    constexpr int kTC = 128 * WC;
    const int64_t tiles_c = (a.cols_pad + kTC - 1) / kTC;
    if constexpr (GROUPED) {
        // padded start rows of the segments, built once per workgroup; the
        // workgroup then walks the row tiles of all segments (tile = blockIdx.x,
        // + gridDim.x, ...) and narrows `a` to each tile's segment
        __shared__ int32_t pad_start[kMaxSegs + 1];
        __shared__ int32_t off[kMaxSegs + 1];
        if ((threadIdx.x >> 6) == 0) {
            wave_offsets(a.nseg, a.seg_offsets, a.rows, off);
            __builtin_amdgcn_wave_barrier();
            wave_prefix(a.nseg, [&](int i) { return (off[i + 1] - off[i] + 127) / 128 * 128; }, pad_start);
        }
        __syncthreads();
        const int64_t tiles = (int64_t)(pad_start[a.nseg] / kTile) * tiles_c;
        for (int64_t tile = blockIdx.x; tile < tiles; tile += gridDim.x) {
            const int64_t rt = tile / tiles_c, tc = tile - rt * tiles_c;
            const int32_t prow = (int32_t)(rt * kTile);
            // the tile's segment (wave-uniform: scalar registers for the narrowed arguments)
            const int e = __builtin_amdgcn_readfirstlane(seg_search(pad_start, a.nseg, prow));
            const int32_t o_e = __builtin_amdgcn_readfirstlane(off[e]);
            const int64_t r_begin = o_e, n_e = (int64_t)__builtin_amdgcn_readfirstlane(off[e + 1]) - o_e;
            const int32_t p_e = __builtin_amdgcn_readfirstlane(pad_start[e]);
            QuantArgs b = a;
            b.x = reinterpret_cast<const uint8_t *>(a.x) + r_begin * a.stride_r * (int64_t)sizeof(T);
            b.index_base += r_begin * a.stride_r;
            b.rows = n_e;
            b.store_rows = (n_e + 127) / 128 * 128;
            b.nbr = b.store_rows / 32;
            if (b.codes) b.codes += (int64_t)p_e * a.ld_codes;
            if (b.codes_t) b.codes_t += p_e / 2;
            if (b.scales) b.scales += (int64_t)(p_e / 32) * a.ld_scales;
            if (b.scales_t) b.scales_t += p_e / 32;
            quantize_tile<T, VEC, SR, ALIGNED8, GROUPED, WC, ONED>(b, (prow - p_e) / kTile, tc);
            __syncthreads();                // the tile's LDS staging is reused by the next
        }
    } else {
        const int64_t tile = blockIdx.x;
        const int64_t tr = tile / tiles_c;
        quantize_tile<T, VEC, SR, ALIGNED8, GROUPED, WC, ONED>(a, tr, tile - tr * tiles_c);
    }
}

template <typename T, bool VEC, bool SR, bool A8, bool G, bool ONED>
hipError_t launch_t(const QuantArgs &a, hipStream_t s)
{
    // 256-column tiles of 8 waves in both rounding modes: the row-packed codes
    // leave as whole 128-byte lines
    constexpr int WC = 2;
    int64_t nb = (a.rows_pad / kTile) * ((a.cols_pad + 128 * WC - 1) / (128 * WC));
    // grouped: each workgroup walks several tiles, so that the segment table is
    // built once per few tiles (the bound covers every padded segment's tiles);
    // 8 per CU keeps the last round of tiles short
    if (G) nb = nb < 8 * (int64_t)cu_count() ? nb : 8 * (int64_t)cu_count();
    hipLaunchKernelGGL((fp4_quantize_kernel<T, VEC, SR, A8, G, WC, ONED>), dim3((unsigned)nb), dim3(256 * WC), 0, s,
                       a);
    return hipGetLastError();
}

template <typename T, bool G, bool ONED>
hipError_t launch_dtype(const QuantArgs &a, bool vec, bool sr, bool a8, hipStream_t s)
{
    if (vec) {
        if (!sr) return launch_t<T, true, false, true, G, ONED>(a, s);
        return a8 ? launch_t<T, true, true, true, G, ONED>(a, s) : launch_t<T, true, true, false, G, ONED>(a, s);
    }
    return sr ? launch_t<T, false, true, true, G, ONED>(a, s) : launch_t<T, false, false, true, G, ONED>(a, s);
}

}  // namespace

hipError_t launch_fp4_quantize(const QuantArgs &a, int dtype_bytes, bool sr, bool oned, hipStream_t stream)
{
    const uintptr_t base = reinterpret_cast<uintptr_t>(a.x);
    const bool vec = a.stride_c == 1 && (base % 16) == 0 && ((a.stride_r * dtype_bytes) % 16) == 0;
    const bool a8 = (a.stride_r % 8) == 0 && (a.index_base % 8) == 0;
    const bool grouped = a.seg_offsets != nullptr;
    if (oned) {
        if (grouped) return hipErrorInvalidValue;
        return dtype_bytes == 4 ? launch_dtype<float, false, true>(a, vec, sr, a8, stream)
                                : launch_dtype<uint16_t, false, true>(a, vec, sr, a8, stream);
    }
    if (dtype_bytes == 4)
        return grouped ? launch_dtype<float, true, false>(a, vec, sr, a8, stream)
                       : launch_dtype<float, false, false>(a, vec, sr, a8, stream);
    return grouped ? launch_dtype<uint16_t, true, false>(a, vec, sr, a8, stream)
                   : launch_dtype<uint16_t, false, false>(a, vec, sr, a8, stream);
}

}  // namespace q2d
