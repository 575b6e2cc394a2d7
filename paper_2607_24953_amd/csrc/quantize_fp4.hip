// Fused 2D-block FP4 quantizer (Sec. 3, Sec. 3.1; App. D, App. E).
//
// One pass over the input: block maximum, truncation-free E8M0 scale, round to
// nearest or Philox stochastic rounding, and both packed layouts (row-packed
// codes and column-packed codes_t) plus the scale grid and its transpose.
//
// Work split: a workgroup of 4 waves owns a 128 x 128 tile, each wave a
// 32 x 128 strip (four 32 x 32 blocks side by side).  Lane l owns an 8 x 8
// sub-block: rows 8*(l/16) .. +7 and columns 8*(l%16) .. +7 of the strip.  A
// row of the sub-block is one 16-byte load (bf16), so every load instruction
// of the wave reads four 256-byte row segments.  The 8 x 8 sub-block makes the
// transposition free: each lane packs eight nibbles per row for codes and eight
// per column for codes_t without any data exchange.  The block maximum is a
// max over the lane's 64 values followed by four cross-lane butterflies (the 16
// lanes of a 32 x 32 block differ in lane bits 0, 1, 4 and 5).
#include "device_common.hpp"
#include "kernels.hpp"

namespace q2d {

namespace {

constexpr int kTile = 128;

template <typename T>
struct Elem;

template <>
struct Elem<float> {
    static __device__ __forceinline__ uint32_t bits(const float *p) { return f_bits(*p); }
    // eight consecutive elements of one row, 16-byte aligned
    static __device__ __forceinline__ void load8(const float *p, uint32_t out[8])
    {
        const uint4 a = *reinterpret_cast<const uint4 *>(p);
        const uint4 b = *reinterpret_cast<const uint4 *>(p + 4);
        out[0] = a.x; out[1] = a.y; out[2] = a.z; out[3] = a.w;
        out[4] = b.x; out[5] = b.y; out[6] = b.z; out[7] = b.w;
    }
};

template <>
struct Elem<uint16_t> {
    static __device__ __forceinline__ uint32_t bits(const uint16_t *p) { return (uint32_t)*p << 16; }
    static __device__ __forceinline__ void load8(const uint16_t *p, uint32_t out[8])
    {
        const uint4 a = *reinterpret_cast<const uint4 *>(p);
        out[0] = a.x << 16; out[1] = a.x & 0xFFFF0000u;
        out[2] = a.y << 16; out[3] = a.y & 0xFFFF0000u;
        out[4] = a.z << 16; out[5] = a.z & 0xFFFF0000u;
        out[6] = a.w << 16; out[7] = a.w & 0xFFFF0000u;
    }
};

// VEC: rows are read as aligned 8-element vectors (stride_c == 1).
// SR: stochastic rounding.  ALIGNED8: every sub-block row starts at a storage
// index that is a multiple of 8, so one Philox block serves its 8 elements.
template <typename T, bool VEC, bool SR, bool ALIGNED8>
__global__ __launch_bounds__(256) void fp4_quantize_kernel(const QuantArgs a)
{
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int64_t tiles_c = a.cols_pad / kTile;
    const int64_t tile = blockIdx.x;
    const int64_t tr = tile / tiles_c, tc = tile - tr * tiles_c;
    const int64_t strip_r = tr * kTile + wave * 32;
    const int rg = lane >> 4, cc = lane & 15;
    const int64_t r0 = strip_r + 8 * rg;
    const int64_t c0 = tc * kTile + 8 * cc;
    const T *x = reinterpret_cast<const T *>(a.x);

    // ---- load the 8 x 8 sub-block as float32 bit patterns (0 outside R x C)
    uint32_t v[8][8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int64_t r = r0 + i;
        if (VEC && r < a.rows && c0 + 8 <= a.cols) {
            Elem<T>::load8(x + r * a.stride_r + c0, v[i]);
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int64_t c = c0 + j;
                v[i][j] = (r < a.rows && c < a.cols) ? Elem<T>::bits(x + r * a.stride_r + c * a.stride_c) : 0u;
            }
        }
    }

    // ---- block maximum on |bits| (NaN > inf > finite, as unsigned integers)
    uint32_t am = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) am = max(am, v[i][j] & 0x7FFFFFFFu);
    am = max(am, (uint32_t)__shfl_xor((int)am, 1));
    am = max(am, (uint32_t)__shfl_xor((int)am, 2));
    am = max(am, (uint32_t)__shfl_xor((int)am, 16));
    am = max(am, (uint32_t)__shfl_xor((int)am, 32));
    const bool finite = am < 0x7F800000u;
    const int e = fp4_block_exponent(am);
    const float inv = inv_pow2(e);

    // ---- encode
    uint32_t rowp[8], colp[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) { rowp[i] = 0; colp[i] = 0; }
    const uint32_t k0 = (uint32_t)a.seed, k1 = (uint32_t)(a.seed >> 32);
    const uint32_t o0 = (uint32_t)a.offset, o1 = (uint32_t)(a.offset >> 32);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        uint32_t w[4] = {0, 0, 0, 0}, w2[4] = {0, 0, 0, 0};
        uint64_t idx0 = 0;
        if (SR && VEC) {
            idx0 = (uint64_t)(a.index_base + (r0 + i) * a.stride_r + c0);
            const uint64_t g = idx0 >> 3;
            philox4x32_10((uint32_t)g, (uint32_t)(g >> 32), o0, o1, k0, k1, w);
            if (!ALIGNED8) {
                const uint64_t g2 = g + 1;
                philox4x32_10((uint32_t)g2, (uint32_t)(g2 >> 32), o0, o1, k0, k1, w2);
            }
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const uint32_t b = v[i][j];
            const float ax = bits_f(b & 0x7FFFFFFFu) * inv;
            uint32_t mag;
            if (SR) {
                uint32_t r16;
                if (VEC) {
                    if (ALIGNED8) {
                        r16 = (w[j >> 1] >> ((j & 1) * 16)) & 0xFFFFu;
                    } else {
                        const uint32_t q = (uint32_t)(idx0 & 7u) + (uint32_t)j;     // 0..14
                        const uint32_t s = q & 7u;
                        const uint32_t wa = (s & 4u) ? ((s & 2u) ? w[3] : w[2]) : ((s & 2u) ? w[1] : w[0]);
                        const uint32_t wb = (s & 4u) ? ((s & 2u) ? w2[3] : w2[2]) : ((s & 2u) ? w2[1] : w2[0]);
                        r16 = ((q < 8u ? wa : wb) >> ((s & 1u) * 16u)) & 0xFFFFu;
                    }
                } else {
                    const uint64_t idx = (uint64_t)(a.index_base + (r0 + i) * a.stride_r + (c0 + j) * a.stride_c);
                    r16 = sr_draw(idx, k0, k1, o0, o1);
                }
                mag = e2m1_sr(ax, r16);
            } else {
                mag = e2m1_rtn(ax);
            }
            const uint32_t code = ((b >> 28) & 8u) | mag;
            rowp[i] |= code << (4 * j);
            colp[j] |= code << (4 * i);
        }
    }
    if (!finite) {
#pragma unroll
        for (int i = 0; i < 8; ++i) { rowp[i] = 0; colp[i] = 0; }
    }

    // ---- stores: codes rows r < R, codes_t rows c < C, scale bytes once per block
    if (a.codes) {
#pragma unroll
        for (int i = 0; i < 8; ++i)
            if (r0 + i < a.rows)
                *reinterpret_cast<uint32_t *>(a.codes + (r0 + i) * a.ld_codes + (c0 >> 1)) = rowp[i];
    }
    if (a.codes_t) {
#pragma unroll
        for (int j = 0; j < 8; ++j)
            if (c0 + j < a.cols)
                *reinterpret_cast<uint32_t *>(a.codes_t + (c0 + j) * a.ld_codes_t + (r0 >> 1)) = colp[j];
    }
    if (rg == 0 && (cc & 3) == 0) {
        const uint8_t sbyte = finite ? (uint8_t)(e + 127) : (uint8_t)0xFF;
        const int64_t rb = strip_r >> 5, cb = c0 >> 5;
        if (a.scales && rb < a.nbr) a.scales[rb * a.ld_scales + cb] = sbyte;
        if (a.scales_t && cb < a.nbc) a.scales_t[cb * a.ld_scales_t + rb] = sbyte;
    }
}

template <typename T, bool VEC, bool SR, bool A8>
hipError_t launch_t(const QuantArgs &a, int64_t nblocks, hipStream_t s)
{
    hipLaunchKernelGGL((fp4_quantize_kernel<T, VEC, SR, A8>), dim3((unsigned)nblocks), dim3(256), 0, s, a);
    return hipGetLastError();
}

template <typename T>
hipError_t launch_dtype(const QuantArgs &a, bool vec, bool sr, bool a8, int64_t nb, hipStream_t s)
{
    if (vec) {
        if (!sr) return launch_t<T, true, false, true>(a, nb, s);
        return a8 ? launch_t<T, true, true, true>(a, nb, s) : launch_t<T, true, true, false>(a, nb, s);
    }
    return sr ? launch_t<T, false, true, true>(a, nb, s) : launch_t<T, false, false, true>(a, nb, s);
}

}  // namespace

hipError_t launch_fp4_quantize(const QuantArgs &a, int dtype_bytes, bool sr, hipStream_t stream)
{
    const int64_t nb = (a.rows_pad / kTile) * (a.cols_pad / kTile);
    const uintptr_t base = reinterpret_cast<uintptr_t>(a.x);
    const bool vec = a.stride_c == 1 && (base % 16) == 0 && ((a.stride_r * dtype_bytes) % 16) == 0;
    const bool a8 = (a.stride_r % 8) == 0 && (a.index_base % 8) == 0;
    if (dtype_bytes == 4) return launch_dtype<float>(a, vec, sr, a8, nb, stream);
    return launch_dtype<uint16_t>(a, vec, sr, a8, nb, stream);
}

}  // namespace q2d
