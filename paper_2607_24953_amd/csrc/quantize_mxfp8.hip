// MXFP8 quantizer for the query/key projections (Sec. 3.2; App. C).
//
// E4M3 codes rounded to nearest even with one truncation-free E8M0 scale per
// 1 x 32 block (smallest power of two S with 448 * S >= block maximum).  One
// pass emits the rowwise copy (blocks along columns, K = cols) and the colwise
// copy (blocks along rows, stored transposed so that K = rows is contiguous),
// which is what the data-gradient and weight-gradient GEMMs read.
//
// Same work split as the FP4 quantizer: 4 waves x (32 x 128) strips, each lane
// an 8 x 8 sub-block.  A 1 x 32 row block spans the 4 lanes that differ in lane
// bits 0-1; a 32 x 1 column block spans the 4 lanes that differ in bits 4-5.
#include "device_common.hpp"
#include "kernels.hpp"

namespace q2d {

namespace {

constexpr int kTile = 128;

__device__ __forceinline__ uint32_t load_bits(const void *x, bool is_f32, int64_t idx)
{
    if (is_f32) return f_bits(reinterpret_cast<const float *>(x)[idx]);
    return (uint32_t)reinterpret_cast<const uint16_t *>(x)[idx] << 16;
}

template <bool F32, bool VEC>
__global__ __launch_bounds__(256) void mxfp8_quantize_kernel(const QuantArgs a)
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
    const bool vec = VEC && c0 + 8 <= a.cols;

    uint32_t v[8][8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int64_t r = r0 + i;
        if (vec && r < a.rows) {
            if (F32) {
                const float *p = reinterpret_cast<const float *>(a.x) + r * a.stride_r + c0;
                const uint4 u0 = *reinterpret_cast<const uint4 *>(p);
                const uint4 u1 = *reinterpret_cast<const uint4 *>(p + 4);
                v[i][0] = u0.x; v[i][1] = u0.y; v[i][2] = u0.z; v[i][3] = u0.w;
                v[i][4] = u1.x; v[i][5] = u1.y; v[i][6] = u1.z; v[i][7] = u1.w;
            } else {
                const uint16_t *p = reinterpret_cast<const uint16_t *>(a.x) + r * a.stride_r + c0;
                const uint4 u = *reinterpret_cast<const uint4 *>(p);
                v[i][0] = u.x << 16; v[i][1] = u.x & 0xFFFF0000u;
                v[i][2] = u.y << 16; v[i][3] = u.y & 0xFFFF0000u;
                v[i][4] = u.z << 16; v[i][5] = u.z & 0xFFFF0000u;
                v[i][6] = u.w << 16; v[i][7] = u.w & 0xFFFF0000u;
            }
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int64_t c = c0 + j;
                v[i][j] = (r < a.rows && c < a.cols) ? load_bits(a.x, F32, r * a.stride_r + c * a.stride_c) : 0u;
            }
        }
    }

    // rowwise (1 x 32) maxima: one per sub-block row, shared by lanes ^1, ^2
    uint32_t rmax[8], cmax[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        uint32_t m = 0;
#pragma unroll
        for (int j = 0; j < 8; ++j) m = max(m, v[i][j] & 0x7FFFFFFFu);
        m = max(m, (uint32_t)__shfl_xor((int)m, 1));
        m = max(m, (uint32_t)__shfl_xor((int)m, 2));
        rmax[i] = m;
    }
    // colwise (32 x 1) maxima: one per sub-block column, shared by lanes ^16, ^32
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        uint32_t m = 0;
#pragma unroll
        for (int i = 0; i < 8; ++i) m = max(m, v[i][j] & 0x7FFFFFFFu);
        m = max(m, (uint32_t)__shfl_xor((int)m, 16));
        m = max(m, (uint32_t)__shfl_xor((int)m, 32));
        cmax[j] = m;
    }

    // ---- rowwise copy
    if (a.codes) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int64_t r = r0 + i;
            const bool finite = rmax[i] < 0x7F800000u;
            const int e = fp8_block_exponent(rmax[i]);
            const float inv = inv_pow2(e);
            uint32_t lo = 0, hi = 0;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const uint32_t b = v[i][j];
                const uint32_t code = finite ? (((b >> 24) & 0x80u) | e4m3_rne(bits_f(b & 0x7FFFFFFFu) * inv)) : 0u;
                if (j < 4) lo |= code << (8 * j); else hi |= code << (8 * (j - 4));
            }
            if (r < a.rows) {
                *reinterpret_cast<uint2 *>(a.codes + r * a.ld_codes + c0) = make_uint2(lo, hi);
                if ((cc & 3) == 0)
                    a.scales[r * a.ld_scales + (c0 >> 5)] = finite ? (uint8_t)(e + 127) : (uint8_t)0xFF;
            }
        }
    }
    // ---- colwise copy, stored transposed
    if (a.codes_t) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int64_t c = c0 + j;
            const bool finite = cmax[j] < 0x7F800000u;
            const int e = fp8_block_exponent(cmax[j]);
            const float inv = inv_pow2(e);
            uint32_t lo = 0, hi = 0;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const uint32_t b = v[i][j];
                const uint32_t code = finite ? (((b >> 24) & 0x80u) | e4m3_rne(bits_f(b & 0x7FFFFFFFu) * inv)) : 0u;
                if (i < 4) lo |= code << (8 * i); else hi |= code << (8 * (i - 4));
            }
            if (c < a.cols) {
                *reinterpret_cast<uint2 *>(a.codes_t + c * a.ld_codes_t + r0) = make_uint2(lo, hi);
                if (rg == 0)
                    a.scales_t[c * a.ld_scales_t + (strip_r >> 5)] = finite ? (uint8_t)(e + 127) : (uint8_t)0xFF;
            }
        }
    }
}

}  // namespace

hipError_t launch_mxfp8_quantize(const QuantArgs &a, int dtype_bytes, hipStream_t stream)
{
    const int64_t nb = (a.rows_pad / kTile) * (a.cols_pad / kTile);
    const uintptr_t base = reinterpret_cast<uintptr_t>(a.x);
    const bool vec = a.stride_c == 1 && (base % 16) == 0 && ((a.stride_r * dtype_bytes) % 16) == 0;
    const dim3 grid((unsigned)nb), block(256);
    if (dtype_bytes == 4) {
        if (vec) hipLaunchKernelGGL((mxfp8_quantize_kernel<true, true>), grid, block, 0, stream, a);
        else hipLaunchKernelGGL((mxfp8_quantize_kernel<true, false>), grid, block, 0, stream, a);
    } else {
        if (vec) hipLaunchKernelGGL((mxfp8_quantize_kernel<false, true>), grid, block, 0, stream, a);
        else hipLaunchKernelGGL((mxfp8_quantize_kernel<false, false>), grid, block, 0, stream, a);
    }
    return hipGetLastError();
}

}  // namespace q2d
