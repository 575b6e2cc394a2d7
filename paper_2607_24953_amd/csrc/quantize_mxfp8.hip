// MXFP8 quantizer for the query/key projections (Sec. 3.2; App. C).
//
// E4M3 codes rounded to nearest even with one truncation-free E8M0 scale per
// 1 x 32 block (smallest power of two S with 448 * S >= block maximum).  One
// pass emits the rowwise copy (blocks along columns, K = cols) and the colwise
// copy (blocks along rows, stored transposed so that K = rows is contiguous),
// which is what the data-gradient and weight-gradient GEMMs read.
//
// Same work split as the FP4 quantizer: 4 waves x (32 x 128) strips, each lane
// an 8 x 8 sub-block (bf16 rows kept packed two elements per register).  A
// 1 x 32 row block spans the 4 lanes that differ in lane bits 0-1; a 32 x 1
// column block spans the 4 lanes that differ in bits 4-5.  The E4M3 codes come
// from gfx950's v_cvt_scalef32_pk_fp8_{bf16,f32} (round to nearest even of
// x / S, two elements per instruction).  Rowwise codes leave as 8-byte stores
// (16 lanes cover a 128-byte row); the colwise codes and both scale grids go
// through LDS and leave as 16- and 4-byte stores.
#include "device_common.hpp"
#include "kernels.hpp"

namespace q2d {

namespace {

constexpr int kTile = 128;

typedef short s2v __attribute__((ext_vector_type(2)));
typedef unsigned int u4v __attribute__((ext_vector_type(4)));

// 16-byte streaming load (the input is read once)
__device__ __forceinline__ uint4 load_stream16(const void *p)
{
    const u4v v = __builtin_nontemporal_load(reinterpret_cast<const u4v *>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t load_bits(const void *x, bool is_f32, int64_t idx)
{
    if (is_f32) return f_bits(reinterpret_cast<const float *>(x)[idx]);
    return (uint32_t)reinterpret_cast<const uint16_t *>(x)[idx] << 16;
}

// E4M3 pair (low element first) into 16-bit word SEL of `old`
template <bool SEL>
__device__ __forceinline__ uint32_t fp8_pair_bf16(uint32_t old, uint32_t packed, float scale)
{
    const s2v r = __builtin_amdgcn_cvt_scalef32_pk_fp8_bf16(__builtin_bit_cast(s2v, old),
                                                            __builtin_bit_cast(bf16x2, packed), scale, SEL);
    return __builtin_bit_cast(uint32_t, r);
}
template <bool SEL>
__device__ __forceinline__ uint32_t fp8_pair_f32(uint32_t old, uint32_t lo, uint32_t hi, float scale)
{
    const s2v r = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(__builtin_bit_cast(s2v, old), bits_f(lo), bits_f(hi),
                                                           scale, SEL);
    return __builtin_bit_cast(uint32_t, r);
}

template <bool F32, bool VEC>
__global__ __launch_bounds__(256) void mxfp8_quantize_kernel(const QuantArgs a)
{
    constexpr bool PK = !F32;                 // bf16: two elements per register
    constexpr int NV = PK ? 4 : 8;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int64_t tiles_c = a.cols_pad / kTile;
    const int64_t tile = blockIdx.x;
    const int64_t tr = tile / tiles_c, tc = tile - tr * tiles_c;
    const int64_t strip_r = tr * kTile + wave * 32;
    const int rg = lane >> 4, cc = lane & 15;
    const int64_t r0 = strip_r + 8 * rg;
    const int64_t c0 = tc * kTile + 8 * cc;

    // ---- load the 8 x 8 sub-block (0 outside R x C)
    uint32_t v[8][NV];
    if (VEC && c0 + 8 <= a.cols) {
        const uint8_t *xr = reinterpret_cast<const uint8_t *>(a.x) + (r0 * a.stride_r + c0) * (F32 ? 4 : 2);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            uint4 q0 = make_uint4(0u, 0u, 0u, 0u), q1 = q0;
            if (r0 + i < a.rows) {
                q0 = load_stream16(xr);
                if (F32) q1 = load_stream16(xr + 16);
            }
            v[i][0] = q0.x; v[i][1] = q0.y; v[i][2] = q0.z; v[i][3] = q0.w;
            if (F32) { v[i][NV - 4] = q1.x; v[i][NV - 3] = q1.y; v[i][NV - 2] = q1.z; v[i][NV - 1] = q1.w; }
            xr += a.stride_r * (F32 ? 4 : 2);
        }
    } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int64_t r = r0 + i;
#pragma unroll
            for (int k = 0; k < NV; ++k) {
                if (PK) {
                    const int64_t c = c0 + 2 * k;
                    const uint32_t lo = (r < a.rows && c < a.cols) ? load_bits(a.x, false, r * a.stride_r + c * a.stride_c) : 0u;
                    const uint32_t hi = (r < a.rows && c + 1 < a.cols) ? load_bits(a.x, false, r * a.stride_r + (c + 1) * a.stride_c) : 0u;
                    v[i][k] = (lo >> 16) | hi;
                } else {
                    const int64_t c = c0 + k;
                    v[i][k] = (r < a.rows && c < a.cols) ? load_bits(a.x, true, r * a.stride_r + c * a.stride_c) : 0u;
                }
            }
        }
    }
    // float32 bit pattern of element (i, j)
    auto elem = [&](int i, int j) -> uint32_t {
        if (PK) return (j & 1) ? (v[i][j >> 1] & 0xFFFF0000u) : (v[i][j >> 1] << 16);
        return v[i][j];
    };

    // ---- block maxima on |bits|: rows (1 x 32, lanes ^1 ^2), columns (32 x 1, lanes ^16 ^32)
    uint32_t rmax[8], cmax[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        uint32_t m = 0;
#pragma unroll
        for (int j = 0; j < 8; ++j) m = max(m, elem(i, j) & 0x7FFFFFFFu);
        m = max(m, (uint32_t)__shfl_xor((int)m, 1));
        m = max(m, (uint32_t)__shfl_xor((int)m, 2));
        rmax[i] = m;
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        uint32_t m = 0;
#pragma unroll
        for (int i = 0; i < 8; ++i) m = max(m, elem(i, j) & 0x7FFFFFFFu);
        m = max(m, (uint32_t)__shfl_xor((int)m, 16));
        m = max(m, (uint32_t)__shfl_xor((int)m, 32));
        cmax[j] = m;
    }

    __shared__ uint32_t st_c[kTile][33];      // column c: 128 codes (rows of the tile) + pad
    __shared__ uint8_t st_sr[kTile][4];       // row scales of the tile's four 1 x 32 blocks
    __shared__ uint8_t st_sc[kTile][4];       // column scales of the four 32 x 1 blocks

    // ---- rowwise copy: 8 codes of row i (two words), stored directly
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int64_t r = r0 + i;
        const bool finite = rmax[i] < 0x7F800000u;
        const int e = fp8_block_exponent(rmax[i]);
        const float scale = bits_f((uint32_t)(127 + e) << 23);
        uint32_t lo = 0, hi = 0;
        if (PK) {
            lo = fp8_pair_bf16<false>(lo, v[i][0], scale);
            lo = fp8_pair_bf16<true>(lo, v[i][PK ? 1 : 0], scale);
            hi = fp8_pair_bf16<false>(hi, v[i][PK ? 2 : 0], scale);
            hi = fp8_pair_bf16<true>(hi, v[i][PK ? 3 : 0], scale);
        } else {
            lo = fp8_pair_f32<false>(lo, elem(i, 0), elem(i, 1), scale);
            lo = fp8_pair_f32<true>(lo, elem(i, 2), elem(i, 3), scale);
            hi = fp8_pair_f32<false>(hi, elem(i, 4), elem(i, 5), scale);
            hi = fp8_pair_f32<true>(hi, elem(i, 6), elem(i, 7), scale);
        }
        if (!finite) { lo = 0; hi = 0; }
        if (a.codes && r < a.rows) *reinterpret_cast<uint2 *>(a.codes + r * a.ld_codes + c0) = make_uint2(lo, hi);
        if ((cc & 3) == 0) st_sr[wave * 32 + 8 * rg + i][cc >> 2] = finite ? (uint8_t)(e + 127) : (uint8_t)0xFF;
    }
    // ---- colwise copy: 8 codes of column j (rows r0 .. r0+7) into LDS
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const bool finite = cmax[j] < 0x7F800000u;
        const int e = fp8_block_exponent(cmax[j]);
        const float scale = bits_f((uint32_t)(127 + e) << 23);
        uint32_t lo = 0, hi = 0;
        if (PK) {
            const int k = j >> 1;
            auto pr = [&](int m) -> uint32_t {
                const uint32_t x0 = v[2 * m][k], x1 = v[2 * m + 1][k];
                return (j & 1) ? ((x0 >> 16) | (x1 & 0xFFFF0000u)) : ((x0 & 0xFFFFu) | (x1 << 16));
            };
            lo = fp8_pair_bf16<false>(lo, pr(0), scale);
            lo = fp8_pair_bf16<true>(lo, pr(1), scale);
            hi = fp8_pair_bf16<false>(hi, pr(2), scale);
            hi = fp8_pair_bf16<true>(hi, pr(3), scale);
        } else {
            lo = fp8_pair_f32<false>(lo, elem(0, j), elem(1, j), scale);
            lo = fp8_pair_f32<true>(lo, elem(2, j), elem(3, j), scale);
            hi = fp8_pair_f32<false>(hi, elem(4, j), elem(5, j), scale);
            hi = fp8_pair_f32<true>(hi, elem(6, j), elem(7, j), scale);
        }
        if (!finite) { lo = 0; hi = 0; }
        st_c[8 * cc + j][wave * 8 + 2 * rg] = lo;
        st_c[8 * cc + j][wave * 8 + 2 * rg + 1] = hi;
        if (rg == 0) st_sc[8 * cc + j][wave] = finite ? (uint8_t)(e + 127) : (uint8_t)0xFF;
    }
    __syncthreads();
    // ---- colwise codes (columns c < C, 16 bytes per lane) and both scale grids
    if (a.codes_t) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int item = threadIdx.x + 256 * q;
            const int line = item >> 3, part = item & 7;
            const int64_t c = tc * kTile + line;
            if (c < a.cols) {
                const uint4 w = make_uint4(st_c[line][4 * part], st_c[line][4 * part + 1],
                                           st_c[line][4 * part + 2], st_c[line][4 * part + 3]);
                *reinterpret_cast<uint4 *>(a.codes_t + c * a.ld_codes_t + tr * kTile + part * 16) = w;
            }
        }
    }
    {
        const int t = threadIdx.x & 127;
        if (threadIdx.x < 128) {
            const int64_t r = tr * kTile + t;
            if (a.scales && r < a.rows)
                *reinterpret_cast<uint32_t *>(a.scales + r * a.ld_scales + tc * 4) =
                    *reinterpret_cast<const uint32_t *>(&st_sr[t][0]);
        } else {
            const int64_t c = tc * kTile + t;
            if (a.scales_t && c < a.cols)
                *reinterpret_cast<uint32_t *>(a.scales_t + c * a.ld_scales_t + tr * 4) =
                    *reinterpret_cast<const uint32_t *>(&st_sc[t][0]);
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
