// Dequantization of one stored copy of a quantized matrix back to R x C values,
// with the per-element scale exponent alongside (optional).
//
// This is what each GEMM of a linear layer effectively multiplies (Sec. 2,
// "Bias induced by scale inconsistency": the forward copy X_fwd = round(X/S_fwd)
// S_fwd and the backward copy X_bwd = round(X/S_bwd) S_bwd).  Dequantizing both
// copies of one tensor in the same R x C orientation gives the scale-difference
// and effective-deviation maps of the forward/backward comparison (Fig. 1): zero
// for 2D blocks, non-zero for 1D blocks.
//
// One workgroup per 128 x 128 output tile.  The tile's codes (128 stored rows of
// 64 bytes for FP4, 128 for MXFP8) are staged in LDS with 16-byte loads; then
// each wave writes 32 output rows, two per instruction, a lane covering four
// consecutive columns (16-byte float32 / 8-byte bfloat16 stores: full 512- or
// 256-byte rows per half wave).  A transposed copy (stored K = rows) is read
// from LDS column-wise.  Values are exact in float32 (an E2M1 or E4M3 code times
// a power of two, rounded once only when it leaves float32 range); bfloat16
// output is the round-to-nearest-even of that value.
#include "device_common.hpp"
#include "kernels.hpp"

namespace q2d {

namespace {

constexpr int kTile = 128;

__device__ __forceinline__ uint16_t bf16_rne(float f)
{
    const uint32_t u = f_bits(f);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0;
    return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

// value of an E2M1 nibble times 2^e
__device__ __forceinline__ float fp4_value(uint32_t n, int e)
{
    const uint32_t m = n & 7u;
    // twice the magnitude: 0, 1, 2, 3, 4, 6, 8, 12
    const uint32_t twice = m < 2u ? m : (2u + (m & 1u)) << ((m >> 1) - 1u);
    const float v = ldexpf((float)twice, e - 1);
    return (n & 8u) ? -v : v;
}

// value of an E4M3FN byte times 2^e (S.1111.111 is NaN)
__device__ __forceinline__ float e4m3_value(uint32_t b, int e)
{
    if ((b & 0x7Fu) == 0x7Fu) return __uint_as_float(0x7FC00000u);
    const uint32_t E = (b >> 3) & 15u, m = b & 7u;
    const float v = E ? ldexpf((float)(8u + m), (int)E - 10 + e) : ldexpf((float)m, e - 9);
    return (b & 0x80u) ? -v : v;
}

// FMT: 0 = FP4 2D blocks, 1 = MXFP8, 2 = FP4 1D blocks.  TRANS: the copy is
// stored with K = rows (element (r, c) in stored row c).
template <int FMT, bool TRANS, bool BF16>
__global__ __launch_bounds__(256) void dequantize_kernel(const DequantArgs a)
{
    constexpr int kRowBytes = FMT == 1 ? 128 : 64;      // bytes of 128 codes
    constexpr int kPitch = kRowBytes + 4;
    __shared__ __attribute__((aligned(16))) uint8_t lds[kTile * kPitch];
    const int64_t tiles_c = (a.cols + kTile - 1) / kTile;
    const int64_t tr = blockIdx.x / tiles_c, tc = blockIdx.x - tr * tiles_c;
    const int64_t r0 = tr * kTile, c0 = tc * kTile;
    const int t = threadIdx.x;

    // ---- stage: stored rows s0 .. s0+127 (rows for a row-packed copy, columns
    // for a transposed one), K bytes of this tile
    {
        const int64_t s0 = TRANS ? c0 : r0, k0 = TRANS ? r0 : c0;
        const int64_t ns = TRANS ? a.cols : a.rows;
        const int sl = t >> 1, half = t & 1;
        constexpr int kVec = kRowBytes / 32;               // 16-byte vectors per thread
        const int64_t s = s0 + sl;
        uint8_t *dst = lds + sl * kPitch + half * (kRowBytes / 2);
#pragma unroll
        for (int v = 0; v < kVec; ++v) {
            uint4 q = make_uint4(0u, 0u, 0u, 0u);
            if (s < ns)
                q = *reinterpret_cast<const uint4 *>(a.codes + s * a.ld_codes + k0 * kRowBytes / kTile +
                                                     half * (kRowBytes / 2) + 16 * v);
            uint32_t *d = reinterpret_cast<uint32_t *>(dst + 16 * v);
            d[0] = q.x; d[1] = q.y; d[2] = q.z; d[3] = q.w;
        }
    }
    __syncthreads();

    // scale byte of stored row s, K index k
    auto scale_byte = [&](int64_t s, int64_t k) -> uint32_t {
        if (FMT == 0) return a.scales[(s >> 5) * a.ld_scales + (k >> 5)];
        if (FMT == 2) return a.scales[(k >> 7) * a.ld_scales + 4 * s + ((k >> 5) & 3)];
        return a.scales[s * a.ld_scales + (k >> 5)];
    };

    const int wave = t >> 6, lane = t & 63;
    const int cg = lane & 31;
    const int64_t c = c0 + 4 * cg;
#pragma unroll 2
    for (int it = 0; it < 16; ++it) {
        const int rl = wave * 32 + 2 * it + (lane >> 5);
        const int64_t r = r0 + rl;
        if (r >= a.rows || c >= a.cols) continue;
        // codes of the four elements (r, c .. c+3)
        uint32_t code[4];
        if (!TRANS) {
            if (FMT == 1) {
                const uint32_t w = *reinterpret_cast<const uint32_t *>(lds + rl * kPitch + 4 * cg);
#pragma unroll
                for (int j = 0; j < 4; ++j) code[j] = (w >> (8 * j)) & 0xFFu;
            } else {
                const uint32_t w = *reinterpret_cast<const uint16_t *>(lds + rl * kPitch + 2 * cg);
#pragma unroll
                for (int j = 0; j < 4; ++j) code[j] = (w >> (4 * j)) & 15u;
            }
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const uint8_t *row = lds + (4 * cg + j) * kPitch;
                code[j] = FMT == 1 ? row[rl] : (row[rl >> 1] >> (4 * (rl & 1))) & 15u;
            }
        }
        // scale bytes: one for a 2D block or a row block (the four columns share
        // it), one per column for column blocks
        uint32_t sb[4];
        if (!TRANS) {
            const uint32_t s = scale_byte(r, c);
#pragma unroll
            for (int j = 0; j < 4; ++j) sb[j] = s;
        } else if (FMT == 0) {
            const uint32_t s = scale_byte(c, r);
#pragma unroll
            for (int j = 0; j < 4; ++j) sb[j] = s;
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) sb[j] = c + j < a.cols ? scale_byte(c + j, r) : 0u;
        }
        float v[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int e = (int)sb[j] - 127;
            v[j] = sb[j] == 0xFFu ? __uint_as_float(0x7FC00000u)
                                  : (FMT == 1 ? e4m3_value(code[j], e) : fp4_value(code[j], e));
        }
        const bool full = c + 4 <= a.cols;
        if (BF16) {
            uint16_t *o = reinterpret_cast<uint16_t *>(a.out) + r * a.ldo + c;
            if (full && a.out_vec) {
                *reinterpret_cast<uint2 *>(o) =
                    make_uint2((uint32_t)bf16_rne(v[0]) | (uint32_t)bf16_rne(v[1]) << 16,
                               (uint32_t)bf16_rne(v[2]) | (uint32_t)bf16_rne(v[3]) << 16);
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (c + j < a.cols) o[j] = bf16_rne(v[j]);
            }
        } else {
            float *o = reinterpret_cast<float *>(a.out) + r * a.ldo + c;
            if (full && a.out_vec) {
                *reinterpret_cast<float4 *>(o) = make_float4(v[0], v[1], v[2], v[3]);
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (c + j < a.cols) o[j] = v[j];
            }
        }
        if (a.exps) {
            int8_t *x = a.exps + r * a.lde + c;
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (c + j < a.cols) x[j] = sb[j] == 0xFFu ? (int8_t)-128 : (int8_t)((int)sb[j] - 127);
        }
    }
}

template <int FMT, bool TRANS>
hipError_t launch_fmt(const DequantArgs &a, hipStream_t s)
{
    const int64_t tiles = ((a.rows + kTile - 1) / kTile) * ((a.cols + kTile - 1) / kTile);
    if (a.out_bf16)
        hipLaunchKernelGGL((dequantize_kernel<FMT, TRANS, true>), dim3((unsigned)tiles), dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL((dequantize_kernel<FMT, TRANS, false>), dim3((unsigned)tiles), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_dequantize(const DequantArgs &a, hipStream_t stream)
{
    const int64_t tiles = ((a.rows + kTile - 1) / kTile) * ((a.cols + kTile - 1) / kTile);
    if (tiles <= 0 || tiles > 0x7FFFFFFF) return hipErrorInvalidValue;
    switch (a.fmt * 2 + (a.transposed ? 1 : 0)) {
    case 0: return launch_fmt<0, false>(a, stream);
    case 1: return launch_fmt<0, true>(a, stream);
    case 2: return launch_fmt<1, false>(a, stream);
    case 3: return launch_fmt<1, true>(a, stream);
    case 4: return launch_fmt<2, false>(a, stream);
    case 5: return launch_fmt<2, true>(a, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace q2d
