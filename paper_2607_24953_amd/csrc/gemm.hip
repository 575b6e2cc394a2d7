// Block-scaled GEMM on CDNA4 scaled MFMA: C[M][N] (+)= A . B^T with K-major
// quantized operands (Sec. 3 "Application to linear layers"; App. C).
//
// v_mfma_scale_f32_32x32x64_f8f6f4 multiplies a 32 x 64 slice of A by a 64 x 32
// slice of B^T.  Lane l holds row (l % 32) and the 32-element K-group (l / 32)
// of each operand and one E8M0 scale byte for that (row, K-group).  For 2D-block
// FP4 the 32 rows of a tile are exactly one block row, so every lane of a row
// tile passes the same block scale and the scale of block (i, j) is replicated
// over the K-group j of its 32 rows; the column-packed copy of an operand has
// the same codes and the same scales with the block index swapped, which is
// what lets one quantization serve Y = X W^T, dX = dY W and dW = dY^T X.  For
// MXFP8 each row has its own scale per K-group.
//
// Tiling: 256 threads, 128 x 128 output tile, 2 x 2 waves of 64 x 64 (2 x 2
// MFMA tiles each), K-tile of 128 elements staged in LDS with double
// buffering.  LDS rows are XOR-swizzled in 16-byte chunks so that the MFMA
// operand reads (32 consecutive rows, same chunk) hit distinct banks.
// Workgroups are remapped so that each XCD (one L2) walks a contiguous band of
// output tiles, grouped by 8 row tiles for operand reuse.
#include "device_common.hpp"
#include "kernels.hpp"

namespace q2d {

namespace {

constexpr int BM = 128, BN = 128, BK = 128;
constexpr int kThreads = 256;
constexpr int kGroupM = 8;
constexpr int kXcds = 8;

template <int FMT>
struct Fmt;

template <>
struct Fmt<kFmtFp4Block2D> {
    static constexpr int kRowBytes = BK / 2;      // 64 bytes of codes per row per K-tile
    static constexpr int kLaneBytes = 16;         // 32 E2M1 codes per lane per MFMA
    static constexpr int kCbsz = 4;               // E2M1
    static constexpr int kScaleRowShift = 5;      // one scale per 32-row block
    static __device__ __forceinline__ int swz(int r) { return ((r >> 1) ^ (r >> 3)) & 3; }
};

template <>
struct Fmt<kFmtMxfp8> {
    static constexpr int kRowBytes = BK;          // 128 bytes per row per K-tile
    static constexpr int kLaneBytes = 32;         // 32 E4M3 codes per lane per MFMA
    static constexpr int kCbsz = 0;               // E4M3
    static constexpr int kScaleRowShift = 0;      // one scale per row and K-group
    static __device__ __forceinline__ int swz(int r) { return (r ^ (r >> 3)) & 7; }
};

__device__ __forceinline__ void tile_coords(int64_t tiles_m, int64_t tiles_n, int64_t &tm, int64_t &tn)
{
    // Hardware dispatch sends consecutive workgroups to consecutive XCDs; give
    // every XCD a contiguous range of the tile order instead.
    const int64_t nb = tiles_m * tiles_n;
    const int64_t bid = blockIdx.x;
    const int64_t xcd = bid % kXcds, local = bid / kXcds;
    const int64_t per = nb / kXcds, rem = nb % kXcds;
    const int64_t t = xcd * per + (xcd < rem ? xcd : rem) + local;
    // grouped order: kGroupM row tiles sweep all column tiles together
    const int64_t span = (int64_t)kGroupM * tiles_n;
    const int64_t grp = t / span;
    const int64_t first = grp * kGroupM;
    const int64_t gsz = (tiles_m - first) < kGroupM ? (tiles_m - first) : kGroupM;
    const int64_t in = t - grp * span;
    tm = first + in % gsz;
    tn = in / gsz;
}

template <int FMT, bool BF16OUT>
__global__ __launch_bounds__(kThreads) void gemm_kernel(const GemmArgs g, int64_t tiles_m, int64_t tiles_n)
{
    using F = Fmt<FMT>;
    constexpr int RB = F::kRowBytes;
    constexpr int NCH = RB / 16;                    // 16-byte chunks per row
    constexpr int LOADS = (BM * NCH) / kThreads;    // chunks per thread per operand
    __shared__ __attribute__((aligned(16))) uint8_t As[2][BM * RB];
    __shared__ __attribute__((aligned(16))) uint8_t Bs[2][BN * RB];

    int64_t tm, tn;
    tile_coords(tiles_m, tiles_n, tm, tn);
    const int64_t m0 = tm * BM, n0 = tn * BN;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int64_t nk = g.K / BK;

    // ---- global -> LDS staging addresses (rows clamped into the operand)
    const uint8_t *ga[LOADS];
    const uint8_t *gb[LOADS];
    int lds_off[LOADS];
#pragma unroll
    for (int s = 0; s < LOADS; ++s) {
        const int q = tid + s * kThreads;
        const int r = q / NCH, c = q % NCH;
        int64_t ra = m0 + r; ra = ra < g.M ? ra : g.M - 1;
        int64_t rb = n0 + r; rb = rb < g.N ? rb : g.N - 1;
        ga[s] = g.a + ra * g.lda + c * 16;
        gb[s] = g.b + rb * g.ldb + c * 16;
        lds_off[s] = r * RB + ((c ^ F::swz(r)) * 16);
    }

    // ---- per-lane scale rows (clamped)
    const uint8_t *sa_row[2];
    const uint8_t *sb_row[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        int64_t ra = m0 + wm * 64 + i * 32 + (lane & 31); ra = ra < g.M ? ra : g.M - 1;
        int64_t rb = n0 + wn * 64 + i * 32 + (lane & 31); rb = rb < g.N ? rb : g.N - 1;
        sa_row[i] = g.sa + (ra >> F::kScaleRowShift) * g.ldsa;
        sb_row[i] = g.sb + (rb >> F::kScaleRowShift) * g.ldsb;
    }

    v16f acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    uint4 ra_reg[LOADS], rb_reg[LOADS];
#pragma unroll
    for (int s = 0; s < LOADS; ++s) {
        ra_reg[s] = *reinterpret_cast<const uint4 *>(ga[s]);
        rb_reg[s] = *reinterpret_cast<const uint4 *>(gb[s]);
    }
#pragma unroll
    for (int s = 0; s < LOADS; ++s) {
        *reinterpret_cast<uint4 *>(&As[0][lds_off[s]]) = ra_reg[s];
        *reinterpret_cast<uint4 *>(&Bs[0][lds_off[s]]) = rb_reg[s];
    }
    __syncthreads();

    const int half = lane >> 5;
    for (int64_t kt = 0; kt < nk; ++kt) {
        const int buf = (int)(kt & 1);
        if (kt + 1 < nk) {
#pragma unroll
            for (int s = 0; s < LOADS; ++s) {
                ra_reg[s] = *reinterpret_cast<const uint4 *>(ga[s] + (kt + 1) * RB);
                rb_reg[s] = *reinterpret_cast<const uint4 *>(gb[s] + (kt + 1) * RB);
            }
        }
        uint32_t swa[2], swb[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            swa[i] = *reinterpret_cast<const uint32_t *>(sa_row[i] + kt * 4);
            swb[i] = *reinterpret_cast<const uint32_t *>(sb_row[i] + kt * 4);
        }
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            v8i af[2], bf[2];
            int sa[2], sb[2];
            const int kg = 2 * ks + half;
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int ra = wm * 64 + i * 32 + (lane & 31);
                const int rb = wn * 64 + i * 32 + (lane & 31);
                const int cbyte = ks * 2 * F::kLaneBytes + half * F::kLaneBytes;   // byte offset in the row
#pragma unroll
                for (int h = 0; h < F::kLaneBytes / 16; ++h) {
                    const int ch = cbyte / 16 + h;
                    const uint4 qa = *reinterpret_cast<const uint4 *>(&As[buf][ra * RB + ((ch ^ F::swz(ra)) * 16)]);
                    const uint4 qb = *reinterpret_cast<const uint4 *>(&Bs[buf][rb * RB + ((ch ^ F::swz(rb)) * 16)]);
                    af[i][4 * h + 0] = (int)qa.x; af[i][4 * h + 1] = (int)qa.y;
                    af[i][4 * h + 2] = (int)qa.z; af[i][4 * h + 3] = (int)qa.w;
                    bf[i][4 * h + 0] = (int)qb.x; bf[i][4 * h + 1] = (int)qb.y;
                    bf[i][4 * h + 2] = (int)qb.z; bf[i][4 * h + 3] = (int)qb.w;
                }
                if (F::kLaneBytes == 16) {
#pragma unroll
                    for (int z = 4; z < 8; ++z) { af[i][z] = 0; bf[i][z] = 0; }
                }
                sa[i] = (int)((swa[i] >> (8 * kg)) & 0xFFu);
                sb[i] = (int)((swb[i] >> (8 * kg)) & 0xFFu);
            }
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                        af[i], bf[j], acc[i][j], F::kCbsz, F::kCbsz, 0, sa[i], 0, sb[j]);
        }
        if (kt + 1 < nk) {
#pragma unroll
            for (int s = 0; s < LOADS; ++s) {
                *reinterpret_cast<uint4 *>(&As[buf ^ 1][lds_off[s]]) = ra_reg[s];
                *reinterpret_cast<uint4 *>(&Bs[buf ^ 1][lds_off[s]]) = rb_reg[s];
            }
        }
        __syncthreads();
    }

    // ---- epilogue: lane holds column (lane % 32) and rows 8*(r/4) + 4*(lane/32) + r%4
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int64_t col = n0 + wn * 64 + j * 32 + (lane & 31);
            if (col >= g.N) continue;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int64_t row = m0 + wm * 64 + i * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
                if (row >= g.M) continue;
                float v = acc[i][j][r];
                if (BF16OUT) {
                    uint16_t *p = reinterpret_cast<uint16_t *>(g.c) + row * g.ldc + col;
                    if (g.accumulate) v += bf16_to_f(*p);
                    *p = f_to_bf16_rne(v);
                } else {
                    float *p = reinterpret_cast<float *>(g.c) + row * g.ldc + col;
                    if (g.accumulate) v += *p;
                    *p = v;
                }
            }
        }
}

template <int FMT, bool BF>
hipError_t launch_t(const GemmArgs &g, hipStream_t s)
{
    const int64_t tm = (g.M + BM - 1) / BM, tn = (g.N + BN - 1) / BN;
    hipLaunchKernelGGL((gemm_kernel<FMT, BF>), dim3((unsigned)(tm * tn)), dim3(kThreads), 0, s, g, tm, tn);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm(const GemmArgs &g, int fmt, int c_is_bf16, hipStream_t stream)
{
    if (fmt == kFmtFp4Block2D)
        return c_is_bf16 ? launch_t<kFmtFp4Block2D, true>(g, stream) : launch_t<kFmtFp4Block2D, false>(g, stream);
    return c_is_bf16 ? launch_t<kFmtMxfp8, true>(g, stream) : launch_t<kFmtMxfp8, false>(g, stream);
}

}  // namespace q2d
