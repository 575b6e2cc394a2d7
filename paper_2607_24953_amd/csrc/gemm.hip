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
// Two kernels.  Problems with at least 128 output tiles of 256 x 256 run on the
// persistent large-tile kernels further down (gemm_fp4_persistent_kernel, also
// the grouped and quantized-output forms, and gemm_fp8_256_kernel).  Smaller
// problems use gemm_kernel: 256 threads, 128 x 128 output tile, 2 x 2 waves of
// 64 x 64 (2 x 2 MFMA tiles each), K-tile of 128 elements staged in LDS with
// double buffering.  LDS rows are XOR-swizzled in 16-byte chunks (Fmt::swz) so
// that the MFMA operand reads hit distinct banks.  Workgroups are remapped so
// that each XCD (one L2) walks a contiguous band of output tiles, grouped by 8
// row tiles for operand reuse.
#include <atomic>
#include <type_traits>
#include <utility>
#include "device_common.hpp"
#include "kernels.hpp"

namespace q2d {

// compute units of the current device (queried once per device)
int cu_count()
{
    static std::atomic<int> cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    int n = cache[dev].load(std::memory_order_relaxed);
    if (n == 0) {
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
        cache[dev].store(n, std::memory_order_relaxed);
    }
    return n;
}

namespace {

constexpr int BM = 128, BN = 128, BK = 128;
constexpr int kThreads = 256;
// row tiles per group of the XCD-aware raster: an XCD's 32 concurrent tiles
// form a 4 x 8 block (measured against 2, 3, 8 and 16: 4 is fastest over the
// 7B shapes, most of all on the short-K GEMMs with large outputs)
constexpr int kGroupM = 4;
constexpr int kXcds = 8;

template <int FMT>
struct Fmt;

// Operand placement measured on gfx950 for v_mfma_scale_f32_32x32x64_f8f6f4:
// with E2M1 operands (4 VGPRs) lane l holds 32 consecutive K values of K-group
// l / 32; with E4M3 operands (8 VGPRs) the first 16 bytes of every lane belong
// to K-group 0 and the last 16 bytes to K-group 1, the two lane halves splitting
// each group.  In both cases lane half h supplies the scale of K-group h.
// chunk(ks, half, h) is the 16-byte chunk of the K-tile row that feeds VGPRs
// 4h..4h+3 of a lane in half `half` for K-substep ks (64 K values).
template <>
struct Fmt<kFmtFp4Block2D> {
    static constexpr int kRowBytes = BK / 2;      // 64 bytes of codes per row per K-tile
    static constexpr int kLaneBytes = 16;         // 32 E2M1 codes per lane per MFMA
    static constexpr int kCbsz = 4;               // E2M1
    static constexpr int kScaleRowShift = 5;      // one scale per 32-row block
    // 16-byte chunk swizzle of 64-byte LDS rows, conflict-free for the fragment
    // reads: rows r and r + 2 (read together with both lane halves) differ in
    // chunk bit 1, and rows r, r + 4, r + 8, r + 12 get four distinct chunks
    // (zero LdsBankConflict measured with rocprofv3)
    static __device__ __forceinline__ int swz(int r) { return ((r & 2) ^ (r >> 2)) & 3; }
    static __device__ __forceinline__ int chunk(int ks, int half, int) { return 2 * ks + half; }
};

template <>
struct Fmt<kFmtMxfp8> {
    static constexpr int kRowBytes = BK;          // 128 bytes per row per K-tile
    static constexpr int kLaneBytes = 32;         // 32 E4M3 codes per lane per MFMA
    static constexpr int kCbsz = 0;               // E4M3
    static constexpr int kScaleRowShift = 0;      // one scale per row and K-group
    // 16-byte chunk swizzle of 128-byte LDS rows: the four rows read together with
    // both lane halves map to distinct chunk pairs, and eight consecutive rows to
    // distinct chunks (zero LdsBankConflict measured with rocprofv3)
    static __device__ __forceinline__ int swz(int r)
    {
        return ((r & 2) << 1) | (((r ^ (r >> 3)) & 1) << 1) | ((r >> 2) & 1);
    }
    static __device__ __forceinline__ int chunk(int ks, int half, int h) { return 4 * ks + 2 * h + half; }
};

__device__ __forceinline__ void tile_coords_of(int64_t bid, int64_t tiles_m, int64_t tiles_n, int64_t &tm, int64_t &tn)
{
    // Hardware dispatch sends consecutive workgroups to consecutive XCDs; give
    // every XCD a contiguous range of the tile order instead.
    const int64_t nb = tiles_m * tiles_n;
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

__device__ __forceinline__ void tile_coords(int64_t tiles_m, int64_t tiles_n, int64_t &tm, int64_t &tn)
{
    tile_coords_of(blockIdx.x, tiles_m, tiles_n, tm, tn);
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
        // 1x32 FP4 scales are K-tile-major words (row offset 4 r, K-tile stride ld)
        sa_row[i] = g.a1d ? g.sa + ra * 4 : g.sa + (ra >> F::kScaleRowShift) * g.ldsa;
        sb_row[i] = g.b1d ? g.sb + rb * 4 : g.sb + (rb >> F::kScaleRowShift) * g.ldsb;
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
            swa[i] = *reinterpret_cast<const uint32_t *>(sa_row[i] + kt * (g.a1d ? g.ldsa : 4));
            swb[i] = *reinterpret_cast<const uint32_t *>(sb_row[i] + kt * (g.b1d ? g.ldsb : 4));
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
#pragma unroll
                for (int h = 0; h < F::kLaneBytes / 16; ++h) {
                    const int ch = F::chunk(ks, half, h);
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

// Large-tile FP4 kernel: 256 x 256 output tile, 4 waves of 128 x 128 (4 x 4
// MFMA tiles, 256 fp32 accumulators per lane held in AGPRs), one wave per
// SIMD.  Per K-tile of 128 each wave issues 32 MFMAs (about 1000 cycles at the
// MFMA rate) against 16 KB of LDS operand reads, half the LDS rate.
//
// Codes move global -> LDS with gfx950's global_load_lds_dwordx4 (each lane
// deposits 16 bytes at M0 + 16 * lane) and the block-scale words with
// global_load_lds_dword, through a ring of kStages LDS stages kept kStages - 1
// K-tiles ahead of the MFMAs.  The loads are issued from inline assembly so
// that the compiler does not serialize them against LDS reads it cannot prove
// disjoint; completion is tracked by hand with vmcnt: every iteration issues
// exactly kDmaPerTile loads per wave (past the last K-tile they re-read it into
// a stage that is never consumed).
constexpr int BM2 = 256, BN2 = 256;
constexpr int kStages = 4;
constexpr int kDmaPerTile = 9;      // per wave: 4 for A, 4 for B, 1 for the scale words
constexpr int kCodeBytes = BM2 * 64;                  // 16 KB per operand per stage

// Wave-uniform 64-bit value (moves it to SGPRs).
__device__ __forceinline__ uint64_t uniform64(uint64_t v)
{
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
    return ((uint64_t)hi << 32) | lo;
}

// global -> LDS, 16 bytes per lane at M0 + 16 * lane; address = sbase + voff
// with a wave-uniform base
__device__ __forceinline__ void lds_dma16(const uint8_t *sbase, uint32_t voff, uint32_t lds_addr)
{
    const uint64_t base = uniform64(reinterpret_cast<uint64_t>(sbase));
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2" ::"s"(lds_addr), "v"(voff), "s"(base)
                 : "memory");
}

// global -> LDS, 4 bytes per lane at M0 + 4 * lane, per-lane 64-bit address
__device__ __forceinline__ void lds_dma4(const uint8_t *src, uint32_t lds_addr)
{
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dword %1, off" ::"s"(lds_addr), "v"(src) : "memory");
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() { asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory"); }

__device__ __forceinline__ void block_barrier() { asm volatile("s_barrier" ::: "memory"); }

// Write a wave's 128 x 128 accumulator block (4 x 4 MFMA tiles) to C; CHECK
// masks rows >= M and columns >= N.  bf16 output rounds to nearest even.  The
// stores are non-temporal: every CU writes its tile at about the same time,
// and C is not read again by the kernel, so it should not displace the operand
// lines the next tiles reuse from L2.
template <bool BF16OUT, bool ACC, bool CHECK>
__device__ __forceinline__ void store_tile(v16f (&acc)[4][4], const GemmArgs &g, int64_t row0, int64_t col0)
{
    const int esize = BF16OUT ? 2 : 4;
    const int64_t ldc_bytes = g.ldc * esize;
    uint8_t *cbase = reinterpret_cast<uint8_t *>(g.c) + row0 * ldc_bytes + col0 * esize;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int roff = i * 32 + 8 * (r >> 2) + (r & 3);
            uint8_t *prow = cbase + roff * ldc_bytes;
            if (CHECK && row0 + roff >= g.M) continue;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (CHECK && col0 + j * 32 >= g.N) continue;
                float v = acc[i][j][r];
                if (BF16OUT) {
                    __bf16 *p = reinterpret_cast<__bf16 *>(prow + j * 32 * 2);
                    if (ACC) v += (float)*p;
                    __builtin_nontemporal_store((__bf16)v, p);
                } else {
                    float *p = reinterpret_cast<float *>(prow + j * 32 * 4);
                    if (ACC) v += *p;
                    __builtin_nontemporal_store(v, p);
                }
            }
            // keep the scheduler from hoisting all 256 accumulator reads at once
            // (they would not fit the VGPR file and would spill)
            __builtin_amdgcn_sched_barrier(0);
        }
}

// Persistent FP4 kernel (the large-tile design above).  The grid holds one
// workgroup per CU, a multiple of the 8 XCDs so that a workgroup keeps its
// XCD's share of the tile order; each walks the tiles u = blockIdx.x,
// blockIdx.x + gridDim.x, ... (ragged K: a serpentine over the tiles sorted by
// cost, TileSpace::step).  The K-tiles of all its tiles form one stream
// through the LDS ring: the loads of the next tile's first K-tiles are in
// flight while the current tile finishes and its accumulators are written, so
// no tile pays the pipeline fill.  Iteration s of the K loop: (A) the 16 MFMAs
// of K-substep 0 of step s while the fragments of substep 1 are read; wait for
// step s + 1 and barrier (every wave now holds step s in registers, so its
// stage is free); (B) the 16 MFMAs of substep 1 while the nine loads of step
// s + kStages go into that stage and the substep-0 fragments and scale words
// of step s + 1 are read.  A load cursor runs kStages steps ahead of the
// MFMAs and addresses each load from the tile it belongs to.  DMA issues and
// LDS reads sit between MFMAs (sched_barrier pins the order).
struct TileRef {
    const uint8_t *a, *sa, *b, *sb;
    uint8_t *c;
    int32_t M, N;          // valid rows of op(A) and op(B) (= rows and columns of C)
    int32_t m0, n0;        // tile origin in C
    uint32_t nk;           // K-tiles
};

template <int GMODE, bool BF16OUT>
struct TileSpace {
    const GemmArgs &g;
    const GroupedArgs &gr;
    int32_t tiles_m, tiles_n;
    const int32_t *pad_start, *tile_start, *seg_start;
    uint32_t total;        // tiles (ragged M: row tiles of all experts x column tiles)
    uint32_t per, rem, span;   // dense and ragged M: XCD share of the tile order; dense: group span

    // Ragged K: u is a position in the tile order sorted by cost, experts by
    // descending K-tile count (tile_start holds that expert order), each expert's
    // tiles in row-major order.  A workgroup takes positions G k + w for even k and
    // G k + G - 1 - w for odd k (G workgroups, w its index): the serpentine over a
    // descending list keeps the K-tiles per workgroup even when a few experts hold
    // most of the tokens.
    __device__ __forceinline__ int32_t expert_at(uint32_t u) const
    {
        return __builtin_amdgcn_readfirstlane(tile_start[u / (uint32_t)(tiles_m * tiles_n)]);
    }
    __device__ __forceinline__ uint32_t nk_of(uint32_t u) const
    {
        if (GMODE != 2) return (uint32_t)(g.K / BK);
        const int32_t e = expert_at(u);
        return (uint32_t)__builtin_amdgcn_readfirstlane((pad_start[e + 1] - pad_start[e]) / BK);
    }
    // the workgroup's next tile after u
    __device__ __forceinline__ uint32_t step(uint32_t u) const
    {
        if (GMODE != 2) return u + gridDim.x;
        const uint32_t k = u / gridDim.x + 1;
        return k * gridDim.x + ((k & 1) ? gridDim.x - 1 - blockIdx.x : blockIdx.x);
    }
    // u, or past the end if u has no K-tile (ragged K: every later position of
    // the cost order is empty too)
    __device__ __forceinline__ uint32_t valid_from(uint32_t u) const
    {
        if (GMODE == 2 && u < total && nk_of(u) == 0) return total;
        return u;
    }
    __device__ __forceinline__ TileRef ref(uint32_t u) const
    {
        TileRef t;
        const int esize = BF16OUT ? 2 : 4;
        t.a = g.a; t.sa = g.sa; t.b = g.b; t.sb = g.sb;
        t.c = reinterpret_cast<uint8_t *>(g.c);
        t.M = (int32_t)g.M; t.N = (int32_t)g.N; t.nk = (uint32_t)(g.K / BK);
        int32_t tm, tn;
        if (GMODE == 0) {
            // as tile_coords, in 32 bits
            const uint32_t xcd = u % kXcds, local = u / kXcds;
            const uint32_t tt = xcd * per + (xcd < rem ? xcd : rem) + local;
            const uint32_t grp = tt / span, first = grp * kGroupM;
            const uint32_t gsz = (uint32_t)tiles_m - first < (uint32_t)kGroupM ? (uint32_t)tiles_m - first : kGroupM;
            const uint32_t in = tt - grp * span;
            tm = (int32_t)(first + in % gsz);
            tn = (int32_t)(in / gsz);
        } else if (GMODE == 1) {
            // A multiple of 8 column tiles: the row-major order already gives each
            // XCD (u mod 8) one column band, i.e. one band of each expert's weight.
            // Otherwise each XCD takes a contiguous range of that order, so an
            // expert's weight bands are fetched into one L2 rather than all eight.
            uint32_t tt = u;
            if (tiles_n % kXcds != 0) {
                const uint32_t xcd = u % kXcds, local = u / kXcds;
                tt = xcd * per + (xcd < rem ? xcd : rem) + local;
            }
            const int32_t rt = (int32_t)(tt / (uint32_t)tiles_n);
            tn = (int32_t)tt - rt * tiles_n;
            const int e = __builtin_amdgcn_readfirstlane(seg_search(tile_start, gr.nseg, rt));
            tm = rt - __builtin_amdgcn_readfirstlane(tile_start[e]);
            const int64_t p_e = __builtin_amdgcn_readfirstlane(pad_start[e]);
            t.a += p_e * g.lda;
            t.sa += (p_e / 32) * g.ldsa;
            const int64_t o0 = __builtin_amdgcn_readfirstlane(seg_start[e]);
            const int64_t o1 = __builtin_amdgcn_readfirstlane(seg_start[e + 1]);
            t.M = (int32_t)(o1 - o0);
            t.c += o0 * g.ldc * esize;
            if (gr.b_group_rows) {
                t.b += (int64_t)e * gr.b_group_rows * g.ldb;
                t.sb += ((int64_t)e * gr.b_group_rows / 32) * g.ldsb;
            } else {
                t.b += (int64_t)e * gr.b_group_k / 2;
                t.sb += (int64_t)e * gr.b_group_k / 32;
            }
        } else {
            const uint32_t per_e = (uint32_t)(tiles_m * tiles_n);
            const int32_t e = expert_at(u);
            const int32_t rest = (int32_t)(u - (u / per_e) * per_e);
            tm = rest / tiles_n;
            tn = rest - tm * tiles_n;
            const int64_t p_e = __builtin_amdgcn_readfirstlane(pad_start[e]);
            t.a += p_e / 2; t.sa += p_e / 32;
            t.b += p_e / 2; t.sb += p_e / 32;
            t.nk = (uint32_t)((__builtin_amdgcn_readfirstlane(pad_start[e + 1]) - p_e) / BK);
            t.c += (int64_t)e * g.M * g.ldc * esize;
        }
        t.m0 = tm * BM2;
        t.n0 = tn * BN2;
        return t;
    }
};

// Write a wave's 128 x 128 accumulator block at cbase (wave-uniform: the
// block's first element) with 32-bit offsets; CHECK masks rows >= rows_left and
// columns >= cols_left.  bf16 output rounds to nearest even.
//
// Inside the persistent tile loop the row offsets would otherwise be hoisted
// out of the loop (they depend only on ldc) and all 256 accumulators copied to
// VGPRs at once; the opaque row stride and the per-element AGPR reads keep the
// epilogue streaming through a few registers.  Non-temporal stores, as in
// store_tile.
template <bool BF16OUT, bool ACC, bool CHECK>
__device__ __forceinline__ void store_block(v16f (&acc)[4][4], uint8_t *cbase, uint32_t ldc_bytes, int rows_left,
                                            int cols_left)
{
    const int lane = threadIdx.x & 63;
    const int col = lane & 31, r4 = 4 * (lane >> 5);
    const int esize = BF16OUT ? 2 : 4;
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" : "+s"(ldc_bytes));   // and the last MFMA results settle
    uint32_t rb = (uint32_t)r4 * ldc_bytes + (uint32_t)(col * esize);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int roff = i * 32 + 8 * (r >> 2) + r4 + (r & 3);
            if (r > 0 || i > 0) rb += (uint32_t)((r & 3) ? 1 : 5) * ldc_bytes;   // next row of this lane
            if (CHECK && roff >= rows_left) continue;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (CHECK && j * 32 + col >= cols_left) continue;
                float v;
                asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(v) : "a"(acc[i][j][r]));
                uint8_t *p = cbase + rb + j * 32 * esize;
                if (BF16OUT) {
                    if (ACC) v += (float)*reinterpret_cast<__bf16 *>(p);
                    __builtin_nontemporal_store((__bf16)v, reinterpret_cast<__bf16 *>(p));
                } else {
                    if (ACC) v += *reinterpret_cast<float *>(p);
                    __builtin_nontemporal_store(v, reinterpret_cast<float *>(p));
                }
            }
            __builtin_amdgcn_sched_barrier(0);
        }
}

// Interleaved columns (the persistent kernels with bf16 output): MFMA tiles 2p
// and 2p + 1 of a wave take B rows 64 p + 2 l and 64 p + 2 l + 1 in lane l, so
// a lane holds two neighbouring output columns of every row it has, and 32
// lanes write a row's 64 columns (128 bytes of bf16) with one store
// instruction.  Whole-line stores: a CU writes about three times faster than
// with the two-byte, half-line stores of the plain column order.
//
// Write a wave's 128 x 128 accumulator block in that layout at cbase (the
// block's first element) as bf16, rounded to nearest even; CHECK masks rows >=
// rows_left and columns >= cols_left.  PAIR: C allows the 4-byte pair stores
// (start and row pitch 4-byte aligned); otherwise each element is stored on
// its own.  Non-temporal stores, as in store_tile.
template <bool ACC, bool CHECK, bool PAIR>
__device__ __forceinline__ void store_block_pairs(v16f (&acc)[4][4], uint8_t *cbase, uint32_t ldc_bytes,
                                                  int rows_left, int cols_left)
{
    typedef __bf16 bf2_t __attribute__((ext_vector_type(2)));
    const int lane = threadIdx.x & 63;
    const int col = 2 * (lane & 31), r4 = 4 * (lane >> 5);
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" : "+s"(ldc_bytes));   // and the last MFMA results settle
    uint32_t rb = (uint32_t)r4 * ldc_bytes + (uint32_t)(col * 2);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int roff = i * 32 + 8 * (r >> 2) + r4 + (r & 3);
            if (r > 0 || i > 0) rb += (uint32_t)((r & 3) ? 1 : 5) * ldc_bytes;   // next row of this lane
            if (CHECK && roff >= rows_left) continue;
#pragma unroll
            for (int jp = 0; jp < 2; ++jp) {
                const int c = 64 * jp + col;            // columns c, c + 1 of the block
                if (CHECK && c >= cols_left) continue;
                float v0, v1;
                asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(v0) : "a"(acc[i][2 * jp][r]));
                asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(v1) : "a"(acc[i][2 * jp + 1][r]));
                uint8_t *p = cbase + rb + 64 * jp * 2;
                const bool both = !CHECK || c + 1 < cols_left;
                if (PAIR && both) {
                    if (ACC) {
                        const bf2_t o = *reinterpret_cast<const bf2_t *>(p);
                        v0 += (float)o.x;
                        v1 += (float)o.y;
                    }
                    const bf2_t b = {(__bf16)v0, (__bf16)v1};
                    __builtin_nontemporal_store(__builtin_bit_cast(uint32_t, b), reinterpret_cast<uint32_t *>(p));
                } else {
                    __bf16 *q = reinterpret_cast<__bf16 *>(p);
                    if (ACC) v0 += (float)q[0];
                    __builtin_nontemporal_store((__bf16)v0, q);
                    if (both) {
                        if (ACC) v1 += (float)q[1];
                        __builtin_nontemporal_store((__bf16)v1, q + 1);
                    }
                }
            }
            __builtin_amdgcn_sched_barrier(0);
        }
}

// Row of B (within a 256-row tile) that feeds MFMA row slot t = 128 h + 32 j + l
// of the interleaved-column layout: 128 h + 64 (j / 2) + 2 l + j % 2.
__device__ __forceinline__ int interleaved_row(int t)
{
    const int j = (t >> 5) & 3, l = t & 31;
    return (t & ~127) + 64 * (j >> 1) + 2 * l + (j & 1);
}

// Quantize a wave's 128 x 128 accumulator block into 2D-block FP4 with round to
// nearest (the quantizer's scale rule and codec, applied to the float32
// result): each 32 x 32 MFMA tile is exactly one block.
//   1. block maxima: each lane's maximum over the 16 values it holds of every
//      tile, then the 16 maxima reduced across the wave together (quad and row
//      permutes, then two lane exchanges), so the reductions overlap; with
//      CHECK, values outside rows_left x cols_left count as 0 (padding gets
//      zero codes, an all-zero block the byte 0x00);
//   2. per 32-row strip i, per tile j:
//      codes_t: a lane holds one column's rows 8q + 4h + 0..3 (h = lane / 32),
//               two bytes per q; the halves h swap one word so that each lane
//               stores 8 consecutive bytes of its column's 16-byte run;
//      codes:   neighbouring columns meet through a quad permute; the even lane
//               packs rows q = 0, 1 and the odd lane rows q = 2, 3, one byte per
//               row, into the wave's LDS strip (32 rows x 64 bytes);
//      scales:  one byte per tile in each grid;
//      then the strip leaves as 16-byte row segments.
// Only the written extent of the layout is touched: codes rows < M, bytes below
// roundup(N, 128) / 2; codes_t rows < N, bytes below roundup(M, 128) / 2.
//
// Stochastic rounding (SR): element (r, c) of the M x N result takes the draw of
// storage index r N + c of a row-major M x N tensor (half (idx & 1) of word
// (idx & 7) >> 1 of the Philox block for counter (idx >> 3, offset)), the draw
// q2d_quantize would give it, and is converted on its own with seed r16 << 16
// (first element of a pair) or r16 << 15 (second).  N is a multiple of 8, so a
// Philox block covers 8 consecutive columns of one row: the wave computes each
// of a tile's 128 blocks once (two per lane) into its LDS table, and every lane
// reads back the 16-bit draws of the 16 elements it holds.
// f(std::integral_constant<int, 0>) ... f(std::integral_constant<int, N - 1>), in order
template <typename F, int... Is>
__device__ __forceinline__ void unroll_seq(F &&f, std::integer_sequence<int, Is...>)
{
    (f(std::integral_constant<int, Is>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void unroll(F &&f)
{
    unroll_seq(f, std::make_integer_sequence<int, N>{});
}

constexpr int kQPitch = 80;                     // LDS strip row pitch (64 bytes + pad)
constexpr int kQStrip = 32 * kQPitch;           // per wave
constexpr int kPRow = 80;                       // Philox table row: four 16-byte blocks + pad
constexpr int kPTab = 32 * kPRow;               // per wave

typedef float f32x2 __attribute__((ext_vector_type(2)));

// SR conversion of a pair into byte `sel` of a zero word (only the nibble the
// caller keeps is defined)
__device__ __forceinline__ uint32_t sr_cvt(int sel, f32x2 v, uint32_t seed, float scale)
{
    switch (sel) {
    case 0: return __builtin_amdgcn_cvt_scalef32_sr_pk_fp4_f32(0u, v, seed, scale, 0);
    case 1: return __builtin_amdgcn_cvt_scalef32_sr_pk_fp4_f32(0u, v, seed, scale, 1);
    case 2: return __builtin_amdgcn_cvt_scalef32_sr_pk_fp4_f32(0u, v, seed, scale, 2);
    default: return __builtin_amdgcn_cvt_scalef32_sr_pk_fp4_f32(0u, v, seed, scale, 3);
    }
}

// byte `sel` of `old` gets the SR codes of the pair (a, b): a with seed ra
// (= r16 << 16) in the low nibble, b with seed rb >> 1 (= r16 << 15) in the high
__device__ __forceinline__ uint32_t sr_pair_into(uint32_t old, int sel, float a, float b, uint32_t ra, uint32_t rb,
                                                 float scale)
{
    const f32x2 v = {a, b};
    const uint32_t lo = sr_cvt(sel, v, ra, scale), hi = sr_cvt(sel, v, rb >> 1, scale);
    return old | (lo & (0x0Fu << (8 * sel))) | (hi & (0xF0u << (8 * sel)));
}

template <bool CHECK, bool SR>
__device__ __forceinline__ void store_qblock(v16f (&acc)[4][4], const GemmArgs &g, uint8_t *strip, uint8_t *ptab,
                                             int r0, int c0, int rows_left, int cols_left)
{
    const int lane = threadIdx.x & 63;
    const int col = lane & 31, h = lane >> 5, odd = lane & 1;
    const int padm = (int)((g.M + 127) / 128 * 128), padn = (int)((g.N + 127) / 128 * 128);
    int dummy = 0;
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" : "+s"(dummy));   // the last MFMA results settle
    auto value = [&](int i, int j, int r) __attribute__((always_inline)) -> float {
        float v;
        asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(v) : "a"(acc[i][j][r]));
        if (CHECK) {
            const int rr = 32 * i + 8 * (r >> 2) + 4 * h + (r & 3);
            if (rr >= rows_left || 32 * j + col >= cols_left) v = 0.0f;
        }
        return v;
    };
    uint32_t am[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            uint32_t m = 0;
#pragma unroll
            for (int r = 0; r < 16; ++r) m = max(m, f_bits(value(i, j, r)) & 0x7FFFFFFFu);
            am[i][j] = m;
        }
    // quad_perm [1,0,3,2], quad_perm [2,3,0,1], row_half_mirror, row_mirror
    auto perm_max = [&](auto ctrl) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                am[i][j] = max(am[i][j], (uint32_t)__builtin_amdgcn_update_dpp((int)am[i][j], (int)am[i][j],
                                                                               decltype(ctrl)::value, 0xF, 0xF, false));
    };
    perm_max(std::integral_constant<int, 0xB1>{});
    perm_max(std::integral_constant<int, 0x4E>{});
    perm_max(std::integral_constant<int, 0x141>{});
    perm_max(std::integral_constant<int, 0x140>{});
#pragma unroll
    for (int m = 16; m < 64; m <<= 1)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) am[i][j] = max(am[i][j], (uint32_t)__shfl_xor((int)am[i][j], m));

    // compile-time tile indices: a runtime loop here would put acc in scratch memory
    unroll<4>([&](auto ic) __attribute__((always_inline)) {
        constexpr int i = decltype(ic)::value;
        const int tr = r0 + 32 * i;                     // strip origin row in C
        unroll<4>([&](auto jc) __attribute__((always_inline)) {
            constexpr int j = decltype(jc)::value;
            const int tc = c0 + 32 * j;                 // tile origin column
            const bool finite = am[i][j] < 0x7F800000u;
            const int e = fp4_block_exponent(am[i][j]);
            const float scale = bits_f((uint32_t)(127 + e) << 23);
            float v[16];
#pragma unroll
            for (int r = 0; r < 16; ++r) v[r] = value(i, j, r);
            // SR draws of the lane's elements (rows 8 (r / 4) + 4 h + r % 4, column col),
            // packed two to a register: rw[k] = draw(2k) | draw(2k + 1) << 16
            uint32_t rw[8];
            if constexpr (SR) {
                // the previous tile's reads of the table come first (in program order)
                __builtin_amdgcn_wave_barrier();
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int t = 0; t < 2; ++t) {
                    const int b = lane + 64 * t, brow = b >> 2, bcg = b & 3;
                    const uint64_t idx = (uint64_t)(uint32_t)(tr + brow) * (uint64_t)g.N + (uint64_t)(tc + 8 * bcg);
                    uint32_t w[4];
                    philox4x32_10((uint32_t)(idx >> 3), (uint32_t)(idx >> 35), (uint32_t)g.offset,
                                  (uint32_t)(g.offset >> 32), (uint32_t)g.seed, (uint32_t)(g.seed >> 32), w);
                    *reinterpret_cast<uint4 *>(ptab + brow * kPRow + 16 * bcg) = make_uint4(w[0], w[1], w[2], w[3]);
                }
                // LDS accesses of one wave complete in order: the reads below see the table.
                // All 16 reads issue back to back, so their latency is paid once.
                __builtin_amdgcn_wave_barrier();
                __builtin_amdgcn_sched_barrier(0);
                const uint8_t *cp = ptab + 16 * (col >> 3) + 4 * ((col & 7) >> 1) + 2 * (col & 1);
#pragma unroll
                for (int k = 0; k < 8; ++k) {
                    const int rl = 8 * (k >> 1) + 4 * h + 2 * (k & 1);        // row of element 2k
                    const uint32_t d0 = *reinterpret_cast<const uint16_t *>(cp + rl * kPRow);
                    const uint32_t d1 = *reinterpret_cast<const uint16_t *>(cp + (rl + 1) * kPRow);
                    rw[k] = d0 | (d1 << 16);
                }
            }
            // the draw of element r, shifted to bits 31..16
            auto rr = [&](int r) __attribute__((always_inline)) -> uint32_t {
                return (r & 1) ? (rw[r >> 1] & 0xFFFF0000u) : (rw[r >> 1] << 16);
            };
            // column-packed: word q/2 byte 2 (q % 2) + k holds rows (8q + 4h + 2k, +1)
            uint32_t w0 = 0, w1 = 0;
            if constexpr (SR) {
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    w0 = sr_pair_into(w0, k, v[2 * k], v[2 * k + 1], rr(2 * k), rr(2 * k + 1), scale);
                    w1 = sr_pair_into(w1, k, v[8 + 2 * k], v[9 + 2 * k], rr(8 + 2 * k), rr(9 + 2 * k), scale);
                }
            } else {
                w0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w0, v[0], v[1], scale, 0);
                w0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w0, v[2], v[3], scale, 1);
                w0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w0, v[4], v[5], scale, 2);
                w0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w0, v[6], v[7], scale, 3);
                w1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w1, v[8], v[9], scale, 0);
                w1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w1, v[10], v[11], scale, 1);
                w1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w1, v[12], v[13], scale, 2);
                w1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w1, v[14], v[15], scale, 3);
            }
            if (!finite) w0 = w1 = 0;
            // half 0 stores bytes 0..7 of the run (q = 0, 1 of both halves), half 1
            // bytes 8..15 (q = 2, 3)
            const uint32_t mine = h ? w1 : w0;
            const uint32_t other = (uint32_t)__shfl_xor((int)(h ? w0 : w1), 32);
            const uint32_t first = h ? other : mine, second = h ? mine : other;
            const uint2 run = make_uint2((first & 0xFFFFu) | (second << 16), (first >> 16) | (second & 0xFFFF0000u));
            if (tc + col < g.N && tr < padm)
                *reinterpret_cast<uint2 *>(g.qct + (int64_t)(tc + col) * g.ldqct + tr / 2 + 8 * h) = run;
            // row-packed: both layouts hold the same code for an element (one block
            // scale; under SR the element's own draw either way), so the row bytes
            // come from the column words.  Nibble r & 7 of w0 (w1) is the code of
            // v[r] for r < 8 (r >= 8).  Of a column pair, the even lane packs rows
            // v[0..7] (its own column low, the neighbour's high), the odd lane rows
            // v[8..15] (the neighbour's low, its own high): one word from the
            // neighbour, then the two words' nibbles zipped into bytes.
            const uint32_t send = odd ? w0 : w1;
            const uint32_t recv = (uint32_t)__builtin_amdgcn_update_dpp((int)send, (int)send, 0xB1, 0xF, 0xF, false);
            const uint32_t lo = odd ? recv : w0, hi = odd ? w1 : recv;
            const uint32_t ev = (lo & 0x0F0F0F0Fu) | ((hi << 4) & 0xF0F0F0F0u);     // byte k: row 2k
            const uint32_t od = ((lo >> 4) & 0x0F0F0F0Fu) | (hi & 0xF0F0F0F0u);     // byte k: row 2k + 1
            uint32_t rowb[2] = {__builtin_amdgcn_perm(od, ev, 0x05010400u), __builtin_amdgcn_perm(od, ev, 0x07030602u)};
            if (!finite) rowb[0] = rowb[1] = 0;
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const int rk = odd ? 8 + k : k;
                const int rl = 8 * (rk >> 2) + 4 * h + (rk & 3);
                strip[rl * kQPitch + 16 * j + (col >> 1)] = (uint8_t)(rowb[k >> 2] >> (8 * (k & 3)));
            }
            if (lane == 0) {
                const uint8_t sbyte = finite ? (uint8_t)(e + 127) : (uint8_t)0xFF;
                if (tr < g.M && tc < padn) g.qs[(int64_t)(tr / 32) * g.ldqs + tc / 32] = sbyte;
                if (tc < g.N && tr < padm) g.qst[(int64_t)(tc / 32) * g.ldqst + tr / 32] = sbyte;
            }
        });
        // the strip's 32 rows x 64 bytes as 16-byte row segments (LDS accesses of
        // one wave complete in order, so the reads see the writes above)
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            const int rl = (lane >> 2) + 16 * k, chunk = lane & 3;
            const uint4 w = *reinterpret_cast<const uint4 *>(strip + rl * kQPitch + 16 * chunk);
            if (tr + rl < g.M && c0 + 32 * chunk < padn)
                *reinterpret_cast<uint4 *>(g.qc + (int64_t)(tr + rl) * g.ldqc + c0 / 2 + 16 * chunk) = w;
        }
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_sched_barrier(0);
    });
}

// SM: bit 0 -- A has 1x32 blocks (one scale per row and K-group: activations
// in the forward GEMM), bit 1 -- B has them (activations in the weight-gradient
// GEMM).  Such an operand's per-row scale words follow the 2D words in each
// stage (1 KB per operand, one load per wave) and every lane reads its own
// row's word instead of the block row's.
template <bool BF16OUT, bool ACC, int GMODE, int SM, bool QOUT = false, bool QSR = false>
__global__ __launch_bounds__(kThreads, 1) void gemm_fp4_persistent_kernel(GemmArgs g, int tiles_m, int tiles_n,
                                                                          const GroupedArgs gr)
{
    using F = Fmt<kFmtFp4Block2D>;
    constexpr int RB = F::kRowBytes;                // 64
    constexpr bool A1 = (SM & 1) != 0, B1 = (SM & 2) != 0;
    constexpr int kDma = kDmaPerTile + A1 + B1;     // 9 .. 11
    constexpr int kWordsA1 = 2 * kCodeBytes + 1024;             // after 2 x codes + 1 KB of 2D scale words: per-row A scale words
    constexpr int kWordsB1 = kWordsA1 + (A1 ? 1024 : 0);       // per-row B scale words
    constexpr int kStageBytes = kWordsB1 + (B1 ? 1024 : 0);
    // interleaved output columns with pair stores for bf16 outputs (3-7 % faster
    // at K <= 4096, where the epilogue weighs most); float32 rows already leave
    // as whole lines, and pairs of them measured slower
    constexpr bool PERM = BF16OUT && !QOUT;
    __shared__ __attribute__((aligned(1024))) uint8_t smem[kStages * kStageBytes];
    __shared__ int32_t pad_start[GMODE == 0 ? 1 : kMaxSegs + 1];
    __shared__ int32_t tile_start[GMODE != 0 ? kMaxSegs + 1 : 1];     // ragged K: the expert cost order
    __shared__ int32_t seg_start[GMODE == 0 ? 1 : kMaxSegs + 1];     // sanitized segment offsets
    __shared__ __attribute__((aligned(16))) uint8_t qstrip[QOUT ? 4 * kQStrip : 16];
    __shared__ __attribute__((aligned(16))) uint8_t ptab[QSR ? 4 * kPTab : 16];

    uint32_t total = (uint32_t)(tiles_m * tiles_n);
    if (GMODE != 0) {
        if ((threadIdx.x >> 6) == 0) {
            wave_offsets(gr.nseg, gr.seg_offsets, gr.total_rows, seg_start);
            __builtin_amdgcn_wave_barrier();
            const int32_t *off = seg_start;
            wave_prefix(gr.nseg, [&](int i) { return (off[i + 1] - off[i] + 127) / 128 * 128; }, pad_start);
            if (GMODE == 1)
                wave_prefix(gr.nseg, [&](int i) { return (off[i + 1] - off[i] + BM2 - 1) / BM2; }, tile_start);
        }
        __syncthreads();
        if (GMODE == 2) {
            // experts by descending K-tile count, ties by index: rank -> expert
            for (int e = threadIdx.x; e < gr.nseg; e += blockDim.x) {
                const int32_t ne = pad_start[e + 1] - pad_start[e];
                int rank = 0;
                for (int f = 0; f < gr.nseg; ++f) {
                    const int32_t nf = pad_start[f + 1] - pad_start[f];
                    rank += (nf > ne || (nf == ne && f < e)) ? 1 : 0;
                }
                tile_start[rank] = e;
            }
            __syncthreads();
        }
        if (GMODE == 1) total = (uint32_t)__builtin_amdgcn_readfirstlane(tile_start[gr.nseg]) * (uint32_t)tiles_n;
        else total = (uint32_t)(gr.nseg * tiles_m * tiles_n);
    }
    const uint32_t nb = (uint32_t)(tiles_m * tiles_n);
    const uint32_t ordered = GMODE == 1 ? total : nb;      // tiles of the XCD-contiguous order
    const TileSpace<GMODE, BF16OUT> ts{g, gr, tiles_m, tiles_n, pad_start, tile_start, seg_start, total,
                                       ordered / kXcds, ordered % kXcds, (uint32_t)(kGroupM * tiles_n)};

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1;
    const int half = lane >> 5;
    const int esize = BF16OUT ? 2 : 4;
    const uint32_t ldc_bytes = (uint32_t)(g.ldc * esize);
    // pair stores need C and its row pitch aligned to two elements
    const bool pair_ok = ((reinterpret_cast<uintptr_t>(g.c) | (uintptr_t)ldc_bytes) & (uintptr_t)(2 * esize - 1)) == 0;

    v16f acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    auto store = [&](const TileRef &t) __attribute__((always_inline)) {
        const int r0 = t.m0 + wm * 128, c0 = t.n0 + wn * 128;
        if constexpr (QOUT) {
            uint8_t *strip = qstrip + wave * kQStrip;
            uint8_t *tab = ptab + (QSR ? wave * kPTab : 0);
            if (t.m0 + BM2 <= t.M && t.n0 + BN2 <= t.N)
                store_qblock<false, QSR>(acc, g, strip, tab, r0, c0, 128, 128);
            else
                store_qblock<true, QSR>(acc, g, strip, tab, r0, c0, t.M - r0, t.N - c0);
        } else {
            uint8_t *cb = t.c + (int64_t)r0 * ldc_bytes + (int64_t)c0 * esize;
            const bool full = t.m0 + BM2 <= t.M && t.n0 + BN2 <= t.N;
            if constexpr (PERM) {
                if (full) {
                    if (pair_ok) store_block_pairs<ACC, false, true>(acc, cb, ldc_bytes, 128, 128);
                    else store_block_pairs<ACC, false, false>(acc, cb, ldc_bytes, 128, 128);
                } else {
                    if (pair_ok) store_block_pairs<ACC, true, true>(acc, cb, ldc_bytes, t.M - r0, t.N - c0);
                    else store_block_pairs<ACC, true, false>(acc, cb, ldc_bytes, t.M - r0, t.N - c0);
                }
            } else if (full) {
                store_block<BF16OUT, ACC, false>(acc, cb, ldc_bytes, 128, 128);
            } else {
                store_block<BF16OUT, ACC, true>(acc, cb, ldc_bytes, t.M - r0, t.N - c0);
            }
        }
    };

    // ragged K: experts without rows give zero tiles (unchanged when accumulating)
    if (GMODE == 2 && !ACC) {
        for (uint32_t u = blockIdx.x; u < total; u += gridDim.x)
            if (ts.nk_of(u) == 0) store(ts.ref(u));
    }

    uint32_t cu = ts.valid_from(blockIdx.x);        // tile being computed
    if (cu >= total) return;

    // per-lane load geometry: DMA j of this wave fills bytes [(4j + wave) * 1024,
    // +1024) of an operand stage: rows 16 (4j + wave) + lane / 4, physical chunk
    // lane % 4 (XOR-swizzled)
    int row[4], c16[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        row[j] = 16 * (4 * j + wave) + (lane >> 2);
        c16[j] = ((lane & 3) ^ F::swz(row[j])) * 16;
    }
    const int sq = lane & 7;                        // scale words: 0-3 A block rows, 4-7 B block rows
    const int srow = sq < 4 ? wm * 128 + sq * 32 : wn * 128 + (sq - 4) * 32;
    const uint32_t lds0 = (uint32_t)(uintptr_t)&smem[0];

    // load cursor: tile lu (lt), K-tile lk; past the last tile it stays on the
    // last K-tile, whose loads then fill a stage that is never read.  The
    // per-lane byte offsets of the tile's rows (and the scale-word source) are
    // set when the cursor enters a tile.
    uint32_t lu = cu, lk = 0;
    TileRef lt = ts.ref(cu);
    TileRef ct = lt;
    uint32_t offA[4], offB[4];
    const uint8_t *lsrc, *lsrcA1 = nullptr, *lsrcB1 = nullptr;
    auto enter = [&]() __attribute__((always_inline)) {
        // 1x32 scales are K-tile-major words: row r of K-tile k at k * ld + 4 r
        if (A1) {
            int r = lt.m0 + 64 * wave + lane; r = r < lt.M ? r : lt.M - 1;
            lsrcA1 = lt.sa + 4 * r;
        }
        if (B1) {
            int r = lt.n0 + (PERM ? interleaved_row(64 * wave + lane) : 64 * wave + lane);
            r = r < lt.N ? r : lt.N - 1;
            lsrcB1 = lt.sb + 4 * r;
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            int ra = lt.m0 + row[j]; ra = ra < lt.M ? ra : lt.M - 1;
            int rb = lt.n0 + (PERM ? interleaved_row(row[j]) : row[j]); rb = rb < lt.N ? rb : lt.N - 1;
            offA[j] = (uint32_t)ra * (uint32_t)g.lda + c16[j];
            offB[j] = (uint32_t)rb * (uint32_t)g.ldb + c16[j];
        }
        const bool isA = sq < 4;
        const int lim = isA ? lt.M : lt.N;
        int r = (isA ? lt.m0 : lt.n0) + srow; r = r < lim ? r : lim - 1;
        lsrc = (isA ? lt.sa : lt.sb) + (uint32_t)(r >> 5) * (uint32_t)(isA ? g.ldsa : g.ldsb);
        // a 1D operand has no block-row words: its lanes read the start of its own
        // word buffer instead (word k of K-tile 0 .. lies inside it for every
        // K-tile k), and the bytes are never used
        if ((A1 && isA) || (B1 && !isA)) lsrc = isA ? lt.sa : lt.sb;
    };
    enter();
    auto advance = [&]() __attribute__((always_inline)) {
        if (++lk < lt.nk) return;
        const uint32_t v = ts.valid_from(ts.step(lu));
        if (v < total) { lu = v; lt = ts.ref(v); lk = 0; enter(); }
        else lk = lt.nk - 1;
    };
    // load k (0 .. kDma-1) of the cursor's K-tile into ring stage `slot`:
    //   k = 0..3 A rows 16 (4k + wave) + ..., 4..7 B likewise, 8 the 2D scale
    //   words, then the per-row words of a 1D A (rows 64 wave + lane) and B
    auto load = [&](uint32_t slot, int k) __attribute__((always_inline)) {
        const uint32_t stage = lds0 + (slot % kStages) * kStageBytes;
        if (k < 4)
            lds_dma16(lt.a + lk * RB, offA[k], stage + (4 * k + wave) * 1024);
        else if (k < 8)
            lds_dma16(lt.b + lk * RB, offB[k - 4], stage + kCodeBytes + (4 * (k - 4) + wave) * 1024);
        else if (k == 8)
            lds_dma4(lsrc + lk * 4, stage + 2 * kCodeBytes + wave * 256);
        else if (k == 9 && A1)
            lds_dma4(lsrcA1 + lk * (uint32_t)g.ldsa, stage + kWordsA1 + wave * 256);
        else
            lds_dma4(lsrcB1 + lk * (uint32_t)g.ldsb, stage + kWordsB1 + wave * 256);
    };
    // scale words of the K-tile in stage `st`: the 2D block-row words (the
    // same for every lane) or a 1D operand's own row words
    auto read_scales = [&](const uint8_t *st, uint32_t (&dA)[4], uint32_t (&dB)[4]) __attribute__((always_inline)) {
        const uint4 wA = *reinterpret_cast<const uint4 *>(st + 2 * kCodeBytes + wave * 256);
        const uint4 wB = *reinterpret_cast<const uint4 *>(st + 2 * kCodeBytes + wave * 256 + 16);
        dA[0] = wA.x; dA[1] = wA.y; dA[2] = wA.z; dA[3] = wA.w;
        dB[0] = wB.x; dB[1] = wB.y; dB[2] = wB.z; dB[3] = wB.w;
        if (A1) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
                dA[i] = *reinterpret_cast<const uint32_t *>(st + kWordsA1 + (wm * 128 + i * 32 + (lane & 31)) * 4);
        }
        if (B1) {
#pragma unroll
            for (int j = 0; j < 4; ++j)
                dB[j] = *reinterpret_cast<const uint32_t *>(st + kWordsB1 + (wn * 128 + j * 32 + (lane & 31)) * 4);
        }
    };

    const int sw = F::swz(lane & 31);
    const int rd_a = (wm * 128 + (lane & 31)) * RB;
    const int rd_b = kCodeBytes + (wn * 128 + (lane & 31)) * RB;
    uint4 fa0[4], fb0[4], fa1[4], fb1[4];
    uint32_t scA[4], scB[4], nA[4], nB[4];

    // the B block-row word of MFMA tile j: with interleaved columns, lanes 0..15
    // (rows 2 l + j % 2 < 32 of the tile pair) take block row 2 (j / 2), lanes
    // 16..31 the next one; 1D words already belong to the lane's own row
    auto bword = [&](const uint32_t (&w)[4], int j) __attribute__((always_inline)) -> uint32_t {
        if (!PERM || B1) return w[j];
        return (lane & 16) ? w[2 * (j >> 1) + 1] : w[2 * (j >> 1)];
    };

#define Q2D_MFMA(fa, fb, scA_, scB_, ks, i, j)                                                          \
    do {                                                                                             \
        const v8i av_ = {(int)fa[i].x, (int)fa[i].y, (int)fa[i].z, (int)fa[i].w, 0, 0, 0, 0};       \
        const v8i bv_ = {(int)fb[j].x, (int)fb[j].y, (int)fb[j].z, (int)fb[j].w, 0, 0, 0, 0};       \
        const int sa_ = (int)((scA_[i] >> (8 * (2 * (ks) + half))) & 0xFFu);                         \
        const int sb_ = (int)((bword(scB_, j) >> (8 * (2 * (ks) + half))) & 0xFFu);                  \
        acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av_, bv_, acc[i][j], F::kCbsz,   \
                                                                    F::kCbsz, 0, sa_, 0, sb_);       \
    } while (0)
#define Q2D_READ(dstA, dstB, st, ks, i)                                                              \
    do {                                                                                             \
        const int cofs_ = ((2 * (ks) + half) ^ sw) * 16;                                             \
        dstA[i] = *reinterpret_cast<const uint4 *>((st) + rd_a + (i) * 32 * RB + cofs_);            \
        dstB[i] = *reinterpret_cast<const uint4 *>((st) + rd_b + (i) * 32 * RB + cofs_);            \
    } while (0)

    // prologue: K-steps 0 .. kStages-1 (the cursor stays on step kStages-1)
    for (uint32_t s = 0; s < kStages; ++s) {
        if (s > 0) advance();
        for (int k = 0; k < kDma; ++k) load(s, k);
    }
    wait_vmcnt<(kStages - 1) * kDma>();
    block_barrier();
    read_scales(smem, scA, scB);
#pragma unroll
    for (int i = 0; i < 4; ++i) Q2D_READ(fa0, fb0, smem, 0, i);

    uint32_t s = 0;                                 // ring step
    for (;;) {
    for (uint32_t ck = 0; ck < ct.nk; ++ck, ++s) {
        // the cursor moves to step s + kStages first: its (rare) switch to the
        // next tile then precedes, rather than splits, the pipelined body
        advance();
        const uint8_t *st = smem + (s % kStages) * kStageBytes;
        // ---- phase A: substep 0 MFMAs; substep 1 reads
#pragma unroll
        for (int i = 0; i < 4; ++i) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                Q2D_MFMA(fa0, fb0, scA, scB, 0, i, j);
                __builtin_amdgcn_sched_barrier(0);
                if (j == 1) {
                    Q2D_READ(fa1, fb1, st, 1, i);
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
        }
        __builtin_amdgcn_s_waitcnt(0xC07F);       // lgkmcnt(0)
        wait_vmcnt<(kStages - 2) * kDma>();
        block_barrier();
        // ---- phase B: substep 1 MFMAs; the nine loads of step s + kStages into
        // the stage of step s; substep 0 reads of step s + 1
        const uint8_t *sn = smem + ((s + 1) % kStages) * kStageBytes;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                Q2D_MFMA(fa1, fb1, scA, scB, 1, i, j);
                __builtin_amdgcn_sched_barrier(0);
                // loads at q = 0, 2, 4, 6, 8, 10, 11, ...; fragment reads at
                // q = 1, 3, 5, 7 (past the last step they are unused); scale
                // words at q = 9
                const int q = 4 * i + j;           // 0..15
                if (q < 8 && (q & 1)) {
                    Q2D_READ(fa0, fb0, sn, 0, q >> 1);
                } else if (q == 9) {
                    read_scales(sn, nA, nB);
                } else if (q < kDma + 5) {
                    load(s + kStages, q < 9 ? q >> 1 : q - 5);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) { scA[i] = nA[i]; scB[i] = nB[i]; }
    }
        // ---- the tile is complete: write it and go on with the next one, whose
        // first K-tiles are already in the ring and first fragments in registers
        store(ct);
        cu = ts.valid_from(ts.step(cu));
        if (cu >= total) break;
        ct = ts.ref(cu);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;
    }
    wait_vmcnt<0>();
#undef Q2D_MFMA
#undef Q2D_READ
}

// Large-tile MXFP8 kernel (the query/key projections): 256 x 256 output tile,
// 4 waves of 128 x 128, E4M3 operands (8 VGPRs per lane per MFMA, 64 cycles
// each).  A stage holds one K-tile of 64 values: 64 bytes per row of A and of B
// (16 KB each), filled by global_load_lds DMA through a ring of kStages
// stages.  Each iteration runs the 16 MFMAs of one K-tile while the next
// K-tile's fragments are read and the stage just consumed is refilled; the
// fragment buffers alternate between two register sets.
//
// Scales: a row's 4-byte word holds the 1x32 scales of two K-tiles of 64, and
// the rows of a tile are ld_scales apart, so a wave's scale load touches one
// line per lane; those loads, not the codes, bound the first version of this
// kernel (without them it ran 27-30 % faster).  S16: each row's 16 bytes for
// eight K-tiles (one group) arrive in one load per operand and wave, into a
// double-buffered side area of the LDS, issued with the codes of the group's
// first K-tile.  Otherwise (K not a multiple of 512, or rows of scales not
// 16-byte aligned) the word of an even K-tile goes into its stage and the odd
// K-tile reuses it.
constexpr int kDma8Codes = 8;                   // per wave per K-tile: 4 A and 4 B code loads
constexpr int kStage8 = 2 * kCodeBytes + 2048;  // word path: codes, then the A and B words
constexpr int kSide8 = 2 * 2 * 256 * 16;        // S16: 2 groups x {A, B} x 256 rows x 16 bytes

template <bool BF16OUT, bool ACC, bool S16>
__global__ __launch_bounds__(kThreads, 1) void gemm_fp8_256_kernel(GemmArgs g, int tiles_m, int tiles_n)
{
    using F = Fmt<kFmtMxfp8>;
    constexpr int RB = 64;                          // bytes per row per K-tile of 64
    constexpr int kStageB = S16 ? 2 * kCodeBytes : kStage8;
    constexpr int kSide = kStages * kStageB;        // S16 side area
    __shared__ __attribute__((aligned(1024))) uint8_t smem[kStages * kStageB + (S16 ? kSide8 : 0)];

    int tm, tn;
    {
        int64_t tm64, tn64;
        tile_coords(tiles_m, tiles_n, tm64, tn64);
        tm = (int)tm64; tn = (int)tn64;
    }
    const int64_t m0 = (int64_t)tm * BM2, n0 = (int64_t)tn * BN2;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1;
    const int half = lane >> 5;
    const uint32_t nk = (uint32_t)(g.K / 64);       // K is a multiple of 128
    const uint32_t nw = (uint32_t)(g.K / 128);      // scale words per row (S16: at least 4)
    // bf16 output: interleaved output columns with pair stores, as in the FP4
    // kernel (the per-row scale words follow their rows)
    constexpr bool PERM = BF16OUT;

    // codes: DMA j of this wave fills bytes [(4j + wave) * 1024, +1024) of an
    // operand stage (rows 16 (4j + wave) + lane / 4, physical chunk lane % 4,
    // the 64-byte-row swizzle of the E2M1 kernel); scales: the wave's DMA
    // covers rows 64 wave + lane of the tile's A and B rows
    uint32_t offA[4], offB[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int row = 16 * (4 * j + wave) + (lane >> 2);
        const int c = (lane & 3) ^ Fmt<kFmtFp4Block2D>::swz(row);
        int64_t ra = m0 + row; ra = ra < g.M ? ra : g.M - 1;
        int64_t rb = n0 + (PERM ? interleaved_row(row) : row); rb = rb < g.N ? rb : g.N - 1;
        offA[j] = (uint32_t)(ra * g.lda + c * 16);
        offB[j] = (uint32_t)(rb * g.ldb + c * 16);
    }
    uint32_t soffA, soffB;
    {
        int64_t ra = m0 + 64 * wave + lane; ra = ra < g.M ? ra : g.M - 1;
        int64_t rb = n0 + (PERM ? interleaved_row(64 * wave + lane) : 64 * wave + lane);
        rb = rb < g.N ? rb : g.N - 1;
        soffA = (uint32_t)(ra * g.ldsa);
        soffB = (uint32_t)(rb * g.ldsb);
    }
    const uint32_t lds0 = (uint32_t)(uintptr_t)&smem[0];
    const int sw = Fmt<kFmtFp4Block2D>::swz(lane & 31);
    const int rd_a = (wm * 128 + (lane & 31)) * RB;
    const int rd_b = kCodeBytes + (wn * 128 + (lane & 31)) * RB;
    // the lane's row words: word path at stage + 2 * kCodeBytes (+ 1024 for B);
    // S16 at side + group buffer * 8192 (+ 4096 for B) + 16 * row
    const int rs_a = S16 ? kSide + (wm * 128 + (lane & 31)) * 16 : 2 * kCodeBytes + (wm * 128 + (lane & 31)) * 4;
    const int rs_b = S16 ? kSide + 4096 + (wn * 128 + (lane & 31)) * 16
                         : 2 * kCodeBytes + 1024 + (wn * 128 + (lane & 31)) * 4;
    constexpr int kRowStride = S16 ? 32 * 16 : 32 * 4;      // words of fragment tile i + 1

    v16f acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    // code loads of K-tile t (part 0..7); past the last K-tile they repeat it
    // into a stage that is never read
    auto dma = [&](uint32_t t, int part) __attribute__((always_inline)) {
        const uint32_t tt = t < nk ? t : nk - 1;
        const uint32_t stage = lds0 + (t % kStages) * kStageB;
        const int jj = part >> 1;
        if ((part & 1) == 0) lds_dma16(g.a + tt * RB, offA[jj], stage + (4 * jj + wave) * 1024);
        else lds_dma16(g.b + tt * RB, offB[jj], stage + kCodeBytes + (4 * jj + wave) * 1024);
    };
    // scale loads: word path, the word of even K-tile t into its stage; S16, the
    // 16 bytes of group p into buffer p & 1 (past the last group, the last one's
    // bytes again: those loads fill a buffer that is never read)
    auto sdma = [&](uint32_t t) __attribute__((always_inline)) {
        if constexpr (S16) {
            const uint32_t p = t >> 3;
            const uint32_t o = 4 * (4 * p < nw - 4 ? 4 * p : nw - 4);
            const uint32_t buf = lds0 + kSide + (p & 1) * 8192;
            lds_dma16(g.sa, soffA + o, buf + wave * 1024);
            lds_dma16(g.sb, soffB + o, buf + 4096 + wave * 1024);
        } else {
            const uint32_t tt = t < nk ? t : nk - 1;
            const uint32_t stage = lds0 + (t % kStages) * kStageB;
            lds_dma4(g.sa + soffA + (tt >> 1) * 4, stage + 2 * kCodeBytes + wave * 256);
            lds_dma4(g.sb + soffB + (tt >> 1) * 4, stage + 2 * kCodeBytes + 1024 + wave * 256);
        }
    };
    // does K-tile t bring scale loads with it
    auto has_scales = [&](uint32_t t) __attribute__((always_inline)) -> bool {
        return S16 ? (t & 7) == 0 : (t & 1) == 0;
    };
    // LDS address of the word of even K-tile t for fragment row base `rs`
    auto word_at = [&](uint32_t t, int rs) __attribute__((always_inline)) -> const uint32_t * {
        if constexpr (S16) {
            const uint32_t p = t >> 3;
            uint32_t w = (t >> 1) - (4 * p < nw - 4 ? 4 * p : nw - 4);
            w = w < 3 ? w : 3;                      // K-tile nk (read, never used) stays in the row's slot
            return reinterpret_cast<const uint32_t *>(smem + rs + (p & 1) * 8192 + 4 * w);
        } else {
            return reinterpret_cast<const uint32_t *>(smem + (t % kStages) * kStageB + rs);
        }
    };

    // fragments of one K-tile: A tile i / B tile j as two 16-byte chunks
    // (chunks half and 2 + half of the row) and the rows' scale words, in two
    // register sets: while one K-tile's MFMAs run on one set, the next
    // K-tile's fragments are read into the other early in the K-tile, so the
    // reads have landed long before their first use
    v8i fa0[4], fb0[4], fa1[4], fb1[4];
    uint32_t sa0[4], sb0[4], sa1[4], sb1[4];
    const int c0 = (half ^ sw) * 16, c1 = ((2 + half) ^ sw) * 16;
#define Q2D_RD8(dst, base, row_off)                                                                  \
    do {                                                                                             \
        const uint4 x0_ = *reinterpret_cast<const uint4 *>((base) + (row_off) + c0);                 \
        const uint4 x1_ = *reinterpret_cast<const uint4 *>((base) + (row_off) + c1);                 \
        dst[0] = (int)x0_.x; dst[1] = (int)x0_.y; dst[2] = (int)x0_.z; dst[3] = (int)x0_.w;          \
        dst[4] = (int)x1_.x; dst[5] = (int)x1_.y; dst[6] = (int)x1_.z; dst[7] = (int)x1_.w;          \
    } while (0)

    // K-tile kt on (fa, fb, sa, sb); the fragments of K-tile kt + 1 into (na, nb,
    // nsa, nsb).  PH = kt mod 8 (S16) or kt mod 2: which K-tiles around kt carry
    // scale loads, so the waits count exactly the loads that may stay outstanding
    auto ktile = [&](auto ph, uint32_t kt, v8i (&fa)[4], v8i (&fb)[4], uint32_t (&sa)[4], uint32_t (&sb)[4],
                     v8i (&na)[4], v8i (&nb)[4], uint32_t (&nsa)[4], uint32_t (&nsb)[4]) __attribute__((always_inline)) {
        constexpr int PH = decltype(ph)::value;
        constexpr bool ODD = (PH & 1) != 0;
        constexpr auto scales_at = [](int t) { return S16 ? (t & 7) == 0 : (t & 1) == 0; };
        // K-tile kt + 1 and its scales landed: the loads of kt + 2 and kt + 3 may not have
        constexpr int kAfter = 2 * kDma8Codes + (scales_at(PH + 2) ? 2 : 0) + (scales_at(PH + 3) ? 2 : 0);
        constexpr bool kScNext = scales_at(PH + kStages);       // K-tile kt + 4's loads include scales
        __builtin_amdgcn_s_waitcnt(0xC07F);                     // lgkmcnt(0): this K-tile's reads done
        wait_vmcnt<kAfter>();
        block_barrier();
        const uint8_t *sn = smem + ((kt + 1) % kStages) * kStageB;   // past the last K-tile: unused reads
        const int byte = 2 * (kt & 1) + half;                   // this K-tile's scale in the row word
#pragma unroll
        for (int i = 0; i < 4; ++i) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int sa_ = (int)((sa[i] >> (8 * byte)) & 0xFFu);
                const int sb_ = (int)((sb[j] >> (8 * byte)) & 0xFFu);
                acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(fa[i], fb[j], acc[i][j], F::kCbsz,
                                                                            F::kCbsz, 0, sa_, 0, sb_);
                __builtin_amdgcn_sched_barrier(0);
                const int q = 4 * i + j;
                if (q < kDma8Codes) {
                    dma(kt + kStages, q);
                    __builtin_amdgcn_sched_barrier(0);
                } else if (q == kDma8Codes && kScNext) {
                    sdma(kt + kStages);
                    __builtin_amdgcn_sched_barrier(0);
                }
                if (q >= 1 && q <= 8) {
                    const int f = (q - 1) >> 1;
                    // an odd K-tile's words are the even one's
                    if (((q - 1) & 1) == 0) {
                        Q2D_RD8(na[f], sn, rd_a + f * 32 * RB);
                        nsa[f] = ODD ? word_at(kt + 1, rs_a + f * kRowStride)[0] : sa[f];
                    } else {
                        Q2D_RD8(nb[f], sn, rd_b + f * 32 * RB);
                        nsb[f] = ODD ? word_at(kt + 1, rs_b + f * kRowStride)[0] : sb[f];
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
        }
    };

    if (nk > 0) {
        for (uint32_t t = 0; t < kStages; ++t) {
            for (int p = 0; p < kDma8Codes; ++p) dma(t, p);
            if (has_scales(t)) sdma(t);
        }
        // K-tile 0 and its scales landed: the loads of K-tiles 1..3 may be outstanding
        // (S16: 3 x 8 code loads; word path: 3 x 8 code loads and 2 scale loads)
        wait_vmcnt<3 * kDma8Codes + (S16 ? 0 : 2)>();
        block_barrier();
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            Q2D_RD8(fa0[i], smem, rd_a + i * 32 * RB);
            Q2D_RD8(fb0[i], smem, rd_b + i * 32 * RB);
            sa0[i] = word_at(0, rs_a + i * kRowStride)[0];
            sb0[i] = word_at(0, rs_b + i * kRowStride)[0];
        }
        using std::integral_constant;
        if constexpr (S16) {
            // nk is a multiple of 8 (K of 512)
            for (uint32_t kt = 0; kt < nk; kt += 8) {
                ktile(integral_constant<int, 0>{}, kt, fa0, fb0, sa0, sb0, fa1, fb1, sa1, sb1);
                ktile(integral_constant<int, 1>{}, kt + 1, fa1, fb1, sa1, sb1, fa0, fb0, sa0, sb0);
                ktile(integral_constant<int, 2>{}, kt + 2, fa0, fb0, sa0, sb0, fa1, fb1, sa1, sb1);
                ktile(integral_constant<int, 3>{}, kt + 3, fa1, fb1, sa1, sb1, fa0, fb0, sa0, sb0);
                ktile(integral_constant<int, 4>{}, kt + 4, fa0, fb0, sa0, sb0, fa1, fb1, sa1, sb1);
                ktile(integral_constant<int, 5>{}, kt + 5, fa1, fb1, sa1, sb1, fa0, fb0, sa0, sb0);
                ktile(integral_constant<int, 6>{}, kt + 6, fa0, fb0, sa0, sb0, fa1, fb1, sa1, sb1);
                ktile(integral_constant<int, 7>{}, kt + 7, fa1, fb1, sa1, sb1, fa0, fb0, sa0, sb0);
            }
        } else {
            // nk is even (K is a multiple of 128)
            for (uint32_t kt = 0; kt < nk; kt += 2) {
                ktile(integral_constant<int, 0>{}, kt, fa0, fb0, sa0, sb0, fa1, fb1, sa1, sb1);
                ktile(integral_constant<int, 1>{}, kt + 1, fa1, fb1, sa1, sb1, fa0, fb0, sa0, sb0);
            }
        }
        wait_vmcnt<0>();
    }
#undef Q2D_RD8

    const bool full = m0 + BM2 <= g.M && n0 + BN2 <= g.N;
    if constexpr (PERM) {
        const uint32_t ldc_bytes = (uint32_t)(g.ldc * 2);
        const bool pair_ok = ((reinterpret_cast<uintptr_t>(g.c) | (uintptr_t)ldc_bytes) & 3u) == 0;
        const int64_t r0 = m0 + wm * 128, cl0 = n0 + wn * 128;
        uint8_t *cb = reinterpret_cast<uint8_t *>(g.c) + r0 * ldc_bytes + cl0 * 2;
        const int rows_left = (int)(g.M - r0), cols_left = (int)(g.N - cl0);
        if (full) {
            if (pair_ok) store_block_pairs<ACC, false, true>(acc, cb, ldc_bytes, 128, 128);
            else store_block_pairs<ACC, false, false>(acc, cb, ldc_bytes, 128, 128);
        } else {
            if (pair_ok) store_block_pairs<ACC, true, true>(acc, cb, ldc_bytes, rows_left, cols_left);
            else store_block_pairs<ACC, true, false>(acc, cb, ldc_bytes, rows_left, cols_left);
        }
    } else {
        const int64_t row0 = m0 + wm * 128 + 4 * half;
        const int64_t col0 = n0 + wn * 128 + (lane & 31);
        if (full) store_tile<BF16OUT, ACC, false>(acc, g, row0, col0);
        else store_tile<BF16OUT, ACC, true>(acc, g, row0, col0);
    }
}


// persistent kernel over at most `tiles` tiles: one workgroup per CU, a
// multiple of 8 (the XCD count) so that every workgroup stays on one XCD's
// share of the tile order
template <bool BF, int GMODE, int SM = 0>
hipError_t launch_persistent(const GemmArgs &g, const GroupedArgs &gr, int tm, int tn, int64_t tiles, hipStream_t s)
{
    int64_t grid = cu_count();
    grid = grid < tiles ? grid : tiles;
    grid = (grid + kXcds - 1) / kXcds * kXcds;
    if (g.accumulate)
        hipLaunchKernelGGL((gemm_fp4_persistent_kernel<BF, true, GMODE, SM>), dim3((unsigned)grid), dim3(kThreads), 0, s,
                           g, tm, tn, gr);
    else
        hipLaunchKernelGGL((gemm_fp4_persistent_kernel<BF, false, GMODE, SM>), dim3((unsigned)grid), dim3(kThreads), 0,
                           s, g, tm, tn, gr);
    return hipGetLastError();
}

// dense: the scale mode of the two operands
template <bool BF>
hipError_t launch_dense(const GemmArgs &g, int tm, int tn, hipStream_t s)
{
    const GroupedArgs none = {nullptr, 0, 0, 0, 0, 0};
    const int64_t tiles = (int64_t)tm * tn;
    switch ((g.a1d ? 1 : 0) | (g.b1d ? 2 : 0)) {
    case 0: return launch_persistent<BF, 0, 0>(g, none, tm, tn, tiles, s);
    case 1: return launch_persistent<BF, 0, 1>(g, none, tm, tn, tiles, s);
    case 2: return launch_persistent<BF, 0, 2>(g, none, tm, tn, tiles, s);
    default: return launch_persistent<BF, 0, 3>(g, none, tm, tn, tiles, s);
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
    // the 256 x 256 kernel once there are enough output tiles to fill the chip
    // (its loads address each operand with 32-bit byte offsets from the K-tile base)
    const bool off32 = g.M * g.lda <= (int64_t(1) << 32) && g.N * g.ldb <= (int64_t(1) << 32);
    if (fmt == kFmtFp4Block2D && off32 && ((g.M + BM2 - 1) / BM2) * ((g.N + BN2 - 1) / BN2) >= 128) {
        const int tm = (int)((g.M + BM2 - 1) / BM2), tn = (int)((g.N + BN2 - 1) / BN2);
        return c_is_bf16 ? launch_dense<true>(g, tm, tn, stream) : launch_dense<false>(g, tm, tn, stream);
    }
    if (fmt == kFmtFp4Block2D)
        return c_is_bf16 ? launch_t<kFmtFp4Block2D, true>(g, stream) : launch_t<kFmtFp4Block2D, false>(g, stream);
    if (off32 && ((g.M + BM2 - 1) / BM2) * ((g.N + BN2 - 1) / BN2) >= 128) {
        const int tm = (int)((g.M + BM2 - 1) / BM2), tn = (int)((g.N + BN2 - 1) / BN2);
        // 16-byte scale loads: whole groups of 8 K-tiles, 16-byte aligned rows
        const bool s16 = g.K % 512 == 0 && g.ldsa % 16 == 0 && g.ldsb % 16 == 0 &&
                         reinterpret_cast<uintptr_t>(g.sa) % 16 == 0 && reinterpret_cast<uintptr_t>(g.sb) % 16 == 0;
        const dim3 grid((unsigned)(tm * tn)), block(kThreads);
        if (s16) {
            if (c_is_bf16) {
                if (g.accumulate) hipLaunchKernelGGL((gemm_fp8_256_kernel<true, true, true>), grid, block, 0, stream, g, tm, tn);
                else hipLaunchKernelGGL((gemm_fp8_256_kernel<true, false, true>), grid, block, 0, stream, g, tm, tn);
            } else {
                if (g.accumulate) hipLaunchKernelGGL((gemm_fp8_256_kernel<false, true, true>), grid, block, 0, stream, g, tm, tn);
                else hipLaunchKernelGGL((gemm_fp8_256_kernel<false, false, true>), grid, block, 0, stream, g, tm, tn);
            }
        } else {
            if (c_is_bf16) {
                if (g.accumulate) hipLaunchKernelGGL((gemm_fp8_256_kernel<true, true, false>), grid, block, 0, stream, g, tm, tn);
                else hipLaunchKernelGGL((gemm_fp8_256_kernel<true, false, false>), grid, block, 0, stream, g, tm, tn);
            } else {
                if (g.accumulate) hipLaunchKernelGGL((gemm_fp8_256_kernel<false, true, false>), grid, block, 0, stream, g, tm, tn);
                else hipLaunchKernelGGL((gemm_fp8_256_kernel<false, false, false>), grid, block, 0, stream, g, tm, tn);
            }
        }
        return hipGetLastError();
    }
    return c_is_bf16 ? launch_t<kFmtMxfp8, true>(g, stream) : launch_t<kFmtMxfp8, false>(g, stream);
}

namespace {

template <int SM, bool QSR>
void launch_quantized_t(const GemmArgs &g, int tm, int tn, int64_t grid, hipStream_t stream)
{
    const GroupedArgs none = {nullptr, 0, 0, 0, 0, 0};
    hipLaunchKernelGGL((gemm_fp4_persistent_kernel<false, false, 0, SM, true, QSR>), dim3((unsigned)grid),
                       dim3(kThreads), 0, stream, g, tm, tn, none);
}

template <bool QSR>
void launch_quantized_sm(const GemmArgs &g, int tm, int tn, int64_t grid, hipStream_t stream)
{
    switch ((g.a1d ? 1 : 0) | (g.b1d ? 2 : 0)) {
    case 0: launch_quantized_t<0, QSR>(g, tm, tn, grid, stream); break;
    case 1: launch_quantized_t<1, QSR>(g, tm, tn, grid, stream); break;
    case 2: launch_quantized_t<2, QSR>(g, tm, tn, grid, stream); break;
    default: launch_quantized_t<3, QSR>(g, tm, tn, grid, stream); break;
    }
}

}  // namespace

hipError_t launch_gemm_quantized(const GemmArgs &g, hipStream_t stream)
{
    const bool off32 = g.M * g.lda <= (int64_t(1) << 32) && g.N * g.ldb <= (int64_t(1) << 32);
    if (!off32) return hipErrorInvalidValue;
    const int tm = (int)((g.M + BM2 - 1) / BM2), tn = (int)((g.N + BN2 - 1) / BN2);
    int64_t grid = cu_count();
    const int64_t tiles = (int64_t)tm * tn;
    grid = grid < tiles ? grid : tiles;
    grid = (grid + kXcds - 1) / kXcds * kXcds;
    if (g.qsr) launch_quantized_sm<true>(g, tm, tn, grid, stream);
    else launch_quantized_sm<false>(g, tm, tn, grid, stream);
    return hipGetLastError();
}

hipError_t launch_grouped_gemm(const GemmArgs &g, const GroupedArgs &gr, int c_is_bf16, hipStream_t stream)
{
    const int tn = (int)((g.N + BN2 - 1) / BN2);
    if (!gr.ragged_k) {
        // row tiles over all experts: at most total_rows / 256 + nseg
        const int rt = (int)((gr.total_rows + BM2 - 1) / BM2) + gr.nseg;
        return c_is_bf16 ? launch_persistent<true, 1>(g, gr, 0, tn, (int64_t)rt * tn, stream)
                         : launch_persistent<false, 1>(g, gr, 0, tn, (int64_t)rt * tn, stream);
    }
    const int tm = (int)((g.M + BM2 - 1) / BM2);
    return c_is_bf16 ? launch_persistent<true, 2>(g, gr, tm, tn, (int64_t)gr.nseg * tm * tn, stream)
                     : launch_persistent<false, 2>(g, gr, tm, tn, (int64_t)gr.nseg * tm * tn, stream);
}

}  // namespace q2d
