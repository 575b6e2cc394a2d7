// Internal kernel-launch interface of libq2d (host and device side).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace q2d {

// compute units of the current device (queried once per device)
int cu_count();

// One 2D-block FP4 or MXFP8 quantization launch over an R x C matrix whose
// element (r, c) sits at x[r*stride_r + c*stride_c].
struct QuantArgs {
    const void *x;
    int64_t rows, cols;            // logical R x C
    int64_t rows_pad, cols_pad;    // R and C rounded up to 128
    int64_t stride_r, stride_c;    // elements
    int64_t index_base;            // added to storage indices before they key the SR stream
    uint64_t seed, offset;
    uint8_t *codes;    int64_t ld_codes;
    uint8_t *codes_t;  int64_t ld_codes_t;
    uint8_t *scales;   int64_t ld_scales;
    uint8_t *scales_t; int64_t ld_scales_t;
    int64_t nbr, nbc;              // scale-grid rows ceil(R/32) and columns ceil(C/32)
    // Grouped (MoE) form: when seg_offsets is set, the rows are nseg segments
    // stored back to back (segment e = rows seg_offsets[e] .. seg_offsets[e+1]);
    // each is quantized as its own matrix and written from padded row
    // P[e] = sum over f < e of roundup(n_f, 128).  rows_pad then bounds the
    // padded rows and `rows` is the total number of input rows.
    const int64_t *seg_offsets;
    int32_t nseg;
    int64_t store_rows;            // rows of codes / scales written (>= rows; padded rows get zeros)
    int32_t block;                 // 2D block edge: 32, or 64 (its scale written to the four 32-entries)
    int32_t floor_scale;           // 2D FP4: floor scale rule with saturation instead of the truncation-free one
};

// 2D blocks, or 1D blocks (oned: 1 x 32 rowwise copy, 32 x 1 colwise copy)
hipError_t launch_fp4_quantize(const QuantArgs &a, int dtype_bytes, bool stochastic, bool oned,
                               hipStream_t stream);
hipError_t launch_mxfp8_quantize(const QuantArgs &a, int dtype_bytes, hipStream_t stream);

// C[M][N] (+)= A . B^T for K-major quantized operands A [M][K], B [N][K].
struct GemmArgs {
    const uint8_t *a;  int64_t lda;     // codes, bytes per row
    const uint8_t *sa; int64_t ldsa;    // scales, bytes per row
    const uint8_t *b;  int64_t ldb;
    const uint8_t *sb; int64_t ldsb;
    void *c;           int64_t ldc;     // elements
    int64_t M, N, K;                    // K rounded up to 128
    int accumulate;
    int a1d, b1d;                       // FP4: operand with one scale per row and K-group (1x32 blocks)
    // quantized output (FP4 GEMM only): C in 2D-block FP4, both orientations
    // (the layout of a q2d_tensor), round to nearest; c is then unused
    uint8_t *qc;  int64_t ldqc;         // codes [M][ldqc]
    uint8_t *qct; int64_t ldqct;        // codes_t [N][ldqct]
    uint8_t *qs;  int64_t ldqs;         // scales [ceil(M/32)][ldqs]
    uint8_t *qst; int64_t ldqst;        // scales_t [ceil(N/32)][ldqst]
    // stochastic rounding of the quantized output: element (r, c) draws the
    // 16-bit value of storage index r * N + c from the Philox stream (seed, offset)
    int qsr;
    uint64_t seed, offset;
};

enum GemmFmt { kFmtFp4Block2D = 0, kFmtMxfp8 = 1 };

// C = op(A) op(B)^T quantized to 2D-block FP4 in the epilogue (g.qc .. set)
hipError_t launch_gemm_quantized(const GemmArgs &g, hipStream_t stream);

hipError_t launch_gemm(const GemmArgs &g, int fmt, int c_is_bf16, hipStream_t stream);

// Grouped (MoE) GEMMs over nseg experts with device segment offsets.
//   ragged M: A = grouped rows (padded), op(B) of expert e is rows
//             [e*N, (e+1)*N) (b_group_rows = N) or K columns [e*K, (e+1)*K)
//             (b_group_rows = 0, b_group_k = K); C rows are the unpadded rows.
//   ragged K: A, B grouped along K (padded), C of expert e at c + e*M*ldc.
struct GroupedArgs {
    const int64_t *seg_offsets;
    int32_t nseg;
    int32_t ragged_k;
    int64_t total_rows;        // sum of segment rows (unpadded)
    int64_t b_group_rows;      // ragged M: rows of op(B) per expert, or 0
    int64_t b_group_k;         // ragged M: K columns of op(B) per expert, or 0
};

hipError_t launch_grouped_gemm(const GemmArgs &g, const GroupedArgs &gr, int c_is_bf16, hipStream_t stream);

// Dequantization of one stored copy back to R x C values (row-major out).
struct DequantArgs {
    const uint8_t *codes;  int64_t ld_codes;    // the copy read: codes, or codes_t (transposed)
    const uint8_t *scales; int64_t ld_scales;   // its scales
    int64_t rows, cols;                         // R x C of the matrix
    int fmt;                                    // 0 FP4 2D blocks, 1 MXFP8, 2 FP4 1D blocks
    int transposed;                             // the copy stores element (r, c) in row c
    void *out; int64_t ldo;                     // elements
    int out_bf16;
    int out_vec;                                // out and ldo allow 4-element vector stores
    int8_t *exps; int64_t lde;                  // optional per-element scale exponents
};

hipError_t launch_dequantize(const DequantArgs &a, hipStream_t stream);

}  // namespace q2d
