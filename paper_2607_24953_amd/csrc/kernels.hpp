// Internal kernel-launch interface of libq2d (host and device side).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace q2d {

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
};

hipError_t launch_fp4_quantize(const QuantArgs &a, int dtype_bytes, bool stochastic,
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
};

enum GemmFmt { kFmtFp4Block2D = 0, kFmtMxfp8 = 1 };

hipError_t launch_gemm(const GemmArgs &g, int fmt, int c_is_bf16, hipStream_t stream);

}  // namespace q2d
