/*
 * q2d.h -- C ABI of libq2d: transposition-invariant 2D-block FP4 quantization
 * and the FP4 / MXFP8 GEMMs of a linear layer on AMD Instinct MI355X (gfx950).
 *
 * The method ("Stable FP4 Training via Transposition-Invariant Block
 * Quantization"):
 *   - a tensor is cut into b x b square blocks; each block gets one
 *     power-of-two scale S = 2^ceil(log2(2M / (Qp - Qn))) from its maximum
 *     magnitude M, with the E2M1 bounds Qp = 6, Qn = -6, so nothing is
 *     clipped (Sec. 3.1; App. D);
 *   - elements are stored as 4-bit E2M1 codes of x / S, rounded to nearest
 *     (forward operands) or stochastically with E[round(x)] = x (gradients)
 *     (Sec. 3.1; App. E);
 *   - a square block keeps its values and its scale under transposition
 *     (Sec. 3; App. D), so each operand of Y = X W^T, dX = dY W and
 *     dW = dY^T X is quantized once and reused transposed (App. C).
 *     libq2d emits the row-packed and the column-packed copy in one pass;
 *     both hold the same codes and the same scales;
 *   - the query/key projections use MXFP8 (E4M3 elements, 1x32 blocks)
 *     instead (Sec. 3.2; App. C).
 *
 * Conventions shared by every entry point:
 *   - Ownership: the caller allocates every buffer; libq2d never allocates,
 *     frees or synchronizes.  Sizes come from q2d_tensor_init.
 *   - Pointers: inputs x and outputs C are device pointers; code and scale
 *     buffers are device pointers; seg_offsets arrays are device pointers;
 *     descriptors (q2d_tensor) live in host memory.
 *   - Ordering: all work is enqueued on `stream` (0 = the null stream) and
 *     is valid in stream order.  No call blocks the host.
 *   - Errors: argument errors are detected on the host before any launch and
 *     returned as a status; nothing is printed, no exception crosses the ABI.
 *     A failed launch returns Q2D_ELAUNCH.  Extents (rows, cols, total rows)
 *     above 2^31, and a strided view whose last storage index
 *     (rows-1)*stride_r + (cols-1)*stride_c reaches 2^47 elements, return
 *     Q2D_EUNSUPPORTED.  Data-dependent conditions are not
 *     errors: a block holding a NaN or an infinity gets scale byte 0xFF (the
 *     E8M0 NaN) and all-zero codes.
 *   - Thread safety: the library keeps no mutable state.
 */
#ifndef Q2D_H
#define Q2D_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* In C++ the enumerations get int as their fixed underlying type, so that any
 * int a C caller passes is a value of the type (and is rejected by the argument
 * checks) rather than undefined behaviour; the size and calling convention are
 * those of int in both languages. */
#ifdef __cplusplus
#define Q2D_ENUM_BASE : int
#else
#define Q2D_ENUM_BASE
#endif

typedef enum Q2D_ENUM_BASE {
    Q2D_OK = 0,
    Q2D_EINVAL = 1,          /* bad argument: null pointer, size, stride, alignment, shape mismatch */
    Q2D_EUNSUPPORTED = 2,    /* valid request this build does not implement (e.g. block 16) */
    Q2D_ELAUNCH = 3          /* the HIP runtime rejected a kernel launch */
} q2d_status;

typedef enum Q2D_ENUM_BASE { Q2D_F32 = 0, Q2D_BF16 = 1 } q2d_dtype;

typedef enum Q2D_ENUM_BASE {
    Q2D_RTN = 0,             /* round to nearest, ties to the even E2M1 code (App. E, forward) */
    Q2D_SR = 1,              /* stochastic rounding, Philox4x32-10, 16 bits per element (App. E) */
    /* Flag OR-ed into Q2D_RTN or Q2D_SR for 2D-block FP4 (q2d_quantize,
     * q2d_grouped_quantize, and the linear-layer calls that use them): the scale
     * rule that the truncation-free ablation removes (Sec. 4.2, Fig. 5; App. G,
     * "Truncation-free scaling").  The block exponent becomes
     * e = floor(log2 M) - 2 (M's leading-bit exponent minus E2M1's largest
     * exponent, clamped to -127) and magnitudes above 6 * 2^e saturate to 6
     * before rounding, so a block maximum with mantissa above 1.5 is clipped by
     * up to 25 %.  Q2D_EUNSUPPORTED for the 1D quantizer. */
    Q2D_FLOOR_SCALE = 0x10
} q2d_round;

typedef enum Q2D_ENUM_BASE {
    Q2D_FMT_FP4_2D = 0,      /* E2M1 codes, one E8M0 scale per 32x32 block (Sec. 3) */
    Q2D_FMT_MXFP8 = 1,       /* E4M3 codes, one E8M0 scale per 1x32 block (Sec. 3.2) */
    Q2D_FMT_FP4_1D = 2       /* E2M1 codes, one E8M0 scale per 1x32 block: activations
                                (Sec. 3, "Application to linear layers"; App. C) */
} q2d_fmt;

/*
 * A quantized R x C matrix in both orientations.
 *
 * FP4_2D (Sec. 3; App. D):
 *   codes    [rows][ld_codes] bytes; byte (r, c/2), low nibble = even c.
 *            Bytes up to roundup(cols,128)/2 of each row are written (padding 0).
 *   codes_t  [cols][ld_codes_t] bytes; byte (c, r/2), low nibble = even r.
 *            Bytes up to roundup(rows,128)/2 of each row are written.
 *   scales   [ceil(rows/32)][ld_scales]: E8M0 byte e+127 of block (r/32, c/32);
 *            entries up to roundup(cols,128)/32 are written (padding 0x00).
 *   scales_t [ceil(cols/32)][ld_scales_t]: the same bytes transposed,
 *            entries up to roundup(rows,128)/32 written.  Every value in
 *            scales_t equals the one in scales: the transposition invariance.
 *   A nibble is sign << 3 | m with m indexing {0, .5, 1, 1.5, 2, 3, 4, 6}.
 *   block 64 (64x64 blocks, the larger block of the block-size trade-off,
 *   Table 4): the same buffers and the same 32-granular scale grids; the byte
 *   of 64x64 block (I, J) fills the four entries (2I..2I+1, 2J..2J+1) that
 *   exist, so every GEMM reads a block-64 tensor exactly as a block-32 one.
 *
 * MXFP8 (Sec. 3.2):
 *   codes    [rows][ld_codes] E4M3 bytes, scales [rows][ld_scales]: one scale
 *            per 1x32 block along columns (K = cols);
 *   codes_t  [cols][ld_codes_t], scales_t [cols][ld_scales_t]: the 32x1
 *            (column-direction) quantization, stored transposed (K = rows).
 *            Unlike FP4_2D, the two copies have different scales.
 *   Rows are padded to multiples of 128 bytes (codes) / 4 bytes (scales) as
 *   for FP4_2D, padding 0.
 *
 * FP4_1D (activations; Sec. 3, "Application to linear layers"; App. C,
 * "Activations"):
 *   codes / codes_t packed exactly as for FP4_2D;
 *   scales   [roundup(cols,128)/128][ld_scales >= 4*rows]: one 4-byte word per
 *            row and K-tile of 128 columns; the scale of the 1x32 block J of
 *            row r (K = cols) is byte J % 4 of word (J / 4, r), i.e.
 *            scales[(J / 4) * ld_scales + 4 r + J % 4];
 *   scales_t [roundup(rows,128)/128][ld_scales_t >= 4*cols]: likewise for the
 *            32x1 block I of column c (K = rows): scales_t[(I / 4) * ld_scales_t
 *            + 4 c + I % 4].
 *   (K-tile-major words put the scales a GEMM K-tile needs for consecutive
 *   rows at consecutive addresses.)
 *   The two copies have different blocks, scales and (in general) codes: the
 *   forward/backward inconsistency of 1D layouts (Sec. 2) that the 2D blocks
 *   of weights and gradients avoid.
 *
 * All leading dimensions are in bytes.  Pointers may be NULL for an
 * orientation the caller does not need (codes with scales, codes_t with
 * scales_t); GEMMs need the orientation their transpose flag selects.
 */
typedef struct {
    int32_t fmt;             /* q2d_fmt */
    int32_t block;           /* block edge: 32, or 64 for FP4_2D */
    int64_t rows, cols;      /* logical shape R x C */
    uint8_t *codes;    int64_t ld_codes;
    uint8_t *codes_t;  int64_t ld_codes_t;
    uint8_t *scales;   int64_t ld_scales;
    uint8_t *scales_t; int64_t ld_scales_t;
} q2d_tensor;

/*
 * Fill `t` with the layout of an R x C matrix (fmt, block, shape and the
 * minimal leading dimensions; pointers set to NULL) and, if `bytes` is not
 * NULL, the byte sizes of its four buffers {codes, codes_t, scales, scales_t}.
 * Host only.  Q2D_EINVAL for rows or cols <= 0; Q2D_EUNSUPPORTED for a block
 * other than 32, except 64 with FP4_2D.
 */
q2d_status q2d_tensor_init(q2d_tensor *t, q2d_fmt fmt, int64_t rows, int64_t cols,
                           int32_t block, int64_t bytes[4]);

/*
 * 2D-block FP4 quantization (Sec. 3, Sec. 3.1; App. D, App. E).
 *
 * x        device pointer to element (0, 0) of an R x C matrix of dtype `dt`;
 *          element (r, c) is x[r*stride_r + c*stride_c] (strides in elements,
 *          > 0).  Views are allowed: stride_c == 1 (row-major) and
 *          stride_r == 1 (a transposed view) take the fast path, other strides
 *          a slower element-wise path.
 * block    32 or 64 (64x64 blocks, Table 4); equal to out->block
 *          (Q2D_EINVAL otherwise).
 * mode     Q2D_RTN or Q2D_SR.  For SR the 16 random bits of the element with
 *          storage index i = r*stride_r + c*stride_c are half (i & 1) of word
 *          (i & 7) >> 1 of Philox4x32-10 with counter (g lo, g hi, offset lo,
 *          offset hi), g = i >> 3, and key (seed lo, seed hi); the magnitude
 *          rounds up iff floor(2^16 * d / delta) + r16 >= 2^16 (d = distance to
 *          the grid point below, delta = grid spacing).  A transposed view
 *          therefore draws the same bits as the matrix it views.
 * out      descriptor from q2d_tensor_init(FP4_2D, rows, cols, block) with device
 *          buffers attached; ld_* may exceed the minimum.  At least one of
 *          codes / codes_t must be set.  Buffers must be 16-byte aligned and
 *          leading dimensions multiples of 16 (codes) and 4 (scales).
 */
q2d_status q2d_quantize(const void *x, q2d_dtype dt, int64_t rows, int64_t cols,
                        int64_t stride_r, int64_t stride_c, int32_t block, q2d_round mode,
                        uint64_t seed, uint64_t offset, q2d_tensor *out, hipStream_t stream);

/*
 * 1D-block FP4 quantization of activations (Sec. 3, "Application to linear
 * layers": activations keep a 1D layout; App. C, "Activations"): one pass
 * writes the rowwise copy (1x32 blocks along columns; codes/scales, read by
 * the forward GEMM) and the colwise copy (32x1 blocks along rows, stored
 * transposed; codes_t/scales_t, read by the weight-gradient GEMM).  Every
 * block gets the truncation-free scale and the E2M1 codec of q2d_quantize;
 * for SR the element's one draw (same storage-index contract) serves both
 * copies.  Arguments, alignment and errors as for q2d_quantize; out from
 * q2d_tensor_init(FP4_1D, rows, cols, 32).
 */
q2d_status q2d_quantize_1d(const void *x, q2d_dtype dt, int64_t rows, int64_t cols,
                           int64_t stride_r, int64_t stride_c, int32_t block, q2d_round mode,
                           uint64_t seed, uint64_t offset, q2d_tensor *out, hipStream_t stream);

/*
 * MXFP8 quantization for the query/key projections (Sec. 3.2; App. C):
 * E4M3 codes rounded to nearest even, one truncation-free E8M0 scale per 1x32
 * block (smallest power of two S with 448 * S >= block maximum).  The rowwise
 * copy (blocks along columns) goes to codes/scales, the colwise copy (blocks
 * along rows, stored transposed) to codes_t/scales_t, both in one pass.
 * Arguments as for q2d_quantize; out from q2d_tensor_init(MXFP8, ...).
 */
q2d_status mxfp8_quantize(const void *x, q2d_dtype dt, int64_t rows, int64_t cols,
                          int64_t stride_r, int64_t stride_c, q2d_tensor *out,
                          hipStream_t stream);

/*
 * C[M][N] (+)= op(A) . op(B)^T on quantized operands (Sec. 3, "Application to
 * linear layers"; App. C), fp32 accumulation on scaled MFMA.
 *
 * op(X) = X (uses codes/scales; K = X.cols) when transX == 0, or X^T (uses
 * codes_t/scales_t; K = X.rows) when transX == 1.  M = rows of op(A),
 * N = rows of op(B); both must have the same K.  FP4_2D and FP4_1D operands
 * may be mixed (1D activations with 2D weights and gradients: App. C); MXFP8
 * pairs only with MXFP8.  Block-64 FP4_2D operands are read as block-32 ones
 * (their scale grids hold each 64x64 block's byte in all four entries).
 *   forward     Y  = X  W^T : q2d_gemm(X, 0, W, 0, ...)
 *   data grad   dX = dY W   : q2d_gemm(dY, 0, W, 1, ...)
 *   weight grad dW = dY^T X : q2d_gemm(dY, 1, X, 1, ...)
 * C        device pointer, row-major with leading dimension ldc (elements,
 *          >= N); c_dt Q2D_F32 or Q2D_BF16 (bf16 rounds to nearest even).
 * accumulate  0: C = result; 1: C += result (read-modify-write in c_dt).
 */
q2d_status q2d_gemm(const q2d_tensor *A, int transA, const q2d_tensor *B, int transB,
                    void *C, q2d_dtype c_dt, int64_t ldc, int accumulate, hipStream_t stream);

/*
 * GEMM with its result quantized in the epilogue: the float32 result C =
 * op(A) op(B)^T (as q2d_gemm computes it, never written out) goes straight
 * into 2D-block FP4 with round to nearest -- the truncation-free scale of each
 * 32x32 block and the E2M1 codec of q2d_quantize -- in both orientations.  The
 * output of one linear layer then enters the next GEMM without a bfloat16
 * round trip through memory (App. C: Y and dX are operands of further GEMMs).
 * Each 32x32 block of C is one 32x32 MFMA tile, so its maximum is found in the
 * tile's registers.
 *
 * A, B, transA, transB as for q2d_gemm (FP4_2D and FP4_1D operands).
 * mode     Q2D_RTN, or Q2D_SR for an output that is a gradient (App. E: the
 *          data gradient dX is the next layer's output gradient, which the
 *          method rounds stochastically).  SR follows q2d_quantize's contract
 *          for a row-major M x N tensor: element (r, c) has storage index
 *          r N + c and draws its 16 bits from the Philox stream (seed,
 *          offset), so the codes equal q2d_quantize(C, SR, seed, offset) of the
 *          float32 result.  N must be a multiple of 8 for SR.
 * seed, offset  the SR stream (ignored for Q2D_RTN).
 * out      descriptor from q2d_tensor_init(FP4_2D, M, N, 32) with all four
 *          buffers attached; written as q2d_quantize writes it (padding
 *          included).  A block holding a NaN or an infinity gets scale 0xFF
 *          and zero codes.
 * Q2D_EUNSUPPORTED for MXFP8 operands, block 64 output, SR with N not a
 * multiple of 8, or operands beyond 4 GiB.  Stream-ordered.
 */
q2d_status q2d_gemm_quantized(const q2d_tensor *A, int transA, const q2d_tensor *B, int transB, q2d_round mode,
                              uint64_t seed, uint64_t offset, q2d_tensor *out, hipStream_t stream);

/*
 * Forward pass of a quantized linear layer Y = X W^T (Sec. 3; App. C):
 * quantizes X [T][K] and W [N][K] (row-major, dtype dt) into qX and qW (both
 * orientations, kept for the backward pass) and runs the forward GEMM into
 * Y [T][N] (row-major, ldy = N, dtype y_dt).  The SR streams of X and W use
 * (seed, offset_x) and (seed, offset_w).  qX may be FP4_1D (the paper's
 * activation layout, App. C): X is then quantized with q2d_quantize_1d and the
 * backward pass's weight gradient reads its 32x1 copy.  Each FP4_2D
 * quantization uses its descriptor's block (32, or 64 for 64x64 blocks).
 */
q2d_status q2d_linear_fwd(const void *X, const void *W, q2d_dtype dt, int64_t T, int64_t N,
                          int64_t K, q2d_round mode_x, q2d_round mode_w, uint64_t seed,
                          uint64_t offset_x, uint64_t offset_w, q2d_tensor *qX, q2d_tensor *qW,
                          void *Y, q2d_dtype y_dt, hipStream_t stream);

/*
 * Backward pass of the same layer (Sec. 3; App. C, App. E): quantizes dY [T][N]
 * into qdY (both orientations) and computes dX = dY W into dX [T][K] and
 * dW = dY^T X into dW [N][K], reusing the forward's qX and qW transposed with
 * their unchanged scales (the straight-through estimator passes dY through the
 * quantizer unchanged).  accumulate_dw: 1 adds into dW.  dY is quantized with
 * qdY's block.
 */
q2d_status q2d_linear_bwd(const void *dY, q2d_dtype dt, const q2d_tensor *qX,
                          const q2d_tensor *qW, q2d_round mode_dy, uint64_t seed,
                          uint64_t offset_dy, q2d_tensor *qdY, void *dX, q2d_dtype dx_dt,
                          void *dW, q2d_dtype dw_dt, int accumulate_dw, hipStream_t stream);

/*
 * Dequantization of one stored copy (Sec. 2, "Bias induced by scale
 * inconsistency"; Fig. 1): the R x C values that a GEMM reading that copy
 * multiplies, in the matrix's own orientation.  copy 0 reads codes/scales (the
 * copy the forward GEMM reads), copy 1 reads codes_t/scales_t (the copy the
 * backward GEMMs read), both mapped back to element (r, c).  For FP4_2D the two
 * copies give identical output (transposition invariance); for FP4_1D and
 * MXFP8 they differ where the rowwise and columnwise blocks have different
 * scales.
 *
 * t        any descriptor from q2d_tensor_init (FP4_2D with block 32 or 64,
 *          FP4_1D, MXFP8) whose chosen copy has buffers attached.
 * out      device pointer, row-major [rows][ldo] (ldo >= cols, elements) of
 *          out_dt.  Q2D_F32: the exact value code * 2^e (E2M1 or E4M3FN code),
 *          rounded once to nearest even only outside float32's range;
 *          Q2D_BF16: round to nearest even of that value.  A block with scale
 *          byte 0xFF, and an E4M3 NaN code, give NaN.
 * exps     optional (NULL to skip) device int8 [rows][lde] (lde >= cols): the
 *          scale exponent e of each element's block, -128 for scale byte 0xFF.
 *          exps of copy 0 minus exps of copy 1 is the scale-difference map.
 * Q2D_EINVAL for a missing buffer, copy not 0 or 1, or leading dimensions
 * below cols.  Stream-ordered; no host synchronisation.
 */
q2d_status q2d_dequantize(const q2d_tensor *t, int copy, void *out, q2d_dtype out_dt, int64_t ldo,
                          int8_t *exps, int64_t lde, hipStream_t stream);

/*
 * Grouped (mixture-of-experts) form.  The rows of x are nseg expert segments
 * stored back to back: segment e is rows seg_offsets[e] .. seg_offsets[e+1]
 * (seg_offsets: device array of nseg + 1 int64, ascending, seg_offsets[0] = 0,
 * seg_offsets[nseg] = rows; 1 <= nseg <= 1024).  Each segment is its own
 * matrix for block quantization (Sec. 3; boundary blocks over valid rows only,
 * App. D): its 2D blocks start at its first row.  It is stored from padded row
 * P[e] = sum over f < e of roundup(n_f, 128) of the output, so every expert's
 * rows (codes) and every expert's K range (codes_t) start 128-aligned; padding
 * rows and nibbles are 0.  Storage indices for the SR stream are those of x
 * (rows counted from x), so a grouped call draws the same bits as quantizing
 * each segment's view of the same buffer.
 *
 * The offsets are read on the device, where they cannot be checked before a
 * launch.  The kernels use o'[i] = min(max(0, seg_offsets[0..i]), rows) (rows
 * = total_rows for the GEMM): a valid table is unchanged, and any other one
 * cannot take a kernel outside x, C or the grouped capacity; its results are
 * those of the table o'.
 *
 * q2d_grouped_tensor_init: layout of the padded form (rows = the capacity
 * roundup(rows + 127 * nseg, 128), cols as given); bytes[] as q2d_tensor_init.
 * Rows beyond the last segment's padded end are not written.  Q2D_EINVAL for
 * rows or cols <= 0 or nseg outside [1, 1024]; Q2D_EUNSUPPORTED for a block
 * other than 32 or a capacity above 2^31 - 1 rows.
 */
q2d_status q2d_grouped_tensor_init(q2d_tensor *t, int64_t rows, int64_t cols, int32_t nseg,
                                   int32_t block, int64_t bytes[4]);

/*
 * Grouped 2D-block FP4 quantization of a row-major [rows, cols] x with row
 * stride stride_r (>= cols) into `out` (from q2d_grouped_tensor_init).  Other
 * arguments and the rounding contract as for q2d_quantize.
 */
q2d_status q2d_grouped_quantize(const void *x, q2d_dtype dt, int64_t rows, int64_t cols,
                                int64_t stride_r, int32_t nseg, const int64_t *seg_offsets,
                                int32_t block, q2d_round mode, uint64_t seed, uint64_t offset,
                                q2d_tensor *out, hipStream_t stream);

/*
 * Grouped GEMMs of the expert FFN (the linear-layer GEMMs of Sec. 3 applied per
 * expert).  total_rows = seg_offsets[nseg] (the host passes it; the offsets stay
 * on the device).  A is a grouped tensor.
 *  transA == 0 (ragged M; forward and data gradient): C[seg_offsets[e] + i] =
 *    A_e[i] . op(B)_e^T for i < n_e.  op(B) is the stack of all experts'
 *    matrices: transB == 0 takes rows [e*N, (e+1)*N) of B (B->rows = nseg*N,
 *    N % 32 == 0, B->cols = K = A->cols); transB == 1 takes K columns
 *    [e*K, (e+1)*K) of B^T (B->rows = nseg*K, K % 128 == 0, N = B->cols).
 *    C is [total_rows][ldc >= N].
 *  transA == 1 (ragged K; weight gradient), transB == 1, B grouped like A:
 *    C_e = A_e^T . B_e (K = n_e, zero-padded to the 128-row boundary), stored at
 *    C + e * A->cols * ldc; C is [nseg * A->cols][ldc >= B->cols].  An empty
 *    expert gets C_e = 0 (or is left unchanged when accumulating).
 * Q2D_EUNSUPPORTED when a code buffer the GEMM reads spans more than 4 GiB.
 */
q2d_status q2d_grouped_gemm(const q2d_tensor *A, int transA, const q2d_tensor *B, int transB,
                            int32_t nseg, const int64_t *seg_offsets, int64_t total_rows, void *C,
                            q2d_dtype c_dt, int64_t ldc, int accumulate, hipStream_t stream);

/* Static description of a status code (never NULL). */
const char *q2d_status_string(q2d_status s);

#ifdef __cplusplus
}
#endif
#endif /* Q2D_H */
