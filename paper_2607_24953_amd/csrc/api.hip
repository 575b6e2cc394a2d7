// C ABI of libq2d: argument validation, layout arithmetic and launches on the
// caller's stream.  No allocation, no synchronization, no printing.
#include "q2d.h"
#include "kernels.hpp"

#include <initializer_list>
#include <stdint.h>

namespace {

using namespace q2d;

constexpr int64_t kPadK = 128;     // K extents are padded to the GEMM K-tile

inline int64_t rup(int64_t a, int64_t m) { return (a + m - 1) / m * m; }
inline int64_t cdiv(int64_t a, int64_t m) { return (a + m - 1) / m; }
inline bool aligned(const void *p, uintptr_t n) { return (reinterpret_cast<uintptr_t>(p) % n) == 0; }

struct Layout {
    int64_t ld_codes, ld_codes_t, ld_scales, ld_scales_t;
    int64_t rows_codes, rows_codes_t, rows_scales, rows_scales_t;
};

Layout layout_of(q2d_fmt fmt, int64_t R, int64_t C)
{
    Layout l;
    if (fmt == Q2D_FMT_FP4_2D) {
        l.ld_codes = rup(C, kPadK) / 2;   l.rows_codes = R;
        l.ld_codes_t = rup(R, kPadK) / 2; l.rows_codes_t = C;
        l.ld_scales = rup(C, kPadK) / 32; l.rows_scales = cdiv(R, 32);
        l.ld_scales_t = rup(R, kPadK) / 32; l.rows_scales_t = cdiv(C, 32);
    } else if (fmt == Q2D_FMT_FP4_1D) {
        // scales: one 4-byte word per row and K-tile, K-tile major
        l.ld_codes = rup(C, kPadK) / 2;   l.rows_codes = R;
        l.ld_codes_t = rup(R, kPadK) / 2; l.rows_codes_t = C;
        l.ld_scales = 4 * R;              l.rows_scales = rup(C, kPadK) / kPadK;
        l.ld_scales_t = 4 * C;            l.rows_scales_t = rup(R, kPadK) / kPadK;
    } else {
        l.ld_codes = rup(C, kPadK);       l.rows_codes = R;
        l.ld_codes_t = rup(R, kPadK);     l.rows_codes_t = C;
        l.ld_scales = rup(C, kPadK) / 32; l.rows_scales = R;
        l.ld_scales_t = rup(R, kPadK) / 32; l.rows_scales_t = C;
    }
    return l;
}

bool valid_dtype(q2d_dtype d) { return d == Q2D_F32 || d == Q2D_BF16; }
int dtype_bytes(q2d_dtype d) { return d == Q2D_F32 ? 4 : 2; }

// Check one orientation's buffers against the minimal layout.
bool check_pair(const uint8_t *codes, int64_t ldc, int64_t min_ldc, const uint8_t *scales,
                int64_t lds, int64_t min_lds)
{
    if (!codes) return true;
    if (!scales) return false;
    if (ldc < min_ldc || (ldc % 16) != 0 || lds < min_lds || (lds % 4) != 0) return false;
    return aligned(codes, 16) && aligned(scales, 4);
}

q2d_status check_tensor(const q2d_tensor *t, q2d_fmt fmt, int64_t R, int64_t C)
{
    if (!t) return Q2D_EINVAL;
    if (t->fmt != fmt || t->rows != R || t->cols != C) return Q2D_EINVAL;
    if (t->block != 32 && !(t->block == 64 && fmt == Q2D_FMT_FP4_2D)) return Q2D_EUNSUPPORTED;
    if (!t->codes && !t->codes_t) return Q2D_EINVAL;
    const Layout l = layout_of(fmt, R, C);
    if (!check_pair(t->codes, t->ld_codes, l.ld_codes, t->scales, t->ld_scales, l.ld_scales)) return Q2D_EINVAL;
    if (!check_pair(t->codes_t, t->ld_codes_t, l.ld_codes_t, t->scales_t, t->ld_scales_t, l.ld_scales_t))
        return Q2D_EINVAL;
    return Q2D_OK;
}

// Build launch arguments; a transposed view (stride_r == 1) is quantized as its
// row-major storage with the two orientations swapped, which leaves every
// element's storage index, block and scale unchanged.
QuantArgs make_quant_args(const void *x, int64_t R, int64_t C, int64_t sr, int64_t sc,
                          uint64_t seed, uint64_t offset, const q2d_tensor *t)
{
    QuantArgs a;
    const bool swap = (sc != 1 && sr == 1);
    a.x = x;
    a.index_base = 0;
    a.seed = seed;
    a.offset = offset;
    if (!swap) {
        a.rows = R; a.cols = C; a.stride_r = sr; a.stride_c = sc;
        a.codes = t->codes;       a.ld_codes = t->ld_codes;
        a.codes_t = t->codes_t;   a.ld_codes_t = t->ld_codes_t;
        a.scales = t->scales;     a.ld_scales = t->ld_scales;
        a.scales_t = t->scales_t; a.ld_scales_t = t->ld_scales_t;
    } else {
        a.rows = C; a.cols = R; a.stride_r = sc; a.stride_c = sr;
        a.codes = t->codes_t;     a.ld_codes = t->ld_codes_t;
        a.codes_t = t->codes;     a.ld_codes_t = t->ld_codes;
        a.scales = t->scales_t;   a.ld_scales = t->ld_scales_t;
        a.scales_t = t->scales;   a.ld_scales_t = t->ld_scales;
    }
    a.rows_pad = rup(a.rows, 128);
    a.cols_pad = rup(a.cols, 128);
    a.nbr = cdiv(a.rows, 32);
    a.nbc = cdiv(a.cols, 32);
    a.seg_offsets = nullptr;
    a.nseg = 0;
    a.store_rows = a.rows;
    a.block = 32;
    a.floor_scale = 0;
    return a;
}

// Padded row capacity of a grouped tensor: every segment starts on a 128-row
// boundary, so sum_e roundup(n_e, 128) <= rows + 127 * nseg.
int64_t grouped_capacity(int64_t rows, int32_t nseg) { return rup(rows + 127 * (int64_t)nseg, 128); }

// The kernels hold segment offsets and padded row starts in 32-bit integers.
constexpr int64_t kMaxGroupedRows = INT32_MAX;

constexpr int32_t kMaxGroups = 1024;

// Matrix extents: positive, and at most 2^31 per dimension, which keeps every
// layout product and padded size far from int64 overflow.
constexpr int64_t kMaxDim = int64_t(1) << 31;

q2d_status check_dims(int64_t R, int64_t C)
{
    if (R <= 0 || C <= 0) return Q2D_EINVAL;
    if (R > kMaxDim || C > kMaxDim) return Q2D_EUNSUPPORTED;
    return Q2D_OK;
}

// The largest storage index a strided view reaches, (R-1) sr + (C-1) sc, must
// stay below 2^47 elements (the kernels form it in 64-bit arithmetic).
constexpr int64_t kMaxIndex = int64_t(1) << 47;

q2d_status check_input(const void *x, q2d_dtype dt, int64_t R, int64_t C, int64_t sr, int64_t sc)
{
    if (!x || !valid_dtype(dt) || sr <= 0 || sc <= 0) return Q2D_EINVAL;
    q2d_status s = check_dims(R, C);
    if (s != Q2D_OK) return s;
    if (!aligned(x, (uintptr_t)dtype_bytes(dt))) return Q2D_EINVAL;
    int64_t a, b, last;
    if (__builtin_mul_overflow(R - 1, sr, &a) || __builtin_mul_overflow(C - 1, sc, &b) ||
        __builtin_add_overflow(a, b, &last) || last >= kMaxIndex)
        return Q2D_EUNSUPPORTED;
    return Q2D_OK;
}

}  // namespace

extern "C" {

q2d_status q2d_tensor_init(q2d_tensor *t, q2d_fmt fmt, int64_t rows, int64_t cols, int32_t block,
                           int64_t bytes[4])
{
    if (!t) return Q2D_EINVAL;
    const q2d_status s = check_dims(rows, cols);
    if (s != Q2D_OK) return s;
    if (fmt != Q2D_FMT_FP4_2D && fmt != Q2D_FMT_MXFP8 && fmt != Q2D_FMT_FP4_1D) return Q2D_EINVAL;
    // 64 x 64 blocks keep the 32-granular scale grid (each block's byte in its
    // four entries), so every GEMM reads them unchanged
    if (block != 32 && !(block == 64 && fmt == Q2D_FMT_FP4_2D)) return Q2D_EUNSUPPORTED;
    const Layout l = layout_of(fmt, rows, cols);
    t->fmt = fmt; t->block = block; t->rows = rows; t->cols = cols;
    t->codes = t->codes_t = t->scales = t->scales_t = nullptr;
    t->ld_codes = l.ld_codes; t->ld_codes_t = l.ld_codes_t;
    t->ld_scales = l.ld_scales; t->ld_scales_t = l.ld_scales_t;
    if (bytes) {
        bytes[0] = l.ld_codes * l.rows_codes;
        bytes[1] = l.ld_codes_t * l.rows_codes_t;
        bytes[2] = l.ld_scales * l.rows_scales;
        bytes[3] = l.ld_scales_t * l.rows_scales_t;
    }
    return Q2D_OK;
}

// The entry points below check every argument before they launch; with
// go == false they only check (the composite linear-layer calls check all of
// their steps before the first launch).
static q2d_status quantize_impl(const void *x, q2d_dtype dt, int64_t rows, int64_t cols, int64_t stride_r,
                                int64_t stride_c, int32_t block, q2d_round mode, uint64_t seed, uint64_t offset,
                                q2d_tensor *out, hipStream_t stream, bool go)
{
    q2d_status s = check_input(x, dt, rows, cols, stride_r, stride_c);
    if (s != Q2D_OK) return s;
    const int rmode = (int)mode & ~Q2D_FLOOR_SCALE;
    if (rmode != Q2D_RTN && rmode != Q2D_SR) return Q2D_EINVAL;
    if (block != 32 && block != 64) return Q2D_EUNSUPPORTED;
    s = check_tensor(out, Q2D_FMT_FP4_2D, rows, cols);
    if (s != Q2D_OK) return s;
    if (out->block != block) return Q2D_EINVAL;
    QuantArgs a = make_quant_args(x, rows, cols, stride_r, stride_c, seed, offset, out);
    a.block = block;
    a.floor_scale = ((int)mode & Q2D_FLOOR_SCALE) != 0;
    if (go && launch_fp4_quantize(a, dtype_bytes(dt), rmode == Q2D_SR, false, stream) != hipSuccess)
        return Q2D_ELAUNCH;
    return Q2D_OK;
}

q2d_status q2d_quantize(const void *x, q2d_dtype dt, int64_t rows, int64_t cols, int64_t stride_r,
                        int64_t stride_c, int32_t block, q2d_round mode, uint64_t seed,
                        uint64_t offset, q2d_tensor *out, hipStream_t stream)
{
    return quantize_impl(x, dt, rows, cols, stride_r, stride_c, block, mode, seed, offset, out, stream, true);
}

static q2d_status quantize_1d_impl(const void *x, q2d_dtype dt, int64_t rows, int64_t cols, int64_t stride_r,
                                   int64_t stride_c, int32_t block, q2d_round mode, uint64_t seed, uint64_t offset,
                                   q2d_tensor *out, hipStream_t stream, bool go)
{
    q2d_status s = check_input(x, dt, rows, cols, stride_r, stride_c);
    if (s != Q2D_OK) return s;
    if ((int)mode & Q2D_FLOOR_SCALE) return Q2D_EUNSUPPORTED;     // the ablation rule is 2D only
    if (mode != Q2D_RTN && mode != Q2D_SR) return Q2D_EINVAL;
    if (block != 32) return Q2D_EUNSUPPORTED;
    s = check_tensor(out, Q2D_FMT_FP4_1D, rows, cols);
    if (s != Q2D_OK) return s;
    if (out->block != 32) return Q2D_EUNSUPPORTED;
    // a transposed view's rowwise blocks are its storage's column blocks: the
    // swap of make_quant_args sends each copy to the right buffers
    const QuantArgs a = make_quant_args(x, rows, cols, stride_r, stride_c, seed, offset, out);
    if (go && launch_fp4_quantize(a, dtype_bytes(dt), mode == Q2D_SR, true, stream) != hipSuccess)
        return Q2D_ELAUNCH;
    return Q2D_OK;
}

q2d_status q2d_quantize_1d(const void *x, q2d_dtype dt, int64_t rows, int64_t cols, int64_t stride_r,
                           int64_t stride_c, int32_t block, q2d_round mode, uint64_t seed, uint64_t offset,
                           q2d_tensor *out, hipStream_t stream)
{
    return quantize_1d_impl(x, dt, rows, cols, stride_r, stride_c, block, mode, seed, offset, out, stream, true);
}

q2d_status mxfp8_quantize(const void *x, q2d_dtype dt, int64_t rows, int64_t cols, int64_t stride_r,
                          int64_t stride_c, q2d_tensor *out, hipStream_t stream)
{
    q2d_status s = check_input(x, dt, rows, cols, stride_r, stride_c);
    if (s != Q2D_OK) return s;
    s = check_tensor(out, Q2D_FMT_MXFP8, rows, cols);
    if (s != Q2D_OK) return s;
    // The two MXFP8 copies use different block directions, so a transposed
    // view is not a relabelling of its storage: always read element-wise.
    QuantArgs a;
    a.x = x; a.rows = rows; a.cols = cols; a.stride_r = stride_r; a.stride_c = stride_c;
    a.index_base = 0; a.seed = 0; a.offset = 0;
    a.codes = out->codes;       a.ld_codes = out->ld_codes;
    a.codes_t = out->codes_t;   a.ld_codes_t = out->ld_codes_t;
    a.scales = out->scales;     a.ld_scales = out->ld_scales;
    a.scales_t = out->scales_t; a.ld_scales_t = out->ld_scales_t;
    a.rows_pad = rup(rows, 128); a.cols_pad = rup(cols, 128);
    a.nbr = rows; a.nbc = cols;
    a.seg_offsets = nullptr; a.nseg = 0; a.store_rows = rows; a.block = 32;
    if (launch_mxfp8_quantize(a, dtype_bytes(dt), stream) != hipSuccess) return Q2D_ELAUNCH;
    return Q2D_OK;
}

// Operands of a GEMM C = op(A) op(B)^T into g (codes, scales, M, N, padded K,
// 1D flags); fp4 tells the FP4 pairing from the MXFP8 one.
static q2d_status gemm_operands(const q2d_tensor *A, int transA, const q2d_tensor *B, int transB, GemmArgs &g, bool &fp4)
{
    if (!A || !B) return Q2D_EINVAL;
    if ((transA != 0 && transA != 1) || (transB != 0 && transB != 1)) return Q2D_EINVAL;
    // FP4 operands may mix 2D and 1D blocks (activations); MXFP8 pairs with MXFP8
    const bool fp4a = A->fmt == Q2D_FMT_FP4_2D || A->fmt == Q2D_FMT_FP4_1D;
    const bool fp4b = B->fmt == Q2D_FMT_FP4_2D || B->fmt == Q2D_FMT_FP4_1D;
    if (!(fp4a && fp4b) && !(A->fmt == Q2D_FMT_MXFP8 && B->fmt == Q2D_FMT_MXFP8)) return Q2D_EINVAL;
    // FP4_2D operands may have 64 x 64 blocks (scales stored 32-granular)
    auto block_ok = [](const q2d_tensor *t) {
        return t->block == 32 || (t->block == 64 && t->fmt == Q2D_FMT_FP4_2D);
    };
    if (!block_ok(A) || !block_ok(B)) return Q2D_EUNSUPPORTED;
    q2d_status s = check_dims(A->rows, A->cols);
    if (s == Q2D_OK) s = check_dims(B->rows, B->cols);
    if (s != Q2D_OK) return s;
    const int64_t M = transA ? A->cols : A->rows, Ka = transA ? A->rows : A->cols;
    const int64_t N = transB ? B->cols : B->rows, Kb = transB ? B->rows : B->cols;
    if (Ka != Kb) return Q2D_EINVAL;
    const Layout la = layout_of((q2d_fmt)A->fmt, A->rows, A->cols), lb = layout_of((q2d_fmt)B->fmt, B->rows, B->cols);
    g = GemmArgs{};
    g.a1d = A->fmt == Q2D_FMT_FP4_1D;
    g.b1d = B->fmt == Q2D_FMT_FP4_1D;
    if (!transA) {
        if (!check_pair(A->codes, A->ld_codes, la.ld_codes, A->scales, A->ld_scales, la.ld_scales) || !A->codes)
            return Q2D_EINVAL;
        g.a = A->codes; g.lda = A->ld_codes; g.sa = A->scales; g.ldsa = A->ld_scales;
    } else {
        if (!check_pair(A->codes_t, A->ld_codes_t, la.ld_codes_t, A->scales_t, A->ld_scales_t, la.ld_scales_t) ||
            !A->codes_t)
            return Q2D_EINVAL;
        g.a = A->codes_t; g.lda = A->ld_codes_t; g.sa = A->scales_t; g.ldsa = A->ld_scales_t;
    }
    if (!transB) {
        if (!check_pair(B->codes, B->ld_codes, lb.ld_codes, B->scales, B->ld_scales, lb.ld_scales) || !B->codes)
            return Q2D_EINVAL;
        g.b = B->codes; g.ldb = B->ld_codes; g.sb = B->scales; g.ldsb = B->ld_scales;
    } else {
        if (!check_pair(B->codes_t, B->ld_codes_t, lb.ld_codes_t, B->scales_t, B->ld_scales_t, lb.ld_scales_t) ||
            !B->codes_t)
            return Q2D_EINVAL;
        g.b = B->codes_t; g.ldb = B->ld_codes_t; g.sb = B->scales_t; g.ldsb = B->ld_scales_t;
    }
    g.M = M; g.N = N; g.K = rup(Ka, kPadK);
    fp4 = fp4a;
    return Q2D_OK;
}

static q2d_status gemm_impl(const q2d_tensor *A, int transA, const q2d_tensor *B, int transB, void *C,
                            q2d_dtype c_dt, int64_t ldc, int accumulate, hipStream_t stream, bool go)
{
    if (!A || !B || !C || !valid_dtype(c_dt)) return Q2D_EINVAL;
    if (accumulate != 0 && accumulate != 1) return Q2D_EINVAL;
    GemmArgs g;
    bool fp4 = false;
    const q2d_status s = gemm_operands(A, transA, B, transB, g, fp4);
    if (s != Q2D_OK) return s;
    if (ldc < g.N) return Q2D_EINVAL;
    if (!aligned(C, (uintptr_t)dtype_bytes(c_dt))) return Q2D_EINVAL;
    g.c = C; g.ldc = ldc;
    g.accumulate = accumulate;
    if (go && launch_gemm(g, fp4 ? kFmtFp4Block2D : kFmtMxfp8, c_dt == Q2D_BF16, stream) != hipSuccess)
        return Q2D_ELAUNCH;
    return Q2D_OK;
}

q2d_status q2d_gemm(const q2d_tensor *A, int transA, const q2d_tensor *B, int transB, void *C,
                    q2d_dtype c_dt, int64_t ldc, int accumulate, hipStream_t stream)
{
    return gemm_impl(A, transA, B, transB, C, c_dt, ldc, accumulate, stream, true);
}

q2d_status q2d_gemm_quantized(const q2d_tensor *A, int transA, const q2d_tensor *B, int transB, q2d_round mode,
                              uint64_t seed, uint64_t offset, q2d_tensor *out, hipStream_t stream)
{
    if (!A || !B || !out) return Q2D_EINVAL;
    if (mode != Q2D_RTN && mode != Q2D_SR) return Q2D_EINVAL;
    GemmArgs g;
    bool fp4 = false;
    q2d_status s = gemm_operands(A, transA, B, transB, g, fp4);
    if (s != Q2D_OK) return s;
    if (!fp4) return Q2D_EUNSUPPORTED;
    s = check_tensor(out, Q2D_FMT_FP4_2D, g.M, g.N);
    if (s != Q2D_OK) return s;
    if (out->block != 32) return Q2D_EUNSUPPORTED;
    if (!out->codes || !out->codes_t) return Q2D_EINVAL;
    // stochastic rounding: the Philox blocks of 8 storage indices stay inside one row
    if (mode == Q2D_SR && (g.N % 8) != 0) return Q2D_EUNSUPPORTED;
    g.qsr = mode == Q2D_SR;
    g.seed = seed;
    g.offset = offset;
    // the epilogue stores 8-byte runs of codes_t
    if (!aligned(out->codes_t, 16) || (out->ld_codes_t % 16) != 0) return Q2D_EINVAL;
    g.qc = out->codes; g.ldqc = out->ld_codes;
    g.qct = out->codes_t; g.ldqct = out->ld_codes_t;
    g.qs = out->scales; g.ldqs = out->ld_scales;
    g.qst = out->scales_t; g.ldqst = out->ld_scales_t;
    if (g.M * g.lda > (int64_t(1) << 32) || g.N * g.ldb > (int64_t(1) << 32)) return Q2D_EUNSUPPORTED;
    if (launch_gemm_quantized(g, stream) != hipSuccess) return Q2D_ELAUNCH;
    return Q2D_OK;
}

q2d_status q2d_linear_fwd(const void *X, const void *W, q2d_dtype dt, int64_t T, int64_t N, int64_t K,
                          q2d_round mode_x, q2d_round mode_w, uint64_t seed, uint64_t offset_x,
                          uint64_t offset_w, q2d_tensor *qX, q2d_tensor *qW, void *Y, q2d_dtype y_dt,
                          hipStream_t stream)
{
    if (!qX || !qW || !qX->codes || !qW->codes) return Q2D_EINVAL;
    // every step is checked (go = false) before the first one is launched
    for (const bool go : {false, true}) {
        q2d_status s = qX->fmt == Q2D_FMT_FP4_1D
                           ? quantize_1d_impl(X, dt, T, K, K, 1, 32, mode_x, seed, offset_x, qX, stream, go)
                           : quantize_impl(X, dt, T, K, K, 1, qX->block, mode_x, seed, offset_x, qX, stream, go);
        if (s == Q2D_OK) s = quantize_impl(W, dt, N, K, K, 1, qW->block, mode_w, seed, offset_w, qW, stream, go);
        if (s == Q2D_OK) s = gemm_impl(qX, 0, qW, 0, Y, y_dt, N, 0, stream, go);
        if (s != Q2D_OK) return s;
    }
    return Q2D_OK;
}

q2d_status q2d_linear_bwd(const void *dY, q2d_dtype dt, const q2d_tensor *qX, const q2d_tensor *qW,
                          q2d_round mode_dy, uint64_t seed, uint64_t offset_dy, q2d_tensor *qdY, void *dX,
                          q2d_dtype dx_dt, void *dW, q2d_dtype dw_dt, int accumulate_dw, hipStream_t stream)
{
    if (!qX || !qW || !qdY) return Q2D_EINVAL;
    const int64_t T = qX->rows, K = qX->cols, N = qW->rows;
    if (qW->cols != K || qdY->rows != T || qdY->cols != N) return Q2D_EINVAL;
    if (!qdY->codes || !qdY->codes_t || !qX->codes_t || !qW->codes_t) return Q2D_EINVAL;
    for (const bool go : {false, true}) {
        q2d_status s = quantize_impl(dY, dt, T, N, N, 1, qdY->block, mode_dy, seed, offset_dy, qdY, stream, go);
        if (s == Q2D_OK) s = gemm_impl(qdY, 0, qW, 1, dX, dx_dt, K, 0, stream, go);
        if (s == Q2D_OK) s = gemm_impl(qdY, 1, qX, 1, dW, dw_dt, K, accumulate_dw, stream, go);
        if (s != Q2D_OK) return s;
    }
    return Q2D_OK;
}

q2d_status q2d_grouped_tensor_init(q2d_tensor *t, int64_t rows, int64_t cols, int32_t nseg, int32_t block,
                                   int64_t bytes[4])
{
    if (nseg <= 0 || nseg > kMaxGroups) return Q2D_EINVAL;
    const q2d_status s = check_dims(rows, cols);
    if (s != Q2D_OK) return s;
    if (block != 32) return Q2D_EUNSUPPORTED;
    if (grouped_capacity(rows, nseg) > kMaxGroupedRows) return Q2D_EUNSUPPORTED;
    return q2d_tensor_init(t, Q2D_FMT_FP4_2D, grouped_capacity(rows, nseg), cols, block, bytes);
}

q2d_status q2d_grouped_quantize(const void *x, q2d_dtype dt, int64_t rows, int64_t cols, int64_t stride_r,
                                int32_t nseg, const int64_t *seg_offsets, int32_t block, q2d_round mode,
                                uint64_t seed, uint64_t offset, q2d_tensor *out, hipStream_t stream)
{
    if (!seg_offsets || nseg <= 0 || nseg > kMaxGroups) return Q2D_EINVAL;
    if (!aligned(seg_offsets, 8)) return Q2D_EINVAL;
    q2d_status s = check_input(x, dt, rows > 0 ? rows : 1, cols, stride_r, 1);
    if (s != Q2D_OK) return s;
    if (rows <= 0 || stride_r < cols) return Q2D_EINVAL;
    const int rmode = (int)mode & ~Q2D_FLOOR_SCALE;
    if (rmode != Q2D_RTN && rmode != Q2D_SR) return Q2D_EINVAL;
    if (block != 32) return Q2D_EUNSUPPORTED;
    const int64_t cap = grouped_capacity(rows, nseg);
    if (cap > kMaxGroupedRows) return Q2D_EUNSUPPORTED;
    s = check_tensor(out, Q2D_FMT_FP4_2D, cap, cols);
    if (s != Q2D_OK) return s;
    if (out->block != 32) return Q2D_EUNSUPPORTED;
    QuantArgs a = make_quant_args(x, rows, cols, stride_r, 1, seed, offset, out);
    a.rows_pad = cap;               // grid bound over padded rows
    a.seg_offsets = seg_offsets;
    a.nseg = nseg;
    a.floor_scale = ((int)mode & Q2D_FLOOR_SCALE) != 0;
    if (launch_fp4_quantize(a, dtype_bytes(dt), rmode == Q2D_SR, false, stream) != hipSuccess) return Q2D_ELAUNCH;
    return Q2D_OK;
}

q2d_status q2d_grouped_gemm(const q2d_tensor *A, int transA, const q2d_tensor *B, int transB, int32_t nseg,
                            const int64_t *seg_offsets, int64_t total_rows, void *C, q2d_dtype c_dt,
                            int64_t ldc, int accumulate, hipStream_t stream)
{
    if (!A || !B || !C || !seg_offsets || !valid_dtype(c_dt)) return Q2D_EINVAL;
    if (nseg <= 0 || nseg > kMaxGroups || total_rows <= 0 || !aligned(seg_offsets, 8)) return Q2D_EINVAL;
    if ((transA != 0 && transA != 1) || (transB != 0 && transB != 1)) return Q2D_EINVAL;
    if (accumulate != 0 && accumulate != 1) return Q2D_EINVAL;
    if (A->fmt != Q2D_FMT_FP4_2D || B->fmt != Q2D_FMT_FP4_2D) return Q2D_EUNSUPPORTED;
    if (A->block != 32 || B->block != 32) return Q2D_EUNSUPPORTED;
    if (!aligned(C, (uintptr_t)dtype_bytes(c_dt))) return Q2D_EINVAL;
    q2d_status s = check_dims(A->rows, A->cols);
    if (s == Q2D_OK) s = check_dims(B->rows, B->cols);
    if (s == Q2D_OK && total_rows > kMaxDim) s = Q2D_EUNSUPPORTED;
    if (s != Q2D_OK) return s;
    const int64_t cap = grouped_capacity(total_rows, nseg);
    if (cap > kMaxGroupedRows) return Q2D_EUNSUPPORTED;
    const Layout la = layout_of(Q2D_FMT_FP4_2D, A->rows, A->cols), lb = layout_of(Q2D_FMT_FP4_2D, B->rows, B->cols);
    GemmArgs g = {};
    g.a1d = g.b1d = 0;
    GroupedArgs gr;
    gr.seg_offsets = seg_offsets;
    gr.nseg = nseg;
    gr.total_rows = total_rows;
    gr.b_group_rows = 0;
    gr.b_group_k = 0;
    if (A->rows != cap) return Q2D_EINVAL;
    if (!transA) {
        // ragged M: grouped A rows times expert e's slice of the stacked op(B)
        gr.ragged_k = 0;
        if (!A->codes || !check_pair(A->codes, A->ld_codes, la.ld_codes, A->scales, A->ld_scales, la.ld_scales))
            return Q2D_EINVAL;
        const int64_t K = A->cols;
        int64_t N;
        if (!transB) {
            if (B->cols != K || B->rows % nseg != 0) return Q2D_EINVAL;
            N = B->rows / nseg;
            if (N % 32 != 0) return Q2D_EUNSUPPORTED;
            if (!B->codes || !check_pair(B->codes, B->ld_codes, lb.ld_codes, B->scales, B->ld_scales, lb.ld_scales))
                return Q2D_EINVAL;
            g.b = B->codes; g.ldb = B->ld_codes; g.sb = B->scales; g.ldsb = B->ld_scales;
            gr.b_group_rows = N;
        } else {
            if (B->rows != (int64_t)nseg * K) return Q2D_EINVAL;
            if (K % 128 != 0) return Q2D_EUNSUPPORTED;
            N = B->cols;
            if (!B->codes_t ||
                !check_pair(B->codes_t, B->ld_codes_t, lb.ld_codes_t, B->scales_t, B->ld_scales_t, lb.ld_scales_t))
                return Q2D_EINVAL;
            g.b = B->codes_t; g.ldb = B->ld_codes_t; g.sb = B->scales_t; g.ldsb = B->ld_scales_t;
            gr.b_group_k = K;
        }
        if (ldc < N) return Q2D_EINVAL;
        g.a = A->codes; g.lda = A->ld_codes; g.sa = A->scales; g.ldsa = A->ld_scales;
        g.M = total_rows; g.N = N; g.K = rup(K, kPadK);
    } else {
        // ragged K: per-expert products of the transposed grouped operands
        gr.ragged_k = 1;
        if (!transB || B->rows != cap) return Q2D_EINVAL;
        if (!A->codes_t ||
            !check_pair(A->codes_t, A->ld_codes_t, la.ld_codes_t, A->scales_t, A->ld_scales_t, la.ld_scales_t))
            return Q2D_EINVAL;
        if (!B->codes_t ||
            !check_pair(B->codes_t, B->ld_codes_t, lb.ld_codes_t, B->scales_t, B->ld_scales_t, lb.ld_scales_t))
            return Q2D_EINVAL;
        if (ldc < B->cols) return Q2D_EINVAL;
        g.a = A->codes_t; g.lda = A->ld_codes_t; g.sa = A->scales_t; g.ldsa = A->ld_scales_t;
        g.b = B->codes_t; g.ldb = B->ld_codes_t; g.sb = B->scales_t; g.ldsb = B->ld_scales_t;
        g.M = A->cols; g.N = B->cols; g.K = 0;
    }
    // the grouped kernel addresses each operand with 32-bit byte offsets
    const int64_t lim = int64_t(1) << 32;
    if ((transA ? A->cols : A->rows) * g.lda > lim || (transB ? B->cols : B->rows) * g.ldb > lim)
        return Q2D_EUNSUPPORTED;
    g.c = C; g.ldc = ldc; g.accumulate = accumulate;
    if (launch_grouped_gemm(g, gr, c_dt == Q2D_BF16, stream) != hipSuccess) return Q2D_ELAUNCH;
    return Q2D_OK;
}

q2d_status q2d_dequantize(const q2d_tensor *t, int copy, void *out, q2d_dtype out_dt, int64_t ldo,
                          int8_t *exps, int64_t lde, hipStream_t stream)
{
    if (!t || !out || (copy != 0 && copy != 1) || !valid_dtype(out_dt)) return Q2D_EINVAL;
    if (t->fmt != Q2D_FMT_FP4_2D && t->fmt != Q2D_FMT_MXFP8 && t->fmt != Q2D_FMT_FP4_1D) return Q2D_EINVAL;
    if (t->block != 32 && !(t->block == 64 && t->fmt == Q2D_FMT_FP4_2D)) return Q2D_EUNSUPPORTED;
    const q2d_status s = check_dims(t->rows, t->cols);
    if (s != Q2D_OK) return s;
    if (ldo < t->cols || (exps && lde < t->cols)) return Q2D_EINVAL;
    const Layout l = layout_of((q2d_fmt)t->fmt, t->rows, t->cols);
    const uint8_t *codes = copy ? t->codes_t : t->codes;
    const uint8_t *scales = copy ? t->scales_t : t->scales;
    const int64_t ldc = copy ? t->ld_codes_t : t->ld_codes, lds = copy ? t->ld_scales_t : t->ld_scales;
    if (!codes || !check_pair(codes, ldc, copy ? l.ld_codes_t : l.ld_codes, scales, lds,
                              copy ? l.ld_scales_t : l.ld_scales))
        return Q2D_EINVAL;
    const int eb = dtype_bytes(out_dt);
    DequantArgs a;
    a.codes = codes; a.ld_codes = ldc;
    a.scales = scales; a.ld_scales = lds;
    a.rows = t->rows; a.cols = t->cols;
    a.fmt = t->fmt == Q2D_FMT_FP4_2D ? 0 : (t->fmt == Q2D_FMT_MXFP8 ? 1 : 2);
    a.transposed = copy;
    a.out = out; a.ldo = ldo;
    a.out_bf16 = out_dt == Q2D_BF16;
    a.out_vec = aligned(out, 4 * eb) && (ldo % 4) == 0;
    a.exps = exps; a.lde = lde;
    if (launch_dequantize(a, stream) != hipSuccess) return Q2D_ELAUNCH;
    return Q2D_OK;
}

const char *q2d_status_string(q2d_status s)
{
    switch (s) {
    case Q2D_OK: return "ok";
    case Q2D_EINVAL: return "invalid argument";
    case Q2D_EUNSUPPORTED: return "unsupported configuration";
    case Q2D_ELAUNCH: return "kernel launch failed";
    }
    return "unknown status";
}

}  // extern "C"
