// Host sanitizer driver for the C ABI's argument checking and layout
// arithmetic (built by tests/test_sanitizers.py: csrc/api.hip compiled for the
// host only with AddressSanitizer and UndefinedBehaviorSanitizer, linked with
// this file).  The kernel launchers are replaced by stubs that record their
// arguments, so no GPU is needed: every entry point runs its checks and builds
// its launch arguments exactly as in the library.  Device pointers are fake,
// suitably aligned addresses that the host code must never dereference
// (AddressSanitizer reports it if it does).
//
// Checked: valid calls reach their launcher with the expected problem sizes;
// invalid ones (null, non-positive, huge or misaligned arguments, mismatched
// operands, bad flags) return the documented status without a launch; and
// no size, however large, makes the host arithmetic overflow.
#include "q2d.h"
#include "kernels.hpp"

#include <stdint.h>
#include <stdio.h>

namespace q2d {
static int g_launches = 0;
static GemmArgs g_gemm;
static QuantArgs g_quant;
hipError_t launch_fp4_quantize(const QuantArgs &a, int, bool, bool, hipStream_t) { ++g_launches; g_quant = a; return hipSuccess; }
hipError_t launch_mxfp8_quantize(const QuantArgs &a, int, hipStream_t) { ++g_launches; g_quant = a; return hipSuccess; }
hipError_t launch_gemm_quantized(const GemmArgs &g, hipStream_t) { ++g_launches; g_gemm = g; return hipSuccess; }
hipError_t launch_gemm(const GemmArgs &g, int, int, hipStream_t) { ++g_launches; g_gemm = g; return hipSuccess; }
hipError_t launch_grouped_gemm(const GemmArgs &g, const GroupedArgs &, int, hipStream_t) { ++g_launches; g_gemm = g; return hipSuccess; }
hipError_t launch_dequantize(const DequantArgs &, hipStream_t) { ++g_launches; return hipSuccess; }
}  // namespace q2d

using q2d::g_launches;

static int failures = 0;
#define CHECK(cond, ...) do { if (!(cond)) { fprintf(stderr, "line %d: ", __LINE__); fprintf(stderr, __VA_ARGS__); fputc('\n', stderr); ++failures; } } while (0)

// a fake device address aligned to 256 bytes
static void *dev(uintptr_t slot) { return reinterpret_cast<void *>(uintptr_t(1) << 40 | slot << 28); }

static q2d_tensor tensor(q2d_fmt fmt, int64_t R, int64_t C, int32_t block, uintptr_t slot)
{
    q2d_tensor t;
    int64_t bytes[4];
    q2d_status s = q2d_tensor_init(&t, fmt, R, C, block, bytes);
    CHECK(s == Q2D_OK, "tensor_init %d %lldx%lld b%d: %d", (int)fmt, (long long)R, (long long)C, block, (int)s);
    t.codes = (uint8_t *)dev(4 * slot);
    t.codes_t = (uint8_t *)dev(4 * slot + 1);
    t.scales = (uint8_t *)dev(4 * slot + 2);
    t.scales_t = (uint8_t *)dev(4 * slot + 3);
    return t;
}

// the status of a call, and whether it launched
#define EXPECT(call, want, launch)                                                                   \
    do {                                                                                           \
        const int before_ = g_launches;                                                            \
        const q2d_status got_ = (call);                                                            \
        CHECK(got_ == (want), "%s: status %d, expected %d", #call, (int)got_, (int)(want));         \
        CHECK((g_launches != before_) == (launch), "%s: launched %d", #call, g_launches - before_); \
    } while (0)

int main()
{
    const hipStream_t st = nullptr;
    const int64_t huge[] = {int64_t(1) << 31 | 1, int64_t(1) << 40, int64_t(1) << 62, INT64_MAX};

    // ---- descriptors and quantization
    for (q2d_fmt f : {Q2D_FMT_FP4_2D, Q2D_FMT_MXFP8, Q2D_FMT_FP4_1D})
        for (int64_t R : {1, 31, 33, 4096, 131072})
            for (int64_t C : {1, 130, 11008}) (void)tensor(f, R, C, 32, 1);
    (void)tensor(Q2D_FMT_FP4_2D, 200, 300, 64, 1);
    q2d_tensor t;
    int64_t bytes[4];
    EXPECT(q2d_tensor_init(nullptr, Q2D_FMT_FP4_2D, 1, 1, 32, bytes), Q2D_EINVAL, false);
    EXPECT(q2d_tensor_init(&t, Q2D_FMT_FP4_2D, 0, 1, 32, bytes), Q2D_EINVAL, false);
    EXPECT(q2d_tensor_init(&t, Q2D_FMT_FP4_2D, 1, -5, 32, bytes), Q2D_EINVAL, false);
    EXPECT(q2d_tensor_init(&t, (q2d_fmt)7, 1, 1, 32, bytes), Q2D_EINVAL, false);
    EXPECT(q2d_tensor_init(&t, Q2D_FMT_FP4_2D, 64, 64, 16, bytes), Q2D_EUNSUPPORTED, false);
    EXPECT(q2d_tensor_init(&t, Q2D_FMT_MXFP8, 64, 64, 64, bytes), Q2D_EUNSUPPORTED, false);
    for (int64_t h : huge) {
        EXPECT(q2d_tensor_init(&t, Q2D_FMT_FP4_2D, h, 64, 32, bytes), Q2D_EUNSUPPORTED, false);
        EXPECT(q2d_tensor_init(&t, Q2D_FMT_FP4_1D, 64, h, 32, bytes), Q2D_EUNSUPPORTED, false);
        EXPECT(q2d_grouped_tensor_init(&t, h, 64, 8, 32, bytes), Q2D_EUNSUPPORTED, false);
    }

    const void *x = dev(60);
    q2d_tensor q = tensor(Q2D_FMT_FP4_2D, 300, 200, 32, 2);
    EXPECT(q2d_quantize(x, Q2D_BF16, 300, 200, 200, 1, 32, Q2D_RTN, 0, 0, &q, st), Q2D_OK, true);
    CHECK(q2d::g_quant.rows == 300 && q2d::g_quant.cols == 200, "quantize sizes");
    EXPECT(q2d_quantize(x, Q2D_F32, 300, 200, 1, 300, 32, Q2D_SR, 1, 2, &q, st), Q2D_OK, true);
    CHECK(q2d::g_quant.rows == 200 && q2d::g_quant.cols == 300, "transposed view is quantized as its storage");
    EXPECT(q2d_quantize(x, Q2D_BF16, 300, 200, 200, 1, 32, (q2d_round)(Q2D_RTN | Q2D_FLOOR_SCALE), 0, 0, &q, st),
           Q2D_OK, true);
    EXPECT(q2d_quantize(nullptr, Q2D_BF16, 300, 200, 200, 1, 32, Q2D_RTN, 0, 0, &q, st), Q2D_EINVAL, false);
    EXPECT(q2d_quantize((const char *)x + 1, Q2D_BF16, 300, 200, 200, 1, 32, Q2D_RTN, 0, 0, &q, st), Q2D_EINVAL, false);
    EXPECT(q2d_quantize(x, Q2D_BF16, 300, 200, 200, 1, 32, (q2d_round)5, 0, 0, &q, st), Q2D_EINVAL, false);
    EXPECT(q2d_quantize(x, Q2D_BF16, 301, 200, 200, 1, 32, Q2D_RTN, 0, 0, &q, st), Q2D_EINVAL, false);
    EXPECT(q2d_quantize(x, Q2D_BF16, 300, 200, 200, 1, 32, Q2D_RTN, 0, 0, nullptr, st), Q2D_EINVAL, false);
    for (int64_t h : huge) {
        EXPECT(q2d_quantize(x, Q2D_BF16, h, 200, 200, 1, 32, Q2D_RTN, 0, 0, &q, st), Q2D_EUNSUPPORTED, false);
        if (h < (int64_t(1) << 40)) continue;
        // strides whose last storage index passes 2^47 elements
        EXPECT(q2d_quantize(x, Q2D_BF16, 300, 200, h, 1, 32, Q2D_RTN, 0, 0, &q, st), Q2D_EUNSUPPORTED, false);
        EXPECT(q2d_quantize(x, Q2D_BF16, 300, 200, 1, h, 32, Q2D_RTN, 0, 0, &q, st), Q2D_EUNSUPPORTED, false);
    }
    q2d_tensor bad = q;
    bad.ld_codes -= 16;
    EXPECT(q2d_quantize(x, Q2D_BF16, 300, 200, 200, 1, 32, Q2D_RTN, 0, 0, &bad, st), Q2D_EINVAL, false);
    bad = q;
    bad.scales = (uint8_t *)bad.scales + 2;
    EXPECT(q2d_quantize(x, Q2D_BF16, 300, 200, 200, 1, 32, Q2D_RTN, 0, 0, &bad, st), Q2D_EINVAL, false);

    q2d_tensor q1 = tensor(Q2D_FMT_FP4_1D, 300, 200, 32, 3);
    EXPECT(q2d_quantize_1d(x, Q2D_BF16, 300, 200, 200, 1, 32, Q2D_SR, 0, 0, &q1, st), Q2D_OK, true);
    EXPECT(q2d_quantize_1d(x, Q2D_BF16, 300, 200, 200, 1, 32, (q2d_round)(Q2D_RTN | Q2D_FLOOR_SCALE), 0, 0, &q1, st),
           Q2D_EUNSUPPORTED, false);
    q2d_tensor q8 = tensor(Q2D_FMT_MXFP8, 300, 200, 32, 4);
    EXPECT(mxfp8_quantize(x, Q2D_F32, 300, 200, 200, 1, &q8, st), Q2D_OK, true);
    EXPECT(mxfp8_quantize(x, Q2D_F32, 300, 200, 200, 1, &q, st), Q2D_EINVAL, false);

    // ---- GEMMs: fwd (X,0,W,0), dX (dY,0,W,1), dW (dY,1,X,1)
    const int64_t T = 1000, N = 700, K = 500;
    q2d_tensor X = tensor(Q2D_FMT_FP4_2D, T, K, 32, 5), W = tensor(Q2D_FMT_FP4_2D, N, K, 32, 6);
    q2d_tensor dY = tensor(Q2D_FMT_FP4_2D, T, N, 32, 7);
    void *C = dev(61);
    EXPECT(q2d_gemm(&X, 0, &W, 0, C, Q2D_F32, N, 0, st), Q2D_OK, true);
    CHECK(q2d::g_gemm.M == T && q2d::g_gemm.N == N && q2d::g_gemm.K == 512, "fwd sizes");
    EXPECT(q2d_gemm(&dY, 0, &W, 1, C, Q2D_BF16, K, 0, st), Q2D_OK, true);
    CHECK(q2d::g_gemm.M == T && q2d::g_gemm.N == K && q2d::g_gemm.K == 768, "dX sizes");
    EXPECT(q2d_gemm(&dY, 1, &X, 1, C, Q2D_F32, K, 1, st), Q2D_OK, true);
    CHECK(q2d::g_gemm.M == N && q2d::g_gemm.N == K && q2d::g_gemm.K == 1024, "dW sizes");
    EXPECT(q2d_gemm(&X, 0, &W, 1, C, Q2D_F32, N, 0, st), Q2D_EINVAL, false);          // K mismatch
    EXPECT(q2d_gemm(&X, 0, &W, 0, C, Q2D_F32, N - 1, 0, st), Q2D_EINVAL, false);      // ldc < N
    EXPECT(q2d_gemm(&X, 2, &W, 0, C, Q2D_F32, N, 0, st), Q2D_EINVAL, false);
    EXPECT(q2d_gemm(&X, 0, &W, 0, C, Q2D_F32, N, 3, st), Q2D_EINVAL, false);
    EXPECT(q2d_gemm(&X, 0, &q8, 0, C, Q2D_F32, N, 0, st), Q2D_EINVAL, false);
    EXPECT(q2d_gemm(nullptr, 0, &W, 0, C, Q2D_F32, N, 0, st), Q2D_EINVAL, false);
    EXPECT(q2d_gemm(&X, 0, &W, 0, (char *)C + 2, Q2D_F32, N, 0, st), Q2D_EINVAL, false);
    q2d_tensor Wrow = W;
    Wrow.codes_t = nullptr;
    Wrow.scales_t = nullptr;
    EXPECT(q2d_gemm(&dY, 0, &Wrow, 1, C, Q2D_BF16, K, 0, st), Q2D_EINVAL, false);     // no column copy
    q2d_tensor Y = tensor(Q2D_FMT_FP4_2D, T, N, 32, 8);
    EXPECT(q2d_gemm_quantized(&X, 0, &W, 0, Q2D_RTN, 0, 0, &Y, st), Q2D_OK, true);
    EXPECT(q2d_gemm_quantized(&X, 0, &W, 0, Q2D_SR, 5, 7, &Y, st), Q2D_EUNSUPPORTED, false);   // N % 8 != 0
    q2d_tensor W8 = tensor(Q2D_FMT_FP4_2D, 704, K, 32, 14), Y8 = tensor(Q2D_FMT_FP4_2D, T, 704, 32, 16);
    EXPECT(q2d_gemm_quantized(&X, 0, &W8, 0, Q2D_SR, 5, 7, &Y8, st), Q2D_OK, true);
    CHECK(q2d::g_gemm.qsr == 1 && q2d::g_gemm.seed == 5 && q2d::g_gemm.offset == 7, "quantized SR stream");
    EXPECT(q2d_gemm_quantized(&X, 0, &W, 0, Q2D_RTN, 5, 7, &Y, st), Q2D_OK, true);
    CHECK(q2d::g_gemm.qsr == 0, "quantized RTN");
    EXPECT(q2d_gemm_quantized(&X, 0, &W, 0, (q2d_round)3, 0, 0, &Y, st), Q2D_EINVAL, false);
    EXPECT(q2d_gemm_quantized(&X, 0, &W, 0, Q2D_RTN, 0, 0, &dY, st), Q2D_OK, true);     // same shape
    EXPECT(q2d_gemm_quantized(&X, 0, &W, 0, Q2D_RTN, 0, 0, &X, st), Q2D_EINVAL, false);

    // ---- linear layer
    q2d_tensor qX = tensor(Q2D_FMT_FP4_2D, T, K, 32, 9), qW = tensor(Q2D_FMT_FP4_2D, N, K, 32, 10);
    q2d_tensor qdY = tensor(Q2D_FMT_FP4_2D, T, N, 32, 11);
    EXPECT(q2d_linear_fwd(x, x, Q2D_BF16, T, N, K, Q2D_RTN, Q2D_RTN, 0, 0, 1, &qX, &qW, C, Q2D_F32, st), Q2D_OK,
           true);
    EXPECT(q2d_linear_bwd(x, Q2D_BF16, &qX, &qW, Q2D_SR, 0, 2, &qdY, C, Q2D_BF16, dev(62), Q2D_F32, 0, st),
           Q2D_OK, true);
    EXPECT(q2d_linear_fwd(x, x, Q2D_BF16, T, N, K + 1, Q2D_RTN, Q2D_RTN, 0, 0, 1, &qX, &qW, C, Q2D_F32, st),
           Q2D_EINVAL, false);
    // a later step's bad argument stops the composite call before its first launch
    EXPECT(q2d_linear_fwd(x, x, Q2D_BF16, T, N, K, Q2D_RTN, Q2D_RTN, 0, 0, 1, &qX, &qW, C, (q2d_dtype)7, st),
           Q2D_EINVAL, false);                                                            // output dtype
    EXPECT(q2d_linear_fwd(x, x, Q2D_BF16, T, N, K, Q2D_RTN, Q2D_RTN, 0, 0, 1, &qX, &qW, (char *)C + 2, Q2D_F32, st),
           Q2D_EINVAL, false);                                                            // misaligned Y
    EXPECT(q2d_linear_fwd(x, x, Q2D_BF16, T, N, K, Q2D_RTN, (q2d_round)9, 0, 0, 1, &qX, &qW, C, Q2D_F32, st),
           Q2D_EINVAL, false);                                                            // W's rounding mode
    q2d_tensor badW = qW;
    badW.ld_codes -= 16;
    EXPECT(q2d_linear_fwd(x, x, Q2D_BF16, T, N, K, Q2D_RTN, Q2D_RTN, 0, 0, 1, &qX, &badW, C, Q2D_F32, st),
           Q2D_EINVAL, false);                                                            // W's layout
    q2d_tensor q8X = tensor(Q2D_FMT_MXFP8, T, K, 32, 13);
    EXPECT(q2d_linear_bwd(x, Q2D_BF16, &q8X, &qW, Q2D_SR, 0, 2, &qdY, C, Q2D_BF16, dev(62), Q2D_F32, 0, st),
           Q2D_EINVAL, false);                                                            // MXFP8 X at the dW GEMM
    EXPECT(q2d_linear_bwd(x, Q2D_BF16, &qX, &qW, Q2D_SR, 0, 2, &qdY, C, Q2D_BF16, dev(62), (q2d_dtype)9, 0, st),
           Q2D_EINVAL, false);                                                            // dW dtype
    EXPECT(q2d_linear_bwd(x, Q2D_BF16, &qX, &qW, Q2D_SR, 0, 2, &qdY, C, Q2D_BF16, dev(62), Q2D_F32, 2, st),
           Q2D_EINVAL, false);                                                            // accumulate flag
    EXPECT(q2d_linear_bwd(x, Q2D_BF16, &qX, &qW, Q2D_SR, 0, 2, &qdY, (char *)C + 1, Q2D_BF16, dev(62), Q2D_F32, 0,
                          st), Q2D_EINVAL, false);                                        // misaligned dX

    // ---- grouped (MoE): 4 experts
    const int32_t E = 4;
    const int64_t rows = 1000;
    q2d_tensor G;
    EXPECT(q2d_grouped_tensor_init(&G, rows, 256, E, 32, bytes), Q2D_OK, false);
    G.codes = (uint8_t *)dev(40); G.codes_t = (uint8_t *)dev(41);
    G.scales = (uint8_t *)dev(42); G.scales_t = (uint8_t *)dev(43);
    const int64_t *offs = (const int64_t *)dev(44);
    EXPECT(q2d_grouped_quantize(x, Q2D_BF16, rows, 256, 256, E, offs, 32, Q2D_RTN, 0, 0, &G, st), Q2D_OK, true);
    EXPECT(q2d_grouped_quantize(x, Q2D_BF16, rows, 256, 256, E, (const int64_t *)((char *)offs + 4), 32, Q2D_RTN,
                                0, 0, &G, st), Q2D_EINVAL, false);
    EXPECT(q2d_grouped_quantize(x, Q2D_BF16, rows, 256, 256, 0, offs, 32, Q2D_RTN, 0, 0, &G, st), Q2D_EINVAL, false);
    EXPECT(q2d_grouped_quantize(x, Q2D_BF16, rows, 256, 256, 5000, offs, 32, Q2D_RTN, 0, 0, &G, st), Q2D_EINVAL,
           false);
    q2d_tensor Wg = tensor(Q2D_FMT_FP4_2D, E * 384, 256, 32, 12);       // stacked [E * N][K]
    EXPECT(q2d_grouped_gemm(&G, 0, &Wg, 0, E, offs, rows, C, Q2D_BF16, 384, 0, st), Q2D_OK, true);
    CHECK(q2d::g_gemm.M == rows && q2d::g_gemm.N == 384 && q2d::g_gemm.K == 256, "grouped fwd sizes");
    q2d_tensor Wd = tensor(Q2D_FMT_FP4_2D, E * 256, 384, 32, 13);       // stacked [E * K][N], read transposed
    EXPECT(q2d_grouped_gemm(&G, 0, &Wd, 1, E, offs, rows, C, Q2D_BF16, 384, 0, st), Q2D_OK, true);
    q2d_tensor Hg;
    EXPECT(q2d_grouped_tensor_init(&Hg, rows, 384, E, 32, bytes), Q2D_OK, false);
    Hg.codes = (uint8_t *)dev(45); Hg.codes_t = (uint8_t *)dev(46);
    Hg.scales = (uint8_t *)dev(47); Hg.scales_t = (uint8_t *)dev(48);
    EXPECT(q2d_grouped_gemm(&Hg, 1, &G, 1, E, offs, rows, C, Q2D_F32, 256, 0, st), Q2D_OK, true);
    EXPECT(q2d_grouped_gemm(&G, 0, &Wg, 0, E, offs, rows + 100000, C, Q2D_BF16, 384, 0, st), Q2D_EINVAL, false);
    for (int64_t h : huge)
        EXPECT(q2d_grouped_gemm(&G, 0, &Wg, 0, E, offs, h, C, Q2D_BF16, 384, 0, st), Q2D_EUNSUPPORTED, false);
    for (int64_t h : huge)
        EXPECT(q2d_grouped_quantize(x, Q2D_BF16, h, 256, 256, E, offs, 32, Q2D_RTN, 0, 0, &G, st), Q2D_EUNSUPPORTED,
               false);
    bad = X;
    bad.cols = INT64_MAX;
    EXPECT(q2d_gemm(&bad, 0, &W, 0, C, Q2D_F32, N, 0, st), Q2D_EUNSUPPORTED, false);
    bad = G;
    bad.rows = int64_t(1) << 62;
    EXPECT(q2d_grouped_gemm(&bad, 0, &Wg, 0, E, offs, rows, C, Q2D_BF16, 384, 0, st), Q2D_EUNSUPPORTED, false);

    // ---- dequantization of either copy
    void *out = dev(63);
    for (int copy = 0; copy < 2; ++copy) {
        EXPECT(q2d_dequantize(&q, copy, out, Q2D_F32, copy ? 300 : 200, (int8_t *)dev(64), copy ? 300 : 200, st),
               Q2D_OK, true);
        EXPECT(q2d_dequantize(&q1, copy, out, Q2D_BF16, copy ? 300 : 200, nullptr, 0, st), Q2D_OK, true);
        EXPECT(q2d_dequantize(&q8, copy, out, Q2D_BF16, copy ? 300 : 200, nullptr, 0, st), Q2D_OK, true);
    }
    EXPECT(q2d_dequantize(&q, 2, out, Q2D_F32, 200, nullptr, 0, st), Q2D_EINVAL, false);
    EXPECT(q2d_dequantize(&q, 0, out, Q2D_F32, 199, nullptr, 0, st), Q2D_EINVAL, false);
    bad = q;
    bad.rows = INT64_MAX;
    EXPECT(q2d_dequantize(&bad, 0, out, Q2D_F32, 200, nullptr, 0, st), Q2D_EUNSUPPORTED, false);

    for (int s = 0; s <= 4; ++s) CHECK(q2d_status_string((q2d_status)s) != nullptr, "status string");

    if (failures) {
        fprintf(stderr, "%d check(s) failed\n", failures);
        return 1;
    }
    printf("sanitize_api: ok\n");
    return 0;
}
