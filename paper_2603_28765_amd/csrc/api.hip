// api.hip -- host side of the C ABI declared in include/ifq.h: argument
// validation (before anything is enqueued) and dispatch to the launchers.
#include <hip/hip_runtime.h>

#include "ifq.h"
#include "launch.h"

namespace {

constexpr uint32_t kKnownFlags =
    IFQ_RHT | IFQ_SR | IFQ_MARGIN_16_17 | IFQ_SCALE_IN | IFQ_AXIS_STRIDED | IFQ_SR_RTN_TYPE;
constexpr int64_t kMaxElems = int64_t(1) << 40;  // keeps every index product in int64

bool valid_format(int f) { return f >= IFQ_FMT_IF4 && f <= IFQ_FMT_NVFP4_BS8; }

int bits_of(int f)
{
    switch (f) {
        case IFQ_FMT_IF3:
        case IFQ_FMT_IF3_BS8: return 3;
        case IFQ_FMT_IF6_E2M3:
        case IFQ_FMT_IF6_E3M2: return 6;
        default: return 4;
    }
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// own_scratch: the partials go to the library's device scratch instead of a
// caller workspace (the allocation-free entry point).
int quantize_impl(int fmt, const void* x, int64_t rows, int64_t cols, int64_t ld_x, uint32_t flags,
                  uint32_t rht_signs, uint64_t seed, uint8_t* codes, uint8_t* scales,
                  float* tensor_scale, void* workspace, size_t workspace_bytes, void* stream,
                  bool own_scratch = false)
{
    if (!valid_format(fmt)) return IFQ_EINVAL;
    if (flags & ~kKnownFlags) return IFQ_EINVAL;
    if (rht_signs > 0xFFFFu) return IFQ_EINVAL;
    if (!tensor_scale) return IFQ_EINVAL;
    if (rows < 0 || cols < 0) return IFQ_ESHAPE;
    if (rows > 0 && cols > 0 && rows > kMaxElems / cols) return IFQ_ESHAPE;
    const bool strided = flags & IFQ_AXIS_STRIDED;
    const int64_t k = strided ? rows : cols;
    if (k % 16) return IFQ_ESHAPE;
    if (!aligned(tensor_scale, 4)) return IFQ_EALIGN;
    const bool empty = rows == 0 || cols == 0;
    if (!empty) {
        if (!x || !codes || !scales) return IFQ_EINVAL;
        if (ld_x < cols) return IFQ_ESHAPE;
        // row-wise groups are read as two 128-bit loads: 16-byte aligned rows;
        // the strided path stages tiles through LDS and takes any alignment
        if (!strided && (!aligned(x, 16) || (ld_x % 8))) return IFQ_EALIGN;
        if (!aligned(x, 2)) return IFQ_EALIGN;
        if (!aligned(codes, 16)) return IFQ_EALIGN;
        if (own_scratch) {
            if (ifq_quantize_workspace_bytes(fmt, rows, cols, flags) > ifq::kScratchBytes)
                return IFQ_EWORKSPACE;
            if (!(flags & IFQ_SCALE_IN)) {
                float* p = nullptr;
                if (ifq::scratch_partials(static_cast<hipStream_t>(stream), &p) != hipSuccess) return IFQ_EHIP;
                workspace = p;
            }
        } else if (!(flags & IFQ_SCALE_IN)) {
            if (!workspace || workspace_bytes < ifq_quantize_workspace_bytes(fmt, rows, cols, flags))
                return IFQ_EWORKSPACE;
            if (!aligned(workspace, 16)) return IFQ_EALIGN;
        }
    }
    ifq::QuantArgs a;
    a.fmt = fmt;
    a.x = static_cast<const uint16_t*>(x);
    a.rows = rows;
    a.cols = cols;
    a.ld = ld_x;
    a.flags = flags;
    a.signs = rht_signs;
    a.seed = seed;
    a.codes = codes;
    a.scales = scales;
    a.tensor_scale = tensor_scale;
    a.partials = static_cast<float*>(workspace);
    return ifq::launch_quantize(a, static_cast<hipStream_t>(stream)) == hipSuccess ? IFQ_OK : IFQ_EHIP;
}

bool dual_format(int f)
{
    return f == IFQ_FMT_IF4 || f == IFQ_FMT_NVFP4 || f == IFQ_FMT_NVINT4 || f == IFQ_FMT_NVFP4_46;
}

int dequantize_impl(int fmt, const uint8_t* codes, const uint8_t* scales, const float* tensor_scale,
                    int64_t rows, int64_t cols, void* out, int out_dtype, void* stream)
{
    if (!valid_format(fmt)) return IFQ_EINVAL;
    if (out_dtype != IFQ_F32 && out_dtype != IFQ_BF16) return IFQ_EINVAL;
    if (rows < 0 || cols < 0) return IFQ_ESHAPE;
    if (cols % 16) return IFQ_ESHAPE;
    if (rows > 0 && cols > 0 && rows > kMaxElems / cols) return IFQ_ESHAPE;
    if (rows == 0 || cols == 0) return IFQ_OK;
    if (!codes || !scales || !tensor_scale || !out) return IFQ_EINVAL;
    if (!aligned(codes, 16) || !aligned(out, 16) || !aligned(tensor_scale, 4)) return IFQ_EALIGN;
    return ifq::launch_dequantize(fmt, codes, scales, tensor_scale, rows, cols, out,
                                  out_dtype == IFQ_BF16, static_cast<hipStream_t>(stream)) == hipSuccess
               ? IFQ_OK
               : IFQ_EHIP;
}

int gemm_impl(int fmt, const uint8_t* a_codes, const uint8_t* a_scales, const float* a_ts,
              const uint8_t* b_codes, const uint8_t* b_scales, const float* b_ts, int64_t M,
              int64_t N, int64_t K, void* c, int64_t ldc, int out_dtype, void* stream)
{
    if (!valid_format(fmt)) return IFQ_EINVAL;
    if (out_dtype != IFQ_F32 && out_dtype != IFQ_BF16) return IFQ_EINVAL;
    if (M < 0 || N < 0 || K < 0) return IFQ_ESHAPE;
    if (K % 16) return IFQ_ESHAPE;
    if ((M > 0 && K > kMaxElems / M) || (N > 0 && K > kMaxElems / N) ||
        (M > 0 && N > 0 && M > kMaxElems / N))
        return IFQ_ESHAPE;
    if (M == 0 || N == 0) return IFQ_OK;
    if (ldc < N) return IFQ_ESHAPE;
    if (!c || !a_ts || !b_ts) return IFQ_EINVAL;
    if (K > 0 && (!a_codes || !a_scales || !b_codes || !b_scales)) return IFQ_EINVAL;
    if (!aligned(a_codes, 16) || !aligned(b_codes, 16) || !aligned(a_ts, 4) || !aligned(b_ts, 4))
        return IFQ_EALIGN;
    if (!aligned(c, out_dtype == IFQ_BF16 ? 2 : 4)) return IFQ_EALIGN;
    ifq::GemmArgs g;
    g.fmt = fmt;
    g.a_codes = a_codes;
    g.a_scales = a_scales;
    g.a_ts = a_ts;
    g.b_codes = b_codes;
    g.b_scales = b_scales;
    g.b_ts = b_ts;
    g.M = M;
    g.N = N;
    g.K = K;
    g.c = c;
    g.ldc = ldc;
    g.out_bf16 = out_dtype == IFQ_BF16;
    return ifq::launch_gemm(g, static_cast<hipStream_t>(stream)) == hipSuccess ? IFQ_OK : IFQ_EHIP;
}

}  // namespace

extern "C" {

int if4_quantize(const void* x, int64_t rows, int64_t cols, int64_t ld_x, uint32_t flags,
                 uint32_t rht_signs, uint64_t seed, uint8_t* codes, uint8_t* scales,
                 float* tensor_scale, void* workspace, size_t workspace_bytes, void* stream)
{
    return quantize_impl(IFQ_FMT_IF4, x, rows, cols, ld_x, flags, rht_signs, seed, codes, scales,
                         tensor_scale, workspace, workspace_bytes, stream);
}

int nvfp4_quantize(const void* x, int64_t rows, int64_t cols, int64_t ld_x, uint32_t flags,
                   uint32_t rht_signs, uint64_t seed, uint8_t* codes, uint8_t* scales,
                   float* tensor_scale, void* workspace, size_t workspace_bytes, void* stream)
{
    return quantize_impl(IFQ_FMT_NVFP4, x, rows, cols, ld_x, flags, rht_signs, seed, codes, scales,
                         tensor_scale, workspace, workspace_bytes, stream);
}

int ifx_quantize(int format, const void* x, int64_t rows, int64_t cols, int64_t ld_x,
                 uint32_t flags, uint32_t rht_signs, uint64_t seed, uint8_t* codes,
                 uint8_t* scales, float* tensor_scale, void* workspace, size_t workspace_bytes,
                 void* stream)
{
    return quantize_impl(format, x, rows, cols, ld_x, flags, rht_signs, seed, codes, scales,
                         tensor_scale, workspace, workspace_bytes, stream);
}

int ifx_quantize_noalloc(int format, const void* x, int64_t rows, int64_t cols, int64_t ld_x,
                         uint32_t flags, uint32_t rht_signs, uint64_t seed, uint8_t* codes,
                         uint8_t* scales, float* tensor_scale, void* stream)
{
    return quantize_impl(format, x, rows, cols, ld_x, flags, rht_signs, seed, codes, scales,
                         tensor_scale, nullptr, 0, stream, true);
}

size_t ifq_quantize_workspace_bytes(int format, int64_t rows, int64_t cols, uint32_t flags)
{
    (void)format;
    (void)rows;
    (void)cols;
    if (flags & IFQ_SCALE_IN) return 0;
    return (size_t)ifq::kMaxPartials * sizeof(float);
}

int if4_dequantize(const uint8_t* codes, const uint8_t* scales, const float* tensor_scale,
                   int64_t rows, int64_t cols, void* out, int out_dtype, void* stream)
{
    return dequantize_impl(IFQ_FMT_IF4, codes, scales, tensor_scale, rows, cols, out, out_dtype, stream);
}

int nvfp4_dequantize(const uint8_t* codes, const uint8_t* scales, const float* tensor_scale,
                     int64_t rows, int64_t cols, void* out, int out_dtype, void* stream)
{
    return dequantize_impl(IFQ_FMT_NVFP4, codes, scales, tensor_scale, rows, cols, out, out_dtype,
                           stream);
}

int ifx_dequantize(int format, const uint8_t* codes, const uint8_t* scales,
                   const float* tensor_scale, int64_t rows, int64_t cols, void* out,
                   int out_dtype, void* stream)
{
    return dequantize_impl(format, codes, scales, tensor_scale, rows, cols, out, out_dtype, stream);
}

int if4_gemm(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_tensor_scale,
             const uint8_t* b_codes, const uint8_t* b_scales, const float* b_tensor_scale,
             int64_t M, int64_t N, int64_t K, void* c, int64_t ldc, int out_dtype, void* stream)
{
    return gemm_impl(IFQ_FMT_IF4, a_codes, a_scales, a_tensor_scale, b_codes, b_scales,
                     b_tensor_scale, M, N, K, c, ldc, out_dtype, stream);
}

int nvfp4_gemm(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_tensor_scale,
               const uint8_t* b_codes, const uint8_t* b_scales, const float* b_tensor_scale,
               int64_t M, int64_t N, int64_t K, void* c, int64_t ldc, int out_dtype, void* stream)
{
    return gemm_impl(IFQ_FMT_NVFP4, a_codes, a_scales, a_tensor_scale, b_codes, b_scales,
                     b_tensor_scale, M, N, K, c, ldc, out_dtype, stream);
}

int ifx_gemm(int format, const uint8_t* a_codes, const uint8_t* a_scales,
             const float* a_tensor_scale, const uint8_t* b_codes, const uint8_t* b_scales,
             const float* b_tensor_scale, int64_t M, int64_t N, int64_t K, void* c, int64_t ldc,
             int out_dtype, void* stream)
{
    return gemm_impl(format, a_codes, a_scales, a_tensor_scale, b_codes, b_scales, b_tensor_scale,
                     M, N, K, c, ldc, out_dtype, stream);
}

size_t ifq_quantize_dual_workspace_bytes(int format, int64_t rows, int64_t cols, uint32_t row_flags,
                                         uint32_t col_flags)
{
    (void)format;
    (void)rows;
    (void)cols;
    if ((row_flags & IFQ_SCALE_IN) && (col_flags & IFQ_SCALE_IN)) return 0;
    return (size_t)2 * ifq::kMaxPartials * sizeof(float);
}

int ifx_quantize_dual(int format, const void* x, int64_t rows, int64_t cols, int64_t ld_x,
                      uint32_t row_flags, uint32_t col_flags, uint32_t rht_signs, uint64_t row_seed,
                      uint64_t col_seed, uint8_t* row_codes, uint8_t* row_scales, float* row_tensor_scale,
                      uint8_t* col_codes, uint8_t* col_scales, float* col_tensor_scale, void* workspace,
                      size_t workspace_bytes, void* stream)
{
    if (!valid_format(format)) return IFQ_EINVAL;
    if ((row_flags | col_flags) & ~kKnownFlags) return IFQ_EINVAL;
    if ((row_flags | col_flags) & IFQ_AXIS_STRIDED) return IFQ_EINVAL;
    if (rht_signs > 0xFFFFu) return IFQ_EINVAL;
    if (!row_tensor_scale || !col_tensor_scale) return IFQ_EINVAL;
    if (!dual_format(format)) return IFQ_EUNSUPPORTED;
    if (rows < 0 || cols < 0) return IFQ_ESHAPE;
    if (rows > 0 && cols > 0 && rows > kMaxElems / cols) return IFQ_ESHAPE;
    if (rows % 16 || cols % 16) return IFQ_ESHAPE;
    if (!aligned(row_tensor_scale, 4) || !aligned(col_tensor_scale, 4)) return IFQ_EALIGN;
    const bool empty = rows == 0 || cols == 0;
    const bool need_ws = !((row_flags & IFQ_SCALE_IN) && (col_flags & IFQ_SCALE_IN));
    if (!empty) {
        if (!x || !row_codes || !row_scales || !col_codes || !col_scales) return IFQ_EINVAL;
        if (ld_x < cols) return IFQ_ESHAPE;
        if (!aligned(x, 2)) return IFQ_EALIGN;
        if (!aligned(row_codes, 16) || !aligned(col_codes, 16)) return IFQ_EALIGN;
        if (need_ws) {
            if (!workspace ||
                workspace_bytes < ifq_quantize_dual_workspace_bytes(format, rows, cols, row_flags, col_flags))
                return IFQ_EWORKSPACE;
            if (!aligned(workspace, 16)) return IFQ_EALIGN;
        }
    }
    ifq::DualArgs a;
    a.fmt = format;
    a.x = static_cast<const uint16_t*>(x);
    a.rows = rows;
    a.cols = cols;
    a.ld = ld_x;
    a.signs = rht_signs;
    float* ws = (need_ws && !empty) ? static_cast<float*>(workspace) : nullptr;
    a.row = {row_flags, row_seed, row_codes, row_scales, row_tensor_scale, ws};
    a.col = {col_flags, col_seed, col_codes, col_scales, col_tensor_scale, ws ? ws + ifq::kMaxPartials : nullptr};
    return ifq::launch_quantize_dual(a, static_cast<hipStream_t>(stream)) == hipSuccess ? IFQ_OK : IFQ_EHIP;
}

int ifq_group_size(int format)
{
    if (!valid_format(format)) return 0;
    return (format == IFQ_FMT_IF4_BS8 || format == IFQ_FMT_IF3_BS8 || format == IFQ_FMT_NVFP4_BS8) ? 8 : 16;
}

size_t ifq_codes_bytes(int format, int64_t rows, int64_t cols)
{
    if (!valid_format(format) || rows < 0 || cols < 0) return 0;
    return (size_t)(rows * cols * bits_of(format) / 8);
}

size_t ifq_scales_bytes(int format, int64_t rows, int64_t cols)
{
    const int g = ifq_group_size(format);
    if (g == 0 || rows < 0 || cols < 0) return 0;
    return (size_t)(rows * (cols / g));
}

const char* ifq_status_string(int status)
{
    switch (status) {
        case IFQ_OK: return "ok";
        case IFQ_EINVAL: return "invalid argument";
        case IFQ_ESHAPE: return "invalid shape";
        case IFQ_EALIGN: return "misaligned pointer or leading dimension";
        case IFQ_EUNSUPPORTED: return "unsupported combination";
        case IFQ_EHIP: return "HIP launch failed";
        case IFQ_EWORKSPACE: return "workspace missing or too small";
        default: return "unknown status";
    }
}

int ifq_abi_version(void) { return IFQ_ABI_VERSION; }

}  // extern "C"
