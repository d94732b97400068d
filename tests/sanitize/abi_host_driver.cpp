// Sanitizer driver for the host side of the C ABI (test infrastructure):
// api.hip's argument validation and dispatch, linked against recording stubs
// of the launchers, built with host-only AddressSanitizer and
// UndefinedBehaviorSanitizer and run by tests/test_sanitizers_cpu.py.  Every
// entry point is called with valid arguments (the stubs check what reaches a
// launcher) and with each kind of invalid one (which must be rejected before
// any launcher runs).
#include <cstdio>
#include <cstdint>
#include <cstring>

#include "ifq.h"
#include "launch.h"

namespace {
int launches = 0;
int bad = 0;
void expect(bool ok, const char* what, int line)
{
    if (!ok) {
        std::fprintf(stderr, "line %d: %s\n", line, what);
        ++bad;
    }
}
#define EXPECT(c) expect((c), #c, __LINE__)
alignas(256) unsigned char dev_scratch[ifq::kScratchBytes];
}  // namespace

namespace ifq {
hipError_t launch_quantize(const QuantArgs& a, hipStream_t)
{
    ++launches;
    EXPECT(a.fmt >= IFQ_FMT_IF4 && a.fmt <= IFQ_FMT_NVFP4_BS8);
    EXPECT(a.tensor_scale != nullptr);
    EXPECT(a.rows == 0 || a.cols == 0 || (a.x && a.codes && a.scales));
    EXPECT((a.flags & IFQ_SCALE_IN) || a.rows == 0 || a.cols == 0 || a.partials != nullptr);
    return hipSuccess;
}
hipError_t launch_quantize_dual(const DualArgs& a, hipStream_t)
{
    ++launches;
    EXPECT(a.rows % 16 == 0 && a.cols % 16 == 0);
    EXPECT(a.row.tensor_scale && a.col.tensor_scale);
    return hipSuccess;
}
hipError_t launch_dequantize(int fmt, const uint8_t* codes, const uint8_t* scales, const float* ts,
                             int64_t rows, int64_t cols, void* out, bool, hipStream_t)
{
    ++launches;
    EXPECT(fmt >= 0 && fmt <= IFQ_FMT_NVFP4_BS8 && codes && scales && ts && out && rows > 0 && cols % 16 == 0);
    return hipSuccess;
}
hipError_t launch_gemm(const GemmArgs& a, hipStream_t)
{
    ++launches;
    EXPECT(a.M > 0 && a.N > 0 && a.K % 16 == 0 && a.c && a.ldc >= a.N);
    return hipSuccess;
}
hipError_t scratch_partials(hipStream_t, float** p)
{
    *p = reinterpret_cast<float*>(dev_scratch);
    return hipSuccess;
}
}  // namespace ifq

int main()
{
    alignas(256) static unsigned char buf[1 << 16];
    void* P = buf;                  // stands in for device memory: never dereferenced here
    unsigned char* U = buf;
    float* F = reinterpret_cast<float*>(buf);
    const size_t WS = ifq_quantize_workspace_bytes(IFQ_FMT_IF4, 64, 64, 0);
    EXPECT(WS > 0 && WS <= ifq::kScratchBytes);
    // valid calls reach the launchers
    for (int fmt = 0; fmt < 10; ++fmt) {
        for (uint32_t fl = 0; fl < 64; ++fl) {
            const int before = launches;
            EXPECT(ifx_quantize(fmt, P, 64, 64, 64, fl, 0xFFFF, 1, U, U, F, P, WS, nullptr) == IFQ_OK);
            EXPECT(ifx_quantize_noalloc(fmt, P, 64, 64, 64, fl, 0, 1, U, U, F, nullptr) == IFQ_OK);
            EXPECT(launches == before + 2);
        }
        EXPECT(ifx_dequantize(fmt, U, U, F, 16, 64, P, IFQ_BF16, nullptr) == IFQ_OK);
        EXPECT(ifx_gemm(fmt, U, U, F, U, U, F, 32, 48, 64, P, 48, IFQ_F32, nullptr) == IFQ_OK);
        EXPECT(ifq_codes_bytes(fmt, 16, 64) > 0 && ifq_scales_bytes(fmt, 16, 64) > 0);
    }
    EXPECT(ifx_quantize_dual(IFQ_FMT_IF4, P, 32, 64, 64, 0, IFQ_RHT, 0, 1, 2, U, U, F, U, U, F, P,
                             ifq_quantize_dual_workspace_bytes(IFQ_FMT_IF4, 32, 64, 0, 0), nullptr) == IFQ_OK);
    // invalid calls are rejected before any launcher
    const int before = launches;
    const int64_t huge = int64_t(1) << 40;
    EXPECT(ifx_quantize(11, P, 64, 64, 64, 0, 0, 0, U, U, F, P, WS, nullptr) == IFQ_EINVAL);
    EXPECT(ifx_quantize(0, P, 64, 64, 64, 1u << 9, 0, 0, U, U, F, P, WS, nullptr) == IFQ_EINVAL);
    EXPECT(ifx_quantize(0, P, 64, 64, 64, 0, 1u << 16, 0, U, U, F, P, WS, nullptr) == IFQ_EINVAL);
    EXPECT(ifx_quantize(0, P, -1, 64, 64, 0, 0, 0, U, U, F, P, WS, nullptr) == IFQ_ESHAPE);
    EXPECT(ifx_quantize(0, P, huge, huge, huge, 0, 0, 0, U, U, F, P, WS, nullptr) == IFQ_ESHAPE);
    EXPECT(ifx_quantize(0, P, 64, 40, 40, 0, 0, 0, U, U, F, P, WS, nullptr) == IFQ_ESHAPE);
    EXPECT(ifx_quantize(0, P, 64, 64, 32, 0, 0, 0, U, U, F, P, WS, nullptr) == IFQ_ESHAPE);
    EXPECT(ifx_quantize(0, U + 2, 64, 64, 64, 0, 0, 0, U, U, F, P, WS, nullptr) == IFQ_EALIGN);
    EXPECT(ifx_quantize(0, P, 64, 64, 64, 0, 0, 0, U, U, F, nullptr, 0, nullptr) == IFQ_EWORKSPACE);
    EXPECT(ifx_quantize(0, P, 64, 64, 64, 0, 0, 0, U, U, F, P, WS - 1, nullptr) == IFQ_EWORKSPACE);
    EXPECT(ifx_quantize_noalloc(0, nullptr, 64, 64, 64, 0, 0, 0, U, U, F, nullptr) == IFQ_EINVAL);
    EXPECT(ifx_quantize_noalloc(0, P, 64, 64, 64, 0, 0, 0, U + 8, U, F, nullptr) == IFQ_EALIGN);
    EXPECT(ifx_dequantize(0, U, U, F, 16, 40, P, IFQ_F32, nullptr) == IFQ_ESHAPE);
    EXPECT(ifx_dequantize(0, U, U, F, huge, huge, P, IFQ_F32, nullptr) == IFQ_ESHAPE);
    EXPECT(ifx_dequantize(0, U, U, F, 16, 64, U + 4, IFQ_F32, nullptr) == IFQ_EALIGN);
    EXPECT(ifx_gemm(0, U, U, F, U, U, F, 32, 48, 64, P, 40, IFQ_F32, nullptr) == IFQ_ESHAPE);
    EXPECT(ifx_gemm(0, U, U, F, U, U, F, huge, huge, huge, P, huge, IFQ_F32, nullptr) == IFQ_ESHAPE);
    EXPECT(ifx_gemm(0, U + 4, U, F, U, U, F, 32, 48, 64, P, 48, IFQ_F32, nullptr) == IFQ_EALIGN);
    EXPECT(ifx_gemm(0, U, U, F, U, U, F, 32, 48, 64, P, 48, 7, nullptr) == IFQ_EINVAL);
    EXPECT(ifx_quantize_dual(IFQ_FMT_IF3, P, 32, 64, 64, 0, 0, 0, 1, 2, U, U, F, U, U, F, P, 4096, nullptr) ==
           IFQ_EUNSUPPORTED);
    EXPECT(ifx_quantize_dual(IFQ_FMT_IF4, P, 40, 64, 64, 0, 0, 0, 1, 2, U, U, F, U, U, F, P, 4096, nullptr) ==
           IFQ_ESHAPE);
    EXPECT(launches == before);
    // empty tensors: the quantizer only publishes alpha = 0, the others do nothing
    EXPECT(ifx_gemm(0, U, U, F, U, U, F, 0, 48, 64, P, 48, IFQ_F32, nullptr) == IFQ_OK);
    EXPECT(ifx_dequantize(0, U, U, F, 0, 64, P, IFQ_F32, nullptr) == IFQ_OK);
    for (int s = -7; s <= 1; ++s) EXPECT(std::strlen(ifq_status_string(s)) > 0);
    EXPECT(ifq_abi_version() == IFQ_ABI_VERSION);
    std::printf("abi host driver: %d launches, %d failures\n", launches, bad);
    return bad != 0;
}
