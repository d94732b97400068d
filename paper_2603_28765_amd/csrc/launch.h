// launch.h -- internal launchers behind the C ABI (host side).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ifq {

// Upper bound on the per-block maxima the tensor-max pass leaves in the
// workspace (one float each).
constexpr int kMaxPartials = 256;

struct QuantArgs {
    int fmt;
    const uint16_t* x;
    int64_t rows, cols, ld;
    uint32_t flags, signs;
    uint64_t seed;
    uint8_t* codes;
    uint8_t* scales;
    float* tensor_scale;
    float* partials;  // workspace
};

hipError_t launch_quantize(const QuantArgs& a, hipStream_t stream);

// The library's own device scratch for the tensor-max partials (one copy per
// GPU, kScratchBytes): its address on the device of `stream` (the current
// device for the null stream), looked up once per device.
constexpr size_t kScratchBytes = kMaxPartials * sizeof(float);
hipError_t scratch_partials(hipStream_t stream, float** ptr);

// One side of the dual quantizer (row-wise or strided output).
struct DualSide {
    uint32_t flags;  // IFQ_* bits of this side (IFQ_AXIS_STRIDED excluded)
    uint64_t seed;
    uint8_t* codes;
    uint8_t* scales;
    float* tensor_scale;
    float* partials;  // kMaxPartials floats of workspace (unused with IFQ_SCALE_IN)
};

struct DualArgs {
    int fmt;
    const uint16_t* x;
    int64_t rows, cols, ld;
    uint32_t signs;
    DualSide row, col;
};

hipError_t launch_quantize_dual(const DualArgs& a, hipStream_t stream);

hipError_t launch_dequantize(int fmt, const uint8_t* codes, const uint8_t* scales,
                             const float* tensor_scale, int64_t rows, int64_t cols, void* out,
                             bool out_bf16, hipStream_t stream);

struct GemmArgs {
    int fmt;
    const uint8_t* a_codes;
    const uint8_t* a_scales;
    const float* a_ts;
    const uint8_t* b_codes;
    const uint8_t* b_scales;
    const float* b_ts;
    int64_t M, N, K;
    void* c;
    int64_t ldc;
    bool out_bf16;
};

hipError_t launch_gemm(const GemmArgs& a, hipStream_t stream);

}  // namespace ifq
