// dequant.hip -- standalone dequantization: q * Delta [* M_FP/M_I] * alpha
// (the dequantized values of Fig. 3a with the tensor scale of Eq. 1), one group of 16 per
// lane, written as fp32 or bf16.
#include "device.h"
#include "launch.h"

namespace ifq {

constexpr int kDqThreads = 256;

template <int FMT, bool OUT_BF16>
__global__ __launch_bounds__(kDqThreads) void dequantize_groups(const uint8_t* __restrict__ codes,
                                                                const uint8_t* __restrict__ scales,
                                                                const float* __restrict__ tensor_scale,
                                                                int64_t ngroups, void* __restrict__ out)
{
    using F = Fmt<FMT>;
    using D = FmtDerived<FMT>;
    const float alpha = *tensor_scale;
    const int64_t stride = (int64_t)gridDim.x * kDqThreads;
    for (int64_t g = (int64_t)blockIdx.x * kDqThreads + threadIdx.x; g < ngroups; g += stride) {
        uint32_t c[kGroup];
        load_unpack16<F::BITS>(codes + g * (2 * F::BITS), c);
        // block size 8: the second half of the 16 values has its own scale byte
        const uint32_t sb0 = F::G == 8 ? scales[2 * g] : scales[g];
        const uint32_t sb1 = F::G == 8 ? scales[2 * g + 1] : sb0;
        float o[kGroup];
#pragma unroll
        for (int j = 0; j < kGroup; ++j) {
            const uint32_t sb = j < 8 ? sb0 : sb1;
            const float delta = e4m3_value(sb);
            const bool is_int = F::KIND == kKindInt || (F::ADAPTIVE && (sb & 0x80u));
            float q;
            if (is_int) {
                q = (float)((int)(c[j] << (32 - F::BITS)) >> (32 - F::BITS));
            } else {
                const uint32_t neg = (c[j] & D::SIGN_BIT) ? 1u : 0u;
                q = __uint_as_float(__float_as_uint(fp_magnitude<FMT>(c[j] & (D::SIGN_BIT - 1u))) |
                                    (neg << 31));
            }
            float t = q * delta;
            if (is_int) t = t * D::K_DN;
            o[j] = t * alpha;
        }
        if constexpr (OUT_BF16) {
            uint32_t p[8];
#pragma unroll
            for (int i = 0; i < 8; ++i)
                p[i] = (uint32_t)f32_to_bf16_rne(o[2 * i]) | ((uint32_t)f32_to_bf16_rne(o[2 * i + 1]) << 16);
            uint4* dst = reinterpret_cast<uint4*>(static_cast<uint16_t*>(out) + g * kGroup);
            dst[0] = make_uint4(p[0], p[1], p[2], p[3]);
            dst[1] = make_uint4(p[4], p[5], p[6], p[7]);
        } else {
            float4* dst = reinterpret_cast<float4*>(static_cast<float*>(out) + g * kGroup);
#pragma unroll
            for (int i = 0; i < 4; ++i) dst[i] = make_float4(o[4 * i], o[4 * i + 1], o[4 * i + 2], o[4 * i + 3]);
        }
    }
}

template <int FMT>
static hipError_t launch_dq(const uint8_t* codes, const uint8_t* scales, const float* ts,
                            int64_t ngroups, void* out, bool bf16, hipStream_t s)
{
    int64_t blocks = std::min<int64_t>((ngroups + kDqThreads - 1) / kDqThreads, 65536);
    if (blocks == 0) return hipSuccess;
    if (bf16)
        hipLaunchKernelGGL((dequantize_groups<FMT, true>), dim3((unsigned)blocks), dim3(kDqThreads), 0, s,
                           codes, scales, ts, ngroups, out);
    else
        hipLaunchKernelGGL((dequantize_groups<FMT, false>), dim3((unsigned)blocks), dim3(kDqThreads), 0, s,
                           codes, scales, ts, ngroups, out);
    return hipGetLastError();
}

hipError_t launch_dequantize(int fmt, const uint8_t* codes, const uint8_t* scales,
                             const float* ts, int64_t rows, int64_t cols, void* out, bool bf16,
                             hipStream_t s)
{
    const int64_t ngroups = rows * (cols / kGroup);
    switch (fmt) {
        case IFQ_FMT_IF4: return launch_dq<IFQ_FMT_IF4>(codes, scales, ts, ngroups, out, bf16, s);
        case IFQ_FMT_NVFP4: return launch_dq<IFQ_FMT_NVFP4>(codes, scales, ts, ngroups, out, bf16, s);
        case IFQ_FMT_IF3: return launch_dq<IFQ_FMT_IF3>(codes, scales, ts, ngroups, out, bf16, s);
        case IFQ_FMT_IF6_E2M3: return launch_dq<IFQ_FMT_IF6_E2M3>(codes, scales, ts, ngroups, out, bf16, s);
        case IFQ_FMT_IF6_E3M2: return launch_dq<IFQ_FMT_IF6_E3M2>(codes, scales, ts, ngroups, out, bf16, s);
        case IFQ_FMT_NVINT4: return launch_dq<IFQ_FMT_NVINT4>(codes, scales, ts, ngroups, out, bf16, s);
        // 4/6 data decode exactly like NVFP4
        case IFQ_FMT_NVFP4_46: return launch_dq<IFQ_FMT_NVFP4>(codes, scales, ts, ngroups, out, bf16, s);
        case IFQ_FMT_IF4_BS8: return launch_dq<IFQ_FMT_IF4_BS8>(codes, scales, ts, ngroups, out, bf16, s);
        case IFQ_FMT_IF3_BS8: return launch_dq<IFQ_FMT_IF3_BS8>(codes, scales, ts, ngroups, out, bf16, s);
        case IFQ_FMT_NVFP4_BS8: return launch_dq<IFQ_FMT_NVFP4_BS8>(codes, scales, ts, ngroups, out, bf16, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace ifq
