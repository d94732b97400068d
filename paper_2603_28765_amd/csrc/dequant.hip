// dequant.hip -- standalone dequantization: q * Delta [* M_FP/M_I] * alpha
// (the dequantized values of Fig. 3a with the tensor scale of Eq. 1), one group of 16 per
// lane, written as fp32 or bf16.
#include "device.h"
#include "launch.h"

namespace ifq {

constexpr int kDqThreads = 256;
typedef uint32_t dq_u32x4 __attribute__((ext_vector_type(4)));

typedef float dq_f32x2 __attribute__((ext_vector_type(2)));

// Codes 2 SEL and 2 SEL + 1 of word w (E2M1) as fp32, exact.
template <int SEL>
__device__ __forceinline__ void fp4_pair(uint32_t w, float (&q)[kGroup], int at)
{
    const dq_f32x2 v = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w, 1.0f, SEL);
    q[at] = v[0];
    q[at + 1] = v[1];
}

// Signed value of FP code c (no branch on the exponent field).
template <int FMT>
__device__ __forceinline__ float fp_code_value(uint32_t c)
{
    using F = Fmt<FMT>;
    using D = FmtDerived<FMT>;
    const uint32_t mi = c & (D::SIGN_BIT - 1u);
    const uint32_t E = mi >> F::MB, M = mi & ((1u << F::MB) - 1u);
    const float sub = (float)M * __uint_as_float((uint32_t)(127 + 1 - D::BIAS - F::MB) << 23);
    const float nor = __uint_as_float(((E - D::BIAS + 127u) << 23) | (M << (23 - F::MB)));
    const float mag = E ? nor : sub;
    return __uint_as_float(__float_as_uint(mag) | ((c & D::SIGN_BIT) ? 0x80000000u : 0u));
}

template <int FMT, bool OUT_BF16>
__global__ __launch_bounds__(kDqThreads) void dequantize_groups(const uint8_t* __restrict__ codes,
                                                                const uint8_t* __restrict__ scales,
                                                                const float* __restrict__ tensor_scale,
                                                                int64_t ngroups, void* __restrict__ out)
{
    using F = Fmt<FMT>;
    using D = FmtDerived<FMT>;
    constexpr bool E2M1 = F::BITS == 4 && F::EB == 2 && F::MB == 1;
    const float alpha = *tensor_scale;
    const int64_t stride = (int64_t)gridDim.x * kDqThreads;
    for (int64_t g = (int64_t)blockIdx.x * kDqThreads + threadIdx.x; g < ngroups; g += stride) {
        uint32_t c[kGroup];
        float qf[kGroup];
        if constexpr (E2M1 && F::KIND != kKindInt) {
            // E2M1 codes two at a time through the hardware converter (exact)
            const uint2 t = *reinterpret_cast<const uint2*>(codes + g * 8);
            fp4_pair<0>(t.x, qf, 0); fp4_pair<1>(t.x, qf, 2); fp4_pair<2>(t.x, qf, 4); fp4_pair<3>(t.x, qf, 6);
            fp4_pair<0>(t.y, qf, 8); fp4_pair<1>(t.y, qf, 10); fp4_pair<2>(t.y, qf, 12); fp4_pair<3>(t.y, qf, 14);
#pragma unroll
            for (int j = 0; j < kGroup; ++j) c[j] = ((j < 8 ? t.x : t.y) >> (4 * (j & 7))) & 15u;
        } else if constexpr (F::BITS == 6) {
            // FP6 codes through the 32-value hardware decode (exact for every
            // code; the stream's codes 0..15 are this group's, 16..31 zeros)
            typedef uint32_t u6v __attribute__((ext_vector_type(6)));
            typedef float f32v __attribute__((ext_vector_type(32)));
            const uint32_t* src = reinterpret_cast<const uint32_t*>(codes + g * 12);
            const u6v r = {src[0], src[1], src[2], 0u, 0u, 0u};
            f32v q;
            if constexpr (F::EB == 2) q = __builtin_amdgcn_cvt_scalef32_pk32_f32_fp6(r, 1.0f);
            else q = __builtin_amdgcn_cvt_scalef32_pk32_f32_bf6(r, 1.0f);
#pragma unroll
            for (int j = 0; j < kGroup; ++j) qf[j] = q[j];
            load_unpack16<6>(codes + g * 12, c);  // the INT codes
        } else {
            load_unpack16<F::BITS>(codes + g * (2 * F::BITS), c);
            if constexpr (F::KIND != kKindInt) {
#pragma unroll
                for (int j = 0; j < kGroup; ++j) qf[j] = fp_code_value<FMT>(c[j]);
            }
        }
        // block size 8: the second half of the 16 values has its own scale byte
        const uint32_t sb0 = F::G == 8 ? scales[2 * g] : scales[g];
        const uint32_t sb1 = F::G == 8 ? scales[2 * g + 1] : sb0;
        const float d0 = e4m3_value(sb0), d1 = e4m3_value(sb1);
        const bool i0 = F::KIND == kKindInt || (F::ADAPTIVE && (sb0 & 0x80u));
        const bool i1 = F::KIND == kKindInt || (F::ADAPTIVE && (sb1 & 0x80u));
        float o[kGroup];
#pragma unroll
        for (int j = 0; j < kGroup; ++j) {
            const bool is_int = j < 8 ? i0 : i1;
            float q;
            if constexpr (F::KIND == kKindInt) {
                q = (float)((int)(c[j] << (32 - F::BITS)) >> (32 - F::BITS));
            } else if constexpr (F::ADAPTIVE) {
                const float qi = (float)((int)(c[j] << (32 - F::BITS)) >> (32 - F::BITS));
                q = is_int ? qi : qf[j];
            } else {
                q = qf[j];
            }
            // the rounding sequence of the oracle: q Delta (exact), times
            // M_FP / M_I for INT groups, times alpha
            const float k = is_int ? D::K_DN : 1.0f;
            o[j] = ((q * (j < 8 ? d0 : d1)) * k) * alpha;
        }
        if constexpr (OUT_BF16) {
            uint32_t p[8];
#pragma unroll
            for (int i = 0; i < 8; ++i)
                p[i] = (uint32_t)f32_to_bf16_rne(o[2 * i]) | ((uint32_t)f32_to_bf16_rne(o[2 * i + 1]) << 16);
            dq_u32x4 lo{p[0], p[1], p[2], p[3]}, hi{p[4], p[5], p[6], p[7]};
            const int64_t g0 = g - (threadIdx.x & 63);  // the wavefront's first group
            if (g0 + 64 <= ngroups) {
                // The wavefront's 64 groups are 2 KiB of output: swap halves
                // across the wavefront so that each store covers 1 KiB
                // contiguously (lane l writes pieces 2(l mod 32) + l/32 and
                // 64 + 2(l mod 32) + l/32), the inverse of the quantizer's
                // load.
#pragma unroll
                for (int d = 0; d < 4; ++d) {
                    const auto r = __builtin_amdgcn_permlane32_swap(lo[d], hi[d], false, false);
                    lo[d] = r[0];
                    hi[d] = r[1];
                }
                const int lane = threadIdx.x & 63;
                const int piece = 2 * (lane & 31) + (lane >> 5);
                dq_u32x4* dst = reinterpret_cast<dq_u32x4*>(static_cast<uint16_t*>(out) + g0 * kGroup);
                // non-temporal: 1-2 us faster here (no gain for fp32 output)
                __builtin_nontemporal_store(lo, dst + piece);
                __builtin_nontemporal_store(hi, dst + 64 + piece);
            } else {
                dq_u32x4* dst = reinterpret_cast<dq_u32x4*>(static_cast<uint16_t*>(out) + g * kGroup);
                dst[0] = lo;
                dst[1] = hi;
            }
        } else {
            dq_u32x4 P[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                P[i] = dq_u32x4{__float_as_uint(o[4 * i]), __float_as_uint(o[4 * i + 1]),
                                __float_as_uint(o[4 * i + 2]), __float_as_uint(o[4 * i + 3])};
            const int64_t g0 = g - (threadIdx.x & 63);  // the wavefront's first group
            if (g0 + 64 <= ngroups) {
                // 4 KiB of output per wavefront: a 4 x 4 transpose of the
                // 16-byte pieces across the wavefront's four 16-lane rows
                // (swap 2 x 2 blocks across the halves, then rows within
                // each half) leaves in lane (row r, column c) piece r of the
                // group of lane (k, c) in P[k], so store k covers 1 KiB
                // contiguously: groups 16k .. 16k + 15.
#pragma unroll
                for (int d = 0; d < 4; ++d) {
                    auto a = __builtin_amdgcn_permlane32_swap(P[0][d], P[2][d], false, false);
                    auto b = __builtin_amdgcn_permlane32_swap(P[1][d], P[3][d], false, false);
                    auto c0 = __builtin_amdgcn_permlane16_swap(a[0], b[0], false, false);
                    auto c1 = __builtin_amdgcn_permlane16_swap(a[1], b[1], false, false);
                    P[0][d] = c0[0];
                    P[1][d] = c0[1];
                    P[2][d] = c1[0];
                    P[3][d] = c1[1];
                }
                const int lane = threadIdx.x & 63;
                dq_u32x4* dst = reinterpret_cast<dq_u32x4*>(static_cast<float*>(out) + g0 * kGroup);
#pragma unroll
                for (int k = 0; k < 4; ++k) dst[64 * k + 4 * (lane & 15) + (lane >> 4)] = P[k];
            } else {
                dq_u32x4* dst = reinterpret_cast<dq_u32x4*>(static_cast<float*>(out) + g * kGroup);
#pragma unroll
                for (int i = 0; i < 4; ++i) dst[i] = P[i];
            }
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
