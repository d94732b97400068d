// gemm.hip -- block-scaled GEMM C = A_hat B_hat^T on packed operands
// (both K-major), gfx950 MFMA.
//
// Per K tile, each thread loads the packed codes and scale bytes of two
// groups, decodes every element to an FP16 value that carries its group
// scale exactly (fold_FP * q * Delta for FP groups, fold_INT * q * Delta for
// INT groups, fold_FP / fold_INT = M_I / M_FP), and stages the decoded tile
// in LDS.  Four wavefronts then run v_mfma_f32_32x32x16_f16 over it with FP32
// accumulation.  Because every decoded operand is exact, one FP32
// accumulation over all of K applies each 16-wide block's scale product and
// its range alignment (1, 6/7 or 36/49 for IF4, Sec. 5.2) at once; the
// epilogue multiplies by alpha_A * alpha_B / fold_FP^2.
//
// Exactness of the FP16 operands: an E4M3 scale has at most 4 significant
// bits and lies in [2^-9, 448]; 7*q_FP and 6*q_INT have at most 5; products
// have at most 9 bits and lie in [3.5*2^-9, 42*448], all normal FP16.
// IF3 uses folds 3 and 4 (at most 6 bits).
#include "device.h"
#include "launch.h"

namespace ifq {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kBM = 128, kBN = 128, kBK = 64;
constexpr int kGemmThreads = 256;
constexpr int kPitch = kBK + 8;  // halves per LDS row (16-byte pad)

template <int FMT> struct Fold;
template <> struct Fold<IFQ_FMT_IF4> { static constexpr float FP = 7.0f, INT = 6.0f; };
template <> struct Fold<IFQ_FMT_NVFP4> { static constexpr float FP = 1.0f, INT = 1.0f; };
template <> struct Fold<IFQ_FMT_IF3> { static constexpr float FP = 3.0f, INT = 4.0f; };

// Decode the 16 codes of one group into fold * value * Delta as FP16.
template <int FMT>
__device__ __forceinline__ void decode_group(const uint32_t (&c)[kGroup], uint32_t sb,
                                             _Float16* dst)
{
    using F = Fmt<FMT>;
    using D = FmtDerived<FMT>;
    const bool is_int = F::ADAPTIVE && (sb & 0x80u);
    const float sc = (is_int ? Fold<FMT>::INT : Fold<FMT>::FP) * e4m3_value(sb);
    _Float16 h[kGroup];
#pragma unroll
    for (int j = 0; j < kGroup; ++j) {
        float q;
        if (is_int) {
            q = (float)((int)(c[j] << (32 - F::BITS)) >> (32 - F::BITS));
        } else {
            const uint32_t neg = (c[j] & D::SIGN_BIT) ? 1u : 0u;
            q = __uint_as_float(__float_as_uint(fp_magnitude<FMT>(c[j] & (D::SIGN_BIT - 1u))) | (neg << 31));
        }
        h[j] = (_Float16)(q * sc);
    }
    uint4* d = reinterpret_cast<uint4*>(dst);
    const uint4* s = reinterpret_cast<const uint4*>(h);
    d[0] = s[0];
    d[1] = s[1];
}

// Stage rows [row0, row0 + kBM) x groups [g0, g0 + kBK/16) of one operand.
template <int FMT>
__device__ __forceinline__ void stage_operand(const uint8_t* __restrict__ codes,
                                              const uint8_t* __restrict__ scales, int64_t nrows,
                                              int64_t gpr, int64_t row0, int64_t g0,
                                              _Float16 (*lds)[kPitch])
{
    constexpr int BITS = Fmt<FMT>::BITS;
    constexpr int GPT = kBM * (kBK / kGroup) / kGemmThreads;  // groups per thread (2)
#pragma unroll
    for (int i = 0; i < GPT; ++i) {
        const int slot = threadIdx.x * GPT + i;
        const int r = slot / (kBK / kGroup), gk = slot % (kBK / kGroup);
        const int64_t row = row0 + r, g = g0 + gk;
        uint32_t c[kGroup];
        uint32_t sb = 0;
        if (row < nrows && g < gpr) {
            load_unpack16<BITS>(codes + (row * gpr + g) * (2 * BITS), c);
            sb = scales[row * gpr + g];
        } else {
#pragma unroll
            for (int j = 0; j < kGroup; ++j) c[j] = 0;
        }
        decode_group<FMT>(c, sb, &lds[r][gk * kGroup]);
    }
}

template <int FMT, bool OUT_BF16>
__global__ __launch_bounds__(kGemmThreads) void gemm_tn(
    const uint8_t* __restrict__ a_codes, const uint8_t* __restrict__ a_scales,
    const float* __restrict__ a_ts, const uint8_t* __restrict__ b_codes,
    const uint8_t* __restrict__ b_scales, const float* __restrict__ b_ts, int64_t M, int64_t N,
    int64_t K, void* __restrict__ C, int64_t ldc)
{
    __shared__ __attribute__((aligned(16))) _Float16 As[kBM][kPitch];
    __shared__ __attribute__((aligned(16))) _Float16 Bs[kBN][kPitch];

    const int64_t m0 = (int64_t)blockIdx.y * kBM, n0 = (int64_t)blockIdx.x * kBN;
    const int64_t gpr = K / kGroup;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = wave >> 1, wn = wave & 1;

    floatx16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

    for (int64_t g0 = 0; g0 < gpr; g0 += kBK / kGroup) {
        stage_operand<FMT>(a_codes, a_scales, M, gpr, m0, g0, As);
        stage_operand<FMT>(b_codes, b_scales, N, gpr, n0, g0, Bs);
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < kBK / 16; ++kk) {
            const int kofs = kk * 16 + (lane >> 5) * 8;
            half8 af[2], bf[2];
#pragma unroll
            for (int i = 0; i < 2; ++i)
                af[i] = *reinterpret_cast<const half8*>(&As[wm * 64 + i * 32 + (lane & 31)][kofs]);
#pragma unroll
            for (int j = 0; j < 2; ++j)
                bf[j] = *reinterpret_cast<const half8*>(&Bs[wn * 64 + j * 32 + (lane & 31)][kofs]);
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(af[i], bf[j], acc[i][j], 0, 0, 0);
        }
        __syncthreads();
    }

    const float sc = (*a_ts * *b_ts) / (Fold<FMT>::FP * Fold<FMT>::FP);
#pragma unroll
    for (int i = 0; i < 2; ++i) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int64_t n = n0 + wn * 64 + j * 32 + (lane & 31);
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int64_t m = m0 + wm * 64 + i * 32 + (e >> 2) * 8 + (lane >> 5) * 4 + (e & 3);
                if (m < M && n < N) {
                    const float v = acc[i][j][e] * sc;
                    if constexpr (OUT_BF16)
                        static_cast<uint16_t*>(C)[m * ldc + n] = f32_to_bf16_rne(v);
                    else
                        static_cast<float*>(C)[m * ldc + n] = v;
                }
            }
        }
    }
}

template <int FMT>
static hipError_t launch_g(const GemmArgs& a, hipStream_t s)
{
    dim3 grid((unsigned)((a.N + kBN - 1) / kBN), (unsigned)((a.M + kBM - 1) / kBM));
    if (grid.x == 0 || grid.y == 0) return hipSuccess;
    if (a.out_bf16)
        hipLaunchKernelGGL((gemm_tn<FMT, true>), grid, dim3(kGemmThreads), 0, s, a.a_codes, a.a_scales,
                           a.a_ts, a.b_codes, a.b_scales, a.b_ts, a.M, a.N, a.K, a.c, a.ldc);
    else
        hipLaunchKernelGGL((gemm_tn<FMT, false>), grid, dim3(kGemmThreads), 0, s, a.a_codes, a.a_scales,
                           a.a_ts, a.b_codes, a.b_scales, a.b_ts, a.M, a.N, a.K, a.c, a.ldc);
    return hipGetLastError();
}

hipError_t launch_gemm(const GemmArgs& a, hipStream_t s)
{
    switch (a.fmt) {
        case IFQ_FMT_IF4: return launch_g<IFQ_FMT_IF4>(a, s);
        case IFQ_FMT_NVFP4: return launch_g<IFQ_FMT_NVFP4>(a, s);
        case IFQ_FMT_IF3: return launch_g<IFQ_FMT_IF3>(a, s);
        default: return hipErrorNotSupported;
    }
}

}  // namespace ifq
