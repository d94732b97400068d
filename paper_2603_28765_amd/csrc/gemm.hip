// gemm.hip -- block-scaled GEMM C = A_hat B_hat^T on packed operands
// (both K-major), gfx950 MFMA.
//
// Operand values.  Every element is decoded to an FP16 number that carries
// its group scale exactly: lambda * fold_FP * q * Delta for FP groups and
// lambda * fold_INT * q * Delta for INT groups, with fold_FP / fold_INT =
// M_I / M_FP (7 and 6 for IF4, lambda = 2^-5; 1 for NVFP4).  One FP32 MFMA
// accumulation over all of K then applies each 16-wide block's scale product
// and its range alignment (1, 6/7 or 36/49 for IF4, Sec. 5.2) at once; the
// epilogue multiplies by alpha_A * alpha_B / (lambda * fold_FP)^2.
// Exactness: an E4M3 scale has at most 4 significant bits and lies in
// [2^-9, 448]; 7 q_FP and 6 q_INT have at most 5, so every operand has at
// most 9 significant bits and lies in [3.5 * 2^-14, 42 * 448 / 32], all
// normal FP16 numbers.
//
// Decode (per pair of elements, one byte of codes):
//   FP  groups: v_cvt_scalef32_pk_f16_fp4 gives (q, q') exactly;
//   INT groups: u = n ^ 8 = q + 8 in [0, 15]; an E4M3 byte 0..15 decodes
//               linearly to u * 2^-9 (v_cvt_scalef32_pk_f16_fp8), so
//               u * 2^-9 * 96 Delta - 1.5 Delta = (6/32) q Delta exactly;
//   then one v_pk_fma_f16 with the group's (K, C) = (7 Delta / 32, 0) or
//   (96 Delta, -1.5 Delta) applies scale and bias to either kind.
//
// Tiling.  A workgroup of 4 wavefronts owns a 256 x 256 tile of C; wavefront
// w owns rows [64 w, 64 w + 64) and all 256 columns (2 x 8
// v_mfma_f32_32x32x16_f16 blocks, 256 accumulators per lane).  Each
// wavefront decodes its own A rows straight into MFMA fragment registers (no
// LDS traffic, no duplicate decode).  B is decoded once per workgroup --
// thread t owns row t of the B tile -- into a double-buffered FP16 LDS stage.
// The K order inside a 64-wide step is permuted the same way for A and B so
// that lane half h of every MFMA holds k in [32 h, 32 h + 32): each lane then
// loads 16 contiguous bytes of A codes per row and step.  Global loads run
// two K steps ahead.  LDS rows hold 64 halves padded to 144 bytes, so the 16
// lanes of a 128-bit access phase touch disjoint banks and every address is a
// per-lane base plus an immediate.
#include <atomic>
#include <type_traits>

#include "device.h"
#include "launch.h"

namespace ifq {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kBM = 256, kBN = 256, kBK = 64;
constexpr int kGemmThreads = 256;
constexpr int kGroupsPerStep = kBK / kGroup;  // 4
constexpr int kPitch = kBK + 8;                // halves per LDS row: 144 bytes
constexpr int kStageHalves = kBN * kPitch;     // one B stage

// Folds: FP operand = FP * q * Delta, INT operand = INT * q * Delta;
// EPI = 1 / (FP * FP) undoes them in the epilogue.
template <int FMT> struct Fold;
template <> struct Fold<IFQ_FMT_IF4> {
    static constexpr float FP = 7.0f / 32.0f, INT = 6.0f / 32.0f, EPI = 1024.0f / 49.0f;
};
template <> struct Fold<IFQ_FMT_NVFP4> { static constexpr float FP = 1.0f, INT = 1.0f, EPI = 1.0f; };
// NVINT4: q Delta / 4 (K = 128 Delta, C = -2 Delta on x = (q + 8) 2^-9); the
// quarter keeps 128 * 448 below the FP16 maximum.
template <> struct Fold<IFQ_FMT_NVINT4> { static constexpr float FP = 0.25f, INT = 0.25f, EPI = 16.0f; };
template <> struct Fold<IFQ_FMT_IF3> { static constexpr float FP = 3.0f, INT = 4.0f, EPI = 1.0f / 9.0f; };
// IF6: FP x 62 and INT x 15 (E2M3, ratio 7.5/31) or x 31 and x 28 (E3M2,
// ratio 28/31), times lambda = 1/4 or 1/8 so that 7.5*62*448*lambda and
// 28*31*448*lambda stay below the FP16 maximum.  With Delta the operand has
// up to 13 significant bits and is rounded once to FP16 (relative error at
// most 2^-12 per operand; the only inexact step of the GEMM besides FP32
// accumulation).
template <> struct Fold<IFQ_FMT_IF6_E2M3> {
    static constexpr float FP = 62.0f / 4.0f, INT = 15.0f / 4.0f, EPI = 1.0f / (15.5f * 15.5f);
};
template <> struct Fold<IFQ_FMT_IF6_E3M2> {
    static constexpr float FP = 31.0f / 8.0f, INT = 28.0f / 8.0f, EPI = 64.0f / 961.0f;
};
// block size 8: the block-16 format's folds, applied per 8 values
template <> struct Fold<IFQ_FMT_IF4_BS8> : Fold<IFQ_FMT_IF4> {};
template <> struct Fold<IFQ_FMT_IF3_BS8> : Fold<IFQ_FMT_IF3> {};
template <> struct Fold<IFQ_FMT_NVFP4_BS8> : Fold<IFQ_FMT_NVFP4> {};

typedef float float2v __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t h2_as_u32(half2v h) { return __builtin_bit_cast(uint32_t, h); }
__device__ __forceinline__ half2v u32_as_h2(uint32_t u) { return __builtin_bit_cast(half2v, u); }

// Keep a value computed on every lane (stops the compiler from sinking its
// computation into a divergent branch in front of a select).
__device__ __forceinline__ uint32_t pin(uint32_t v)
{
    asm volatile("" : "+v"(v));
    return v;
}

// (K, C) of two groups whose scale bytes are the low and high byte of sw:
// lane 0 of each half2 belongs to the low byte's group.
template <int FMT>
__device__ __forceinline__ void pair_scales(uint32_t sw, uint32_t& K, uint32_t& Cb)
{
    const half2v d = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(sw & 0x7F7Fu, 1.0f, false);  // E4M3 -> FP16
    if constexpr (Fmt<FMT>::KIND == kKindInt) {
        const half2v ki = {(_Float16)128.0f, (_Float16)128.0f}, cn = {(_Float16)-2.0f, (_Float16)-2.0f};
        K = h2_as_u32(d * ki);
        Cb = h2_as_u32(d * cn);
    } else if constexpr (Fmt<FMT>::ADAPTIVE && Fmt<FMT>::BITS == 4) {
        half2v ki, kf, cn;
        ki[0] = (_Float16)96.0f; ki[1] = (_Float16)96.0f;
        kf[0] = (_Float16)Fold<FMT>::FP; kf[1] = (_Float16)Fold<FMT>::FP;
        cn[0] = (_Float16)-1.5f; cn[1] = (_Float16)-1.5f;
        const uint32_t KI = h2_as_u32(d * ki), KF = h2_as_u32(d * kf), CN = h2_as_u32(d * cn);
        // 0xFFFF in a half whose group is INT (sign bit of its scale byte)
        const uint32_t m = __builtin_amdgcn_perm(sw << 8, sw, 0x08080A0Au);
        K = (KI & m) | (KF & ~m);
        Cb = CN & m;
    } else if constexpr (Fmt<FMT>::BITS == 4) {
        half2v f;
        f[0] = (_Float16)Fold<FMT>::FP; f[1] = (_Float16)Fold<FMT>::FP;
        K = h2_as_u32(d * f);
        Cb = 0;
    } else {
        K = h2_as_u32(d);  // IF3 applies its folds to the element values
        Cb = 0;
    }
}

__device__ __forceinline__ uint32_t bcast_lo(uint32_t v) { return __builtin_amdgcn_perm(v, v, 0x01000100u); }
__device__ __forceinline__ uint32_t bcast_hi(uint32_t v) { return __builtin_amdgcn_perm(v, v, 0x03020302u); }

// Four FP16 operand pairs from one dword of IF4/NVFP4 codes (elements 2i, 2i+1
// in byte i), for a group with broadcast scale pair (k2, c2).
template <int FMT>
__device__ __forceinline__ void decode_word(uint32_t w, bool is_int, uint32_t k2, uint32_t c2,
                                            uint32_t (&out)[4])
{
    uint32_t x[4];
    x[0] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 1.0f, 0));
    x[1] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 1.0f, 1));
    x[2] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 1.0f, 2));
    x[3] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 1.0f, 3));
    if constexpr (Fmt<FMT>::ADAPTIVE) {
        const uint32_t wu = w ^ 0x88888888u;
        const uint32_t lo = wu & 0x0F0F0F0Fu, hi = (wu >> 4) & 0x0F0F0F0Fu;
        const uint32_t d0 = __builtin_amdgcn_perm(hi, lo, 0x05010400u);  // u0 u1 u2 u3
        const uint32_t d1 = __builtin_amdgcn_perm(hi, lo, 0x07030602u);  // u4 u5 u6 u7
        const uint32_t y0 = pin(h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp8(d0, 1.0f, false)));
        const uint32_t y1 = pin(h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp8(d0, 1.0f, true)));
        const uint32_t y2 = pin(h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp8(d1, 1.0f, false)));
        const uint32_t y3 = pin(h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp8(d1, 1.0f, true)));
        x[0] = is_int ? y0 : x[0];
        x[1] = is_int ? y1 : x[1];
        x[2] = is_int ? y2 : x[2];
        x[3] = is_int ? y3 : x[3];
    } else if constexpr (Fmt<FMT>::KIND == kKindInt) {
        (void)is_int;
        const uint32_t wu = w ^ 0x88888888u;
        const uint32_t lo = wu & 0x0F0F0F0Fu, hi = (wu >> 4) & 0x0F0F0F0Fu;
        const uint32_t d0 = __builtin_amdgcn_perm(hi, lo, 0x05010400u);
        const uint32_t d1 = __builtin_amdgcn_perm(hi, lo, 0x07030602u);
        x[0] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp8(d0, 1.0f, false));
        x[1] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp8(d0, 1.0f, true));
        x[2] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp8(d1, 1.0f, false));
        x[3] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp8(d1, 1.0f, true));
    }
    const half2v K = u32_as_h2(k2), C = u32_as_h2(c2);
#pragma unroll
    for (int i = 0; i < 4; ++i) out[i] = h2_as_u32(__builtin_elementwise_fma(u32_as_h2(x[i]), K, C));
}

typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

// The four three-bit codes in bits 0-11 of t, one per byte (code k in bits
// 0-2 of byte k, the other bits zero), as v_perm selectors; bits of t above
// 11 are ignored.  One packed shift makes the 16-bit lanes bits 0-15 and
// 6-15 of t (codes 0 and 2 at bit 0 of their lane, codes 1 and 3 at bit 3);
// a shift of the word by 5 moves codes 1 and 3 to bytes 1 and 3, and the
// masks keep each code's three bits.
__device__ __forceinline__ uint32_t spread3x4(uint32_t t)
{
    const unsigned short s = (unsigned short)t;
    const uint32_t y = __builtin_bit_cast(uint32_t, u16x2{s, s} >> u16x2{0, 6});
    return (y & 0x00070007u) | ((y << 5) & 0x07000700u);
}

// Sixteen three-bit IF3 codes (48 bits) -> 8 FP16 operand pairs: 3 q (FP) or
// 4 q (INT), times Delta (at most 6 significant bits, exact).  Codes 0-7 use
// (is_int0, k20), codes 8-15 (is_int1, k21): the same for block size 16.
// Each run of 4 codes is spread to bytes, one v_perm looks up the E4M3 byte
// of its folded value (3 x E2M0 sign-magnitude, or 4 x INT3 two's
// complement -- small integers, exact in E4M3), the FP8 converter turns
// it into FP16 and one FP16 multiply applies Delta (k2 = Delta in both
// halves; the product has at most 6 significant bits).
__device__ __forceinline__ void decode_if3_group(uint64_t bitsv, bool is_int0, uint32_t k20, bool is_int1,
                                                 uint32_t k21, uint32_t (&out)[8])
{
    // bytes 0..7 = code 0..7: FP {0, 3, 6, 12, -0, -3, -6, -12}; INT {0, 4, 8, 12, -16, -12, -8, -4}
    constexpr uint32_t kFpLo = 0x544C4400u, kFpHi = 0xD4CCC480u;
    constexpr uint32_t kIntLo = 0x54504800u, kIntHi = 0xC8D0D4D8u;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const bool is_int = q < 2 ? is_int0 : is_int1;
        const half2v K = u32_as_h2(q < 2 ? k20 : k21);
        const uint32_t sel = spread3x4((uint32_t)(bitsv >> (12 * q)));
        const uint32_t e = __builtin_amdgcn_perm(is_int ? kIntHi : kFpHi, is_int ? kIntLo : kFpLo, sel);
        out[2 * q] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp8(e, 1.0f, false) * K);
        out[2 * q + 1] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp8(e, 1.0f, true) * K);
    }
}

// Sixteen six-bit IF6 codes (96 bits in w[0..2], code j at bits 6j) -> 8
// FP16 operand pairs: Fold::FP * q (FP, sign-magnitude ExMy) or Fold::INT * q
// (INT6 two's complement), times Delta, rounded once to FP16.  FP codes go
// through the gfx950 FP6 converter (E2M3: fp6, E3M2: bf6; 32 codes per
// instruction, the upper 16 unused) to exact FP16 values; INT codes become
// FP16 exactly through the bits of 1056 + q (int6_pair); one FP16 multiply by
// the exact fold constant (Fold * Delta has at most 9 significant bits)
// rounds the product once, as the FP32 product rounded to FP16 would.
typedef int v6i32 __attribute__((ext_vector_type(6)));
typedef _Float16 v32f16 __attribute__((ext_vector_type(32)));

// Codes 2i and 2i + 1 of an INT6 group as an exact FP16 pair (q, q'): the
// pair's 12 bits lie in half HI of x, code 2i at bit S0 and code 2i + 1 at
// bit S1 of that half.  One packed shift moves each code to bit 0 of its
// lane; the mask keeps its six bits, and the exclusive or flips its sign bit
// (n ^ 32 = q + 32 in [0, 63]) and sets the exponent of 1024, whose ulp is 1:
// the lane reads 1056 + q, and one subtraction leaves q.
template <int HI, int S0, int S1>
__device__ __forceinline__ half2v int6_pair(uint32_t x)
{
    const unsigned short s = HI ? (unsigned short)(x >> 16) : (unsigned short)x;
    const u16x2 v = u16x2{s, s} >> u16x2{(unsigned short)S0, (unsigned short)S1};
    const uint32_t b = (__builtin_bit_cast(uint32_t, v) & 0x003F003Fu) ^ 0x64206420u;
    return __builtin_bit_cast(half2v, b) - half2v{(_Float16)1056.0f, (_Float16)1056.0f};
}

template <int FMT>
__device__ __forceinline__ void decode_if6_group(const uint32_t* w, bool is_int, uint32_t k2, uint32_t (&out)[8])
{
    // k2 = Delta in both halves (exact FP16); the folds are exact FP16 too
    const half2v D = u32_as_h2(k2);
    const half2v KF = D * half2v{(_Float16)Fold<FMT>::FP, (_Float16)Fold<FMT>::FP};
    const half2v KI = D * half2v{(_Float16)Fold<FMT>::INT, (_Float16)Fold<FMT>::INT};
    const uint32_t im = 0u - (uint32_t)is_int;  // all-ones in an INT group: branch-free select
    const half2v KS = u32_as_h2((h2_as_u32(KI) & im) | (h2_as_u32(KF) & ~im));
    const v6i32 src = {(int)w[0], (int)w[1], (int)w[2], 0, 0, 0};
    v32f16 f;
    if constexpr (Fmt<FMT>::EB == 2)
        f = __builtin_amdgcn_cvt_scalef32_pk32_f16_fp6(src, 1.0f);
    else
        f = __builtin_amdgcn_cvt_scalef32_pk32_f16_bf6(src, 1.0f);
    // pair i = codes 2i, 2i + 1 at bits 12 i .. 12 i + 11: pairs 0, 3, 4 and
    // 7 lie in one half of a word; xa = bits 8-39 holds pairs 1 and 2, xb =
    // bits 56-87 pairs 5 and 6
    const uint32_t xa = __builtin_amdgcn_alignbit(w[1], w[0], 8);
    const uint32_t xb = __builtin_amdgcn_alignbit(w[2], w[1], 24);
    half2v hv[8];
    hv[0] = int6_pair<0, 0, 6>(w[0]);
    hv[1] = int6_pair<0, 4, 10>(xa);
    hv[2] = int6_pair<1, 0, 6>(xa);
    hv[3] = int6_pair<0, 4, 10>(w[1]);
    hv[4] = int6_pair<1, 0, 6>(w[1]);
    hv[5] = int6_pair<0, 4, 10>(xb);
    hv[6] = int6_pair<1, 0, 6>(xb);
    hv[7] = int6_pair<1, 4, 10>(w[2]);
    // the group's own pair and constant, then one rounding of their product
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const half2v fv = {f[2 * i], f[2 * i + 1]};
        const uint32_t x = (h2_as_u32(hv[i]) & im) | (h2_as_u32(fv) & ~im);
        out[i] = h2_as_u32(u32_as_h2(x) * KS);
    }
}

// ------------------------------------------------- single-conversion decode
// Shared by the fast kernel and the general one for 4-bit codes.
namespace dec {

// Fold constants of the two groups whose scale bytes are the low and high
// byte of sw, one half each: the operand is K x + C, x the converted code.
//   IF4 FP group : K = 14 Delta, C = 0 (x = E2M1 value times 2^-6)
//   IF4 INT group: K = 96 Delta, C = -1.5 Delta (x = (q + 8) 2^-9)
//   NVFP4        : K = Delta, C = 0 (x = E2M1 value)
//   NVINT4       : K = 128 Delta, C = -2 Delta (every group INT)
// For IF4 the E4M3 conversion keeps the indicator bit as the sign (d = -Delta
// for INT groups), so max(14 d, -96 d) and min(1.5 d, 0) select the
// constants without masks; C != 0 marks an INT group (an INT group with
// Delta = 0 decodes to zeros either way).
struct KC {
    half2v K, C;
};

template <int FMT>
__device__ __forceinline__ KC pair_kc(uint32_t sw)
{
    KC r;
    if constexpr (Fmt<FMT>::BITS == 3) {
        // IF3: K = Delta (the folds 3 and 4 live in the code tables), C = the
        // signed Delta, negative exactly for INT groups (only its sign is used)
        r.K = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(sw & 0x7F7Fu, 1.0f, false);
        r.C = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(sw, 1.0f, false);
    } else if constexpr (Fmt<FMT>::KIND == kKindInt) {
        const half2v d = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(sw & 0x7F7Fu, 1.0f, false);
        const half2v ki = {(_Float16)128.0f, (_Float16)128.0f}, cn = {(_Float16)-2.0f, (_Float16)-2.0f};
        r.K = d * ki;
        r.C = d * cn;
    } else if constexpr (Fmt<FMT>::ADAPTIVE) {
        const half2v d = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(sw, 1.0f, false);
        constexpr float kf = Fold<FMT>::FP * 64.0f;
        const half2v f = {(_Float16)kf, (_Float16)kf};
        const half2v fi = {(_Float16)-96.0f, (_Float16)-96.0f};
        const half2v c = {(_Float16)1.5f, (_Float16)1.5f};
        const half2v z = {(_Float16)0.0f, (_Float16)0.0f};
        r.K = __builtin_elementwise_max(d * f, d * fi);
        r.C = __builtin_elementwise_min(d * c, z);
    } else {
        const half2v f = {(_Float16)Fold<FMT>::FP, (_Float16)Fold<FMT>::FP};
        r.K = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(sw & 0x7F7Fu, 1.0f, false) * f;
        r.C = half2v{(_Float16)0.0f, (_Float16)0.0f};
    }
    return r;
}

// Per-group selector of the IF4 byte mapping: M = all ones, P = 0 for an INT
// group, M = 0, P = 2 for an FP group (unused by the other formats).  M is
// the sign of the group's C (negative exactly for INT groups; a zero INT
// scale gives C = -0 or +0, and K = 0 makes the group zero either way).
struct TypeSel {
    uint32_t M, P;
};

template <int FMT, int HS>
__device__ __forceinline__ TypeSel type_sel(const KC& kc)
{
    if constexpr (Fmt<FMT>::ADAPTIVE) {
        const int32_t cb = (int32_t)h2_as_u32(kc.C);
        const uint32_t m = (uint32_t)(HS ? (cb >> 31) : ((cb << 16) >> 31));
        return TypeSel{m, ~m & 2u};
    } else {
        return TypeSel{0u, 0u};
    }
}

// IF4 codes as E4M3 bytes, one code per byte (d holds a code in the low
// nibble of each byte).  FP group: the sign goes to bit 7 and the three
// magnitude bits to bits 2..4, which is the E4M3 pattern of the E2M1 value
// times 2^-6 (subnormal 0.5 included).  INT group: n ^ 8, the E4M3 pattern
// of (q + 8) 2^-9.  Both types thus share one conversion per two codes.
__device__ __forceinline__ uint32_t if4_bytes(uint32_t d, const TypeSel& ts)
{
    const uint32_t a = d & 0x07070707u;
    const uint32_t sg = (d ^ ts.M) & 0x08080808u;
    return ((sg << ts.P) | a) << ts.P;
}

// Empty asm statements that pin a stage's results to a program point: the
// slice schedule below places each decode stage between two MFMAs, and
// without them instruction selection would sink every stage to the last
// use of its results.
template <bool ON> __device__ __forceinline__ void pin(uint32_t& a)
{
    if constexpr (ON) asm volatile("" : "+v"(a));
}
template <bool ON> __device__ __forceinline__ void pin4(uint32_t (&a)[4])
{
    if constexpr (ON) asm volatile("" : "+v"(a[0]), "+v"(a[1]), "+v"(a[2]), "+v"(a[3]));
}

// Decode of one dword w of eight 4-bit codes (code 2i in the low nibble of
// byte i) into four FP16 operand pairs, in four stages of a few VALU
// operations each.  The E4M3 paths (IF4, NVINT4) convert the even codes
// (low nibbles) and the odd codes (high nibbles) as two byte vectors, so the
// pairs come out as (0, 2), (4, 6), (1, 3), (5, 7); NVFP4 converts nibble
// pairs in place: (0, 1), (2, 3), (4, 5), (6, 7).  Both operands of a GEMM
// are decoded alike, so either order is the same contraction over K.
//   s1: even codes to bytes (IF4, NVINT4) or the E2M1 conversions (NVFP4)
//   s2: odd codes to bytes
//   s3: E4M3 conversions
//   s4: K x + C
struct WordDec {
    uint32_t d0, d1;
    uint32_t x[4];
    uint32_t w, tlo, thi;   // IF3: the word and its code tables
};

// IF3 words: 8 three-bit codes, code i at bits 3i (24 bits; what lies above
// bit 23 is ignored).  The selector bytes of four codes (one code per byte)
// index a v_perm table of the E4M3 bytes of their folded values: 3 x E2M0
// (sign-magnitude) for FP groups, 4 x INT3 (two's complement) for INT
// groups -- small integers, exact in E4M3 and after the FP8 conversion in
// FP16; one FP16 multiply by Delta then gives the operand (at most 6
// significant bits, exact).
// bytes 0..7 = code 0..7: FP {0, 3, 6, 12, -0, -3, -6, -12}; INT {0, 4, 8, 12, -16, -12, -8, -4}
constexpr uint32_t kIf3FpLo = 0x544C4400u, kIf3FpHi = 0xD4CCC480u;
constexpr uint32_t kIf3IntLo = 0x54504800u, kIf3IntHi = 0xC8D0D4D8u;

template <int FMT, bool PIN>
__device__ __forceinline__ void wd_s1(uint32_t w, const TypeSel& ts, WordDec& s)
{
    if constexpr (Fmt<FMT>::BITS == 3) {
        s.w = w;
        s.d0 = spread3x4(w);
        pin<PIN>(s.d0);
    } else if constexpr (Fmt<FMT>::KIND == kKindInt) {
        s.d0 = (w & 0x0F0F0F0Fu) ^ 0x08080808u;
        pin<PIN>(s.d0);
    } else if constexpr (Fmt<FMT>::ADAPTIVE) {
        s.d0 = if4_bytes(w, ts);
        pin<PIN>(s.d0);
    } else {
        s.x[0] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 1.0f, 0));
        s.x[1] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 1.0f, 1));
        s.x[2] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 1.0f, 2));
        s.x[3] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 1.0f, 3));
        pin4<PIN>(s.x);
    }
}

template <int FMT, bool PIN>
__device__ __forceinline__ void wd_s2(uint32_t w, const TypeSel& ts, WordDec& s)
{
    if constexpr (Fmt<FMT>::BITS == 3) {
        // the group's table (M: all ones for an INT group), codes 0-3
        s.tlo = kIf3FpLo ^ ((kIf3FpLo ^ kIf3IntLo) & ts.M);
        s.thi = kIf3FpHi ^ ((kIf3FpHi ^ kIf3IntHi) & ts.M);
        const uint32_t e = __builtin_amdgcn_perm(s.thi, s.tlo, s.d0);
        s.x[0] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp8(e, 1.0f, false));
        s.x[1] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp8(e, 1.0f, true));
        if constexpr (PIN) asm volatile("" : "+v"(s.x[0]), "+v"(s.x[1]), "+v"(s.tlo), "+v"(s.thi));
    } else if constexpr (Fmt<FMT>::KIND == kKindInt || Fmt<FMT>::ADAPTIVE) {
        const uint32_t w4 = w >> 4;
        if constexpr (Fmt<FMT>::KIND == kKindInt) s.d1 = (w4 & 0x0F0F0F0Fu) ^ 0x08080808u;
        else s.d1 = if4_bytes(w4, ts);
        pin<PIN>(s.d1);
    }
}

template <int FMT, bool PIN>
__device__ __forceinline__ void wd_s3(WordDec& s)
{
    if constexpr (Fmt<FMT>::BITS == 3) {
        s.d1 = spread3x4(s.w >> 12);   // codes 4-7
        pin<PIN>(s.d1);
    } else if constexpr (Fmt<FMT>::KIND == kKindInt || Fmt<FMT>::ADAPTIVE) {
        s.x[0] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp8(s.d0, 1.0f, false));
        s.x[1] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp8(s.d0, 1.0f, true));
        s.x[2] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp8(s.d1, 1.0f, false));
        s.x[3] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp8(s.d1, 1.0f, true));
        pin4<PIN>(s.x);
    }
}

template <int FMT, int HS, bool PIN>
__device__ __forceinline__ void wd_s4(const WordDec& s, const KC& kc, uint32_t (&out)[4])
{
    const half2v K2 = {kc.K[HS], kc.K[HS]};
    if constexpr (Fmt<FMT>::BITS == 3) {
        const uint32_t e = __builtin_amdgcn_perm(s.thi, s.tlo, s.d1);
        const half2v x2 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(e, 1.0f, false);
        const half2v x3 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(e, 1.0f, true);
        out[0] = h2_as_u32(u32_as_h2(s.x[0]) * K2);
        out[1] = h2_as_u32(u32_as_h2(s.x[1]) * K2);
        out[2] = h2_as_u32(x2 * K2);
        out[3] = h2_as_u32(x3 * K2);
    } else {
        const half2v C2 = {kc.C[HS], kc.C[HS]};
#pragma unroll
        for (int i = 0; i < 4; ++i) out[i] = h2_as_u32(__builtin_elementwise_fma(u32_as_h2(s.x[i]), K2, C2));
    }
    pin4<PIN>(out);
}

// Two words w[0], w[1] of a block-size-8 unit: word 0 with the constants of
// half 0 of kc, word 1 with half 1.
template <int FMT>
__device__ __forceinline__ void decode_words_kc2(const uint32_t* w, const KC& kc, uint32_t (&out)[8])
{
    const TypeSel t0 = type_sel<FMT, 0>(kc), t1 = type_sel<FMT, 1>(kc);
    WordDec a, b;
    uint32_t o0[4], o1[4];
    wd_s1<FMT, false>(w[0], t0, a);
    wd_s2<FMT, false>(w[0], t0, a);
    wd_s3<FMT, false>(a);
    wd_s4<FMT, 0, false>(a, kc, o0);
    wd_s1<FMT, false>(w[1], t1, b);
    wd_s2<FMT, false>(w[1], t1, b);
    wd_s3<FMT, false>(b);
    wd_s4<FMT, 1, false>(b, kc, o1);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        out[i] = o0[i];
        out[4 + i] = o1[i];
    }
}

// One group (two dwords w[0], w[1]) with the constants of half HS of kc,
// all stages in a row.
template <int FMT, int HS>
__device__ __forceinline__ void decode_group_kc(const uint32_t* w, const KC& kc, uint32_t (&out)[8])
{
    const TypeSel ts = type_sel<FMT, HS>(kc);
    WordDec a, b;
    uint32_t o0[4], o1[4];
    wd_s1<FMT, false>(w[0], ts, a);
    wd_s2<FMT, false>(w[0], ts, a);
    wd_s3<FMT, false>(a);
    wd_s4<FMT, HS, false>(a, kc, o0);
    wd_s1<FMT, false>(w[1], ts, b);
    wd_s2<FMT, false>(w[1], ts, b);
    wd_s3<FMT, false>(b);
    wd_s4<FMT, HS, false>(b, kc, o1);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        out[i] = o0[i];
        out[4 + i] = o1[i];
    }
}

}  // namespace dec

// ------------------------------------------------------------ raw chunks
// A: one lane's 32 k-values of one row for one step (2 groups);
// B: one thread's 64 k-values of one row (4 groups).  IF3 keeps 6-byte groups.
// Scale bytes of a chunk: one per 16 values, two for block size 8.
template <int FMT> using ScaleBits = typename std::conditional<Fmt<FMT>::G == 8, uint64_t, uint32_t>::type;
template <int FMT> struct RawA { uint32_t w[4]; ScaleBits<FMT> sb; };
template <> struct RawA<IFQ_FMT_IF3> { uint16_t h[6]; uint32_t sb; };
template <> struct RawA<IFQ_FMT_IF3_BS8> { uint16_t h[6]; uint64_t sb; };
template <int FMT> struct RawB { uint32_t w[8]; ScaleBits<FMT> sb; };
template <> struct RawB<IFQ_FMT_IF3> { uint16_t h[12]; uint32_t sb; };
template <> struct RawB<IFQ_FMT_IF3_BS8> { uint16_t h[12]; uint64_t sb; };
template <> struct RawA<IFQ_FMT_IF6_E2M3> { uint32_t w[6]; uint32_t sb; };
template <> struct RawA<IFQ_FMT_IF6_E3M2> { uint32_t w[6]; uint32_t sb; };
template <> struct RawB<IFQ_FMT_IF6_E2M3> { uint32_t w[12]; uint32_t sb; };
template <> struct RawB<IFQ_FMT_IF6_E3M2> { uint32_t w[12]; uint32_t sb; };

// Load `ng` groups (2 or 4) of one row starting at group g0 into words /
// halves.  Interior tiles (EDGE = false) load without guards.
template <int FMT, bool EDGE, int NG>
__device__ __forceinline__ void load_groups(const uint8_t* __restrict__ codes,
                                            const uint8_t* __restrict__ scales, int64_t row,
                                            int64_t nrows, int64_t gpr, int64_t g0,
                                            uint32_t* w, uint16_t* h, ScaleBits<FMT>& sb)
{
    constexpr int BITS = Fmt<FMT>::BITS;
    constexpr int SPG = Fmt<FMT>::G == 8 ? 2 : 1;  // scale bytes per 16 values
    const uint8_t* cp = codes + (row * gpr + g0) * (2 * BITS);
    const uint8_t* sp = scales + (row * gpr + g0) * SPG;
    if constexpr (BITS == 4 && !EDGE) {
        const uint4 a = *reinterpret_cast<const uint4*>(cp);
        w[0] = a.x; w[1] = a.y; w[2] = a.z; w[3] = a.w;
        if constexpr (NG == 4) {
            const uint4 b = *reinterpret_cast<const uint4*>(cp + 16);
            w[4] = b.x; w[5] = b.y; w[6] = b.z; w[7] = b.w;
        }
        if constexpr (SPG == 2 && NG == 4) {
            const uint32_t* sp4 = reinterpret_cast<const uint32_t*>(sp);  // 4-byte aligned
            sb = (uint64_t)sp4[0] | ((uint64_t)sp4[1] << 32);
        } else if constexpr (SPG == 2 || NG == 4) {
            sb = *reinterpret_cast<const uint32_t*>(sp);
        } else {
            sb = *reinterpret_cast<const uint16_t*>(sp);
        }
    } else if constexpr (BITS == 6 && !EDGE) {
        // interior tiles (K % 128 == 0, 16-byte aligned codes): a row's NG
        // groups are 12 NG contiguous bytes, 16-byte aligned for NG = 4 and
        // 8-byte aligned for NG = 2
        if constexpr (NG == 4) {
#pragma unroll
            for (int i = 0; i < 3; ++i) {
                const uint4 v = reinterpret_cast<const uint4*>(cp)[i];
                w[4 * i] = v.x; w[4 * i + 1] = v.y; w[4 * i + 2] = v.z; w[4 * i + 3] = v.w;
            }
            sb = *reinterpret_cast<const uint32_t*>(sp);
        } else {
#pragma unroll
            for (int i = 0; i < 3; ++i) {
                const uint2 v = reinterpret_cast<const uint2*>(cp)[i];
                w[2 * i] = v.x; w[2 * i + 1] = v.y;
            }
            sb = *reinterpret_cast<const uint16_t*>(sp);
        }
    } else if constexpr (BITS == 3 && !EDGE) {
        // interior tiles: 6 NG contiguous bytes, 8-byte aligned for NG = 4
        // and 4-byte aligned for NG = 2 (8-byte pieces, then dwords)
        if constexpr (NG == 4) {
#pragma unroll
            for (int i = 0; i < 3; ++i) {
                const uint2 v = reinterpret_cast<const uint2*>(cp)[i];
                h[4 * i] = (uint16_t)v.x; h[4 * i + 1] = (uint16_t)(v.x >> 16);
                h[4 * i + 2] = (uint16_t)v.y; h[4 * i + 3] = (uint16_t)(v.y >> 16);
            }
        } else {
            const uint32_t* c4 = reinterpret_cast<const uint32_t*>(cp);
#pragma unroll
            for (int i = 0; i < 3; ++i) { h[2 * i] = (uint16_t)c4[i]; h[2 * i + 1] = (uint16_t)(c4[i] >> 16); }
        }
        // scale bytes as for 4-bit codes (two per 16 values with block size 8)
        if constexpr (SPG == 2 && NG == 4) {
            const uint32_t* sp4 = reinterpret_cast<const uint32_t*>(sp);
            sb = (uint64_t)sp4[0] | ((uint64_t)sp4[1] << 32);
        } else if constexpr (SPG == 2 || NG == 4) {
            sb = *reinterpret_cast<const uint32_t*>(sp);
        } else {
            sb = *reinterpret_cast<const uint16_t*>(sp);
        }
    } else {
        const bool row_ok = row < nrows;
        sb = 0;
#pragma unroll
        for (int g = 0; g < NG; ++g) {
            const bool ok = row_ok && g0 + g < gpr;
            if constexpr (BITS == 4) {
                const uint2 t = ok ? *reinterpret_cast<const uint2*>(cp + 8 * g) : make_uint2(0, 0);
                w[2 * g] = t.x;
                w[2 * g + 1] = t.y;
            } else if constexpr (BITS == 6) {
                const uint32_t* p = reinterpret_cast<const uint32_t*>(cp + 12 * g);
                w[3 * g] = ok ? p[0] : 0u;
                w[3 * g + 1] = ok ? p[1] : 0u;
                w[3 * g + 2] = ok ? p[2] : 0u;
            } else {
                const uint16_t* p = reinterpret_cast<const uint16_t*>(cp + 6 * g);
                h[3 * g] = ok ? p[0] : (uint16_t)0;
                h[3 * g + 1] = ok ? p[1] : (uint16_t)0;
                h[3 * g + 2] = ok ? p[2] : (uint16_t)0;
            }
            if constexpr (SPG == 2) {
                sb |= (ok ? (ScaleBits<FMT>)sp[2 * g] | ((ScaleBits<FMT>)sp[2 * g + 1] << 8) : 0) << (16 * g);
            } else {
                sb |= (ok ? (uint32_t)sp[g] : 0u) << (8 * g);
            }
        }
    }
}

template <int FMT, bool EDGE>
__device__ __forceinline__ void load_a(const uint8_t* __restrict__ codes, const uint8_t* __restrict__ scales,
                                       int64_t row, int64_t nrows, int64_t gpr, int64_t g0, RawA<FMT>& r)
{
    if constexpr (Fmt<FMT>::BITS != 3)
        load_groups<FMT, EDGE, 2>(codes, scales, row, nrows, gpr, g0, r.w, nullptr, r.sb);
    else
        load_groups<FMT, EDGE, 2>(codes, scales, row, nrows, gpr, g0, nullptr, r.h, r.sb);
}

template <int FMT, bool EDGE>
__device__ __forceinline__ void load_b(const uint8_t* __restrict__ codes, const uint8_t* __restrict__ scales,
                                       int64_t row, int64_t nrows, int64_t gpr, int64_t g0, RawB<FMT>& r)
{
    if constexpr (Fmt<FMT>::BITS != 3)
        load_groups<FMT, EDGE, 4>(codes, scales, row, nrows, gpr, g0, r.w, nullptr, r.sb);
    else
        load_groups<FMT, EDGE, 4>(codes, scales, row, nrows, gpr, g0, nullptr, r.h, r.sb);
}

// Decode group g of a raw chunk (whose scale bytes are sb) into 8 operand pairs.
template <int FMT>
__device__ __forceinline__ void decode_group(const uint32_t* w, const uint16_t* h, ScaleBits<FMT> sb, int g,
                                             uint32_t (&out)[8])
{
    if constexpr (Fmt<FMT>::BITS == 4) {
        // 4-bit codes: one conversion per two codes for both group types
        // (dec::); with block size 8 the two scale bytes of these 16 values
        // hold the constants of codes 0-7 (low byte, word 0) and 8-15 (high
        // byte, word 1), with block size 16 the pair of groups g & ~1, g | 1
        if constexpr (Fmt<FMT>::G == 8) {
            const dec::KC kc = dec::pair_kc<FMT>((uint32_t)(sb >> (16 * g)) & 0xFFFFu);
            dec::decode_words_kc2<FMT>(w + 2 * g, kc, out);
        } else {
            const dec::KC kc = dec::pair_kc<FMT>((uint32_t)(sb >> (16 * (g >> 1))) & 0xFFFFu);
            if (g & 1)
                dec::decode_group_kc<FMT, 1>(w + 2 * g, kc, out);
            else
                dec::decode_group_kc<FMT, 0>(w + 2 * g, kc, out);
        }
        return;
    } else if constexpr (Fmt<FMT>::G == 8) {
        // block size 8: the two scale bytes of these 16 values hold the
        // constants of codes 0-7 (low byte) and 8-15 (high byte)
        const uint32_t sw = (uint32_t)(sb >> (16 * g)) & 0xFFFFu;
        uint32_t K, Cb;
        pair_scales<FMT>(sw, K, Cb);
        const bool i0 = Fmt<FMT>::ADAPTIVE && ((sw >> 7) & 1u), i1 = Fmt<FMT>::ADAPTIVE && ((sw >> 15) & 1u);
        {
            const uint64_t bitsv = (uint64_t)h[3 * g] | ((uint64_t)h[3 * g + 1] << 16) |
                                   ((uint64_t)h[3 * g + 2] << 32);
            decode_if3_group(bitsv, i0, bcast_lo(K), i1, bcast_hi(K), out);
        }
        return;
    } else {
    const uint32_t sw = (sb >> (16 * (g >> 1))) & 0xFFFFu;
    uint32_t K, Cb;
    pair_scales<FMT>(sw, K, Cb);
    const uint32_t k2 = (g & 1) ? bcast_hi(K) : bcast_lo(K);
    const uint32_t c2 = (g & 1) ? bcast_hi(Cb) : bcast_lo(Cb);
    const bool is_int = Fmt<FMT>::ADAPTIVE && ((sb >> (8 * g + 7)) & 1u);
    if constexpr (Fmt<FMT>::BITS == 4) {
        uint32_t o0[4], o1[4];
        decode_word<FMT>(w[2 * g], is_int, k2, c2, o0);
        decode_word<FMT>(w[2 * g + 1], is_int, k2, c2, o1);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            out[i] = o0[i];
            out[4 + i] = o1[i];
        }
    } else if constexpr (Fmt<FMT>::BITS == 6) {
        decode_if6_group<FMT>(w + 3 * g, is_int, k2, out);
    } else {
        const uint64_t bitsv = (uint64_t)h[3 * g] | ((uint64_t)h[3 * g + 1] << 16) |
                               ((uint64_t)h[3 * g + 2] << 32);
        decode_if3_group(bitsv, is_int, k2, is_int, k2, out);
    }
    }
}

// Decode B group g of thread t's row into the LDS stage (natural k order).
template <int FMT>
__device__ __forceinline__ void decode_b(const RawB<FMT>& r, _Float16* stage, int t, int g)
{
    uint32_t v[8];
    if constexpr (Fmt<FMT>::BITS != 3)
        decode_group<FMT>(r.w, nullptr, r.sb, g, v);
    else
        decode_group<FMT>(nullptr, r.h, r.sb, g, v);
    uint4* p = reinterpret_cast<uint4*>(stage + t * kPitch + g * kGroup);
    p[0] = make_uint4(v[0], v[1], v[2], v[3]);
    p[1] = make_uint4(v[4], v[5], v[6], v[7]);
}

// Decode A group gg (0 or 1) of a lane's row chunk into the fragments of K
// slices 2 gg and 2 gg + 1.
template <int FMT>
__device__ __forceinline__ void decode_a(const RawA<FMT>& r, int gg, half8& f0, half8& f1)
{
    uint32_t v[8];
    if constexpr (Fmt<FMT>::BITS != 3)
        decode_group<FMT>(r.w, nullptr, r.sb, gg, v);
    else
        decode_group<FMT>(nullptr, r.h, r.sb, gg, v);
    uint4 a = make_uint4(v[0], v[1], v[2], v[3]), b = make_uint4(v[4], v[5], v[6], v[7]);
    f0 = __builtin_bit_cast(half8, a);
    f1 = __builtin_bit_cast(half8, b);
}

__device__ __forceinline__ void read_bfrags(const _Float16* Bs, int kk, int lane, half8 (&bf)[8])
{
    const int kofs = 32 * (lane >> 5) + 8 * kk;
#pragma unroll
    for (int j = 0; j < 8; ++j)
        bf[j] = *reinterpret_cast<const half8*>(Bs + (j * 32 + (lane & 31)) * kPitch + kofs);
}

// Register state carried across K steps.  Slots alternate with the step
// parity P (the loop is unrolled by two so that no slot is ever copied): raw
// A chunks of steps s (slot P) and s + 1 (slot P ^ 1); raw B of step s + 2
// (slot P, decoded during step s) and s + 3 (slot P ^ 1, loading).
template <int FMT, bool EDGE> struct TileState {
    RawA<FMT> a[2][2];     // [slot][row block i]
    RawB<FMT> b[2];        // [slot]
    half8 af[2][2][2];     // [group gg][row block i][slice parity]
    half8 bf[2][8];        // B fragments, double buffered over slices
};

// Wait for this wavefront's LDS writes, then meet the other wavefronts.
// (A full __syncthreads() would also wait for every outstanding global load.)
__device__ __forceinline__ void lds_barrier()
{
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// One 64-wide K step s.  B is staged in a ring of three LDS buffers: step s
// reads stage s % 3, decodes B of step s + 2 into stage (s + 2) % 3 and, in
// its last slice, prefetches the first B fragments of step s + 1 from stage
// (s + 1) % 3, which the barrier closing step s - 1 made visible; so no
// slice waits on a fresh LDS read after the barrier.  Slice kk multiplies
// the B fragments of the slice with A fragments in registers while one B
// group and one A decode unit are produced -- this step's second A group
// (slices 2, 3) at kk = 0, 1 and the next step's first group (slices 0, 1) at
// kk = 2, 3.  Loads beyond the last step are clamped to it (harmless extra
// work that keeps the loop free of branches).
template <int FMT, bool EDGE, int P>
__device__ __forceinline__ void gemm_step(int s, int nsteps, const uint8_t* __restrict__ a_codes,
                                          const uint8_t* __restrict__ a_scales,
                                          const uint8_t* __restrict__ b_codes,
                                          const uint8_t* __restrict__ b_scales, int64_t M,
                                          int64_t N, int64_t gpr, int64_t arow0, int64_t n0,
                                          TileState<FMT, EDGE>& st, const _Float16* Bs,
                                          const _Float16* Bn, _Float16* Bd, floatx16 (&acc)[2][8])
{
    const int t = threadIdx.x;
    const int lane = t & 63;
    const int h = lane >> 5;
    const int64_t g3 = (int64_t)min(s + 3, nsteps - 1) * kGroupsPerStep;
    const int64_t g2 = (int64_t)min(s + 2, nsteps - 1) * kGroupsPerStep;
    load_b<FMT, EDGE>(b_codes, b_scales, n0 + t, N, gpr, g3, st.b[P ^ 1]);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
        const int f = kk & 1;
        if (kk < 3)
            read_bfrags(Bs, kk + 1, lane, st.bf[f ^ 1]);
        else
            read_bfrags(Bn, 0, lane, st.bf[f ^ 1]);
        decode_b<FMT>(st.b[P], Bd, t, kk);
        if (kk < 2) {
            decode_a<FMT>(st.a[P][kk], 1, st.af[1][kk][0], st.af[1][kk][1]);
        } else {
            if (kk == 2) {
                // this step's A chunks are fully decoded: refill them with step s + 2
#pragma unroll
                for (int i = 0; i < 2; ++i)
                    load_a<FMT, EDGE>(a_codes, a_scales, arow0 + 32 * i, M, gpr, g2 + 2 * h, st.a[P][i]);
            }
            decode_a<FMT>(st.a[P ^ 1][kk - 2], 0, st.af[0][kk - 2][0], st.af[0][kk - 2][1]);
        }
        const int gg = kk >> 1, par = kk & 1;
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 8; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(st.af[gg][i][par], st.bf[f][j], acc[i][j], 0, 0, 0);
        // VALU operations placed after each MFMA: the slice's decode spread
        // over its 16 MFMAs (IF6 and IF3 with block size 8 decode about 7 per
        // MFMA, the other formats of this kernel at most 6)
        constexpr int kValu = (Fmt<FMT>::BITS == 6 || (Fmt<FMT>::BITS == 3 && Fmt<FMT>::G == 8)) ? 8 : 6;
#pragma unroll
        for (int m = 0; m < 16; ++m) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x002, kValu, 0);
            if (m < 8) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            if (m == 3 || m == 7) __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
    }
    lds_barrier();
}

// Scale the accumulators by alpha_A alpha_B / (lambda fold_FP)^2 and store
// the 256 x 256 tile (lane layout of v_mfma_f32_32x32x16_f16: column
// lane % 32, rows 8 (e / 4) + 4 (lane / 32) + e % 4 of each 32 x 32 block).
template <int FMT, bool OUT_BF16, bool EDGE>
__device__ __forceinline__ void store_tile(const floatx16 (&acc)[2][8], const float* __restrict__ a_ts,
                                           const float* __restrict__ b_ts, int64_t M, int64_t N,
                                           void* __restrict__ C, int64_t ldc, int64_t m0, int64_t n0,
                                           bool add = false)
{
    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    const int h = lane >> 5;
    const float sc = (*a_ts * *b_ts) * Fold<FMT>::EPI;
    if constexpr (!OUT_BF16 && !EDGE) {
        if (add) {
            // one K half of a split tile: its share of the product, added into
            // the zeroed output by the hardware atomic
            float* c = static_cast<float*>(C);
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const int64_t n = n0 + j * 32 + (lane & 31);
#pragma unroll
                    for (int e = 0; e < 16; ++e) {
                        const int64_t m = m0 + 64 * wave + i * 32 + (e >> 2) * 8 + h * 4 + (e & 3);
                        unsafeAtomicAdd(c + m * ldc + n, acc[i][j][e] * sc);
                    }
                }
            return;
        }
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int64_t n = n0 + j * 32 + (lane & 31);
#pragma unroll
            for (int e = 0; e < 16; e += 2) {
                // elements e and e + 1 are rows m and m + 1 of column n
                const int64_t m = m0 + 64 * wave + i * 32 + (e >> 2) * 8 + h * 4 + (e & 3);
                const float v0 = acc[i][j][e] * sc, v1 = acc[i][j][e + 1] * sc;
                if constexpr (OUT_BF16) {
                    // both rounded to nearest even by one v_cvt_pk_bf16_f32; the
                    // second row is stored from the high half
                    const float2v v = {v0, v1};
                    const uint32_t u = __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2v));
                    uint16_t* c = static_cast<uint16_t*>(C);
                    if (!EDGE || (m < M && n < N)) c[m * ldc + n] = (uint16_t)u;
                    if (!EDGE || (m + 1 < M && n < N)) c[(m + 1) * ldc + n] = (uint16_t)(u >> 16);
                } else {
                    float* c = static_cast<float*>(C);
                    if (!EDGE || (m < M && n < N)) c[m * ldc + n] = v0;
                    if (!EDGE || (m + 1 < M && n < N)) c[(m + 1) * ldc + n] = v1;
                }
            }
        }
    }
}

template <int FMT, bool OUT_BF16, bool EDGE>
__device__ __forceinline__ void gemm_tile(const uint8_t* __restrict__ a_codes,
                                          const uint8_t* __restrict__ a_scales,
                                          const float* __restrict__ a_ts,
                                          const uint8_t* __restrict__ b_codes,
                                          const uint8_t* __restrict__ b_scales,
                                          const float* __restrict__ b_ts, int64_t M, int64_t N,
                                          int64_t K, void* __restrict__ C, int64_t ldc,
                                          int64_t m0, int64_t n0, _Float16 (*lds)[kStageHalves])
{
    const int64_t gpr = K / kGroup;
    // steps run in pairs; a padding step (EDGE tiles only: interior tiles have
    // K % 128 == 0) loads guarded, zero-filled groups and adds nothing
    const int nsteps = 2 * (int)((gpr + 2 * kGroupsPerStep - 1) / (2 * kGroupsPerStep));
    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    const int h = lane >> 5;
    const int64_t arow0 = m0 + 64 * wave + (lane & 31);  // row of block i is arow0 + 32 i

    floatx16 acc[2][8];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

    if (nsteps > 0) {
        TileState<FMT, EDGE> st;
        const int64_t g1 = (int64_t)min(1, nsteps - 1) * kGroupsPerStep;
        const int64_t g2 = (int64_t)min(2, nsteps - 1) * kGroupsPerStep;
        RawB<FMT> b0;
        load_b<FMT, EDGE>(b_codes, b_scales, n0 + t, N, gpr, 0, b0);
        load_b<FMT, EDGE>(b_codes, b_scales, n0 + t, N, gpr, g1, st.b[1]);
        load_b<FMT, EDGE>(b_codes, b_scales, n0 + t, N, gpr, g2, st.b[0]);
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            load_a<FMT, EDGE>(a_codes, a_scales, arow0 + 32 * i, M, gpr, 2 * h, st.a[0][i]);
            load_a<FMT, EDGE>(a_codes, a_scales, arow0 + 32 * i, M, gpr, g1 + 2 * h, st.a[1][i]);
        }
#pragma unroll
        for (int g = 0; g < kGroupsPerStep; ++g) {
            decode_b<FMT>(b0, lds[0], t, g);
            decode_b<FMT>(st.b[1], lds[1], t, g);
        }
#pragma unroll
        for (int i = 0; i < 2; ++i) decode_a<FMT>(st.a[0][i], 0, st.af[0][i][0], st.af[0][i][1]);
        lds_barrier();
        read_bfrags(lds[0], 0, lane, st.bf[0]);
        // stage indices of steps s, s + 1, s + 2
        int r0 = 0, r1 = 1, r2 = 2;
        for (int s = 0; s < nsteps; s += 2) {
            gemm_step<FMT, EDGE, 0>(s, nsteps, a_codes, a_scales, b_codes, b_scales, M, N, gpr, arow0,
                                    n0, st, lds[r0], lds[r1], lds[r2], acc);
            gemm_step<FMT, EDGE, 1>(s + 1, nsteps, a_codes, a_scales, b_codes, b_scales, M, N, gpr,
                                    arow0, n0, st, lds[r1], lds[r2], lds[r0], acc);
            // advance the ring by two steps
            const int n0r = r2, n1r = r0, n2r = r1;
            r0 = n0r;
            r1 = n1r;
            r2 = n2r;
        }
    }

    store_tile<FMT, OUT_BF16, EDGE>(acc, a_ts, b_ts, M, N, C, ldc, m0, n0);
}

// Tile of workgroup blockIdx.x.  Workgroup ids are dealt round robin to the
// 8 XCDs; they are remapped so that each XCD walks a contiguous range of tile
// ids, and tile ids are ordered in bands of 4 tile rows (column-major inside
// a band), so the 32 workgroups resident on one XCD form a 4 x 8 block of
// tiles that share A and B rows in its L2.
__device__ __forceinline__ void band_tile(int tile, int tiles_m, int tiles_n, int& tm, int& tn)
{
    constexpr int GM = 4;
    const int band = tile / (GM * tiles_n);
    const int first_m = band * GM;
    const int gm = min(tiles_m - first_m, GM);
    const int in_band = tile - band * GM * tiles_n;
    tm = first_m + in_band % gm;
    tn = in_band / gm;
}

__device__ __forceinline__ void tile_coords(int tiles_m, int tiles_n, int& tm, int& tn)
{
    const int nwg = gridDim.x;
    const int bid = blockIdx.x;
    const int tile = (nwg % 8 == 0) ? (bid % 8) * (nwg / 8) + bid / 8 : bid;
    band_tile(tile, tiles_m, tiles_n, tm, tn);
}

// Split tail (fast path, fp32 output): tiles [0, t_full) run whole, tiles
// [t_full, t_full + t_split) as two halves of K each, whose products are
// added into the zeroed output.  With t_full % 8 == 0 and t_split % 4 == 0,
// every XCD takes t_full / 8 whole tiles (a contiguous range, first) and
// t_split / 4 halves, so the halves fill the last round on every XCD;
// otherwise blocks take whole tiles, then halves, in order.  Returns the
// tile; half = -1 for a whole tile, else the K half.
__device__ __forceinline__ int split_tile(int t_full, int t_split, int& half)
{
    const int nwg = gridDim.x, bid = blockIdx.x;
    half = -1;
    if (t_split == 0) return (nwg % 8 == 0) ? (bid % 8) * (nwg / 8) + bid / 8 : bid;
    int j;
    if (t_full % 8 == 0 && t_split % 4 == 0) {
        const int x = bid % 8, p = bid / 8, fpx = t_full / 8;
        if (p < fpx) return x * fpx + p;
        j = x * (t_split / 4) + (p - fpx);
    } else {
        if (bid < t_full) return bid;
        j = bid - t_full;
    }
    half = j & 1;
    return t_full + (j >> 1);
}

// ------------------------------------------------------- fast interior path
// Interior tiles of 4-bit formats with K % 512 == 0 and 16-byte aligned
// operands.  Same tiling and operand values as above; what changes is how
// the packed operands reach the kernel.  Row-major codes give each row only
// 32 bytes per K step, so per-lane row loads touch a different cache line in
// every lane and every step (and scale bytes far more so).  Here operands
// arrive in line-sized, coalesced pieces:
//   B codes: two K steps (64 bytes per row) per chunk, copied straight into
//            LDS by global_load_lds (four lanes per row), two chunk slots;
//   scales : eight K steps (32 bytes per row, A and B) per chunk, the same
//            way, two slots;
//   A codes: 32 bytes per lane and chunk (both 16-byte halves of one row's
//            64 bytes are read by the lane pair that owns the row), straight
//            into registers, two slots.
// K order.  Within a 2-step chunk (8 groups), lane half h of every MFMA
// holds groups 4h .. 4h + 3; step j of the chunk uses groups 4h + 2j and
// 4h + 2j + 1 (slices 0, 1 and 2, 3).  The B stage of step j therefore holds,
// per row, groups 2j, 2j + 1 (half 0) and 4 + 2j, 5 + 2j (half 1).
// Loads are issued from inline assembly and waited for with explicit
// vmcnt counts (the compiler's own tracking would wait for every copy into
// LDS before any LDS access); the counts below follow the fixed issue order
// of the four-step loop body:
//   odd step,  slice 0: 4 copies of B codes (+ 2 copies of scales at step 1)
//   odd step,  slice 2: 4 loads of A codes
// Decoded B stages are 128-byte rows whose 16-byte pieces are XOR-swizzled
// by swz8(row) = (row % 8) ^ ((row / 8) % 2), raw B rows (64 bytes) by
// swz4(row) = ((row / 2) % 4) ^ ((row / 8) % 2): both keep the row-wise
// accesses (consecutive lanes on consecutive rows) free of bank conflicts
// whether a 128-bit access is served 8 lanes over 32 banks or 16 lanes over
// 64 banks at a time.
namespace fast {

using namespace dec;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr int kStageBytes = kBN * kBK * 2;       // decoded B stage, 32 KiB
constexpr int kRawBytes = kBN * 64;              // B codes of one chunk, 16 KiB
// Code bytes of a row per 2-step chunk and of a B chunk: 64 and 16 KiB for
// 4-bit codes, 48 and 12 KiB for IF3.
template <int BITS> constexpr int kChunkB = BITS == 3 ? 48 : 64;
template <int BITS> constexpr int kRawBytesF = kBN * kChunkB<BITS>;
constexpr int kSclBytes = (kBM + kBN) * 32;      // scales of one 8-step chunk, 16 KiB
constexpr int kSclB = kBM * 32;                  // offset of the B rows in a scale chunk

__device__ __forceinline__ int swz8(int row) { return (row & 7) ^ ((row >> 3) & 1); }
// IF3 raw rows (32 bytes of pieces 0 and 1): piece p at position p ^ swz2(row)
__device__ __forceinline__ int swz2(int row) { return (row >> 3) & 1; }
__device__ __forceinline__ int swz4(int row) { return ((row >> 1) & 3) ^ ((row >> 3) & 1); }

__device__ __forceinline__ uint32_t lds_off(const void* p)
{
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// 16 bytes per lane from global memory (wave-uniform base + this lane's
// 32-bit offset) into LDS at lds + 16 * lane (lds is wave-uniform).
__device__ __forceinline__ void copy16(const uint8_t* base, uint32_t voff, uint32_t lds)
{
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(base),
                 "s"(lds)
                 : "memory", "m0");
}

// 16 bytes per lane from base + voff + OFS into registers.
template <int OFS> __device__ __forceinline__ u32x4 load16(const uint8_t* base, uint32_t voff)
{
    u32x4 v;
    asm volatile("global_load_dwordx4 %0, %1, %2 offset:%3" : "=v"(v) : "v"(voff), "s"(base), "n"(OFS) : "memory");
    return v;
}

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// 8 bytes per lane from base + voff + OFS into registers.
template <int OFS> __device__ __forceinline__ u32x2 load8(const uint8_t* base, uint32_t voff)
{
    u32x2 v;
    asm volatile("global_load_dwordx2 %0, %1, %2 offset:%3" : "=v"(v) : "v"(voff), "s"(base), "n"(OFS) : "memory");
    return v;
}

template <int N> __device__ __forceinline__ void vm_wait()
{
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Wait as above and mark the four registers of an A chunk as produced here.
template <int N> __device__ __forceinline__ void vm_wait(u32x4& a, u32x4& b, u32x4& c, u32x4& d)
{
    asm volatile("s_waitcnt vmcnt(%4)" : "+v"(a), "+v"(b), "+v"(c), "+v"(d) : "n"(N) : "memory");
}

// The same for IF3's A chunk (16 + 8 bytes per row block).
template <int N> __device__ __forceinline__ void vm_wait(u32x4& a, u32x2& b, u32x4& c, u32x2& d)
{
    asm volatile("s_waitcnt vmcnt(%4)" : "+v"(a), "+v"(b), "+v"(c), "+v"(d) : "n"(N) : "memory");
}

// Drain every load before the epilogue.  The A registers of both slots are
// operands: the compiler cannot see the asm loads as loads, so without them
// the last (unused) A prefetch's registers count as free after the loop and
// may be reassigned (e.g. to a store address) while that load is still
// writing them.
__device__ __forceinline__ void vm_drain(u32x4 (&a)[2][2][2])
{
    asm volatile("s_waitcnt vmcnt(0)"
                 : "+v"(a[0][0][0]), "+v"(a[0][0][1]), "+v"(a[0][1][0]), "+v"(a[0][1][1]),
                   "+v"(a[1][0][0]), "+v"(a[1][0][1]), "+v"(a[1][1][0]), "+v"(a[1][1][1])
                 :
                 : "memory");
}

__device__ __forceinline__ void vm_drain(u32x4 (&a)[2][2][2], u32x2 (&a3)[2][2])
{
    asm volatile("s_waitcnt vmcnt(0)"
                 : "+v"(a[0][0][0]), "+v"(a3[0][0]), "+v"(a[0][1][0]), "+v"(a3[0][1]),
                   "+v"(a[1][0][0]), "+v"(a3[1][0]), "+v"(a[1][1][0]), "+v"(a3[1][1])
                 :
                 : "memory");
}

struct Ctx {
    const uint8_t* a_codes;
    const uint8_t* a_scales;
    const uint8_t* b_codes;
    const uint8_t* b_scales;
    int64_t rowb;    // bytes per code row (K / 2)
    int64_t gpr;     // scale bytes per row (K / 16, or K / 8 for block size 8)
    int nch;         // 2-step chunks
    int nsc;         // scale chunks (8 steps, or 4 for block size 8: 32 bytes per row either way)
    int64_t m0, n0;
    uint8_t* dec;    // 3 decoded stages
    uint8_t* raw;    // 2 raw B slots
    uint8_t* scl;    // 2 scale slots
    // Loop-invariant parts of the copy and load addresses: wave-uniform bases
    // of the tile's first row (codes and scales of A and B) and per-lane
    // 32-bit byte offsets from them (a tile spans 256 rows, so every offset
    // is below 256 * max(rowb, gpr)).
    const uint8_t* a_row0;
    const uint8_t* b_row0;
    const uint8_t* as_row0;
    const uint8_t* bs_row0;
    uint32_t vb[4];      // B code copy q: row (4 q + wave) 16 + lane / 4, piece (lane % 4) ^ swz4(row)
                         // (IF3: q < 2 row 64 wave + 32 q + lane / 2, piece (lane % 2) ^ swz2(row);
                         // q = 2 row 64 wave + lane, piece 2)
    uint32_t vs[2];      // scale copy q: row (2 wave + q) 32 + lane / 2, half lane % 2
    uint32_t va[2];      // A code loads: row arow_local + 32 i, bytes 32 h .. (IF3: 24 h ..)
    uint32_t lds_raw;    // LDS byte address of raw slot 0 (wave-uniform)
    uint32_t lds_scl;    // LDS byte address of scale slot 0 (wave-uniform)
    int wave;            // wave-uniform wavefront index
};

// SPG: scale bytes per 16 values (1, or 2 for block size 8).
template <int FMT> constexpr int kSpg = Fmt<FMT>::G == 8 ? 2 : 1;
template <int SPG> using SclWord = typename std::conditional<SPG == 2, uint64_t, uint32_t>::type;

template <int SPG, int BITS = 4> struct StateT {
    u32x4 a[2][2][2];        // A codes [chunk slot][row block][16-byte half] (IF3: first 16 bytes)
    typename std::conditional<BITS == 3, u32x2[2][2], char>::type a3;  // IF3: the last 8 bytes
    SclWord<SPG> as[2][2];   // A scale bytes [chunk slot][row block] (4 groups)
    uint32_t bw[8];          // B codes of the next decode (4 groups, decode order)
    SclWord<SPG> bs;         // their scale bytes
    KC akc[2];               // A fold constants [row block]: of the pair in use, or
                             // (block size 8) of the second group of the step
    KC akf;                  // (block size 8) constants of the A group decoded in
                             // the next slice, when it is the first group of a step
    KC bkc;                  // constants of the B group(s) decoded in the next slice
    half8 af[2][2][2];       // A fragments [group gg][row block][slice parity]
    half8 bf[2][8];          // B fragments, double buffered over slices
};
template <int FMT> using StateF = StateT<kSpg<FMT>, Fmt<FMT>::BITS>;

// The two words (8 codes each) of IF3 group g of a run of 48-bit groups in
// dwords D: group g starts at bit 48 g; word 0 holds codes 0-7 (bits 0-23 of
// the group), word 1 codes 8-15 (bits above 23 are ignored by the decode).
__device__ __forceinline__ void group_words3(const uint32_t* D, int g, uint32_t& w0, uint32_t& w1)
{
    const int m = 3 * (g >> 1);
    if (g & 1) {
        w0 = __builtin_amdgcn_alignbit(D[m + 2], D[m + 1], 16);
        w1 = D[m + 2] >> 8;
    } else {
        w0 = D[m];
        w1 = __builtin_amdgcn_alignbit(D[m + 1], D[m], 24);
    }
}

// B codes of chunk cc (rows n0 .. n0 + 255, 64 bytes each) into raw slot:
// instruction q of wave w covers rows 16 (4 q + w) .. + 15, four lanes per
// row; piece p of a row is stored at position p ^ swz4(row).
// (Q0 .. Q1 - 1: the copies issued by this call.)
// IF3 chunks (48 bytes a row) take three instructions per wave: q = 0, 1
// copy pieces 0 and 1 of rows 64 wave + 32 q .. + 31 (two lanes per row)
// into the slot's first 8 KiB (32 bytes a row), q = 2 piece 2 of rows
// 64 wave .. + 63 (one lane per row) into its last 4 KiB.
template <int BITS = 4, int Q0 = 0, int Q1 = (BITS == 3 ? 3 : 4)>
__device__ __forceinline__ void copy_b_chunk(const Ctx& x, int cc, int slot)
{
    const uint8_t* base = x.b_row0 + (int64_t)cc * kChunkB<BITS>;
#pragma unroll
    for (int q = Q0; q < Q1; ++q) {
        if constexpr (BITS == 3)
            copy16(base, x.vb[q], x.lds_raw + slot * kRawBytesF<3> +
                                      (q < 2 ? (64 * x.wave + 32 * q) * 32 : kBN * 32 + 64 * x.wave * 16));
        else
            copy16(base, x.vb[q], x.lds_raw + slot * kRawBytes + (4 * q + x.wave) * 16 * 64);
    }
}

// Half `hf` of scale chunk e (hf 0: the A rows, 1: the B rows): 8
// instructions of 32 rows x 32 bytes, two per wave.
template <int Q0 = 0, int Q1 = 2>
__device__ __forceinline__ void copy_scales(const Ctx& x, int e, int hf, int slot)
{
    const uint8_t* base = (hf ? x.bs_row0 : x.as_row0) + (int64_t)e * 32;
#pragma unroll
    for (int q = Q0; q < Q1; ++q)
        copy16(base, x.vs[q], x.lds_scl + slot * kSclBytes + hf * kSclB + (2 * x.wave + q) * 32 * 32);
}

// A codes of chunk cc for this lane: rows arow0 + 32 i, bytes 32 h .. 32 h + 31.
__device__ __forceinline__ void load_a_chunk(const Ctx& x, int cc, u32x4 (&a)[2][2])
{
    const uint8_t* base = x.a_row0 + (int64_t)cc * 64;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        a[i][0] = load16<0>(base, x.va[i]);
        a[i][1] = load16<16>(base, x.va[i]);
    }
}

// IF3: 24 bytes a lane and row block (groups 4 h .. 4 h + 3 of the chunk).
__device__ __forceinline__ void load_a_chunk(const Ctx& x, int cc, u32x4 (&a)[2][2], u32x2 (&a3)[2])
{
    const uint8_t* base = x.a_row0 + (int64_t)cc * 48;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        a[i][0] = load16<0>(base, x.va[i]);
        a3[i] = load8<16>(base, x.va[i]);
    }
}

template <int FMT>
__device__ __forceinline__ void load_a_any(const Ctx& x, int cc, StateF<FMT>& st, int slot)
{
    if constexpr (Fmt<FMT>::BITS == 3)
        load_a_chunk(x, cc, st.a[slot], st.a3[slot]);
    else
        load_a_chunk(x, cc, st.a[slot]);
}

// The two words of local group G (0..3) of the lane's A chunk in (slot, row block).
template <int FMT, int G>
__device__ __forceinline__ void a_words(const StateF<FMT>& st, int slot, int rb, uint32_t& w0, uint32_t& w1)
{
    if constexpr (Fmt<FMT>::BITS == 3) {
        const u32x4 v = st.a[slot][rb][0];
        const u32x2 u = st.a3[slot][rb];
        const uint32_t D[6] = {v.x, v.y, v.z, v.w, u.x, u.y};
        group_words3(D, G, w0, w1);
    } else {
        w0 = st.a[slot][rb][G >> 1][2 * (G & 1)];
        w1 = st.a[slot][rb][G >> 1][2 * (G & 1) + 1];
    }
}

// Wait for the A chunk in `slot` (N loads may stay outstanding).
template <int FMT, int N>
__device__ __forceinline__ void vm_wait_a(StateF<FMT>& st, int slot)
{
    if constexpr (Fmt<FMT>::BITS == 3)
        vm_wait<N>(st.a[slot][0][0], st.a3[slot][0], st.a[slot][1][0], st.a3[slot][1]);
    else
        vm_wait<N>(st.a[slot][0][0], st.a[slot][0][1], st.a[slot][1][0], st.a[slot][1][1]);
}

// Scale bytes of A chunk c for this lane (4 groups per row block; two
// bytes per group with block size 8, whose scale chunks hold 2 code chunks).
template <int SPG>
__device__ __forceinline__ void read_a_scales(const Ctx& x, int c, int arow_local, int h, SclWord<SPG> (&as)[2])
{
    if constexpr (SPG == 1) {
        const uint8_t* sl = x.scl + ((c >> 2) & 1) * kSclBytes;
#pragma unroll
        for (int i = 0; i < 2; ++i)
            as[i] = *reinterpret_cast<const uint32_t*>(sl + (arow_local + 32 * i) * 32 + 8 * (c & 3) + 4 * h);
    } else {
        const uint8_t* sl = x.scl + ((c >> 1) & 1) * kSclBytes;
#pragma unroll
        for (int i = 0; i < 2; ++i)
            as[i] = *reinterpret_cast<const uint64_t*>(sl + (arow_local + 32 * i) * 32 + 16 * (c & 1) + 8 * h);
    }
}

// B codes and scale bytes that step s decodes (B of step s + 2) -- chunk
// (s + 2) / 2, step j = s % 2 of it -- for row t: the LDS reads
// (read_b_raw_issue) and, a few slots later, the unpacking into the state
// (read_b_raw_finish), so that no wait for these reads falls right behind
// them.
template <int SPG> struct RawRead {
    u32x4 lo, hi, mid;   // (mid: IF3 only)
    typename std::conditional<SPG == 2, u32x4, uint2>::type v;
};

// IF3 reads the whole 48-byte row of the chunk (pieces 0, 1, 2).
template <int SPG, int BITS = 4>
__device__ __forceinline__ void read_b_raw_issue(const Ctx& x, int sd, RawRead<SPG>& r)
{
    const int t = threadIdx.x;
    const int c = sd >> 1, j = sd & 1;
    if constexpr (BITS == 3) {
        const uint8_t* rs = x.raw + (c & 1) * kRawBytesF<3>;
        const int sw = swz2(t);
        r.lo = *reinterpret_cast<const u32x4*>(rs + t * 32 + 16 * sw);
        r.mid = *reinterpret_cast<const u32x4*>(rs + t * 32 + 16 * (1 ^ sw));
        r.hi = *reinterpret_cast<const u32x4*>(rs + kBN * 32 + t * 16);
    } else {
        const uint8_t* rs = x.raw + (c & 1) * kRawBytes + t * 64;
        const int sw = swz4(t);
        r.lo = *reinterpret_cast<const u32x4*>(rs + 16 * (j ^ sw));
        r.hi = *reinterpret_cast<const u32x4*>(rs + 16 * ((2 + j) ^ sw));
    }
    if constexpr (SPG == 1)
        r.v = *reinterpret_cast<const uint2*>(x.scl + ((c >> 2) & 1) * kSclBytes + kSclB + t * 32 + 8 * (c & 3));
    else
        r.v = *reinterpret_cast<const u32x4*>(x.scl + ((c >> 1) & 1) * kSclBytes + kSclB + t * 32 + 16 * (c & 1));
}

// J: the step of the chunk (sd % 2).  IF3: the words of groups 2 J, 2 J + 1,
// 4 + 2 J, 5 + 2 J of the row.
template <int SPG, int BITS, int J>
__device__ __forceinline__ void read_b_raw_finish(const RawRead<SPG>& r, StateT<SPG, BITS>& st)
{
    constexpr int j = J;
    if constexpr (BITS == 3) {
        const uint32_t D[12] = {r.lo.x, r.lo.y, r.lo.z, r.lo.w, r.mid.x, r.mid.y,
                                r.mid.z, r.mid.w, r.hi.x, r.hi.y, r.hi.z, r.hi.w};
#pragma unroll
        for (int G = 0; G < 4; ++G) group_words3(D, (G < 2 ? 0 : 4) + 2 * j + (G & 1), st.bw[2 * G], st.bw[2 * G + 1]);
    } else {
        st.bw[0] = r.lo.x; st.bw[1] = r.lo.y; st.bw[2] = r.lo.z; st.bw[3] = r.lo.w;
        st.bw[4] = r.hi.x; st.bw[5] = r.hi.y; st.bw[6] = r.hi.z; st.bw[7] = r.hi.w;
    }
    if constexpr (SPG == 1) {
        st.bs = __builtin_amdgcn_perm(r.v.y, r.v.x, j ? 0x07060302u : 0x05040100u);
    } else {
        // 16 bytes of chunk c: groups 2j, 2j + 1 at bytes 4j .. 4j + 3 and
        // groups 4 + 2j, 5 + 2j at bytes 8 + 4j .. 8 + 4j + 3
        st.bs = j ? ((uint64_t)r.v.y | ((uint64_t)r.v.w << 32)) : ((uint64_t)r.v.x | ((uint64_t)r.v.z << 32));
    }
}

template <int SPG, int BITS, int J>
__device__ __forceinline__ void read_b_raw(const Ctx& x, int sd, StateT<SPG, BITS>& st)
{
    RawRead<SPG> r;
    read_b_raw_issue<SPG, BITS>(x, sd, r);
    read_b_raw_finish<SPG, BITS, J>(r, st);
}

// Decode B group G (0..3, decode order) of row t into stage `stg`: halves
// 16 G .. 16 G + 15, i.e. pieces 2 G and 2 G + 1 (swizzled); kc holds the
// constants of groups 2 (G / 2) and 2 (G / 2) + 1.
template <int FMT, int G>
__device__ __forceinline__ void decode_b_fast(const StateF<FMT>& st, const KC& kc, uint8_t* stg)
{
    const int t = threadIdx.x;
    uint32_t v[8];
    if constexpr (kSpg<FMT> == 2)
        decode_words_kc2<FMT>(st.bw + 2 * G, kc, v);
    else
        decode_group_kc<FMT, G & 1>(st.bw + 2 * G, kc, v);
    const int sw = swz8(t);
    uint8_t* row = stg + t * 128;
    *reinterpret_cast<u32x4*>(row + 16 * ((2 * G) ^ sw)) = u32x4{v[0], v[1], v[2], v[3]};
    *reinterpret_cast<u32x4*>(row + 16 * ((2 * G + 1) ^ sw)) = u32x4{v[4], v[5], v[6], v[7]};
}

template <int FMT>
__device__ __forceinline__ void decode_b_all(const StateF<FMT>& st, uint8_t* stg)
{
    if constexpr (kSpg<FMT> == 2) {
        decode_b_fast<FMT, 0>(st, pair_kc<FMT>((uint32_t)st.bs & 0xFFFFu), stg);
        decode_b_fast<FMT, 1>(st, pair_kc<FMT>((uint32_t)(st.bs >> 16) & 0xFFFFu), stg);
        decode_b_fast<FMT, 2>(st, pair_kc<FMT>((uint32_t)(st.bs >> 32) & 0xFFFFu), stg);
        decode_b_fast<FMT, 3>(st, pair_kc<FMT>((uint32_t)(st.bs >> 48)), stg);
    } else {
        const KC k0 = pair_kc<FMT>(st.bs & 0xFFFFu), k1 = pair_kc<FMT>(st.bs >> 16);
        decode_b_fast<FMT, 0>(st, k0, stg);
        decode_b_fast<FMT, 1>(st, k0, stg);
        decode_b_fast<FMT, 2>(st, k1, stg);
        decode_b_fast<FMT, 3>(st, k1, stg);
    }
}

// Decode local group G (0..3) of the lane's A chunk (one row block) with the
// constants kc of its pair.
template <int FMT, int G>
__device__ __forceinline__ void decode_a_fast(const StateF<FMT>& st, int slot, int rb, const KC& kc, half8& f0,
                                              half8& f1)
{
    uint32_t w[2];
    a_words<FMT, G>(st, slot, rb, w[0], w[1]);
    uint32_t v[8];
    if constexpr (kSpg<FMT> == 2)
        decode_words_kc2<FMT>(w, kc, v);   // kc: this group's two scale bytes
    else
        decode_group_kc<FMT, G & 1>(w, kc, v);
    f0 = __builtin_bit_cast(half8, u32x4{v[0], v[1], v[2], v[3]});
    f1 = __builtin_bit_cast(half8, u32x4{v[4], v[5], v[6], v[7]});
}

__device__ __forceinline__ void read_bfrags_fast(const uint8_t* stg, int kk, int lane, half8 (&bf)[8])
{
    const int h = lane >> 5;
    const uint8_t* base = stg + (lane & 31) * 128 + 16 * ((4 * h + kk) ^ swz8(lane & 31));
#pragma unroll
    for (int j = 0; j < 8; ++j) bf[j] = *reinterpret_cast<const half8*>(base + j * 32 * 128);
}

// B fragment j0 of slice kk of a decoded stage.
__device__ __forceinline__ void read_bfrag1(const uint8_t* stg, int kk, int lane, half8 (&bf)[8], int j0)
{
    const int h = lane >> 5;
    const uint8_t* base = stg + (lane & 31) * 128 + 16 * ((4 * h + kk) ^ swz8(lane & 31));
    bf[j0] = *reinterpret_cast<const half8*>(base + j0 * 32 * 128);
}

// One K step s = 4 u + Q of the four-step loop body.  c = s / 2 is the A
// chunk of this step (slot CS = Q / 2), j = Q % 2 the step within it.
// Each slice kk issues its 16 MFMAs one per slot and places, after each,
// one piece of the slice's other work, fenced with sched_barrier so that
// the matrix core never waits behind a long run of VALU work:
//   slots 0..7 : the next slice's B fragments (one LDS read per slot)
//   slots 1..8 : decode of one B group (stages of its two words), stored
//                to the stage of step s + 2 at slot 8
//   slots 9..15: decode of one A group into the fragments of a later slice
//                (this step's second group at kk = 0, 1; the next step's
//                first group at kk = 2, 3)
// Every MFMA operand was produced at least one slice earlier.
template <int FMT, int Q>
__device__ __forceinline__ void step(const Ctx& x, StateF<FMT>& st, int s, int64_t arow0, int arow_local,
                                     uint8_t* Bs, uint8_t* Bn, uint8_t* Bd, floatx16 (&acc)[2][8])
{
    constexpr int j = Q & 1, CS = Q >> 1;
    constexpr int SPG = kSpg<FMT>;
    constexpr int BITS = Fmt<FMT>::BITS;
    const int t = threadIdx.x;
    const int lane = t & 63;
    const int h = lane >> 5;
    const int c = s >> 1;
    const int swb = swz8(t);
    // Odd steps copy B codes of chunk c + 3 (slots 4-7 of slice 0) and, where
    // due, half of a scale chunk (slots 10, 11); even steps read the A scale
    // bytes of chunk c + 1 (slot 4).
    const int cb = min(c + 3, x.nch - 1);
    constexpr bool SCOPY = (SPG == 1 && Q == 1) || (SPG == 2 && j == 1);
    int se = 0, shf = 0;
    if constexpr (SPG == 1 && Q == 1) {
        // scale chunk e = (u + 3) / 2, half (u + 1) % 2, for u = s / 4
        const int u = s >> 2;
        se = (u + 3) >> 1;
        shf = (u + 1) & 1;
    } else if constexpr (SPG == 2 && j == 1) {
        // 4-step scale chunks: e = u + 2, its A half at Q = 1, its B half at Q = 3
        se = (s >> 2) + 2;
        shf = Q >> 1;
    }
    const int sec = min(se, x.nsc - 1);
    RawRead<SPG> rr;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
        const int f = kk & 1, gg = kk >> 1, par = kk & 1;
        const uint8_t* nstg = kk < 3 ? Bs : Bn;
        const int nkk = kk < 3 ? kk + 1 : 0;
        WordDec b0, b1, a0, a1;
#define IFQ_MFMA(m) \
    acc[(m) >> 3][(m) & 7] = __builtin_amdgcn_mfma_f32_32x32x16_f16(st.af[gg][(m) >> 3][par], st.bf[f][(m) & 7], \
                                                                      acc[(m) >> 3][(m) & 7], 0, 0, 0)
#define IFQ_SLOT_END() __builtin_amdgcn_sched_barrier(0)
        IFQ_MFMA(0);
        read_bfrag1(nstg, nkk, lane, st.bf[f ^ 1], 0);
        // constants of this slice's B group (computed in an earlier slot:
        // for block size 16 from the pair of groups 2 (kk / 2), 2 (kk / 2) + 1,
        // for block size 8 from group kk's two bytes)
        const KC bkc = st.bkc;
        // word 0 and word 1 of the group: the same half of bkc, or (block size
        // 8) halves 0 and 1
        const TypeSel bts = (SPG == 1 && (kk & 1)) ? type_sel<FMT, 1>(bkc) : type_sel<FMT, 0>(bkc);
        const TypeSel bts1 = (SPG == 1 && !(kk & 1)) ? type_sel<FMT, 0>(bkc) : type_sel<FMT, 1>(bkc);
        IFQ_SLOT_END();
        IFQ_MFMA(1);
        read_bfrag1(nstg, nkk, lane, st.bf[f ^ 1], 1);
        wd_s1<FMT, true>(st.bw[2 * kk], bts, b0);
        IFQ_SLOT_END();
        IFQ_MFMA(2);
        read_bfrag1(nstg, nkk, lane, st.bf[f ^ 1], 2);
        wd_s2<FMT, true>(st.bw[2 * kk], bts, b0);
        IFQ_SLOT_END();
        IFQ_MFMA(3);
        read_bfrag1(nstg, nkk, lane, st.bf[f ^ 1], 3);
        wd_s3<FMT, true>(b0);
        IFQ_SLOT_END();
        IFQ_MFMA(4);
        read_bfrag1(nstg, nkk, lane, st.bf[f ^ 1], 4);
        if (kk == 0) {
            if constexpr (j == 1) copy_b_chunk<BITS, 0, 1>(x, cb, CS ^ 1);
            else read_a_scales<SPG>(x, min(c + 1, x.nch - 1), arow_local, h, st.as[CS ^ 1]);
        }
        if (kk == 3) read_b_raw_issue<SPG, BITS>(x, s + 3, rr);
        uint32_t v0[4], v1[4];
        if (SPG == 1 && (kk & 1)) wd_s4<FMT, 1, true>(b0, bkc, v0); else wd_s4<FMT, 0, true>(b0, bkc, v0);
        IFQ_SLOT_END();
        IFQ_MFMA(5);
        read_bfrag1(nstg, nkk, lane, st.bf[f ^ 1], 5);
        if constexpr (j == 1) if (kk == 0) copy_b_chunk<BITS, 1, 2>(x, cb, CS ^ 1);
        wd_s1<FMT, true>(st.bw[2 * kk + 1], bts1, b1);
        IFQ_SLOT_END();
        IFQ_MFMA(6);
        read_bfrag1(nstg, nkk, lane, st.bf[f ^ 1], 6);
        if constexpr (j == 1) if (kk == 0) copy_b_chunk<BITS, 2, 3>(x, cb, CS ^ 1);
        wd_s2<FMT, true>(st.bw[2 * kk + 1], bts1, b1);
        IFQ_SLOT_END();
        IFQ_MFMA(7);
        read_bfrag1(nstg, nkk, lane, st.bf[f ^ 1], 7);
        if constexpr (j == 1 && BITS == 4) if (kk == 0) copy_b_chunk<BITS, 3, 4>(x, cb, CS ^ 1);
        wd_s3<FMT, true>(b1);
        IFQ_SLOT_END();
        IFQ_MFMA(8);
        if (SPG == 2 || (kk & 1)) wd_s4<FMT, 1, true>(b1, bkc, v1); else wd_s4<FMT, 0, true>(b1, bkc, v1);
        {
            // B group kk of row t: pieces 2 kk and 2 kk + 1 of the stage row
            uint8_t* row = Bd + t * 128;
            *reinterpret_cast<u32x4*>(row + 16 * ((2 * kk) ^ swb)) = u32x4{v0[0], v0[1], v0[2], v0[3]};
            *reinterpret_cast<u32x4*>(row + 16 * ((2 * kk + 1) ^ swb)) = u32x4{v1[0], v1[1], v1[2], v1[3]};
        }
        IFQ_SLOT_END();
        IFQ_MFMA(9);
        // the A group of this slice: kk < 2: local group 2 j + 1 of chunk c,
        // row block kk (constants computed with group 2 j); kk >= 2: the
        // first group of the next step, row block kk - 2 -- local group 0 of
        // chunk c + 1 (j = 1, loaded two steps ago; then slot CS, whose last
        // group was decoded at kk = 1, is refilled) or local group 2 of chunk
        // c (j = 0)
        // (block size 8: the constants of each group come from its own two
        // scale bytes -- the first group's here, the second's kept for the
        // next step -- word 0 with half 0, word 1 with half 1)
        uint32_t aw0, aw1;
        KC akc;
        if (kk < 2) {
            a_words<FMT, 2 * j + 1>(st, CS, kk, aw0, aw1);
            akc = st.akc[kk];
        } else {
            if constexpr (j == 1) {
                if (kk == 2) {
                    // outstanding after the wait: this step's B code copies (4, IF3: 3)
                    // and, where issued, 2 scale copies
                    constexpr int NB = BITS == 3 ? 3 : 4;
                    vm_wait_a<FMT, (SPG == 2 || Q == 1) ? NB + 2 : NB>(st, CS ^ 1);
                    load_a_any<FMT>(x, min(c + 2, x.nch - 1), st, CS);
                }
                a_words<FMT, 0>(st, CS ^ 1, kk - 2, aw0, aw1);
            } else {
                a_words<FMT, 2>(st, CS, kk - 2, aw0, aw1);
            }
            // constants computed in slot 13 of the previous slice
            akc = SPG == 1 ? st.akc[kk - 2] : st.akf;
        }
        const TypeSel ats = (SPG == 1 && kk < 2) ? type_sel<FMT, 1>(akc) : type_sel<FMT, 0>(akc);
        const TypeSel ats1 = (SPG == 1 && kk >= 2) ? type_sel<FMT, 0>(akc) : type_sel<FMT, 1>(akc);
        wd_s1<FMT, true>(aw0, ats, a0);
        IFQ_SLOT_END();
        IFQ_MFMA(10);
        if constexpr (SCOPY) if (kk == 0) copy_scales<0, 1>(x, sec, shf, se & 1);
        wd_s2<FMT, true>(aw0, ats, a0);
        IFQ_SLOT_END();
        IFQ_MFMA(11);
        if constexpr (SCOPY) if (kk == 0) copy_scales<1, 2>(x, sec, shf, se & 1);
        wd_s3<FMT, true>(a0);
        IFQ_SLOT_END();
        IFQ_MFMA(12);
        if constexpr (SPG == 1) {
            if (kk == 1) st.bkc = pair_kc<FMT>(st.bs >> 16);
        } else {
            if (kk < 3) st.bkc = pair_kc<FMT>((uint32_t)(st.bs >> (16 * (kk + 1))) & 0xFFFFu);
        }
        uint32_t o0[4], o1[4];
        if (SPG == 1 && kk < 2) wd_s4<FMT, 1, true>(a0, akc, o0); else wd_s4<FMT, 0, true>(a0, akc, o0);
        wd_s1<FMT, true>(aw1, ats1, a1);
        IFQ_SLOT_END();
        IFQ_MFMA(13);
        if (kk == 1 || kk == 2) {
            // constants of the first A group of the next step (row block kk - 1),
            // decoded in slice kk + 1 (its slot is free: slice kk decodes row
            // block kk % 2 with akc[kk % 2], block size 8 with its own copy)
            const int rb = kk - 1;
            if constexpr (j == 1) {
                if constexpr (SPG == 1) {
                    st.akc[rb] = pair_kc<FMT>(st.as[CS ^ 1][rb] & 0xFFFFu);
                } else {
                    st.akf = pair_kc<FMT>((uint32_t)st.as[CS ^ 1][rb] & 0xFFFFu);
                    st.akc[rb] = pair_kc<FMT>((uint32_t)(st.as[CS ^ 1][rb] >> 16) & 0xFFFFu);
                }
            } else {
                if constexpr (SPG == 1) {
                    st.akc[rb] = pair_kc<FMT>(st.as[CS][rb] >> 16);
                } else {
                    st.akf = pair_kc<FMT>((uint32_t)(st.as[CS][rb] >> 32) & 0xFFFFu);
                    st.akc[rb] = pair_kc<FMT>((uint32_t)(st.as[CS][rb] >> 48));
                }
            }
        }
        wd_s2<FMT, true>(aw1, ats1, a1);
        IFQ_SLOT_END();
        IFQ_MFMA(14);
        if (kk == 3) {
            // B codes, scales and constants of the next step's first group
            read_b_raw_finish<SPG, BITS, (Q + 1) & 1>(rr, st);
            st.bkc = pair_kc<FMT>((uint32_t)st.bs & 0xFFFFu);
        }
        wd_s3<FMT, true>(a1);
        IFQ_SLOT_END();
        IFQ_MFMA(15);
        if (SPG == 2 || kk < 2) wd_s4<FMT, 1, true>(a1, akc, o1); else wd_s4<FMT, 0, true>(a1, akc, o1);
        {
            const half8 f0 = __builtin_bit_cast(half8, u32x4{o0[0], o0[1], o0[2], o0[3]});
            const half8 f1 = __builtin_bit_cast(half8, u32x4{o1[0], o1[1], o1[2], o1[3]});
            st.af[kk < 2 ? 1 : 0][kk & 1][0] = f0;
            st.af[kk < 2 ? 1 : 0][kk & 1][1] = f1;
        }

        IFQ_SLOT_END();
#undef IFQ_MFMA
#undef IFQ_SLOT_END
    }
    // even steps: the copies of the last odd step (B codes, scales) must have
    // landed before the barrier makes them visible
    if constexpr (j == 0) vm_wait<4>();
    lds_barrier();
}

template <int FMT, bool OUT_BF16>
__device__ __forceinline__ void tile(const uint8_t* __restrict__ a_codes, const uint8_t* __restrict__ a_scales,
                                     const float* __restrict__ a_ts, const uint8_t* __restrict__ b_codes,
                                     const uint8_t* __restrict__ b_scales, const float* __restrict__ b_ts,
                                     int64_t M, int64_t N, int64_t K, void* __restrict__ C, int64_t ldc,
                                     int64_t m0, int64_t n0, uint8_t* dec, uint8_t* raw, uint8_t* scl,
                                     int64_t k0, int64_t klen, bool add)
{
    // K values [k0, k0 + klen) of the rows (k0 and klen multiples of 512);
    // the row pitches come from the whole K
    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    const int h = lane >> 5;
    const int arow_local = 64 * wave + (lane & 31);
    const int64_t arow0 = m0 + arow_local;
    constexpr int SPG = kSpg<FMT>;
    constexpr int BITS = Fmt<FMT>::BITS;
    Ctx x;
    x.a_codes = a_codes;
    x.a_scales = a_scales;
    x.b_codes = b_codes;
    x.b_scales = b_scales;
    x.rowb = K * BITS / 8;
    x.gpr = SPG * (K / kGroup);
    x.nch = (int)(klen / 128);
    x.nsc = (int)(klen / (512 / SPG));
    x.m0 = m0;
    x.n0 = n0;
    x.dec = dec;
    x.raw = raw;
    x.scl = scl;
    x.a_row0 = a_codes + m0 * x.rowb + k0 * BITS / 8;
    x.b_row0 = b_codes + n0 * x.rowb + k0 * BITS / 8;
    x.as_row0 = a_scales + m0 * x.gpr + SPG * (k0 / kGroup);
    x.bs_row0 = b_scales + n0 * x.gpr + SPG * (k0 / kGroup);
    x.wave = __builtin_amdgcn_readfirstlane(wave);
    x.lds_raw = __builtin_amdgcn_readfirstlane(lds_off(raw));
    x.lds_scl = __builtin_amdgcn_readfirstlane(lds_off(scl));
    if constexpr (BITS == 3) {
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const int r = 64 * wave + 32 * q + (lane >> 1);
            x.vb[q] = (uint32_t)(r * x.rowb) + 16u * (uint32_t)((lane & 1) ^ swz2(r));
        }
        x.vb[2] = (uint32_t)((64 * wave + lane) * x.rowb) + 32u;
        x.vb[3] = 0;
    } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int r = (4 * q + wave) * 16 + (lane >> 2);
            x.vb[q] = (uint32_t)(r * x.rowb) + 16u * (uint32_t)((lane & 3) ^ swz4(r));
        }
    }
#pragma unroll
    for (int q = 0; q < 2; ++q)
        x.vs[q] = (uint32_t)(((2 * wave + q) * 32 + (lane >> 1)) * x.gpr) + 16u * (uint32_t)(lane & 1);
#pragma unroll
    for (int i = 0; i < 2; ++i)
        x.va[i] = (uint32_t)((arow_local + 32 * i) * x.rowb) + (BITS == 3 ? 24u : 32u) * (uint32_t)h;
    const int nsteps = (int)(klen / kBK);

    floatx16 acc[2][8];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int jb = 0; jb < 8; ++jb)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][jb][e] = 0.0f;

    StateF<FMT> st;
    // prologue: B codes of chunks 0, 1; scale chunk 0 and the A half of
    // chunk 1 (block size 8: scale chunks 0 and 1 whole); A codes of chunk 0
    copy_b_chunk<BITS>(x, 0, 0);
    copy_b_chunk<BITS>(x, min(1, x.nch - 1), 1);
    copy_scales(x, 0, 0, 0);
    copy_scales(x, 0, 1, 0);
    copy_scales(x, min(1, x.nsc - 1), 0, 1);
    if constexpr (SPG == 2) copy_scales(x, min(1, x.nsc - 1), 1, 1);
    load_a_any<FMT>(x, 0, st, 0);
    vm_wait_a<FMT, 0>(st, 0);
    lds_barrier();
    int r0 = 0, r1 = 1, r2 = 2;
    read_b_raw<SPG, BITS, 0>(x, 0, st);
    decode_b_all<FMT>(st, dec + r0 * kStageBytes);
    read_b_raw<SPG, BITS, 1>(x, 1, st);
    decode_b_all<FMT>(st, dec + r1 * kStageBytes);
    read_b_raw<SPG, BITS, 0>(x, 2, st);
    st.bkc = pair_kc<FMT>((uint32_t)st.bs & 0xFFFFu);
    read_a_scales<SPG>(x, 0, arow_local, h, st.as[0]);
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        if constexpr (SPG == 1) {
            st.akc[i] = pair_kc<FMT>(st.as[0][i] & 0xFFFFu);
            decode_a_fast<FMT, 0>(st, 0, i, st.akc[i], st.af[0][i][0], st.af[0][i][1]);
        } else {
            st.akc[i] = pair_kc<FMT>((uint32_t)(st.as[0][i] >> 16) & 0xFFFFu);
            decode_a_fast<FMT, 0>(st, 0, i, pair_kc<FMT>((uint32_t)st.as[0][i] & 0xFFFFu), st.af[0][i][0],
                                  st.af[0][i][1]);
        }
    }
    lds_barrier();
    // the odd step before step 0: B codes of chunk 2 into slot 0, A codes of chunk 1
    copy_b_chunk<BITS>(x, min(2, x.nch - 1), 0);
    load_a_any<FMT>(x, min(1, x.nch - 1), st, 1);
    read_bfrags_fast(dec + r0 * kStageBytes, 0, lane, st.bf[0]);

    for (int s = 0; s < nsteps; s += 4) {
        step<FMT, 0>(x, st, s, arow0, arow_local, dec + r0 * kStageBytes, dec + r1 * kStageBytes,
                     dec + r2 * kStageBytes, acc);
        step<FMT, 1>(x, st, s + 1, arow0, arow_local, dec + r1 * kStageBytes, dec + r2 * kStageBytes,
                     dec + r0 * kStageBytes, acc);
        step<FMT, 2>(x, st, s + 2, arow0, arow_local, dec + r2 * kStageBytes, dec + r0 * kStageBytes,
                     dec + r1 * kStageBytes, acc);
        step<FMT, 3>(x, st, s + 3, arow0, arow_local, dec + r0 * kStageBytes, dec + r1 * kStageBytes,
                     dec + r2 * kStageBytes, acc);
        // advance the ring by four steps (one position)
        const int t0 = r1;
        r1 = r2;
        r2 = r0;
        r0 = t0;
    }
    if constexpr (BITS == 3)
        vm_drain(st.a, st.a3);
    else
        vm_drain(st.a);
    store_tile<FMT, OUT_BF16, false>(acc, a_ts, b_ts, M, N, C, ldc, m0, n0, add);
}

}  // namespace fast

// Interior tiles on the fast path (4-bit formats, K % 512 == 0, 16-byte
// aligned operands), with the same XCD-aware tile order as below.
template <int FMT, bool OUT_BF16>
__global__ __launch_bounds__(kGemmThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void gemm_tn_fast(const uint8_t* __restrict__ a_codes, const uint8_t* __restrict__ a_scales,
                  const float* __restrict__ a_ts, const uint8_t* __restrict__ b_codes,
                  const uint8_t* __restrict__ b_scales, const float* __restrict__ b_ts,
                  int64_t M, int64_t N, int64_t K, void* __restrict__ C, int64_t ldc,
                  int tiles_m, int tiles_n, int t_full, int t_split)
{
    __shared__ __attribute__((aligned(16))) uint8_t dec[3 * fast::kStageBytes];
    __shared__ __attribute__((aligned(16))) uint8_t raw[2 * fast::kRawBytesF<Fmt<FMT>::BITS>];
    __shared__ __attribute__((aligned(16))) uint8_t scl[2 * fast::kSclBytes];
    int half;
    const int tile = split_tile(t_full, OUT_BF16 ? 0 : t_split, half);
    int tm, tn;
    band_tile(tile, tiles_m, tiles_n, tm, tn);
    const int64_t klen = half < 0 ? K : K / 2;
    fast::tile<FMT, OUT_BF16>(a_codes, a_scales, a_ts, b_codes, b_scales, b_ts, M, N, K, C, ldc,
                              (int64_t)tm * kBM, (int64_t)tn * kBN, dec, raw, scl,
                              half > 0 ? klen : 0, klen, half >= 0);
}

// Zeroes the output tiles [t_full, t_full + gridDim.x) of the band order
// (fp32, ldc % 4 == 0, 16-byte aligned C), ahead of the split halves' atomic
// additions.
__global__ __launch_bounds__(256) void zero_split_tiles(float* __restrict__ C, int64_t ldc, int t_full,
                                                        int tiles_m, int tiles_n)
{
    int tm, tn;
    band_tile(t_full + (int)blockIdx.x, tiles_m, tiles_n, tm, tn);
    float* base = C + (int64_t)tm * kBM * ldc + (int64_t)tn * kBN;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const float4 z = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    for (int r = wave; r < kBM; r += 4) reinterpret_cast<float4*>(base + (int64_t)r * ldc)[lane] = z;
}

// Interior tiles: every row, column and K group in range (K % 128 == 0,
// 4-byte aligned scale rows).
template <int FMT, bool OUT_BF16>
__global__ __launch_bounds__(kGemmThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void gemm_tn_interior(const uint8_t* __restrict__ a_codes, const uint8_t* __restrict__ a_scales,
                      const float* __restrict__ a_ts, const uint8_t* __restrict__ b_codes,
                      const uint8_t* __restrict__ b_scales, const float* __restrict__ b_ts,
                      int64_t M, int64_t N, int64_t K, void* __restrict__ C, int64_t ldc,
                      int tiles_m, int tiles_n)
{
    __shared__ __attribute__((aligned(16))) _Float16 lds[3][kStageHalves];
    int tm, tn;
    tile_coords(tiles_m, tiles_n, tm, tn);
    gemm_tile<FMT, OUT_BF16, false>(a_codes, a_scales, a_ts, b_codes, b_scales, b_ts, M, N, K, C,
                                    ldc, (int64_t)tm * kBM, (int64_t)tn * kBN, lds);
}

// Boundary tiles: the last tile row and column (or every tile when K or the
// scale rows rule out the interior path), with guarded loads and stores.
// Tiles [0, full_m * ext_n) cover rows below full_m * 256 in the columns
// from n_start; the rest cover the last tile row.
template <int FMT, bool OUT_BF16>
__global__ __launch_bounds__(kGemmThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void gemm_tn_edge(const uint8_t* __restrict__ a_codes, const uint8_t* __restrict__ a_scales,
                  const float* __restrict__ a_ts, const uint8_t* __restrict__ b_codes,
                  const uint8_t* __restrict__ b_scales, const float* __restrict__ b_ts, int64_t M,
                  int64_t N, int64_t K, void* __restrict__ C, int64_t ldc, int full_m,
                  int n_start_tile, int ext_n, int tiles_n)
{
    __shared__ __attribute__((aligned(16))) _Float16 lds[3][kStageHalves];
    const int bid = blockIdx.x;
    int tm, tn;
    if (bid < full_m * ext_n) {
        tm = bid / ext_n;
        tn = n_start_tile + bid % ext_n;
    } else {
        tm = full_m + (bid - full_m * ext_n) / tiles_n;
        tn = (bid - full_m * ext_n) % tiles_n;
    }
    gemm_tile<FMT, OUT_BF16, true>(a_codes, a_scales, a_ts, b_codes, b_scales, b_ts, M, N, K, C,
                                   ldc, (int64_t)tm * kBM, (int64_t)tn * kBN, lds);
}

// Compute units of the current device, cached per device (a racing first
// query repeats the same answer); 0 when it cannot be read.
static int device_cus()
{
    static std::atomic<int> cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
    int v = cache[dev].load(std::memory_order_relaxed);
    if (v == 0) {
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
        cache[dev].store(v, std::memory_order_relaxed);
    }
    return v;
}

template <int FMT>
static hipError_t launch_g(const GemmArgs& a, hipStream_t s)
{
    const int64_t tiles_m = (a.M + kBM - 1) / kBM, tiles_n = (a.N + kBN - 1) / kBN;
    if (tiles_m == 0 || tiles_n == 0) return hipSuccess;
    if (tiles_m * tiles_n > (int64_t)1 << 30) return hipErrorInvalidValue;
    // interior tiles load whole row chunks: K % 128 == 0, 4-byte aligned scale
    // rows, 16-byte aligned codes (as the API requires)
    const bool interior_ok = (a.K % (2 * kBK)) == 0 && ((uintptr_t)a.a_scales % 4) == 0 &&
                             ((uintptr_t)a.b_scales % 4) == 0 && ((uintptr_t)a.a_codes % 16) == 0 &&
                             ((uintptr_t)a.b_codes % 16) == 0;
    const int64_t full_m = interior_ok ? a.M / kBM : 0;
    const int64_t full_n = interior_ok ? a.N / kBN : 0;
    {
      if (full_m * full_n > 0) {
        // (K <= 2^24 keeps the fast kernel's 32-bit per-lane offsets, below
        // 256 code rows of K * bits / 8 bytes, in range)
        const bool fast_ok = (Fmt<FMT>::BITS == 4 || Fmt<FMT>::BITS == 3) && (a.K % 512) == 0 &&
                             a.K <= ((int64_t)1 << 24) &&
                             ((uintptr_t)a.a_codes % 16) == 0 &&
                             ((uintptr_t)a.b_codes % 16) == 0 && ((uintptr_t)a.a_scales % 16) == 0 &&
                             ((uintptr_t)a.b_scales % 16) == 0;
        const dim3 grid((unsigned)(full_m * full_n)), block(kGemmThreads);
#define IFQ_GEMM_ARGS a.a_codes, a.a_scales, a.a_ts, a.b_codes, a.b_scales, a.b_ts, a.M, a.N, a.K, a.c, a.ldc, \
                      (int)full_m, (int)full_n
        bool done = false;
        // fast path: 4-bit codes with one scale per 16 or per 8 values, IF3 with
        // one per 16 (IF3 with block size 8 spills there and runs the general
        // kernel)
        if constexpr (Fmt<FMT>::BITS == 4 || (Fmt<FMT>::BITS == 3 && Fmt<FMT>::G == 16)) {
            // fp32 output: when the last round of tiles would leave at least
            // half of the compute units idle, those tiles run as two K halves
            // each (K % 1024 == 0), added into their zeroed output
            int t_full = (int)(full_m * full_n), t_split = 0;
            if (fast_ok && !a.out_bf16 && (a.K % 1024) == 0 && (a.ldc % 4) == 0 &&
                ((uintptr_t)a.c % 16) == 0) {
                const int64_t cus = device_cus();
                const int64_t tail = cus > 0 ? (full_m * full_n) % cus : 0;
                if (tail > 0 && 2 * tail <= cus) {
                    t_split = (int)tail;
                    t_full -= t_split;
                }
            }
            if (t_split > 0) {
                hipLaunchKernelGGL(zero_split_tiles, dim3((unsigned)t_split), dim3(256), 0, s,
                                   static_cast<float*>(a.c), a.ldc, t_full, (int)full_m, (int)full_n);
                hipError_t e = hipGetLastError();
                if (e != hipSuccess) return e;
            }
            const dim3 fgrid((unsigned)(t_full + 2 * t_split));
            if (fast_ok && a.out_bf16)
                hipLaunchKernelGGL((gemm_tn_fast<FMT, true>), fgrid, block, 0, s, IFQ_GEMM_ARGS, t_full, 0);
            else if (fast_ok)
                hipLaunchKernelGGL((gemm_tn_fast<FMT, false>), fgrid, block, 0, s, IFQ_GEMM_ARGS, t_full,
                                   t_split);
            done = fast_ok;
        }
        if (!done && a.out_bf16)
            hipLaunchKernelGGL((gemm_tn_interior<FMT, true>), grid, block, 0, s, IFQ_GEMM_ARGS);
        else if (!done)
            hipLaunchKernelGGL((gemm_tn_interior<FMT, false>), grid, block, 0, s, IFQ_GEMM_ARGS);
#undef IFQ_GEMM_ARGS
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
      }
    }
    // remaining tiles: columns [full_n, tiles_n) of rows [0, full_m), then all of rows [full_m, tiles_m)
    const int64_t ext_n = (full_m * full_n > 0) ? tiles_n - full_n : tiles_n;
    const int64_t fm = (full_m * full_n > 0) ? full_m : 0;
    const int64_t n_start = (full_m * full_n > 0) ? full_n : 0;
    const int64_t nedge = fm * ext_n + (tiles_m - fm) * tiles_n;
    if (nedge > 0) {
        if (a.out_bf16)
            hipLaunchKernelGGL((gemm_tn_edge<FMT, true>), dim3((unsigned)nedge), dim3(kGemmThreads), 0,
                               s, a.a_codes, a.a_scales, a.a_ts, a.b_codes, a.b_scales, a.b_ts, a.M,
                               a.N, a.K, a.c, a.ldc, (int)fm, (int)n_start, (int)ext_n, (int)tiles_n);
        else
            hipLaunchKernelGGL((gemm_tn_edge<FMT, false>), dim3((unsigned)nedge), dim3(kGemmThreads), 0,
                               s, a.a_codes, a.a_scales, a.a_ts, a.b_codes, a.b_scales, a.b_ts, a.M,
                               a.N, a.K, a.c, a.ldc, (int)fm, (int)n_start, (int)ext_n, (int)tiles_n);
        return hipGetLastError();
    }
    return hipSuccess;
}

hipError_t launch_gemm(const GemmArgs& a, hipStream_t s)
{
    switch (a.fmt) {
        case IFQ_FMT_IF4: return launch_g<IFQ_FMT_IF4>(a, s);
        case IFQ_FMT_NVFP4: return launch_g<IFQ_FMT_NVFP4>(a, s);
        case IFQ_FMT_IF3: return launch_g<IFQ_FMT_IF3>(a, s);
        case IFQ_FMT_IF6_E2M3: return launch_g<IFQ_FMT_IF6_E2M3>(a, s);
        case IFQ_FMT_IF6_E3M2: return launch_g<IFQ_FMT_IF6_E3M2>(a, s);
        case IFQ_FMT_NVINT4: return launch_g<IFQ_FMT_NVINT4>(a, s);
        // 4/6 operands are NVFP4 data (E2M1 codes, E4M3 scales, bit 7 clear)
        case IFQ_FMT_NVFP4_46: return launch_g<IFQ_FMT_NVFP4>(a, s);
        case IFQ_FMT_IF4_BS8: return launch_g<IFQ_FMT_IF4_BS8>(a, s);
        case IFQ_FMT_IF3_BS8: return launch_g<IFQ_FMT_IF3_BS8>(a, s);
        case IFQ_FMT_NVFP4_BS8: return launch_g<IFQ_FMT_NVFP4_BS8>(a, s);
        default: return hipErrorNotSupported;
    }
}

}  // namespace ifq
