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
template <> struct Fold<IFQ_FMT_IF3> { static constexpr float FP = 3.0f, INT = 4.0f, EPI = 1.0f / 9.0f; };

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
    if constexpr (Fmt<FMT>::ADAPTIVE && Fmt<FMT>::BITS == 4) {
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
    }
    const half2v K = u32_as_h2(k2), C = u32_as_h2(c2);
#pragma unroll
    for (int i = 0; i < 4; ++i) out[i] = h2_as_u32(__builtin_elementwise_fma(u32_as_h2(x[i]), K, C));
}

// Sixteen three-bit IF3 codes (48 bits) -> 8 FP16 operand pairs: 3 q (FP) or
// 4 q (INT), times Delta (at most 6 significant bits, exact).
__device__ __forceinline__ void decode_if3_group(uint64_t bitsv, bool is_int, uint32_t k2,
                                                 uint32_t (&out)[8])
{
    using D = FmtDerived<IFQ_FMT_IF3>;
    const half2v K = u32_as_h2(k2);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        half2v hv;
#pragma unroll
        for (int e = 0; e < 2; ++e) {
            const uint32_t c = (uint32_t)(bitsv >> (3 * (2 * i + e))) & 7u;
            const float qi = (float)((int)(c << 29) >> 29);
            const float mag = fp_magnitude<IFQ_FMT_IF3>(c & 3u);
            const float qf = (c & D::SIGN_BIT) ? -mag : mag;
            hv[e] = (_Float16)(is_int ? qi * Fold<IFQ_FMT_IF3>::INT : qf * Fold<IFQ_FMT_IF3>::FP);
        }
        out[i] = h2_as_u32(hv * K);
    }
}

// ------------------------------------------------------------ raw chunks
// A: one lane's 32 k-values of one row for one step (2 groups);
// B: one thread's 64 k-values of one row (4 groups).  IF3 keeps 6-byte groups.
template <int FMT> struct RawA { uint32_t w[4]; uint32_t sb; };
template <> struct RawA<IFQ_FMT_IF3> { uint16_t h[6]; uint32_t sb; };
template <int FMT> struct RawB { uint32_t w[8]; uint32_t sb; };
template <> struct RawB<IFQ_FMT_IF3> { uint16_t h[12]; uint32_t sb; };

// Load `ng` groups (2 or 4) of one row starting at group g0 into words /
// halves.  Interior tiles (EDGE = false) load without guards.
template <int FMT, bool EDGE, int NG>
__device__ __forceinline__ void load_groups(const uint8_t* __restrict__ codes,
                                            const uint8_t* __restrict__ scales, int64_t row,
                                            int64_t nrows, int64_t gpr, int64_t g0,
                                            uint32_t* w, uint16_t* h, uint32_t& sb)
{
    constexpr int BITS = Fmt<FMT>::BITS;
    const uint8_t* cp = codes + (row * gpr + g0) * (2 * BITS);
    const uint8_t* sp = scales + row * gpr + g0;
    if constexpr (BITS == 4 && !EDGE) {
        const uint4 a = *reinterpret_cast<const uint4*>(cp);
        w[0] = a.x; w[1] = a.y; w[2] = a.z; w[3] = a.w;
        if constexpr (NG == 4) {
            const uint4 b = *reinterpret_cast<const uint4*>(cp + 16);
            w[4] = b.x; w[5] = b.y; w[6] = b.z; w[7] = b.w;
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
            } else {
                const uint16_t* p = reinterpret_cast<const uint16_t*>(cp + 6 * g);
                h[3 * g] = ok ? p[0] : (uint16_t)0;
                h[3 * g + 1] = ok ? p[1] : (uint16_t)0;
                h[3 * g + 2] = ok ? p[2] : (uint16_t)0;
            }
            sb |= (ok ? (uint32_t)sp[g] : 0u) << (8 * g);
        }
    }
}

template <int FMT, bool EDGE>
__device__ __forceinline__ void load_a(const uint8_t* __restrict__ codes, const uint8_t* __restrict__ scales,
                                       int64_t row, int64_t nrows, int64_t gpr, int64_t g0, RawA<FMT>& r)
{
    if constexpr (Fmt<FMT>::BITS == 4)
        load_groups<FMT, EDGE, 2>(codes, scales, row, nrows, gpr, g0, r.w, nullptr, r.sb);
    else
        load_groups<FMT, EDGE, 2>(codes, scales, row, nrows, gpr, g0, nullptr, r.h, r.sb);
}

template <int FMT, bool EDGE>
__device__ __forceinline__ void load_b(const uint8_t* __restrict__ codes, const uint8_t* __restrict__ scales,
                                       int64_t row, int64_t nrows, int64_t gpr, int64_t g0, RawB<FMT>& r)
{
    if constexpr (Fmt<FMT>::BITS == 4)
        load_groups<FMT, EDGE, 4>(codes, scales, row, nrows, gpr, g0, r.w, nullptr, r.sb);
    else
        load_groups<FMT, EDGE, 4>(codes, scales, row, nrows, gpr, g0, nullptr, r.h, r.sb);
}

// Decode group g of a raw chunk (whose scale bytes are sb) into 8 operand pairs.
template <int FMT>
__device__ __forceinline__ void decode_group(const uint32_t* w, const uint16_t* h, uint32_t sb, int g,
                                             uint32_t (&out)[8])
{
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
    } else {
        const uint64_t bitsv = (uint64_t)h[3 * g] | ((uint64_t)h[3 * g + 1] << 16) |
                               ((uint64_t)h[3 * g + 2] << 32);
        decode_if3_group(bitsv, is_int, k2, out);
    }
}

// Decode B group g of thread t's row into the LDS stage (natural k order).
template <int FMT>
__device__ __forceinline__ void decode_b(const RawB<FMT>& r, _Float16* stage, int t, int g)
{
    uint32_t v[8];
    if constexpr (Fmt<FMT>::BITS == 4)
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
    if constexpr (Fmt<FMT>::BITS == 4)
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

template <int FMT, bool EDGE> struct TileState {
    RawA<FMT> a_cur[2], a_nxt[2];  // [row block i]: this step, next step
    RawB<FMT> b_nxt, b_fill;       // next step (decoded now), step + 2 (loading)
    half8 af[2][2][2];             // [group gg][row block i][slice parity]
};

// One 64-wide K step.  Slice kk multiplies B fragments read from LDS stage
// `cur` with A fragments in registers while: the B fragments of slice kk + 1
// are read, one B group of the next step is decoded into stage cur ^ 1, and
// one A decode unit is produced -- this step's second group (slices 2, 3) at
// kk = 0, 1 and the next step's first group (slices 0, 1) at kk = 2, 3.
// Loads of step s + 2 are clamped to the last step (harmless extra work that
// keeps the loop free of branches).
template <int FMT, bool EDGE>
__device__ __forceinline__ void gemm_step(int s, int nsteps, const uint8_t* __restrict__ a_codes,
                                          const uint8_t* __restrict__ a_scales,
                                          const uint8_t* __restrict__ b_codes,
                                          const uint8_t* __restrict__ b_scales, int64_t M,
                                          int64_t N, int64_t gpr, int64_t arow0, int64_t n0,
                                          TileState<FMT, EDGE>& st, _Float16 (*lds)[kStageHalves],
                                          int cur, floatx16 (&acc)[2][8])
{
    const int t = threadIdx.x;
    const int lane = t & 63;
    const int h = lane >> 5;
    const _Float16* Bs = lds[cur];
    _Float16* Bd = lds[cur ^ 1];
    half8 bf[2][8];
    read_bfrags(Bs, 0, lane, bf[0]);
    const int64_t g2 = (int64_t)min(s + 2, nsteps - 1) * kGroupsPerStep;
    load_b<FMT, EDGE>(b_codes, b_scales, n0 + t, N, gpr, g2, st.b_fill);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
        const int f = kk & 1;
        if (kk < 3) read_bfrags(Bs, kk + 1, lane, bf[f ^ 1]);
        decode_b<FMT>(st.b_nxt, Bd, t, kk);
        if (kk < 2) {
            decode_a<FMT>(st.a_cur[kk], 1, st.af[1][kk][0], st.af[1][kk][1]);
        } else {
            if (kk == 2) {
                // this step's A chunks are fully decoded: refill them with step s + 2
#pragma unroll
                for (int i = 0; i < 2; ++i)
                    load_a<FMT, EDGE>(a_codes, a_scales, arow0 + 32 * i, M, gpr, g2 + 2 * h, st.a_cur[i]);
            }
            decode_a<FMT>(st.a_nxt[kk - 2], 0, st.af[0][kk - 2][0], st.af[0][kk - 2][1]);
        }
        const int gg = kk >> 1, par = kk & 1;
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 8; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(st.af[gg][i][par], bf[f][j], acc[i][j], 0, 0, 0);
#pragma unroll
        for (int m = 0; m < 16; ++m) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);
            if (m < 8) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            if (m == 3 || m == 7) __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
    }
    __syncthreads();
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
    const int nsteps = (int)((gpr + kGroupsPerStep - 1) / kGroupsPerStep);
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
        RawB<FMT> b0;
        load_b<FMT, EDGE>(b_codes, b_scales, n0 + t, N, gpr, 0, b0);
        load_b<FMT, EDGE>(b_codes, b_scales, n0 + t, N, gpr, g1, st.b_nxt);
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            load_a<FMT, EDGE>(a_codes, a_scales, arow0 + 32 * i, M, gpr, 2 * h, st.a_cur[i]);
            load_a<FMT, EDGE>(a_codes, a_scales, arow0 + 32 * i, M, gpr, g1 + 2 * h, st.a_nxt[i]);
        }
#pragma unroll
        for (int g = 0; g < kGroupsPerStep; ++g) decode_b<FMT>(b0, lds[0], t, g);
#pragma unroll
        for (int i = 0; i < 2; ++i) decode_a<FMT>(st.a_cur[i], 0, st.af[0][i][0], st.af[0][i][1]);
        __syncthreads();
        for (int s = 0; s < nsteps; ++s) {
            gemm_step<FMT, EDGE>(s, nsteps, a_codes, a_scales, b_codes, b_scales, M, N, gpr, arow0,
                                 n0, st, lds, s & 1, acc);
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const RawA<FMT> ta = st.a_cur[i];
                st.a_cur[i] = st.a_nxt[i];
                st.a_nxt[i] = ta;
            }
            const RawB<FMT> tb = st.b_nxt;
            st.b_nxt = st.b_fill;
            st.b_fill = tb;
        }
    }

    const float sc = (*a_ts * *b_ts) * Fold<FMT>::EPI;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int64_t n = n0 + j * 32 + (lane & 31);
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int64_t m = m0 + 64 * wave + i * 32 + (e >> 2) * 8 + h * 4 + (e & 3);
                if (!EDGE || (m < M && n < N)) {
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

// Interior tiles: every row, column and K group in range (K % 64 == 0,
// 4-byte aligned scale rows).  Workgroup ids are dealt round robin to the 8
// XCDs; they are remapped so that each XCD walks a contiguous range of tile
// ids, and tile ids are ordered in bands of 4 tile rows (column-major inside
// a band), so the 32 workgroups resident on one XCD form a 4 x 8 block of
// tiles that share A and B rows in its L2.
template <int FMT, bool OUT_BF16>
__global__ __launch_bounds__(kGemmThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void gemm_tn_interior(const uint8_t* __restrict__ a_codes, const uint8_t* __restrict__ a_scales,
                      const float* __restrict__ a_ts, const uint8_t* __restrict__ b_codes,
                      const uint8_t* __restrict__ b_scales, const float* __restrict__ b_ts,
                      int64_t M, int64_t N, int64_t K, void* __restrict__ C, int64_t ldc,
                      int tiles_m, int tiles_n)
{
    __shared__ __attribute__((aligned(16))) _Float16 lds[2][kStageHalves];
    const int nwg = gridDim.x;
    const int bid = blockIdx.x;
    const int tile = (nwg % 8 == 0) ? (bid % 8) * (nwg / 8) + bid / 8 : bid;
    constexpr int GM = 4;
    const int band = tile / (GM * tiles_n);
    const int first_m = band * GM;
    const int gm = min(tiles_m - first_m, GM);
    const int in_band = tile - band * GM * tiles_n;
    const int tm = first_m + in_band % gm, tn = in_band / gm;
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
    __shared__ __attribute__((aligned(16))) _Float16 lds[2][kStageHalves];
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

template <int FMT>
static hipError_t launch_g(const GemmArgs& a, hipStream_t s)
{
    const int64_t tiles_m = (a.M + kBM - 1) / kBM, tiles_n = (a.N + kBN - 1) / kBN;
    if (tiles_m == 0 || tiles_n == 0) return hipSuccess;
    if (tiles_m * tiles_n > (int64_t)1 << 30) return hipErrorInvalidValue;
    const bool interior_ok = (a.K % kBK) == 0 && ((uintptr_t)a.a_scales % 4) == 0 &&
                             ((uintptr_t)a.b_scales % 4) == 0 && Fmt<FMT>::BITS == 4;
    const int64_t full_m = interior_ok ? a.M / kBM : 0;
    const int64_t full_n = interior_ok ? a.N / kBN : 0;
    if constexpr (Fmt<FMT>::BITS == 4) {
      if (full_m * full_n > 0) {
        if (a.out_bf16)
            hipLaunchKernelGGL((gemm_tn_interior<FMT, true>), dim3((unsigned)(full_m * full_n)),
                               dim3(kGemmThreads), 0, s, a.a_codes, a.a_scales, a.a_ts, a.b_codes,
                               a.b_scales, a.b_ts, a.M, a.N, a.K, a.c, a.ldc, (int)full_m, (int)full_n);
        else
            hipLaunchKernelGGL((gemm_tn_interior<FMT, false>), dim3((unsigned)(full_m * full_n)),
                               dim3(kGemmThreads), 0, s, a.a_codes, a.a_scales, a.a_ts, a.b_codes,
                               a.b_scales, a.b_ts, a.M, a.N, a.K, a.c, a.ldc, (int)full_m, (int)full_n);
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
        default: return hipErrorNotSupported;
    }
}

}  // namespace ifq
