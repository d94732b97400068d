// gemm.hip -- block-scaled GEMM C = A_hat B_hat^T on packed operands
// (both K-major), gfx950 MFMA.
//
// Operand values.  Every element is decoded to an FP16 number that carries
// its group scale exactly: fold_FP * q * Delta for FP groups and
// fold_INT * q * Delta for INT groups, with fold_FP / fold_INT = M_I / M_FP
// (7 and 6 for IF4, 3 and 4 for IF3, 1 for NVFP4).  One FP32 MFMA
// accumulation over all of K then applies each 16-wide block's scale product
// and its range alignment (1, 6/7 or 36/49 for IF4, Sec. 5.2) at once, and the
// epilogue multiplies by alpha_A * alpha_B / fold_FP^2.  Exactness: an E4M3
// scale has at most 4 significant bits and lies in [2^-9, 448]; 7 q_FP and
// 6 q_INT have at most 5, so every product has at most 9 bits and lies in
// [3.5 * 2^-9, 42 * 448], all normal FP16 numbers.
//
// Tiling.  A workgroup of 4 wavefronts owns a 256 x 256 tile of C; each
// wavefront owns 128 x 128 (4 x 4 v_mfma_f32_32x32x16_f16 blocks, 256
// accumulators per lane).  Per 64-wide K step every thread loads the packed
// codes and scale bytes of one A row and one B row (8 groups), decodes them
// into the next FP16 LDS stage while the MFMAs consume the current one, so
// each element is decoded exactly once per workgroup.  Global loads run two
// K steps ahead in a two-slot register ring.  LDS rows hold 64 halves padded
// to 144 bytes: consecutive rows start 36 banks apart, so the 16 lanes of a
// 128-bit access phase touch disjoint banks, and every fragment and store
// address is a per-lane base plus an immediate offset.
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
constexpr int kStageHalves = kBM * kPitch;     // one operand, one stage

template <int FMT> struct Fold;
template <> struct Fold<IFQ_FMT_IF4> { static constexpr float FP = 7.0f, INT = 6.0f; };
template <> struct Fold<IFQ_FMT_NVFP4> { static constexpr float FP = 1.0f, INT = 1.0f; };
template <> struct Fold<IFQ_FMT_IF3> { static constexpr float FP = 3.0f, INT = 4.0f; };

__device__ __forceinline__ uint32_t h2_as_u32(half2v h) { return __builtin_bit_cast(uint32_t, h); }
__device__ __forceinline__ half2v u32_as_h2(uint32_t u) { return __builtin_bit_cast(half2v, u); }

// Raw packed data of one operand row for one K step (4 groups).
template <int FMT> struct RawChunk;
template <> struct RawChunk<IFQ_FMT_IF4> { uint32_t w[8]; uint32_t sb; };
template <> struct RawChunk<IFQ_FMT_NVFP4> { uint32_t w[8]; uint32_t sb; };
template <> struct RawChunk<IFQ_FMT_IF3> { uint16_t h[12]; uint32_t sb; };

// Interior tiles (EDGE = false) have every row and group in range and
// 4-byte aligned scale rows, so they load without guards.
template <int FMT, bool EDGE>
__device__ __forceinline__ void load_chunk(const uint8_t* __restrict__ codes,
                                           const uint8_t* __restrict__ scales, int64_t row,
                                           int64_t nrows, int64_t gpr, int64_t g0,
                                           RawChunk<FMT>& rc)
{
    constexpr int BITS = Fmt<FMT>::BITS;
    const bool row_ok = row < nrows;
    const int64_t gvalid = gpr - g0;  // groups of this chunk inside K
    const uint8_t* cp = codes + (row * gpr + g0) * (2 * BITS);
    const uint8_t* sp = scales + row * gpr + g0;
    if constexpr (BITS == 4 && !EDGE) {
        uint4 a = *reinterpret_cast<const uint4*>(cp);
        uint4 b = *reinterpret_cast<const uint4*>(cp + 16);
        rc.w[0] = a.x; rc.w[1] = a.y; rc.w[2] = a.z; rc.w[3] = a.w;
        rc.w[4] = b.x; rc.w[5] = b.y; rc.w[6] = b.z; rc.w[7] = b.w;
        rc.sb = *reinterpret_cast<const uint32_t*>(sp);
    } else if constexpr (BITS == 4) {
        if (row_ok && gvalid >= 4 && ((uintptr_t)cp & 15) == 0) {
            uint4 a = *reinterpret_cast<const uint4*>(cp);
            uint4 b = *reinterpret_cast<const uint4*>(cp + 16);
            rc.w[0] = a.x; rc.w[1] = a.y; rc.w[2] = a.z; rc.w[3] = a.w;
            rc.w[4] = b.x; rc.w[5] = b.y; rc.w[6] = b.z; rc.w[7] = b.w;
            if (((uintptr_t)sp & 3) == 0) {
                rc.sb = *reinterpret_cast<const uint32_t*>(sp);
            } else {
                rc.sb = (uint32_t)sp[0] | ((uint32_t)sp[1] << 8) | ((uint32_t)sp[2] << 16) |
                        ((uint32_t)sp[3] << 24);
            }
        } else {
            rc.sb = 0;
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const bool ok = row_ok && g < gvalid;
                uint2 t = ok ? *reinterpret_cast<const uint2*>(cp + 8 * g) : make_uint2(0, 0);
                rc.w[2 * g] = t.x;
                rc.w[2 * g + 1] = t.y;
                rc.sb |= (ok ? (uint32_t)sp[g] : 0u) << (8 * g);
            }
        }
    } else {
        rc.sb = 0;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const bool ok = row_ok && g < gvalid;
            const uint16_t* p = reinterpret_cast<const uint16_t*>(cp + 6 * g);
            rc.h[3 * g] = ok ? p[0] : (uint16_t)0;
            rc.h[3 * g + 1] = ok ? p[1] : (uint16_t)0;
            rc.h[3 * g + 2] = ok ? p[2] : (uint16_t)0;
            rc.sb |= (ok ? (uint32_t)sp[g] : 0u) << (8 * g);
        }
    }
}

// v_and_or_b32: (x & m) | o in one VALU op (the compiler splits it in two
// when both masks are literals).
__device__ __forceinline__ uint32_t and_or(uint32_t x, uint32_t m, uint32_t o)
{
    uint32_t r;
    asm("v_and_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"(x), "v"(m), "v"(o));
    return r;
}

// Keep a value computed on every lane (stops the compiler from sinking its
// computation into a divergent branch in front of a select).
__device__ __forceinline__ uint32_t pin(uint32_t v)
{
    asm volatile("" : "+v"(v));
    return v;
}

// Per-group FP16 scale pairs (fold * Delta, fold * Delta) of a chunk's 4 groups.
template <int FMT>
__device__ __forceinline__ void chunk_scales(uint32_t sb4, uint32_t (&k2)[4])
{
    const uint32_t mag = sb4 & 0x7F7F7F7Fu;
    const half2v d01 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(mag, 1.0f, false);  // E4M3 -> FP16
    const half2v d23 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(mag, 1.0f, true);
    const _Float16 d[4] = {d01[0], d01[1], d23[0], d23[1]};
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        const bool is_int = Fmt<FMT>::ADAPTIVE && ((sb4 >> (8 * g + 7)) & 1u);
        const _Float16 fold = is_int ? (_Float16)Fold<FMT>::INT : (_Float16)Fold<FMT>::FP;
        half2v kk;
        kk[0] = d[g] * fold;  // exact: at most 7 significant bits
        kk[1] = kk[0];
        k2[g] = h2_as_u32(kk);
    }
}

// Decode group g (0..3) of a raw chunk into 8 FP16 pairs (elements 2i, 2i+1).
template <int FMT>
__device__ __forceinline__ void decode_group(const RawChunk<FMT>& rc, int g, uint32_t k2u,
                                             uint32_t (&out)[8])
{
    using F = Fmt<FMT>;
    const half2v k2 = u32_as_h2(k2u);
    if constexpr (F::BITS == 4) {
        const uint32_t w0 = rc.w[2 * g], w1 = rc.w[2 * g + 1];
        // FP: hardware E2M1 -> FP16 decode of byte i (low nibble first)
        uint32_t f[8];
        f[0] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w0, 1.0f, 0));
        f[1] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w0, 1.0f, 1));
        f[2] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w0, 1.0f, 2));
        f[3] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w0, 1.0f, 3));
        f[4] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w1, 1.0f, 0));
        f[5] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w1, 1.0f, 1));
        f[6] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w1, 1.0f, 2));
        f[7] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w1, 1.0f, 3));
        if constexpr (F::ADAPTIVE) {
            // INT: (n ^ 8) = q + 8 in [1, 15]; FP16 bits 0x6400 | (n ^ 8) = 1032 + q
            const bool is_int = (rc.sb >> (8 * g + 7)) & 1u;
            const uint32_t a0 = w0 ^ 0x88888888u, a1 = w1 ^ 0x88888888u;
            const uint32_t b0 = a0 >> 4, b1 = a1 >> 4;
            const uint32_t nib = 0x000F000Fu, magic = 0x64006400u;
            half2v bias;
            bias[0] = (_Float16)-1032.0f;
            bias[1] = (_Float16)-1032.0f;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const uint32_t sel = 0x0C000C00u | ((4u + i) << 16) | (uint32_t)i;
                const uint32_t p0 = and_or(__builtin_amdgcn_perm(b0, a0, sel), nib, magic);
                const uint32_t p1 = and_or(__builtin_amdgcn_perm(b1, a1, sel), nib, magic);
                const uint32_t s0 = pin(h2_as_u32(u32_as_h2(p0) + bias));
                const uint32_t s1 = pin(h2_as_u32(u32_as_h2(p1) + bias));
                f[i] = is_int ? s0 : f[i];
                f[4 + i] = is_int ? s1 : f[4 + i];
            }
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) out[i] = h2_as_u32(u32_as_h2(f[i]) * k2);
    } else {
        // IF3: 16 three-bit codes in 48 bits
        using D = FmtDerived<FMT>;
        const bool is_int = (rc.sb >> (8 * g + 7)) & 1u;
        const uint64_t bitsv = (uint64_t)rc.h[3 * g] | ((uint64_t)rc.h[3 * g + 1] << 16) |
                               ((uint64_t)rc.h[3 * g + 2] << 32);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            _Float16 v[2];
#pragma unroll
            for (int e = 0; e < 2; ++e) {
                const uint32_t c = (uint32_t)(bitsv >> (3 * (2 * i + e))) & 7u;
                const float qi = (float)((int)(c << 29) >> 29);
                const float qf = (c & D::SIGN_BIT) ? -fp_magnitude<FMT>(c & 3u) : fp_magnitude<FMT>(c & 3u);
                v[e] = (_Float16)(is_int ? qi : qf);
            }
            half2v hv;
            hv[0] = v[0];
            hv[1] = v[1];
            out[i] = h2_as_u32(hv * k2);
        }
    }
}

// Write the 16 decoded values of group g of `row` into an LDS stage.
__device__ __forceinline__ void store_group(_Float16* stage, int row, int g, const uint32_t (&v)[8])
{
    uint4* p0 = reinterpret_cast<uint4*>(stage + row * kPitch + (2 * g) * 8);
    uint4* p1 = reinterpret_cast<uint4*>(stage + row * kPitch + (2 * g + 1) * 8);
    *p0 = make_uint4(v[0], v[1], v[2], v[3]);
    *p1 = make_uint4(v[4], v[5], v[6], v[7]);
}

template <int FMT>
__device__ __forceinline__ void decode_store(const RawChunk<FMT>& rc, const uint32_t (&k2)[4],
                                             _Float16* stage, int row, int g)
{
    uint32_t v[8];
    decode_group<FMT>(rc, g, k2[g], v);
    store_group(stage, row, g, v);
}

// Fragments of one 16-wide K slice: 4 A blocks and 4 B blocks of 32 rows.
__device__ __forceinline__ void read_frags(const _Float16* As, const _Float16* Bs, int kk, int lane,
                                           int wm, int wn, half8 (&af)[4], half8 (&bf)[4])
{
    const int chunk = 2 * kk + (lane >> 5);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int r = wm * 128 + i * 32 + (lane & 31);
        af[i] = *reinterpret_cast<const half8*>(As + r * kPitch + chunk * 8);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int r = wn * 128 + j * 32 + (lane & 31);
        bf[j] = *reinterpret_cast<const half8*>(Bs + r * kPitch + chunk * 8);
    }
}

// One 64-wide K step: multiply LDS stage `cur` while decoding the next step's
// raw chunks (nxt_a, nxt_b) into the other stage, and load step s + 2 into
// (fill_a, fill_b) -- clamped to the last step: the extra loads and decodes
// near the end are harmless and keep the loop free of branches.  Fragments
// for slice kk + 1 are read while slice kk multiplies; the scheduling hints
// spread the decode (about 7 VALU operations per MFMA) and the LDS traffic
// between the MFMAs.
template <int FMT, bool EDGE>
__device__ __forceinline__ void gemm_step(int s, int nsteps, const uint8_t* __restrict__ a_codes,
                                          const uint8_t* __restrict__ a_scales,
                                          const uint8_t* __restrict__ b_codes,
                                          const uint8_t* __restrict__ b_scales, int64_t M,
                                          int64_t N, int64_t gpr, int64_t m0, int64_t n0,
                                          const RawChunk<FMT>& nxt_a, const RawChunk<FMT>& nxt_b,
                                          RawChunk<FMT>& fill_a, RawChunk<FMT>& fill_b,
                                          _Float16 (*lds)[2][kStageHalves], int cur,
                                          floatx16 (&acc)[4][4])
{
    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const _Float16* As = lds[cur][0];
    const _Float16* Bs = lds[cur][1];
    _Float16* Ad = lds[cur ^ 1][0];
    _Float16* Bd = lds[cur ^ 1][1];
    half8 af[2][4], bf[2][4];
    read_frags(As, Bs, 0, lane, wm, wn, af[0], bf[0]);
    uint32_t ka[4], kb[4];
    chunk_scales<FMT>(nxt_a.sb, ka);
    chunk_scales<FMT>(nxt_b.sb, kb);
    const int64_t gload = (int64_t)min(s + 2, nsteps - 1) * kGroupsPerStep;
    load_chunk<FMT, EDGE>(a_codes, a_scales, m0 + t, M, gpr, gload, fill_a);
    load_chunk<FMT, EDGE>(b_codes, b_scales, n0 + t, N, gpr, gload, fill_b);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
        const int f = kk & 1;
        if (kk < 3) read_frags(As, Bs, kk + 1, lane, wm, wn, af[f ^ 1], bf[f ^ 1]);
        decode_store<FMT>(nxt_a, ka, Ad, t, kk);
        decode_store<FMT>(nxt_b, kb, Bd, t, kk);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(af[f][i], bf[f][j], acc[i][j], 0, 0, 0);
        // interleave: MFMA, VALU x7, with the 8 fragment reads and the 4
        // decoded-tile writes spread over the first MFMAs
#pragma unroll
        for (int m = 0; m < 16; ++m) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x002, 7, 0);
            if (m < 8) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            if (m % 4 == 1) __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
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
                                          int64_t m0, int64_t n0, _Float16 (*lds)[2][kStageHalves])
{
    const int64_t gpr = K / kGroup;
    const int nsteps = (int)((gpr + kGroupsPerStep - 1) / kGroupsPerStep);
    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    const int wm = wave >> 1, wn = wave & 1;

    floatx16 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

    if (nsteps > 0) {
        RawChunk<FMT> a_nxt, b_nxt, a_fill, b_fill;
        load_chunk<FMT, EDGE>(a_codes, a_scales, m0 + t, M, gpr, 0, a_fill);
        load_chunk<FMT, EDGE>(b_codes, b_scales, n0 + t, N, gpr, 0, b_fill);
        const int64_t g1 = (int64_t)min(1, nsteps - 1) * kGroupsPerStep;
        load_chunk<FMT, EDGE>(a_codes, a_scales, m0 + t, M, gpr, g1, a_nxt);
        load_chunk<FMT, EDGE>(b_codes, b_scales, n0 + t, N, gpr, g1, b_nxt);
        uint32_t ka[4], kb[4];
        chunk_scales<FMT>(a_fill.sb, ka);
        chunk_scales<FMT>(b_fill.sb, kb);
#pragma unroll
        for (int g = 0; g < kGroupsPerStep; ++g) {
            decode_store<FMT>(a_fill, ka, lds[0][0], t, g);
            decode_store<FMT>(b_fill, kb, lds[0][1], t, g);
        }
        __syncthreads();
        for (int s = 0; s < nsteps; ++s) {
            gemm_step<FMT, EDGE>(s, nsteps, a_codes, a_scales, b_codes, b_scales, M, N, gpr, m0, n0,
                                 a_nxt, b_nxt, a_fill, b_fill, lds, s & 1, acc);
            const RawChunk<FMT> ta = a_nxt, tb = b_nxt;
            a_nxt = a_fill;
            b_nxt = b_fill;
            a_fill = ta;
            b_fill = tb;
        }
    }

    const float sc = (*a_ts * *b_ts) / (Fold<FMT>::FP * Fold<FMT>::FP);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t n = n0 + wn * 128 + j * 32 + (lane & 31);
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int64_t m = m0 + wm * 128 + i * 32 + (e >> 2) * 8 + (lane >> 5) * 4 + (e & 3);
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
// XCDs; they are remapped so that each XCD walks a contiguous band of tiles
// in row-major order, so the workgroups resident on one XCD share A rows in
// its L2.
template <int FMT, bool OUT_BF16>
__global__ __launch_bounds__(kGemmThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void gemm_tn_interior(const uint8_t* __restrict__ a_codes, const uint8_t* __restrict__ a_scales,
                      const float* __restrict__ a_ts, const uint8_t* __restrict__ b_codes,
                      const uint8_t* __restrict__ b_scales, const float* __restrict__ b_ts,
                      int64_t M, int64_t N, int64_t K, void* __restrict__ C, int64_t ldc,
                      int tiles_n)
{
    __shared__ __attribute__((aligned(16))) _Float16 lds[2][2][kStageHalves];
    const int nwg = gridDim.x;
    const int bid = blockIdx.x;
    const int tile = (nwg % 8 == 0) ? (bid % 8) * (nwg / 8) + bid / 8 : bid;
    const int64_t m0 = (int64_t)(tile / tiles_n) * kBM, n0 = (int64_t)(tile % tiles_n) * kBN;
    gemm_tile<FMT, OUT_BF16, false>(a_codes, a_scales, a_ts, b_codes, b_scales, b_ts, M, N, K, C,
                                    ldc, m0, n0, lds);
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
    __shared__ __attribute__((aligned(16))) _Float16 lds[2][2][kStageHalves];
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
                               a.b_scales, a.b_ts, a.M, a.N, a.K, a.c, a.ldc, (int)full_n);
        else
            hipLaunchKernelGGL((gemm_tn_interior<FMT, false>), dim3((unsigned)(full_m * full_n)),
                               dim3(kGemmThreads), 0, s, a.a_codes, a.a_scales, a.a_ts, a.b_codes,
                               a.b_scales, a.b_ts, a.M, a.N, a.K, a.c, a.ldc, (int)full_n);
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
