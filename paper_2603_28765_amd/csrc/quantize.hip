// quantize.hip -- tensor maximum and block quantizer kernels (gfx950).
//
// Pass 1 (tensor_max_*): every block reduces max|v| over its share of the
// groups (after the RHT when it is on) and writes one float to the
// workspace.  Pass 2 (quantize_*): every block re-reduces those partials to
// the same amax, so each computes the same alpha = amax / (M * 448) (Eq. 1);
// block (0,0) publishes it.  Then one lane quantizes one group of 16 values
// at a time (Eq. 2 and Fig. 3a) and stores its packed codes and scale byte.
//
// Row-wise: a group is 32 contiguous bytes of bf16, read with two 128-bit
// loads.  Strided axis: a 64x64 tile is staged through LDS so that a lane
// can gather 16 consecutive rows of one column.
#include <mutex>

#include "device.h"
#include "launch.h"

namespace ifq {

constexpr int kThreads = 256;

__device__ __forceinline__ float wave_max(float m)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off, 64));
    return m;
}

// Block-wide max (NT threads, red[NT / 64]); result valid in every thread.
template <int NT = kThreads>
__device__ __forceinline__ float block_max(float m, float* red)
{
    m = wave_max(m);
    const int wid = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) red[wid] = m;
    __syncthreads();
    float r = red[0];
#pragma unroll
    for (int i = 1; i < NT / 64; ++i) r = fmaxf(r, red[i]);
    __syncthreads();
    return r;
}

// Workgroup size of the tensor-max passes.  Their grid is capped at
// kMaxPartials workgroups (one partial each), so with the RHT -- about 130
// VALU operations per group of 16 -- 256-thread workgroups leave one
// wavefront per SIMD; 1024 threads give four.
template <bool RHT> constexpr int kMaxThreads = RHT ? 1024 : kThreads;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// 16 bf16 values (two 16-byte pieces, low piece first) as floats
__device__ __forceinline__ void unpack_group(u32x4 a, u32x4 b, float (&v)[kGroup])
{
    v[0] = bf16lo(a.x);  v[1] = bf16hi(a.x);  v[2] = bf16lo(a.y);  v[3] = bf16hi(a.y);
    v[4] = bf16lo(a.z);  v[5] = bf16hi(a.z);  v[6] = bf16lo(a.w);  v[7] = bf16hi(a.w);
    v[8] = bf16lo(b.x);  v[9] = bf16hi(b.x);  v[10] = bf16lo(b.y); v[11] = bf16hi(b.y);
    v[12] = bf16lo(b.z); v[13] = bf16hi(b.z); v[14] = bf16lo(b.w); v[15] = bf16hi(b.w);
}

// 64 consecutive groups (2 KiB at p, 16-byte aligned) read by one wavefront
// with two loads that each cover 1 KiB contiguously (a lane's two 16-byte
// pieces of one group would otherwise sit 32 bytes apart in every load, and
// each load would touch twice the cache lines): lane l reads pieces
// 2(l mod 32) + l/32 and 64 + 2(l mod 32) + l/32.  Lane l < 32 then holds the
// first half of group l and of group 32 + l, lane l + 32 their second halves;
// one swap across the wavefront's halves per dword leaves group l whole in
// lane l.  Every lane of the wavefront must be active.
__device__ __forceinline__ void load_wave_raw(const uint16_t* p, u32x4& a, u32x4& b)
{
    const int lane = threadIdx.x & 63;
    const int piece = 2 * (lane & 31) + (lane >> 5);
    const u32x4* q = reinterpret_cast<const u32x4*>(p);
    a = __builtin_nontemporal_load(q + piece);
    b = __builtin_nontemporal_load(q + 64 + piece);
}

// A group's 16 values from its raw bytes (wave: as loaded by load_wave_raw,
// else its two 16-byte pieces), with the RHT when RHT is set.  SCALE (the
// quantize passes): the transform as rht16 computes it.  Otherwise (the
// tensor-max passes, which scale their maximum instead): signs flipped on
// the packed bf16 pairs and the butterflies, without the 1/4.  (Flipping
// the packed pairs measured slower in the quantize pass.)
template <bool RHT, bool SCALE>
__device__ __forceinline__ void row_group_values(u32x4 a, u32x4 b, bool wave, uint32_t signs, float (&v)[kGroup])
{
    u32x4 lo = a, hi = b;
    if (wave) {
#pragma unroll
        for (int d = 0; d < 4; ++d) {
            const auto r = __builtin_amdgcn_permlane32_swap(a[d], b[d], false, false);
            lo[d] = r[0];
            hi[d] = r[1];
        }
    }
    if constexpr (RHT && !SCALE) {
#pragma unroll
        for (int d = 0; d < 4; ++d) {
            lo[d] ^= rht_pair_mask(signs, d);
            hi[d] ^= rht_pair_mask(signs, d + 4);
        }
    }
    unpack_group(lo, hi, v);
    if constexpr (RHT) {
        if constexpr (SCALE)
            rht16(v, signs);
        else
            hadamard16(v);
    }
}

// Raw bytes of group gc of row r: whole-wavefront loads when the wavefront's
// 64 groups lie in the row (returns true; row_group_values then assembles
// lane l's group), else the group's own two 16-byte pieces (returns false).
__device__ __forceinline__ bool load_row_group(const uint16_t* x, int64_t r, int64_t ld, int64_t gc,
                                               int64_t gpr, u32x4& a, u32x4& b)
{
    const int64_t gc0 = gc - (threadIdx.x & 63);  // the wavefront's first group
    if (gc0 + 64 <= gpr) {
        load_wave_raw(x + r * ld + gc0 * kGroup, a, b);
        return true;
    }
    const u32x4* q = reinterpret_cast<const u32x4*>(x + r * ld + gc * kGroup);
    a = __builtin_nontemporal_load(q);
    b = __builtin_nontemporal_load(q + 1);
    return false;
}

// alpha for this launch: the caller's, or Eq. 1 from the pass-1 partials.
__device__ __forceinline__ float resolve_alpha(bool scale_in, float* tensor_scale,
                                               const float* partials, int npartials,
                                               float denom_alpha, float* red)
{
    if (scale_in) return *tensor_scale;
    float m = 0.0f;
    for (int i = threadIdx.x; i < npartials; i += kThreads) m = fmaxf(m, partials[i]);
    m = block_max(m, red);
    float alpha = m / denom_alpha;
    if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) *tensor_scale = alpha;
    return alpha;
}

// Non-temporal stores: the outputs are written once and not read back by
// this launch, and streaming them past the caches keeps the write path at
// full rate (a wavefront's stores still cover whole lines).
template <int BITS> __device__ __forceinline__ void store_packed_nt(uint8_t* dst, const Packed<BITS>& p)
{
    if constexpr (BITS == 4) {
        __builtin_nontemporal_store(u32x2{p.w[0], p.w[1]}, reinterpret_cast<u32x2*>(dst));
    } else if constexpr (BITS == 6) {
        uint32_t* d = reinterpret_cast<uint32_t*>(dst);
        __builtin_nontemporal_store(p.w[0], d);
        __builtin_nontemporal_store(p.w[1], d + 1);
        __builtin_nontemporal_store(p.w[2], d + 2);
    } else {
        uint16_t* d = reinterpret_cast<uint16_t*>(dst);
        __builtin_nontemporal_store((uint16_t)p.w[0], d);
        __builtin_nontemporal_store((uint16_t)(p.w[0] >> 16), d + 1);
        __builtin_nontemporal_store((uint16_t)p.w[1], d + 2);
    }
}

// Quantize one (transformed) group and store its codes and scale byte.
template <int FMT, bool SR, bool NTS = false>
__device__ __forceinline__ void quantize_store(const float (&v)[kGroup], float alpha, const Div& denom,
                                               uint64_t seed, int64_t gi, uint8_t* __restrict__ codes,
                                               uint8_t* __restrict__ scales, int qflags)
{
    constexpr int BITS = Fmt<FMT>::BITS;
    Packed<BITS> p;
    const uint32_t sb = quantize_any<FMT, SR>(v, alpha, denom, qflags, seed, gi, p);
    if constexpr (NTS) {
        store_packed_nt<BITS>(codes + gi * (2 * BITS), p);
        if constexpr (Fmt<FMT>::G == 8) {
            __builtin_nontemporal_store((uint16_t)sb, reinterpret_cast<uint16_t*>(scales + 2 * gi));
        } else {
            __builtin_nontemporal_store((uint8_t)sb, scales + gi);
        }
    } else {
        store_packed<BITS>(codes + gi * (2 * BITS), p);
        if constexpr (Fmt<FMT>::G == 8) {
            scales[2 * gi] = (uint8_t)sb;
            scales[2 * gi + 1] = (uint8_t)(sb >> 8);
        } else {
            scales[gi] = (uint8_t)sb;
        }
    }
}

// --------------------------------------------------------------- row-wise

template <bool RHT, int NT = kMaxThreads<RHT>>
__global__ __launch_bounds__(NT) void tensor_max_rows(const uint16_t* __restrict__ x,
                                                      int64_t nrows, int64_t gpr,
                                                      int64_t ld, uint32_t signs,
                                                      float* __restrict__ partials)
{
    __shared__ float red[NT / 64];
    float m = 0.0f;
    const int64_t stride = (int64_t)gridDim.x * NT;
    for (int64_t r = blockIdx.y; r < nrows; r += gridDim.y) {
        int64_t gc = (int64_t)blockIdx.x * NT + threadIdx.x;
        const int64_t gc0 = gc - (threadIdx.x & 63);  // the wavefront's first group
        // four chunks of 64 groups in flight per wavefront: the grid is small
        // (at most kMaxPartials blocks), so bytes in flight come from unrolling.
        // The condition is the same in every lane of a wavefront.
        for (int64_t w0 = gc0; w0 + 3 * stride + 64 <= gpr; w0 += 4 * stride, gc += 4 * stride) {
            u32x4 a[4], b[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) load_wave_raw(x + r * ld + (w0 + u * stride) * kGroup, a[u], b[u]);
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                float v[kGroup];
                // without the RHT, which group a value is in does not matter
                row_group_values<RHT, false>(a[u], b[u], RHT, signs, v);
#pragma unroll
                for (int j = 0; j < kGroup; ++j) m = fmaxf(m, fabsf(v[j]));
            }
        }
        for (; gc < gpr; gc += stride) {
            const u32x4* q = reinterpret_cast<const u32x4*>(x + r * ld + gc * kGroup);
            float v[kGroup];
            row_group_values<RHT, false>(__builtin_nontemporal_load(q), __builtin_nontemporal_load(q + 1), false,
                                         signs, v);
#pragma unroll
            for (int j = 0; j < kGroup; ++j) m = fmaxf(m, fabsf(v[j]));
        }
    }
    if constexpr (RHT) m *= 0.25f;  // exact: the maximum of the transformed values
    m = block_max<NT>(m, red);
    if (threadIdx.x == 0) partials[blockIdx.y * gridDim.x + blockIdx.x] = m;
}

// ONE: the grid has a thread for every group of every row (nrows <= the
// grid's rows), so a thread quantizes at most one group and the kernel has
// no loop -- and none of the loop's 64-bit address registers, which keeps
// the IF4 kernel within 64 VGPRs (eight wavefronts per SIMD).
template <int FMT, bool RHT, bool SR, bool ONE>
__global__ __launch_bounds__(kThreads) void quantize_rows(
    const uint16_t* __restrict__ x, int64_t nrows, int64_t gpr, int64_t ld, uint32_t signs,
    uint64_t seed, int qflags, float scale_max, float denom_alpha, int scale_in,
    const float* __restrict__ partials, int npartials, uint8_t* __restrict__ codes,
    uint8_t* __restrict__ scales, float* tensor_scale)
{
    constexpr int BITS = Fmt<FMT>::BITS;
    __shared__ float red[kThreads / 64];
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    const int64_t gc_first = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    // One value per thread -- its pass-1 partial maximum, or alpha itself when
    // it is supplied -- then the block's first group are loaded before alpha
    // is reduced: loads complete in order, so the reduction waits only for
    // the first and the group's HBM latency overlaps it.  Both loads are
    // unconditional (a lane without a group reads group 0 and drops it), so
    // the wait for the first one stays partial.
    static_assert(kMaxPartials <= kThreads, "one partial per thread");
    const float* one = scale_in ? tensor_scale : partials + min((int)threadIdx.x, npartials - 1);
    const float first = *one;
    u32x4 pa, pb;
    bool pwave;
    {
        const int64_t w0 = gc_first - (threadIdx.x & 63);  // the wavefront's first group
        const bool row_ok = blockIdx.y < nrows;
        pwave = row_ok && w0 + 64 <= gpr;                  // the same in every lane
        if (pwave) {
            load_wave_raw(x + (int64_t)blockIdx.y * ld + w0 * kGroup, pa, pb);
        } else {
            const bool mine = row_ok && gc_first < gpr;
            const u32x4* q = reinterpret_cast<const u32x4*>(
                x + (mine ? (int64_t)blockIdx.y * ld + gc_first * kGroup : 0));
            pa = __builtin_nontemporal_load(q);
            pb = __builtin_nontemporal_load(q + 1);
        }
    }
    float alpha = first;
    if (!scale_in) {
        alpha = block_max((int)threadIdx.x < npartials ? first : 0.0f, red) / denom_alpha;
        if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) *tensor_scale = alpha;
    }
    const Div denom = make_div(alpha, alpha * scale_max);
    if constexpr (ONE) {
        // a wavefront with pwave has all 64 of its groups in the row, so
        // every lane takes part in row_group_values' cross-lane swaps
        if (blockIdx.y < nrows && gc_first < gpr) {
            float v[kGroup];
            row_group_values<RHT, true>(pa, pb, pwave, signs, v);
            quantize_store<FMT, SR, true>(v, alpha, denom, seed, (int64_t)blockIdx.y * gpr + gc_first, codes,
                                          scales, qflags);
        }
        return;
    }
    for (int64_t r = blockIdx.y; r < nrows; r += gridDim.y) {
        for (int64_t gc = gc_first; gc < gpr; gc += stride) {
            u32x4 a = pa, b = pb;
            bool wave = pwave;
            if (r != blockIdx.y || gc != gc_first) wave = load_row_group(x, r, ld, gc, gpr, a, b);
            float v[kGroup];
            row_group_values<RHT, true>(a, b, wave, signs, v);
            const int64_t gi = r * gpr + gc;
            quantize_store<FMT, SR, true>(v, alpha, denom, seed, gi, codes, scales, qflags);
        }
    }
}

// ---------------------------------------------------- strided (token) axis
// Tile: kTR rows (kTR/16 groups per column) x kTC columns of X, staged as
// bf16 in LDS.  Thread t handles column t % kTC and group t / kTC.
constexpr int kTR = 64, kTC = 64;

__device__ __forceinline__ void stage_tile(const uint16_t* __restrict__ x, int64_t rows,
                                           int64_t cols, int64_t ld, int64_t r0, int64_t c0,
                                           bool vec, uint16_t (*tile)[kTC + 2])
{
    // kTR rows x kTC columns = kTR * kTC / 8 chunks of 8 values
#pragma unroll
    for (int i = 0; i < kTR * kTC / 8 / kThreads; ++i) {
        const int ch = threadIdx.x + i * kThreads;
        const int rr = ch / (kTC / 8), cc = (ch % (kTC / 8)) * 8;
        const int64_t gr = r0 + rr, gcol = c0 + cc;
        uint16_t tmp[8];
        if (vec && gr < rows && gcol + 8 <= cols) {
            uint4 q = *reinterpret_cast<const uint4*>(x + gr * ld + gcol);
            tmp[0] = (uint16_t)q.x; tmp[1] = (uint16_t)(q.x >> 16);
            tmp[2] = (uint16_t)q.y; tmp[3] = (uint16_t)(q.y >> 16);
            tmp[4] = (uint16_t)q.z; tmp[5] = (uint16_t)(q.z >> 16);
            tmp[6] = (uint16_t)q.w; tmp[7] = (uint16_t)(q.w >> 16);
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e)
                tmp[e] = (gr < rows && gcol + e < cols) ? x[gr * ld + gcol + e] : (uint16_t)0;
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) tile[rr][cc + e] = tmp[e];
    }
}

template <bool RHT>
__global__ __launch_bounds__(kThreads) void tensor_max_strided(const uint16_t* __restrict__ x,
                                                               int64_t rows, int64_t cols,
                                                               int64_t ld, int vec, uint32_t signs,
                                                               float* __restrict__ partials)
{
    __shared__ uint16_t tile[kTR][kTC + 2];
    __shared__ float red[kThreads / 64];
    float m = 0.0f;
    const int c = threadIdx.x % kTC, q = threadIdx.x / kTC;
    for (int64_t c0 = (int64_t)blockIdx.x * kTC; c0 < cols; c0 += (int64_t)gridDim.x * kTC) {
        for (int64_t r0 = (int64_t)blockIdx.y * kTR; r0 < rows; r0 += (int64_t)gridDim.y * kTR) {
            stage_tile(x, rows, cols, ld, r0, c0, vec != 0, tile);
            __syncthreads();
            float v[kGroup];
#pragma unroll
            for (int j = 0; j < kGroup; ++j) v[j] = __uint_as_float((uint32_t)tile[q * kGroup + j][c] << 16);
            if constexpr (RHT) rht16(v, signs);  // rows beyond the matrix are zero groups
#pragma unroll
            for (int j = 0; j < kGroup; ++j) m = fmaxf(m, fabsf(v[j]));
            __syncthreads();
        }
    }
    m = block_max(m, red);
    if (threadIdx.x == 0) partials[blockIdx.y * gridDim.x + blockIdx.x] = m;
}

template <int FMT, bool RHT, bool SR>
__global__ __launch_bounds__(kThreads) void quantize_strided(
    const uint16_t* __restrict__ x, int64_t rows, int64_t cols, int64_t ld, int vec,
    uint32_t signs, uint64_t seed, int qflags, float scale_max, float denom_alpha, int scale_in,
    const float* __restrict__ partials, int npartials, uint8_t* __restrict__ codes,
    uint8_t* __restrict__ scales, float* tensor_scale)
{
    constexpr int BITS = Fmt<FMT>::BITS;
    __shared__ uint16_t tile[kTR][kTC + 2];
    __shared__ float red[kThreads / 64];
    const float alpha = resolve_alpha(scale_in, tensor_scale, partials, npartials, denom_alpha, red);
    const Div denom = make_div(alpha, alpha * scale_max);
    const int64_t gpr = rows / kGroup;  // groups per output row (= per column of X)
    const int c = threadIdx.x % kTC, q = threadIdx.x / kTC;
    for (int64_t c0 = (int64_t)blockIdx.x * kTC; c0 < cols; c0 += (int64_t)gridDim.x * kTC) {
        for (int64_t r0 = (int64_t)blockIdx.y * kTR; r0 < rows; r0 += (int64_t)gridDim.y * kTR) {
            stage_tile(x, rows, cols, ld, r0, c0, vec != 0, tile);
            __syncthreads();
            const int64_t col = c0 + c, g = r0 / kGroup + q;
            if (col < cols && g < gpr) {
                float v[kGroup];
#pragma unroll
                for (int j = 0; j < kGroup; ++j)
                    v[j] = __uint_as_float((uint32_t)tile[q * kGroup + j][c] << 16);
                if constexpr (RHT) rht16(v, signs);
                const int64_t gi = col * gpr + g;
                quantize_store<FMT, SR>(v, alpha, denom, seed, gi, codes, scales, qflags);
            }
            __syncthreads();
        }
    }
}

// ------------------------------------------- strided axis, register path
// When rows are 16-byte aligned (x and ld) and cols % 8 == 0, a lane loads
// the same 16 bytes (8 columns) from 16 consecutive rows: one wave
// instruction reads 1 KiB of one row, fully coalesced.  The lane then holds
// 8 complete column groups in 16 registers and quantizes them one after
// another -- no LDS and no barriers.  In the tensor-max pass every
// wavefront of a block covers the block's 512 columns (64 lanes x 8
// columns), and wavefront w of a block of W wavefronts takes row groups w,
// w + W, ... of the block's row range.
constexpr int kColsPerBlock = 64 * 8;          // 512: every wave spans the block's 512 columns

typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void load_col_block(const uint16_t* __restrict__ p, int64_t ld, u32x4v (&r)[kGroup])
{
#pragma unroll
    for (int j = 0; j < kGroup; ++j) r[j] = __builtin_nontemporal_load(reinterpret_cast<const u32x4v*>(p + j * ld));
}

// The RHT signs of a 16 x 8 bf16 block: row j is element j of each of the 8
// column groups, so one exclusive or per dword flips both of its values.
__device__ __forceinline__ void sign_rows(u32x4v (&r)[kGroup], uint32_t signs)
{
#pragma unroll
    for (int j = 0; j < kGroup; ++j) r[j] ^= ((signs >> j) & 1u) ? 0x80008000u : 0u;
}

// Column c (0..7) of the 16 x 8 bf16 block as 16 floats.
__device__ __forceinline__ void column_of(const u32x4v (&r)[kGroup], int c, float (&v)[kGroup])
{
#pragma unroll
    for (int j = 0; j < kGroup; ++j) {
        const uint32_t w = r[j][c >> 1];
        v[j] = (c & 1) ? bf16hi(w) : bf16lo(w);
    }
}

template <bool RHT, int NT = kMaxThreads<RHT>>
__global__ __launch_bounds__(NT) void tensor_max_cols(const uint16_t* __restrict__ x,
                                                      int64_t rows, int64_t cols, int64_t ld,
                                                      uint32_t signs, float* __restrict__ partials)
{
    __shared__ float red[NT / 64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t ngroups = rows / kGroup;
    float m = 0.0f;
    for (int64_t cb = blockIdx.x; cb * kColsPerBlock < cols; cb += gridDim.x) {
        const int64_t col = cb * kColsPerBlock + 8 * lane;
        if (col >= cols) continue;
        for (int64_t g = (int64_t)blockIdx.y * (NT / 64) + wave; g < ngroups; g += (int64_t)gridDim.y * (NT / 64)) {
            u32x4v r[kGroup];
            load_col_block(x + g * kGroup * ld + col, ld, r);
            if constexpr (RHT) sign_rows(r, signs);
#pragma unroll
            for (int c = 0; c < 8; ++c) {
                float v[kGroup];
                column_of(r, c, v);
                if constexpr (RHT) hadamard16(v);
#pragma unroll
                for (int j = 0; j < kGroup; ++j) m = fmaxf(m, fabsf(v[j]));
            }
        }
    }
    if constexpr (RHT) m *= 0.25f;  // exact: the maximum of the transformed values
    m = block_max<NT>(m, red);
    if (threadIdx.x == 0) partials[blockIdx.y * gridDim.x + blockIdx.x] = m;
}

// Pass 2 of the register path.  A block owns a tile of 64 columns x 1024
// rows (64 groups per output row) and stages its output in LDS (36 KiB) so
// that every output row segment -- 512 bytes of codes, 64 of scales -- is
// written as whole cache lines, with non-temporal stores (measured against
// 2048-row tiles: more workgroups in flight, 20 % faster with round to
// nearest).  Lane l of wavefront w handles column chunk
// l / 8 (8 columns) and group l % 8 of the wavefront's 8 groups per round;
// one load instruction reads 16 B from each of 8 rows' 128-byte column
// segments.  LDS rows are XOR-swizzled by 8 (col / 8) slots, which keeps the
// 8-byte code writes of a 32-lane pass on distinct banks.
constexpr int kColTile = 64;          // columns (output rows) per block
constexpr int kGrpTile = 64;          // groups per output row per block
constexpr int kCodeRowBytes = kGrpTile * 8;

// IF4 with stochastic rounding needs about 190 VGPRs, which allows two
// wavefronts per SIMD; asking for three (at most 168 VGPRs, a few values
// spilled to scratch) measured faster on dY 8192 x 14336 (137 -> 128 us).
template <int FMT, bool RHT, bool SR>
__global__ __launch_bounds__(kThreads)
__attribute__((amdgpu_waves_per_eu(SR && Fmt<FMT>::ADAPTIVE ? 3 : 1))) void quantize_cols(
    const uint16_t* __restrict__ x, int64_t rows, int64_t cols, int64_t ld, uint32_t signs,
    uint64_t seed, int qflags, float scale_max, float denom_alpha, int scale_in,
    const float* __restrict__ partials, int npartials, uint8_t* __restrict__ codes,
    uint8_t* __restrict__ scales, float* tensor_scale)
{
    static_assert(Fmt<FMT>::BITS == 4, "register path stores 8-byte code groups");
    __shared__ __attribute__((aligned(16))) uint8_t lcodes[kColTile * kCodeRowBytes];
    __shared__ __attribute__((aligned(16))) uint8_t lscales[kColTile * kGrpTile];
    __shared__ float red[kThreads / 64];
    const float alpha = resolve_alpha(scale_in, tensor_scale, partials, npartials, denom_alpha, red);
    const Div denom = make_div(alpha, alpha * scale_max);
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int64_t ngroups = rows / kGroup;  // groups per output row (= per column of X)
    const int64_t c0 = (int64_t)blockIdx.x * kColTile, g0 = (int64_t)blockIdx.y * kGrpTile;
    const int ntg = (int)min<int64_t>(kGrpTile, ngroups - g0);
    const int ncol = (int)min<int64_t>(kColTile, cols - c0);
    const int cc = lane >> 3, q = lane & 7;
    const int sw = 8 * cc;  // swizzle of the LDS rows 8 cc .. 8 cc + 7
    for (int rg = 0; rg < ntg; rg += 32) {
        const int gl = rg + 8 * wave + q;
        if (gl < ntg && 8 * cc < ncol) {
            u32x4v r[kGroup];
            load_col_block(x + (g0 + gl) * kGroup * ld + c0 + 8 * cc, ld, r);
            if constexpr (RHT) sign_rows(r, signs);
#pragma unroll
            for (int c = 0; c < 8; ++c) {
                float v[kGroup];
                column_of(r, c, v);
                if constexpr (RHT) {
                    hadamard16(v);
#pragma unroll
                    for (int j = 0; j < kGroup; ++j) v[j] = v[j] * 0.25f;
                }
                const int64_t gi = (c0 + 8 * cc + c) * ngroups + g0 + gl;  // SR counter: global group index
                Packed<4> pp;
                const uint32_t sb = quantize_any<FMT, SR>(v, alpha, denom, qflags, seed, gi, pp);
                const uint2 pk = make_uint2(pp.w[0], pp.w[1]);
                const int row = 8 * cc + c;
                *reinterpret_cast<uint2*>(lcodes + row * kCodeRowBytes + (gl ^ sw) * 8) = pk;
                lscales[row * kGrpTile + (gl ^ sw)] = (uint8_t)sb;
            }
        }
    }
    __syncthreads();
    // codes: ncol rows x ntg * 8 bytes, 16-byte pieces (groups 2p, 2p + 1)
    const int ppr = ntg / 2;
    for (int idx = t; idx < ncol * ppr; idx += kThreads) {
        const int row = idx / ppr, pc = idx % ppr;
        const int s = 8 * (row >> 3);
        const uint4 v = *reinterpret_cast<const uint4*>(lcodes + row * kCodeRowBytes + ((2 * pc) ^ s) * 8);
        __builtin_nontemporal_store(u32x4{v.x, v.y, v.z, v.w},
                                    reinterpret_cast<u32x4*>(codes + ((c0 + row) * ngroups + g0 + 2 * pc) * 8));
    }
    // scales: ncol rows x ntg bytes, 16-byte pieces (bytes keep the swizzle of 8-slot blocks)
    const int spr = ntg / 16;
    for (int idx = t; idx < ncol * spr; idx += kThreads) {
        const int row = idx / spr, pc = idx % spr;
        const int s = 8 * (row >> 3);
        uint32_t w4[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            uint32_t wv = 0;
#pragma unroll
            for (int b = 0; b < 4; ++b)
                wv |= (uint32_t)lscales[row * kGrpTile + ((16 * pc + 4 * k + b) ^ s)] << (8 * b);
            w4[k] = wv;
        }
        __builtin_nontemporal_store(u32x4{w4[0], w4[1], w4[2], w4[3]},
                                    reinterpret_cast<u32x4*>(scales + (c0 + row) * ngroups + g0 + 16 * pc));
    }
}

__global__ void write_scalar(float* p, float v) { *p = v; }

// ------------------------------------------- dual layouts from one read
// Training needs each of X, W and dY packed both ways: along its columns
// (row-wise) and along its rows (strided, the packed form of the
// transpose).  One launch per pass reads each 64 x 64 tile once into LDS;
// thread t then takes column group (column t % 64, group t / 64) for the
// strided output and row group (row t / 4, group t % 4) for the row-wise
// output, each side with its own RHT / SR / margin / alpha.  Results equal
// two separate quantizer calls bit for bit.
struct DualSideK {
    uint8_t* codes;
    uint8_t* scales;
    float* tensor_scale;
    const float* partials;
    uint64_t seed;
    float scale_max, denom_alpha;
    int qflags, rht, scale_in;
};

struct DualK {
    const uint16_t* x;
    int64_t rows, cols, ld;
    int vec, npartials;
    uint32_t signs;
    DualSideK row, col;
};

__device__ __forceinline__ void tile_col_group(uint16_t (*tile)[kTC + 2], int c, int q, float (&v)[kGroup])
{
#pragma unroll
    for (int j = 0; j < kGroup; ++j) v[j] = __uint_as_float((uint32_t)tile[q * kGroup + j][c] << 16);
}

__device__ __forceinline__ void tile_row_group(uint16_t (*tile)[kTC + 2], int r, int g, float (&v)[kGroup])
{
    // row pitch 132 bytes: 4-byte aligned pairs
    const uint32_t* p = reinterpret_cast<const uint32_t*>(&tile[r][kGroup * g]);
#pragma unroll
    for (int i = 0; i < kGroup / 2; ++i) {
        const uint32_t w = p[i];
        v[2 * i] = bf16lo(w);
        v[2 * i + 1] = bf16hi(w);
    }
}

__global__ __launch_bounds__(kThreads) void tensor_max_dual(DualK a, float* __restrict__ part_row,
                                                            float* __restrict__ part_col)
{
    __shared__ __attribute__((aligned(16))) uint16_t tile[kTR][kTC + 2];
    __shared__ float red[kThreads / 64];
    float mr = 0.0f, mc = 0.0f;
    const int t = threadIdx.x;
    const int c = t % kTC, q = t / kTC, r = t / 4, g = t % 4;
    for (int64_t c0 = (int64_t)blockIdx.x * kTC; c0 < a.cols; c0 += (int64_t)gridDim.x * kTC) {
        for (int64_t r0 = (int64_t)blockIdx.y * kTR; r0 < a.rows; r0 += (int64_t)gridDim.y * kTR) {
            stage_tile(a.x, a.rows, a.cols, a.ld, r0, c0, a.vec != 0, tile);
            __syncthreads();
            // elements outside the matrix are staged as zeros: they do not
            // change a maximum, and an RHT of a zero-padded group is only
            // taken where the whole group is inside
            float v[kGroup];
            if (c0 + c < a.cols && r0 + kGroup * q < a.rows) {
                tile_col_group(tile, c, q, v);
                if (a.col.rht) rht16(v, a.signs);
#pragma unroll
                for (int j = 0; j < kGroup; ++j) mc = fmaxf(mc, fabsf(v[j]));
            }
            if (r0 + r < a.rows && c0 + kGroup * g < a.cols) {
                tile_row_group(tile, r, g, v);
                if (a.row.rht) rht16(v, a.signs);
#pragma unroll
                for (int j = 0; j < kGroup; ++j) mr = fmaxf(mr, fabsf(v[j]));
            }
            __syncthreads();
        }
    }
    mr = block_max(mr, red);
    mc = block_max(mc, red);
    if (t == 0) {
        part_row[blockIdx.y * gridDim.x + blockIdx.x] = mr;
        part_col[blockIdx.y * gridDim.x + blockIdx.x] = mc;
    }
}

template <int FMT, bool SR_ROW, bool SR_COL>
__global__ __launch_bounds__(kThreads) void quantize_dual(DualK a)
{
    __shared__ __attribute__((aligned(16))) uint16_t tile[kTR][kTC + 2];
    __shared__ float red[kThreads / 64];
    const float alpha_r = resolve_alpha(a.row.scale_in, a.row.tensor_scale, a.row.partials, a.npartials,
                                        a.row.denom_alpha, red);
    const float alpha_c = resolve_alpha(a.col.scale_in, a.col.tensor_scale, a.col.partials, a.npartials,
                                        a.col.denom_alpha, red);
    const Div denom_r = make_div(alpha_r, alpha_r * a.row.scale_max);
    const Div denom_c = make_div(alpha_c, alpha_c * a.col.scale_max);
    const int64_t gpr_r = a.cols / kGroup, gpr_c = a.rows / kGroup;
    const int t = threadIdx.x;
    const int c = t % kTC, q = t / kTC, r = t / 4, g = t % 4;
    for (int64_t c0 = (int64_t)blockIdx.x * kTC; c0 < a.cols; c0 += (int64_t)gridDim.x * kTC) {
        for (int64_t r0 = (int64_t)blockIdx.y * kTR; r0 < a.rows; r0 += (int64_t)gridDim.y * kTR) {
            stage_tile(a.x, a.rows, a.cols, a.ld, r0, c0, a.vec != 0, tile);
            __syncthreads();
            float v[kGroup];
            const int64_t col = c0 + c, gc = r0 / kGroup + q;
            if (col < a.cols && gc < gpr_c) {
                tile_col_group(tile, c, q, v);
                if (a.col.rht) rht16(v, a.signs);
                quantize_store<FMT, SR_COL>(v, alpha_c, denom_c, a.col.seed, col * gpr_c + gc, a.col.codes,
                                            a.col.scales, a.col.qflags);
            }
            const int64_t row = r0 + r, gr = c0 / kGroup + g;
            if (row < a.rows && gr < gpr_r) {
                tile_row_group(tile, r, g, v);
                if (a.row.rht) rht16(v, a.signs);
                quantize_store<FMT, SR_ROW>(v, alpha_r, denom_r, a.row.seed, row * gpr_r + gr, a.row.codes,
                                            a.row.scales, a.row.qflags);
            }
            __syncthreads();
        }
    }
}


// ------------------------------------------------------------- launcher

static inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// 128-bit tile loads need 16-byte aligned row starts; otherwise stage by element.
static inline int strided_vec_ok(const QuantArgs& a)
{
    return (reinterpret_cast<uintptr_t>(a.x) % 16 == 0 && a.ld % 8 == 0) ? 1 : 0;
}

// The register path loads 16 bytes (8 columns) per lane and row and stores
// 16-byte pieces of codes and scales: 4-bit formats, 16-byte aligned rows of
// X, cols % 8 == 0, and 16 groups per output row multiple (rows % 256 == 0)
// with 16-byte aligned code and scale buffers.
static inline bool strided_load_ok(const QuantArgs& a)
{
    return reinterpret_cast<uintptr_t>(a.x) % 16 == 0 && a.ld % 8 == 0 && a.cols % 8 == 0;
}

template <int FMT>
static inline bool strided_cols_ok(const QuantArgs& a)
{
    return Fmt<FMT>::BITS == 4 && Fmt<FMT>::G == 16 && strided_load_ok(a) && (a.rows / kGroup) % 16 == 0 &&
           a.rows / kGroup / kGrpTile < 65536 && reinterpret_cast<uintptr_t>(a.codes) % 16 == 0 &&
           reinterpret_cast<uintptr_t>(a.scales) % 16 == 0;
}

template <int FMT, bool RHT, bool SR>
static hipError_t launch_q(const QuantArgs& a, hipStream_t s, int npartials, float scale_max,
                           float denom_alpha)
{
    const int scale_in = (a.flags & IFQ_SCALE_IN) ? 1 : 0;
    const int qflags = ((a.flags & IFQ_SR_RTN_TYPE) ? kQSrRtnType : 0) |
                       ((a.flags & IFQ_MARGIN_16_17) ? kQMargin : 0);
    if constexpr (Fmt<FMT>::BITS == 4 && Fmt<FMT>::G == 16) {
        if ((a.flags & IFQ_AXIS_STRIDED) && strided_cols_ok<FMT>(a)) {
            dim3 grid((unsigned)cdiv(a.cols, kColTile), (unsigned)cdiv(a.rows / kGroup, kGrpTile));
            hipLaunchKernelGGL((quantize_cols<FMT, RHT, SR>), grid, dim3(kThreads), 0, s, a.x, a.rows,
                               a.cols, a.ld, a.signs, a.seed, qflags, scale_max, denom_alpha, scale_in, a.partials,
                               npartials, a.codes, a.scales, a.tensor_scale);
            return hipGetLastError();
        }
    }
    if (a.flags & IFQ_AXIS_STRIDED) {
        dim3 grid((unsigned)cdiv(a.cols, kTC), (unsigned)std::min<int64_t>(cdiv(a.rows, kTR), 65535));
        hipLaunchKernelGGL((quantize_strided<FMT, RHT, SR>), grid, dim3(kThreads), 0, s, a.x,
                           a.rows, a.cols, a.ld, strided_vec_ok(a), a.signs, a.seed, qflags, scale_max, denom_alpha, scale_in,
                           a.partials, npartials, a.codes, a.scales, a.tensor_scale);
    } else {
        const bool flat = a.ld == a.cols;
        const int64_t nrows = flat ? 1 : a.rows;
        const int64_t gpr = flat ? a.rows * a.cols / kGroup : a.cols / kGroup;
        const int64_t ld = flat ? 0 : a.ld;
        dim3 grid((unsigned)cdiv(gpr, kThreads), (unsigned)std::min<int64_t>(nrows, 65535));
        if (nrows <= 65535)
            hipLaunchKernelGGL((quantize_rows<FMT, RHT, SR, true>), grid, dim3(kThreads), 0, s, a.x, nrows,
                               gpr, ld, a.signs, a.seed, qflags, scale_max, denom_alpha, scale_in, a.partials,
                               npartials, a.codes, a.scales, a.tensor_scale);
        else
            hipLaunchKernelGGL((quantize_rows<FMT, RHT, SR, false>), grid, dim3(kThreads), 0, s, a.x, nrows,
                               gpr, ld, a.signs, a.seed, qflags, scale_max, denom_alpha, scale_in, a.partials,
                               npartials, a.codes, a.scales, a.tensor_scale);
    }
    return hipGetLastError();
}

template <bool RHT>
static hipError_t launch_tensor_max(const QuantArgs& a, hipStream_t s, int* npartials)
{
    if ((a.flags & IFQ_AXIS_STRIDED) && strided_load_ok(a)) {
        int64_t bx = std::min<int64_t>(cdiv(a.cols, kColsPerBlock), kMaxPartials);
        int64_t by = std::max<int64_t>(
            1, std::min<int64_t>(cdiv(a.rows / kGroup, kMaxThreads<RHT> / 64), kMaxPartials / bx));
        *npartials = (int)(bx * by);
        hipLaunchKernelGGL((tensor_max_cols<RHT>), dim3((unsigned)bx, (unsigned)by), dim3(kMaxThreads<RHT>), 0,
                           s, a.x, a.rows, a.cols, a.ld, a.signs, a.partials);
    } else if (a.flags & IFQ_AXIS_STRIDED) {
        int64_t tx = cdiv(a.cols, kTC), ty = cdiv(a.rows, kTR);
        int64_t bx = std::min<int64_t>(tx, kMaxPartials);
        int64_t by = std::max<int64_t>(1, std::min<int64_t>(ty, kMaxPartials / bx));
        *npartials = (int)(bx * by);
        hipLaunchKernelGGL((tensor_max_strided<RHT>), dim3((unsigned)bx, (unsigned)by), dim3(kThreads),
                           0, s, a.x, a.rows, a.cols, a.ld, strided_vec_ok(a), a.signs, a.partials);
    } else {
        const bool flat = a.ld == a.cols;
        const int64_t nrows = flat ? 1 : a.rows;
        const int64_t gpr = flat ? a.rows * a.cols / kGroup : a.cols / kGroup;
        const int64_t ld = flat ? 0 : a.ld;
        int64_t by = std::min<int64_t>(nrows, kMaxPartials);
        int64_t bx = std::max<int64_t>(1, std::min<int64_t>(cdiv(gpr, kMaxThreads<RHT>), kMaxPartials / by));
        *npartials = (int)(bx * by);
        hipLaunchKernelGGL((tensor_max_rows<RHT>), dim3((unsigned)bx, (unsigned)by), dim3(kMaxThreads<RHT>), 0,
                           s, a.x, nrows, gpr, ld, a.signs, a.partials);
    }
    return hipGetLastError();
}

template <int FMT>
static hipError_t dispatch_fmt(const QuantArgs& a, hipStream_t s, int npartials, float scale_max,
                               float denom_alpha)
{
    const bool rht = a.flags & IFQ_RHT, sr = a.flags & IFQ_SR;
    if (rht && sr) return launch_q<FMT, true, true>(a, s, npartials, scale_max, denom_alpha);
    if (rht) return launch_q<FMT, true, false>(a, s, npartials, scale_max, denom_alpha);
    if (sr) return launch_q<FMT, false, true>(a, s, npartials, scale_max, denom_alpha);
    return launch_q<FMT, false, false>(a, s, npartials, scale_max, denom_alpha);
}

template <int FMT> static void targets(float& m, float& a8)
{
    m = Fmt<FMT>::M;
    a8 = Fmt<FMT>::A8;
}

hipError_t launch_quantize(const QuantArgs& a, hipStream_t s)
{
    // M and the E4M3 factor of Eq. 1-2 (M * 16/17 with the gradient margin
    // of Sec. 4.1)
    float scale_max = 0.0f, a8 = 0.0f;
    switch (a.fmt) {
        case IFQ_FMT_IF4: targets<IFQ_FMT_IF4>(scale_max, a8); break;
        case IFQ_FMT_NVFP4: targets<IFQ_FMT_NVFP4>(scale_max, a8); break;
        case IFQ_FMT_IF3: targets<IFQ_FMT_IF3>(scale_max, a8); break;
        case IFQ_FMT_IF6_E2M3: targets<IFQ_FMT_IF6_E2M3>(scale_max, a8); break;
        case IFQ_FMT_IF6_E3M2: targets<IFQ_FMT_IF6_E3M2>(scale_max, a8); break;
        case IFQ_FMT_NVINT4: targets<IFQ_FMT_NVINT4>(scale_max, a8); break;
        case IFQ_FMT_NVFP4_46: targets<IFQ_FMT_NVFP4_46>(scale_max, a8); break;
        case IFQ_FMT_IF4_BS8: targets<IFQ_FMT_IF4_BS8>(scale_max, a8); break;
        case IFQ_FMT_IF3_BS8: targets<IFQ_FMT_IF3_BS8>(scale_max, a8); break;
        case IFQ_FMT_NVFP4_BS8: targets<IFQ_FMT_NVFP4_BS8>(scale_max, a8); break;
        default: return hipErrorInvalidValue;
    }
    if (a.flags & IFQ_MARGIN_16_17) scale_max = (float)((double)scale_max * 16.0 / 17.0);
    const float denom_alpha = scale_max * a8;
    const bool scale_in = a.flags & IFQ_SCALE_IN;

    if (a.rows == 0 || a.cols == 0) {  // empty tensor: alpha = 0, nothing to quantize
        if (!scale_in) hipLaunchKernelGGL(write_scalar, dim3(1), dim3(1), 0, s, a.tensor_scale, 0.0f);
        return hipGetLastError();
    }
    int npartials = 0;
    if (!scale_in) {
        hipError_t e = (a.flags & IFQ_RHT) ? launch_tensor_max<true>(a, s, &npartials)
                                            : launch_tensor_max<false>(a, s, &npartials);
        if (e != hipSuccess) return e;
    }
    switch (a.fmt) {
        case IFQ_FMT_IF4: return dispatch_fmt<IFQ_FMT_IF4>(a, s, npartials, scale_max, denom_alpha);
        case IFQ_FMT_NVFP4: return dispatch_fmt<IFQ_FMT_NVFP4>(a, s, npartials, scale_max, denom_alpha);
        case IFQ_FMT_IF3: return dispatch_fmt<IFQ_FMT_IF3>(a, s, npartials, scale_max, denom_alpha);
        case IFQ_FMT_IF6_E2M3: return dispatch_fmt<IFQ_FMT_IF6_E2M3>(a, s, npartials, scale_max, denom_alpha);
        case IFQ_FMT_IF6_E3M2: return dispatch_fmt<IFQ_FMT_IF6_E3M2>(a, s, npartials, scale_max, denom_alpha);
        case IFQ_FMT_NVINT4: return dispatch_fmt<IFQ_FMT_NVINT4>(a, s, npartials, scale_max, denom_alpha);
        case IFQ_FMT_NVFP4_46: return dispatch_fmt<IFQ_FMT_NVFP4_46>(a, s, npartials, scale_max, denom_alpha);
        case IFQ_FMT_IF4_BS8: return dispatch_fmt<IFQ_FMT_IF4_BS8>(a, s, npartials, scale_max, denom_alpha);
        case IFQ_FMT_IF3_BS8: return dispatch_fmt<IFQ_FMT_IF3_BS8>(a, s, npartials, scale_max, denom_alpha);
        default: return dispatch_fmt<IFQ_FMT_NVFP4_BS8>(a, s, npartials, scale_max, denom_alpha);
    }
}

// Register path of the dual quantizer (the strided register layout of
// quantize_cols / tensor_max_cols, same conditions).  A lane holds 16 rows x
// 8 columns; the lane holding the other 8 columns of the same 16 rows is its
// DPP partner (CTRL: row_ror:8 for lane ^ 8, quad_perm [1,0,3,2] for
// lane ^ 1).  Each sends the half the other needs -- the even-chunk lane keeps
// rows 0-7, the odd one rows 8-15 -- so after 32 dword moves each lane holds 8
// complete row groups: row 8 * odd + j, columns 0-15 of the pair.
template <int CTRL>
__device__ __forceinline__ void row_group_of_pair(const u32x4v (&r)[kGroup], bool odd, int j, float (&v)[kGroup])
{
    u32x4v send = odd ? r[j] : r[8 + j];
    u32x4v recv;
#pragma unroll
    for (int e = 0; e < 4; ++e)
        recv[e] = (uint32_t)__builtin_amdgcn_mov_dpp((int)send[e], CTRL, 0xF, 0xF, false);
    const u32x4v lo = odd ? recv : r[j];
    const u32x4v hi = odd ? r[8 + j] : recv;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        v[2 * i] = bf16lo(lo[i]);
        v[2 * i + 1] = bf16hi(lo[i]);
        v[8 + 2 * i] = bf16lo(hi[i]);
        v[8 + 2 * i + 1] = bf16hi(hi[i]);
    }
}

constexpr int kDppRor8 = 0x128;    // row_ror:8 -> lane ^ 8 within 16-lane rows
constexpr int kDppSwap1 = 0xB1;    // quad_perm [1,0,3,2] -> lane ^ 1

__global__ __launch_bounds__(kThreads) void tensor_max_cols_dual(DualK a, float* __restrict__ part_row,
                                                                 float* __restrict__ part_col)
{
    __shared__ float red[kThreads / 64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t ngroups = a.rows / kGroup;
    const bool odd = lane & 1;  // chunk 8 * lane: partner lane ^ 1
    float mr = 0.0f, mc = 0.0f;
    for (int64_t cb = blockIdx.x; cb * kColsPerBlock < a.cols; cb += gridDim.x) {
        const int64_t col = cb * kColsPerBlock + 8 * lane;
        if (col >= a.cols) continue;  // cols % 16 == 0: partners leave together
        for (int64_t g = (int64_t)blockIdx.y * 4 + wave; g < ngroups; g += (int64_t)gridDim.y * 4) {
            u32x4v r[kGroup];
            load_col_block(a.x + g * kGroup * a.ld + col, a.ld, r);
#pragma unroll
            for (int c = 0; c < 8; ++c) {
                float v[kGroup];
                column_of(r, c, v);
                if (!a.row.rht) {
#pragma unroll
                    for (int j = 0; j < kGroup; ++j) mr = fmaxf(mr, fabsf(v[j]));
                }
                if (a.col.rht) rht16(v, a.signs);
#pragma unroll
                for (int j = 0; j < kGroup; ++j) mc = fmaxf(mc, fabsf(v[j]));
            }
            if (a.row.rht) {
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    float v[kGroup];
                    row_group_of_pair<kDppSwap1>(r, odd, j, v);
                    rht16(v, a.signs);
#pragma unroll
                    for (int e = 0; e < kGroup; ++e) mr = fmaxf(mr, fabsf(v[e]));
                }
            }
        }
    }
    mr = block_max(mr, red);
    mc = block_max(mc, red);
    if (threadIdx.x == 0) {
        part_row[blockIdx.y * gridDim.x + blockIdx.x] = mr;
        part_col[blockIdx.y * gridDim.x + blockIdx.x] = mc;
    }
}

// Pass 2 with round-to-nearest on both sides: quantize_cols' tile (64
// columns x 1024 rows, strided output staged in LDS and written as whole
// lines) plus the row-wise groups of the same registers, stored directly
// (8 code bytes and one scale byte per group; the four groups of a pair row
// are contiguous).
template <int FMT, bool SR_ROW, bool SR_COL>
__global__ __launch_bounds__(kThreads) void quantize_cols_dual(DualK a)
{
    __shared__ __attribute__((aligned(16))) uint8_t lcodes[kColTile * kCodeRowBytes];
    __shared__ __attribute__((aligned(16))) uint8_t lscales[kColTile * kGrpTile];
    __shared__ float red[kThreads / 64];
    const float alpha_r = resolve_alpha(a.row.scale_in, a.row.tensor_scale, a.row.partials, a.npartials,
                                        a.row.denom_alpha, red);
    const float alpha_c = resolve_alpha(a.col.scale_in, a.col.tensor_scale, a.col.partials, a.npartials,
                                        a.col.denom_alpha, red);
    const Div denom_r = make_div(alpha_r, alpha_r * a.row.scale_max);
    const Div denom_c = make_div(alpha_c, alpha_c * a.col.scale_max);
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int64_t ngroups = a.rows / kGroup, gpr_r = a.cols / kGroup;
    const int64_t c0 = (int64_t)blockIdx.x * kColTile, g0 = (int64_t)blockIdx.y * kGrpTile;
    const int ntg = (int)min<int64_t>(kGrpTile, ngroups - g0);
    const int ncol = (int)min<int64_t>(kColTile, a.cols - c0);
    const int cc = lane >> 3, q = lane & 7;
    const bool odd = cc & 1;
    const int sw = 8 * cc;
    for (int rg = 0; rg < ntg; rg += 32) {
        const int gl = rg + 8 * wave + q;
        // ncol is a multiple of 16, so both chunks of a pair pass or fail together
        if (gl < ntg && 8 * cc < ncol) {
            u32x4v r[kGroup];
            load_col_block(a.x + (g0 + gl) * kGroup * a.ld + c0 + 8 * cc, a.ld, r);
#pragma unroll
            for (int c = 0; c < 8; ++c) {
                float v[kGroup];
                column_of(r, c, v);
                if (a.col.rht) rht16(v, a.signs);
                const int64_t gi = (c0 + 8 * cc + c) * ngroups + g0 + gl;
                Packed<4> pp;
                const uint32_t sb = quantize_any<FMT, SR_COL>(v, alpha_c, denom_c, a.col.qflags, a.col.seed, gi, pp);
                const int row = 8 * cc + c;
                *reinterpret_cast<uint2*>(lcodes + row * kCodeRowBytes + (gl ^ sw) * 8) = make_uint2(pp.w[0], pp.w[1]);
                lscales[row * kGrpTile + (gl ^ sw)] = (uint8_t)sb;
            }
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                float v[kGroup];
                row_group_of_pair<kDppRor8>(r, odd, j, v);
                if (a.row.rht) rht16(v, a.signs);
                const int64_t row = (g0 + gl) * kGroup + 8 * (odd ? 1 : 0) + j;
                const int64_t gi = row * gpr_r + c0 / kGroup + (cc >> 1);
                Packed<4> pp;
                const uint32_t sb = quantize_any<FMT, SR_ROW>(v, alpha_r, denom_r, a.row.qflags, a.row.seed, gi, pp);
                *reinterpret_cast<uint2*>(a.row.codes + gi * 8) = make_uint2(pp.w[0], pp.w[1]);
                a.row.scales[gi] = (uint8_t)sb;
            }
        }
    }
    __syncthreads();
    uint8_t* codes = a.col.codes;
    uint8_t* scales = a.col.scales;
    const int ppr = ntg / 2;
    for (int idx = t; idx < ncol * ppr; idx += kThreads) {
        const int row = idx / ppr, pc = idx % ppr;
        const int s = 8 * (row >> 3);
        const uint4 v = *reinterpret_cast<const uint4*>(lcodes + row * kCodeRowBytes + ((2 * pc) ^ s) * 8);
        __builtin_nontemporal_store(u32x4{v.x, v.y, v.z, v.w},
                                    reinterpret_cast<u32x4*>(codes + ((c0 + row) * ngroups + g0 + 2 * pc) * 8));
    }
    const int spr = ntg / 16;
    for (int idx = t; idx < ncol * spr; idx += kThreads) {
        const int row = idx / spr, pc = idx % spr;
        const int s = 8 * (row >> 3);
        uint32_t w4[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            uint32_t wv = 0;
#pragma unroll
            for (int b = 0; b < 4; ++b)
                wv |= (uint32_t)lscales[row * kGrpTile + ((16 * pc + 4 * k + b) ^ s)] << (8 * b);
            w4[k] = wv;
        }
        __builtin_nontemporal_store(u32x4{w4[0], w4[1], w4[2], w4[3]},
                                    reinterpret_cast<u32x4*>(scales + (c0 + row) * ngroups + g0 + 16 * pc));
    }
}

// Round-to-nearest on both sides only (SR sides take the single-layout kernels).
template <int FMT>
static hipError_t launch_cols_dual_fmt(const DualK& k, dim3 grid, hipStream_t s)
{
    hipLaunchKernelGGL((quantize_cols_dual<FMT, false, false>), grid, dim3(kThreads), 0, s, k);
    return hipGetLastError();
}

template <int FMT>
static hipError_t launch_dual_fmt(const DualK& k, dim3 grid, bool sr_r, bool sr_c, hipStream_t s)
{
    if (sr_r && sr_c) hipLaunchKernelGGL((quantize_dual<FMT, true, true>), grid, dim3(kThreads), 0, s, k);
    else if (sr_r) hipLaunchKernelGGL((quantize_dual<FMT, true, false>), grid, dim3(kThreads), 0, s, k);
    else if (sr_c) hipLaunchKernelGGL((quantize_dual<FMT, false, true>), grid, dim3(kThreads), 0, s, k);
    else hipLaunchKernelGGL((quantize_dual<FMT, false, false>), grid, dim3(kThreads), 0, s, k);
    return hipGetLastError();
}

static void dual_side(const DualSide& d, float m, float a8, DualSideK& k)
{
    k.codes = d.codes;
    k.scales = d.scales;
    k.tensor_scale = d.tensor_scale;
    k.partials = d.partials;
    k.seed = d.seed;
    k.scale_max = (d.flags & IFQ_MARGIN_16_17) ? (float)((double)m * 16.0 / 17.0) : m;
    k.denom_alpha = k.scale_max * a8;
    k.qflags = ((d.flags & IFQ_SR_RTN_TYPE) ? kQSrRtnType : 0) | ((d.flags & IFQ_MARGIN_16_17) ? kQMargin : 0);
    k.rht = (d.flags & IFQ_RHT) ? 1 : 0;
    k.scale_in = (d.flags & IFQ_SCALE_IN) ? 1 : 0;
}

// 4-bit training formats only (the caller has checked the format).
hipError_t launch_quantize_dual(const DualArgs& a, hipStream_t s)
{
    float m = 0.0f, a8 = 0.0f;
    switch (a.fmt) {
        case IFQ_FMT_IF4: targets<IFQ_FMT_IF4>(m, a8); break;
        case IFQ_FMT_NVFP4: targets<IFQ_FMT_NVFP4>(m, a8); break;
        case IFQ_FMT_NVINT4: targets<IFQ_FMT_NVINT4>(m, a8); break;
        case IFQ_FMT_NVFP4_46: targets<IFQ_FMT_NVFP4_46>(m, a8); break;
        default: return hipErrorInvalidValue;
    }
    DualK k;
    k.x = a.x;
    k.rows = a.rows;
    k.cols = a.cols;
    k.ld = a.ld;
    k.vec = (reinterpret_cast<uintptr_t>(a.x) % 16 == 0 && a.ld % 8 == 0) ? 1 : 0;
    k.signs = a.signs;
    dual_side(a.row, m, a8, k.row);
    dual_side(a.col, m, a8, k.col);
    if (a.rows == 0 || a.cols == 0) {  // empty tensor: alpha = 0 on each side that computes it
        if (!k.row.scale_in) hipLaunchKernelGGL(write_scalar, dim3(1), dim3(1), 0, s, a.row.tensor_scale, 0.0f);
        if (!k.col.scale_in) hipLaunchKernelGGL(write_scalar, dim3(1), dim3(1), 0, s, a.col.tensor_scale, 0.0f);
        return hipGetLastError();
    }
    // register path: 16-byte aligned rows of X, 16 groups per output row
    // multiple (rows % 256 == 0), 16-byte aligned strided codes and scales
    const bool regs = k.vec && (a.rows / kGroup) % 16 == 0 && a.rows / kGroup / kGrpTile < 65536 &&
                      reinterpret_cast<uintptr_t>(a.col.codes) % 16 == 0 &&
                      reinterpret_cast<uintptr_t>(a.col.scales) % 16 == 0;
    if (regs) {
        k.npartials = 0;
        if (!(k.row.scale_in && k.col.scale_in)) {
            const int64_t bx = std::min<int64_t>(cdiv(a.cols, kColsPerBlock), kMaxPartials);
            const int64_t by = std::max<int64_t>(1, std::min<int64_t>(cdiv(a.rows / kGroup, 4), kMaxPartials / bx));
            k.npartials = (int)(bx * by);
            hipLaunchKernelGGL(tensor_max_cols_dual, dim3((unsigned)bx, (unsigned)by), dim3(kThreads), 0, s, k,
                               a.row.partials, a.col.partials);
            hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
        }
        const bool sr_r = a.row.flags & IFQ_SR, sr_c = a.col.flags & IFQ_SR;
        if (sr_r || sr_c) {
            // Stochastic rounding makes the quantize pass VALU-bound with
            // long dependent chains: one fused kernel (about 250 VGPRs, one
            // wavefront per SIMD) loses to the single-layout kernels, which
            // run at higher occupancy; reading X twice costs nothing there.
            // Both take their alpha from the fused maxima above.
            QuantArgs qr{a.fmt, a.x, a.rows, a.cols, a.ld, a.row.flags, a.signs, a.row.seed, a.row.codes,
                         a.row.scales, a.row.tensor_scale, a.row.partials};
            QuantArgs qc{a.fmt, a.x, a.rows, a.cols, a.ld, a.col.flags | IFQ_AXIS_STRIDED, a.signs, a.col.seed,
                         a.col.codes, a.col.scales, a.col.tensor_scale, a.col.partials};
            hipError_t e = hipSuccess;
            switch (a.fmt) {
                case IFQ_FMT_IF4:
                    e = dispatch_fmt<IFQ_FMT_IF4>(qr, s, k.npartials, k.row.scale_max, k.row.denom_alpha);
                    if (e == hipSuccess)
                        e = dispatch_fmt<IFQ_FMT_IF4>(qc, s, k.npartials, k.col.scale_max, k.col.denom_alpha);
                    break;
                case IFQ_FMT_NVFP4:
                    e = dispatch_fmt<IFQ_FMT_NVFP4>(qr, s, k.npartials, k.row.scale_max, k.row.denom_alpha);
                    if (e == hipSuccess)
                        e = dispatch_fmt<IFQ_FMT_NVFP4>(qc, s, k.npartials, k.col.scale_max, k.col.denom_alpha);
                    break;
                case IFQ_FMT_NVINT4:
                    e = dispatch_fmt<IFQ_FMT_NVINT4>(qr, s, k.npartials, k.row.scale_max, k.row.denom_alpha);
                    if (e == hipSuccess)
                        e = dispatch_fmt<IFQ_FMT_NVINT4>(qc, s, k.npartials, k.col.scale_max, k.col.denom_alpha);
                    break;
                default:
                    e = dispatch_fmt<IFQ_FMT_NVFP4_46>(qr, s, k.npartials, k.row.scale_max, k.row.denom_alpha);
                    if (e == hipSuccess)
                        e = dispatch_fmt<IFQ_FMT_NVFP4_46>(qc, s, k.npartials, k.col.scale_max, k.col.denom_alpha);
                    break;
            }
            return e;
        }
        const dim3 grid((unsigned)cdiv(a.cols, kColTile), (unsigned)cdiv(a.rows / kGroup, kGrpTile));
        switch (a.fmt) {
            case IFQ_FMT_IF4: return launch_cols_dual_fmt<IFQ_FMT_IF4>(k, grid, s);
            case IFQ_FMT_NVFP4: return launch_cols_dual_fmt<IFQ_FMT_NVFP4>(k, grid, s);
            case IFQ_FMT_NVINT4: return launch_cols_dual_fmt<IFQ_FMT_NVINT4>(k, grid, s);
            default: return launch_cols_dual_fmt<IFQ_FMT_NVFP4_46>(k, grid, s);
        }
    }
    const int64_t tx = cdiv(a.cols, kTC), ty = cdiv(a.rows, kTR);
    k.npartials = 0;
    if (!(k.row.scale_in && k.col.scale_in)) {
        const int64_t bx = std::min<int64_t>(tx, kMaxPartials);
        const int64_t by = std::max<int64_t>(1, std::min<int64_t>(ty, kMaxPartials / bx));
        k.npartials = (int)(bx * by);
        // both sides' maxima are written (a side with alpha supplied ignores its own)
        hipLaunchKernelGGL(tensor_max_dual, dim3((unsigned)bx, (unsigned)by), dim3(kThreads), 0, s, k,
                           a.row.partials, a.col.partials);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const dim3 grid((unsigned)tx, (unsigned)std::min<int64_t>(ty, 65535));
    const bool sr_r = a.row.flags & IFQ_SR, sr_c = a.col.flags & IFQ_SR;
    switch (a.fmt) {
        case IFQ_FMT_IF4: return launch_dual_fmt<IFQ_FMT_IF4>(k, grid, sr_r, sr_c, s);
        case IFQ_FMT_NVFP4: return launch_dual_fmt<IFQ_FMT_NVFP4>(k, grid, sr_r, sr_c, s);
        case IFQ_FMT_NVINT4: return launch_dual_fmt<IFQ_FMT_NVINT4>(k, grid, sr_r, sr_c, s);
        default: return launch_dual_fmt<IFQ_FMT_NVFP4_46>(k, grid, sr_r, sr_c, s);
    }
}

// Scratch of the allocation-free quantize entry point: room for the
// per-block maxima of the tensor-max pass.  Every GPU the library runs on
// holds its own copy until the process ends.  In host code the array's name
// is not a device address; the address is taken once per device, with that
// device current, from hipGetSymbolAddress and kept in scratch_ptr.
static __device__ __align__(256) float scratch[kMaxPartials];
static_assert(sizeof(scratch) == kScratchBytes, "scratch size");

namespace {
constexpr int kMaxScratchDevices = 64;
std::mutex scratch_mu;
float* scratch_ptr[kMaxScratchDevices];
}  // namespace

hipError_t scratch_partials(hipStream_t s, float** ptr)
{
    int dev = -1;
    hipError_t e = s ? hipStreamGetDevice(s, &dev) : hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxScratchDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(scratch_mu);
    if (!scratch_ptr[dev]) {
        int cur = -1;
        e = hipGetDevice(&cur);
        if (e != hipSuccess) return e;
        if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return e;
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (cur != dev) {
            const hipError_t e2 = hipSetDevice(cur);
            if (e == hipSuccess) e = e2;
        }
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        scratch_ptr[dev] = static_cast<float*>(p);
    }
    *ptr = scratch_ptr[dev];
    return hipSuccess;
}

}  // namespace ifq
