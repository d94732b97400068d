/*
 * ifq.h -- C ABI of the IF4 quantized-linear hot path on AMD Instinct
 * MI355X (gfx950): the adaptive block-scaled quantizer and the block-scaled
 * GEMM of "Adaptive Block-Scaled Data Types", with NVFP4, IF3, IF6, NVINT4
 * and NVFP4-with-4/6 variants for comparison.
 *
 * Format (Sec. 3).  A tensor X is stored as
 *   - one FP32 tensor scale  alpha = max|X| / (M_FP * 448)           (Eq. 1)
 *   - one byte per group of 16 values along the grouped axis K:
 *       bits 0-6  E4M3 magnitude of the group scale
 *                 Delta = max|X_g| / (alpha * M_FP) rounded to E4M3  (Eq. 2)
 *       bit 7     1 = the group holds scaled integers, 0 = FP elements
 *                 (the otherwise unused sign bit of the scale, Sec. 3)
 *   - 16 element codes per group, packed as a little-endian bit stream
 *     (code j at bits [j*b, j*b + b) of the group's 2b bytes).  For IF4 that
 *     puts element 2i in the low nibble of byte i.  FP codes are sign-
 *     magnitude ExMy; INT codes are two's complement in [-M_I, M_I].
 * A value decodes as  q * Delta * alpha  for FP groups and
 * q * Delta * (M_FP / M_I) * alpha  for INT groups (the 6/7 method, Sec. 3;
 * factors 4/3, 7.5/31 and 28/31 for IF3 and IF6 per the Sec. 5.1 footnote).
 *
 *   format      bits  FP element     M_FP   INT    M_I
 *   IF4         4     E2M1           6      INT4   7     (Sec. 3, Fig. 3a)
 *   NVFP4       4     E2M1           6      --     --    (FP only; bit 7 = 0)
 *   IF3         3     E2M0           4      INT3   3     (Sec. 5.1, Table 6)
 *   IF6_E2M3    6     E2M3           7.5    INT6   31    (Sec. 5.1, Table 6)
 *   IF6_E3M2    6     E3M2           28     INT6   31    (Sec. 5.1, Table 6)
 *   NVINT4      4     --             --     INT4   7     (INT only, Sec. 2)
 *   NVFP4_46    4     E2M1           6      --     --    (FP only, 4/6, Sec. 3)
 *   IF4_BS8, IF3_BS8, NVFP4_BS8: IF4, IF3 and NVFP4 with one scale per 8
 *                values instead of 16 (Sec. 5.1; Table 6 in App. D: 5.0, 4.0, 5.0 bits per
 *                parameter).  Scales are [R, K/8]; the two scale bytes of
 *                values 16i .. 16i+15 are adjacent, and their codes fill the
 *                same 2b bytes as one block-16 group.  SR draws of group g
 *                (its scale byte index) are the first 8 of counter g.
 *
 * NVINT4 groups are scaled straight to M_I = 7 (Delta = max|X_g| / (alpha * 7),
 * alpha = max|X| / (7 * 448), Table 1), decode as q * Delta * alpha, and keep
 * bit 7 of the scale clear.  NVFP4_46 (Four Over Six) computes alpha =
 * max|X| / (6 * 256) (Table 1), scales each group both to a maximum of 6 and
 * to a maximum of 4, rounds onto E2M1 each time and keeps the scaling whose
 * dequantized group has the smaller squared error (ties keep 6); the stored
 * data then decode exactly like NVFP4.
 *
 * Layouts (row-major, no padding):
 *   codes   uint8 [R, K * bits / 8]      scales  uint8 [R, K / G]
 * with G = 16 values per scale byte (8 for the *_BS8 formats)
 * where R is the number of logical rows and K (a multiple of 16) is the
 * grouped axis.
 *
 * Conventions for every call:
 *   - Pointers marked (device) are HIP device pointers; the caller allocates
 *     and owns all memory; the library keeps no state and allocates nothing.
 *   - `stream` is a hipStream_t (NULL = the legacy default stream).  All
 *     work is enqueued asynchronously on it; no call synchronises.
 *   - Arguments are validated on the host before anything is enqueued; a
 *     negative return value means nothing was launched.  IFQ_EHIP means a
 *     launch was rejected by the runtime (outputs are then undefined).
 *     Faults inside kernels surface at the caller's next synchronisation.
 *   - Inputs must be finite.
 *   - Calls are thread-safe; concurrent calls must not share outputs or a
 *     workspace.
 */
#ifndef IFQ_H
#define IFQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define IFQ_ABI_VERSION 2

typedef enum ifq_status {
    IFQ_OK = 0,
    IFQ_EINVAL = -1,        /* null pointer, unknown flag, format or dtype */
    IFQ_ESHAPE = -2,        /* negative size, K not a multiple of 16, ld too small, too large */
    IFQ_EALIGN = -3,        /* a pointer or leading dimension breaks the alignment rules */
    IFQ_EUNSUPPORTED = -4,  /* valid but not implemented combination */
    IFQ_EHIP = -5,          /* the HIP runtime rejected a launch */
    IFQ_EWORKSPACE = -6     /* workspace missing or smaller than required */
} ifq_status;

typedef enum ifq_format {
    IFQ_FMT_IF4 = 0,
    IFQ_FMT_NVFP4 = 1,
    IFQ_FMT_IF3 = 2,
    IFQ_FMT_IF6_E2M3 = 3,
    IFQ_FMT_IF6_E3M2 = 4,
    IFQ_FMT_NVINT4 = 5,
    IFQ_FMT_NVFP4_46 = 6,
    IFQ_FMT_IF4_BS8 = 7,
    IFQ_FMT_IF3_BS8 = 8,
    IFQ_FMT_NVFP4_BS8 = 9
} ifq_format;

typedef enum ifq_dtype { IFQ_F32 = 0, IFQ_BF16 = 1 } ifq_dtype;

/* quantizer flags */
enum {
    IFQ_RHT = 1u,          /* 16-point random Hadamard transform of each group first */
    IFQ_SR = 2u,           /* stochastic rounding of both candidates */
    IFQ_MARGIN_16_17 = 4u, /* scales computed against M * 16/17 (Sec. 4.1); for
                              NVFP4_46 both targets, 6 and 4, take the factor */
    IFQ_SCALE_IN = 8u,     /* *tensor_scale is an input instead of Eq. 1's output */
    IFQ_AXIS_STRIDED = 16u, /* groups run along rows; output describes X transposed */
    IFQ_SR_RTN_TYPE = 32u   /* with IFQ_SR: decide FP or INT (for NVFP4_46: the
                               scaling to 6 or 4) on the round-to-nearest
                               candidates, then round stochastically in that type
                               (the unbiased alternative of App. B); no effect
                               without IFQ_SR or for NVFP4 and NVINT4 */
};

/* ------------------------------------------------------------ quantize --
 * Quantize a bf16 matrix X (rows x cols, row stride ld_x elements).
 * Follows Eq. 1 and 2 and Fig. 3a of the paper: alpha from the tensor
 * maximum, Delta per group rounded to E4M3, then for IF formats both an FP
 * and a scaled-INT candidate with the INT one kept only if its squared
 * error is strictly smaller (Fig. 3a (selection)).
 *
 *   x             (device) bf16 [rows, ld_x], ld_x >= cols; row-wise: 16-byte
 *                 aligned with ld_x % 8 == 0; strided axis: any alignment
 *   flags         IFQ_* bits above.  IFQ_RHT applies v = (1/4) H16 diag(s) x
 *                 to every group (Sylvester order H16[i][j] =
 *                 (-1)^popcount(i&j), s_j = -1 where bit j of rht_signs is
 *                 set); the tensor scale is then taken over the transformed
 *                 values.  IFQ_SR draws 16 uniform 16-bit numbers per group
 *                 from Philox4x32-10 (key = seed, counter = (group index lo,
 *                 group index hi, block 0/1, 0), group index = position of
 *                 its scale byte) and shares draw j between the two
 *                 candidates of element j.
 *   rht_signs     16-bit sign mask (upper bits must be zero)
 *   seed          Philox key for IFQ_SR
 *   codes         (device) uint8 [R, K*bits/8], 16-byte aligned
 *   scales        (device) uint8 [R, K/G] (G = ifq_group_size(format))
 *                 Row-wise: R = rows, K = cols (cols % 16 == 0).
 *                 IFQ_AXIS_STRIDED: R = cols, K = rows (rows % 16 == 0): the
 *                 output is the packed form of X^T, K-major as the GEMM
 *                 expects (e.g. dY^T and X^T of a weight gradient).
 *   tensor_scale  (device) one float: written with alpha, or read when
 *                 IFQ_SCALE_IN is set.  A group whose alpha * Delta is zero or
 *                 below FLT_MIN (this includes alpha = 0 and an all-zero
 *                 tensor) is stored as scale 0 and codes 0; for NVFP4_46 that
 *                 is decided on the scaling to 4 (the larger Delta), and a
 *                 scaling to 6 below FLT_MIN leaves the scaling to 4.
 *   workspace     (device) at least ifq_quantize_workspace_bytes() bytes,
 *                 256-byte aligned, no initial contents required; may be
 *                 NULL when that size is 0.
 */
int if4_quantize(const void* x, int64_t rows, int64_t cols, int64_t ld_x, uint32_t flags,
                 uint32_t rht_signs, uint64_t seed, uint8_t* codes, uint8_t* scales,
                 float* tensor_scale, void* workspace, size_t workspace_bytes, void* stream);

/* NVFP4 (Fig. 3a up to the FP candidate): same arguments, bit 7 of every scale is 0. */
int nvfp4_quantize(const void* x, int64_t rows, int64_t cols, int64_t ld_x, uint32_t flags,
                   uint32_t rht_signs, uint64_t seed, uint8_t* codes, uint8_t* scales,
                   float* tensor_scale, void* workspace, size_t workspace_bytes, void* stream);

/* Any format (IF3 and IF6 of Sec. 5.1, NVINT4, NVFP4_46 and the block-size-8
 * formats included); same arguments, scales [R, K / ifq_group_size()]. */
int ifx_quantize(int format, const void* x, int64_t rows, int64_t cols, int64_t ld_x,
                 uint32_t flags, uint32_t rht_signs, uint64_t seed, uint8_t* codes,
                 uint8_t* scales, float* tensor_scale, void* workspace, size_t workspace_bytes,
                 void* stream);

/* ifx_quantize without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  Same arguments, checks and results as
 * ifx_quantize, bit for bit.  The per-block maxima of the tensor-max pass go
 * to a 1 KiB scratch array inside the library, one per GPU, held until the
 * process ends; its address is looked up once per device (the device of
 * `stream`, or the current device for the null stream).  The scratch holds
 * at most 256 partial maxima whatever the tensor size, so no size is
 * rejected for it; a requirement above its 1 KiB (none today) would return
 * IFQ_EWORKSPACE.  Nothing in it needs to start at zero: each call writes
 * every entry it reads.  Calls on one GPU share the scratch: calls that can
 * overlap in time on one GPU (different streams without ordering) race and
 * must not be made.  Allocates nothing (no hipMalloc, no library allocation).
 */
int ifx_quantize_noalloc(int format, const void* x, int64_t rows, int64_t cols, int64_t ld_x,
                         uint32_t flags, uint32_t rht_signs, uint64_t seed, uint8_t* codes,
                         uint8_t* scales, float* tensor_scale, void* stream);

/* Bytes of device workspace the quantizer needs (0 with IFQ_SCALE_IN). */
size_t ifq_quantize_workspace_bytes(int format, int64_t rows, int64_t cols, uint32_t flags);

/* ------------------------------------------------------- dual quantize --
 * Both packed layouts of one bf16 matrix X: the row-wise form (groups along
 * cols: codes [rows, cols*b/8], scales [rows, cols/16]) and the strided form
 * (groups along rows, describing X^T: codes [cols, rows*b/8], scales
 * [cols, rows/16]).  One pass reads X once for both tensor maxima; the
 * quantize pass reads it once more for both layouts when neither side uses
 * IFQ_SR, and once per layout otherwise (stochastic rounding makes that pass
 * arithmetic-bound, where separate kernels are faster).  A linear layer's
 * training step needs X, W and dY both ways (Sec. 4.1: the forward GEMM, the
 * activation gradient dX = dY W and the weight gradient dW = dY^T X contract
 * over different axes); the results are bit-identical to
 *   ifx_quantize(format, x, ..., row_flags, rht_signs, row_seed, row_*) and
 *   ifx_quantize(format, x, ..., col_flags | IFQ_AXIS_STRIDED, rht_signs,
 *                col_seed, col_*).
 *   format        IFQ_FMT_IF4, IFQ_FMT_NVFP4, IFQ_FMT_NVINT4 or
 *                 IFQ_FMT_NVFP4_46 (others: IFQ_EUNSUPPORTED)
 *   x             (device) bf16 [rows, ld_x], ld_x >= cols, 2-byte aligned;
 *                 rows % 16 == 0 and cols % 16 == 0
 *   row_flags, col_flags  IFQ_RHT, IFQ_SR, IFQ_MARGIN_16_17, IFQ_SCALE_IN,
 *                 IFQ_SR_RTN_TYPE per side (IFQ_AXIS_STRIDED is rejected);
 *                 each side has its own alpha (its RHT changes the values)
 *   rht_signs     16-bit sign mask shared by both sides
 *   row_seed, col_seed  Philox keys of the two sides (IFQ_SR)
 *   row_codes, col_codes  (device) 16-byte aligned; row_scales, col_scales
 *   row_tensor_scale, col_tensor_scale  (device) written, or read with
 *                 IFQ_SCALE_IN on that side
 *   workspace     (device) ifq_quantize_dual_workspace_bytes() bytes, 16-byte
 *                 aligned (0 when both sides have IFQ_SCALE_IN)
 */
int ifx_quantize_dual(int format, const void* x, int64_t rows, int64_t cols, int64_t ld_x,
                      uint32_t row_flags, uint32_t col_flags, uint32_t rht_signs, uint64_t row_seed,
                      uint64_t col_seed, uint8_t* row_codes, uint8_t* row_scales, float* row_tensor_scale,
                      uint8_t* col_codes, uint8_t* col_scales, float* col_tensor_scale, void* workspace,
                      size_t workspace_bytes, void* stream);

size_t ifq_quantize_dual_workspace_bytes(int format, int64_t rows, int64_t cols, uint32_t row_flags,
                                         uint32_t col_flags);

/* ---------------------------------------------------------- dequantize --
 * out[r, k] = q * Delta * (M_FP/M_I if INT) * alpha (the factor is 1 for
 * NVINT4), evaluated as three fp32 multiplies in that order (the dequantized values of Fig. 3a with alpha restored); the
 * bf16 output is the round-to-nearest-even of that fp32 value.
 *   codes, scales  (device) packed [R, K] as written by the quantizer
 *   tensor_scale   (device) alpha
 *   out            (device) [rows, cols] contiguous, fp32 or bf16 (out_dtype),
 *                  16-byte aligned
 */
int if4_dequantize(const uint8_t* codes, const uint8_t* scales, const float* tensor_scale,
                   int64_t rows, int64_t cols, void* out, int out_dtype, void* stream);
int nvfp4_dequantize(const uint8_t* codes, const uint8_t* scales, const float* tensor_scale,
                     int64_t rows, int64_t cols, void* out, int out_dtype, void* stream);
int ifx_dequantize(int format, const uint8_t* codes, const uint8_t* scales,
                   const float* tensor_scale, int64_t rows, int64_t cols, void* out,
                   int out_dtype, void* stream);

/* ---------------------------------------------------------------- GEMM --
 * C[m, n] = sum_k A[m, k] * B[n, k] over the dequantized values of two
 * packed operands that share the grouped axis K ("TN": Y = X W^T, or
 * dW = dY^T X with both operands quantized along the token axis).  This is
 * the block-scaled dot product of Sec. 5.2: per 16-wide K block the product
 * of the two group scales, times 1, 6/7 or 36/49 by the two group types,
 * accumulated in FP32.  Here each element is decoded to an FP16 MFMA operand
 * that carries its group scale exactly (7 q Delta for FP groups, 6 q Delta
 * for INT groups), so one FP32 accumulation over all of K applies every
 * block's scale pair and range alignment; alpha_A * alpha_B / 49 is applied
 * once at the end.  NVFP4, NVFP4_46, NVINT4 (q Delta / 4) and IF3 operands
 * are exact the same way; IF6
 * operands (62 q Delta and 15 q Delta for E2M3, 31 q Delta and 28 q Delta
 * for E3M2, Sec. 5.1 ratios) need up to 13 significant bits and are rounded
 * once to FP16 (relative error at most 2^-12 per operand).
 *   a_codes, a_scales  (device) A packed [M, K]; b_* : B packed [N, K]
 *   a_tensor_scale, b_tensor_scale  (device) alpha of A and of B
 *   c                  (device) [M, ldc] fp32 or bf16 (out_dtype); ldc >= N
 *   code pointers 16-byte aligned; K % 16 == 0.
 * fp32 output with K % 1024 == 0, c 16-byte aligned and ldc % 4 == 0: when
 * the last round of 256 x 256 tiles would leave at least half of the
 * device's compute units idle, those tiles are computed as two K halves
 * whose shares are added by atomics into their output, zeroed first in the
 * same stream.  A sum of two terms into zero does not depend on their order,
 * so the result is deterministic for a given shape and device (it differs
 * from the whole-K accumulation by one rounding); other work must not touch
 * c while the call runs.
 */
int if4_gemm(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_tensor_scale,
             const uint8_t* b_codes, const uint8_t* b_scales, const float* b_tensor_scale,
             int64_t M, int64_t N, int64_t K, void* c, int64_t ldc, int out_dtype, void* stream);
int nvfp4_gemm(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_tensor_scale,
               const uint8_t* b_codes, const uint8_t* b_scales, const float* b_tensor_scale,
               int64_t M, int64_t N, int64_t K, void* c, int64_t ldc, int out_dtype,
               void* stream);
int ifx_gemm(int format, const uint8_t* a_codes, const uint8_t* a_scales,
             const float* a_tensor_scale, const uint8_t* b_codes, const uint8_t* b_scales,
             const float* b_tensor_scale, int64_t M, int64_t N, int64_t K, void* c,
             int64_t ldc, int out_dtype, void* stream);

/* ---------------------------------------------------------- host helpers */
/* Buffer sizes of a packed [rows, cols] tensor (cols = the grouped axis K);
 * 0 for an unknown format or a negative size. */
size_t ifq_codes_bytes(int format, int64_t rows, int64_t cols);  /* rows * cols * bits / 8 */
size_t ifq_scales_bytes(int format, int64_t rows, int64_t cols); /* rows * (cols / group size) */
int ifq_group_size(int format);  /* values per scale byte: 16, or 8 for the *_BS8 formats;
                                    0 for an unknown format */
const char* ifq_status_string(int status);
int ifq_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* IFQ_H */
