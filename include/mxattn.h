/*
 * mxattn.h -- C ABI of libmxattn: MXFP4 attention forward for MI355X (gfx950).
 *
 * The library implements the hot path of "MXAttention: Data-Free Optimal
 * Scaling and Pre-Normalization Quantization for MXFP4 Attention":
 *
 *   1. an MXFP4 quantizer (32-element E2M1 blocks sharing one E8M0
 *      power-of-two scale) with either the OCP floor scale rule
 *      e = floor(log2 M) - 2 (Sec. 2, Eq. ocp_scale) or the Universal Optimal
 *      Scaling rule e = ceil(log2(M / 7.25)) (Sec. 4.1, Algorithm 1);
 *   2. a fused flash-style attention forward on MXFP4 Q, K, V: S = Q^K^T on
 *      block-scaled FP4 matrix cores, online softmax, in-register MXFP4
 *      quantization of the unnormalized exponential tile, and O~ += P^V^ on
 *      FP4 matrix cores (Algorithm 2 without its Hadamard rotation).
 *
 * Everything is asynchronous on the caller's HIP stream.  All tensor
 * pointers are device pointers owned by the caller; the library never frees
 * or retains them.  Arguments are validated before anything is launched; on
 * an error nothing is launched and a nonzero status is returned.  The library
 * never aborts, prints or throws.  Inputs must be finite (not checked).
 *
 * Layouts (row-major, bf16 = IEEE binary32 truncated to its top 16 bits):
 *   Q, K, V, O        bf16 [B, H, N, d], d = 128.
 *   head-dim blocks   (block_axis = 3, used for Q and K): 32 consecutive
 *                     channels of one token.
 *                     codes  uint8 [B, H, N, d/2]   element 2i in the low
 *                                                   nibble of byte i
 *                     scales uint8 [B, H, N, d/32]  E8M0 (bias 127)
 *   token blocks      (block_axis = 2, used for V): 32 consecutive tokens of
 *                     one channel; the last block of a row is padded with +0.
 *                     codes  uint8 [B, H, d, nb*16] nb = ceil(N/32), tokens
 *                                                   contiguous per channel
 *                     scales uint8 [B, H, d, nb]
 *   A 4-bit code is sign(1) | magnitude index(3) into the E2M1 grid
 *   {0, 0.5, 1, 1.5, 2, 3, 4, 6} (Sec. 2, "MXFP4 Block Quantization").
 *
 * Rounding of the quantizer (readings of the paper, which says only "round
 * to nearest with saturation at +-6"): ties go to the even code, magnitudes
 * above 6 saturate to 6, the code keeps the input's sign bit even for a zero
 * magnitude, the E8M0 exponent is clamped to [-127, 127], and an all-zero
 * block gets scale byte 127 (sigma = 1, as Algorithm 1 states).
 */
#ifndef MXATTN_H
#define MXATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Scale rule, row-sum placement and rotation (rows of the paper's
 * sequential ablation, Sec. 5.4):
 *   MXATTN_OCP_VANILLA  OCP floor rule for Q, K, V and P~; direct placement:
 *                       l accumulates the unquantized P~ (Eq.
 *                       direct_mxfp4_tile, Sec. 4.2).
 *   MXATTN_UOS          UOS rule (Algorithm 1) everywhere; direct placement.
 *   MXATTN_UOS_PNQ      UOS rule everywhere; Pre-Normalization Quantization:
 *                       l accumulates the quantized P^ that also feeds the PV
 *                       product (Eqs. pnq_tile_contribution and
 *                       pnq_online_update; Algorithm 2).
 *   MXATTN_UOS_PNQ_ROT  as MXATTN_UOS_PNQ, and Q and K are multiplied by the
 *                       fixed Hadamard rotation R_H = H/sqrt(128) before
 *                       quantization (Sec. 4.3; Algorithm 2, its first two
 *                       steps): Sylvester ordering, formed in fp32 by the
 *                       radix-2 fast Walsh-Hadamard transform (stages
 *                       h = 1, 2, ..., 64, pairs (a, b) -> (a + b, a - b)),
 *                       then one fp32 multiply by fp32(1/sqrt(128)); the
 *                       fp32 result is quantized directly.  V is not
 *                       rotated.  Since (Q R_H)(K R_H)^T = Q K^T, the
 *                       attention the operands represent is unchanged. */
typedef enum {
    MXATTN_OCP_VANILLA = 0,
    MXATTN_UOS = 1,
    MXATTN_UOS_PNQ = 2,
    MXATTN_UOS_PNQ_ROT = 3
} mxattn_mode;

typedef enum {
    MXATTN_OK = 0,
    MXATTN_ERR_NULL = 1,        /* a required pointer is NULL              */
    MXATTN_ERR_SHAPE = 2,       /* B, H or N < 1, beyond a size limit, or an
                                   output that overlaps an input            */
    MXATTN_ERR_ALIGN = 3,       /* a pointer is not 16-byte aligned         */
    MXATTN_ERR_MODE = 4,        /* mode is not an mxattn_mode value         */
    MXATTN_ERR_AXIS = 5,        /* block_axis is not 2 or 3                 */
    MXATTN_ERR_UNSUPPORTED = 6, /* d != 128                                 */
    MXATTN_ERR_OOM = 7,         /* workspace allocation failed              */
    MXATTN_ERR_HIP = 8,         /* a HIP call failed; see mxattn_last_error */
    MXATTN_ERR_BOUNDARY = 9,    /* a scale boundary q outside [4, 8], a
                                   boundary count outside [1, 64], or a
                                   pre-scale gamma not in (0, 3e38)         */
    MXATTN_ERR_SCRATCH = 10     /* the problem needs more than the static
                                   scratch of mxattn_cross_attend_noalloc   */
} mxattn_status;

#define MXATTN_AXIS_TOKENS 2   /* blocks along N (V)      */
#define MXATTN_AXIS_HEAD_DIM 3 /* blocks along d (Q and K) */
#define MXATTN_MAX_BOUNDARIES 64 /* boundaries per mxattn_qmax_sse call */

/* MXFP4-quantize a bf16 tensor x [B, H, N, d] (Algorithm 1 with the scale
 * rule of `mode`: OCP floor for MXATTN_OCP_VANILLA, UOS otherwise).  With
 * MXATTN_UOS_PNQ_ROT and block_axis MXATTN_AXIS_HEAD_DIM the rows are first
 * rotated by R_H (Q and K of that mode); along MXATTN_AXIS_TOKENS that mode
 * quantizes like MXATTN_UOS_PNQ.
 *   x       device, bf16 [B, H, N, d], 16-byte aligned
 *   codes   device, layout of `block_axis` above, 16-byte aligned,
 *           mxattn_codes_bytes() bytes
 *   scales  device, layout of `block_axis` above, mxattn_scales_bytes() bytes
 *   stream  hipStream_t to run on (NULL: the null stream)
 * Returns MXATTN_OK or an error status; nothing is launched on error. */
int mxattn_quantize(const void* x, uint8_t* codes, uint8_t* scales, int block_axis, int mode,
                    int64_t B, int64_t H, int64_t N, int64_t d, void* stream);

/* MXFP4-quantize with the ceil scale rule of a general boundary q: each
 * block takes the smallest exponent e with M <= q 2^e (Eq. scale_definition,
 * Eq. uos_mapping), clamped to [-127, 127].  q = 6 is TFS, q = 7 the OAS rule
 * at 32-element blocks (App. "Relation to OAS and the OCP Endpoint
 * Convention"), q = 7.25 UOS (identical to mxattn_quantize in a UOS mode) and
 * q = 8 the ceil form of the OCP boundary (which differs from the floor rule
 * of MXATTN_OCP_VANILLA only where M is a power of two).  Layouts, rounding
 * and alignment as mxattn_quantize; no rotation.
 *   qmax    the boundary q, 4 <= q <= 8 (MXATTN_ERR_BOUNDARY otherwise)
 * Returns MXATTN_OK or an error status; nothing is launched on error. */
int mxattn_quantize_qmax(const void* x, uint8_t* codes, uint8_t* scales, int block_axis, double qmax,
                         int64_t B, int64_t H, int64_t N, int64_t d, void* stream);

/* Per-(batch, head) sum of squared MXFP4 quantization errors
 * sum_i (x_i - Q_q(x_i))^2 of x [B, H, N, d], blocked along block_axis, for
 * each boundary qs[j] of the ceil rule above: the per-tensor MSE sweep of
 * the paper's empirical check of the boundary (Sec. 5.5, Table
 * cx_distribution, which sweeps q from 6.00 to 8.00 in steps of 0.05).
 * Token blocks count their +0 padding, which adds no error.
 *   x       device bf16 [B, H, N, d], 16-byte aligned, finite
 *   qs      HOST array of nq boundaries, each 4 <= q <= 8, read before the
 *           call returns; 1 <= nq <= MXATTN_MAX_BOUNDARIES
 *   sse     device fp64 [B*H, nq], 8-byte aligned, written in full
 * Sums are formed in fp64 (each element's squared error exactly); the order
 * of additions within a workgroup is not fixed, so repeated calls may differ
 * in the last bits.  Uses stream-ordered workspace (the library's pool,
 * see mxattn_release_workspace): 2056 bytes per workgroup, about 2048 workgroups or one per
 * (batch, head) if there are more, so about 2 KiB * max(B*H, 2048).
 * Returns MXATTN_OK, MXATTN_ERR_OOM, or another error status. */
int mxattn_qmax_sse(const void* x, int block_axis, const double* qs, int nq, double* sse, int64_t B,
                    int64_t H, int64_t N, int64_t d, void* stream);

/* Row-sum diagnostics of MXFP4-quantized attention probabilities (Sec. 5.5,
 * "Validation of Pre-Normalization Quantization", Fig. pnq_rowsum): what
 * direct block quantization of a materialized, normalized P does to the mass
 * of each row, which PNQ avoids.  Per row, stats holds 8 fp64 values
 *   [0] sum_j Q(x_j) / gamma        the row sum after quantization
 *   [1] sum_j p_j                    the row sum before
 *   [2] zeroing     sum of Q(x_j)/gamma - p_j over p_j > 0 with Q(x_j) = 0
 *   [3] saturation  ... over x_j / sigma > 6 (above the largest E2M1 value)
 *   [4] down        ... over the other entries with Q(x_j) < x_j
 *   [5] up          ... over Q(x_j) > x_j
 *   [6] exact       ... over Q(x_j) = x_j
 *   [7] entropy     -sum_{p_j > 0} p_j ln p_j (nats)
 * with x_j = fp32(gamma * p_j) quantized in blocks of 32 consecutive entries
 * of the row (the last block padded with +0) by the scale rule of `mode`
 * (OCP floor for MXATTN_OCP_VANILLA, UOS otherwise), and 1/gamma rounded to
 * fp64.  gamma is the single "pre-quant global scaling" factor of
 * Fig. pnq_rowsum (C); gamma = 1 quantizes P as it is.  [0] - [1] equals
 * [2] + ... + [6] up to rounding.  Sums are fp64 (each term exact but the
 * entropy's, which uses the fp32 base-2 logarithm); workgroup reductions run
 * in a fixed order.
 *
 * mxattn_softmax_rows materializes p = softmax(q k^T / sqrt(d)) for the query
 * rows [row0, row0 + rows) of every (batch, head): S on the bf16 matrix cores
 * with fp32 accumulation, p = 2^(s log2(e)/sqrt(d) - m) / L in fp32 (entries
 * below 2^-126 flush to 0).
 *   q       device bf16 [B, H, Nq, d]; k device bf16 [B, H, Nkv, d]
 *   p       device fp32 [B, H, rows, ld], ld >= Nkv, ld % 4 == 0; entries
 *           past Nkv up to the next multiple of 4 are set to 0, the rest of
 *           [Nkv, ld) is not written
 * mxattn_rowsum_diag quantizes given rows:
 *   p       device fp32 [rows, ld], entries >= 0 (first N of each row used),
 *           ld >= N, ld % 4 == 0, 16-byte aligned
 *   stats   device fp64 [rows, 8]
 * mxattn_attention_rowsum_diag computes the same statistics for every query
 * row of q against k without materializing P: the probabilities are formed
 * exactly as mxattn_softmax_rows forms them and quantized in registers, so
 * the result equals mxattn_rowsum_diag applied to mxattn_softmax_rows up to
 * the order of the fp64 additions.  No workspace.
 *   stats   device fp64 [B, H, Nq, 8]
 * All three return MXATTN_OK or an error status; nothing is launched on
 * error. */
int mxattn_softmax_rows(const void* q, const void* k, float* p, int64_t B, int64_t H, int64_t Nq,
                        int64_t Nkv, int64_t d, int64_t row0, int64_t rows, int64_t ld, void* stream);
int mxattn_rowsum_diag(const float* p, int64_t rows, int64_t N, int64_t ld, int mode, float gamma,
                       double* stats, void* stream);
int mxattn_attention_rowsum_diag(const void* q, const void* k, int64_t B, int64_t H, int64_t Nq,
                                 int64_t Nkv, int64_t d, int mode, float gamma, double* stats,
                                 void* stream);

/* MXFP4 attention forward O = softmax(Q K^T / sqrt(d)) V with MXFP4 Q, K, V
 * and MXFP4 P~ (Algorithm 2, with its Hadamard rotation in mode
 * MXATTN_UOS_PNQ_ROT only; non-causal, no mask besides the sequence end).
 * Quantizes K along d and V along N into stream-ordered workspace (from
 * the library's pool on `stream`, see mxattn_release_workspace; about 0.53
 * bytes per element of each of K and V), then runs the fused kernel, which quantizes Q along d in
 * its prologue with codes bit-identical to mxattn_quantize's; in
 * MXATTN_UOS_PNQ_ROT, Q is rotated and quantized into the workspace first
 * (0.53 bytes per element more).
 *   q, k, v  device bf16 [B, H, N, d], 16-byte aligned
 *   out      device bf16 [B, H, N, d], 16-byte aligned; MXATTN_ERR_SHAPE if
 *            it shares a byte with q, k or v
 * Size limits (MXATTN_ERR_SHAPE otherwise): N <= 2^24 keys (the kernel
 * addresses one head's quantized K and V with 32-bit byte offsets) and
 * B * H * ceil(N / 128) <= 2^30 query tiles.
 * Returns MXATTN_OK, MXATTN_ERR_OOM if the workspace cannot be allocated, or
 * another error status; nothing is launched on an argument error. */
int mxattn_forward(const void* q, const void* k, const void* v, void* out, int64_t B, int64_t H,
                   int64_t N, int64_t d, int mode, void* stream);

/* The fused attention kernel alone, on already quantized operands (the
 * layouts above: Q and K blocked along d, V blocked along N).  The scale rule
 * of `mode` applies to the in-kernel quantization of P~; `mode` also selects
 * direct or PNQ placement.  All pointers are device pointers; code arrays
 * and `out` are 16-byte aligned, k_scales 4-byte aligned, the other scale
 * arrays may have any alignment.  MXATTN_ERR_SHAPE if `out` shares a byte
 * with any code or scale array. */
int mxattn_attend(const uint8_t* q_codes, const uint8_t* q_scales, const uint8_t* k_codes,
                  const uint8_t* k_scales, const uint8_t* v_codes, const uint8_t* v_scales,
                  void* out, int64_t B, int64_t H, int64_t N, int64_t d, int mode, void* stream);

/* Attention with different query and key/value lengths (cross-attention:
 * video queries attending to a short text sequence; the paper's Wan2.2 has
 * separate cross-attention modules, Sec. 5.1).  q and out are [B, H, Nq, d],
 * k and v are [B, H, Nkv, d]; the quantized variants take Q^ blocked along d
 * with Nq rows, K^ blocked along d with Nkv rows and V^ blocked along Nkv.
 * Otherwise as mxattn_forward / mxattn_attend, which are these calls with
 * Nq = Nkv = N; the key limit N <= 2^24 applies to Nkv. */
int mxattn_cross_forward(const void* q, const void* k, const void* v, void* out, int64_t B,
                         int64_t H, int64_t Nq, int64_t Nkv, int64_t d, int mode, void* stream);
int mxattn_cross_attend(const uint8_t* q_codes, const uint8_t* q_scales, const uint8_t* k_codes,
                        const uint8_t* k_scales, const uint8_t* v_codes, const uint8_t* v_scales,
                        void* out, int64_t B, int64_t H, int64_t Nq, int64_t Nkv, int64_t d, int mode,
                        void* stream);

/* mxattn_cross_attend without any allocation, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * and harnesses that forbid allocation.  Same arguments, checks and result
 * as mxattn_cross_attend (bit-identical output, the same kernels); it calls
 * no hipMalloc, hipMallocAsync, hipFree or any allocating routine.  Its one
 * buffer beyond the inputs and `out`, the K^ and V^ scales rearranged into
 * the kernel's operand order (1 KiB per (batch, head) and 128-key tile), is
 * a static device array of MXATTN_NOALLOC_SCRATCH_BYTES that each device the
 * library runs on holds until the process ends.  Limit: B * H * ceil(Nkv /
 * 128) <= 32768 (e.g. H = 40 heads of up to 104 832 keys), else
 * MXATTN_ERR_SCRATCH with a message in mxattn_last_error and nothing
 * launched.  The array is fully rewritten by every call before it is read,
 * but all calls on one device share it: calls that overlap in time on one
 * device (different streams without ordering between them) race and give
 * undefined results.  The first call on a device looks up the array's
 * device address (hipGetSymbolAddress); MXATTN_ERR_HIP if that fails. */
#define MXATTN_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
int mxattn_cross_attend_noalloc(const uint8_t* q_codes, const uint8_t* q_scales, const uint8_t* k_codes,
                                const uint8_t* k_scales, const uint8_t* v_codes, const uint8_t* v_scales,
                                void* out, int64_t B, int64_t H, int64_t Nq, int64_t Nkv, int64_t d,
                                int mode, void* stream);

/* Sizes of the code and scale arrays of a [B, H, N, d] tensor blocked along
 * `block_axis`; 0 for invalid arguments. */
size_t mxattn_codes_bytes(int block_axis, int64_t B, int64_t H, int64_t N, int64_t d);
size_t mxattn_scales_bytes(int block_axis, int64_t B, int64_t H, int64_t N, int64_t d);

/* KV tile width B_c of the fused kernel: the running maximum is updated once
 * per B_c keys, in increasing key order (this fixes which exponentials are
 * quantized together; see Sec. 2, Eq. online_attention). */
int mxattn_kv_tile(void);

/* Query rows handled by one workgroup of the fused kernel. */
int mxattn_query_tile(void);

/* Static description of a status code. */
const char* mxattn_status_string(int status);

/* Detail of the last MXATTN_ERR_HIP or MXATTN_ERR_OOM on the calling
 * thread ("" if none). */
const char* mxattn_last_error(void);

/* Workspace.  mxattn_forward, mxattn_cross_forward, mxattn_attend,
 * mxattn_cross_attend and mxattn_qmax_sse take their workspace, stream-
 * ordered, from a memory pool that belongs to the library (one per device,
 * created on first use; the device's default pool is left as it is).  The
 * pool keeps freed workspace for the next call rather than returning it to
 * the driver.  mxattn_release_workspace returns all of the current device's
 * cached workspace that no call still uses; call it after the streams that
 * ran the library's calls have completed, e.g. before a phase of a pipeline
 * that needs the memory.  Returns MXATTN_OK or MXATTN_ERR_HIP. */
int mxattn_release_workspace(void);

/* ABI version (major * 100 + minor). */
int mxattn_version(void);

#ifdef __cplusplus
}
#endif

#endif /* MXATTN_H */
