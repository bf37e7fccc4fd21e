/*
 * mxref.c -- CPU oracle for the MXFP4 attention hot path of "MXAttention:
 * Data-Free Optimal Scaling and Pre-Normalization Quantization for MXFP4
 * Attention".
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path links, loads or
 * calls this file; only the tests, the smoke check and the CPU-baseline leg
 * of the benchmark do.  It shares no code, header, table or constant with
 * the HIP library: every grid value, rule and constant below is restated
 * here from the paper.
 *
 * It is deliberately plain and slow: brute-force argmin over the E2M1 grid,
 * scale exponents found by search instead of by logarithms, and the online
 * softmax recurrence run one query row at a time in fp64 (with the fp32
 * rounding points of the kernel contract mirrored where stated).
 *
 * What is computed, and where the paper states it:
 *   - E2M1 grid and the element quantizer Q_sigma(v) = sigma * Pi_G(v/sigma),
 *     round to nearest with saturation at +-6: Sec. 2, "MXFP4 Block
 *     Quantization" (Eq. mxfp4_quantizer) and App. B (grid + thresholds).
 *   - OCP floor rule e = floor(log2 M) - 2: Eq. ocp_scale, App. "Relation to
 *     OAS and the OCP Endpoint Convention" (Eq. app_ocp_floor).
 *   - UOS rule e = ceil(log2(M / 7.25)), all-zero block -> sigma = 1:
 *     Algorithm 1 (UOS-Based MXFP4 Block Quantization), Eq. uos_mapping.
 *   - Generic ceil boundary q: e = ceil(log2(M / q)) (Eq. scale_definition,
 *     Eq. uos_mapping) for 4 <= q <= 8, covering TFS (q = 6), OAS (q = 7,
 *     App. "Relation to OAS and the OCP Endpoint Convention"), UOS (7.25) and
 *     the ceil form of OCP (8); the per-head squared-error sweep over q of
 *     the empirical check in Sec. 5.5 (Table cx_distribution).
 *   - Row-sum diagnostics of block-quantized materialized probabilities:
 *     Sec. 5.5 ("Validation of Pre-Normalization Quantization", Fig.
 *     pnq_rowsum): per-row quantized mass, its split into zeroing,
 *     saturation, downward and upward rounding, and the row entropy.
 *   - Online softmax recurrence: Sec. 2 Eqs. online_attention /
 *     online_attention_output; direct placement: Eq. direct_mxfp4_tile;
 *     PNQ: Eqs. pnq_tile_contribution / pnq_online_update; Algorithm 2
 *     (MXAttention Forward Pass) without its Hadamard rotation.
 *   - Effective full-row form with beta_j = exp(m_j - m_final): App. "Full
 *     Online-Softmax Form of PNQ" (Lemma pnq_effective_full_row) and App.
 *     "Full-Row Mismatch under Direct Placement" (Eq. pnq_direct_full_rowsum).
 *   - Exact attention S = QK^T/sqrt(d), P = softmax(S), O = PV: Eq.
 *     standard_attention.
 *
 * Readings where the paper is silent (each also listed in the design notes):
 *   - ties of the nearest-grid projection go to the even magnitude index
 *     (the OCP round-to-nearest-even convention);
 *   - the code keeps the input's sign bit even when the magnitude rounds to
 *     zero; element 2i sits in the low nibble of byte i;
 *   - the E8M0 exponent is clamped to [-127, 127] (byte = e + 127, 0xFF is
 *     never produced); an all-zero block gets byte 127 (sigma = 1);
 *   - blocks are aligned to absolute multiples of 32 along their axis and a
 *     ragged tail block is padded with +0;
 *   - kernel precision contract (exact == 0): s = fp32(exact q.k),
 *     m' = max(m', RD(c * max s)) where RD rounds the exact product down to
 *     fp32, t = fmaf(s, c, -m'), p~ = fp32(2^t) flushed to 0 below 2^-126,
 *     with c = fp32(log2(e) / sqrt(d)); the running state (alpha, l, O~) is
 *     kept in fp64 here.  Rounding the maximum down gives the row maximum
 *     t >= 0, hence P~ in [1, 1 + 2^-20] and Q(P~) = 1 under both rules, as
 *     App. "Positive PNQ Normalization Factor" requires of exact arithmetic
 *     (rounding to nearest would let P~ fall just below 1, where the OCP rule
 *     drops an octave and saturates it to 0.75);
 *   - the running maximum is updated once per KV tile of width block_c, in
 *     increasing key order, with no lazy rescaling.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <unistd.h>

/* Nonnegative E2M1 grid G+ (Sec. 2 and App. B).  The array index is the
 * 3-bit magnitude field of the code. */
static const double E2M1_GRID[8] = {0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0};

enum { RULE_OCP = 0, RULE_UOS = 1, RULE_IDENTITY = 2 };

/* UOS boundary q* = 29/4 (Theorem 1, Eq. uos_optimal_qmax). */
static const double UOS_QMAX = 7.25;

/* ------------------------------------------------------------------ */
/* Scalars                                                             */
/* ------------------------------------------------------------------ */

static double bf16_bits_to_double(uint16_t b) {
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* Shared-scale exponent of a nonzero block with maximum magnitude M > 0,
 * found by search over integers (no logarithm):
 *   UOS: the smallest e with M <= 7.25 * 2^e        (= ceil(log2(M/7.25)))
 *   OCP: the largest  e with 2^(e+2) <= M           (= floor(log2 M) - 2)
 * The search starts from an exponent that provably lies on the wrong side of
 * the condition and walks one step at a time.  The result is not clamped. */
static int scale_exponent_unclamped(double M, int rule) {
    int base = ilogb(M); /* 2^base <= M < 2^(base+1) */
    if (rule == RULE_UOS) {
        int e = base - 4; /* 7.25*2^(base-4) < 2^(base-1) < M: condition false */
        while (!(M <= UOS_QMAX * ldexp(1.0, e))) e++;
        return e;
    } else {
        int e = base + 2; /* 2^(base+4) > M: condition false */
        while (!(ldexp(1.0, e + 2) <= M)) e--;
        return e;
    }
}

long mxref_scale_exponent(double M, int rule) {
    if (!(M > 0.0)) return 0; /* all-zero block: sigma = 1 */
    int e = scale_exponent_unclamped(M, rule);
    if (e < -127) e = -127;
    if (e > 127) e = 127;
    return e;
}

/* Nearest grid index of a nonnegative normalized magnitude x by brute-force
 * argmin over the finite grid.  The finite grid makes saturation automatic
 * (every x > 5 is nearest to 6).  Ties go to the even index. */
static int nearest_grid_index(double x) {
    int best = 0;
    double bd = fabs(x - E2M1_GRID[0]);
    for (int i = 1; i < 8; i++) {
        double dd = fabs(x - E2M1_GRID[i]);
        if (dd < bd || (dd == bd && (i % 2) == 0)) {
            best = i;
            bd = dd;
        }
    }
    return best;
}

/* Quantize one block of n (<= 32) values; missing tail elements count as +0.
 * Writes one 4-bit code per element (low nibble of out_codes[i]) and returns
 * the E8M0 byte. */
static uint8_t quantize_block(const double* v, int n, int rule, uint8_t* out_codes) {
    double M = 0.0;
    for (int i = 0; i < n; i++) {
        double a = fabs(v[i]);
        if (a > M) M = a;
    }
    if (M == 0.0) { /* Algorithm 1: all-zero block -> sigma = 1, p_i = 0 */
        for (int i = 0; i < n; i++) out_codes[i] = (uint8_t)(signbit(v[i]) ? 8 : 0);
        return 127;
    }
    int e = (int)mxref_scale_exponent(M, rule);
    for (int i = 0; i < n; i++) {
        double x = ldexp(fabs(v[i]), -e); /* |v| / sigma, exact */
        int idx = nearest_grid_index(x);
        out_codes[i] = (uint8_t)((signbit(v[i]) ? 8 : 0) | idx);
    }
    return (uint8_t)(e + 127);
}

/* Block quantizer on caller-given values, one code per output byte.  Used by
 * the tests for the scalar pins. */
int mxref_quantize_block(const double* v, int n, int rule, uint8_t* codes, uint8_t* scale) {
    if (n < 1 || n > 32 || (rule != RULE_OCP && rule != RULE_UOS)) return -1;
    *scale = quantize_block(v, n, rule, codes);
    return 0;
}

double mxref_decode(uint8_t code, uint8_t scale_byte) {
    double g = E2M1_GRID[code & 7];
    if (code & 8) g = -g;
    return ldexp(g, (int)scale_byte - 127);
}

/* Round a double to the nearest bf16 (ties to even), returned as bits. */
static uint16_t double_to_bf16_bits(double x) {
    if (x == 0.0) return signbit(x) ? 0x8000 : 0;
    int ex;
    double m = frexp(fabs(x), &ex);        /* |x| = m * 2^ex, m in [0.5, 1) */
    double r = nearbyint(ldexp(m, 8));     /* 8 significant bits, RNE */
    double y = ldexp(r, ex - 8);
    float f = (float)y;                    /* exact: y has 8 significant bits */
    if (signbit(x)) f = -f;
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    return (uint16_t)(u >> 16);
}

void mxref_round_bf16(const double* x, int64_t n, uint16_t* out) {
    for (int64_t i = 0; i < n; i++) out[i] = double_to_bf16_bits(x[i]);
}

/* ------------------------------------------------------------------ */
/* Threading helper                                                    */
/* ------------------------------------------------------------------ */

typedef void (*range_fn)(void* ctx, int64_t begin, int64_t end);

typedef struct {
    range_fn fn;
    void* ctx;
    int64_t begin, end;
} range_job;

static void* range_thread(void* p) {
    range_job* j = (range_job*)p;
    j->fn(j->ctx, j->begin, j->end);
    return NULL;
}

static int resolve_threads(int nthreads) {
    if (nthreads > 0) return nthreads;
    long n = sysconf(_SC_NPROCESSORS_ONLN);
    return n > 0 ? (int)n : 1;
}

static void parallel_for(int64_t n, int nthreads, range_fn fn, void* ctx) {
    int nt = resolve_threads(nthreads);
    if (nt > 256) nt = 256;
    if (n < nt) nt = (int)(n > 0 ? n : 1);
    if (nt <= 1) {
        fn(ctx, 0, n);
        return;
    }
    pthread_t th[256];
    range_job jobs[256];
    for (int t = 0; t < nt; t++) {
        jobs[t].fn = fn;
        jobs[t].ctx = ctx;
        jobs[t].begin = n * t / nt;
        jobs[t].end = n * (t + 1) / nt;
        pthread_create(&th[t], NULL, range_thread, &jobs[t]);
    }
    for (int t = 0; t < nt; t++) pthread_join(th[t], NULL);
}

/* ------------------------------------------------------------------ */
/* Tensor quantizers                                                   */
/* ------------------------------------------------------------------ */

/* Blocks along the last axis: x is [rows, d] bf16 with d a multiple of 32.
 * codes [rows, d/2] (element 2i in the low nibble), scales [rows, d/32]. */
typedef struct {
    const uint16_t* x;
    int64_t d;
    int rule;
    uint8_t* codes;
    uint8_t* scales;
} qrows_ctx;

static void qrows_range(void* p, int64_t r0, int64_t r1) {
    qrows_ctx* c = (qrows_ctx*)p;
    double v[32];
    uint8_t cd[32];
    for (int64_t r = r0; r < r1; r++) {
        for (int64_t b = 0; b < c->d / 32; b++) {
            const uint16_t* src = c->x + r * c->d + b * 32;
            for (int i = 0; i < 32; i++) v[i] = bf16_bits_to_double(src[i]);
            c->scales[r * (c->d / 32) + b] = quantize_block(v, 32, c->rule, cd);
            uint8_t* dst = c->codes + r * (c->d / 2) + b * 16;
            for (int i = 0; i < 16; i++) dst[i] = (uint8_t)(cd[2 * i] | (cd[2 * i + 1] << 4));
        }
    }
}

int mxref_quantize_rows(const uint16_t* x, int64_t rows, int64_t d, int rule, uint8_t* codes,
                        uint8_t* scales, int nthreads) {
    if (d <= 0 || d % 32 != 0 || rows < 0) return -1;
    if (rule != RULE_OCP && rule != RULE_UOS) return -1;
    qrows_ctx c = {x, d, rule, codes, scales};
    parallel_for(rows, nthreads, qrows_range, &c);
    return 0;
}

/* ------------------------------------------------------------------ */
/* Fixed Hadamard rotation of Q and K (Sec. 4.3, Algorithm 2)          */
/* ------------------------------------------------------------------ */

/* x <- x R_H for one row of d = 2^k values, R_H = H / sqrt(d) with H the
 * Sylvester Hadamard matrix, H[i][j] = (-1)^popcount(i & j) (symmetric, and
 * orthogonal once scaled).  The paper fixes neither the size, the ordering
 * nor the arithmetic; the reading here (shared with the GPU kernel's
 * contract): natural Sylvester ordering without random signs, formed in fp32
 * by the radix-2 fast Walsh-Hadamard transform with its stages in the order
 * h = 1, 2, 4, ..., d/2, each stage mapping every pair (a, b) = (x[i], x[i+h])
 * with bit h of i clear to (a + b, a - b), then one fp32 multiplication of
 * each element by fp32(1/sqrt(d)). */
void mxref_hadamard_f32(float* x, int64_t d) {
    for (int64_t h = 1; h < d; h *= 2) {
        for (int64_t i = 0; i < d; i++) {
            if (i & h) continue;
            float a = x[i], b = x[i + h];
            x[i] = a + b;
            x[i + h] = a - b;
        }
    }
    const float s = (float)(1.0 / sqrt((double)d));
    for (int64_t i = 0; i < d; i++) x[i] = x[i] * s;
}

/* Rows rotated by R_H, then quantized along the last axis as
 * mxref_quantize_rows does (from the fp32 rotated values). */
static void qrows_rot_range(void* p, int64_t r0, int64_t r1) {
    qrows_ctx* c = (qrows_ctx*)p;
    float y[128];
    double v[32];
    uint8_t cd[32];
    for (int64_t r = r0; r < r1; r++) {
        for (int64_t i = 0; i < c->d; i++) y[i] = (float)bf16_bits_to_double(c->x[r * c->d + i]);
        mxref_hadamard_f32(y, c->d);
        for (int64_t b = 0; b < c->d / 32; b++) {
            for (int i = 0; i < 32; i++) v[i] = (double)y[b * 32 + i];
            c->scales[r * (c->d / 32) + b] = quantize_block(v, 32, c->rule, cd);
            uint8_t* dst = c->codes + r * (c->d / 2) + b * 16;
            for (int i = 0; i < 16; i++) dst[i] = (uint8_t)(cd[2 * i] | (cd[2 * i + 1] << 4));
        }
    }
}

int mxref_quantize_rows_rotated(const uint16_t* x, int64_t rows, int64_t d, int rule, uint8_t* codes,
                                uint8_t* scales, int nthreads) {
    if (d != 128 || rows < 0) return -1;
    if (rule != RULE_OCP && rule != RULE_UOS) return -1;
    qrows_ctx c = {x, d, rule, codes, scales};
    parallel_for(rows, nthreads, qrows_rot_range, &c);
    return 0;
}

/* ------------------------------------------------------------------ */
/* Generic boundary family q (Sec. 4.1, Theorem 1; App. "Relation to    */
/* OAS and the OCP Endpoint Convention")                               */
/* ------------------------------------------------------------------ */

/* The ceil rule with boundary q: e = the smallest integer with M <= q 2^e
 * (= ceil(log2(M/q))), clamped to [-127, 127]; q = 7.25 is UOS, q = 6 maps
 * every block maximum into (3, 6] (no clipping), q = 8 is the ceil form of
 * the OCP boundary.  Found by search, for 4 <= q <= 8. */
static int scale_exponent_qmax(double M, double q) {
    int e = ilogb(M) - 4; /* q 2^e <= 2^(ilogb(M)-1) < M: condition false */
    while (!(M <= q * ldexp(1.0, e))) e++;
    if (e < -127) e = -127;
    if (e > 127) e = 127;
    return e;
}

static uint8_t quantize_block_qmax(const double* v, int n, double q, uint8_t* out_codes) {
    double M = 0.0;
    for (int i = 0; i < n; i++)
        if (fabs(v[i]) > M) M = fabs(v[i]);
    if (M == 0.0) {
        for (int i = 0; i < n; i++) out_codes[i] = (uint8_t)(signbit(v[i]) ? 8 : 0);
        return 127;
    }
    int e = scale_exponent_qmax(M, q);
    for (int i = 0; i < n; i++) {
        int idx = nearest_grid_index(ldexp(fabs(v[i]), -e));
        out_codes[i] = (uint8_t)((signbit(v[i]) ? 8 : 0) | idx);
    }
    return (uint8_t)(e + 127);
}

int mxref_quantize_block_qmax(const double* v, int n, double q, uint8_t* codes, uint8_t* scale) {
    if (n < 1 || n > 32 || !(q >= 4.0 && q <= 8.0)) return -1;
    *scale = quantize_block_qmax(v, n, q, codes);
    return 0;
}

/* Blocks along the last axis with boundary q: x [rows, d] bf16 -> codes
 * [rows, d/2], scales [rows, d/32], as mxref_quantize_rows. */
int mxref_quantize_rows_qmax(const uint16_t* x, int64_t rows, int64_t d, double q, uint8_t* codes,
                             uint8_t* scales) {
    if (d <= 0 || d % 32 != 0 || rows < 0 || !(q >= 4.0 && q <= 8.0)) return -1;
    double v[32];
    uint8_t cd[32];
    for (int64_t r = 0; r < rows; r++)
        for (int64_t b = 0; b < d / 32; b++) {
            for (int i = 0; i < 32; i++) v[i] = bf16_bits_to_double(x[r * d + b * 32 + i]);
            scales[r * (d / 32) + b] = quantize_block_qmax(v, 32, q, cd);
            for (int i = 0; i < 16; i++) codes[r * (d / 2) + b * 16 + i] = (uint8_t)(cd[2 * i] | (cd[2 * i + 1] << 4));
        }
    return 0;
}

/* Sum over a head's blocks of the squared quantization error sum_i (v_i -
 * Q_q(v_i))^2, for each boundary in qs[0..nq): the per-tensor MSE sweep of
 * the empirical check of Sec. 5.5 (Table cx_distribution).  axis 3: blocks
 * along d of x [heads, N, d]; axis 2: blocks of 32 consecutive tokens per
 * channel, the last one padded with +0 (padding adds no error).  sse is
 * [heads, nq], fp64. */
typedef struct {
    const uint16_t* x;
    int64_t N, d;
    int axis;
    const double* qs;
    int nq;
    double* sse;
} sse_ctx;

static void sse_range(void* p, int64_t h0, int64_t h1) {
    sse_ctx* c = (sse_ctx*)p;
    double v[32];
    uint8_t cd[32];
    const int64_t nb = (c->N + 31) / 32;
    for (int64_t h = h0; h < h1; h++) {
        const uint16_t* xh = c->x + h * c->N * c->d;
        for (int j = 0; j < c->nq; j++) c->sse[h * c->nq + j] = 0.0;
        const int64_t nblocks = c->axis == 3 ? c->N * (c->d / 32) : c->d * nb;
        for (int64_t blk = 0; blk < nblocks; blk++) {
            if (c->axis == 3) {
                const int64_t r = blk / (c->d / 32), b = blk % (c->d / 32);
                for (int i = 0; i < 32; i++) v[i] = bf16_bits_to_double(xh[r * c->d + b * 32 + i]);
            } else {
                const int64_t ch = blk / nb, b = blk % nb;
                for (int i = 0; i < 32; i++) {
                    const int64_t t = b * 32 + i;
                    v[i] = t < c->N ? bf16_bits_to_double(xh[t * c->d + ch]) : 0.0;
                }
            }
            for (int j = 0; j < c->nq; j++) {
                uint8_t sc = quantize_block_qmax(v, 32, c->qs[j], cd);
                double acc = 0.0;
                for (int i = 0; i < 32; i++) {
                    const double err = v[i] - mxref_decode(cd[i], sc);
                    acc += err * err;
                }
                c->sse[h * c->nq + j] += acc;
            }
        }
    }
}

int mxref_qmax_sse(const uint16_t* x, int64_t heads, int64_t N, int64_t d, int axis, const double* qs,
                   int nq, double* sse, int nthreads) {
    if (heads < 0 || N < 1 || d <= 0 || d % 32 != 0 || (axis != 2 && axis != 3) || nq < 1) return -1;
    for (int j = 0; j < nq; j++)
        if (!(qs[j] >= 4.0 && qs[j] <= 8.0)) return -1;
    sse_ctx c = {x, N, d, axis, qs, nq, sse};
    parallel_for(heads, nthreads, sse_range, &c);
    return 0;
}

/* Blocks along the token axis: x is [heads, N, d] bf16.  For each (head,
 * channel) the N tokens form ceil(N/32) blocks of 32 consecutive tokens, the
 * last one padded with +0.  codes [heads, d, nb*16], scales [heads, d, nb]
 * with nb = ceil(N/32): tokens contiguous per channel. */
typedef struct {
    const uint16_t* x;
    int64_t N, d, nb;
    int rule;
    uint8_t* codes;
    uint8_t* scales;
} qkeys_ctx;

static void qkeys_range(void* p, int64_t i0, int64_t i1) {
    qkeys_ctx* c = (qkeys_ctx*)p;
    double v[32];
    uint8_t cd[32];
    for (int64_t i = i0; i < i1; i++) { /* i = head * d + channel */
        int64_t h = i / c->d, ch = i % c->d;
        const uint16_t* base = c->x + h * c->N * c->d + ch;
        for (int64_t b = 0; b < c->nb; b++) {
            for (int k = 0; k < 32; k++) {
                int64_t n = b * 32 + k;
                v[k] = n < c->N ? bf16_bits_to_double(base[n * c->d]) : 0.0;
            }
            c->scales[i * c->nb + b] = quantize_block(v, 32, c->rule, cd);
            uint8_t* dst = c->codes + i * c->nb * 16 + b * 16;
            for (int k = 0; k < 16; k++) dst[k] = (uint8_t)(cd[2 * k] | (cd[2 * k + 1] << 4));
        }
    }
}

int mxref_quantize_keys(const uint16_t* x, int64_t heads, int64_t N, int64_t d, int rule,
                        uint8_t* codes, uint8_t* scales, int nthreads) {
    if (N <= 0 || d <= 0 || heads < 0) return -1;
    if (rule != RULE_OCP && rule != RULE_UOS) return -1;
    qkeys_ctx c = {x, N, d, (N + 31) / 32, rule, codes, scales};
    parallel_for(heads * d, nthreads, qkeys_range, &c);
    return 0;
}

/* Dequantize a row-blocked tensor: codes [rows, d/2], scales [rows, d/32]
 * -> out [rows, d] doubles. */
void mxref_dequant_rows(const uint8_t* codes, const uint8_t* scales, int64_t rows, int64_t d,
                        double* out) {
    for (int64_t r = 0; r < rows; r++)
        for (int64_t c = 0; c < d; c++) {
            uint8_t byte = codes[r * (d / 2) + c / 2];
            uint8_t code = (c % 2 == 0) ? (byte & 15) : (byte >> 4);
            out[r * d + c] = mxref_decode(code, scales[r * (d / 32) + c / 32]);
        }
}

/* Dequantize one head of a token-blocked tensor: codes [d, nb*16],
 * scales [d, nb] -> out [N, d] doubles (token-major). */
void mxref_dequant_keys(const uint8_t* codes, const uint8_t* scales, int64_t N, int64_t d,
                        double* out) {
    int64_t nb = (N + 31) / 32;
    for (int64_t c = 0; c < d; c++)
        for (int64_t n = 0; n < N; n++) {
            uint8_t byte = codes[c * nb * 16 + n / 2];
            uint8_t code = (n % 2 == 0) ? (byte & 15) : (byte >> 4);
            out[n * d + c] = mxref_decode(code, scales[c * nb + n / 32]);
        }
}

/* ------------------------------------------------------------------ */
/* Attention                                                           */
/* ------------------------------------------------------------------ */

/* Tiled online-softmax attention for a set of query rows of one head.
 *
 *   qrows  [n_rows, d]  query rows (dequantized Q^ values, or raw values)
 *   keys   [N, d]       K^ (token-major)
 *   vals   [N, d]       V^ (token-major)
 *   p_rule RULE_OCP / RULE_UOS quantize each tile's exponentials in 32-key
 *          blocks; RULE_IDENTITY leaves them unquantized (P^ = P~)
 *   pnq    0: l += sum(P~) (direct placement); 1: l += sum(P^) (PNQ)
 *   exact  0: kernel fp32 contract for s, m', t, p~; 1: fp64 throughout
 *   block_c KV tile width (a multiple of 32 unless p_rule is identity)
 *   out    [n_rows, d] O = O~ / l in fp64
 *   diag   [n_rows, 8] or NULL:
 *          0 l, 1 induced row sum (sum_j beta_j sum P^_j) / l,
 *          2 l rebuilt from the unrolled form, 3 max |O - O_unrolled|,
 *          4 number of tiles, 5 number of tiles where the max rose,
 *          6 elements of P~ within 4 fp32 ulps of an E2M1 decision threshold
 *            of their block (near_threshold), 7 blocks whose maximum lies
 *            within 4 fp32 ulps of an end of its scale rule's range
 *            (near_boundary).  Columns 6 and 7 audit the exponential: an
 *            exp2 that is faithful rather than correctly rounded can move
 *            exactly these elements to a neighbouring code (or these blocks
 *            to a neighbouring scale); every other element's code is fixed
 *            by the fp32 argument t alone.
 */
/* Distance, in units of the fp32 spacing just above x > 0, within which a
 * value counts as "near" a decision point in the exponential audit. */
static int near_f32(double x, double point) {
    const float xf = (float)x;
    const double ulp = (double)nextafterf(xf, INFINITY) - (double)xf;
    return fabs(x - point) <= 4.0 * ulp;
}

/* E2M1 decision thresholds: the midpoints between neighbouring grid values
 * (App. B), in units of the block scale. */
static const double E2M1_MIDPOINTS[7] = {0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0};

/* Audit of one quantized block of fp32 exponentials p[0..n) with scale byte
 * sc: adds the number of elements near a decision threshold to *near_el and
 * one to *near_blk when the block maximum is near an end of the rule's
 * normalized range (UOS (3.625, 7.25] sigma, OCP [4, 8) sigma), unless the
 * block holds the row maximum. */
static void audit_block(const double* p, int64_t n, uint8_t sc, int rule, double* near_el,
                        double* near_blk) {
    const double sigma = ldexp(1.0, (int)sc - 127);
    double M = 0.0;
    for (int64_t i = 0; i < n; i++) {
        if (p[i] > M) M = p[i];
        if (!(p[i] > 0.0)) continue;
        for (int k = 0; k < 7; k++)
            if (near_f32(p[i], E2M1_MIDPOINTS[k] * sigma)) {
                *near_el += 1.0;
                break;
            }
    }
    /* a block holding the row maximum has M in [1, 1 + 2^-20]: exp2 of an
     * argument t >= 0 is never below 1, so its scale cannot move */
    if (!(M > 0.0) || M >= 1.0) return;
    const double lo = (rule == RULE_UOS ? 0.5 * UOS_QMAX : 4.0) * sigma;
    const double hi = (rule == RULE_UOS ? UOS_QMAX : 8.0) * sigma;
    if (near_f32(M, lo) || near_f32(M, hi)) *near_blk += 1.0;
}

typedef struct {
    const double* q;
    const double* k;
    const double* v;
    int64_t N, d, block_c;
    int p_rule, pnq, exact;
    double* out;
    double* diag;
} attn_ctx;

static void attn_range(void* p, int64_t r0, int64_t r1) {
    attn_ctx* A = (attn_ctx*)p;
    const int64_t N = A->N, d = A->d, bc = A->block_c;
    const int64_t ntiles = (N + bc - 1) / bc;
    const double c64 = 1.4426950408889634 / sqrt((double)d); /* log2(e)/sqrt(d) */
    const float c32 = (float)c64;
    double* s = (double*)malloc(sizeof(double) * bc);
    double* pt = (double*)malloc(sizeof(double) * bc);
    double* ph = (double*)malloc(sizeof(double) * bc);
    double* o = (double*)malloc(sizeof(double) * d);
    /* per-tile records for the unrolled (effective full-row) form */
    double* tm = NULL;
    double* tmass_hat = NULL;
    double* tmass_l = NULL;
    double* tO = NULL;
    if (A->diag) {
        tm = (double*)malloc(sizeof(double) * ntiles);
        tmass_hat = (double*)malloc(sizeof(double) * ntiles);
        tmass_l = (double*)malloc(sizeof(double) * ntiles);
        tO = (double*)malloc(sizeof(double) * ntiles * d);
    }
    uint8_t cd[32];

    for (int64_t r = r0; r < r1; r++) {
        const double* qr = A->q + r * d;
        double m = -INFINITY, l = 0.0;
        double near_el = 0.0, near_blk = 0.0;
        int rises = 0;
        for (int64_t c = 0; c < d; c++) o[c] = 0.0;

        for (int64_t j = 0; j < ntiles; j++) {
            int64_t k0 = j * bc;
            int64_t n = (k0 + bc <= N) ? bc : N - k0; /* valid keys in this tile */

            /* S_ij = Q_i K_j^T (the 1/sqrt(d) factor is folded into c) */
            double smax = -INFINITY;
            for (int64_t t = 0; t < n; t++) {
                const double* kr = A->k + (k0 + t) * d;
                double acc = 0.0;
                for (int64_t c = 0; c < d; c++) acc += qr[c] * kr[c];
                s[t] = A->exact ? acc : (double)(float)acc;
                if (s[t] > smax) smax = s[t];
            }
            /* m_new = max(m, rowmax(S_ij)) in log2 units */
            double u;
            if (A->exact) {
                u = smax * c64;
            } else {
                /* largest fp32 not above c * max s (exact product in fp64) */
                double prod = (double)c32 * smax;
                float u32 = (float)prod;
                if ((double)u32 > prod) u32 = nextafterf(u32, -INFINITY);
                u = u32;
            }
            double m_new = u > m ? u : m;
            if (j > 0 && m_new > m) rises++;
            double alpha = exp2(m - m_new); /* 0 on the first tile */

            /* P~ = exp(S - m_new) */
            for (int64_t t = 0; t < n; t++) {
                if (A->exact) {
                    pt[t] = exp2(s[t] * c64 - m_new);
                } else {
                    float tt = fmaf((float)s[t], c32, (float)(-m_new));
                    float pv = (float)exp2((double)tt);
                    if (pv < 1.17549435e-38f) pv = 0.0f; /* below 2^-126 -> 0 */
                    pt[t] = pv;
                }
            }
            for (int64_t t = n; t < bc; t++) pt[t] = 0.0; /* tail padding */

            /* P^ = Q*(P~) in 32-key blocks aligned to absolute key index */
            if (A->p_rule == RULE_IDENTITY) {
                for (int64_t t = 0; t < n; t++) ph[t] = pt[t];
            } else {
                for (int64_t b = 0; b < bc; b += 32) {
                    int64_t nv = n - b;
                    if (nv <= 0) break;
                    if (nv > 32) nv = 32;
                    uint8_t sc = quantize_block(pt + b, 32, A->p_rule, cd);
                    for (int64_t t = 0; t < nv; t++) ph[b + t] = mxref_decode(cd[t], sc);
                    if (A->diag && !A->exact) audit_block(pt + b, nv, sc, A->p_rule, &near_el, &near_blk);
                }
            }

            double mass_t = 0.0, mass_h = 0.0;
            for (int64_t t = 0; t < n; t++) {
                mass_t += pt[t];
                mass_h += ph[t];
            }
            double dl = A->pnq ? mass_h : mass_t;
            l = alpha * l + dl;
            for (int64_t c = 0; c < d; c++) o[c] *= alpha;
            if (A->diag) {
                double* oj = tO + j * d;
                for (int64_t c = 0; c < d; c++) oj[c] = 0.0;
                for (int64_t t = 0; t < n; t++) {
                    const double* vr = A->v + (k0 + t) * d;
                    for (int64_t c = 0; c < d; c++) oj[c] += ph[t] * vr[c];
                }
                for (int64_t c = 0; c < d; c++) o[c] += oj[c];
                tm[j] = m_new;
                tmass_hat[j] = mass_h;
                tmass_l[j] = dl;
            } else {
                for (int64_t t = 0; t < n; t++) {
                    const double* vr = A->v + (k0 + t) * d;
                    for (int64_t c = 0; c < d; c++) o[c] += ph[t] * vr[c];
                }
            }
            m = m_new;
        }

        double* orow = A->out + r * d;
        for (int64_t c = 0; c < d; c++) orow[c] = o[c] / l;

        if (A->diag) {
            /* beta_j = exp(m_j - m_final); unrolled l and O~ */
            double lu = 0.0, mass = 0.0, maxdiff = 0.0;
            for (int64_t j = 0; j < ntiles; j++) {
                double beta = exp2(tm[j] - m);
                lu += beta * tmass_l[j];
                mass += beta * tmass_hat[j];
            }
            for (int64_t c = 0; c < d; c++) {
                double ou = 0.0;
                for (int64_t j = 0; j < ntiles; j++) ou += exp2(tm[j] - m) * tO[j * d + c];
                double df = fabs(ou / lu - orow[c]);
                if (df > maxdiff) maxdiff = df;
            }
            double* dg = A->diag + r * 8;
            dg[0] = l;
            dg[1] = mass / l;
            dg[2] = lu;
            dg[3] = maxdiff;
            dg[4] = (double)ntiles;
            dg[5] = (double)rises;
            dg[6] = near_el;
            dg[7] = near_blk;
        }
    }
    free(s);
    free(pt);
    free(ph);
    free(o);
    free(tm);
    free(tmass_hat);
    free(tmass_l);
    free(tO);
}

int mxref_attention_rows(const double* qrows, const double* keys, const double* vals, int64_t N,
                         int64_t d, int64_t n_rows, int p_rule, int pnq, int exact,
                         int64_t block_c, double* out, double* diag, int nthreads) {
    if (N <= 0 || d <= 0 || n_rows < 0 || block_c <= 0) return -1;
    if (p_rule != RULE_OCP && p_rule != RULE_UOS && p_rule != RULE_IDENTITY) return -1;
    if (p_rule != RULE_IDENTITY && block_c % 32 != 0) return -1;
    attn_ctx A = {qrows, keys, vals, N, d, block_c, p_rule, pnq, exact, out, diag};
    parallel_for(n_rows, nthreads, attn_range, &A);
    return 0;
}

/* Exact attention of Eq. standard_attention for a set of query rows of one
 * head, two-pass softmax in fp64:  out = softmax(q K^T / sqrt(d)) V. */
typedef struct {
    const double* q;
    const double* k;
    const double* v;
    int64_t N, d;
    double* out;
} exact_ctx;

static void exact_range(void* p, int64_t r0, int64_t r1) {
    exact_ctx* E = (exact_ctx*)p;
    const int64_t N = E->N, d = E->d;
    double* s = (double*)malloc(sizeof(double) * N);
    const double scale = 1.0 / sqrt((double)d);
    for (int64_t r = r0; r < r1; r++) {
        const double* qr = E->q + r * d;
        double mx = -INFINITY;
        for (int64_t n = 0; n < N; n++) {
            double acc = 0.0;
            for (int64_t c = 0; c < d; c++) acc += qr[c] * E->k[n * d + c];
            s[n] = acc * scale;
            if (s[n] > mx) mx = s[n];
        }
        double sum = 0.0;
        for (int64_t n = 0; n < N; n++) {
            s[n] = exp(s[n] - mx);
            sum += s[n];
        }
        double* orow = E->out + r * d;
        for (int64_t c = 0; c < d; c++) orow[c] = 0.0;
        for (int64_t n = 0; n < N; n++) {
            double w = s[n] / sum;
            for (int64_t c = 0; c < d; c++) orow[c] += w * E->v[n * d + c];
        }
    }
    free(s);
}

int mxref_attention_exact_rows(const double* qrows, const double* keys, const double* vals,
                               int64_t N, int64_t d, int64_t n_rows, double* out, int nthreads) {
    if (N <= 0 || d <= 0 || n_rows < 0) return -1;
    exact_ctx E = {qrows, keys, vals, N, d, out};
    parallel_for(n_rows, nthreads, exact_range, &E);
    return 0;
}

/* ------------------------------------------------------------------ */
/* Row-sum diagnostics on materialized probabilities (Sec. 5.5,         */
/* "Validation of Pre-Normalization Quantization", Fig. pnq_rowsum)     */
/* ------------------------------------------------------------------ */

/* Exact softmax rows P[r, n] = softmax_n(q_r . k_n / sqrt(d)) in fp64 (Eq.
 * standard_attention without the product with V). */
typedef struct {
    const double* q;
    const double* k;
    int64_t N, d;
    double* P;
} softmax_ctx;

static void softmax_range(void* p, int64_t r0, int64_t r1) {
    softmax_ctx* C = (softmax_ctx*)p;
    const int64_t N = C->N, d = C->d;
    const double scale = 1.0 / sqrt((double)d);
    for (int64_t r = r0; r < r1; r++) {
        const double* qr = C->q + r * d;
        double* prow = C->P + r * N;
        double mx = -INFINITY;
        for (int64_t n = 0; n < N; n++) {
            double acc = 0.0;
            for (int64_t c = 0; c < d; c++) acc += qr[c] * C->k[n * d + c];
            prow[n] = acc * scale;
            if (prow[n] > mx) mx = prow[n];
        }
        double sum = 0.0;
        for (int64_t n = 0; n < N; n++) {
            prow[n] = exp(prow[n] - mx);
            sum += prow[n];
        }
        for (int64_t n = 0; n < N; n++) prow[n] /= sum;
    }
}

int mxref_softmax_rows(const double* qrows, const double* keys, int64_t N, int64_t d, int64_t n_rows,
                       double* P, int nthreads) {
    if (N <= 0 || d <= 0 || n_rows < 0) return -1;
    softmax_ctx C = {qrows, keys, N, d, P};
    parallel_for(n_rows, nthreads, softmax_range, &C);
    return 0;
}

/* What block-wise MXFP4 quantization does to the mass of each row of a
 * materialized probability matrix (the diagnostic of Fig. pnq_rowsum).
 * P is fp32 [rows, ld], N valid entries per row (p >= 0), blocks of 32
 * consecutive entries from the row start, the last one padded with +0.
 * Each entry is pre-scaled x = fl32(gamma * p) (the "pre-quant global
 * scaling" baseline of Fig. pnq_rowsum (C); gamma = 1 is plain
 * quantization), quantized with the block's scale rule to Q(x), and
 * contributes Q(x) * g - p with g = fl64(1 / gamma).  Entries fall in one of
 *   zeroing     p > 0 and Q(x) = 0
 *   saturation  x / sigma > 6 (above the largest E2M1 magnitude)
 *   down        0 < Q(x) < x otherwise
 *   up          Q(x) > x
 *   exact       Q(x) = x
 * stats[r] = {sum_j Q(x_j) g, sum_j p_j, zeroing, saturation, down, up,
 * exact, -sum_{p_j > 0} p_j ln p_j}; the row sum minus the mass equals the
 * sum of the five contributions. */
typedef struct {
    const float* P;
    int64_t N, ld;
    int rule;
    float gamma;
    double* stats;
} diag_ctx;

static void diag_range(void* p, int64_t r0, int64_t r1) {
    diag_ctx* C = (diag_ctx*)p;
    const double g = 1.0 / (double)C->gamma;
    double x[32];
    uint8_t cd[32];
    for (int64_t r = r0; r < r1; r++) {
        const float* prow = C->P + r * C->ld;
        double st[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        for (int64_t b = 0; b < C->N; b += 32) {
            const int n = (int)((C->N - b) < 32 ? (C->N - b) : 32);
            for (int i = 0; i < n; i++) x[i] = (double)(float)(C->gamma * prow[b + i]);
            const uint8_t sc = quantize_block(x, n, C->rule, cd);
            const double sigma = ldexp(1.0, (int)sc - 127);
            for (int i = 0; i < n; i++) {
                const double pj = (double)prow[b + i];
                const double qx = mxref_decode(cd[i], sc);
                const double c = qx * g - pj;
                int cls;
                if (pj > 0.0 && (cd[i] & 7) == 0)
                    cls = 2;
                else if (x[i] > 6.0 * sigma)
                    cls = 3;
                else if (qx < x[i])
                    cls = 4;
                else if (qx > x[i])
                    cls = 5;
                else
                    cls = 6;
                st[0] += qx * g;
                st[1] += pj;
                st[cls] += c;
                if (pj > 0.0) st[7] -= pj * log(pj);
            }
        }
        memcpy(C->stats + r * 8, st, sizeof st);
    }
}

int mxref_rowsum_diag(const float* P, int64_t rows, int64_t N, int64_t ld, int rule, float gamma,
                      double* stats, int nthreads) {
    if (rows < 0 || N < 1 || ld < N || (rule != RULE_OCP && rule != RULE_UOS) || !(gamma > 0.0f))
        return -1;
    diag_ctx C = {P, N, ld, rule, gamma, stats};
    parallel_for(rows, nthreads, diag_range, &C);
    return 0;
}

int mxref_threads(int nthreads) { return resolve_threads(nthreads); }
