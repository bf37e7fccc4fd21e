// attention.hip -- fused MXFP4 flash attention forward for gfx950.
//
// One workgroup = 4 waves = 128 query rows of one (batch, head); each wave
// owns 32 query rows.  The kernel walks the keys in tiles of 128 (the KV tile
// B_c) in increasing order, as Algorithm 2 does, and for each tile:
//
//   1. reads the tile's MXFP4 K^ and V^ codes and E8M0 scales from LDS (the
//      tiles after it are already in flight into the other LDS stages,
//      copied by buffer loads straight into LDS);
//   2. S^T = K^ Q^T on the block-scaled FP4 matrix cores
//      (V_MFMA_SCALE_F32_32X32X64_F8F6F4, fp32 accumulation);
//   3. online softmax in registers: running maximum m, correction
//      alpha = exp2(m_old - m_new), P~ = exp2(s*c - m_new) with
//      c = log2(e)/sqrt(d)  (Sec. 2, Eq. online_attention);
//   4. quantizes P~ in 32-key blocks in registers with the mode's scale rule
//      straight into the FP4 operand layout of the PV product (Algorithm 2,
//      P^ = Q*(P~));
//   5. l = alpha*l + sum(P~) (direct placement, Eq. direct_mxfp4_tile) or
//      l = alpha*l + sum(P^) (PNQ, Eq. pnq_online_update);  the PNQ row sum
//      of the dequantized P^ is accumulated on the matrix cores (RowSum);
//   6. O~^T = diag(alpha) O~^T + V^T P^T on the FP4 matrix cores, one
//      64-key chunk at a time, so the first chunk's products run while the
//      second chunk's P~ is formed.
//
// After the last tile O = O~ / l is rounded to bf16 (Eq.
// online_attention_output).  For long key sequences the steps of
// consecutive tiles overlap (attention_pipelined_kernel: the score products
// of tile j + 1 and the second PV chunk of tile j - 1 run during the softmax
// of tile j); key sequences of at most four tiles stay in LDS for the whole
// workgroup (attention_resident_kernel).
//
// Layouts chosen so that no lane shuffles are needed between the two
// products: with S^T (keys as rows) each lane holds the scores of ONE query
// for 16 keys of a 32x32 tile.  The key order of the K^ rows fed to the S
// product is permuted so that after two tiles (64 keys) lane (query q,
// half h) holds exactly keys 32h..32h+31 of that 64-key chunk in natural
// order: one complete MXFP4 block of P~, which is both the unit of the P~
// quantization and the B-operand layout of the 32x32x64 PV product.
//
// The softmax path (one FMA, one exp, half an FP4 conversion and half a
// 3-way max per score) costs about twice the matrix-core time of the two
// products, so the kernel is bound by vector-ALU issue; two workgroups per CU
// give each SIMD two waves, whose matrix-core work overlaps the other's
// softmax (not for free: vector instructions issue about a third slower
// while another wave's FP4 32x32x64 products execute).
//
// Arithmetic contract (mirrored by the CPU oracle):
//   s     fp32 accumulation of exact FP4 products (matrix core)
//   m'    max(m', RD(c * max s)), RD = largest fp32 <= the exact product
//   t     fmaf(s, c, -m')
//   P~    v_exp_f32(t): faithful (<1 ulp), flushes results below 2^-126
//   scale from the block maximum of P~ (exp2 of the block's largest t)
//   P^    the gfx950 FP4 conversion of P~ / 2^e (round to nearest, ties to
//         the even code, saturating)
#include <type_traits>

#include "device_common.h"
#include "launch.h"

namespace mxattn {
namespace {

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * 64;
constexpr int kQw = 32;  // query rows per wave

// LDS stage layout (bytes)
constexpr int kKcOff = 0;      // K^ codes: 128 rows x 64 B, rows in MFMA order
constexpr int kVcOff = 8192;   // V^ codes: 128 rows (channels) x 64 B (128 keys)
constexpr int kKsOff = 16384;  // K^ scales: 64 lanes x 8 B, in MFMA operand order
constexpr int kVsOff = 16896;  // V^ scales: 64 lanes x 8 B, in MFMA operand order
constexpr int kStageBytes = 17408;
constexpr int kOutStageBytes = 2048;  // per wave: 8 output rows of 256 B
// Short key sequences are bound by the output stores, long ones by the
// softmax: the resident kernel stages its output rows through LDS (fully
// coalesced 1 KiB stores, four dependent LDS round trips) up to this many
// key tiles and stores 16 bytes per lane directly above it.
constexpr int kStagedStoreMaxTiles = 2;

// 16-byte slot swizzle of a 64-byte LDS row: any 16 consecutive rows read at
// the same logical slot hit 16 distinct 16-byte bank groups.
__device__ __forceinline__ int swz(int row) { return ((row >> 1) ^ (row >> 2)) & 3; }

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// Global -> LDS copy of one tile's K^ and V^ codes (16 KiB) with gfx950
// buffer loads that write to LDS: lane i of a wave-wide load writes the 16
// bytes it fetched to LDS base + 16*i, so each lane fetches whatever chunk
// belongs at its slot of the permuted, swizzled layout.  Nothing passes
// through VGPRs; completion is tracked by vmcnt.  Wave w copies LDS bytes
// [2048 w, 2048 w + 2048) of each of the two 8 KiB code regions, and wave 0
// also the tile's K^ and V^ scales, already in the lanes' MFMA operand order
// (tile_scales_kernel).  Each source is a buffer resource over one head's
// array: a lane's offset within a tile is fixed, the tile's offset is a
// scalar, so no per-tile address arithmetic runs on the vector units.  In the
// last tile, K^ rows of keys past N lie past the end of the head's array and
// read as zero (buffer range check; their scores are masked anyway); V^ key
// blocks past the end of a channel row read the start of the next row (zeros
// after the last row).  Those V^ values meet P^ entries that are zero, and
// FP4 codes and E8M0 scales are always finite, so they contribute nothing.
struct TileLoader {
    __amdgpu_buffer_rsrc_t kc;  // this head's K^ codes [N, 64]
    __amdgpu_buffer_rsrc_t vc;  // this head's V^ codes [128, nb * 16]
    __amdgpu_buffer_rsrc_t sc;  // this head's operand-order scales [ntiles, 1024]
    uint32_t koff[2];           // lane offsets (bytes) within a tile
    uint32_t voff[2];
    int wave, lane;

    // raw buffer, 32-bit data format (word 3 of the gfx9 buffer descriptor)
    static constexpr int kRsrcFlags = 0x00020000;

    __device__ __forceinline__ TileLoader(const AttnArgs& a, int bh, int wave_, int lane_)
        : wave(wave_), lane(lane_) {
        const int ntiles = (a.N + 127) / 128;
        kc = __builtin_amdgcn_make_buffer_rsrc((void*)(a.kc + (int64_t)bh * a.N * 64), 0, a.N * 64, kRsrcFlags);
        vc = __builtin_amdgcn_make_buffer_rsrc((void*)(a.vc + (int64_t)bh * 128 * a.nb * 16), 0,
                                               128 * a.nb * 16, kRsrcFlags);
        sc = __builtin_amdgcn_make_buffer_rsrc((void*)(a.sc + (int64_t)bh * ntiles * 1024), 0, ntiles * 1024,
                                               kRsrcFlags);
#pragma unroll
        for (int it = 0; it < 2; it++) {
            const int p = (2 * wave + it) * 64 + lane;  // 16-byte slot of the region
            const int row = p >> 2;
            // K^: LDS row 64 c + 32 j + r is A-row r of the S product for
            // 32-key tile j of 64-key chunk c, and holds key
            // 64 c + 32 ((r >> 2) & 1) + 16 j + 4 (r >> 3) + (r & 3).  In the
            // 32x32 output layout accumulator i of lane (q, h) is A-row
            // 8 (i / 4) + 4 h + (i % 4), so after both tiles of a chunk lane
            // (q, h) holds keys 32 h .. 32 h + 31 of the chunk in order.  The
            // slot is the channel block.  V^: row = channel, slot -> key block
            // (same swizzle).
            const int r = row & 31, j = (row >> 5) & 1, c = row >> 6;
            const int key = 64 * c + 32 * ((r >> 2) & 1) + 16 * j + 4 * (r >> 3) + (r & 3);
            const int db = (p & 3) ^ swz(row);
            koff[it] = (uint32_t)(key * 64 + db * 16);
            voff[it] = (uint32_t)((row * a.nb + db) * 16);
        }
    }

    __device__ __forceinline__ void load(uint8_t* st, int tile_) const {
        // the tile index is wave-uniform; stating it keeps the offsets in
        // scalar registers (a vector one would need a loop per load)
        const int tile = __builtin_amdgcn_readfirstlane(tile_);
#pragma unroll
        for (int it = 0; it < 2; it++) {
            __builtin_amdgcn_raw_ptr_buffer_load_lds(kc, (lds_ptr_t)(st + kKcOff + (2 * wave + it) * 1024), 16,
                                                     (int)koff[it], tile * 8192, 0, 0);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(vc, (lds_ptr_t)(st + kVcOff + (2 * wave + it) * 1024), 16,
                                                     (int)voff[it], tile * 64, 0, 0);
        }
        if (wave == 0)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(sc, (lds_ptr_t)(st + kKsOff), 16, lane * 16, tile * 1024, 0, 0);
    }
};

// Maxima of scores, which are finite or -inf (masked keys), never NaN: the
// NaN-propagating maximum needs no quieting of its operands and fuses into
// the 3-input form.
__device__ __forceinline__ float max2f(float a, float b) { return __builtin_elementwise_maximum(a, b); }
__device__ __forceinline__ float max3f(float a, float b, float c) { return max2f(max2f(a, b), c); }

// Largest of the 32 scores of one P~ block (the lane's 16 + 16 accumulators
// of the two 32-key S products of a chunk): two independent chains.
__device__ __forceinline__ float block_max32(const v16f& a, const v16f& b) {
    float x = max3f(a[0], a[1], a[2]);
    float y = max3f(b[0], b[1], b[2]);
#pragma unroll
    for (int i = 3; i < 15; i += 2) {
        x = max3f(x, a[i], a[i + 1]);
        y = max3f(y, b[i], b[i + 1]);
    }
    return max2f(max3f(x, a[15], b[15]), y);
}

__device__ __forceinline__ float max_with_other_half(float x) {
    // lanes l and l^32 hold the two halves of one query row
    const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, x),
                                                    __builtin_bit_cast(uint32_t, x), false, false);
    return max2f(__builtin_bit_cast(float, (uint32_t)r[0]), __builtin_bit_cast(float, (uint32_t)r[1]));
}

// c * x rounded towards -inf: the round-to-nearest product, stepped one ulp
// down when it exceeds the exact product (the FMA gives the exact residual).
// x is finite.
__device__ __forceinline__ float mul_rd(float c, float x) {
    const float u = c * x;
    const uint32_t ub = __builtin_bit_cast(uint32_t, u);
    // one ulp towards -inf: magnitude down for u > 0, up for u < 0 (and
    // -0 -> the negative denormal); u = +0 never rounds up a negative product
    const uint32_t down = ub - (uint32_t)(((int32_t)ub >> 31) | 1);
    return __builtin_bit_cast(float, __builtin_fmaf(c, x, -u) < 0.f ? down : ub);
}

// E8M0 byte of a P~ block from the bits of its maximum M (0 <= M <= 1 + 2^-20):
// e + 127 = E - 2 under the OCP floor rule and E - 2 + [fraction > 0x680000]
// under UOS (as scale_exponent_f32), where adding 0x17FFFF carries into the
// exponent field exactly when the 23-bit fraction exceeds 0x680000; clamped
// at byte 0 (e >= -127).  A block whose maximum underflowed to 0 holds only
// zeros, so its codes are all zero and its scale affects nothing: it gets
// byte 0 here rather than the 127 of an all-zero input block.
template <int kRule>
__device__ __forceinline__ uint32_t p_scale_byte(uint32_t mbits) {
    const int E = (int)((mbits + (kRule == kRuleUos ? 0x17FFFFu : 0u)) >> 23);
    return (uint32_t)max(E - 2, 0);
}

// LDS reads are ordinary loads from __shared__ arrays.  A lane reads its
// 8-byte scale slot and the two 16-byte slots of row q of a stage (rows
// 32 i + q share q's swizzle); every other row and region is an immediate
// offset of the same per-lane address.
typedef int v4i __attribute__((ext_vector_type(4)));
struct LaneOff {
    uint32_t sc, lo, hi;
};
__device__ __forceinline__ LaneOff lane_off(int q, int h, int lane) {
    return {(uint32_t)(lane * 8), (uint32_t)(q * 64 + 16 * ((0 + h) ^ swz(q))),
            (uint32_t)(q * 64 + 16 * ((2 + h) ^ swz(q)))};
}
template <int kOff>
__device__ __forceinline__ v4i ld128(const uint8_t* stage, uint32_t off) {
    return *reinterpret_cast<const v4i*>(stage + kOff + off);
}
template <int kOff>
__device__ __forceinline__ uint2 ld64(const uint8_t* stage, uint32_t off) {
    return *reinterpret_cast<const uint2*>(stage + kOff + off);
}
__device__ __forceinline__ v8i fp4_v(v4i x) {
    v8i r;
    r[0] = x[0];
    r[1] = x[1];
    r[2] = x[2];
    r[3] = x[3];
    r[4] = 0;
    r[5] = 0;
    r[6] = 0;
    r[7] = 0;
    return r;
}

template <int kScaleOpsel>
__device__ __forceinline__ v16f mfma_fp4(v8i a, v8i b, v16f c, int sa, int sb) {
    return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 4, 4, kScaleOpsel, sa, 0, sb);
}

typedef float v4f __attribute__((ext_vector_type(4)));

// 16x16x128 FP4 product with E8M0 block scales: lane l supplies row (A) or
// column (B) l % 16 for the 32 K-values 32 (l / 16) ... 32 (l / 16) + 31
// and their scale; D row 4 (l / 16) + i, column l % 16 is accumulator i.
__device__ __forceinline__ v4f mfma16_fp4(v8i a, v8i b, v4f c, int sa, int sb) {
    return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 4, 4, 0, sa, 0, sb);
}

// The row sum l.  Direct placement: l is this lane's half of its row's sum
// of P~ (the two halves are added at the end).  PNQ: L accumulates the sum of
// the dequantized P^ on the matrix cores.  Read as a 16x16x128 B operand, the
// P^ registers of a 64-key chunk hold, for column n, K-groups 0..3 = query n
// keys 0-31, query n+16 keys 0-31, query n keys 32-63, query n+16 keys 32-63;
// with FP4 1.0 in row 0 at K-groups 0 and 2 and in row 1 at K-groups 1 and 3
// (row_sum_selector), D row 0 / row 1 of column n is the chunk's sum for
// query n / n + 16.  So lanes 0-15 hold the row sums of the wave's queries
// q (L[0]) and q + 16 (L[1]); L of the other lanes stays 0.
struct RowSum {
    float l;
    v4f L;
};

// The A operand of that product: FP4 1.0 (code 0b0010) in every position of
// row 0 at K-groups 0 and 2 and of row 1 at K-groups 1 and 3, zero elsewhere.
__device__ __forceinline__ v8i row_sum_selector(int lane) {
    const int row = lane & 15, group = lane >> 4;
    const bool one = (row == 0 && (group & 1) == 0) || (row == 1 && (group & 1) == 1);
    v8i r;
#pragma unroll
    for (int i = 0; i < 8; i++) r[i] = (one && i < 4) ? 0x22222222 : 0;
    return r;
}

__device__ __forceinline__ uint32_t cvt_fp4x2(uint32_t old, float a, float b, float scale, int sel) {
    switch (sel) {
        case 0: return __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(old, a, b, scale, 0);
        case 1: return __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(old, a, b, scale, 1);
        case 2: return __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(old, a, b, scale, 2);
        default: return __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(old, a, b, scale, 3);
    }
}

// The Q^ operands of S^T = K^ Q^T for one query row: lane (q, h) holds channel
// blocks h and 2 + h of its query (the B operands of the products over
// channels 0-63 and 64-127) and their E8M0 scales.
struct QOperands {
    v8i b0, b1;
    int s0, s1;
};

// From Q^ quantized beforehand ([BH, Nq, 64] codes, [BH, Nq, 4] scales).
__device__ __forceinline__ QOperands q_operands(const AttnArgs& a, int64_t row, int h) {
    const uint8_t* qrow = a.qc + row * 64;
    return {fp4_operand(*reinterpret_cast<const uint4*>(qrow + 16 * h)),
            fp4_operand(*reinterpret_cast<const uint4*>(qrow + 16 * (2 + h))), (int)a.qs[row * 4 + h],
            (int)a.qs[row * 4 + 2 + h]};
}

// The two bf16 channel blocks (32 values each) of a query row that lane half
// h quantizes itself: channels 32 h .. 32 h + 31 and 64 + 32 h .. 64 + 32 h + 31.
struct QRaw {
    uint4 v[8];
};
__device__ __forceinline__ QRaw q_raw(const AttnArgs& a, int64_t row, int h) {
    const uint4* src = reinterpret_cast<const uint4*>(a.qraw + row * 128);
    QRaw r;
#pragma unroll
    for (int k = 0; k < 4; k++) {
        r.v[k] = src[4 * h + k];
        r.v[4 + k] = src[8 + 4 * h + k];
    }
    return r;
}

// One 32-value block quantized exactly as quantize_headdim_kernel does it
// (Algorithm 1 with the mode's rule): the block maximum on the bf16
// magnitude bits, its E8M0 exponent (an all-zero block gets sigma = 1) and
// the gfx950 FP4 conversion, so the codes are bit-identical to that kernel's.
template <int kRule>
__device__ __forceinline__ v8i quantize_q_block(const uint4* v, int& sbyte) {
    uint32_t m = 0;
#pragma unroll
    for (int k = 0; k < 4; k++) {
        const uint32_t w[4] = {v[k].x, v[k].y, v[k].z, v[k].w};
#pragma unroll
        for (int e = 0; e < 4; e++) m = max(m, max(w[e] & 0x7FFFu, (w[e] >> 16) & 0x7FFFu));
    }
    const uint32_t sb = (m == 0) ? 127u : (uint32_t)(scale_exponent_bf16<kRule>(m) + 127);
    const float sf = e8m0_as_f32(sb);
    uint32_t c[4];
#pragma unroll
    for (int k = 0; k < 4; k++) {
        uint32_t x = 0;
        x = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(x, __builtin_bit_cast(bf16x2, v[k].x), sf, 0);
        x = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(x, __builtin_bit_cast(bf16x2, v[k].y), sf, 1);
        x = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(x, __builtin_bit_cast(bf16x2, v[k].z), sf, 2);
        x = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(x, __builtin_bit_cast(bf16x2, v[k].w), sf, 3);
        c[k] = x;
    }
    sbyte = (int)sb;
    return fp4_operand(make_uint4(c[0], c[1], c[2], c[3]));
}

template <int kRule>
__device__ __forceinline__ QOperands quantize_q(const QRaw& r) {
    QOperands o;
    o.b0 = quantize_q_block<kRule>(r.v, o.s0);
    o.b1 = quantize_q_block<kRule>(r.v + 4, o.s1);
    return o;
}

// Scores of keys at or past the end of the sequence set to -inf: S[c][jj][i]
// is key 64 c + 16 jj + i past the lane's first key, `valid` keys of which
// exist.  Whole-vector integer arithmetic, one bit-field select per score
// (-inf's bits where the key index reaches the limit), so no per-score
// condition masks are held in scalar registers.
typedef int v16i __attribute__((ext_vector_type(16)));
__device__ __forceinline__ void mask_tail(v16f (&S)[2][2], int valid) {
    const v16i idx = {0, 1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 11, 12, 13, 14, 15};
#pragma unroll
    for (int c = 0; c < 2; c++)
#pragma unroll
        for (int jj = 0; jj < 2; jj++) {
            const v16i mk = ((valid - 1 - 64 * c - 16 * jj) - idx) >> 31;  // all ones past the end
            const v16i b = __builtin_bit_cast(v16i, S[c][jj]);
            S[c][jj] = __builtin_bit_cast(v16f, (mk & (int)0xFF800000u) | (~mk & b));
        }
}

// One KV tile of Algorithm 2 for the wave's 32 query rows, read from the LDS
// stage at `st`: S^T = K^ Q^T, the online-softmax update of (m, l), P^ and
// O~^T += V^T P^T.  Reads LDS only; the caller owns loads and barriers.
// kFirst: the row's first tile, which sets m, l and O~ instead of updating
// them (the rescale by alpha = 0 of a zero O~ and l is skipped, and the first
// products accumulate onto zero), so they need no initial values.
template <int kRule, bool kPnq, bool kFirst = false>
__device__ __forceinline__ void attend_tile(const uint8_t* st, const LaneOff& lo, int tile, int N, int h,
                                            const QOperands& qo, const v8i& sel, float& m, RowSum& rs,
                                            v16f (&O)[4]) {
    const float cl = 0.12751743082459868f;  // fp32(log2(e) / sqrt(128))
    const v8i& qB0 = qo.b0;
    const v8i& qB1 = qo.b1;
    const int qS0 = qo.s0, qS1 = qo.s1;
    const uint2 ksb = ld64<kKsOff>(st, lo.sc);
    const uint2 vsb = ld64<kVsOff>(st, lo.sc);

    // ---- K^ operands for the 8 S products (chunk c, tile j, half hf):
    // row 64 c + 32 j + q
    v8i kop[2][2][2];
#pragma unroll
    for (int c = 0; c < 2; c++) {
        kop[c][0][0] = fp4_v(ld128<kKcOff + 0 * 2048>(st + 4096 * c, lo.lo));
        kop[c][0][1] = fp4_v(ld128<kKcOff + 0 * 2048>(st + 4096 * c, lo.hi));
        kop[c][1][0] = fp4_v(ld128<kKcOff + 1 * 2048>(st + 4096 * c, lo.lo));
        kop[c][1][1] = fp4_v(ld128<kKcOff + 1 * 2048>(st + 4096 * c, lo.hi));
    }

    // ---- S^T = K^ Q^T: S[c][j][i] is key 64c + 32h + 16j + i of the tile
    v16f S[2][2];
#pragma unroll
    for (int c = 0; c < 2; c++) {
        const int sreg = c == 0 ? (int)ksb.x : (int)ksb.y;
#pragma unroll
        for (int j = 0; j < 2; j++) {
            v16f acc;
#pragma unroll
            for (int i = 0; i < 16; i++) acc[i] = 0.f;
            if (j == 0) {
                acc = mfma_fp4<0>(kop[c][j][0], qB0, acc, sreg, qS0);
                acc = mfma_fp4<1>(kop[c][j][1], qB1, acc, sreg, qS1);
            } else {
                acc = mfma_fp4<2>(kop[c][j][0], qB0, acc, sreg, qS0);
                acc = mfma_fp4<3>(kop[c][j][1], qB1, acc, sreg, qS1);
            }
            S[c][j] = acc;
        }
    }

    // ---- V^ operands for the PV products (read now, used after softmax):
    // row (channel) 32 n + q
    v8i vop[4][2];
#pragma unroll
    for (int n = 0; n < 4; n++) {
        vop[n][0] = fp4_v(ld128<kVcOff>(st + 2048 * n, lo.lo));
        vop[n][1] = fp4_v(ld128<kVcOff>(st + 2048 * n, lo.hi));
    }

    // ---- mask keys past the end of the sequence (last tile only)
    const int k0 = tile * 128;
    if (k0 + 128 > N) {
#pragma unroll
        for (int c = 0; c < 2; c++)
#pragma unroll
            for (int j = 0; j < 2; j++)
#pragma unroll
                for (int i = 0; i < 16; i++)
                    if (k0 + 64 * c + 32 * h + 16 * j + i >= N) S[c][j][i] = -__builtin_inff();
    }

    // ---- running maximum: the block maxima (one P~ block per lane and
    // chunk), the tile maximum of the row across the lane pair
    float bmax[2];
#pragma unroll
    for (int c = 0; c < 2; c++) bmax[c] = block_max32(S[c][0], S[c][1]);
    float rmax = max_with_other_half(max2f(bmax[0], bmax[1]));
    const float m_new = kFirst ? mul_rd(cl, rmax) : max2f(m, mul_rd(cl, rmax));
    const float alpha = kFirst ? 0.f : __builtin_amdgcn_exp2f(m - m_new);  // 0 on the first tile
    m = m_new;

    // ---- O~^T rescale, then per 64-key chunk: P~ -> P^ and that chunk's PV
    // products (so chunk 0's products run under chunk 1's softmax)
    if (!kFirst && __any(alpha != 1.f)) {
#pragma unroll
        for (int n = 0; n < 4; n++)
#pragma unroll
            for (int i = 0; i < 16; i++) O[n][i] *= alpha;
        if (kPnq) {
            // lane q < 16 holds the sums of queries q and q + 16: the second
            // takes alpha of lane q + 16 (row 1 of the first operand swaps
            // with row 0 of the second)
            const uint32_t ab = __builtin_bit_cast(uint32_t, alpha);
            const auto r = __builtin_amdgcn_permlane16_swap(ab, ab, false, false);
            rs.L[0] *= alpha;
            rs.L[1] *= __builtin_bit_cast(float, (uint32_t)r[1]);
        }
    }
    float lsum = 0.f;
#pragma unroll
    for (int c = 0; c < 2; c++) {
        const float mb = __builtin_amdgcn_exp2f(__builtin_fmaf(bmax[c], cl, -m_new));
        const uint32_t sbyte = p_scale_byte<kRule>(__builtin_bit_cast(uint32_t, mb));
        const float sf = e8m0_as_f32(sbyte);
        const int psc = (int)sbyte;
        uint32_t w[4];
#pragma unroll
        for (int n = 0; n < 32; n += 2) {
            const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(S[c][n >> 4][n & 15], cl, -m_new));
            const float p1 =
                __builtin_amdgcn_exp2f(__builtin_fmaf(S[c][(n + 1) >> 4][(n + 1) & 15], cl, -m_new));
            if (!kPnq) lsum += p0 + p1;
            const uint32_t prev = (n & 7) == 0 ? __builtin_bit_cast(uint32_t, p0) : w[n >> 3];
            w[n >> 3] = cvt_fp4x2(prev, p0, p1, sf, (n & 7) >> 1);
        }
        const v8i P = fp4_operand(make_uint4(w[0], w[1], w[2], w[3]));
        if (kFirst && c == 0) {
            const v16f zero = {};
            if (kPnq) rs.L = mfma16_fp4(sel, P, v4f{0.f, 0.f, 0.f, 0.f}, 127, psc);
            O[0] = mfma_fp4<0>(vop[0][0], P, zero, (int)vsb.x, psc);
            O[1] = mfma_fp4<2>(vop[1][0], P, zero, (int)vsb.x, psc);
            O[2] = mfma_fp4<0>(vop[2][0], P, zero, (int)vsb.y, psc);
            O[3] = mfma_fp4<2>(vop[3][0], P, zero, (int)vsb.y, psc);
            continue;
        }
        if (kPnq) rs.L = mfma16_fp4(sel, P, rs.L, 127, psc);
        // scale byte 2 (n & 1) + c of the register of channel rows 32 n
        if (c == 0) {
            O[0] = mfma_fp4<0>(vop[0][0], P, O[0], (int)vsb.x, psc);
            O[1] = mfma_fp4<2>(vop[1][0], P, O[1], (int)vsb.x, psc);
            O[2] = mfma_fp4<0>(vop[2][0], P, O[2], (int)vsb.y, psc);
            O[3] = mfma_fp4<2>(vop[3][0], P, O[3], (int)vsb.y, psc);
        } else {
            O[0] = mfma_fp4<1>(vop[0][1], P, O[0], (int)vsb.x, psc);
            O[1] = mfma_fp4<3>(vop[1][1], P, O[1], (int)vsb.x, psc);
            O[2] = mfma_fp4<1>(vop[2][1], P, O[2], (int)vsb.y, psc);
            O[3] = mfma_fp4<3>(vop[3][1], P, O[3], (int)vsb.y, psc);
        }
    }
    if (!kPnq) rs.l = kFirst ? lsum : alpha * rs.l + lsum;
}

// O = O~ / l rounded to bf16 (Eq. online_attention_output), as O~ times the
// fp32 reciprocal of l; lane (q, h) holds channels 32 n + 8 g + 4 h + (0..3)
// of its query row.
typedef float f32x2 __attribute__((ext_vector_type(2)));

template <bool kPnq>
__device__ __forceinline__ void store_rows(const AttnArgs& a, int64_t rowbase, int qi, int q, int h, int lane,
                                           uint8_t* stage, bool staged, const RowSum& rs,
                                           const v16f (&O)[4]) {
    float ltot;
    if (kPnq) {
        // the sums of queries q and q + 16 sit in lane q & 15 (RowSum)
        const float l0 = __shfl(rs.L[0], q & 15), l1 = __shfl(rs.L[1], q & 15);
        ltot = q < 16 ? l0 : l1;
    } else {
        ltot = rs.l + __shfl_xor(rs.l, 32);
    }
    const float inv = 1.0f / ltot;  // one division, then 64 products
    // w[n][g]: channels 32 n + 8 g + 4 h .. + 3 of the row as two bf16 pairs
    // (round to nearest even with the packed hardware conversion)
    uint32_t w[4][4][2];
#pragma unroll
    for (int n = 0; n < 4; n++)
#pragma unroll
        for (int g = 0; g < 4; g++) {
            const f32x2 lo = {O[n][4 * g + 0] * inv, O[n][4 * g + 1] * inv};
            const f32x2 hi = {O[n][4 * g + 2] * inv, O[n][4 * g + 3] * inv};
            w[n][g][0] = __builtin_bit_cast(uint32_t, __builtin_convertvector(lo, bf16x2));
            w[n][g][1] = __builtin_bit_cast(uint32_t, __builtin_convertvector(hi, bf16x2));
        }
    // Lanes q and q + 32 hold the row's channel groups 8 g .. 8 g + 7 in
    // halves.  Swapping the lanes 32-63 of the even-g words with the lanes
    // 0-31 of the odd-g words gives lane h all eight channels of group
    // g = 2 j + h, i.e. 16 contiguous bytes per (n, j).
#pragma unroll
    for (int n = 0; n < 4; n++)
#pragma unroll
        for (int j = 0; j < 2; j++)
#pragma unroll
            for (int k = 0; k < 2; k++) {
                const auto r = __builtin_amdgcn_permlane32_swap(w[n][2 * j][k], w[n][2 * j + 1][k], false, false);
                w[n][2 * j][k] = (uint32_t)r[0];
                w[n][2 * j + 1][k] = (uint32_t)r[1];
            }
    if (!staged) {
        if (qi < a.Nq) {
            uint16_t* dst = a.out + (rowbase + qi) * 128 + 8 * h;
#pragma unroll
            for (int n = 0; n < 4; n++)
#pragma unroll
                for (int j = 0; j < 2; j++)
                    *reinterpret_cast<uint4*>(dst + 32 * n + 16 * j) =
                        make_uint4(w[n][2 * j][0], w[n][2 * j][1], w[n][2 * j + 1][0], w[n][2 * j + 1][1]);
        }
        return;
    }
    // Staged: the wave's 32 output rows are contiguous in memory (8 KiB).
    // They go through the wave's 2 KiB LDS buffer 8 rows at a time: the 16
    // lanes of those rows write them in, then every lane copies 2 x 16 bytes
    // out, so each store instruction writes 1 KiB of consecutive rows.  The
    // 16-byte slot of a row is XOR-ed with the row index to spread the writes
    // of the 8 rows over the banks.
    const int q0 = qi - q;  // first row of the wave
#pragma unroll
    for (int pass = 0; pass < 4; pass++) {
        if ((q >> 3) == pass) {
            const int row = q & 7;
#pragma unroll
            for (int n = 0; n < 4; n++)
#pragma unroll
                for (int j = 0; j < 2; j++) {
                    const int slot = (4 * n + 2 * j + h) ^ row;
                    *reinterpret_cast<uint4*>(stage + row * 256 + slot * 16) =
                        make_uint4(w[n][2 * j][0], w[n][2 * j][1], w[n][2 * j + 1][0], w[n][2 * j + 1][1]);
                }
        }
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int k = 0; k < 2; k++) {
            const int byte = 1024 * k + 16 * lane;  // of the 8 rows, 2 KiB
            const int row = byte >> 8, slot = (byte >> 4) & 15;
            const uint4 v = *reinterpret_cast<const uint4*>(stage + row * 256 + (slot ^ row) * 16);
            const int r = q0 + 8 * pass + row;
            if (r < a.Nq) *reinterpret_cast<uint4*>(a.out + (int64_t)(rowbase + r) * 128 + slot * 8) = v;
        }
        __builtin_amdgcn_wave_barrier();
    }
}

// ---------------------------------------------------------------------------
// Long key sequences: the same tile computation, software-pipelined: the
// score products of tile j + 1 are issued during the softmax of tile j (each
// as soon as the score registers it overwrites have been consumed) and the
// second PV chunk of a tile is deferred into the next one, so that no wave
// waits for its own score products before its maximum and no LDS read sits
// right before the product that consumes it.  On video720p this runs as fast
// as a two-stage loop that issues each tile's score products as one group and
// waits for them (the vector-ALU issue rate of the softmax bounds both), with
// results identical bit for bit; it is kept because its LDS reads are
// ordinary loads (see below) and its tail masking holds no per-score masks in
// scalar registers.
//
// Per KV tile j of a wave (stage s = j mod 3 holds tile j's K^, V^ and scales):
//   A  read tile j-1's chunk-1 V^ operands; block and row maxima of S(j),
//      the running maximum and alpha.
//   B  wait for tile j+1's loads, barrier, start tile j+2's loads (into the
//      stage of tile j-1, read for the last time in A); tile j-1's deferred
//      chunk-1 products (O~ += V^ P^ and the PNQ row sum) threaded through
//      the first half of chunk 0's softmax; then the rescale of O~ and l by
//      alpha.
//   C  the rest of chunk 0, its products with V^ threaded through chunk 1's
//      softmax, and the score products of tile j+1, each issued as soon as
//      the score registers it overwrites have been consumed.
// Every accumulator still receives its terms in the same order as in
// attend_tile (O~: chunk 0 then chunk 1 of each tile, then the next tile's
// rescale), so the results are identical.
//
// The three stages are separate LDS arrays read by ordinary loads, so the
// compiler orders them against the buffer-to-LDS copies by their arrays
// (a read of one stage never waits for the copies into another).
constexpr int kPipeStages = 3;

// The K^ operands of the score products of one tile in `stage`: rows
// 64 c + 32 jj + q, channel blocks h (lo) and 2 + h (hi).
struct KOperands {
    v4i lo[2][2], hi[2][2];
};
__device__ __forceinline__ KOperands k_operands(const uint8_t* stage, const LaneOff& lo) {
    KOperands k;
    k.lo[0][0] = ld128<kKcOff + 0 * 2048>(stage, lo.lo);
    k.hi[0][0] = ld128<kKcOff + 0 * 2048>(stage, lo.hi);
    k.lo[0][1] = ld128<kKcOff + 1 * 2048>(stage, lo.lo);
    k.hi[0][1] = ld128<kKcOff + 1 * 2048>(stage, lo.hi);
    k.lo[1][0] = ld128<kKcOff + 2 * 2048>(stage, lo.lo);
    k.hi[1][0] = ld128<kKcOff + 2 * 2048>(stage, lo.hi);
    k.lo[1][1] = ld128<kKcOff + 3 * 2048>(stage, lo.lo);
    k.hi[1][1] = ld128<kKcOff + 3 * 2048>(stage, lo.hi);
    return k;
}

// The two score products of S[c][jj] (keys 64 c + 32 h + 16 jj + i of the
// tile).
template <int kC, int kJ>
__device__ __forceinline__ v16f score_pair(const KOperands& k, const QOperands& qo, uint2 ksb) {
    const int sreg = kC == 0 ? (int)ksb.x : (int)ksb.y;
    const v16f zero = {};
    v16f acc = mfma_fp4<2 * kJ>(fp4_v(k.lo[kC][kJ]), qo.b0, zero, sreg, qo.s0);
    return mfma_fp4<2 * kJ + 1>(fp4_v(k.hi[kC][kJ]), qo.b1, acc, sreg, qo.s1);
}

// The V^ operands of chunk kC of a tile in `stage` (channel rows 32 n + q).
struct VOperands {
    v4i v[4];
};
template <int kC>
__device__ __forceinline__ VOperands v_operands(const uint8_t* stage, const LaneOff& lo) {
    const uint32_t off = kC == 0 ? lo.lo : lo.hi;
    return {{ld128<kVcOff + 0 * 2048>(stage, off), ld128<kVcOff + 1 * 2048>(stage, off),
             ld128<kVcOff + 2 * 2048>(stage, off), ld128<kVcOff + 3 * 2048>(stage, off)}};
}

// O~ += V^ P^ for chunk kC of a tile, and the PNQ row sum of that chunk.
template <bool kPnq, int kC>
__device__ __forceinline__ void pv_chunk(const VOperands& vo, const v8i& P, int psc, uint2 vsb, const v8i& sel,
                                         RowSum& rs, v16f (&O)[4]) {
    if (kPnq) rs.L = mfma16_fp4(sel, P, rs.L, 127, psc);
    O[0] = mfma_fp4<kC>(fp4_v(vo.v[0]), P, O[0], (int)vsb.x, psc);
    O[1] = mfma_fp4<2 + kC>(fp4_v(vo.v[1]), P, O[1], (int)vsb.x, psc);
    O[2] = mfma_fp4<kC>(fp4_v(vo.v[2]), P, O[2], (int)vsb.y, psc);
    O[3] = mfma_fp4<2 + kC>(fp4_v(vo.v[3]), P, O[3], (int)vsb.y, psc);
}

// P~ of one 32-key block (this lane's S[c][0] and S[c][1]) -> its E8M0 byte
// and FP4 codes; the direct placement's row sum of P~ is added to lsum.
template <int kRule, bool kPnq, int kHalf>
__device__ __forceinline__ void softmax_half(const v16f& Sh, float m_new, float sf, uint32_t (&w)[4],
                                             float& lsum) {
    const float cl = 0.12751743082459868f;  // fp32(log2(e) / sqrt(128))
#pragma unroll
    for (int n = 0; n < 16; n += 2) {
        const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(Sh[n], cl, -m_new));
        const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(Sh[n + 1], cl, -m_new));
        if (!kPnq) lsum += p0 + p1;
        const int k = 16 * kHalf + n;  // key within the block
        const uint32_t prev = (k & 7) == 0 ? __builtin_bit_cast(uint32_t, p0) : w[k >> 3];
        w[k >> 3] = cvt_fp4x2(prev, p0, p1, sf, (k & 7) >> 1);
    }
}

template <int kRule>
__device__ __forceinline__ uint32_t block_scale(float bmax, float m_new) {
    const float cl = 0.12751743082459868f;
    const float mb = __builtin_amdgcn_exp2f(__builtin_fmaf(bmax, cl, -m_new));
    return p_scale_byte<kRule>(__builtin_bit_cast(uint32_t, mb));
}

// State a wave carries from one KV tile to the next.
struct PipeState {
    v16f S[2][2];  // scores of the current tile
    v16f O[4];
    RowSum rs;
    float m;
    v8i P1;        // P^ of the previous tile's chunk 1 (its products are deferred)
    int psc1;
    uint2 vsb1;    // V^ scales of the previous tile
};

// Keeps the computation of its operands ahead of this point: an empty asm
// statement that takes them as inputs (no instruction is emitted).  It stops
// the compiler from sinking work past a branch into the block that uses it
// (the exponentials of a chunk past the rescale branch, the next tile's score
// products past the loop exit), which would regroup the products.  Operands
// written by matrix-core products are named only to place the product's
// issue, never read.
template <typename T>
__device__ __forceinline__ void pin_one(const T& x) {
    asm volatile("" ::"v"(x));
}
template <typename... T>
__device__ __forceinline__ void pin_here(const T&... x) {
    (pin_one(x), ...);
}

// One KV tile j in stage kS: see the description above.  Stages kS + 1 and
// kS + 2 (mod 3) hold tiles j + 1 and j - 1.
template <int kRule, bool kPnq, int kS>
__device__ __forceinline__ void pipe_tile(uint8_t* const (&stages)[kPipeStages], const TileLoader& loader,
                                          const LaneOff& lo, int j, int ntiles, int N, int h, const QOperands& qo,
                                          const v8i& sel, PipeState& ps) {
    const float cl = 0.12751743082459868f;
    const uint8_t* cur = stages[kS];
    const uint8_t* nxt = stages[(kS + 1) % kPipeStages];
    const uint8_t* prv = stages[(kS + 2) % kPipeStages];

    // ---- A: tile j-1's chunk-1 V^ operands (its stage is reloaded after the
    // barrier below), the maxima of S(j), the running maximum and alpha
    const VOperands vprev = v_operands<1>(prv, lo);
    const int k0 = j * 128;
    if (k0 + 128 > N) mask_tail(ps.S, N - k0 - 32 * h);
    float bmax[2];
#pragma unroll
    for (int c = 0; c < 2; c++) bmax[c] = block_max32(ps.S[c][0], ps.S[c][1]);
    const float rmax = max_with_other_half(max2f(bmax[0], bmax[1]));
    const float m_new = max2f(ps.m, mul_rd(cl, rmax));
    const float alpha = __builtin_amdgcn_exp2f(ps.m - m_new);  // 0 on the first tile
    ps.m = m_new;

    // ---- B: tile j+1 landed everywhere, and every wave has read tile j-1's
    // stage for the last time, so it takes tile j+2
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (j + 2 < ntiles) loader.load(stages[(kS + 2) % kPipeStages], j + 2);

    // region 1: every LDS read of the rest of the tile; tile j-1's chunk-1
    // products (on the first tile P^ = 0 with finite scales, which adds
    // exactly zero) under chunk 0's first half, then the first score
    // products of tile j+1 into the registers that half freed.  Each score
    // pair of tile j+1 is issued as soon as the softmax has consumed the
    // scores it overwrites, which spreads the products evenly over the
    // tile's vector work (issuing them in two groups of four was slower).
    // After the last tile, the
    // score products read a stage that holds an older tile (every stage is
    // in bounds) and their results are unused: 8 products per query tile, in
    // exchange for branch-free tile code.
    const uint2 vsb = ld64<kVsOff>(cur, lo.sc);
    const uint2 ksb = ld64<kKsOff>(nxt, lo.sc);
    const KOperands kn = k_operands(nxt, lo);
    const VOperands vc0 = v_operands<0>(cur, lo);
    pv_chunk<kPnq, 1>(vprev, ps.P1, ps.psc1, ps.vsb1, sel, ps.rs, ps.O);
    float lsum = 0.f;
    uint32_t w0[4], w1[4];
    const uint32_t sb0 = block_scale<kRule>(bmax[0], m_new);
    const float sf0 = e8m0_as_f32(sb0);
    softmax_half<kRule, kPnq, 0>(ps.S[0][0], m_new, sf0, w0, lsum);
    ps.S[0][0] = score_pair<0, 0>(kn, qo, ksb);
    pin_here(ps.S[0][0][0], w0[0], w0[1], lsum, ps.O[0][0], ps.O[1][0], ps.O[2][0], ps.O[3][0], ps.rs.L[0], ksb,
             vsb, kn.lo[0][0], kn.hi[0][0], kn.lo[0][1], kn.hi[0][1], kn.lo[1][0], kn.hi[1][0], kn.lo[1][1],
             kn.hi[1][1], vc0.v[0], vc0.v[1], vc0.v[2], vc0.v[3]);

    // the rescale of O~ and l by alpha follows the products above
    if (__any(alpha != 1.f)) {
#pragma unroll
        for (int n = 0; n < 4; n++)
#pragma unroll
            for (int i = 0; i < 16; i++) ps.O[n][i] *= alpha;
        if (kPnq) {
            const uint32_t ab = __builtin_bit_cast(uint32_t, alpha);
            const auto r = __builtin_amdgcn_permlane16_swap(ab, ab, false, false);
            ps.rs.L[0] *= alpha;
            ps.rs.L[1] *= __builtin_bit_cast(float, (uint32_t)r[1]);
        }
    }

    // region 2: the rest of chunk 0, chunk 0's products, chunk 1, with the
    // score products of tile j+1 issued as score registers become free
    softmax_half<kRule, kPnq, 1>(ps.S[0][1], m_new, sf0, w0, lsum);
    ps.S[0][1] = score_pair<0, 1>(kn, qo, ksb);
    const v8i P0 = fp4_operand(make_uint4(w0[0], w0[1], w0[2], w0[3]));
    pv_chunk<kPnq, 0>(vc0, P0, (int)sb0, vsb, sel, ps.rs, ps.O);
    const uint32_t sb1 = block_scale<kRule>(bmax[1], m_new);
    const float sf1 = e8m0_as_f32(sb1);
    softmax_half<kRule, kPnq, 0>(ps.S[1][0], m_new, sf1, w1, lsum);
    ps.S[1][0] = score_pair<1, 0>(kn, qo, ksb);
    pin_here(ps.S[1][0][0], w1[0], w1[1]);
    softmax_half<kRule, kPnq, 1>(ps.S[1][1], m_new, sf1, w1, lsum);
    ps.S[1][1] = score_pair<1, 1>(kn, qo, ksb);
    pin_here(ps.S[0][0][0], ps.S[0][1][0], ps.S[1][0][0], ps.S[1][1][0], ps.O[0][0], ps.O[1][0], ps.O[2][0],
             ps.O[3][0]);
    ps.P1 = fp4_operand(make_uint4(w1[0], w1[1], w1[2], w1[3]));
    ps.psc1 = (int)sb1;
    ps.vsb1 = vsb;
    if (!kPnq) ps.rs.l = alpha * ps.rs.l + lsum;
}

template <int kRule, bool kPnq, bool kQraw>
__global__ __launch_bounds__(kThreads, 2) void attention_pipelined_kernel(AttnArgs a) {
    __shared__ __attribute__((aligned(16))) uint8_t st0[kStageBytes];
    __shared__ __attribute__((aligned(16))) uint8_t st1[kStageBytes];
    __shared__ __attribute__((aligned(16))) uint8_t st2[kStageBytes];
    uint8_t* const stages[kPipeStages] = {st0, st1, st2};
    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63;
    const int q = lane & 31, h = lane >> 5;

    const int L = blockIdx.x;
    const int logical = (L & 7) * a.per_xcd + (L >> 3);
    if (logical >= a.total_tiles) return;
    const int bh = logical / a.qtiles;
    const int qt = logical - bh * a.qtiles;
    const int N = a.N;
    const int Nq = a.Nq;
    const int64_t rowbase = (int64_t)bh * Nq;
    const int qi = qt * kQueryTile + wave * kQw + q;
    const int qic = min(qi, Nq - 1);
    const int ntiles = (N + 127) / 128;

    const TileLoader loader(a, bh, wave, lane);
    loader.load(st0, 0);
    if (ntiles > 1) loader.load(st1, 1);

    QOperands qo;
    if constexpr (kQraw)
        qo = quantize_q<kRule>(q_raw(a, rowbase + qic, h));
    else
        qo = q_operands(a, rowbase + qic, h);
    const v8i sel = row_sum_selector(lane);
    const LaneOff lo = lane_off(q, h, lane);

    PipeState ps;
    ps.m = -__builtin_inff();
    ps.rs.l = 0.f;
    ps.rs.L = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int n = 0; n < 4; n++)
#pragma unroll
        for (int i = 0; i < 16; i++) ps.O[n][i] = 0.f;
    // the deferred products of "tile -1": P^ = 0 with finite scales
    ps.P1 = v8i{};
    ps.psc1 = 127;
    ps.vsb1 = make_uint2(0x7F7F7F7Fu, 0x7F7F7F7Fu);

    __builtin_amdgcn_s_waitcnt(0);  // tiles 0 and 1 landed
    __syncthreads();
    {
        const uint2 ksb = ld64<kKsOff>(st0, lo.sc);
        const KOperands k0 = k_operands(st0, lo);
        ps.S[0][0] = score_pair<0, 0>(k0, qo, ksb);
        ps.S[0][1] = score_pair<0, 1>(k0, qo, ksb);
        ps.S[1][0] = score_pair<1, 0>(k0, qo, ksb);
        ps.S[1][1] = score_pair<1, 1>(k0, qo, ksb);
    }
    for (int j = 0;; j += 3) {
        pipe_tile<kRule, kPnq, 0>(stages, loader, lo, j, ntiles, N, h, qo, sel, ps);
        if (j + 1 >= ntiles) break;
        pipe_tile<kRule, kPnq, 1>(stages, loader, lo, j + 1, ntiles, N, h, qo, sel, ps);
        if (j + 2 >= ntiles) break;
        pipe_tile<kRule, kPnq, 2>(stages, loader, lo, j + 2, ntiles, N, h, qo, sel, ps);
        if (j + 3 >= ntiles) break;
    }
    // the last tile's chunk-1 products (its stage is (ntiles - 1) mod 3)
    const int last = (ntiles - 1) % kPipeStages;
    pv_chunk<kPnq, 1>(v_operands<1>(last == 0 ? st0 : (last == 1 ? st1 : st2), lo), ps.P1, ps.psc1, ps.vsb1, sel,
                      ps.rs, ps.O);

    store_rows<kPnq>(a, rowbase, qi, q, h, lane, nullptr, false, ps.rs, ps.O);
}

// Short key sequences (cross-attention over a text context, at most
// kResidentKeys keys): the workgroup copies all of the head's K^ and V^ tiles
// into LDS once and then runs several query tiles of that head against them,
// with no per-tile loads or barriers; each query tile is the same computation
// as in the streaming kernel.
constexpr int kResidentTiles = kResidentKeys / 128;
static_assert(kStagedStoreMaxTiles < kResidentTiles && kWaves * kOutStageBytes <= kStageBytes,
              "the output staging buffers fit in an unused tile slot");

template <int kRule, bool kPnq, bool kQraw>
__global__ __launch_bounds__(kThreads, 2) void attention_resident_kernel(AttnArgs a) {
    __shared__ __attribute__((aligned(16))) uint8_t lds[kResidentTiles * kStageBytes];
    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63;
    const int q = lane & 31, h = lane >> 5;

    const int L = blockIdx.x;
    const int logical = (L & 7) * a.per_xcd + (L >> 3);
    if (logical >= a.total_tiles) return;
    const int bh = logical / a.nchunks;
    const int chunk = logical - bh * a.nchunks;
    // the head's query tiles split as evenly as possible over nchunks
    const int qt0 = (int)((int64_t)chunk * a.qtiles / a.nchunks);
    const int qt1 = (int)((int64_t)(chunk + 1) * a.qtiles / a.nchunks);
    const int N = a.N;
    const int Nq = a.Nq;
    const int64_t rowbase = (int64_t)bh * Nq;
    const int ntiles = (N + 127) / 128;
    // staging goes to the first unused tile slot
    const bool staged = ntiles <= kStagedStoreMaxTiles;
    uint8_t* const ostage = lds + ntiles * kStageBytes + wave * kOutStageBytes;

    const TileLoader loader(a, bh, wave, lane);
    for (int t = 0; t < ntiles; t++) loader.load(lds + t * kStageBytes, t);

    const v8i sel = row_sum_selector(lane);
    const LaneOff lo = lane_off(q, h, lane);

    __builtin_amdgcn_s_waitcnt(0);  // this wave's direct LDS loads landed
    __syncthreads();                // and every other wave's

    // the Q^ operands (or the bf16 rows to quantize) of the first query tile;
    // each later one is fetched while the previous tile is processed
    auto q_row = [&](int qt) { return rowbase + min(qt * kQueryTile + wave * kQw + q, Nq - 1); };
    using QFetch = std::conditional_t<kQraw, QRaw, QOperands>;
    auto fetch = [&](int qt) -> QFetch {
        if constexpr (kQraw)
            return q_raw(a, q_row(qt), h);
        else
            return q_operands(a, q_row(qt), h);
    };
    // The next query tile's operands are formed from its fetched rows before
    // this tile's output stores are issued.  vmcnt counts loads and stores
    // alike and the number of stores is not static (row guards, staging), so a
    // wait for the fetched registers placed after the stores would wait for
    // the stores as well, once per query tile.  Quantized operands are read
    // by an empty asm statement to pin that wait before the stores; raw rows
    // are read by their quantization.
    auto operands = [&](QFetch f) -> QOperands {
        if constexpr (kQraw) {
            return quantize_q<kRule>(f);
        } else {
            asm volatile("" : "+v"(f.b0), "+v"(f.b1), "+v"(f.s0), "+v"(f.s1));
            return f;
        }
    };
    QOperands qo = operands(fetch(qt0));

    for (int qt = qt0; qt < qt1; qt++) {
        const int qi = qt * kQueryTile + wave * kQw + q;
        // the last query tile fetches itself again: no branch around the loads
        const QFetch next = fetch(min(qt + 1, qt1 - 1));

        // set by the first tile (N >= 1, so there is one)
        float m;
        RowSum rs;
        v16f O[4];
        attend_tile<kRule, kPnq, true>(lds, lo, 0, N, h, qo, sel, m, rs, O);
        for (int tile = 1; tile < ntiles; tile++)
            attend_tile<kRule, kPnq>(lds + tile * kStageBytes, lo, tile, N, h, qo, sel, m, rs, O);

        const QOperands qn = operands(next);
        store_rows<kPnq>(a, rowbase, qi, q, h, lane, ostage, staged, rs, O);
        qo = qn;
    }
}

}  // namespace

// E8M0 scales of K^ ([BH, N, 4]) and V^ ([BH, 128, nb]) rearranged into the
// order of the attention kernel's MFMA scale operands: per head and 128-key
// tile, 512 bytes of K^ scales then 512 bytes of V^ scales, 8 bytes per lane.
// K^: lane r + 32*(db&1), byte 4c + 2j + (db>>1) holds the scale of channel
// block db of the key in A-row r of S product (chunk c, tile j).  V^: lane
// (d&31) + 32*(kb&1), byte 2*(d>>5) + (kb>>1) holds the scale of channel d,
// key block kb of the tile.  Keys past N repeat key N-1 and blocks past the
// end repeat the last block, as the code loads do.
__global__ __launch_bounds__(256) void tile_scales_kernel(const uint8_t* __restrict__ ks,
                                                          const uint8_t* __restrict__ vs,
                                                          uint8_t* __restrict__ out, int N, int nb,
                                                          int ntiles, int64_t total) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;  // (head, tile, K|V, lane)
    if (i >= total) return;
    const int L = (int)(i & 63);
    const int half = (int)((i >> 6) & 1);
    const int64_t ht = i >> 7;
    const int t = (int)(ht % ntiles);
    const int64_t bh = ht / ntiles;
    uint32_t lo = 0, hi = 0;
#pragma unroll
    for (int e = 0; e < 8; e++) {
        uint32_t b;
        if (half == 0) {
            const int r = L & 31, c = e >> 2, j = (e >> 1) & 1, db = 2 * (e & 1) + (L >> 5);
            const int w = (r & 3) | ((r >> 3) << 2) | (j << 4) | (((r >> 2) & 1) << 5);
            const int key = min(t * 128 + 64 * c + w, N - 1);
            b = ks[(bh * N + key) * 4 + db];
        } else {
            const int d = 32 * (e >> 1) + (L & 31), kb = 2 * (e & 1) + (L >> 5);
            b = vs[(bh * 128 + d) * nb + min(4 * t + kb, nb - 1)];
        }
        if (e < 4)
            lo |= b << (8 * e);
        else
            hi |= b << (8 * (e - 4));
    }
    *reinterpret_cast<uint2*>(out + ht * 1024 + half * 512 + L * 8) = make_uint2(lo, hi);
}

hipError_t launch_tile_scales(const uint8_t* ks, const uint8_t* vs, uint8_t* out, int64_t BH, int64_t N,
                              hipStream_t stream) {
    const int ntiles = (int)((N + 127) / 128);
    const int64_t total = BH * ntiles * 128;
    const dim3 grid((unsigned)((total + 255) / 256));
    tile_scales_kernel<<<grid, 256, 0, stream>>>(ks, vs, out, (int)N, (int)((N + 31) / 32), ntiles, total);
    return hipGetLastError();
}

template <bool kQraw>
static void launch_attention_q(const AttnArgs& a, int mode, dim3 grid, hipStream_t stream) {
    if (a.N <= kResidentKeys) {
        switch (mode) {
            case 0: attention_resident_kernel<kRuleOcp, false, kQraw><<<grid, kThreads, 0, stream>>>(a); break;
            case 1: attention_resident_kernel<kRuleUos, false, kQraw><<<grid, kThreads, 0, stream>>>(a); break;
            default: attention_resident_kernel<kRuleUos, true, kQraw><<<grid, kThreads, 0, stream>>>(a); break;
        }
        return;
    }
    switch (mode) {
        case 0: attention_pipelined_kernel<kRuleOcp, false, kQraw><<<grid, kThreads, 0, stream>>>(a); break;
        case 1: attention_pipelined_kernel<kRuleUos, false, kQraw><<<grid, kThreads, 0, stream>>>(a); break;
        default: attention_pipelined_kernel<kRuleUos, true, kQraw><<<grid, kThreads, 0, stream>>>(a); break;
    }
}

hipError_t launch_attention(const AttnArgs& a, int mode, hipStream_t stream) {
    const dim3 grid((unsigned)(8 * a.per_xcd));
    if (a.qraw)
        launch_attention_q<true>(a, mode, grid, stream);
    else
        launch_attention_q<false>(a, mode, grid, stream);
    return hipGetLastError();
}

}  // namespace mxattn
