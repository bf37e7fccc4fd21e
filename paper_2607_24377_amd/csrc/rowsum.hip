// rowsum.hip -- row-sum diagnostics of MXFP4-quantized attention
// probabilities for gfx950 (Sec. 5.5, "Validation of Pre-Normalization
// Quantization", Fig. pnq_rowsum).
//
// The paper measures what direct MXFP4 quantization does to the mass of each
// row of a materialized probability matrix P = softmax(Q K^T / sqrt(d)).  Two
// kernels:
//
//   attn_rows_kernel    S^T on the bf16 matrix cores (V_MFMA_F32_32X32X16_BF16,
//                       fp32 accumulation), then two passes over the keys: the
//                       first for each row's maximum and normalizer, the
//                       second forming p = 2^(t - m) / L in fp32 and either
//                       storing it (a materialized tile of P) or quantizing it
//                       in 32-key blocks in registers and accumulating the
//                       row statistics below, so that whole tensors are
//                       diagnosed without writing P;
//   rowsum_diag_kernel  the statistics of a given fp32 P: each row quantized
//                       in 32-entry blocks (optionally pre-scaled by gamma),
//                       reduced to the quantized mass, the unquantized mass,
//                       the contributions Q(x)/gamma - p of zeroed,
//                       saturated, rounded-down, rounded-up and exact
//                       entries, and the entropy -sum p ln p.
//
// Both quantize with the same per-entry arithmetic (diag_add), so on the same
// p they classify every entry identically and their fp64 sums differ only in
// the order of additions.  rowsum_diag_kernel is HBM-bound (4 bytes of P per
// entry read once); attn_rows_kernel in its diagnostic form reads only Q and
// K and is bound by the two score passes and the per-entry VALU work.
#include <cmath>

#include "device_common.h"
#include "launch.h"

namespace mxattn {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kRowsPerWg = 128;   // query rows per softmax workgroup (4 waves x 32)
constexpr int kKeyTile = 128;     // keys staged in LDS per step
constexpr int kLdsRow = 272;      // bytes per staged key row (256 + 16 of padding)
constexpr float kNegBig = -3.0e38f;

// Stage keys [tile * 128, tile * 128 + 128) of one head into LDS (zeros past Nkv).
__device__ __forceinline__ void stage_keys(uint8_t* lds, const uint4* kh, int tile, int Nkv) {
#pragma unroll
    for (int it = 0; it < 8; it++) {
        const int c = threadIdx.x + 256 * it;  // 16-byte chunk of the tile
        const int key = c >> 4, part = c & 15;
        const int gk = tile * kKeyTile + key;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (gk < Nkv) v = kh[(int64_t)gk * 16 + part];
        *reinterpret_cast<uint4*>(lds + key * kLdsRow + part * 16) = v;
    }
}

// S^T for 32 keys (sub-tile j of the staged tile, as A rows) x 32 queries
// (this wave's, as B columns): lane (col, h) supplies key 32 j + col and query
// col, each with channels 16 s + 8 h .. + 7 per 16-channel step s.
__device__ __forceinline__ v16f scores_t(const bf16x8* qb, const uint8_t* lds, int j, int col, int h) {
    v16f acc;
#pragma unroll
    for (int i = 0; i < 16; i++) acc[i] = 0.f;
    const uint8_t* row = lds + (32 * j + col) * kLdsRow + 16 * h;
#pragma unroll
    for (int s = 0; s < 8; s++) {
        const bf16x8 ka = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(row + 32 * s));
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qb[s], acc, 0, 0, 0);
    }
    return acc;
}

// Accumulator i of lane (col, h) holds the score of query col with key
// (A row) 8 (i / 4) + 4 h + (i % 4) of the 32-key sub-tile: a lane holds 16
// of the 32 keys of its query, its partner lane col + 32 (1 - 2h) the rest.
__device__ __forceinline__ int acc_key(int i, int h) { return 8 * (i >> 2) + 4 * h + (i & 3); }

// log2 of a positive fp32, subnormals included (the hardware logarithm takes
// them as zero): a subnormal is scaled by 2^32 into the normal range first.
__device__ __forceinline__ float log2_full(float p) {
    return p < 1.17549435e-38f ? __builtin_amdgcn_logf(p * 4294967296.0f) - 32.0f : __builtin_amdgcn_logf(p);
}

// Adds one entry's terms to the row statistics (see mxattn.h): p the
// probability, xs = gamma p / sigma (exact), r its E2M1 value from the
// 4-bit code, sig = sigma in fp64, g = fp64(1 / gamma).
__device__ __forceinline__ void diag_add(double* st, float p, float xs, float r, uint32_t code,
                                         double sig, double g) {
    const double pd = (double)p;
    const double qv = (double)r * sig * g;
    const double cj = qv - pd;
    const bool zer = p > 0.f && (code & 7u) == 0u;
    const bool sat = !zer && xs > 6.0f;
    const bool dn = !zer && !sat && r < xs;
    const bool up = !zer && !sat && r > xs;
    const bool ex = !zer && !sat && !dn && !up;
    st[0] += qv;
    st[1] += pd;
    st[2] += zer ? cj : 0.0;
    st[3] += sat ? cj : 0.0;
    st[4] += dn ? cj : 0.0;
    st[5] += up ? cj : 0.0;
    st[6] += ex ? cj : 0.0;
    st[7] += p > 0.f ? (double)(p * log2_full(p)) : 0.0;  // p log2 p; scaled by -ln 2 at the end
}

// Shared-scale exponent of a block from the bits of its largest magnitude.
template <int kRule>
__device__ __forceinline__ int block_exponent_f32(uint32_t mb) {
    return mb == 0 ? 0 : scale_exponent_f32<kRule>(mb);
}

// Rows of attention probabilities: S^T on the bf16 matrix cores, pass 1 the
// row maximum m and normalizer L of t = s c, pass 2 p = 2^(t - m) / L, then
// kOut = 0: p stored as fp32 rows; kOut = 1 (UOS) or 2 (OCP): p quantized in
// 32-key blocks in registers and the row statistics of rowsum_diag_kernel
// accumulated, so the diagnostic of a whole tensor never materializes P.
template <int kOut>
__global__ __launch_bounds__(256) void attn_rows_kernel(SoftmaxRowsArgs a) {
    __shared__ __attribute__((aligned(16))) uint8_t lds[kKeyTile * kLdsRow];
    const int bh = blockIdx.x / a.qtiles, qt = blockIdx.x % a.qtiles;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int col = lane & 31, h = lane >> 5;
    const int lr = qt * kRowsPerWg + 32 * wave + col;  // this lane's local query row
    const bool row_ok = lr < a.rows;

    // Q operand (B columns): query row lr (clamped; only valid rows are written)
    const int lq = min(lr, a.rows - 1);
    const uint4* qrow = reinterpret_cast<const uint4*>(a.q) + ((int64_t)bh * a.Nq + a.row0 + lq) * 16;
    bf16x8 qb[8];
#pragma unroll
    for (int s = 0; s < 8; s++) qb[s] = __builtin_bit_cast(bf16x8, qrow[2 * s + h]);

    const uint4* kh = reinterpret_cast<const uint4*>(a.k) + (int64_t)bh * a.Nkv * 16;
    const int tiles = (a.Nkv + kKeyTile - 1) / kKeyTile;

    // pass 1: running maximum and normalizer of this lane's 16-key shares
    float m = kNegBig, l = 0.f;
    for (int t = 0; t < tiles; t++) {
        __syncthreads();
        stage_keys(lds, kh, t, a.Nkv);
        __syncthreads();
        v16f sv[4];
#pragma unroll
        for (int j = 0; j < 4; j++) sv[j] = scores_t(qb, lds, j, col, h);
        float tm = kNegBig;
#pragma unroll
        for (int j = 0; j < 4; j++)
#pragma unroll
            for (int i = 0; i < 16; i++) {
                const bool valid = t * kKeyTile + 32 * j + acc_key(i, h) < a.Nkv;
                sv[j][i] = valid ? sv[j][i] * a.c : -INFINITY;
                tm = fmaxf(tm, sv[j][i]);
            }
        const float mn = fmaxf(m, tm);
        float acc = l * __builtin_amdgcn_exp2f(m - mn);
#pragma unroll
        for (int j = 0; j < 4; j++)
#pragma unroll
            for (int i = 0; i < 16; i++) acc += __builtin_amdgcn_exp2f(sv[j][i] - mn);
        m = mn;
        l = acc;
    }
    {  // the two halves of the row
        const float mo = __shfl_xor(m, 32);
        const float lo = __shfl_xor(l, 32);
        const float mn = fmaxf(m, mo);
        l = l * __builtin_amdgcn_exp2f(m - mn) + lo * __builtin_amdgcn_exp2f(mo - mn);
        m = mn;
    }
    const float inv = 1.0f / l;

    double st[8];
#pragma unroll
    for (int i = 0; i < 8; i++) st[i] = 0.0;

    // pass 2
    for (int t = 0; t < tiles; t++) {
        __syncthreads();
        stage_keys(lds, kh, t, a.Nkv);
        __syncthreads();
#pragma unroll
        for (int j = 0; j < 4; j++) {
            const v16f sv = scores_t(qb, lds, j, col, h);
            const int key0 = t * kKeyTile + 32 * j;
            float p[16];
#pragma unroll
            for (int i = 0; i < 16; i++)
                p[i] = key0 + acc_key(i, h) < a.Nkv ? __builtin_amdgcn_exp2f(sv[i] * a.c - m) * inv : 0.f;
            if constexpr (kOut == 0) {
                // keys key0 + 8 (i/4) + 4 h + 0..3 as one 16-byte store each
                if (row_ok) {
                    float* prow = a.p + ((int64_t)bh * a.rows + lr) * a.ld;
#pragma unroll
                    for (int g = 0; g < 4; g++) {
                        const int key = key0 + 8 * g + 4 * h;
                        if (key < a.Nkv)
                            *reinterpret_cast<float4*>(prow + key) =
                                make_float4(p[4 * g], p[4 * g + 1], p[4 * g + 2], p[4 * g + 3]);
                    }
                }
            } else {
                constexpr int kRule = kOut == 1 ? kRuleUos : kRuleOcp;
                float x[16];
                uint32_t mb = 0;
#pragma unroll
                for (int i = 0; i < 16; i++) {
                    x[i] = a.gamma * p[i];
                    mb = max(mb, __builtin_bit_cast(uint32_t, x[i]) & 0x7FFFFFFFu);
                }
                mb = max(mb, (uint32_t)__shfl_xor((int)mb, 32));  // the block's other 16 keys
                const int ex = block_exponent_f32<kRule>(mb);
                const float sf = e8m0_as_f32((uint32_t)(ex + 127));
                const float invs = __builtin_bit_cast(float, (uint32_t)(127 - ex) << 23);
                const double sig = __builtin_bit_cast(double, (uint64_t)(ex + 1023) << 52);
#pragma unroll
                for (int i = 0; i < 16; i += 2) {
                    const uint32_t c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, x[i], x[i + 1], sf, 0);
                    const auto r = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(c, 1.0f, 0);
                    diag_add(st, p[i], x[i] * invs, r[0], c & 0xFu, sig, a.g);
                    diag_add(st, p[i + 1], x[i + 1] * invs, r[1], (c >> 4) & 0xFu, sig, a.g);
                }
            }
        }
    }
    if constexpr (kOut != 0) {
#pragma unroll
        for (int i = 0; i < 8; i++) st[i] += __shfl_xor(st[i], 32);
        st[7] *= -0.6931471805599453;  // -sum p ln p = -ln 2 sum p log2 p
        if (row_ok && h == 0) {
            double* dst = a.stats + ((int64_t)bh * a.Nq + a.row0 + lr) * 8;
#pragma unroll
            for (int i = 0; i < 8; i++) dst[i] = st[i];
        }
    }
}

// One workgroup per row; 8 lanes per 32-entry block, 4 entries per lane.
template <int kRule>
__global__ __launch_bounds__(256) void rowsum_diag_kernel(RowsumDiagArgs a) {
    __shared__ double red[4][8];
    const int64_t r = blockIdx.x;
    const float* prow = a.p + r * a.ld;
    double st[8];
#pragma unroll
    for (int i = 0; i < 8; i++) st[i] = 0.0;

    for (int64_t base = 0; base < a.N; base += 1024) {
        const int64_t j = base + 4 * threadIdx.x;  // 4 entries of block j / 32
        float p[4] = {0.f, 0.f, 0.f, 0.f};
        if (j < a.N) {
            const float4 v = *reinterpret_cast<const float4*>(prow + j);
            p[0] = v.x;
            p[1] = j + 1 < a.N ? v.y : 0.f;
            p[2] = j + 2 < a.N ? v.z : 0.f;
            p[3] = j + 3 < a.N ? v.w : 0.f;
        }
        float x[4];
        uint32_t mb = 0;
#pragma unroll
        for (int e = 0; e < 4; e++) {
            x[e] = a.gamma * p[e];
            mb = max(mb, __builtin_bit_cast(uint32_t, x[e]) & 0x7FFFFFFFu);
        }
        mb = max(mb, (uint32_t)__shfl_xor((int)mb, 1));
        mb = max(mb, (uint32_t)__shfl_xor((int)mb, 2));
        mb = max(mb, (uint32_t)__shfl_xor((int)mb, 4));
        const int ex = block_exponent_f32<kRule>(mb);
        const float sf = e8m0_as_f32((uint32_t)(ex + 127));
        const float inv = __builtin_bit_cast(float, (uint32_t)(127 - ex) << 23);  // 2^-ex, normal
        const double sig = __builtin_bit_cast(double, (uint64_t)(ex + 1023) << 52);
        uint32_t c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, x[0], x[1], sf, 0);
        c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c, x[2], x[3], sf, 1);
        const auto r01 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(c, 1.0f, 0);
        const auto r23 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(c, 1.0f, 1);
        const float rq[4] = {r01[0], r01[1], r23[0], r23[1]};
#pragma unroll
        for (int e = 0; e < 4; e++) diag_add(st, p[e], x[e] * inv, rq[e], (c >> (4 * e)) & 0xFu, sig, a.g);
    }
    // -sum p ln p = -ln 2 * sum p log2 p
    st[7] *= -0.6931471805599453;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
#pragma unroll
        for (int i = 0; i < 8; i++) st[i] += __shfl_xor(st[i], off);
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0)
#pragma unroll
        for (int i = 0; i < 8; i++) red[wave][i] = st[i];
    __syncthreads();
    if (threadIdx.x < 8) {
        const int i = threadIdx.x;
        const double v = (red[0][i] + red[1][i]) + (red[2][i] + red[3][i]);
        const int64_t head = r / a.rows_per_head, lr = r % a.rows_per_head;
        a.stats[((head * a.out_rows_per_head) + a.out_row0 + lr) * 8 + i] = v;
    }
}

}  // namespace

hipError_t launch_attn_rows(const SoftmaxRowsArgs& args, int64_t BH, int out, hipStream_t stream) {
    SoftmaxRowsArgs a = args;
    a.qtiles = (a.rows + kRowsPerWg - 1) / kRowsPerWg;
    a.c = 0.12751743082459868f;  // fp32(log2(e) / sqrt(128))
    const dim3 grid((unsigned)(BH * a.qtiles));
    if (out == kRowsStoreP)
        attn_rows_kernel<0><<<grid, 256, 0, stream>>>(a);
    else if (out == kRowsDiagUos)
        attn_rows_kernel<1><<<grid, 256, 0, stream>>>(a);
    else
        attn_rows_kernel<2><<<grid, 256, 0, stream>>>(a);
    return hipGetLastError();
}

hipError_t launch_rowsum_diag(const RowsumDiagArgs& a, int64_t rows, int rule, hipStream_t stream) {
    if (rows == 0) return hipSuccess;
    if (rule == kRuleUos)
        rowsum_diag_kernel<kRuleUos><<<dim3((unsigned)rows), 256, 0, stream>>>(a);
    else
        rowsum_diag_kernel<kRuleOcp><<<dim3((unsigned)rows), 256, 0, stream>>>(a);
    return hipGetLastError();
}

}  // namespace mxattn
