// quantize.hip -- MXFP4 block quantizers for gfx950 (Algorithm 1 with the UOS
// rule, the OCP floor scale rule, or the ceil rule of a general boundary q).
//
// Both kernels stream bf16 from HBM once and write 4-bit codes plus one E8M0
// byte per 32 elements (2.53125 bytes of traffic per element).  The E2M1
// rounding itself is done by the gfx950 scaled FP4 conversion, which rounds to
// nearest with ties to the even code, saturates at +-6 and keeps the sign bit
// (the same readings the library documents for the quantizer).
#include <cmath>

#include "device_common.h"
#include "launch.h"

namespace mxattn {

// The bf16 inputs are read exactly once: non-temporal loads keep them from
// displacing cached lines (measured ~10 % faster than ordinary loads here).
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 nt_load(const uint4* p) {
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
    return make_uint4(v[0], v[1], v[2], v[3]);
}

// ---------------------------------------------------------------------------
// Blocks along the head dimension (Q and K).  A thread owns 8 consecutive
// elements (one 16-byte chunk) in each of two grid-strided passes, both
// loaded before either is quantized; the 4 threads of a 32-element block are
// adjacent lanes and exchange their maxima with two lane swaps.
// ---------------------------------------------------------------------------
// Cross-lane exchanges inside a row of 16 lanes with DPP moves (no LDS
// traffic): the value of lane i ^ kM.  xor 1 and 2 are quad permutations;
// xor 4 and 8 compose the half-row mirror (lane i ^ 7) with the quad
// reversal (^ 3) or with the row mirror (^ 15).
template <int kM>
__device__ __forceinline__ int lane_xor(int v) {
    constexpr int kQuadXor1 = 0xB1, kQuadXor2 = 0x4E, kQuadRev = 0x1B, kRowMirror = 0x140, kHalfMirror = 0x141;
    if constexpr (kM == 1) {
        return __builtin_amdgcn_mov_dpp(v, kQuadXor1, 0xF, 0xF, false);
    } else if constexpr (kM == 2) {
        return __builtin_amdgcn_mov_dpp(v, kQuadXor2, 0xF, 0xF, false);
    } else if constexpr (kM == 4) {
        const int h = __builtin_amdgcn_mov_dpp(v, kHalfMirror, 0xF, 0xF, false);
        return __builtin_amdgcn_mov_dpp(h, kQuadRev, 0xF, 0xF, false);
    } else {
        static_assert(kM == 8, "xor within a row of 16 lanes");
        const int h = __builtin_amdgcn_mov_dpp(v, kHalfMirror, 0xF, 0xF, false);
        return __builtin_amdgcn_mov_dpp(h, kRowMirror, 0xF, 0xF, false);
    }
}
template <int kM>
__device__ __forceinline__ float lane_xor(float v) {
    return __builtin_bit_cast(float, lane_xor<kM>(__builtin_bit_cast(int, v)));
}

// One cross-lane butterfly stage of the Walsh-Hadamard transform over the
// lanes of a row (partners differ in bit kM of the lane's index t): lane t gets
// a + b (lower partner) or a - b (upper), with a the lower lane's value; fma
// with +-1 rounds exactly as the add or subtract.
template <int kM>
__device__ __forceinline__ void butterfly_lanes(float (&y)[8], int t) {
    const float sgn = (t & kM) ? -1.f : 1.f;
#pragma unroll
    for (int e = 0; e < 8; e++) y[e] = __builtin_fmaf(sgn, y[e], lane_xor<kM>(y[e]));
}

// Quantizes the 16-byte chunk v (8 elements) of chunk index i.
template <int kRule>
__device__ __forceinline__ void quantize_chunk(uint4 v, int64_t i, bool valid, uint32_t* __restrict__ codes,
                                               uint8_t* __restrict__ scales, Boundary bq) {
    // block maximum of |x| on the bf16 bit patterns (order-preserving for
    // nonnegative finite values)
    uint32_t m = 0;
    m = max(m, v.x & 0x7FFFu);
    m = max(m, (v.x >> 16) & 0x7FFFu);
    m = max(m, v.y & 0x7FFFu);
    m = max(m, (v.y >> 16) & 0x7FFFu);
    m = max(m, v.z & 0x7FFFu);
    m = max(m, (v.z >> 16) & 0x7FFFu);
    m = max(m, v.w & 0x7FFFu);
    m = max(m, (v.w >> 16) & 0x7FFFu);
    m = max(m, (uint32_t)lane_xor<1>((int)m));
    m = max(m, (uint32_t)lane_xor<2>((int)m));
    // all-zero block: sigma = 1 (Algorithm 1); codes come out as signed zeros
    const uint32_t sbyte = (m == 0) ? 127u : (uint32_t)(block_exponent_bf16<kRule>(m, bq) + 127);
    const float sf = e8m0_as_f32(sbyte);
    uint32_t c = 0;
    c = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(c, __builtin_bit_cast(bf16x2, v.x), sf, 0);
    c = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(c, __builtin_bit_cast(bf16x2, v.y), sf, 1);
    c = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(c, __builtin_bit_cast(bf16x2, v.z), sf, 2);
    c = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(c, __builtin_bit_cast(bf16x2, v.w), sf, 3);
    if (valid) {
        codes[i] = c;
        if ((i & 3) == 0) scales[i >> 2] = (uint8_t)sbyte;
    }
}

template <int kRule>
__global__ __launch_bounds__(256) void quantize_headdim_kernel(const uint4* __restrict__ x,
                                                               uint32_t* __restrict__ codes,
                                                               uint8_t* __restrict__ scales,
                                                               int64_t n_chunks, Boundary bq) {
    const int64_t stride = (int64_t)gridDim.x * 256;
    const int64_t i0 = (int64_t)blockIdx.x * 256 + threadIdx.x;
    uint4 v[2];
#pragma unroll
    for (int k = 0; k < 2; k++) {
        const int64_t i = i0 + k * stride;
        v[k] = i < n_chunks ? nt_load(x + i) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int k = 0; k < 2; k++) {
        const int64_t i = i0 + k * stride;
        quantize_chunk<kRule>(v[k], i, i < n_chunks, codes, scales, bq);
    }
}

// ---------------------------------------------------------------------------
// Rotated head-dimension blocks (Q and K of the rotated mode): each row of 128
// is multiplied by R_H = H/sqrt(128) (Sylvester Hadamard, Sec. 4.3, Algorithm
// 2) before the block quantization above.  The product is the radix-2 fast
// Walsh-Hadamard transform in fp32, stages h = 1, 2, 4, ..., 64, each mapping
// (x[i], x[i+h]) (bit h of i clear) to (a + b, a - b), then one fp32 multiply
// by fp32(1/sqrt(128)); the 8 threads of a row hold 16 consecutive elements
// each, so stages 1-8 run in registers and stages 16-64 exchange with the
// thread whose index in the row differs in bit 0, 1 or 2 (DPP moves inside the
// row of lanes).  Every operation is a single correctly
// rounded fp32 add, subtract or multiply in a fixed order, so the result is
// bit-identical to any other evaluation in that order.
// ---------------------------------------------------------------------------
template <int kRule>
__global__ __launch_bounds__(256) void quantize_headdim_rot_kernel(const uint4* __restrict__ x,
                                                                   uint2* __restrict__ codes,
                                                                   uint8_t* __restrict__ scales,
                                                                   int64_t n_threads) {
    // 8 lanes per row of 128, 16 consecutive elements (two chunks) each
    const int64_t g = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const bool valid = g < n_threads;
    uint4 v0 = make_uint4(0, 0, 0, 0), v1 = v0;
    if (valid) {
        v0 = nt_load(x + 2 * g);
        v1 = nt_load(x + 2 * g + 1);
    }
    const int t = threadIdx.x & 7;  // thread within the row: elements 16t..16t+15

    float y[16];
    const uint32_t w[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
#pragma unroll
    for (int e = 0; e < 8; e++) {
        y[2 * e] = __builtin_bit_cast(float, w[e] << 16);
        y[2 * e + 1] = __builtin_bit_cast(float, w[e] & 0xFFFF0000u);
    }
#pragma unroll
    for (int h = 1; h < 16; h *= 2) {
#pragma unroll
        for (int e = 0; e < 16; e++) {
            if (e & h) continue;
            const float a = y[e], b = y[e + h];
            y[e] = a + b;
            y[e + h] = a - b;
        }
    }
#pragma unroll
    for (int half = 0; half < 2; half++) {
        float (&yh)[8] = *reinterpret_cast<float(*)[8]>(&y[8 * half]);
        butterfly_lanes<1>(yh, t);
    }
#pragma unroll
    for (int half = 0; half < 2; half++) {
        float (&yh)[8] = *reinterpret_cast<float(*)[8]>(&y[8 * half]);
        butterfly_lanes<2>(yh, t);
    }
#pragma unroll
    for (int half = 0; half < 2; half++) {
        float (&yh)[8] = *reinterpret_cast<float(*)[8]>(&y[8 * half]);
        butterfly_lanes<4>(yh, t);
    }
    const float rs = 0.0883883476483184405f;  // fp32(1/sqrt(128))
#pragma unroll
    for (int e = 0; e < 16; e++) y[e] = y[e] * rs;

    // block maximum of |y| on the fp32 bit patterns: two lanes per block
    uint32_t m = 0;
#pragma unroll
    for (int e = 0; e < 16; e++) m = max(m, __builtin_bit_cast(uint32_t, y[e]) & 0x7FFFFFFFu);
    m = max(m, (uint32_t)lane_xor<1>((int)m));
    const uint32_t sbyte = (m == 0) ? 127u : (uint32_t)(scale_exponent_f32<kRule>(m) + 127);
    const float sf = e8m0_as_f32(sbyte);

    uint32_t c0 = 0, c1 = 0;
    c0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c0, y[0], y[1], sf, 0);
    c0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c0, y[2], y[3], sf, 1);
    c0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c0, y[4], y[5], sf, 2);
    c0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c0, y[6], y[7], sf, 3);
    c1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c1, y[8], y[9], sf, 0);
    c1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c1, y[10], y[11], sf, 1);
    c1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c1, y[12], y[13], sf, 2);
    c1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c1, y[14], y[15], sf, 3);
    if (valid) {
        codes[g] = make_uint2(c0, c1);
        if ((g & 1) == 0) scales[g >> 1] = (uint8_t)sbyte;
    }
}

// ---------------------------------------------------------------------------
// Blocks along the token axis (V).  A group of 256 tokens x 128 channels of
// one head (64 KiB of bf16) is staged in LDS from coalesced 16-byte loads;
// tokens past N are staged as +0 (the zero padding of the last block).  Wave
// w of 8 then quantizes channel pairs 8w..8w+7 over the group's eight 32-token
// blocks, lane (pair p, block b) owning one block of two channels.  Output
// rows are tokens-contiguous per channel (16 code bytes and one scale byte per
// (channel, 32-token block)), so the eight lanes of a pair write the pair's
// 128 code bytes of this group, one whole 128-byte line per channel row, in
// one store instruction.  (Groups of 128 tokens wrote half lines, 64 bytes
// into each of 128 rows far apart, and took 5 % longer.)  The code may
// quantize kGroupsPerWg consecutive groups per workgroup, loading the next
// group into registers while the current one is quantized; one group per
// workgroup measured fastest with 256-token groups.
constexpr int kVqTokens = 256;
constexpr int kVqThreads = 512;
constexpr int kGroupsPerWg = 1;  // token groups per workgroup

// Two bf16 values (a packed pair) to FP4 codes divided by `scale`, into byte
// `sel` of `old` (the conversion takes the byte index as an immediate).
__device__ __forceinline__ uint32_t cvt_fp4x2_bf16(uint32_t old, uint32_t pair, float scale, int sel) {
    const bf16x2 v = __builtin_bit_cast(bf16x2, pair);
    switch (sel) {
        case 0: return __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(old, v, scale, 0);
        case 1: return __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(old, v, scale, 1);
        case 2: return __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(old, v, scale, 2);
        default: return __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(old, v, scale, 3);
    }
}

template <int kRule>
__global__ __launch_bounds__(kVqThreads) void quantize_tokens_kernel(const uint4* __restrict__ x,
                                                              uint8_t* __restrict__ codes,
                                                              uint8_t* __restrict__ scales, int N,
                                                              int nb, int groups, int per_xcd, int total,
                                                              Boundary bq) {
    // [token][64 dwords = 128 bf16]; the 32-token block b of the group is
    // stored with its dword columns XOR-ed by 8 b, so that the eight lanes
    // reading the same channel pair in eight blocks hit eight bank groups
    __shared__ uint32_t tile[kVqTokens * 64];
    const int tid = threadIdx.x;
    // consecutive workgroup ids go round-robin over the 8 XCDs: give each XCD
    // a contiguous range of (head, group), so that neighbouring groups, whose
    // outputs share cache lines in every channel row, meet in one L2 and
    // reach HBM as whole lines
    const int L = blockIdx.x;
    const int logical = (L & 7) * per_xcd + (L >> 3);
    const int first = logical * kGroupsPerWg;
    if (first >= total) return;
    const int last = min(first + kGroupsPerWg, total);

    // group lg = (head, group) of this XCD's range, 16 chunks of 16 B per token
    auto fetch = [&](int lg, uint4 (&r)[8]) {
        const int bh = lg / groups, g = lg % groups;
        const uint4* src = x + (int64_t)bh * N * 16;
#pragma unroll
        for (int k = 0; k < 8; k++) {
            const int ch = tid + kVqThreads * k;
            const int tok = ch >> 4, part = ch & 15;
            r[k] = (g * kVqTokens + tok < N) ? nt_load(src + (int64_t)(g * kVqTokens + tok) * 16 + part)
                                             : make_uint4(0, 0, 0, 0);
        }
    };
    uint4 buf[8];
    fetch(first, buf);
    for (int lg = first; lg < last; lg++) {
        __syncthreads();  // the previous group's LDS reads are done
#pragma unroll
        for (int k = 0; k < 8; k++) {
            const int ch = tid + kVqThreads * k;
            const int tok = ch >> 4, part = ch & 15;
            *reinterpret_cast<uint4*>(&tile[tok * 64 + ((part * 4) ^ (8 * (tok >> 5)))]) = buf[k];
        }
        __syncthreads();
        if (lg + 1 < last) fetch(lg + 1, buf);  // in flight while this group is quantized
        const int bh = lg / groups, g = lg % groups;

        // wave w: channel pairs 8 w .. 8 w + 7; lane: pair p = lane / 8, token
        // block b = lane % 8 of the group.  The eight lanes of a pair write the
        // pair's eight 16-byte code chunks of this group next to each other.
        const int w = tid >> 6, lane = tid & 63;
        const int p = lane >> 3, b = lane & 7;
        const int cp = 8 * w + p;  // channels 2cp, 2cp+1 (dword column cp)
        const int blk = 8 * g + b;
        if (blk < nb) {
            uint32_t col[32];
            uint32_t m0 = 0, m1 = 0;
#pragma unroll
            for (int t = 0; t < 32; t++) {
                uint32_t d = tile[(32 * b + t) * 64 + (cp ^ (8 * b))];
                col[t] = d;
                m0 = max(m0, d & 0x7FFFu);
                m1 = max(m1, (d >> 16) & 0x7FFFu);
            }
            const uint32_t s0 = (m0 == 0) ? 127u : (uint32_t)(block_exponent_bf16<kRule>(m0, bq) + 127);
            const uint32_t s1 = (m1 == 0) ? 127u : (uint32_t)(block_exponent_bf16<kRule>(m1, bq) + 127);
            const float f0 = e8m0_as_f32(s0), f1 = e8m0_as_f32(s1);

            uint32_t c0[4] = {0, 0, 0, 0}, c1[4] = {0, 0, 0, 0};
#pragma unroll
            for (int t = 0; t < 32; t += 2) {
                // (token t, token t+1) pairs of each channel
                uint32_t lo = __builtin_amdgcn_perm(col[t + 1], col[t], 0x05040100u);  // low halves
                uint32_t hi = __builtin_amdgcn_perm(col[t + 1], col[t], 0x07060302u);  // high halves
                const int word = t >> 3, sel = (t & 7) >> 1;
                c0[word] = cvt_fp4x2_bf16(c0[word], lo, f0, sel);
                c1[word] = cvt_fp4x2_bf16(c1[word], hi, f1, sel);
            }
            const int64_t row0 = (int64_t)bh * 128 + 2 * cp;
            *reinterpret_cast<uint4*>(codes + (row0 * nb + blk) * 16) = make_uint4(c0[0], c0[1], c0[2], c0[3]);
            *reinterpret_cast<uint4*>(codes + ((row0 + 1) * nb + blk) * 16) = make_uint4(c1[0], c1[1], c1[2], c1[3]);
            scales[row0 * nb + blk] = (uint8_t)s0;
            scales[(row0 + 1) * nb + blk] = (uint8_t)s1;
        }
    }
}

// Kernel argument of the kRuleQmax rule for boundary q (4 <= q <= 8).
Boundary boundary_of(double q) {
    Boundary b;
    b.thr = (int)std::floor(32.0 * (q - 4.0));
    b.pow2_down = q == 8.0 ? 1 : 0;
    return b;
}

hipError_t launch_quantize_headdim(const void* x, uint8_t* codes, uint8_t* scales, int64_t rows,
                                   int rule, hipStream_t stream, double qmax) {
    const int64_t n_chunks = rows * 16;  // d = 128: 16 chunks of 8 elements per row
    if (n_chunks == 0) return hipSuccess;
    const dim3 grid((unsigned)(((n_chunks + 2 - 1) / 2 + 255) / 256));
    const Boundary bq = boundary_of(rule == kRuleQmax ? qmax : 7.25);
    if (rule == kRuleUos)
        quantize_headdim_kernel<kRuleUos><<<grid, 256, 0, stream>>>(
            (const uint4*)x, (uint32_t*)codes, scales, n_chunks, bq);
    else if (rule == kRuleQmax)
        quantize_headdim_kernel<kRuleQmax><<<grid, 256, 0, stream>>>(
            (const uint4*)x, (uint32_t*)codes, scales, n_chunks, bq);
    else
        quantize_headdim_kernel<kRuleOcp><<<grid, 256, 0, stream>>>(
            (const uint4*)x, (uint32_t*)codes, scales, n_chunks, bq);
    return hipGetLastError();
}

hipError_t launch_quantize_headdim_rotated(const void* x, uint8_t* codes, uint8_t* scales, int64_t rows,
                                           int rule, hipStream_t stream) {
    const int64_t n_threads = rows * 8;
    if (n_threads == 0) return hipSuccess;
    const dim3 grid((unsigned)((n_threads + 255) / 256));
    if (rule == kRuleUos)
        quantize_headdim_rot_kernel<kRuleUos><<<grid, 256, 0, stream>>>(
            (const uint4*)x, (uint2*)codes, scales, n_threads);
    else
        quantize_headdim_rot_kernel<kRuleOcp><<<grid, 256, 0, stream>>>(
            (const uint4*)x, (uint2*)codes, scales, n_threads);
    return hipGetLastError();
}

hipError_t launch_quantize_tokens(const void* x, uint8_t* codes, uint8_t* scales, int64_t BH,
                                  int64_t N, int rule, hipStream_t stream, double qmax) {
    const int nb = (int)((N + 31) / 32);
    const int groups = (int)((N + kVqTokens - 1) / kVqTokens);
    const int total = (int)(BH * groups);
    const int wgs = (total + kGroupsPerWg - 1) / kGroupsPerWg;
    const int per_xcd = (wgs + 7) / 8;
    const dim3 grid((unsigned)(8 * per_xcd));
    const Boundary bq = boundary_of(rule == kRuleQmax ? qmax : 7.25);
    if (rule == kRuleUos)
        quantize_tokens_kernel<kRuleUos><<<grid, kVqThreads, 0, stream>>>((const uint4*)x, codes, scales,
                                                                    (int)N, nb, groups, per_xcd, total, bq);
    else if (rule == kRuleQmax)
        quantize_tokens_kernel<kRuleQmax><<<grid, kVqThreads, 0, stream>>>((const uint4*)x, codes, scales,
                                                                     (int)N, nb, groups, per_xcd, total, bq);
    else
        quantize_tokens_kernel<kRuleOcp><<<grid, kVqThreads, 0, stream>>>((const uint4*)x, codes, scales,
                                                                    (int)N, nb, groups, per_xcd, total, bq);
    return hipGetLastError();
}

}  // namespace mxattn
