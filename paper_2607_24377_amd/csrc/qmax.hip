// qmax.hip -- per-head MXFP4 squared-error sweep over scale boundaries q for
// gfx950 (the per-tensor MSE comparison of Sec. 5.5, Table cx_distribution,
// over the ceil family of Eq. scale_definition).
//
// For a block whose bf16 maximum is M = (1 + F/128) 2^(E-127), every boundary
// 4 <= q <= 8 selects one of three exponents (device_common.h): E-129 when
// F <= thr(q), E-128 otherwise, and E-130 for q = 8 when M is a power of two.
// One pass over the tensor therefore computes each block's squared error
// under those three exponents and adds them to a per-head histogram over F:
//     A[F] += sse(E-128),   B[F] += sse(E-129),   C += sse(E-130) if F = 0.
// For boundary q_j the head's total is then the sum over F of
//     F > thr_j ? A[F] : (F == 0 && pow2_down_j ? C : B[F]),
// so the pass costs the same for any number of boundaries.  Exponents are
// clamped to [-127, 127]; for maxima below 2^-126 (and all-zero blocks) the
// three clamp to the same value and so do the three sums.
//
// Squared errors: with xs = x 2^-e (exact: a product with a power of two)
// and r the E2M1 value of the block's code for x (the scaled FP4 conversion,
// decoded back at scale 1), err = xs - r is exact in fp32 for bf16 x, and so
// is err^2; groups of 8 are summed in fp32 (exactly but for elements that
// round to zero, see oct_sse), then in fp64, and the block sum is scaled by
// 2^(2e).  The pass reads x once from HBM (2 bytes per element) and is the
// only large traffic; the histograms go through LDS (fp64 LDS atomics, so the
// order of additions inside a workgroup varies from run to run) and then,
// per workgroup, to a small workspace that one more kernel reduces in a
// fixed order.
#include <cmath>

#include "device_common.h"
#include "launch.h"

namespace mxattn {

namespace {

constexpr int kBins = 257;          // A[0..127], B[0..127], C
constexpr int kTargetGroups = 2048;  // workgroups per launch (8 per CU)
constexpr int kTokGroup = 128;       // tokens staged per workgroup step (token blocks)

struct BoundaryList {
    int thr[kMaxBoundaries];
    int down[kMaxBoundaries];
};

__device__ __forceinline__ int clamp_e(int e) { return e < -127 ? -127 : (e > 127 ? 127 : e); }

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __builtin_bit_cast(float, w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __builtin_bit_cast(float, w & 0xFFFF0000u); }

// Sum of (x 2^-e - r)^2 over the two bf16 elements of `pair`, whose 4-bit
// codes the scaled conversion puts in byte 0 of the result, in fp32.
__device__ __forceinline__ float pair_sse(uint32_t pair, int e) {
    const float sf = e8m0_as_f32((uint32_t)(e + 127));
    const uint32_t c = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(0u, __builtin_bit_cast(bf16x2, pair), sf, 0);
    const auto r = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(c, 1.0f, 0);
    // 2^-e as a normal fp32 (e <= 126 here: bf16 maxima have E <= 254)
    const float inv = __builtin_bit_cast(float, (uint32_t)(127 - e) << 23);
    const float d0 = bf16_lo(pair) * inv - r[0];
    const float d1 = bf16_hi(pair) * inv - r[1];
    return fmaf(d0, d0, d1 * d1);
}

// Squared error of 8 elements (4 bf16 pairs) under exponent e.  Each term is
// exact in fp32; so is their fp32 sum unless an element rounds to zero with
// bits below 2^-18 of its scaled value (the other terms are multiples of
// 2^-18 below 4 and add up to less than 2^5), so the partial carries at most
// the error of a 7-addition fp32 sum of nonnegative terms, 7 * 2^-24 of it.
__device__ __forceinline__ double oct_sse(uint32_t a, uint32_t b, uint32_t c, uint32_t d, int e) {
    return (double)((pair_sse(a, e) + pair_sse(b, e)) + (pair_sse(c, e) + pair_sse(d, e)));
}

__device__ __forceinline__ void hist_zero(double* h) {
    for (int i = threadIdx.x; i < kBins; i += blockDim.x) h[i] = 0.0;
}

__device__ __forceinline__ void hist_add(double* h, uint32_t mbits, double sp, double s0, double sm) {
    const int F = (int)(mbits & 0x7Fu);
    atomicAdd(&h[F], sp);
    atomicAdd(&h[128 + F], s0);
    if (F == 0) atomicAdd(&h[256], sm);
}

// Blocks along d (rows of 128 = 4 blocks): as the head-dim quantizer, each
// thread owns 8 consecutive elements and 4 adjacent lanes form a block.  A
// workgroup covers rows [c * rows_per_chunk, ...) of one head, 16 rows per
// step.
__global__ __launch_bounds__(256) void sse_hist_headdim_kernel(const uint4* __restrict__ x,
                                                               double* __restrict__ partial,
                                                               int64_t N, int64_t rows_per_chunk,
                                                               int chunks) {
    __shared__ double hist[kBins];
    const int bh = blockIdx.x / chunks, c = blockIdx.x % chunks;
    hist_zero(hist);
    __syncthreads();

    const int64_t r0 = (int64_t)c * rows_per_chunk;
    const int64_t r1 = min(N, r0 + rows_per_chunk);
    const uint4* src = x + (int64_t)bh * N * 16;
    for (int64_t base = r0; base < r1; base += 16) {  // same trip count in every lane
        const int64_t row = base + (threadIdx.x >> 4);
        const bool valid = row < r1;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (valid) v = src[row * 16 + (threadIdx.x & 15)];
        uint32_t m = 0;
        m = max(m, v.x & 0x7FFFu);
        m = max(m, (v.x >> 16) & 0x7FFFu);
        m = max(m, v.y & 0x7FFFu);
        m = max(m, (v.y >> 16) & 0x7FFFu);
        m = max(m, v.z & 0x7FFFu);
        m = max(m, (v.z >> 16) & 0x7FFFu);
        m = max(m, v.w & 0x7FFFu);
        m = max(m, (v.w >> 16) & 0x7FFFu);
        m = max(m, (uint32_t)__shfl_xor((int)m, 1));
        m = max(m, (uint32_t)__shfl_xor((int)m, 2));
        const int E = (int)(m >> 7);
        const int ep = clamp_e(E - 128), e0 = clamp_e(E - 129), em = clamp_e(E - 130);
        // E - 130 is used only for a power-of-two maximum (F = 0)
        const bool pow2 = (m & 0x7Fu) == 0;
        double sp = oct_sse(v.x, v.y, v.z, v.w, ep);
        double s0 = oct_sse(v.x, v.y, v.z, v.w, e0);
        double sm = pow2 ? oct_sse(v.x, v.y, v.z, v.w, em) : 0.0;
        sp += __shfl_xor(sp, 1);
        s0 += __shfl_xor(s0, 1);
        sm += __shfl_xor(sm, 1);
        sp += __shfl_xor(sp, 2);
        s0 += __shfl_xor(s0, 2);
        sm += __shfl_xor(sm, 2);
        if (valid && (threadIdx.x & 3) == 0)
            hist_add(hist, m, ldexp(sp, 2 * ep), ldexp(s0, 2 * e0), ldexp(sm, 2 * em));
    }
    __syncthreads();
    double* dst = partial + (int64_t)blockIdx.x * kBins;
    for (int i = threadIdx.x; i < kBins; i += blockDim.x) dst[i] = hist[i];
}

// Blocks along the tokens (32 tokens of one channel; the last block padded
// with +0, which adds no error): a workgroup stages 128 tokens x 128 channels
// in LDS, wave w takes token block w of the group and each lane a pair of
// channels.  A workgroup covers token groups [c * groups_per_chunk, ...).
__global__ __launch_bounds__(256) void sse_hist_tokens_kernel(const uint4* __restrict__ x,
                                                              double* __restrict__ partial, int N,
                                                              int groups, int groups_per_chunk,
                                                              int chunks) {
    __shared__ uint32_t tile[kTokGroup * 64];  // [token][64 dwords = 128 bf16]
    __shared__ double hist[kBins];
    const int tid = threadIdx.x;
    const int bh = blockIdx.x / chunks, c = blockIdx.x % chunks;
    hist_zero(hist);

    const uint4* src = x + (int64_t)bh * N * 16;
    const int g0 = c * groups_per_chunk, g1 = min(groups, g0 + groups_per_chunk);
    const int w = tid >> 6, cp = tid & 63;
    for (int g = g0; g < g1; g++) {
        const int tok0 = g * kTokGroup;
        __syncthreads();  // previous group's reads (and the zeroed histogram)
#pragma unroll
        for (int k = 0; k < 8; k++) {
            const int ch = tid + 256 * k;
            const int tok = ch >> 4, part = ch & 15;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (tok0 + tok < N) v = src[(int64_t)(tok0 + tok) * 16 + part];
            *reinterpret_cast<uint4*>(&tile[tok * 64 + part * 4]) = v;
        }
        __syncthreads();
        if (tok0 + 32 * w >= N) continue;  // block entirely past the sequence end

        uint32_t col[32];
        uint32_t m0 = 0, m1 = 0;
#pragma unroll
        for (int t = 0; t < 32; t++) {
            const uint32_t d = tile[(32 * w + t) * 64 + cp];
            col[t] = d;
            m0 = max(m0, d & 0x7FFFu);
            m1 = max(m1, (d >> 16) & 0x7FFFu);
        }
#pragma unroll
        for (int ch = 0; ch < 2; ch++) {
            const uint32_t m = ch ? m1 : m0;
            const int E = (int)(m >> 7);
            const int ep = clamp_e(E - 128), e0 = clamp_e(E - 129), em = clamp_e(E - 130);
            double sp = 0.0, s0 = 0.0, sm = 0.0;
            const uint32_t sel = ch ? 0x07060302u : 0x05040100u;
#pragma unroll
            for (int t = 0; t < 32; t += 8) {
                // (token t + 2i, token t + 2i + 1) of this channel as bf16 pairs
                const uint32_t p0 = __builtin_amdgcn_perm(col[t + 1], col[t], sel);
                const uint32_t p1 = __builtin_amdgcn_perm(col[t + 3], col[t + 2], sel);
                const uint32_t p2 = __builtin_amdgcn_perm(col[t + 5], col[t + 4], sel);
                const uint32_t p3 = __builtin_amdgcn_perm(col[t + 7], col[t + 6], sel);
                sp += oct_sse(p0, p1, p2, p3, ep);
                s0 += oct_sse(p0, p1, p2, p3, e0);
                if ((m & 0x7Fu) == 0) sm += oct_sse(p0, p1, p2, p3, em);  // used for F = 0 only
            }
            hist_add(hist, m, ldexp(sp, 2 * ep), ldexp(s0, 2 * e0), ldexp(sm, 2 * em));
        }
    }
    __syncthreads();
    double* dst = partial + (int64_t)blockIdx.x * kBins;
    for (int i = tid; i < kBins; i += blockDim.x) dst[i] = hist[i];
}

// One workgroup per head: sums the chunks' histograms in chunk order, then
// forms each boundary's total in bin order.
__global__ __launch_bounds__(256) void sse_reduce_kernel(const double* __restrict__ partial, int chunks,
                                                         BoundaryList bl, int nq, double* __restrict__ sse) {
    __shared__ double hist[kBins];
    const int bh = blockIdx.x;
    const double* src = partial + (int64_t)bh * chunks * kBins;
    for (int i = threadIdx.x; i < kBins; i += blockDim.x) {
        double acc = 0.0;
        for (int c = 0; c < chunks; c++) acc += src[(int64_t)c * kBins + i];
        hist[i] = acc;
    }
    __syncthreads();
    const int j = threadIdx.x;
    if (j < nq) {
        double tot = 0.0;
        for (int F = 0; F < 128; F++) {
            if (F > bl.thr[j])
                tot += hist[F];
            else if (F == 0 && bl.down[j])
                tot += hist[256];
            else
                tot += hist[128 + F];
        }
        sse[(int64_t)bh * nq + j] = tot;
    }
}

// Workgroups per head and the work each takes.
struct Split {
    int chunks;
    int64_t per_chunk;  // rows (head-dim blocks) or token groups (token blocks)
};

Split split_of(int axis, int64_t BH, int64_t N) {
    const int64_t units = axis == 3 ? (N + 15) / 16 : (N + kTokGroup - 1) / kTokGroup;
    int64_t chunks = (kTargetGroups + BH - 1) / BH;
    if (chunks > units) chunks = units;
    if (chunks < 1) chunks = 1;
    int64_t per = (units + chunks - 1) / chunks;  // in 16-row steps or token groups
    chunks = (units + per - 1) / per;
    Split s;
    s.chunks = (int)chunks;
    s.per_chunk = axis == 3 ? per * 16 : per;
    return s;
}

}  // namespace

int64_t qmax_sse_workspace_bytes(int axis, int64_t BH, int64_t N) {
    return BH * split_of(axis, BH, N).chunks * kBins * (int64_t)sizeof(double);
}

hipError_t launch_qmax_sse(const void* x, int axis, const double* qs, int nq, double* sse,
                           void* workspace, int64_t BH, int64_t N, hipStream_t stream) {
    const Split sp = split_of(axis, BH, N);
    double* partial = static_cast<double*>(workspace);
    const dim3 grid((unsigned)(BH * sp.chunks));
    if (axis == 3) {
        sse_hist_headdim_kernel<<<grid, 256, 0, stream>>>((const uint4*)x, partial, N, sp.per_chunk,
                                                          sp.chunks);
    } else {
        const int groups = (int)((N + kTokGroup - 1) / kTokGroup);
        sse_hist_tokens_kernel<<<grid, 256, 0, stream>>>((const uint4*)x, partial, (int)N, groups,
                                                         (int)sp.per_chunk, sp.chunks);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    BoundaryList bl;
    for (int j = 0; j < kMaxBoundaries; j++) {
        const Boundary b = boundary_of(j < nq ? qs[j] : 7.25);
        bl.thr[j] = b.thr;
        bl.down[j] = b.pow2_down;
    }
    sse_reduce_kernel<<<dim3((unsigned)BH), 256, 0, stream>>>(partial, sp.chunks, bl, nq, sse);
    return hipGetLastError();
}

}  // namespace mxattn
