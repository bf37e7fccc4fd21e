// bench_issue.hip -- instruction issue rates of the attention kernel's
// per-score instruction mix on gfx950, alone and next to FP4 matrix-core
// work of other waves of the same SIMD.
//
// One workgroup per CU (256 workgroups) of 4 * S waves, so S waves per SIMD
// (S = 1 to 4)
// (wave w runs on SIMD w % 4, slot w / 4).  Slot 0 of every SIMD runs the
// stream under test ("A"); every other slot runs stream "B", which repeats
// until all A waves of the workgroup have finished (a flag in LDS, polled
// once per B iteration, with an iteration cap so that every wave exits), so
// each A wave is measured entirely while B is running.  With B = same, every
// slot runs A for the same number of iterations and the SIMD time is the
// slowest wave's.  Cycles come from s_memtime (the shader clock).
//
// Streams (per iteration), written as inline assembly so that the order is
// fixed; every instruction's operands are independent of the matrix-core
// results, and no vector instruction reads a register an MFMA wrote inside
// the timed loop:
//   fma      64 v_fma_f32
//   exp      64 v_exp_f32
//   cvt      32 v_cvt_scalef32_pk_fp4_f32 (two fp32 values each)
//   max3     32 v_maximum3_f32
//   soft     the per-score mix of one wave-tile: 64 fma, 64 exp, 32 cvt,
//            32 max3, in groups of 8 scores (8 fma, 8 exp, 4 cvt, 4 max3)
//   mfma32   16 V_MFMA_SCALE_F32_32X32X64_F8F6F4 (FP4 x FP4), 4 accumulators
//   mfma16   32 V_MFMA_SCALE_F32_16X16X128_F8F6F4 (FP4 x FP4), 8 accumulators
//            (the same matrix-core time as mfma32)
//   soft+m32 soft with one 32x32x64 MFMA after every 4 scores' worth of
//            softmax instructions (16 per iteration)
//   soft+m16 soft with one 16x16x128 MFMA after every 2 scores (32)
//   tile     the whole vector and matrix-core mix of one wave-tile of the
//            attention kernel as compiled: soft, 16 32x32x64 and 2 16x16x128
//            products in the kernel's order (the previous tile's second PV
//            chunk and the first score pair under the first quarter of the
//            softmax, a score pair and the first PV chunk under the second,
//            a score pair under each of the last two), plus 3 FMA, 3 exp,
//            3 max3, 20 integer operations and 11 multiplies (the rescale of
//            O~, which runs on about 16 % of tiles, averaged)
//   idle     nothing (the wave exits at once)
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

typedef float v16f __attribute__((ext_vector_type(16)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef int v4i __attribute__((ext_vector_type(4)));

enum Kind { kIdle, kFma, kExp, kCvt, kMax3, kSoft, kMfma32, kMfma16, kSoftM32, kSoftM16, kTile, kNumKinds };
static const char* kNames[kNumKinds] = {"idle", "fma", "exp", "cvt", "max3", "soft", "mfma32", "mfma16",
                                        "soft+m32", "soft+m16", "tile"};

constexpr int kIters = 512;        // A iterations
constexpr int kMaxBIters = 1 << 16;  // cap on B iterations (B stops when A is done)

#define FMA8(x)                                                                                         \
    asm volatile(                                                                                       \
        "v_fma_f32 %0, %0, %8, %9\n v_fma_f32 %1, %1, %8, %9\n v_fma_f32 %2, %2, %8, %9\n"           \
        " v_fma_f32 %3, %3, %8, %9\n v_fma_f32 %4, %4, %8, %9\n v_fma_f32 %5, %5, %8, %9\n"          \
        " v_fma_f32 %6, %6, %8, %9\n v_fma_f32 %7, %7, %8, %9"                                         \
        : "+v"(x[0]), "+v"(x[1]), "+v"(x[2]), "+v"(x[3]), "+v"(x[4]), "+v"(x[5]), "+v"(x[6]), "+v"(x[7]) \
        : "v"(c1), "v"(c2))
#define EXP8(x)                                                                                           \
    asm volatile(                                                                                         \
        "v_exp_f32 %0, %0\n v_exp_f32 %1, %1\n v_exp_f32 %2, %2\n v_exp_f32 %3, %3\n"                   \
        " v_exp_f32 %4, %4\n v_exp_f32 %5, %5\n v_exp_f32 %6, %6\n v_exp_f32 %7, %7"                    \
        : "+v"(x[0]), "+v"(x[1]), "+v"(x[2]), "+v"(x[3]), "+v"(x[4]), "+v"(x[5]), "+v"(x[6]), "+v"(x[7]))
#define CVT4(x, w)                                                                                      \
    asm volatile(                                                                                       \
        "v_cvt_scalef32_pk_fp4_f32 %0, %4, %5, %12\n v_cvt_scalef32_pk_fp4_f32 %1, %6, %7, %12\n"      \
        " v_cvt_scalef32_pk_fp4_f32 %2, %8, %9, %12\n v_cvt_scalef32_pk_fp4_f32 %3, %10, %11, %12"     \
        : "+v"(w[0]), "+v"(w[1]), "+v"(w[2]), "+v"(w[3])                                               \
        : "v"(x[0]), "v"(x[1]), "v"(x[2]), "v"(x[3]), "v"(x[4]), "v"(x[5]), "v"(x[6]), "v"(x[7]), "v"(one))
#define MAX4(x, w)                                                                                      \
    asm volatile(                                                                                       \
        "v_maximum3_f32 %0, %0, %4, %5\n v_maximum3_f32 %1, %1, %6, %7\n"                              \
        " v_maximum3_f32 %2, %2, %8, %9\n v_maximum3_f32 %3, %3, %10, %11"                             \
        : "+v"(w[0]), "+v"(w[1]), "+v"(w[2]), "+v"(w[3])                                               \
        : "v"(x[0]), "v"(x[1]), "v"(x[2]), "v"(x[3]), "v"(x[4]), "v"(x[5]), "v"(x[6]), "v"(x[7]))
#define M32(acc)                                                                                        \
    asm volatile("v_mfma_scale_f32_32x32x64_f8f6f4 %0, %1, %2, %0, %3, %3 op_sel_hi:[0,0,0] cbsz:4 blgp:4" \
                 : "+v"(acc) : "v"(a4), "v"(b4), "v"(sc))
#define M16(acc)                                                                                        \
    asm volatile("v_mfma_scale_f32_16x16x128_f8f6f4 %0, %1, %2, %0, %3, %3 op_sel_hi:[0,0,0] cbsz:4 blgp:4" \
                 : "+v"(acc) : "v"(a4), "v"(b4), "v"(sc))

// 8 scores of the softmax mix on x (and y for the maxima)
#define SOFT8(x, y) \
    FMA8(x);        \
    EXP8(x);        \
    CVT4(x, w);     \
    MAX4(y, mx)

template <int K>
constexpr bool uses_m32() { return K == kMfma32 || K == kSoftM32 || K == kTile; }
template <int K>
constexpr bool uses_m16() { return K == kMfma16 || K == kSoftM16 || K == kTile; }

// One iteration of stream K.
template <int K>
__device__ __forceinline__ void iteration(float (&x)[8], float (&y)[8], float (&mx)[4], uint32_t (&w)[4],
                                          float (&z)[4], uint32_t (&ii)[4], v16f (&acc32)[4], v4f (&acc16)[8],
                                          const v4i& a4, const v4i& b4, const int& sc, float c1, float c2,
                                          float one) {
    if constexpr (K == kFma) {
        FMA8(x); FMA8(y); FMA8(x); FMA8(y); FMA8(x); FMA8(y); FMA8(x); FMA8(y);
    } else if constexpr (K == kExp) {
        EXP8(x); EXP8(y); EXP8(x); EXP8(y); EXP8(x); EXP8(y); EXP8(x); EXP8(y);
    } else if constexpr (K == kCvt) {
        CVT4(x, w); CVT4(y, w); CVT4(x, w); CVT4(y, w); CVT4(x, w); CVT4(y, w); CVT4(x, w); CVT4(y, w);
    } else if constexpr (K == kMax3) {
        MAX4(x, mx); MAX4(y, mx); MAX4(x, mx); MAX4(y, mx); MAX4(x, mx); MAX4(y, mx); MAX4(x, mx); MAX4(y, mx);
    } else if constexpr (K == kSoft) {
#pragma unroll
        for (int r = 0; r < 4; r++) {
            SOFT8(x, y);
            SOFT8(y, x);
        }
    } else if constexpr (K == kMfma32) {
#pragma unroll
        for (int r = 0; r < 4; r++) {
            M32(acc32[0]); M32(acc32[1]); M32(acc32[2]); M32(acc32[3]);
        }
    } else if constexpr (K == kMfma16) {
#pragma unroll
        for (int r = 0; r < 4; r++) {
            M16(acc16[0]); M16(acc16[1]); M16(acc16[2]); M16(acc16[3]);
            M16(acc16[4]); M16(acc16[5]); M16(acc16[6]); M16(acc16[7]);
        }
    } else if constexpr (K == kSoftM32) {
        // one MFMA per 4 scores: 2 per group of 8
#pragma unroll
        for (int r = 0; r < 4; r++) {
            FMA8(x); M32(acc32[0]); EXP8(x); CVT4(x, w); MAX4(y, mx); M32(acc32[1]);
            FMA8(y); M32(acc32[2]); EXP8(y); CVT4(y, w); MAX4(x, mx); M32(acc32[3]);
        }
    } else if constexpr (K == kSoftM16) {
        // one MFMA per 2 scores: 4 per group of 8
#pragma unroll
        for (int r = 0; r < 4; r++) {
            FMA8(x); M16(acc16[0]); EXP8(x); M16(acc16[1]); CVT4(x, w); M16(acc16[2]); MAX4(y, mx); M16(acc16[3]);
            FMA8(y); M16(acc16[4]); EXP8(y); M16(acc16[5]); CVT4(y, w); M16(acc16[6]); MAX4(x, mx); M16(acc16[7]);
        }
    } else if constexpr (K == kTile) {
        // first quarter: the previous tile's second PV chunk, the first score pair
        FMA8(x); M32(acc32[0]); EXP8(x); M32(acc32[1]); CVT4(x, w); M32(acc32[2]); MAX4(y, mx); M32(acc32[3]);
        FMA8(y); M16(acc16[0]); EXP8(y); M32(acc32[0]); CVT4(y, w); MAX4(x, mx); M32(acc32[1]);
        // second quarter: a score pair, the first PV chunk
        FMA8(x); M32(acc32[2]); EXP8(x); M32(acc32[3]); CVT4(x, w); M32(acc32[0]); MAX4(y, mx); M32(acc32[1]);
        FMA8(y); M32(acc32[2]); EXP8(y); M32(acc32[3]); CVT4(y, w); M16(acc16[1]); MAX4(x, mx);
        // third and fourth quarters: a score pair each
        FMA8(x); EXP8(x); M32(acc32[0]); CVT4(x, w); MAX4(y, mx);
        FMA8(y); EXP8(y); M32(acc32[1]); CVT4(y, w); MAX4(x, mx);
        FMA8(x); EXP8(x); M32(acc32[2]); CVT4(x, w); MAX4(y, mx);
        FMA8(y); EXP8(y); M32(acc32[3]); CVT4(y, w); MAX4(x, mx);
        // the rest of the tile's vector work
#pragma unroll
        for (int i = 0; i < 3; i++) {
            asm volatile("v_fma_f32 %0, %0, %1, %2" : "+v"(z[i]) : "v"(c1), "v"(c2));
            asm volatile("v_exp_f32 %0, %0" : "+v"(z[i + 1]));
            asm volatile("v_maximum3_f32 %0, %0, %1, %2" : "+v"(z[3 - i]) : "v"(x[i]), "v"(y[i]));
        }
#pragma unroll
        for (int i = 0; i < 20; i++) asm volatile("v_add_u32 %0, %0, %1" : "+v"(ii[i & 3]) : "v"(w[i & 3]));
#pragma unroll
        for (int i = 0; i < 11; i++) asm volatile("v_mul_f32 %0, %0, %1" : "+v"(z[i & 3]) : "v"(one));
    }
}

// KB < 0: every slot runs KA for kIters iterations (throughput of the waves
// of one SIMD running the same stream).
template <int KA, int KB>
__global__ __launch_bounds__(1024, 1) void issue_kernel(long long* out) {
    __shared__ int done_count;
    const int wave = threadIdx.x >> 6;
    const int nwaves = blockDim.x >> 6;
    const int slot = wave >> 2;
    const bool is_a = KB < 0 || slot == 0;
    const int n_a = KB < 0 ? nwaves : 4;
    if (threadIdx.x == 0) done_count = 0;

    float x[8], y[8], mx[4] = {0.f, 0.f, 0.f, 0.f}, z[4] = {-0.5f, -0.25f, -0.125f, -1.f};
    uint32_t ii[4] = {1, 2, 3, 4};
    uint32_t w[4] = {0, 0, 0, 0};
    for (int i = 0; i < 8; i++) {
        x[i] = 1e-3f * (float)(i + 1 + (threadIdx.x & 7));
        y[i] = -1e-3f * (float)(i + 2);
    }
    // t = -t - 1 keeps the fma/exp chains bounded (t -> 2^t -> -2^t - 1 ...)
    const float c1 = -1.0f, c2 = -1.0f, one = 1.0f;
    v4i a4 = {0x22222222, 0x22222222, 0x22222222, 0x22222222};  // FP4 1.0 everywhere
    v4i b4 = a4;
    int sc = 127;  // E8M0 2^0
    v16f acc32[4];
    v4f acc16[8];
    for (int k = 0; k < 4; k++)
        for (int i = 0; i < 16; i++) acc32[k][i] = 0.f;
    for (int k = 0; k < 8; k++)
        for (int i = 0; i < 4; i++) acc16[k][i] = 0.f;
    asm volatile("" : "+v"(a4), "+v"(b4), "+v"(sc));
    __syncthreads();
    // operand registers were written by vector instructions just above
    asm volatile("s_nop 7\n s_nop 7");

    const long long t0 = __builtin_amdgcn_s_memtime();
    int iters = 0;
    if (is_a) {
        for (int it = 0; it < kIters; it++) {
            iteration<KA>(x, y, mx, w, z, ii, acc32, acc16, a4, b4, sc, c1, c2, one);
            iters++;
        }
    } else if constexpr (KB >= 0) {
        for (int it = 0; it < kMaxBIters; it++) {
            // stop once every A wave has finished
            if (__builtin_amdgcn_readfirstlane(*(volatile int*)&done_count) >= n_a) break;
            iteration<KB>(x, y, mx, w, z, ii, acc32, acc16, a4, b4, sc, c1, c2, one);
            iters++;
        }
    }
    const long long t1 = __builtin_amdgcn_s_memtime();
    // let the last MFMAs retire before their results are read
    asm volatile("s_nop 7\n s_nop 7\n s_nop 7\n s_nop 7");
    if (is_a && (threadIdx.x & 63) == 0) atomicAdd(&done_count, 1);

    float s = 0.f;
    for (int i = 0; i < 8; i++) s += x[i] + y[i];
    for (int i = 0; i < 4; i++) s += __builtin_bit_cast(float, w[i] ^ ii[i]) + mx[i] + z[i];
    if constexpr (uses_m32<KA>() || (KB >= 0 && uses_m32<KB>()))
        for (int k = 0; k < 4; k++) s += acc32[k][threadIdx.x & 15];
    if constexpr (uses_m16<KA>() || (KB >= 0 && uses_m16<KB>()))
        for (int k = 0; k < 8; k++) s += acc16[k][threadIdx.x & 3];
    if ((threadIdx.x & 63) == 0) {
        long long* o = out + ((size_t)blockIdx.x * 16 + wave) * 3;
        o[0] = t1 - t0;
        o[1] = iters;
        o[2] = (long long)__builtin_bit_cast(int, s);  // keeps the streams live
    }
}

typedef void (*KernelFn)(long long*);
template <int KA, int KB>
KernelFn kfn() { return issue_kernel<KA, KB>; }

struct Result {
    double a_cycles_per_iter;  // median over A waves
    double simd_cycles_per_wave_iter;  // (all A waves on one SIMD) / iterations
    double b_iters_per_a;      // median B iterations completed per A wave's run
};

static Result run(KernelFn fn, int kindB, int slots, long long* d, std::vector<long long>& h) {
    const int nblk = 256;
    (void)hipMemset(d, 0, h.size() * sizeof(long long));
    hipLaunchKernelGGL(fn, dim3(nblk), dim3(slots * 256), 0, 0, d);
    if (hipDeviceSynchronize() != hipSuccess) {
        std::fprintf(stderr, "kernel failed\n");
        std::exit(1);
    }
    (void)hipMemcpy(h.data(), d, h.size() * sizeof(long long), hipMemcpyDeviceToHost);
    std::vector<double> a, simd, b;
    for (int blk = 0; blk < nblk; blk++) {
        for (int simd_i = 0; simd_i < 4; simd_i++) {
            long long tmax = 0;
            int na = 0;
            for (int sl = 0; sl < slots; sl++) {
                const int wv = sl * 4 + simd_i;
                const long long* o = &h[((size_t)blk * 16 + wv) * 3];
                const bool is_a = kindB < 0 || sl == 0;
                if (is_a) {
                    a.push_back((double)o[0] / kIters);
                    tmax = std::max(tmax, o[0]);
                    na++;
                } else {
                    b.push_back((double)o[1]);
                }
            }
            simd.push_back((double)tmax / ((double)kIters * na));
        }
    }
    auto med = [](std::vector<double>& v) {
        if (v.empty()) return 0.0;
        std::sort(v.begin(), v.end());
        return v[v.size() / 2];
    };
    return {med(a), med(simd), med(b) / 1.0};
}

int main() {
    long long* d = nullptr;
    std::vector<long long> h((size_t)256 * 16 * 3);
    if (hipMalloc(&d, h.size() * sizeof(long long)) != hipSuccess) return 1;
    run(kfn<kFma, -1>(), -1, 1, d, h);  // warm-up
    std::printf("# per-iteration work: fma/exp 64 instr, cvt/max3 32, soft 64 fma + 64 exp + 32 cvt + 32 max3,\n");
    std::printf("# mfma32 16 x 32x32x64, mfma16 32 x 16x16x128 (the same matrix-core work)\n");
    std::printf("%-10s %-10s %5s %14s %18s %10s\n", "A", "B", "waves", "A cyc/iter", "SIMD cyc/wave-iter",
                "B iters");
    struct Alone { int k; KernelFn f; };
    const Alone alone[] = {{kFma, kfn<kFma, -1>()},         {kExp, kfn<kExp, -1>()},
                           {kCvt, kfn<kCvt, -1>()},         {kMax3, kfn<kMax3, -1>()},
                           {kSoft, kfn<kSoft, -1>()},       {kMfma32, kfn<kMfma32, -1>()},
                           {kMfma16, kfn<kMfma16, -1>()},   {kSoftM32, kfn<kSoftM32, -1>()},
                           {kSoftM16, kfn<kSoftM16, -1>()},   {kTile, kfn<kTile, -1>()}};
    for (const Alone& a : alone)
        for (int slots : {1, 2, 3, 4}) {
            Result r = run(a.f, -1, slots, d, h);
            std::printf("%-10s %-10s %5d %14.1f %18.1f %10s\n", kNames[a.k], "(same)", slots, r.a_cycles_per_iter,
                        r.simd_cycles_per_wave_iter, "-");
        }
    struct Pair { int a, b; KernelFn f; };
    const Pair pairs[] = {
        {kFma, kMfma32, kfn<kFma, kMfma32>()},   {kExp, kMfma32, kfn<kExp, kMfma32>()},
        {kCvt, kMfma32, kfn<kCvt, kMfma32>()},   {kMax3, kMfma32, kfn<kMax3, kMfma32>()},
        {kSoft, kMfma32, kfn<kSoft, kMfma32>()}, {kFma, kMfma16, kfn<kFma, kMfma16>()},
        {kExp, kMfma16, kfn<kExp, kMfma16>()},   {kCvt, kMfma16, kfn<kCvt, kMfma16>()},
        {kMax3, kMfma16, kfn<kMax3, kMfma16>()}, {kSoft, kMfma16, kfn<kSoft, kMfma16>()},
        {kSoft, kSoft, kfn<kSoft, kSoft>()},     {kMfma32, kSoft, kfn<kMfma32, kSoft>()},
        {kMfma16, kSoft, kfn<kMfma16, kSoft>()}, {kFma, kExp, kfn<kFma, kExp>()},
        {kExp, kFma, kfn<kExp, kFma>()},         {kCvt, kExp, kfn<kCvt, kExp>()}};
    for (const Pair& p : pairs)
        for (int slots : {2, 3, 4}) {
            Result r = run(p.f, p.b, slots, d, h);
            std::printf("%-10s %-10s %5d %14.1f %18s %10.0f\n", kNames[p.a], kNames[p.b], slots,
                        r.a_cycles_per_iter, "-", r.b_iters_per_a);
        }
    (void)hipFree(d);
    return 0;
}
