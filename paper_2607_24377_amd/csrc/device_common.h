// device_common.h -- device helpers shared by the gfx950 kernels of libmxattn.
//
// FP4 (E2M1) matrix-core operands, E8M0 scale selection, bf16 packing.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "launch.h"

namespace mxattn {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Shared-scale exponent of a block from the bits of its maximum magnitude M
// given as a normal fp32 (M >= 2^-126):
//   OCP floor rule  e = floor(log2 M) - 2                (Sec. 2, Eq. ocp_scale)
//   UOS rule        e = ceil(log2(M / 7.25))             (Algorithm 1)
// With M = 1.f * 2^(E-127): floor(log2 M) = E - 127, and M <= 7.25 * 2^(E-129)
// exactly when 1.f <= 1.8125, i.e. when the 23-bit fraction is <= 0x680000;
// otherwise the UOS exponent is one larger.  The result is clamped below at
// -127 (the E8M0 range); it cannot exceed 127 for finite fp32.
template <int kRule>
__device__ __forceinline__ int scale_exponent_f32(uint32_t mbits) {
    int E = (int)(mbits >> 23);
    int e = E - 129;
    if (kRule == kRuleUos) e += ((mbits & 0x7FFFFFu) > 0x680000u) ? 1 : 0;
    return e < -127 ? -127 : e;
}

// Same rule from the bits of a bf16 magnitude (sign cleared).  bf16 values
// below 2^-126 (exponent field 0) need an exponent below -127 under both
// rules, so they clamp to -127.  The UOS fraction threshold 0x680000 of fp32
// is 0x68 in bf16's 7-bit fraction.
template <int kRule>
__device__ __forceinline__ int scale_exponent_bf16(uint32_t mbits) {
    int E = (int)(mbits >> 7);
    if (E == 0) return -127;
    int e = E - 129;
    if (kRule == kRuleUos) e += ((mbits & 0x7Fu) > 0x68u) ? 1 : 0;
    return e < -127 ? -127 : e;
}

// Ceil rule with a general boundary 4 <= q <= 8 (Eq. scale_definition): the
// smallest e with M <= q 2^e, clamped to [-127, 127].  With the bf16 maximum
// M = (1 + F/128) 2^(E-127), e = E - 129 exactly when 1 + F/128 <= q/4, i.e.
// F <= 32 (q - 4); otherwise E - 128 (1 + F/128 < 2 <= q/2).  A power of two
// (F = 0) also satisfies 1 <= q/8 when q = 8 and takes E - 130.  The host
// passes thr = floor(32 (q - 4)) (exact for a binary64 q in [4, 8]) and
// pow2_down = (q == 8).  bf16 maxima below 2^-126 clamp to -127 as above.
struct Boundary {
    int thr;
    int pow2_down;
};

// Host side: the Boundary of q (defined in quantize.hip).
Boundary boundary_of(double q);

__device__ __forceinline__ int scale_exponent_bf16_q(uint32_t mbits, Boundary b) {
    const int E = (int)(mbits >> 7);
    if (E == 0) return -127;
    const int F = (int)(mbits & 0x7Fu);
    int e = E - 129 + (F > b.thr ? 1 : 0) - ((F == 0 && b.pow2_down) ? 1 : 0);
    return e < -127 ? -127 : (e > 127 ? 127 : e);
}

template <int kRule>
__device__ __forceinline__ int block_exponent_bf16(uint32_t mbits, Boundary b) {
    if constexpr (kRule == kRuleQmax)
        return scale_exponent_bf16_q(mbits, b);
    else
        return scale_exponent_bf16<kRule>(mbits);
}

// The fp32 whose exponent field is the E8M0 byte: the scale operand of the
// gfx950 FP4 conversions, which divide by 2^(exponent field - 127).
__device__ __forceinline__ float e8m0_as_f32(uint32_t byte) {
    return __builtin_bit_cast(float, byte << 23);
}

__device__ __forceinline__ v8i fp4_operand(uint4 v) {
    v8i r;
    r[0] = (int)v.x;
    r[1] = (int)v.y;
    r[2] = (int)v.z;
    r[3] = (int)v.w;
    r[4] = 0;
    r[5] = 0;
    r[6] = 0;
    r[7] = 0;
    return r;
}

}  // namespace mxattn
