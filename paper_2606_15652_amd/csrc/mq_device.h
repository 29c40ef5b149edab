// Internal device helpers of libmq (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>
#include <stdint.h>

#include "mq.h"

namespace mq {

constexpr int kGroup = 128;       // weight group length along K == residual block edge
constexpr int kGroupBytes = 64;   // packed bytes of one group of one row
constexpr int kQmax = 7;

typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- scalars --
__device__ __forceinline__ float half_bits_to_float(uint16_t b) {
    return __half2float(__ushort_as_half(b));
}
__device__ __forceinline__ uint16_t float_to_half_bits(float f) {
    return __half_as_ushort(__float2half_rn(f));
}

// Scale of a symmetric 4-bit quantiser with row/group maximum `amax`:
// fp16_rn(fp32(amax) / 7).  The library is built with correctly rounded fp32
// division (-fhip-fp32-correctly-rounded-divide-sqrt, no fast-math).
__device__ __forceinline__ uint16_t scale_bits_from_amax(float amax) {
    return float_to_half_bits(amax / (float)kQmax);
}

// Code of x for scale s (s != 0): clamp(round_half_even(x / s), -7, 7).
// x is fp16 or fp32 and s is fp16, so the tie points t*s (t = k + 1/2) have at
// most 15 significant bits: an x that is not a tie lies at least 2^-24
// (relative) away from one, more than half an fp32 ulp at t, so the correctly
// rounded fp32 quotient rounds exactly as the real quotient does.
__device__ __forceinline__ int quant_code(float x, float s) {
    float r = rintf(x / s);
    r = fminf(fmaxf(r, -(float)kQmax), (float)kQmax);
    return (int)r;
}

// ------------------------------------------------------------------ unpack --
// 16 packed bytes (32 nibbles, elements 2j in low and 2j+1 in high nibbles)
// -> two MFMA operands of 16 int8 each, holding 16 * code:
//   lo = the even elements, hi = the odd elements (same byte positions).
// Masking the high nibble in place yields 16 * (signed code) as an int8, and
// shifting the low nibble up by 4 does the same for the even element, so the
// integer products are 256x the code products; callers remove the factor.
__device__ __forceinline__ void unpack_nibbles(const uint4 p, i32x4& lo, i32x4& hi) {
    const uint32_t m = 0xF0F0F0F0u;
    hi = i32x4{(int)(p.x & m), (int)(p.y & m), (int)(p.z & m), (int)(p.w & m)};
    lo = i32x4{(int)((p.x << 4) & m), (int)((p.y << 4) & m),
               (int)((p.z << 4) & m), (int)((p.w << 4) & m)};
}

// D = A(16x64 int8) * B(64x16 int8) + C, int32.  Lane l supplies row l%16 of A
// and column l%16 of B for its quarter (l/16) of K; it receives
// D[4*(l/16) + r][l%16], r = 0..3.
__device__ __forceinline__ i32x4 mfma_i8(const i32x4 a, const i32x4 b, const i32x4 c) {
    return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ uint4 ldg16(const uint8_t* p) {
    return *reinterpret_cast<const uint4*>(p);
}

__device__ __forceinline__ uint16_t ldg_u16(const void* base, int64_t idx) {
    return reinterpret_cast<const uint16_t*>(base)[idx];
}

// ----------------------------------------------------------- reductions --
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
    for (int off = 32; off > 0; off >>= 1) {
        uint32_t o = __shfl_xor(v, off, 64);
        v = o > v ? o : v;
    }
    return v;
}

}  // namespace mq

// Host-side helpers shared by the API translation units.
namespace mq_host {

inline bool aligned(const void* p, size_t a) {
    return (reinterpret_cast<uintptr_t>(p) % a) == 0;
}

inline bool shape_ok(int N, int K) {
    return K >= 128 && N >= 128 && (K % 128) == 0 && (N % 128) == 0 &&
           K <= (1 << 20) && N <= (1 << 24);
}

inline mq_status launch_status() {
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? MQ_OK : MQ_ERR_HIP;
}

}  // namespace mq_host
