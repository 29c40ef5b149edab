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

typedef int32_t i32x2 __attribute__((ext_vector_type(2)));
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
__device__ __forceinline__ uint16_t scale_bits_from_amax(float amax, int qmax = kQmax) {
    return float_to_half_bits(amax / (float)qmax);
}

// |code| of an fp16 x for an fp16 scale s > 0 (the activation quantiser):
// min(7, round_half_even(|x| / s)), given inv_s = the correctly rounded fp32
// 1 / s.  x and s are fp16 values, so a
// quotient that is not a tie lies at least 2^-14 from every half-integer
// (2|x| - (2k+1) s is a non-zero multiple of the finer of the two exponents'
// units).  q0 = |x| inv_s is within 2^-20 of |x| / s; one correction step
// (r = |x| - q0 s is exact: on a tie q0 - (k + 1/2) is a few units of the
// last place, times s representable) makes q1 exactly k + 1/2 on a tie and
// keeps it within 2^-22 otherwise, so rint (ties to even) gives the code.
__device__ __forceinline__ float quant_mag(float ax, float s, float inv_s) {
    const float q0 = ax * inv_s;
    const float r = __builtin_fmaf(-q0, s, ax);
    const float q1 = __builtin_fmaf(r, inv_s, q0);
    return fminf(rintf(q1), (float)kQmax);
}

// Code of x for scale s > 0 (inv_s = 1 / s, rounded any way):
// clamp(round_half_even(x / s), -7, 7).
// x is fp16 or fp32 and s is fp16, so the tie points t*s (t = k + 1/2) have at
// most 15 significant bits: an x that is not a tie lies at least 2^-24
// (relative) away from one, more than half an fp32 ulp at t, so rounding the
// exact quotient (below) gives what the correctly rounded fp32 quotient does.
// No division: q = rint(x * inv_s) is within one of the result; e = x - q s
// is exact (an fma: for q != 0 both terms are multiples of half an ulp of s
// and |e| is at most about s; for q = 0, e = x); comparing |e| with s/2
// (exact) moves q to the nearest integer, ties to the even one.
// (The argument does not depend on the size of q: it holds for the INT8
// activation codes of the W4A8 variant, qmax = 127, as well.)
__device__ __forceinline__ int quant_code_max(float x, float s, float inv_s, int qmax) {
    float q = rintf(x * inv_s);
    const float e = __builtin_fmaf(-q, s, x);
    const float h = 0.5f * s;
    const float ae = fabsf(e);
    const bool odd = ((int)q & 1) != 0;
    if (ae > h || (ae == h && odd)) q += e > 0.f ? 1.f : -1.f;
    q = fminf(fmaxf(q, -(float)qmax), (float)qmax);
    return (int)q;
}
__device__ __forceinline__ int quant_code(float x, float s, float inv_s) {
    return quant_code_max(x, s, inv_s, kQmax);
}

// --------------------------------------------------- W4A8 activation codes --
// An INT8 code x in [-127, 127] is stored as x = 8 h + l with h = floor(x / 8)
// in [-16, 15] and l in [0, 7]: h as an fp8 e4m3 byte (every integer up to 16
// in magnitude is exact), l as a folded 4-bit code (e2m3 subnormal l / 8).
// The matrix instruction then sums h (q/8) and (l/8)(q/8) exactly, and the
// two products chained give the group sum / 64 as for W4A4.
constexpr int kQmax8 = 127;
// Byte offset, inside the 128-byte high-plane piece of a row and group, of the
// 16-code chunk c (codes 16c .. 16c + 15).  A lane of the matrix instruction
// reads 32 bytes at 32 (l / 16) and, for an fp8 operand, takes them as the
// codes 16 (l / 16) + 0..15 and 64 + 16 (l / 16) + 0..15 of the group (the
// pairing with the fp6 operand's codes 32 (l / 16) + 0..31 of the folded
// layout, measured on the GPU by the raw-sum parity tests).
__device__ __forceinline__ int hi_chunk_offset(int c) { return 32 * (c & 3) + 16 * (c >> 2); }

// e4m3 byte of an integer h with |h| <= 16 (sign, exponent bias 7, 3 mantissa bits)
__device__ __forceinline__ uint32_t e4m3_of_int(int h) {
    const uint32_t a = (uint32_t)(h < 0 ? -h : h);
    if (a == 0u) return 0u;
    const int e = 31 - __builtin_clz(a);
    const uint32_t m = ((a << 3) >> e) & 7u;
    return (h < 0 ? 0x80u : 0u) | ((uint32_t)(e + 7) << 3) | m;
}
// integer value of an e4m3 byte written by e4m3_of_int
__device__ __forceinline__ int int_of_e4m3(uint32_t b) {
    if ((b & 0x7Fu) == 0u) return 0;
    const int e = (int)((b >> 3) & 15u) - 7;
    const int a = (int)(((8u + (b & 7u)) << e) >> 3);
    return (b & 0x80u) ? -a : a;
}

// ---------------------------------------------------------- packed codes --
// Storage of 4-bit codes (q in [-7, 7]): a row of K codes is K/16 chunks of
// 8 bytes, chunk c holding codes 16c .. 16c + 15.  Code e of a chunk is the
// 6-bit field f = 32 [q < 0] + |q| at bit 6e of a 96-bit word (o0, o1, o2);
// read as an fp6 e2m3 value a field with zero exponent is the subnormal
// sign * |q| / 8, so a chunk expands into MFMA operand dwords with a mask per
// word.  The two exponent bits of every field are zero, and those of o0 (kFoldA)
// and of o1 (kFoldB) together are exactly the bits o2 can use, so the chunk is
// stored folded as  P0 = o0 | (o2 & kFoldA),  P1 = o1 | (o2 & kFoldB).
constexpr uint32_t kFoldA = 0x18618618u;   // bits 6e+3, 6e+4 inside word 0
constexpr uint32_t kFoldB = 0x86186186u;   // bits 6e+3, 6e+4 inside word 1

typedef int32_t i32x8 __attribute__((ext_vector_type(8)));

// 16 codes -> the 96-bit word (o0, o1, o2) of their 6-bit fields
__device__ __forceinline__ void code_fields(const int (&q)[16], uint32_t (&o)[3]) {
    o[0] = o[1] = o[2] = 0u;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
        const uint32_t f = (q[e] < 0 ? 32u : 0u) | (uint32_t)(q[e] < 0 ? -q[e] : q[e]);
        const int bit = 6 * e, w = bit >> 5, off = bit & 31;
        o[w] |= f << off;
        if (off > 26) o[w + 1] |= f >> (32 - off);
    }
}

// 16 codes -> one folded chunk (quantisers)
__device__ __forceinline__ uint2 fold_codes(const int (&q)[16]) {
    uint32_t o[3];
    code_fields(q, o);
    return make_uint2(o[0] | (o[2] & kFoldA), o[1] | (o[2] & kFoldB));
}

// code e (0..15) of a 96-bit field word
__device__ __forceinline__ int field_code(const uint32_t (&o)[3], int e) {
    const int bit = 6 * e, w = bit >> 5, off = bit & 31;
    uint32_t f = o[w] >> off;
    if (off > 26) f |= o[w + 1] << (32 - off);
    const int mag = (int)(f & 7u);
    return (f & 32u) ? -mag : mag;
}

// code e (0..15) of a folded chunk
__device__ __forceinline__ int chunk_code(uint32_t p0, uint32_t p1, int e) {
    const uint32_t o[3] = {p0 & ~kFoldA, p1 & ~kFoldB, (p0 & kFoldA) | (p1 & kFoldB)};
    return field_code(o, e);
}

// 16 bytes = two chunks (32 codes) -> the six e2m3 dwords of one MFMA lane
// operand (dwords 6, 7 unused): 4 bit operations per chunk.
__device__ __forceinline__ i32x8 unfold_codes(const uint4 p) {
    return i32x8{(int)(p.x & ~kFoldA), (int)(p.y & ~kFoldB), (int)((p.x & kFoldA) | (p.y & kFoldB)),
                 (int)(p.z & ~kFoldA), (int)(p.w & ~kFoldB), (int)((p.z & kFoldA) | (p.w & kFoldB)),
                 0, 0};
}

// D = A (16 x 128) B^T + C in fp32 on e2m3 operands: lane l supplies row l%16
// of A and of B for its quarter l/16 of K (32 codes, one 16-byte pair of
// chunks) and receives D[4 * (l/16) + r][l%16], r = 0..3.  Products of codes
// are exact and so is their sum: D = (sum of code products) / 64.
__device__ __forceinline__ f32x4 mfma_codes(const i32x8 a, const i32x8 b, const f32x4 c) {
    return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 2, 2, 0, 0, 0, 0);
}
// the same with A given as 32 e4m3 bytes per lane (eight dwords, k order):
// D = A (16 x 128, fp8) B^T (fp6 codes) + C
__device__ __forceinline__ f32x4 mfma_e4m3_codes(const i32x8 a, const i32x8 b, const f32x4 c) {
    return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 2, 0, 0, 0, 0);
}
// removes the 1/64 of the e2m3 encoding (exact)
constexpr float kCodeScale = 64.0f;

// ------------------------------------------------- activation quantiser --
// Largest |x| of 8 fp16 values, as fp16 bits with the sign cleared (an
// order-preserving integer maximum for finite values): packed 16-bit maxima.
typedef uint16_t u16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ u16x2 abs_bits2(uint32_t w) {
    return __builtin_bit_cast(u16x2, w & 0x7FFF7FFFu);
}
__device__ __forceinline__ u16x2 chunk_absmax2(const uint4 v) {
    return __builtin_elementwise_max(__builtin_elementwise_max(abs_bits2(v.x), abs_bits2(v.y)),
                                     __builtin_elementwise_max(abs_bits2(v.z), abs_bits2(v.w)));
}
__device__ __forceinline__ uint32_t chunk_absmax_bits(const uint4 v) {
    const u16x2 m = chunk_absmax2(v);
    return m.x > m.y ? m.x : m.y;
}
// the same over two 16-byte loads (16 fp16)
__device__ __forceinline__ uint32_t chunk_absmax_bits(const uint4 v0, const uint4 v1) {
    const u16x2 m = __builtin_elementwise_max(chunk_absmax2(v0), chunk_absmax2(v1));
    return m.x > m.y ? m.x : m.y;
}

// 16 fp16 (two 16-byte loads) -> 16 codes for scale s (inv_s = 1 / s) -> one
// folded chunk.  Each 6-bit field is the code's magnitude with x's sign bit
// at bit 5 when the code is not zero (as fold_codes writes it), laid out at
// bit 6e of the 96-bit word and folded.
__device__ __forceinline__ uint32_t code_field(uint32_t h16, float s, float inv_s) {
    // quant_mag's steps on the signed value (every step is sign-symmetric);
    // adding +0 turns a negative zero into +0, so the sign bit of q is set
    // exactly for the negative codes
    const float x = half_bits_to_float((uint16_t)h16);
    const float q0 = x * inv_s;
    const float r = __builtin_fmaf(-q0, s, x);
    const float q = rintf(__builtin_fmaf(r, inv_s, q0)) + 0.0f;
    const uint32_t m = min((uint32_t)fabsf(q), (uint32_t)kQmax);
    return m | ((__float_as_uint(q) >> 31) << 5);
}
// 16 fp16 -> the 96-bit word (o0, o1, o2) of their 6-bit code fields
__device__ __forceinline__ void quant_fields(const uint4 v0, const uint4 v1, float s, float inv_s,
                                             uint32_t& o0, uint32_t& o1, uint32_t& o2) {
    if (s == 0.0f) {
        o0 = o1 = o2 = 0u;
        return;
    }
    const uint32_t w[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
    uint32_t f[16];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        f[2 * i] = code_field(w[i] & 0xFFFFu, s, inv_s);
        f[2 * i + 1] = code_field(w[i] >> 16, s, inv_s);
    }
    o0 = f[0] | (f[1] << 6) | (f[2] << 12) | (f[3] << 18) | (f[4] << 24) | (f[5] << 30);
    o1 = (f[5] >> 2) | (f[6] << 4) | (f[7] << 10) | (f[8] << 16) | (f[9] << 22) | (f[10] << 28);
    o2 = (f[10] >> 4) | (f[11] << 2) | (f[12] << 8) | (f[13] << 14) | (f[14] << 20) | (f[15] << 26);
}
__device__ __forceinline__ uint2 quant_chunk(const uint4 v0, const uint4 v1, float s, float inv_s) {
    uint32_t o0, o1, o2;
    quant_fields(v0, v1, s, inv_s, o0, o1, o2);
    return make_uint2(o0 | (o2 & kFoldA), o1 | (o2 & kFoldB));
}

// ----------------------------------------------------- device group order --
// Packed rows (Xq, Wq) are stored group-major: the 64-byte piece of row r and
// 128-code group g sits at byte (g rows + r) 64, so every 128-row x 128-code
// tile is one contiguous run and the tiles of neighbouring row blocks are
// neighbours in memory.  Weight scales are stored [K/128][N]: s_w of (row n,
// group g) at element g N + n, 256 contiguous bytes per tile.
__device__ __forceinline__ int64_t piece_offset(int rows, int r, int g) {
    return ((int64_t)g * rows + r) * kGroupBytes;
}
__device__ __forceinline__ int64_t wscale_index(int N, int n, int g) {
    return (int64_t)g * N + n;
}

// ------------------------------------------------ activation operand order --
// Activation codes (Xq of mq_quantize_act) are stored in the matrix
// instruction's operand form, so the GEMMs read them with no bit work: the
// 32 codes of quarter j (codes 32j .. 32j + 31 of a 128-code group) are one
// 192-bit word of their 6-bit fields (code e at bit 6e, the fields of the
// packed layout, not folded), six dwords d0 .. d5.  Main plane: d0 .. d3 of
// quarter j of (row r, group g) at byte (g M + r) 64 + 16 j; tail plane, from
// byte G M 64 on: d4, d5 at byte G M 64 + (g M + r) 32 + 8 j.  A 16-row piece
// of the main plane is 1 KB contiguous, like the packed rows, and so are the
// tails of 32 rows.
constexpr int kActGroupBytes = 96;   // bytes of one group of one row (64 main + 32 tail)
__device__ __forceinline__ int64_t act_main_offset(int M, int r, int g) {
    return ((int64_t)g * M + r) * 64;
}
__device__ __forceinline__ int64_t act_tail_offset(int M, int G, int r, int g, int j) {
    return (int64_t)G * M * 64 + ((int64_t)g * M + r) * 32 + 8 * j;
}
// the operand of quarter j from its main (d0 .. d3) and tail (d4, d5) parts
__device__ __forceinline__ i32x8 act_operand(const uint4 m, const uint2 t) {
    return i32x8{(int)m.x, (int)m.y, (int)m.z, (int)m.w, (int)t.x, (int)t.y, 0, 0};
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
