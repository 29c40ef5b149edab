// Conversion between the canonical 4-bit interchange layout and the
// library's storage layout (both documented in mq.h).
//
// Canonical: one two's-complement code per nibble, two per byte, the even k
// in the low nibble, rows of K/2 bytes in k order; weight scales [N][K/128].
// Library: weights (Wq, Rq) as folded sign-magnitude chunks of 16 codes,
// packed rows of Wq in group order, weight scales [K/128][N], residual blocks
// in their [nnzb][128][64] order; activations (Xq) in the fp6 matrix
// instruction's operand form (act_main_offset / act_tail_offset).
//
// The paper fixes no bit layout (Section 4.2 fuses layout packing with
// quantisation); these conversions let a caller that holds plain int4 codes
// use the fused layer, with the method's codes in [-7, 7] (Eq. (1) with
// q_max = 7).  Offline work: one thread per 16-code chunk.
#include "mq_device.h"

namespace mq {

// 8 canonical bytes (16 nibbles) -> 16 codes; -8 saturates to -7 and is counted
__device__ __forceinline__ int nibbles_to_codes(uint2 v, int (&q)[16]) {
    int bad = 0;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
        const uint32_t w = e < 8 ? v.x : v.y;
        const int nib = (int)((w >> (4 * (e & 7))) & 0xFu);
        int c = nib >= 8 ? nib - 16 : nib;
        if (c == -8) {
            c = -kQmax;
            ++bad;
        }
        q[e] = c;
    }
    return bad;
}

// folded chunk -> 8 canonical bytes
__device__ __forceinline__ uint2 chunk_to_nibbles(uint2 ch) {
    uint32_t lo = 0u, hi = 0u;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
        const uint32_t nib = (uint32_t)chunk_code(ch.x, ch.y, e) & 0xFu;
        if (e < 8) lo |= nib << (4 * e);
        else hi |= nib << (4 * (e - 8));
    }
    return make_uint2(lo, hi);
}

// Packed rows.  Chunk c of row r: canonical bytes 8c of row r (stride ld
// bytes); library bytes piece_offset(rows, r, c / 8) + 8 (c % 8) when GROUPED,
// else 8c of row r (stride K/2: residual blocks).
template <bool TO_LIB, bool GROUPED>
__global__ __launch_bounds__(256) void repack_rows_kernel(const uint8_t* __restrict__ src, uint8_t* __restrict__ dst,
                                                          int rows, int K, int ld, int32_t* __restrict__ n_invalid) {
    const int cpr = K / 16;                                   // chunks per row
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (int64_t)rows * cpr) return;
    const int r = (int)(idx / cpr), c = (int)(idx % cpr);
    const int64_t canon = (int64_t)r * ld + 8 * c;
    const int64_t lib = GROUPED ? piece_offset(rows, r, c / 8) + 8 * (c % 8) : (int64_t)r * (K / 2) + 8 * c;
    if constexpr (TO_LIB) {
        int q[16];
        const int bad = nibbles_to_codes(*reinterpret_cast<const uint2*>(src + canon), q);
        *reinterpret_cast<uint2*>(dst + lib) = fold_codes(q);
        if (bad && n_invalid) atomicAdd(n_invalid, bad);
    } else {
        *reinterpret_cast<uint2*>(dst + canon) = chunk_to_nibbles(*reinterpret_cast<const uint2*>(src + lib));
    }
}

// Activation rows: chunk c of row r (canonical bytes 8c of row r, stride ld)
// <-> half c % 2 of quarter (c / 2) % 4 of group c / 8 in the operand layout
// (dwords d0 .. d2 of the quarter for an even chunk, d3 and the tail d4, d5
// for an odd one).
template <bool TO_LIB>
__global__ __launch_bounds__(256) void repack_act_kernel(const uint8_t* __restrict__ src, uint8_t* __restrict__ dst,
                                                         int rows, int K, int ld, int32_t* __restrict__ n_invalid) {
    const int cpr = K / 16, G = K / kGroup;
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (int64_t)rows * cpr) return;
    const int r = (int)(idx / cpr), c = (int)(idx % cpr);
    const int g = c >> 3, j = (c >> 1) & 3;
    const int64_t canon = (int64_t)r * ld + 8 * c;
    const int64_t main = act_main_offset(rows, r, g) + 16 * j;
    const int64_t tail = act_tail_offset(rows, G, r, g, j);
    if constexpr (TO_LIB) {
        int q[16];
        const int bad = nibbles_to_codes(*reinterpret_cast<const uint2*>(src + canon), q);
        uint32_t o[3];
        code_fields(q, o);
        if ((c & 1) == 0) {
            *reinterpret_cast<uint3*>(dst + main) = make_uint3(o[0], o[1], o[2]);
        } else {
            *reinterpret_cast<uint32_t*>(dst + main + 12) = o[0];
            *reinterpret_cast<uint2*>(dst + tail) = make_uint2(o[1], o[2]);
        }
        if (bad && n_invalid) atomicAdd(n_invalid, bad);
    } else {
        uint32_t o[3];
        if ((c & 1) == 0) {
            const uint3 v = *reinterpret_cast<const uint3*>(src + main);
            o[0] = v.x, o[1] = v.y, o[2] = v.z;
        } else {
            const uint2 t = *reinterpret_cast<const uint2*>(src + tail);
            o[0] = *reinterpret_cast<const uint32_t*>(src + main + 12), o[1] = t.x, o[2] = t.y;
        }
        uint32_t lo = 0u, hi = 0u;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const uint32_t nib = (uint32_t)field_code(o, e) & 0xFu;
            if (e < 8) lo |= nib << (4 * e);
            else hi |= nib << (4 * (e - 8));
        }
        *reinterpret_cast<uint2*>(dst + canon) = make_uint2(lo, hi);
    }
}

// Weight scales: canonical [N][G] <-> library [G][N]
template <bool TO_LIB>
__global__ __launch_bounds__(256) void repack_scales_kernel(const uint16_t* __restrict__ src,
                                                            uint16_t* __restrict__ dst, int N, int G) {
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (int64_t)N * G) return;
    const int n = (int)(idx / G), g = (int)(idx % G);
    if constexpr (TO_LIB) dst[wscale_index(N, n, g)] = src[idx];
    else dst[idx] = src[wscale_index(N, n, g)];
}

// W4A8 activation codes: library layout (e4m3 high plane, folded low plane,
// both in group order) <-> canonical int8 rows [rows, ld].  One thread per 16
// codes; -128 (not a code of the method) is stored as -127 and counted.
template <bool TO_LIB>
__global__ __launch_bounds__(256) void repack_act8_kernel(const uint8_t* __restrict__ src, uint8_t* __restrict__ dst,
                                                          int rows, int K, int ld, int32_t* __restrict__ n_invalid) {
    const int cpr = K / 16;
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (int64_t)rows * cpr) return;
    const int r = (int)(idx / cpr), c = (int)(idx % cpr);
    const int g = c >> 3, cc = c & 7;
    const int64_t canon = (int64_t)r * ld + 16 * c;
    const uint8_t* lib_src = TO_LIB ? nullptr : src;
    uint8_t* lib_dst = TO_LIB ? dst : nullptr;
    const int64_t hi_off = ((int64_t)g * rows + r) * 128 + hi_chunk_offset(cc);
    const int64_t lo_off = (int64_t)rows * K + piece_offset(rows, r, g) + 8 * cc;
    if constexpr (TO_LIB) {
        const uint4 v = *reinterpret_cast<const uint4*>(src + canon);
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
        int l[16], bad = 0;
        uint32_t hb[4] = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            int q = (int)(int8_t)(uint8_t)(w[e >> 2] >> (8 * (e & 3)));
            if (q == -128) {
                q = -kQmax8;
                ++bad;
            }
            const int h = q >> 3;
            l[e] = q - 8 * h;
            hb[e >> 2] |= e4m3_of_int(h) << (8 * (e & 3));
        }
        *reinterpret_cast<uint4*>(lib_dst + hi_off) = make_uint4(hb[0], hb[1], hb[2], hb[3]);
        *reinterpret_cast<uint2*>(lib_dst + lo_off) = fold_codes(l);
        if (bad && n_invalid) atomicAdd(n_invalid, bad);
    } else {
        const uint4 hv = *reinterpret_cast<const uint4*>(lib_src + hi_off);
        const uint2 lv = *reinterpret_cast<const uint2*>(lib_src + lo_off);
        const uint32_t hw[4] = {hv.x, hv.y, hv.z, hv.w};
        uint32_t ow[4] = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const int h = int_of_e4m3((hw[e >> 2] >> (8 * (e & 3))) & 0xFFu);
            const int q = 8 * h + chunk_code(lv.x, lv.y, e);
            ow[e >> 2] |= ((uint32_t)q & 0xFFu) << (8 * (e & 3));
        }
        *reinterpret_cast<uint4*>(dst + canon) = make_uint4(ow[0], ow[1], ow[2], ow[3]);
    }
}

static unsigned blocks_for(int64_t n) { return (unsigned)((n + 255) / 256); }

template <bool TO_LIB, bool GROUPED>
static mq_status rows_launch(const uint8_t* src, uint8_t* dst, int rows, int K, int ld, int32_t* n_invalid,
                             hipStream_t stream) {
    const int64_t n = (int64_t)rows * (K / 16);
    if (n == 0) return MQ_OK;
    hipLaunchKernelGGL((repack_rows_kernel<TO_LIB, GROUPED>), dim3(blocks_for(n)), dim3(256), 0, stream, src, dst,
                       rows, K, ld, n_invalid);
    return mq_host::launch_status();
}

template <bool TO_LIB>
static mq_status act_launch(const uint8_t* src, uint8_t* dst, int rows, int K, int ld, int32_t* n_invalid,
                            hipStream_t stream) {
    const int64_t n = (int64_t)rows * (K / 16);
    if (n == 0) return MQ_OK;
    hipLaunchKernelGGL((repack_act_kernel<TO_LIB>), dim3(blocks_for(n)), dim3(256), 0, stream, src, dst, rows, K,
                       ld, n_invalid);
    return mq_host::launch_status();
}

static bool k_ok(int K) { return K >= 128 && K % 128 == 0 && K <= (1 << 20); }

template <bool TO_LIB>
static mq_status weights(int N, int K, const uint8_t* Wsrc, const void* ssrc, int nnzb, const uint8_t* Rsrc,
                         uint8_t* Wdst, void* sdst, uint8_t* Rdst, int32_t* n_invalid, hipStream_t stream) {
    if (N < 0 || K < 0 || nnzb < 0) return MQ_ERR_INVALID_ARG;
    if (!mq_host::shape_ok(N, K)) return MQ_ERR_UNSUPPORTED_SHAPE;
    if ((int64_t)nnzb > (int64_t)(N / kGroup) * (K / kGroup)) return MQ_ERR_INVALID_ARG;
    if (!Wsrc || !Wdst || (ssrc == nullptr) != (sdst == nullptr) || (nnzb > 0 && (!Rsrc || !Rdst)))
        return MQ_ERR_INVALID_ARG;
    if (!mq_host::aligned(Wsrc, 8) || !mq_host::aligned(Wdst, 16) || (ssrc && !mq_host::aligned(ssrc, 2)) ||
        (sdst && !mq_host::aligned(sdst, 2)) || (Rsrc && !mq_host::aligned(Rsrc, 8)) ||
        (Rdst && !mq_host::aligned(Rdst, 16)) || (n_invalid && !mq_host::aligned(n_invalid, 4)))
        return MQ_ERR_MISALIGNED;
    // the library side must be 16-byte aligned, the canonical side 8-byte
    if (!TO_LIB && (!mq_host::aligned(Wsrc, 16) || (Rsrc && !mq_host::aligned(Rsrc, 16)))) return MQ_ERR_MISALIGNED;
    mq_status st = rows_launch<TO_LIB, true>(Wsrc, Wdst, N, K, K / 2, n_invalid, stream);
    if (st != MQ_OK) return st;
    if (ssrc) {
        const int G = K / kGroup;
        hipLaunchKernelGGL((repack_scales_kernel<TO_LIB>), dim3(blocks_for((int64_t)N * G)), dim3(256), 0, stream,
                           static_cast<const uint16_t*>(ssrc), static_cast<uint16_t*>(sdst), N, G);
        st = mq_host::launch_status();
        if (st != MQ_OK) return st;
    }
    if (nnzb > 0) return rows_launch<TO_LIB, false>(Rsrc, Rdst, nnzb * kGroup, kGroup, kGroup / 2, n_invalid, stream);
    return MQ_OK;
}

}  // namespace mq

using namespace mq;

extern "C" mq_status mq_repack_weights(int N, int K, const uint8_t* Wq_c, const void* s_w_c, int nnzb,
                                       const uint8_t* Rq_c, uint8_t* Wq, void* s_w, uint8_t* Rq,
                                       int32_t* n_invalid, hipStream_t stream) {
    return weights<true>(N, K, Wq_c, s_w_c, nnzb, Rq_c, Wq, s_w, Rq, n_invalid, stream);
}

extern "C" mq_status mq_unpack_weights(int N, int K, const uint8_t* Wq, const void* s_w, int nnzb,
                                       const uint8_t* Rq, uint8_t* Wq_c, void* s_w_c, uint8_t* Rq_c,
                                       hipStream_t stream) {
    return weights<false>(N, K, Wq, s_w, nnzb, Rq, Wq_c, s_w_c, Rq_c, nullptr, stream);
}

extern "C" mq_status mq_repack_act(int M, int K, const uint8_t* Xq_c, int ldq, uint8_t* Xq, int32_t* n_invalid,
                                   hipStream_t stream) {
    if (M < 0 || K < 0) return MQ_ERR_INVALID_ARG;
    if (!k_ok(K) || M > (1 << 24) || ldq < K / 2 || ldq % 8 != 0) return MQ_ERR_UNSUPPORTED_SHAPE;
    if (M == 0) return MQ_OK;
    if (!Xq_c || !Xq) return MQ_ERR_INVALID_ARG;
    if (!mq_host::aligned(Xq_c, 8) || !mq_host::aligned(Xq, 16) || (n_invalid && !mq_host::aligned(n_invalid, 4)))
        return MQ_ERR_MISALIGNED;
    return act_launch<true>(Xq_c, Xq, M, K, ldq, n_invalid, stream);
}

extern "C" mq_status mq_unpack_act(int M, int K, const uint8_t* Xq, uint8_t* Xq_c, int ldq, hipStream_t stream) {
    if (M < 0 || K < 0) return MQ_ERR_INVALID_ARG;
    if (!k_ok(K) || M > (1 << 24) || ldq < K / 2 || ldq % 8 != 0) return MQ_ERR_UNSUPPORTED_SHAPE;
    if (M == 0) return MQ_OK;
    if (!Xq_c || !Xq) return MQ_ERR_INVALID_ARG;
    if (!mq_host::aligned(Xq_c, 8) || !mq_host::aligned(Xq, 16)) return MQ_ERR_MISALIGNED;
    return act_launch<false>(Xq, Xq_c, M, K, ldq, nullptr, stream);
}

extern "C" mq_status mq_repack_act8(int M, int K, const int8_t* Xc, int ldq, uint8_t* Xq8, int32_t* n_invalid,
                                    hipStream_t stream) {
    if (M < 0 || K < 0) return MQ_ERR_INVALID_ARG;
    if (!k_ok(K) || M > (1 << 24) || ldq < K || ldq % 16 != 0) return MQ_ERR_UNSUPPORTED_SHAPE;
    if (M == 0) return MQ_OK;
    if (!Xc || !Xq8) return MQ_ERR_INVALID_ARG;
    if (!mq_host::aligned(Xc, 16) || !mq_host::aligned(Xq8, 16) || (n_invalid && !mq_host::aligned(n_invalid, 4)))
        return MQ_ERR_MISALIGNED;
    const int64_t n = (int64_t)M * (K / 16);
    hipLaunchKernelGGL((repack_act8_kernel<true>), dim3(blocks_for(n)), dim3(256), 0, stream,
                       reinterpret_cast<const uint8_t*>(Xc), Xq8, M, K, ldq, n_invalid);
    return mq_host::launch_status();
}

extern "C" mq_status mq_unpack_act8(int M, int K, const uint8_t* Xq8, int8_t* Xc, int ldq, hipStream_t stream) {
    if (M < 0 || K < 0) return MQ_ERR_INVALID_ARG;
    if (!k_ok(K) || M > (1 << 24) || ldq < K || ldq % 16 != 0) return MQ_ERR_UNSUPPORTED_SHAPE;
    if (M == 0) return MQ_OK;
    if (!Xc || !Xq8) return MQ_ERR_INVALID_ARG;
    if (!mq_host::aligned(Xc, 16) || !mq_host::aligned(Xq8, 16)) return MQ_ERR_MISALIGNED;
    const int64_t n = (int64_t)M * (K / 16);
    hipLaunchKernelGGL((repack_act8_kernel<false>), dim3(blocks_for(n)), dim3(256), 0, stream, Xq8,
                       reinterpret_cast<uint8_t*>(Xc), M, K, ldq, nullptr);
    return mq_host::launch_status();
}
