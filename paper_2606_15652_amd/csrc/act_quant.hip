// Per-token symmetric INT4 activation quantisation fused with code packing
// (Section 2, Eq. (1) applied per row; Section 4.2 "Kernel Fusion": layout
// packing is fused with quantisation).
//
// One workgroup of 256 threads per token row.  Each thread owns 32-byte
// chunks (16 fp16) of the row; the row maximum of |x| is taken on the fp16 bit
// patterns with the sign cleared (an order-preserving integer max for finite
// values, packed 16-bit maxima), reduced across the wave with xor-shuffles and
// across the four waves through LDS.  Codes are then formed from the
// registers (rows up to CPT * 4096 elements) or by re-reading the row (longer
// rows), with the division-free exact rounding of quant_mag, and written in
// the matrix instruction's operand form (act_main_offset / act_tail_offset):
// the 16 codes of an even chunk are dwords d0 .. d2 of their quarter, those of
// the odd chunk d3 .. d5.  The pair of threads of a quarter exchange d3, so
// that the even thread writes the quarter's 16 main-plane bytes and the odd
// one its 8 tail bytes (the quarters of a group are then 64 and 32 contiguous
// bytes).
#include "mq_device.h"

namespace mq {

constexpr int kActThreads = 256;

// Row of workgroup b.  Workgroups go to the eight XCDs in turn (b % 8), and
// neighbouring rows share the 128-byte lines of the operand planes (a row
// writes 64 and 32 bytes of each group's main and tail pieces), so each XCD
// takes a contiguous range of rows: the lines are then written whole from one
// L2.  A bijection on [0, M): XCD x holds rows x per + min(x, rem) on.
__device__ __forceinline__ int xcd_row(int b, int M) {
    const int x = b % 8, k = b / 8, per = M / 8, rem = M % 8;
    return x * per + min(x, rem) + k;
}

// CPT > 0: the row stays in registers (CPT chunks per thread); CPT == 0: the
// row is read twice.
template <int CPT>
__global__ __launch_bounds__(kActThreads) void act_quant_kernel(
    const uint16_t* __restrict__ X, int M, int K, int ldx,
    uint8_t* __restrict__ Xq, uint16_t* __restrict__ s_x) {
    __shared__ uint32_t red[kActThreads / 64];
    const int m = xcd_row(blockIdx.x, M);
    const int t = threadIdx.x;
    const uint16_t* row = X + (int64_t)m * ldx;
    const int nchunks = K / 16, G = K / 128;
    // chunk c (codes 16c .. 16c+15) is half c % 2 of quarter (c / 2) % 4 of group c / 8
    // (both threads of a pair are active or neither: K / 16 is even)
    auto store = [&](int c, const uint4 v0, const uint4 v1, float s, float inv_s) {
        uint32_t o0, o1, o2;
        quant_fields(v0, v1, s, inv_s, o0, o1, o2);
        const uint32_t d3 = __shfl_down(o0, 1, 64);          // the odd neighbour's o0
        const int g = c >> 3, j = (c >> 1) & 3;
        if ((c & 1) == 0)
            *reinterpret_cast<uint4*>(Xq + act_main_offset(M, m, g) + 16 * j) = make_uint4(o0, o1, o2, d3);
        else
            *reinterpret_cast<uint2*>(Xq + act_tail_offset(M, G, m, g, j)) = make_uint2(o1, o2);
    };

    uint32_t amax = 0;
    uint4 v[CPT > 0 ? CPT : 1][2];
    if constexpr (CPT > 0) {
#pragma unroll
        for (int i = 0; i < CPT; ++i) {
            const int c = t + i * kActThreads;
            if (c < nchunks) {
                v[i][0] = *reinterpret_cast<const uint4*>(row + 16 * c);
                v[i][1] = *reinterpret_cast<const uint4*>(row + 16 * c + 8);
                const uint32_t cm = chunk_absmax_bits(v[i][0], v[i][1]);
                amax = cm > amax ? cm : amax;
            }
        }
    } else {
        for (int c = t; c < nchunks; c += kActThreads) {
            const uint32_t cm = chunk_absmax_bits(*reinterpret_cast<const uint4*>(row + 16 * c),
                                                  *reinterpret_cast<const uint4*>(row + 16 * c + 8));
            amax = cm > amax ? cm : amax;
        }
    }
    amax = wave_max_u32(amax);
    if ((t & 63) == 0) red[t >> 6] = amax;
    __syncthreads();
    amax = red[0];
#pragma unroll
    for (int w = 1; w < kActThreads / 64; ++w) amax = red[w] > amax ? red[w] : amax;

    const uint16_t sb = scale_bits_from_amax(half_bits_to_float((uint16_t)amax));
    const float s = half_bits_to_float(sb);
    const float inv_s = 1.0f / s;
    if (t == 0) s_x[m] = sb;

    if constexpr (CPT > 0) {
#pragma unroll
        for (int i = 0; i < CPT; ++i) {
            const int c = t + i * kActThreads;
            if (c < nchunks) store(c, v[i][0], v[i][1], s, inv_s);
        }
    } else {
        for (int c = t; c < nchunks; c += kActThreads)
            store(c, *reinterpret_cast<const uint4*>(row + 16 * c), *reinterpret_cast<const uint4*>(row + 16 * c + 8),
                  s, inv_s);
    }
}

// ---------------------------------------------------------------------------
// W4A8: per-token symmetric INT8 codes (Eq. (1) with q_max = 127; the W4A8
// setting of the appendix "Implementation Details", per-token dynamic
// activation quantisation), written as x = 8 h + l: the e4m3 bytes of h in
// the high plane (piece (row, group) of 128 bytes at (g M + m) 128, chunks
// placed by hi_chunk_offset) and the
// folded 4-bit codes l in [0, 7] in the low plane (M K bytes on, the W4A4
// group order).  Same row structure as act_quant_kernel.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void quant8_chunk(const uint4 v0, const uint4 v1, float s, float inv_s,
                                             uint4& hi, uint2& lo) {
    const uint32_t w[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
    int l[16];
    uint32_t hb[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int e = 0; e < 16; ++e) {
        const float x = half_bits_to_float((uint16_t)(e & 1 ? w[e >> 1] >> 16 : w[e >> 1] & 0xFFFFu));
        const int q = s == 0.0f ? 0 : quant_code_max(x, s, inv_s, kQmax8);
        const int h = q >> 3;                                    // floor(q / 8)
        l[e] = q - 8 * h;
        hb[e >> 2] |= e4m3_of_int(h) << (8 * (e & 3));
    }
    hi = make_uint4(hb[0], hb[1], hb[2], hb[3]);
    lo = fold_codes(l);
}

template <int CPT>
__global__ __launch_bounds__(kActThreads) void act_quant8_kernel(
    const uint16_t* __restrict__ X, int M, int K, int ldx,
    uint8_t* __restrict__ Xq8, uint16_t* __restrict__ s_x) {
    __shared__ uint32_t red[kActThreads / 64];
    const int m = xcd_row(blockIdx.x, M);
    const int t = threadIdx.x;
    const uint16_t* row = X + (int64_t)m * ldx;
    const int nchunks = K / 16;
    uint8_t* lo_plane = Xq8 + (int64_t)M * K;
    auto store = [&](int c, const uint4 v0, const uint4 v1, float s, float inv_s) {
        uint4 hi;
        uint2 lo;
        quant8_chunk(v0, v1, s, inv_s, hi, lo);
        const int g = c >> 3, cc = c & 7;
        *reinterpret_cast<uint4*>(Xq8 + ((int64_t)g * M + m) * 128 + hi_chunk_offset(cc)) = hi;
        *reinterpret_cast<uint2*>(lo_plane + piece_offset(M, m, g) + 8 * cc) = lo;
    };

    uint32_t amax = 0;
    uint4 v[CPT > 0 ? CPT : 1][2];
    if constexpr (CPT > 0) {
#pragma unroll
        for (int i = 0; i < CPT; ++i) {
            const int c = t + i * kActThreads;
            if (c < nchunks) {
                v[i][0] = *reinterpret_cast<const uint4*>(row + 16 * c);
                v[i][1] = *reinterpret_cast<const uint4*>(row + 16 * c + 8);
                const uint32_t cm = chunk_absmax_bits(v[i][0], v[i][1]);
                amax = cm > amax ? cm : amax;
            }
        }
    } else {
        for (int c = t; c < nchunks; c += kActThreads) {
            const uint32_t cm = chunk_absmax_bits(*reinterpret_cast<const uint4*>(row + 16 * c),
                                                  *reinterpret_cast<const uint4*>(row + 16 * c + 8));
            amax = cm > amax ? cm : amax;
        }
    }
    amax = wave_max_u32(amax);
    if ((t & 63) == 0) red[t >> 6] = amax;
    __syncthreads();
    amax = red[0];
#pragma unroll
    for (int w = 1; w < kActThreads / 64; ++w) amax = red[w] > amax ? red[w] : amax;

    const uint16_t sb = scale_bits_from_amax(half_bits_to_float((uint16_t)amax), kQmax8);
    const float s = half_bits_to_float(sb);
    const float inv_s = 1.0f / s;
    if (t == 0) s_x[m] = sb;

    if constexpr (CPT > 0) {
#pragma unroll
        for (int i = 0; i < CPT; ++i) {
            const int c = t + i * kActThreads;
            if (c < nchunks) store(c, v[i][0], v[i][1], s, inv_s);
        }
    } else {
        for (int c = t; c < nchunks; c += kActThreads)
            store(c, *reinterpret_cast<const uint4*>(row + 16 * c), *reinterpret_cast<const uint4*>(row + 16 * c + 8),
                  s, inv_s);
    }
}

}  // namespace mq

using namespace mq;

extern "C" mq_status mq_quantize_act8(const void* X, int M, int K, int ldx,
                                      uint8_t* Xq8, void* s_x, hipStream_t stream) {
    if (M < 0 || K < 0) return MQ_ERR_INVALID_ARG;
    if (M > (1 << 24) || K < 128 || K % 128 != 0 || K > (1 << 20) || ldx < K || ldx % 8 != 0)
        return MQ_ERR_UNSUPPORTED_SHAPE;
    if (M == 0) return MQ_OK;
    if (!X || !Xq8 || !s_x) return MQ_ERR_INVALID_ARG;
    if (!mq_host::aligned(X, 16) || !mq_host::aligned(Xq8, 16) || !mq_host::aligned(s_x, 2))
        return MQ_ERR_MISALIGNED;
    const auto* x = static_cast<const uint16_t*>(X);
    auto* s = static_cast<uint16_t*>(s_x);
    const int chunks_per_thread = (K / 16 + kActThreads - 1) / kActThreads;
    dim3 grid(M), block(kActThreads);
    if (chunks_per_thread <= 1)
        hipLaunchKernelGGL(act_quant8_kernel<1>, grid, block, 0, stream, x, M, K, ldx, Xq8, s);
    else if (chunks_per_thread <= 2)
        hipLaunchKernelGGL(act_quant8_kernel<2>, grid, block, 0, stream, x, M, K, ldx, Xq8, s);
    else if (chunks_per_thread <= 4)
        hipLaunchKernelGGL(act_quant8_kernel<4>, grid, block, 0, stream, x, M, K, ldx, Xq8, s);
    else if (chunks_per_thread <= 8)
        hipLaunchKernelGGL(act_quant8_kernel<8>, grid, block, 0, stream, x, M, K, ldx, Xq8, s);
    else
        hipLaunchKernelGGL(act_quant8_kernel<0>, grid, block, 0, stream, x, M, K, ldx, Xq8, s);
    return mq_host::launch_status();
}

extern "C" mq_status mq_quantize_act(const void* X, int M, int K, int ldx,
                                     uint8_t* Xq, void* s_x, hipStream_t stream) {
    if (M < 0 || K < 0) return MQ_ERR_INVALID_ARG;
    if (M > (1 << 24) || K < 128 || K % 128 != 0 || K > (1 << 20) || ldx < K || ldx % 8 != 0)
        return MQ_ERR_UNSUPPORTED_SHAPE;
    if (M == 0) return MQ_OK;
    if (!X || !Xq || !s_x) return MQ_ERR_INVALID_ARG;
    if (!mq_host::aligned(X, 16) || !mq_host::aligned(Xq, 16) || !mq_host::aligned(s_x, 2))
        return MQ_ERR_MISALIGNED;
    const auto* x = static_cast<const uint16_t*>(X);
    auto* s = static_cast<uint16_t*>(s_x);
    const int chunks_per_thread = (K / 16 + kActThreads - 1) / kActThreads;
    dim3 grid(M), block(kActThreads);
    if (chunks_per_thread <= 1)
        hipLaunchKernelGGL(act_quant_kernel<1>, grid, block, 0, stream, x, M, K, ldx, Xq, s);
    else if (chunks_per_thread <= 2)
        hipLaunchKernelGGL(act_quant_kernel<2>, grid, block, 0, stream, x, M, K, ldx, Xq, s);
    else if (chunks_per_thread <= 4)
        hipLaunchKernelGGL(act_quant_kernel<4>, grid, block, 0, stream, x, M, K, ldx, Xq, s);
    else if (chunks_per_thread <= 8)
        hipLaunchKernelGGL(act_quant_kernel<8>, grid, block, 0, stream, x, M, K, ldx, Xq, s);
    else if (chunks_per_thread <= 16)
        hipLaunchKernelGGL(act_quant_kernel<16>, grid, block, 0, stream, x, M, K, ldx, Xq, s);
    else
        hipLaunchKernelGGL(act_quant_kernel<0>, grid, block, 0, stream, x, M, K, ldx, Xq, s);
    return mq_host::launch_status();
}
