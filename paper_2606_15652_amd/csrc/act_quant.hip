// Per-token symmetric INT4 activation quantisation fused with nibble packing
// (Section 2, Eq. (1) applied per row; Section 4.2 "Kernel Fusion": layout
// packing is fused with quantisation).
//
// One workgroup of 256 threads per token row.  Each thread owns 16-byte
// chunks (8 fp16) of the row; the row maximum of |x| is taken on the fp16 bit
// patterns with the sign cleared (an order-preserving integer max for finite
// values), reduced across the wave with xor-shuffles and across the four waves
// through LDS.  Codes are then formed from the registers (rows up to
// CPT * 2048 elements) or by re-reading the row (longer rows), and written as
// 4 packed bytes per chunk: fully coalesced 16-byte loads, 4-byte stores.
#include "mq_device.h"

namespace mq {

constexpr int kActThreads = 256;

__device__ __forceinline__ uint32_t chunk_absmax_bits(const uint4 v) {
    uint32_t m = 0;
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        uint32_t lo = w[i] & 0x7FFFu, hi = (w[i] >> 16) & 0x7FFFu;
        m = lo > m ? lo : m;
        m = hi > m ? hi : m;
    }
    return m;
}

// 8 fp16 -> 8 codes -> 4 packed bytes (element 2j low nibble, 2j+1 high).
__device__ __forceinline__ uint32_t quant_chunk(const uint4 v, float s) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    uint32_t out = 0;
    if (s == 0.0f) return 0u;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        int q0 = quant_code(half_bits_to_float((uint16_t)(w[i] & 0xFFFFu)), s);
        int q1 = quant_code(half_bits_to_float((uint16_t)(w[i] >> 16)), s);
        uint32_t byte = ((uint32_t)q0 & 0xFu) | (((uint32_t)q1 & 0xFu) << 4);
        out |= byte << (8 * i);
    }
    return out;
}

// CPT > 0: the row stays in registers (CPT chunks per thread); CPT == 0: the
// row is read twice.
template <int CPT>
__global__ __launch_bounds__(kActThreads) void act_quant_kernel(
    const uint16_t* __restrict__ X, int K, int ldx,
    uint8_t* __restrict__ Xq, uint16_t* __restrict__ s_x) {
    __shared__ uint32_t red[kActThreads / 64];
    const int m = blockIdx.x;
    const int t = threadIdx.x;
    const uint16_t* row = X + (int64_t)m * ldx;
    uint32_t* out = reinterpret_cast<uint32_t*>(Xq + (int64_t)m * (K / 2));
    const int nchunks = K / 8;

    uint32_t amax = 0;
    uint4 v[CPT > 0 ? CPT : 1];
    if constexpr (CPT > 0) {
#pragma unroll
        for (int i = 0; i < CPT; ++i) {
            const int c = t + i * kActThreads;
            if (c < nchunks) {
                v[i] = *reinterpret_cast<const uint4*>(row + 8 * c);
                const uint32_t cm = chunk_absmax_bits(v[i]);
                amax = cm > amax ? cm : amax;
            }
        }
    } else {
        for (int c = t; c < nchunks; c += kActThreads) {
            const uint32_t cm = chunk_absmax_bits(*reinterpret_cast<const uint4*>(row + 8 * c));
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
    if (t == 0) s_x[m] = sb;

    if constexpr (CPT > 0) {
#pragma unroll
        for (int i = 0; i < CPT; ++i) {
            const int c = t + i * kActThreads;
            if (c < nchunks) out[c] = quant_chunk(v[i], s);
        }
    } else {
        for (int c = t; c < nchunks; c += kActThreads)
            out[c] = quant_chunk(*reinterpret_cast<const uint4*>(row + 8 * c), s);
    }
}

}  // namespace mq

using namespace mq;

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
    const int chunks_per_thread = (K / 8 + kActThreads - 1) / kActThreads;
    dim3 grid(M), block(kActThreads);
    if (chunks_per_thread <= 1)
        hipLaunchKernelGGL(act_quant_kernel<1>, grid, block, 0, stream, x, K, ldx, Xq, s);
    else if (chunks_per_thread <= 2)
        hipLaunchKernelGGL(act_quant_kernel<2>, grid, block, 0, stream, x, K, ldx, Xq, s);
    else if (chunks_per_thread <= 4)
        hipLaunchKernelGGL(act_quant_kernel<4>, grid, block, 0, stream, x, K, ldx, Xq, s);
    else if (chunks_per_thread <= 8)
        hipLaunchKernelGGL(act_quant_kernel<8>, grid, block, 0, stream, x, K, ldx, Xq, s);
    else if (chunks_per_thread <= 16)
        hipLaunchKernelGGL(act_quant_kernel<16>, grid, block, 0, stream, x, K, ldx, Xq, s);
    else
        hipLaunchKernelGGL(act_quant_kernel<0>, grid, block, 0, stream, x, K, ldx, Xq, s);
    return mq_host::launch_status();
}
