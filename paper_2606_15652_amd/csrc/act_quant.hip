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
// rows), with the division-free exact rounding of quant_mag, and written as
// one folded 8-byte chunk per 16 codes in the device group order
// (piece_offset): coalesced 16-byte loads, 8-byte stores.
#include "mq_device.h"

namespace mq {

constexpr int kActThreads = 256;

// CPT > 0: the row stays in registers (CPT chunks per thread); CPT == 0: the
// row is read twice.
template <int CPT>
__global__ __launch_bounds__(kActThreads) void act_quant_kernel(
    const uint16_t* __restrict__ X, int M, int K, int ldx,
    uint8_t* __restrict__ Xq, uint16_t* __restrict__ s_x) {
    __shared__ uint32_t red[kActThreads / 64];
    const int m = blockIdx.x;
    const int t = threadIdx.x;
    const uint16_t* row = X + (int64_t)m * ldx;
    const int nchunks = K / 16;
    // chunk c (codes 16c .. 16c+15) is chunk c % 8 of the piece of group c / 8
    auto out = [&](int c) -> uint2& {
        return *reinterpret_cast<uint2*>(Xq + piece_offset(M, m, c >> 3) + (c & 7) * 8);
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
            if (c < nchunks) out(c) = quant_chunk(v[i][0], v[i][1], s, inv_s);
        }
    } else {
        for (int c = t; c < nchunks; c += kActThreads)
            out(c) = quant_chunk(*reinterpret_cast<const uint4*>(row + 16 * c),
                                 *reinterpret_cast<const uint4*>(row + 16 * c + 8), s, inv_s);
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
