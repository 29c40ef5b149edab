// The unfused three-kernel pipeline that the fused kernel replaces (Section
// 4.2 "Kernel Fusion", Fig. 3: dense 4-bit GEMM, a separate sparse residual
// GEMM, then a reduce-add).  It is a comparison baseline, not the hot path:
//
//   1. dense:     Y   = fp16(s_x * sum_g s_w A_b)          (the fused kernels, no residual blocks)
//   2. residual:  P   = sum_g s_r A_r (fp32, [M, N])       (reloads Xq from memory)
//   3. reduce-add: Y <- fp16(f32(Y) + s_x * P)              (block rows that hold residual blocks)
//
// The residual kernel and the reduce-add touch only block rows with at least
// one residual block; P is left unwritten (and unread) elsewhere.
#include "mq_device.h"

namespace mq {

// Residual kernel: a workgroup of four waves owns a 64 x 128 tile (64 rows of
// the output, one 128-column block row); wave w owns rows 16 w .. 16 w + 15
// as eight 16 x 16 sub-tiles.  For each residual block (nb, kb) of the block
// row it multiplies the X rows' group kb (from memory) with the block's R
// tile (from memory, shared through L2), scales each block row's sums by s_r
// and accumulates in fp32.
__global__ __launch_bounds__(256) void residual_only_kernel(int M, int N, const uint8_t* __restrict__ Xq,
                                                            const int32_t* __restrict__ rowptr,
                                                            const int32_t* __restrict__ res_kb,
                                                            const uint8_t* __restrict__ Rq,
                                                            const uint16_t* __restrict__ s_r,
                                                            float* __restrict__ P) {
    const int nb = blockIdx.y;
    const int rp = rowptr[nb], re = rowptr[nb + 1];
    if (rp == re) return;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int lrow = lane & 15, lq = lane >> 4;
    const int m0 = blockIdx.x * 64 + 16 * wave;
    const int xr = m0 + lrow;
    f32x4 acc[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) acc[c] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int p = rp; p < re; ++p) {
        const int g = res_kb[p];
        uint4 xa = make_uint4(0u, 0u, 0u, 0u);
        if (xr < M) xa = ldg16(Xq + piece_offset(M, xr, g) + 16 * lq);
        const i32x8 av = unfold_codes(xa);
        const uint8_t* rt = Rq + (int64_t)p * kGroup * kGroupBytes;
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            const int row = 16 * c + lrow;                       // row of the R tile
            const i32x8 bv = unfold_codes(ldg16(rt + row * kGroupBytes + 16 * lq));
            const f32x4 t = mfma_codes(av, bv, f32x4{0.f, 0.f, 0.f, 0.f});
            const float sr = half_bits_to_float(s_r[(int64_t)p * kGroup + row]) * kCodeScale;
#pragma unroll
            for (int r = 0; r < 4; ++r) acc[c][r] = __builtin_fmaf(sr, t[r], acc[c][r]);
        }
    }
    // lane holds rows 4 (lane / 16) + r of each sub-tile, column lane % 16
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int m = m0 + 4 * lq + r;
        if (m >= M) continue;
#pragma unroll
        for (int c = 0; c < 8; ++c) P[(int64_t)m * N + nb * kGroup + 16 * c + lrow] = acc[c][r];
    }
}

// Y[m, n] <- fp16(f32(Y[m, n]) + s_x[m] P[m, n]) on block rows with blocks.
__global__ __launch_bounds__(256) void reduce_add_kernel(int M, int N, const int32_t* __restrict__ rowptr,
                                                         const float* __restrict__ P,
                                                         const uint16_t* __restrict__ s_x,
                                                         uint16_t* __restrict__ Y, int ldy) {
    const int nb = blockIdx.y;
    if (rowptr[nb] == rowptr[nb + 1]) return;
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (int64_t)M * kGroup) return;
    const int m = (int)(idx / kGroup), n = nb * kGroup + (int)(idx % kGroup);
    const float y = half_bits_to_float(Y[(int64_t)m * ldy + n]);
    Y[(int64_t)m * ldy + n] = float_to_half_bits(y + half_bits_to_float(s_x[m]) * P[(int64_t)m * N + n]);
}

}  // namespace mq

using namespace mq;

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

extern "C" size_t mq_unfused_workspace_size(int M, int N, int K) {
    if (M <= 0 || !mq_host::shape_ok(N, K)) return 0;
    return align256((size_t)M * N * sizeof(float)) + mq_fused_gemm_workspace_size(M, N, K);
}

extern "C" mq_status mq_unfused_gemm(int M, int N, int K, const uint8_t* Xq, const void* s_x, const uint8_t* Wq,
                                     const void* s_w, const int32_t* res_rowptr, const int32_t* res_kb, int nnzb,
                                     const uint8_t* Rq, const void* s_r, void* Y, int ldy, void* workspace,
                                     size_t ws_bytes, hipStream_t stream) {
    if (M < 0 || N < 0 || K < 0 || nnzb < 0) return MQ_ERR_INVALID_ARG;
    if (!mq_host::shape_ok(N, K) || M > (1 << 24)) return MQ_ERR_UNSUPPORTED_SHAPE;
    if ((int64_t)nnzb > (int64_t)(N / kGroup) * (K / kGroup)) return MQ_ERR_INVALID_ARG;
    if (ldy < N || ldy % 8 != 0 || N / kGroup > 65535) return MQ_ERR_UNSUPPORTED_SHAPE;
    const size_t need = mq_unfused_workspace_size(M, N, K);
    if (ws_bytes < need) return MQ_ERR_WORKSPACE;
    if (M == 0) return MQ_OK;
    if (!Xq || !s_x || !Wq || !s_w || !Y || !workspace || (nnzb > 0 && (!res_rowptr || !res_kb || !Rq || !s_r)))
        return MQ_ERR_INVALID_ARG;
    if (!mq_host::aligned(Xq, 16) || !mq_host::aligned(Wq, 16) || (Rq && !mq_host::aligned(Rq, 16)) ||
        !mq_host::aligned(workspace, 16) || !mq_host::aligned(s_x, 2) || !mq_host::aligned(Y, 2))
        return MQ_ERR_MISALIGNED;
    float* P = static_cast<float*>(workspace);
    uint8_t* gws = static_cast<uint8_t*>(workspace) + align256((size_t)M * N * sizeof(float));
    const size_t gws_bytes = ws_bytes - align256((size_t)M * N * sizeof(float));
    // 1. dense W4A4 GEMM (no residual blocks)
    mq_status st = mq_fused_gemm(M, N, K, Xq, s_x, Wq, s_w, nullptr, nullptr, 0, nullptr, nullptr, Y, ldy,
                                 gws_bytes ? gws : nullptr, gws_bytes, stream);
    if (st != MQ_OK || nnzb == 0) return st;
    // 2. sparse residual GEMM into P
    const int NB = N / kGroup;
    hipLaunchKernelGGL(residual_only_kernel, dim3((unsigned)((M + 63) / 64), (unsigned)NB), dim3(256), 0, stream, M,
                       N, Xq, res_rowptr, res_kb, Rq, static_cast<const uint16_t*>(s_r), P);
    st = mq_host::launch_status();
    if (st != MQ_OK) return st;
    // 3. reduce-add
    hipLaunchKernelGGL(reduce_add_kernel, dim3((unsigned)(((int64_t)M * kGroup + 255) / 256), (unsigned)NB),
                       dim3(256), 0, stream, M, N, res_rowptr, P, static_cast<const uint16_t*>(s_x),
                       static_cast<uint16_t*>(Y), ldy);
    return mq_host::launch_status();
}
