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

// Residual kernel: a workgroup of eight waves owns a (16 WGMR) x 128 tile (one
// 128-column block row); WGMR waves along M, each with 16 rows and the eight
// 16-column sub-tiles, and 8 / WGMR splits of the block row's CSR entries
// (contiguous runs).  Each wave streams its blocks through a two-stage
// register ring (X fragment of the block's group and R fragments, read from
// memory), scales each block row's sums by s_r, and the splits are added
// through LDS in split order.  WGMR = 1 for M <= 16, else 4.
template <int WGMR>
__global__ __launch_bounds__(512) void gemm_residual_kernel(int M, int N, int K, const uint8_t* __restrict__ Xq,
                                                            const int32_t* __restrict__ rowptr,
                                                            const int32_t* __restrict__ res_kb,
                                                            const uint8_t* __restrict__ Rq,
                                                            const uint16_t* __restrict__ s_r,
                                                            float* __restrict__ P) {
    constexpr int KS = 8 / WGMR;
    __shared__ __attribute__((aligned(16))) float red[8][32][64];
    const int nb = blockIdx.y;
    const int rp = rowptr[nb], cnt = rowptr[nb + 1] - rp;
    if (cnt == 0) return;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = wave % WGMR, split = wave / WGMR;
    const int lrow = lane & 15, lq = lane >> 4;
    const int m0 = blockIdx.x * 16 * WGMR + 16 * wm;
    const int xr = m0 + lrow;
    const int per = cnt / KS, extra = cnt % KS;
    const int pb = rp + split * per + min(split, extra);
    const int ne = per + (split < extra ? 1 : 0);

    const int G = K / kGroup;
    struct Stage {
        uint4 x, r[8];
        uint2 xt;
        uint16_t s[8];
    };
    auto load = [&](Stage& S, int e) {
        S.x = make_uint4(0u, 0u, 0u, 0u);
        S.xt = make_uint2(0u, 0u);
        if (e >= ne) return;
        const int p = pb + e;
        const int g = res_kb[p];
        if (xr < M) {
            S.x = ldg16(Xq + act_main_offset(M, xr, g) + 16 * lq);
            S.xt = *reinterpret_cast<const uint2*>(Xq + act_tail_offset(M, G, xr, g, lq));
        }
        const uint8_t* rt = Rq + (int64_t)p * kGroup * kGroupBytes;
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            S.r[c] = ldg16(rt + (16 * c + lrow) * kGroupBytes + 16 * lq);
            S.s[c] = s_r[(int64_t)p * kGroup + 16 * c + lrow];
        }
    };
    f32x4 acc[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) acc[c] = f32x4{0.f, 0.f, 0.f, 0.f};
    auto compute = [&](const Stage& S) {
        const i32x8 av = act_operand(S.x, S.xt);
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            const f32x4 t = mfma_codes(av, unfold_codes(S.r[c]), f32x4{0.f, 0.f, 0.f, 0.f});
            const float sr = half_bits_to_float(S.s[c]) * kCodeScale;
#pragma unroll
            for (int r = 0; r < 4; ++r) acc[c][r] = __builtin_fmaf(sr, t[r], acc[c][r]);
        }
#pragma unroll
        for (int c = 0; c < 8; ++c) asm volatile("" : "+v"(acc[c]));   // epilogue completes in this block
    };
    Stage S0, S1;
    load(S0, 0);
    load(S1, 1);
    for (int e = 0; e < ne; e += 2) {
        compute(S0);
        load(S0, e + 2);
        if (e + 1 < ne) compute(S1);
        load(S1, e + 3);
    }
    // lane holds rows 4 (lane / 16) + r of each sub-tile, column lane % 16
#pragma unroll
    for (int c = 0; c < 8; ++c)
#pragma unroll
        for (int r = 0; r < 4; ++r) red[wave][c * 4 + r][lane] = acc[c][r];
    __syncthreads();
    if (split != 0) return;
#pragma unroll
    for (int c = 0; c < 8; ++c)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int m = m0 + 4 * lq + r;
            float v = 0.f;
            for (int k = 0; k < KS; ++k) v += red[k * WGMR + wm][c * 4 + r][lane];
            if (m < M) P[(int64_t)m * N + nb * kGroup + 16 * c + lrow] = v;
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
    if (M <= 16)
        hipLaunchKernelGGL((gemm_residual_kernel<1>), dim3(1u, (unsigned)NB), dim3(512), 0, stream, M, N, K, Xq,
                           res_rowptr, res_kb, Rq, static_cast<const uint16_t*>(s_r), P);
    else
        hipLaunchKernelGGL((gemm_residual_kernel<4>), dim3((unsigned)((M + 63) / 64), (unsigned)NB), dim3(512), 0,
                           stream, M, N, K, Xq, res_rowptr, res_kb, Rq, static_cast<const uint16_t*>(s_r), P);
    st = mq_host::launch_status();
    if (st != MQ_OK) return st;
    // 3. reduce-add
    hipLaunchKernelGGL(reduce_add_kernel, dim3((unsigned)(((int64_t)M * kGroup + 255) / 256), (unsigned)NB),
                       dim3(256), 0, stream, M, N, res_rowptr, P, static_cast<const uint16_t*>(s_x),
                       static_cast<uint16_t*>(Y), ldy);
    return mq_host::launch_status();
}
