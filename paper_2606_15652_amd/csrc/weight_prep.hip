// Offline weight preparation: dense 4-bit base, residual block scores, top-K
// block selection and the sparse 4-bit residual (Section 3 Eq. (4);
// Section 4.1 and Alg. 1).  Not on the timed path: the kernels favour plain,
// deterministic code over speed.
#include "mq_device.h"

#include <float.h>

namespace mq {

// ---------------------------------------------------------------------------
// Base quantisation: one thread per (row n, group g), Eq. (1) over 128 values.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void quant_base_kernel(
    const float* __restrict__ W, int N, int K, int ldw,
    uint8_t* __restrict__ Wq, uint16_t* __restrict__ s_w) {
    const int G = K / kGroup;
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (int64_t)N * G) return;
    const int n = (int)(idx / G), g = (int)(idx % G);
    const float4* src = reinterpret_cast<const float4*>(W + (int64_t)n * ldw + (int64_t)g * kGroup);
    float amax = 0.0f;
    for (int i = 0; i < kGroup / 4; ++i) {
        const float4 v = src[i];
        amax = fmaxf(amax, fmaxf(fmaxf(fabsf(v.x), fabsf(v.y)), fmaxf(fabsf(v.z), fabsf(v.w))));
    }
    const uint16_t sb = scale_bits_from_amax(amax);
    const float s = half_bits_to_float(sb);
    s_w[wscale_index(N, n, g)] = sb;
    const float inv_s = 1.0f / s;
    uint2* dst = reinterpret_cast<uint2*>(Wq + piece_offset(N, n, g));
    for (int c = 0; c < kGroup / 16; ++c) {   // one folded chunk per 16 elements
        int q[16];
        for (int i = 0; i < 4; ++i) {
            const float4 v = src[c * 4 + i];
            q[4 * i + 0] = s == 0.0f ? 0 : quant_code(v.x, s, inv_s);
            q[4 * i + 1] = s == 0.0f ? 0 : quant_code(v.y, s, inv_s);
            q[4 * i + 2] = s == 0.0f ? 0 : quant_code(v.z, s, inv_s);
            q[4 * i + 3] = s == 0.0f ? 0 : quant_code(v.w, s, inv_s);
        }
        dst[c] = fold_codes(q);
    }
}

__device__ __forceinline__ int code_at(const uint8_t* packed_row, int k) {
    const uint2 ch = reinterpret_cast<const uint2*>(packed_row)[k >> 4];
    return chunk_code(ch.x, ch.y, k & 15);
}

// R = W - s q in fp32: s * q is exact (11-bit significand times |q| <= 8), so
// the difference is rounded once.
__device__ __forceinline__ float residual_at(float w, float s, int q) {
    const float deq = s * (float)q;
    return w - deq;
}

// ---------------------------------------------------------------------------
// ||R_B||_F^2 per 128x128 block: one 128-thread workgroup per block, thread r
// sums its row in fp64 in column order, thread 0 then adds the 128 row sums
// in row order.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(128) void score_frob_kernel(
    const float* __restrict__ W, int N, int K, int ldw,
    const uint8_t* __restrict__ Wq, const uint16_t* __restrict__ s_w,
    double* __restrict__ score) {
    __shared__ double rows[kGroup];
    const int KB = K / kGroup;
    const int nb = blockIdx.x / KB, kb = blockIdx.x % KB;
    const int r = threadIdx.x;
    const int n = nb * kGroup + r;
    const float* w = W + (int64_t)n * ldw + (int64_t)kb * kGroup;
    const uint8_t* q = Wq + piece_offset(N, n, kb);
    const float s = half_bits_to_float(s_w[wscale_index(N, n, kb)]);
    double acc = 0.0;
    for (int c = 0; c < kGroup; ++c) {
        const double rv = residual_at(w[c], s, code_at(q, c));
        acc += rv * rv;
    }
    rows[r] = acc;
    __syncthreads();
    if (r == 0) {
        double tot = 0.0;
        for (int i = 0; i < kGroup; ++i) tot += rows[i];
        score[blockIdx.x] = tot;
    }
}

// ---------------------------------------------------------------------------
// Diagonal Hessian h_j = (2/T) sum_t X[t,j]^2: one thread per channel, fp64.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void hessian_diag_kernel(
    const uint16_t* __restrict__ X, int T, int K, int ldx, double* __restrict__ h) {
    const int j = blockIdx.x * blockDim.x + threadIdx.x;
    if (j >= K) return;
    double acc = 0.0;
    for (int t = 0; t < T; ++t) {
        const double x = half_bits_to_float(X[(int64_t)t * ldx + j]);
        acc += x * x;
    }
    h[j] = 2.0 / (double)T * acc;
}

// Quantise one 128-long residual row held in registers-by-recomputation:
// returns the fp16 scale bits; codes are produced by quant_code on demand.
__device__ __forceinline__ uint16_t residual_row_scale(const float* w, const uint8_t* q, float s) {
    float amax = 0.0f;
    for (int c = 0; c < kGroup; ++c) amax = fmaxf(amax, fabsf(residual_at(w[c], s, code_at(q, c))));
    return scale_bits_from_amax(amax);
}

// ---------------------------------------------------------------------------
// Delta-Hessian score (Alg. 1): per block, sum_B h_j R^2 - sum_B h_j (R - Q(R))^2,
// clamped at 0; Q(R) with one scale per block row.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(128) void score_dhessian_kernel(
    const float* __restrict__ W, int N, int K, int ldw,
    const uint8_t* __restrict__ Wq, const uint16_t* __restrict__ s_w,
    const double* __restrict__ h, double* __restrict__ score) {
    __shared__ double before_s[kGroup], after_s[kGroup];
    const int KB = K / kGroup;
    const int nb = blockIdx.x / KB, kb = blockIdx.x % KB;
    const int r = threadIdx.x;
    const int n = nb * kGroup + r;
    const float* w = W + (int64_t)n * ldw + (int64_t)kb * kGroup;
    const uint8_t* q = Wq + piece_offset(N, n, kb);
    const float s = half_bits_to_float(s_w[wscale_index(N, n, kb)]);
    const uint16_t srb = residual_row_scale(w, q, s);
    const float sr = half_bits_to_float(srb);
    double before = 0.0, after = 0.0;
    for (int c = 0; c < kGroup; ++c) {
        const float rv = residual_at(w[c], s, code_at(q, c));
        const int rq = sr == 0.0f ? 0 : quant_code(rv, sr, 1.0f / sr);
        const double hj = h[kb * kGroup + c];
        const double e = (double)rv - (double)sr * (double)rq;
        before += hj * (double)rv * (double)rv;
        after += hj * e * e;
    }
    before_s[r] = before;
    after_s[r] = after;
    __syncthreads();
    if (r == 0) {
        double b = 0.0, a = 0.0;
        for (int i = 0; i < kGroup; ++i) { b += before_s[i]; a += after_s[i]; }
        const double d = b - a;
        score[blockIdx.x] = d > 0.0 ? d : 0.0;
    }
}

// ---------------------------------------------------------------------------
// Top-K selection.  Block i is selected iff its rank
//   #{ j : s_j > s_i  or  (s_j == s_i and j < i) }
// is below nnzb.  One workgroup per block row computes the ranks of that row's
// blocks against all scores (staged through LDS); pass 0 stores the row's
// count, a single-workgroup scan turns counts into row pointers, and pass 1
// recomputes the same ranks and writes the row's ascending column list.
// ---------------------------------------------------------------------------
constexpr int kSelThreads = 256;

__device__ __forceinline__ bool beats(double sj, int j, double si, int i) {
    return sj > si || (sj == si && j < i);
}

template <int PASS>
__global__ __launch_bounds__(kSelThreads) void select_rows_kernel(
    const double* __restrict__ score, int NB, int KB, int nnzb,
    int32_t* __restrict__ rowptr, int32_t* __restrict__ kb_out) {
    __shared__ double chunk[kSelThreads];
    __shared__ int warp_cnt[kSelThreads / 64];
    __shared__ int base_s;
    const int nb = blockIdx.x;
    const int n = NB * KB;
    const int t = threadIdx.x;
    if (t == 0) base_s = PASS == 1 ? rowptr[nb] : 0;
    __syncthreads();
    for (int kb0 = 0; kb0 < KB; kb0 += kSelThreads) {
        const int kb = kb0 + t;
        const bool valid = kb < KB;
        const int i = nb * KB + (valid ? kb : 0);
        const double si = score[i];
        int rank = 0;
        for (int j0 = 0; j0 < n; j0 += kSelThreads) {
            __syncthreads();
            chunk[t] = (j0 + t < n) ? score[j0 + t] : -DBL_MAX;
            __syncthreads();
            const int lim = min(kSelThreads, n - j0);
            for (int u = 0; u < lim; ++u) rank += beats(chunk[u], j0 + u, si, i) ? 1 : 0;
        }
        const bool sel = valid && rank < nnzb;
        // ordered compaction of the selected columns of this batch
        const uint64_t ballot = __ballot(sel);
        const int lane = t & 63, wv = t >> 6;
        const int before_in_wave = __popcll(ballot & ((lane == 0) ? 0ull : (~0ull >> (64 - lane))));
        if (lane == 0) warp_cnt[wv] = __popcll(ballot);
        __syncthreads();
        int before_waves = 0, total = 0;
        for (int w = 0; w < kSelThreads / 64; ++w) {
            if (w < wv) before_waves += warp_cnt[w];
            total += warp_cnt[w];
        }
        const int pos = base_s + before_waves + before_in_wave;
        // ranks form a permutation for finite scores, so pos < nnzb; the bound
        // also keeps non-finite input from writing past the output
        if (PASS == 1 && sel && pos < nnzb) kb_out[pos] = kb;
        __syncthreads();
        if (t == 0) base_s += total;
        __syncthreads();
    }
    if (PASS == 0 && t == 0) rowptr[nb + 1] = base_s;
}

__global__ void scan_rowptr_kernel(int32_t* rowptr, int NB) {
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    rowptr[0] = 0;
    for (int i = 0; i < NB; ++i) rowptr[i + 1] += rowptr[i];
}

// ---------------------------------------------------------------------------
// Residual quantisation on the selected blocks: one 128-thread workgroup per
// block p, thread r = block row.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(128) void quant_residual_kernel(
    const float* __restrict__ W, int N, int K, int ldw,
    const uint8_t* __restrict__ Wq, const uint16_t* __restrict__ s_w,
    const int32_t* __restrict__ rowptr, const int32_t* __restrict__ res_kb, int NB,
    uint8_t* __restrict__ Rq, uint16_t* __restrict__ s_r) {
    const int p = blockIdx.x;
    // block row of entry p: largest nb with rowptr[nb] <= p
    int lo = 0, hi = NB - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) / 2;
        if (rowptr[mid] <= p) lo = mid; else hi = mid - 1;
    }
    const int nb = lo, kb = res_kb[p];
    const int r = threadIdx.x;
    const int n = nb * kGroup + r;
    const float* w = W + (int64_t)n * ldw + (int64_t)kb * kGroup;
    const uint8_t* q = Wq + piece_offset(N, n, kb);
    const float s = half_bits_to_float(s_w[wscale_index(N, n, kb)]);
    const uint16_t srb = residual_row_scale(w, q, s);
    const float sr = half_bits_to_float(srb);
    s_r[(int64_t)p * kGroup + r] = srb;
    uint2* dst = reinterpret_cast<uint2*>(Rq + ((int64_t)p * kGroup + r) * kGroupBytes);
    for (int c = 0; c < kGroup / 16; ++c) {
        int rq[16];
        for (int e = 0; e < 16; ++e) {
            const int k = 16 * c + e;
            const float rv = residual_at(w[k], s, code_at(q, k));
            rq[e] = sr == 0.0f ? 0 : quant_code(rv, sr, 1.0f / sr);
        }
        dst[c] = fold_codes(rq);
    }
}

}  // namespace mq

using namespace mq;

static mq_status check_weight_args(const float* W, int N, int K, int ldw,
                                   const void* Wq, const void* s_w) {
    if (N < 0 || K < 0) return MQ_ERR_INVALID_ARG;
    if (!mq_host::shape_ok(N, K) || ldw < K || ldw % 4 != 0) return MQ_ERR_UNSUPPORTED_SHAPE;
    if (!W || !Wq || !s_w) return MQ_ERR_INVALID_ARG;
    if (!mq_host::aligned(W, 16) || !mq_host::aligned(Wq, 16) || !mq_host::aligned(s_w, 2))
        return MQ_ERR_MISALIGNED;
    return MQ_OK;
}

extern "C" mq_status mq_quantize_weight(const float* W, int N, int K, int ldw,
                                        uint8_t* Wq, void* s_w, double* score,
                                        hipStream_t stream) {
    mq_status st = check_weight_args(W, N, K, ldw, Wq, s_w);
    if (st != MQ_OK) return st;
    if (score && !mq_host::aligned(score, 8)) return MQ_ERR_MISALIGNED;
    const int64_t jobs = (int64_t)N * (K / kGroup);
    hipLaunchKernelGGL(quant_base_kernel, dim3((unsigned)((jobs + 255) / 256)), dim3(256), 0, stream,
                       W, N, K, ldw, Wq, static_cast<uint16_t*>(s_w));
    st = mq_host::launch_status();
    if (st != MQ_OK || !score) return st;
    const int nblk = (N / kGroup) * (K / kGroup);
    hipLaunchKernelGGL(score_frob_kernel, dim3(nblk), dim3(128), 0, stream,
                       W, N, K, ldw, Wq, static_cast<const uint16_t*>(s_w), score);
    return mq_host::launch_status();
}

extern "C" mq_status mq_hessian_diag(const void* X, int T, int K, int ldx, double* h,
                                     hipStream_t stream) {
    if (T <= 0 || K <= 0 || ldx < K) return MQ_ERR_INVALID_ARG;
    if (!X || !h) return MQ_ERR_INVALID_ARG;
    if (!mq_host::aligned(X, 2) || !mq_host::aligned(h, 8)) return MQ_ERR_MISALIGNED;
    hipLaunchKernelGGL(hessian_diag_kernel, dim3((K + 255) / 256), dim3(256), 0, stream,
                       static_cast<const uint16_t*>(X), T, K, ldx, h);
    return mq_host::launch_status();
}

extern "C" mq_status mq_block_scores_dhessian(const float* W, int N, int K, int ldw,
                                              const uint8_t* Wq, const void* s_w,
                                              const double* h, double* score,
                                              hipStream_t stream) {
    mq_status st = check_weight_args(W, N, K, ldw, Wq, s_w);
    if (st != MQ_OK) return st;
    if (!h || !score) return MQ_ERR_INVALID_ARG;
    if (!mq_host::aligned(h, 8) || !mq_host::aligned(score, 8)) return MQ_ERR_MISALIGNED;
    const int nblk = (N / kGroup) * (K / kGroup);
    hipLaunchKernelGGL(score_dhessian_kernel, dim3(nblk), dim3(128), 0, stream,
                       W, N, K, ldw, Wq, static_cast<const uint16_t*>(s_w), h, score);
    return mq_host::launch_status();
}

extern "C" mq_status mq_select_blocks(const double* score, int NB, int KB, int nnzb,
                                      int32_t* res_rowptr, int32_t* res_kb,
                                      hipStream_t stream) {
    if (NB <= 0 || KB <= 0 || nnzb < 0) return MQ_ERR_INVALID_ARG;
    if ((int64_t)NB * KB > (1 << 24)) return MQ_ERR_UNSUPPORTED_SHAPE;
    if ((int64_t)nnzb > (int64_t)NB * KB) return MQ_ERR_INVALID_ARG;
    if (!score || !res_rowptr || (nnzb > 0 && !res_kb)) return MQ_ERR_INVALID_ARG;
    if (!mq_host::aligned(score, 8) || !mq_host::aligned(res_rowptr, 4) ||
        (res_kb && !mq_host::aligned(res_kb, 4)))
        return MQ_ERR_MISALIGNED;
    hipLaunchKernelGGL(select_rows_kernel<0>, dim3(NB), dim3(kSelThreads), 0, stream,
                       score, NB, KB, nnzb, res_rowptr, res_kb);
    mq_status st = mq_host::launch_status();
    if (st != MQ_OK) return st;
    hipLaunchKernelGGL(scan_rowptr_kernel, dim3(1), dim3(1), 0, stream, res_rowptr, NB);
    st = mq_host::launch_status();
    if (st != MQ_OK || nnzb == 0) return st;
    hipLaunchKernelGGL(select_rows_kernel<1>, dim3(NB), dim3(kSelThreads), 0, stream,
                       score, NB, KB, nnzb, res_rowptr, res_kb);
    return mq_host::launch_status();
}

extern "C" mq_status mq_quantize_residual(const float* W, int N, int K, int ldw,
                                          const uint8_t* Wq, const void* s_w,
                                          const int32_t* res_rowptr, const int32_t* res_kb,
                                          int nnzb, uint8_t* Rq, void* s_r,
                                          hipStream_t stream) {
    mq_status st = check_weight_args(W, N, K, ldw, Wq, s_w);
    if (st != MQ_OK) return st;
    if (nnzb < 0 || (int64_t)nnzb > (int64_t)(N / kGroup) * (K / kGroup)) return MQ_ERR_INVALID_ARG;
    if (nnzb == 0) return MQ_OK;
    if (!res_rowptr || !res_kb || !Rq || !s_r) return MQ_ERR_INVALID_ARG;
    if (!mq_host::aligned(res_rowptr, 4) || !mq_host::aligned(res_kb, 4) ||
        !mq_host::aligned(Rq, 16) || !mq_host::aligned(s_r, 2))
        return MQ_ERR_MISALIGNED;
    hipLaunchKernelGGL(quant_residual_kernel, dim3(nnzb), dim3(128), 0, stream,
                       W, N, K, ldw, Wq, static_cast<const uint16_t*>(s_w),
                       res_rowptr, res_kb, N / kGroup, Rq, static_cast<uint16_t*>(s_r));
    return mq_host::launch_status();
}
