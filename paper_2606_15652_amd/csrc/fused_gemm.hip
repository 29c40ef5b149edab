// Fused dense + sparse-residual W4A4 GEMM for gfx950 (Section 3 Eq. (4) with
// the scale factorisation of Eq. (2) applied per 128-group; Section 4.2
// "Kernel Fusion" and "Overlapped pipeline").
//
//   Y[m,n] = s_x[m] * sum_g ( s_w[n,g] A_b[m,n,g] + s_r[p,n%128] A_r[m,n,g] )
//
// CDNA4 has no 4-bit matrix instruction, so packed nibbles are widened in
// registers to int8 (16 * code, see unpack_nibbles) and fed to
// v_mfma_i32_16x16x64_i8.  One MFMA pair covers one 128-long group of a 16x16
// output sub-tile; its int32 result is the exact group sum (times 256), which
// the epilogue converts and scales into an fp32 accumulator.  The residual
// blocks of the tile's 128-row block row are walked in the same K-loop: when
// the CSR's next column equals the current group, the residual fragments are
// multiplied with the activation fragments already staged for the dense term
// and accumulated into the same output registers.
//
// Two kernel families share that inner step:
//  * tiled  (prefill):  a workgroup owns a BM x BN output tile; the packed
//    activation tile of each group is widened once per workgroup into an LDS
//    double buffer (XOR-swizzled 16-byte chunks) and shared by all waves, each
//    wave streams its own weight rows straight from global memory into
//    registers, one group ahead of the MFMAs.
//  * skinny (decode, small M): a workgroup owns 16 output columns and all M
//    rows; its waves split the K-loop, each streaming a contiguous run of
//    groups, and the fp32 partial tiles are reduced through LDS in wave order
//    (deterministic).
#include "mq_device.h"

#include <type_traits>

namespace mq {

struct GemmArgs {
    int M, N, K;
    const uint8_t* Xq;
    const uint16_t* s_x;
    const uint8_t* Wq;
    const uint16_t* s_w;
    const int32_t* rowptr;   // may be null when nnzb == 0
    const int32_t* res_kb;
    const uint8_t* Rq;
    const uint16_t* s_r;
    uint16_t* Y;
    int ldy;
    int32_t* Tb;             // raw mode outputs
    int32_t* Tr;
};

// 1/256 removes the 16 x 16 factor of the nibble widening (exact).
constexpr float kUnscale = 1.0f / 256.0f;

// One m sub-tile row of one group: base MFMA pair + epilogue for each of the
// WN column sub-tiles, then (HAS_RES) the residual MFMA pair + epilogue.  The
// caller picks HAS_RES once per group, so this is straight-line code and every
// MFMA result is converted inside the basic block that produced it (the
// compiler's MFMA-to-VALU wait states are only placed reliably within a block).
template <int WN, bool RAW, bool HAS_RES>
__device__ __forceinline__ void group_row(const i32x4 alo, const i32x4 ahi,
                                          const i32x4 (&wlo)[WN], const i32x4 (&whi)[WN],
                                          const i32x4 (&rlo)[WN], const i32x4 (&rhi)[WN],
                                          const float (&sw_f)[WN], const float (&sr_f)[WN],
                                          f32x4 (&acc)[WN], i32x4 (&iacc)[WN], i32x4 (&racc)[WN]) {
#pragma unroll
    for (int j = 0; j < WN; ++j) {
        i32x4 s = mfma_i8(alo, wlo[j], i32x4{0, 0, 0, 0});
        s = mfma_i8(ahi, whi[j], s);
        if constexpr (RAW) {
#pragma unroll
            for (int r = 0; r < 4; ++r) iacc[j][r] += s[r] >> 8;  // exact: s is 256 x the sum
        } else {
#pragma unroll
            for (int r = 0; r < 4; ++r) acc[j][r] += sw_f[j] * (float)s[r];
        }
    }
    if constexpr (HAS_RES) {
#pragma unroll
        for (int j = 0; j < WN; ++j) {
            i32x4 s = mfma_i8(alo, rlo[j], i32x4{0, 0, 0, 0});
            s = mfma_i8(ahi, rhi[j], s);
            if constexpr (RAW) {
#pragma unroll
                for (int r = 0; r < 4; ++r) racc[j][r] += s[r] >> 8;
            } else {
#pragma unroll
                for (int r = 0; r < 4; ++r) acc[j][r] += sr_f[j] * (float)s[r];
            }
        }
    }
}

// --------------------------------------------------------------------------
// Tiled kernel
// --------------------------------------------------------------------------
// WM: 16-row sub-tiles per wave along M; WN: 16-column sub-tiles per wave
// along N; NW: waves per workgroup, all along N (they share the X tile).
template <int WM, int WN, int NW, bool RAW>
__global__ __launch_bounds__(64 * NW) void gemm_tiled_kernel(GemmArgs a) {
    constexpr int BM = 16 * WM;
    constexpr int BN = 16 * WN * NW;
    constexpr int kThreads = 64 * NW;
    constexpr int kXChunks = BM * 4;                       // 16-byte packed chunks per group
    constexpr int kXPerThread = (kXChunks + kThreads - 1) / kThreads;
    constexpr int kRowBytes = 128;                         // widened int8 row of one group
    static_assert(WN * 16 <= 128 && 128 % (WN * 16) == 0, "wave columns must sit in one block row");

    __shared__ __attribute__((aligned(16))) uint8_t xs[2][BM * kRowBytes];

    const int M = a.M, N = a.N, K = a.K;
    const int G = K / kGroup;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int tiles_n = (N + BN - 1) / BN;
    const int tm = blockIdx.x / tiles_n, tn = blockIdx.x % tiles_n;
    const int m0 = tm * BM;
    const int wn0 = tn * BN + wave * 16 * WN;
    const bool active = wn0 < N;                            // N % 128 == 0: whole wave in or out
    const int64_t ldk = K / 2;

    // residual walk for this wave's block row
    int rp = 0, rend = 0;
    if (active && a.rowptr) {
        const int nb = wn0 / 128;
        rp = a.rowptr[nb];
        rend = a.rowptr[nb + 1];
    }
    const int rrow0 = (wn0 % 128);                          // first row of this wave inside the block

    // per-lane pointers
    const int lrow = lane & 15, lq = lane >> 4;
    const uint8_t* wbase = a.Wq + (int64_t)(wn0 + lrow) * ldk + lq * 16;
    const uint16_t* swbase = a.s_w + (int64_t)(wn0 + lrow) * G;

    // --- prefetch state (group g) ---
    uint4 xpk[kXPerThread];
    uint4 wpk[WN], rpk[WN];
    uint16_t swb[WN], srb[WN];
#pragma unroll
    for (int j = 0; j < WN; ++j) {
        wpk[j] = rpk[j] = make_uint4(0, 0, 0, 0);
        swb[j] = srb[j] = 0;
    }
    int cur_p = -1;

    auto load_x = [&](int g, uint4* dst) {
#pragma unroll
        for (int i = 0; i < kXPerThread; ++i) {
            const int c = threadIdx.x + i * kThreads;
            const int row = c >> 2, q = c & 3;
            dst[i] = make_uint4(0, 0, 0, 0);
            if (c < kXChunks && m0 + row < M)
                dst[i] = ldg16(a.Xq + (int64_t)(m0 + row) * ldk + (int64_t)g * kGroupBytes + q * 16);
        }
    };
    auto load_w = [&](int g) {
        if (!active) return;
#pragma unroll
        for (int j = 0; j < WN; ++j) {
            wpk[j] = ldg16(wbase + (int64_t)j * 16 * ldk + (int64_t)g * kGroupBytes);
            if constexpr (!RAW) swb[j] = swbase[(int64_t)j * 16 * G + g];
        }
    };
    auto load_r = [&](int p) {
        const uint8_t* rb = a.Rq + ((int64_t)p * 128 + rrow0 + lrow) * kGroupBytes + lq * 16;
#pragma unroll
        for (int j = 0; j < WN; ++j) {
            rpk[j] = ldg16(rb + j * 16 * kGroupBytes);
            if constexpr (!RAW) srb[j] = a.s_r[(int64_t)p * 128 + rrow0 + j * 16 + lrow];
        }
    };
    // residual entry for group g (advances the walk)
    auto res_for = [&](int g) -> int {
        if (rp < rend && a.res_kb[rp] == g) return rp++;
        return -1;
    };

    f32x4 acc[WM][WN];
    i32x4 iacc[WM][WN], racc[WM][WN];
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
        for (int j = 0; j < WN; ++j) {
            acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
            iacc[i][j] = i32x4{0, 0, 0, 0};
            racc[i][j] = i32x4{0, 0, 0, 0};
        }

    load_x(0, xpk);
    load_w(0);
    if (active) {
        cur_p = res_for(0);
        if (cur_p >= 0) load_r(cur_p);
    }

    for (int g = 0; g < G; ++g) {
        const int buf = g & 1;
        // widen this group's activation chunks into LDS
#pragma unroll
        for (int i = 0; i < kXPerThread; ++i) {
            const int c = threadIdx.x + i * kThreads;
            if (c < kXChunks) {
                const int row = c >> 2, q = c & 3;
                i32x4 lo, hi;
                unpack_nibbles(xpk[i], lo, hi);
                const int sw = row & 7;
                uint8_t* rb = &xs[buf][row * kRowBytes];
                *reinterpret_cast<i32x4*>(rb + (((2 * q) ^ sw) << 4)) = lo;
                *reinterpret_cast<i32x4*>(rb + (((2 * q + 1) ^ sw) << 4)) = hi;
            }
        }
        // widen this group's weight (and residual) fragments
        i32x4 wlo[WN], whi[WN], rlo[WN], rhi[WN];
        float sw_f[WN], sr_f[WN];
        const int p = cur_p;
#pragma unroll
        for (int j = 0; j < WN; ++j) { rlo[j] = rhi[j] = i32x4{0, 0, 0, 0}; sw_f[j] = sr_f[j] = 0.f; }
#pragma unroll
        for (int j = 0; j < WN; ++j) {
            unpack_nibbles(wpk[j], wlo[j], whi[j]);
            if constexpr (!RAW) sw_f[j] = half_bits_to_float(swb[j]) * kUnscale;
            if (p >= 0) {
                unpack_nibbles(rpk[j], rlo[j], rhi[j]);
                if constexpr (!RAW) sr_f[j] = half_bits_to_float(srb[j]) * kUnscale;
            }
        }
        // prefetch group g+1
        if (g + 1 < G) {
            load_x(g + 1, xpk);
            load_w(g + 1);
            cur_p = -1;
            if (active) {
                cur_p = res_for(g + 1);
                if (cur_p >= 0) load_r(cur_p);
            }
        }
        __syncthreads();
        if (active) {
            auto tiles = [&](auto has_res) {
                constexpr bool HR = decltype(has_res)::value;
#pragma unroll
                for (int i = 0; i < WM; ++i) {
                    const int row = i * 16 + lrow;
                    const int sw = row & 7;
                    const uint8_t* rb = &xs[buf][row * kRowBytes];
                    const i32x4 alo = *reinterpret_cast<const i32x4*>(rb + (((2 * lq) ^ sw) << 4));
                    const i32x4 ahi = *reinterpret_cast<const i32x4*>(rb + (((2 * lq + 1) ^ sw) << 4));
                    group_row<WN, RAW, HR>(alo, ahi, wlo, whi, rlo, rhi, sw_f, sr_f, acc[i], iacc[i], racc[i]);
                }
            };
            if (p >= 0) tiles(std::true_type{});
            else tiles(std::false_type{});
        }
    }

    if (!active) return;
    // epilogue: lane holds rows 4*(lane/16)+r of each sub-tile, column lane%16
#pragma unroll
    for (int i = 0; i < WM; ++i) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int m = m0 + i * 16 + 4 * lq + r;
            if (m >= M) continue;
            if constexpr (RAW) {
#pragma unroll
                for (int j = 0; j < WN; ++j) {
                    const int n = wn0 + j * 16 + lrow;
                    a.Tb[(int64_t)m * N + n] = iacc[i][j][r];
                    a.Tr[(int64_t)m * N + n] = racc[i][j][r];
                }
            } else {
                const float sx = half_bits_to_float(a.s_x[m]);
#pragma unroll
                for (int j = 0; j < WN; ++j) {
                    const int n = wn0 + j * 16 + lrow;
                    a.Y[(int64_t)m * a.ldy + n] = float_to_half_bits(sx * acc[i][j][r]);
                }
            }
        }
    }
}

// --------------------------------------------------------------------------
// Skinny kernel: 16 * WN output columns per workgroup, all M (<= 16 * WM)
// rows, the K-loop split over NW waves.
// --------------------------------------------------------------------------
template <int WM, int WN, int NW, bool RAW>
__global__ __launch_bounds__(64 * NW) void gemm_skinny_kernel(GemmArgs a) {
    static_assert(WN * 16 <= 128 && 128 % (WN * 16) == 0, "workgroup columns must sit in one block row");
    // reduction buffer: fp32 partials, or (raw mode) int32 base and residual sums
    constexpr int kSlotsPerWave = WM * WN * 4 * (RAW ? 2 : 1);
    __shared__ __attribute__((aligned(16))) uint32_t red[NW][kSlotsPerWave][64];

    const int M = a.M, K = a.K, N = a.N;
    const int G = K / kGroup;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int n0 = blockIdx.x * 16 * WN;
    const int64_t ldk = K / 2;
    const int lrow = lane & 15, lq = lane >> 4;

    // contiguous run of groups for this wave
    const int per = G / NW, extra = G % NW;
    const int gb = wave * per + (wave < extra ? wave : extra);
    const int ge = gb + per + (wave < extra ? 1 : 0);

    // residual walk: first entry of the block row with column >= gb
    int rp = 0, rend = 0;
    if (a.rowptr) {
        const int nb = n0 / 128;
        rp = a.rowptr[nb];
        rend = a.rowptr[nb + 1];
        while (rp < rend && a.res_kb[rp] < gb) ++rp;
    }
    const int rrow0 = n0 % 128;

    const uint8_t* wbase = a.Wq + (int64_t)(n0 + lrow) * ldk + lq * 16;
    const uint16_t* swbase = a.s_w + (int64_t)(n0 + lrow) * G;

    f32x4 acc[WM][WN];
    i32x4 iacc[WM][WN], racc[WM][WN];
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
        for (int j = 0; j < WN; ++j) {
            acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
            iacc[i][j] = i32x4{0, 0, 0, 0};
            racc[i][j] = i32x4{0, 0, 0, 0};
        }

    uint4 xpk[WM], wpk[WN], rpk[WN];
    uint16_t swb[WN], srb[WN];
    int cur_p = -1;
    auto load = [&](int g) {
#pragma unroll
        for (int i = 0; i < WM; ++i) {
            const int row = i * 16 + lrow;
            xpk[i] = make_uint4(0, 0, 0, 0);
            if (row < M) xpk[i] = ldg16(a.Xq + (int64_t)row * ldk + (int64_t)g * kGroupBytes + lq * 16);
        }
#pragma unroll
        for (int j = 0; j < WN; ++j) {
            wpk[j] = ldg16(wbase + (int64_t)j * 16 * ldk + (int64_t)g * kGroupBytes);
            if constexpr (!RAW) swb[j] = swbase[(int64_t)j * 16 * G + g];
        }
        cur_p = -1;
        if (rp < rend && a.res_kb[rp] == g) {
            cur_p = rp++;
            const uint8_t* rb = a.Rq + ((int64_t)cur_p * 128 + rrow0 + lrow) * kGroupBytes + lq * 16;
#pragma unroll
            for (int j = 0; j < WN; ++j) {
                rpk[j] = ldg16(rb + j * 16 * kGroupBytes);
                if constexpr (!RAW) srb[j] = a.s_r[(int64_t)cur_p * 128 + rrow0 + j * 16 + lrow];
            }
        }
    };

    if (gb < ge) load(gb);
    for (int g = gb; g < ge; ++g) {
        i32x4 alo[WM], ahi[WM], wlo[WN], whi[WN], rlo[WN], rhi[WN];
        float sw_f[WN], sr_f[WN];
        const int p = cur_p;
#pragma unroll
        for (int j = 0; j < WN; ++j) { rlo[j] = rhi[j] = i32x4{0, 0, 0, 0}; sw_f[j] = sr_f[j] = 0.f; }
#pragma unroll
        for (int i = 0; i < WM; ++i) unpack_nibbles(xpk[i], alo[i], ahi[i]);
#pragma unroll
        for (int j = 0; j < WN; ++j) {
            unpack_nibbles(wpk[j], wlo[j], whi[j]);
            if constexpr (!RAW) sw_f[j] = half_bits_to_float(swb[j]) * kUnscale;
            if (p >= 0) {
                unpack_nibbles(rpk[j], rlo[j], rhi[j]);
                if constexpr (!RAW) sr_f[j] = half_bits_to_float(srb[j]) * kUnscale;
            }
        }
        if (g + 1 < ge) load(g + 1);
        auto tiles = [&](auto has_res) {
            constexpr bool HR = decltype(has_res)::value;
#pragma unroll
            for (int i = 0; i < WM; ++i)
                group_row<WN, RAW, HR>(alo[i], ahi[i], wlo, whi, rlo, rhi, sw_f, sr_f, acc[i], iacc[i], racc[i]);
        };
        if (p >= 0) tiles(std::true_type{});
        else tiles(std::false_type{});
    }

    // cross-wave reduction in wave order
    if constexpr (RAW) {
#pragma unroll
        for (int i = 0; i < WM; ++i)
#pragma unroll
            for (int j = 0; j < WN; ++j)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    red[wave][((i * WN + j) * 4 + r) * 2 + 0][lane] = (uint32_t)iacc[i][j][r];
                    red[wave][((i * WN + j) * 4 + r) * 2 + 1][lane] = (uint32_t)racc[i][j][r];
                }
    } else {
#pragma unroll
        for (int i = 0; i < WM; ++i)
#pragma unroll
            for (int j = 0; j < WN; ++j)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    red[wave][(i * WN + j) * 4 + r][lane] = __float_as_uint(acc[i][j][r]);
    }
    __syncthreads();
    // each thread finishes (slot, lane) pairs
    constexpr int kSlots = WM * WN * 4;
    for (int e = threadIdx.x; e < kSlots * 64; e += 64 * NW) {
        const int slot = e / 64, l = e % 64;
        const int ij = slot / 4, r = slot % 4;
        const int i = ij / WN, j = ij % WN;
        const int m = i * 16 + 4 * (l >> 4) + r;
        const int n = n0 + j * 16 + (l & 15);
        if (m >= M) continue;
        if constexpr (RAW) {
            int32_t tb = 0, tr = 0;
            for (int w = 0; w < NW; ++w) {
                tb += (int32_t)red[w][slot * 2 + 0][l];
                tr += (int32_t)red[w][slot * 2 + 1][l];
            }
            a.Tb[(int64_t)m * N + n] = tb;
            a.Tr[(int64_t)m * N + n] = tr;
        } else {
            float v = 0.f;
            for (int w = 0; w < NW; ++w) v += __uint_as_float(red[w][slot][l]);
            a.Y[(int64_t)m * a.ldy + n] = float_to_half_bits(half_bits_to_float(a.s_x[m]) * v);
        }
    }
}

// --------------------------------------------------------------------------
// Host dispatch
// --------------------------------------------------------------------------
constexpr int kSkinnyMaxM = 32;

template <bool RAW>
static mq_status launch(mq_variant variant, const GemmArgs& a, hipStream_t stream) {
    if (variant == MQ_VARIANT_AUTO) variant = a.M <= 32 ? MQ_VARIANT_SKINNY : MQ_VARIANT_TILED;
    if (variant == MQ_VARIANT_SKINNY && a.M > kSkinnyMaxM) variant = MQ_VARIANT_TILED;
    if (variant == MQ_VARIANT_SKINNY) {
        constexpr int NW = 8;
        const dim3 grid(a.N / 16), block(64 * NW);
        if (a.M <= 16)
            hipLaunchKernelGGL((gemm_skinny_kernel<1, 1, NW, RAW>), grid, block, 0, stream, a);
        else
            hipLaunchKernelGGL((gemm_skinny_kernel<2, 1, NW, RAW>), grid, block, 0, stream, a);
    } else {
        constexpr int WM = 4, WN = 4, NW = 4;
        constexpr int BM = 16 * WM, BN = 16 * WN * NW;
        const int64_t tiles = (int64_t)((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
        if (tiles > 0x7fffffff) return MQ_ERR_UNSUPPORTED_SHAPE;
        hipLaunchKernelGGL((gemm_tiled_kernel<WM, WN, NW, RAW>), dim3((unsigned)tiles), dim3(64 * NW),
                           0, stream, a);
    }
    return mq_host::launch_status();
}

static mq_status check_common(int M, int N, int K, const uint8_t* Xq, const uint8_t* Wq,
                              const int32_t* rowptr, const int32_t* res_kb, int nnzb,
                              const uint8_t* Rq) {
    if (M < 0 || N < 0 || K < 0 || nnzb < 0) return MQ_ERR_INVALID_ARG;
    if (!mq_host::shape_ok(N, K) || M > (1 << 24)) return MQ_ERR_UNSUPPORTED_SHAPE;
    if ((int64_t)nnzb > (int64_t)(N / 128) * (K / 128)) return MQ_ERR_INVALID_ARG;
    if (M > 0 && (!Xq || !Wq)) return MQ_ERR_INVALID_ARG;
    if (nnzb > 0 && (!rowptr || !res_kb || !Rq)) return MQ_ERR_INVALID_ARG;
    if ((Xq && !mq_host::aligned(Xq, 16)) || (Wq && !mq_host::aligned(Wq, 16)) ||
        (Rq && !mq_host::aligned(Rq, 16)) || (rowptr && !mq_host::aligned(rowptr, 4)) ||
        (res_kb && !mq_host::aligned(res_kb, 4)))
        return MQ_ERR_MISALIGNED;
    return MQ_OK;
}

}  // namespace mq

using namespace mq;

extern "C" size_t mq_fused_gemm_workspace_size(int M, int N, int K) {
    (void)M; (void)N; (void)K;
    return 0;
}

extern "C" mq_status mq_fused_gemm_variant(mq_variant variant, int M, int N, int K,
                                           const uint8_t* Xq, const void* s_x,
                                           const uint8_t* Wq, const void* s_w,
                                           const int32_t* res_rowptr, const int32_t* res_kb, int nnzb,
                                           const uint8_t* Rq, const void* s_r,
                                           void* Y, int ldy,
                                           void* workspace, size_t ws_bytes, hipStream_t stream) {
    (void)workspace;
    if (variant < MQ_VARIANT_AUTO || variant > MQ_VARIANT_TILED) return MQ_ERR_INVALID_ARG;
    mq_status st = check_common(M, N, K, Xq, Wq, res_rowptr, res_kb, nnzb, Rq);
    if (st != MQ_OK) return st;
    if (ldy < N || ldy % 8 != 0) return MQ_ERR_UNSUPPORTED_SHAPE;
    if (ws_bytes < mq_fused_gemm_workspace_size(M, N, K)) return MQ_ERR_WORKSPACE;
    if (M == 0) return MQ_OK;
    if (!s_x || !s_w || !Y || (nnzb > 0 && !s_r)) return MQ_ERR_INVALID_ARG;
    if (!mq_host::aligned(s_x, 2) || !mq_host::aligned(s_w, 2) || !mq_host::aligned(Y, 2) ||
        (s_r && !mq_host::aligned(s_r, 2)))
        return MQ_ERR_MISALIGNED;
    GemmArgs a{M, N, K, Xq, static_cast<const uint16_t*>(s_x), Wq, static_cast<const uint16_t*>(s_w),
               nnzb > 0 ? res_rowptr : nullptr, res_kb, Rq, static_cast<const uint16_t*>(s_r),
               static_cast<uint16_t*>(Y), ldy, nullptr, nullptr};
    return launch<false>(variant, a, stream);
}

extern "C" mq_status mq_fused_gemm(int M, int N, int K,
                                   const uint8_t* Xq, const void* s_x,
                                   const uint8_t* Wq, const void* s_w,
                                   const int32_t* res_rowptr, const int32_t* res_kb, int nnzb,
                                   const uint8_t* Rq, const void* s_r,
                                   void* Y, int ldy,
                                   void* workspace, size_t ws_bytes, hipStream_t stream) {
    return mq_fused_gemm_variant(MQ_VARIANT_AUTO, M, N, K, Xq, s_x, Wq, s_w, res_rowptr, res_kb,
                                 nnzb, Rq, s_r, Y, ldy, workspace, ws_bytes, stream);
}

extern "C" mq_status mq_fused_gemm_acc_i32(mq_variant variant, int M, int N, int K,
                                           const uint8_t* Xq,
                                           const uint8_t* Wq,
                                           const int32_t* res_rowptr, const int32_t* res_kb, int nnzb,
                                           const uint8_t* Rq,
                                           int32_t* Tb, int32_t* Tr, hipStream_t stream) {
    if (variant < MQ_VARIANT_AUTO || variant > MQ_VARIANT_TILED) return MQ_ERR_INVALID_ARG;
    mq_status st = check_common(M, N, K, Xq, Wq, res_rowptr, res_kb, nnzb, Rq);
    if (st != MQ_OK) return st;
    if (M == 0) return MQ_OK;
    if (!Tb || !Tr) return MQ_ERR_INVALID_ARG;
    if (!mq_host::aligned(Tb, 4) || !mq_host::aligned(Tr, 4)) return MQ_ERR_MISALIGNED;
    GemmArgs a{M, N, K, Xq, nullptr, Wq, nullptr, nnzb > 0 ? res_rowptr : nullptr, res_kb, Rq,
               nullptr, nullptr, 0, Tb, Tr};
    return launch<true>(variant, a, stream);
}
