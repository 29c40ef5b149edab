// Fused dense + sparse-residual W4A4 GEMM for gfx950 (Section 3 Eq. (4) with
// the scale factorisation of Eq. (2) applied per 128-group; Section 4.2
// "Kernel Fusion" and "Overlapped pipeline").
//
//   Y[m,n] = s_x[m] * sum_g ( s_w[n,g] A_b[m,n,g] + s_r[p,n%128] A_r[m,n,g] )
//
// CDNA4 has no 4-bit integer matrix instruction.  The packed codes are stored
// so that a 16-byte pair of chunks expands with four bit operations per chunk
// into the operand of v_mfma_f32_16x16x128_f8f6f4 read as fp6 e2m3, where each
// code q is the exact subnormal q/8 (unfold_codes).  One instruction covers
// one whole 128-long group of a 16x16 output sub-tile, its fp32 result is the
// exact group sum / 64, and the epilogue is one fma per element and group with
// the scale times 64.  The residual blocks of the tile's 128-row block row are
// walked in the same K-loop: when the CSR's next column equals the current
// group, the residual fragments are multiplied with the activation fragments
// already staged for the dense term and accumulated into the same output
// registers.
//
// Two kernel families share that inner step:
//  * tiled  (prefill):  a workgroup owns a 256 x 256 (eight waves, one per CU)
//    or 128 x 128 (four waves, two per CU) output tile; the packed X, W and
//    (when present) R tiles of each group are copied by the LDS DMA into a
//    3-stage ring.
//  * streaming (decode and medium M): the eight waves of a workgroup split
//    the K groups, and the tile's residual blocks, into contiguous runs; each
//    wave streams its run through a ring of register stages (no LDS staging,
//    no barrier until the end), and the partial tiles are added through LDS
//    in wave order (deterministic).  Decode (M <= 32): all rows, 16, 32 or 64
//    columns.  Medium M: 64 x 64 (or 32 x 64) tiles, each wave the whole tile
//    over an eighth of K, so every operand piece is read once per workgroup.
#include "mq_device.h"

#include <stddef.h>

#include <mutex>
#include <type_traits>

namespace mq {

// Kernel arguments.  Pointer use by mode: the fp16 path (mq_fused_gemm*) reads
// s_x, s_w, s_r and writes Y; the raw-sum path (mq_fused_gemm_acc_i32) passes
// s_x = s_w = s_r = Y = nullptr and writes Tb, Tr.  rowptr is null when there
// are no residual blocks; res_kb, Rq (and s_r) are only read for entries of it.
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
    const uint16_t* X;       // fused-quantisation decode path: fp16 activations
    int ldx;
    int nnzb;
    int rank_rows;           // tiled kernels: order block rows by residual count (one-round grids)
    int y16;                 // Y 16-byte aligned: the tiled kernels store Y in 16-byte row pieces
    // byte sizes of Xq, Wq, Rq, s_w, s_r (each below 2 GB) and buffer
    // resources spanning each whole operand (set by launch())
    uint32_t xq_bytes, wq_bytes, rq_bytes, sw_bytes, sr_bytes;
    i32x4 rx, rw, rr, rsw, rsr;
};

// Keeps a value in registers at this point of the program: an empty volatile
// asm that reads and writes it, so everything producing it (MFMA results and
// their epilogue) must complete before the asm, inside the current block.
template <typename T>
__device__ __forceinline__ void pin(T& v) {
    asm volatile("" : "+v"(v));
}

// One m sub-tile row of one group: base MFMA + epilogue for each of the WN
// column sub-tiles, then (HAS_RES) the residual MFMA + epilogue.  sw / sr carry
// the scales times kCodeScale.  The caller picks HAS_RES once per group, so
// this is straight-line code and every MFMA result is consumed inside the
// basic block that produced it (the compiler's MFMA-to-VALU wait states are
// only placed reliably within a block).  Raw mode adds the exact integer group
// sums instead.
template <int WN, bool RAW, bool HAS_RES>
__device__ __forceinline__ void group_row(const i32x8 a, const i32x8 (&w)[WN], const i32x8 (&rr)[WN],
                                          const float (&sw)[WN], const float (&sr)[WN],
                                          f32x4 (&acc)[WN], i32x4 (&iacc)[WN], i32x4 (&racc)[WN]) {
    const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < WN; ++j) {
        const f32x4 t = mfma_codes(a, w[j], zero);
        if constexpr (RAW) {
#pragma unroll
            for (int r = 0; r < 4; ++r) iacc[j][r] += (int)(t[r] * kCodeScale);   // exact integer
        } else {
#pragma unroll
            for (int r = 0; r < 4; ++r) acc[j][r] = __builtin_fmaf(sw[j], t[r], acc[j][r]);
        }
    }
    if constexpr (HAS_RES) {
#pragma unroll
        for (int j = 0; j < WN; ++j) {
            const f32x4 t = mfma_codes(a, rr[j], zero);
            if constexpr (RAW) {
#pragma unroll
                for (int r = 0; r < 4; ++r) racc[j][r] += (int)(t[r] * kCodeScale);
            } else {
#pragma unroll
                for (int r = 0; r < 4; ++r) acc[j][r] = __builtin_fmaf(sr[j], t[r], acc[j][r]);
            }
        }
    }
}

// --------------------------------------------------------------------------
// Tiled kernel
// --------------------------------------------------------------------------
// Workgroup: 2 x WAVES_N waves owning a (32 WMB) x (64 WAVES_N) output tile:
// <8, 4> is 256 x 256 with eight waves, one workgroup per CU; <4, 2> is
// 128 x 128 with four waves, two per CU.  Wave (wm, wn) owns WMB sub-tile
// rows of 16 and four 16-column sub-tiles at tile columns 16 (wn + WAVES_N c),
// interleaved so that every wave has sub-tiles in each 128-column residual
// block row of the tile.
//
// Per 128-K group the packed X tile, W tile, the group's weight scales and,
// for block rows with a residual block at this group, the R tiles and their
// scales go by LDS DMA (buffer loads that write LDS directly, no staging
// registers) into one slot of a 3-stage ring.  One barrier per group, in the
// middle of the dense pass: it publishes group g + 1 (each wave first waits
// for its own loads) and frees the slot of group g - 1, into which the waves
// with wm == 0 then issue the loads of group g + 2; every wave reads its next
// group's W fragments, scales and first A fragment into registers right
// after it.  The DMA does not raise the compiler's wait counters, so the
// kernel waits on the vector-memory counter itself (wait_loads_and_sync).
//
// Loads use per-tile buffer resources over operands in device group order, so
// each load instruction reads 1 KB of whole 64-byte rows, contiguous.  16-byte
// chunks are XOR-swizzled by (row >> 1) & 3 inside 64-byte rows, which makes
// the 16-lane fragment reads conflict-free (LDS serves 8 lanes of 16 B per
// 128-byte bank window).
//
// After the dense pass, one residual pass per block row with a block at this
// group: every wave re-reads the staged X fragments and multiplies its
// sub-tiles of that block row, accumulating into the same registers.  With
// split-K (SPLIT), workgroup z handles a contiguous run of groups and writes
// fp32 partial sums; reduce_splits_kernel adds them in split order
// (deterministic) and applies s_x.
constexpr int kTB = 128;
constexpr int kRankMaxNB = 512;     // block rows the tiled kernel ranks by residual count
constexpr uint32_t kPastEnd = 0x80000000u;   // buffer offset past every operand (< 2 GB): reads zero

__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ ((row >> 1) & 3); }

// Tile order: blocks are dealt to the 8 XCDs round-robin, so give each XCD a
// contiguous range of a grouped tile order (the CUs of one XCD then share
// operand strips in their L2).
constexpr int kGroupM = 8;
__device__ __forceinline__ void tile_coords(int b, int tiles_m, int tiles_n, int& tm, int& tn) {
    const int nt = tiles_m * tiles_n;
    const int xcd = b % 8, k = b / 8;
    const int per = nt / 8, rem = nt % 8;
    const int t = xcd < rem ? xcd * (per + 1) + k : rem * (per + 1) + (xcd - rem) * per + k;
    // grouped order inside the range: bands of kGroupM tile rows, M fastest
    // within a band, so the tiles an XCD holds at once form a near-square
    // patch and share its L2 for both operands
    const int band = t / (kGroupM * tiles_n);
    const int first = band * kGroupM;
    const int h = min(tiles_m - first, kGroupM);
    const int r = t - band * kGroupM * tiles_n;
    tm = first + r % h;
    tn = r / h;
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ uint4 bload16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    const i32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
    return make_uint4((uint32_t)v[0], (uint32_t)v[1], (uint32_t)v[2], (uint32_t)v[3]);
}

typedef __attribute__((address_space(3))) void* lds_ptr_t;
typedef __attribute__((address_space(4))) int32_t cint32_t;   // read-only (scalar-loadable) int32

// LDS DMA (buffer loads that write LDS, lane l's bytes at dst + size * l),
// issued from inline assembly so that the compiler does not track them: its
// wait-count pass would otherwise make every later LDS read wait for all of
// them, including the prefetches of later groups.  The kernel waits for them
// itself (wait_loads_and_sync), before the barrier that publishes a stage.
// The compiler's own vector-memory waits stay correct: loads return in order,
// so loads it does not know of can only make its waits longer.
// Buffer descriptor words: base[31:0]; base[47:32] (stride 0); byte size;
// raw-buffer flags.
__device__ __forceinline__ i32x4 buf_desc(const void* base, uint32_t bytes) {
    const uint64_t b = reinterpret_cast<uint64_t>(base);
    return i32x4{(int)(uint32_t)b, (int)((uint32_t)(b >> 32) & 0xFFFFu), (int)bytes, 0x00020000};
}
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    return (uint32_t)(uintptr_t)(lds_ptr_t)p;
}
// reads at LDS byte address addr (aligned to the size read)
__device__ __forceinline__ uint4 lds_read16(uint32_t addr) {
    const i32x4 v = *(__attribute__((address_space(3))) const i32x4*)(uintptr_t)addr;
    return make_uint4((uint32_t)v[0], (uint32_t)v[1], (uint32_t)v[2], (uint32_t)v[3]);
}
__device__ __forceinline__ uint2 lds_read8(uint32_t addr) {
    const i32x2 v = *(__attribute__((address_space(3))) const i32x2*)(uintptr_t)addr;
    return make_uint2((uint32_t)v[0], (uint32_t)v[1]);
}
__device__ __forceinline__ uint16_t lds_read2(uint32_t addr) {
    return *(__attribute__((address_space(3))) const uint16_t*)(uintptr_t)addr;
}
// An LDS DMA reads M0; after an SALU write of M0 it needs one wait state
// (the compiler adds none inside inline assembly, hence the s_nop).  The
// destination and the resource are wave-uniform; readfirstlane makes that
// explicit, so they are always in scalar registers (a no-op when they are).
__device__ __forceinline__ i32x4 uniform4(const i32x4 d) {
    return i32x4{__builtin_amdgcn_readfirstlane(d[0]), __builtin_amdgcn_readfirstlane(d[1]),
                 __builtin_amdgcn_readfirstlane(d[2]), __builtin_amdgcn_readfirstlane(d[3])};
}
// Four 1 KB blocks at dst + 1024 k from voff + 1024 k (k = 0 .. 3): the
// instruction's immediate offset moves both the memory and the LDS address.
__device__ __forceinline__ void dma16x4(const i32x4 desc, uint32_t dst, uint32_t voff) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\t"
                 "buffer_load_dwordx4 %1, %2, 0 offen lds\n\t"
                 "buffer_load_dwordx4 %1, %2, 0 offen offset:1024 lds\n\t"
                 "buffer_load_dwordx4 %1, %2, 0 offen offset:2048 lds\n\t"
                 "buffer_load_dwordx4 %1, %2, 0 offen offset:3072 lds"
                 :: "s"(__builtin_amdgcn_readfirstlane(dst)), "v"(voff), "s"(uniform4(desc)) : "memory", "m0");
}
// one 1 KB block with a scalar offset added to the memory address
__device__ __forceinline__ void dma16s(const i32x4 desc, uint32_t dst, uint32_t voff, uint32_t soff) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
                 :: "s"(__builtin_amdgcn_readfirstlane(dst)), "v"(voff), "s"(uniform4(desc)),
                    "s"(__builtin_amdgcn_readfirstlane(soff)) : "memory", "m0");
}
__device__ __forceinline__ void dma4(const i32x4 desc, uint32_t dst, uint32_t voff) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dword %1, %2, 0 offen lds"
                 :: "s"(__builtin_amdgcn_readfirstlane(dst)), "v"(voff), "s"(uniform4(desc)) : "memory", "m0");
}

// f(std::integral_constant<int, I>{}) for I = 0 .. N-1, in order
template <int I, int N, typename F>
__device__ __forceinline__ void static_for_from(F&& f) {
    if constexpr (I < N) {
        f(std::integral_constant<int, I>{});
        static_for_from<I + 1, N>(f);
    }
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
    static_for_from<0, N>(f);
}

// Waits until all of this wave's vector-memory loads have landed (the LDS DMA
// does not raise the compiler's own waits), then meets the other waves of
// the workgroup.
__device__ __forceinline__ void wait_loads_and_sync() {
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Waits until at most n (0 .. 15) of this wave's vector-memory loads are in
// flight, then meets the other waves.  s_waitcnt takes an immediate, hence
// one case per count (a larger n waits as for 15, i.e. longer).
__device__ __forceinline__ void wait_vm_and_sync(int n) {
#define MQ_WAIT_CASE(k) \
    case k: asm volatile("s_waitcnt vmcnt(" #k ") lgkmcnt(0)\n\ts_barrier" ::: "memory"); break;
    switch (n) {
        MQ_WAIT_CASE(0) MQ_WAIT_CASE(1) MQ_WAIT_CASE(2) MQ_WAIT_CASE(3) MQ_WAIT_CASE(4) MQ_WAIT_CASE(5)
        MQ_WAIT_CASE(6) MQ_WAIT_CASE(7) MQ_WAIT_CASE(8) MQ_WAIT_CASE(9) MQ_WAIT_CASE(10) MQ_WAIT_CASE(11)
        MQ_WAIT_CASE(12) MQ_WAIT_CASE(13) MQ_WAIT_CASE(14)
        default: asm volatile("s_waitcnt vmcnt(15) lgkmcnt(0)\n\ts_barrier" ::: "memory"); break;
    }
#undef MQ_WAIT_CASE
}

// Tile geometry: two waves along M of WMB 16-row sub-tiles each, WAVES_N
// waves along N of 64 columns each.  <4, 2>: 128 x 128 tile, 4 waves, two
// workgroups per CU; <8, 4>: 256 x 256 tile, 8 waves, one workgroup per CU
// (half the L2 -> LDS bytes per output, the L2 being the busiest unit).
template <int WMB, int WAVES_N>
struct TileShape {
    static constexpr int kWaves = 2 * WAVES_N;
    static constexpr int kThreads = 64 * kWaves;
    static constexpr int kTM = 2 * 16 * WMB;
    static constexpr int kTN = 64 * WAVES_N;
    static constexpr int kBlockRows = kTN / kTB;          // residual block rows per tile
    static constexpr int kPerCU = kWaves == 4 ? 2 : 1;
    static_assert(kTM / 16 == 2 * kWaves && kTN / 16 == 2 * kWaves, "two 1 KB load blocks per wave and operand");
};

template <int WMB, int WAVES_N, bool RAW, bool SPLIT>
__global__ __launch_bounds__(128 * WAVES_N, (WAVES_N == 2 ? 2 : 1))   // TileShape's kThreads, kPerCU
void gemm_tiled_kernel(GemmArgs a, int groups_per_split, float* __restrict__ part) {
    using TS = TileShape<WMB, WAVES_N>;
    static_assert(TS::kThreads == 128 * WAVES_N && TS::kPerCU == (WAVES_N == 2 ? 2 : 1), "launch bounds");
    constexpr int WM = WMB, WN = 4;
    constexpr int kRow = kGroupBytes;                       // 64 bytes per row per group (W rows, X main plane)
    constexpr int kTile = kTB * kRow;                       // 8 KB: one 128-row tile
    constexpr int TM = TS::kTM, TN = TS::kTN, NBR = TS::kBlockRows, kWaves = TS::kWaves;
    constexpr int kCPerBR = WN / NBR;                       // a wave's sub-tiles per block row
    constexpr int kStages = 3;
    static_assert((NBR == 1 || NBR == 2) && kWaves == 4 * NBR, "one or two block rows, four waves per block row");
    // X, W and weight scales: three slots, loaded two groups ahead; residual
    // tiles and their scales: two slots, loaded one group ahead (they are only
    // read after the dense pass).  Arrays by kind, so that a read of a slot
    // known at compile time is one lane address plus an immediate offset.
    struct Ring {
        uint8_t x[kStages][TM * kRow];                      // activation main plane, 16-byte chunks swizzled
        uint8_t xt[kStages][2][TM * 16];                    // activation tail plane: [quarter pair][row]
        uint8_t w[kStages][TN * kRow];
        uint32_t sw[kStages][TN / 2];                       // fp16 scales, two per dword
        uint8_t r[2][NBR][kTile];
        uint32_t sr[2][NBR][kTB / 2];
        int cnt[kRankMaxNB];                                // residual blocks per block row (ranking)
        int sel[NBR];
    };
    __shared__ __attribute__((aligned(16))) Ring L;

    const int M = a.M, N = a.N, K = a.K;
    const int G = K / kGroup;
    const int t = threadIdx.x;
    const int lane = t & 63;
    const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    const int lrow = lane & 15, lq = lane >> 4;
    const int tiles_m = (M + TM - 1) / TM, tiles_n = N / TN;
    int tm, tn;
    tile_coords(blockIdx.x, tiles_m, tiles_n, tm, tn);
    const int m0 = tm * TM;
    const int gb = SPLIT ? blockIdx.y * groups_per_split : 0;
    const int ge = SPLIT ? min(G, gb + groups_per_split) : G;

    // The tile's block rows br[b] (128 output columns each).  Every tile
    // takes all K groups, so its time is set by its residual blocks: tile
    // column tn takes the block rows of rank tn (and, with two block rows, of
    // rank NB - 1 - tn) in the order of decreasing residual-block count (ties:
    // lower index first), which pairs the heaviest block row with the
    // lightest, and gives the lowest tile columns -- the first workgroups
    // dispatched -- the heaviest work.  Each workgroup ranks the block rows
    // itself (NB <= kRankMaxNB), when the host asks for it: in grids that run
    // in one round, where nothing else balances the tiles (in longer grids a
    // workgroup that finishes early takes the next tile, and the ranking's
    // cost would be paid by every workgroup).
    const int NB = N / kTB;
    int br[NBR];
#pragma unroll
    for (int b = 0; b < NBR; ++b) br[b] = tn * NBR + b;
    if (a.rank_rows && a.rowptr && NB <= kRankMaxNB) {
        for (int u = t; u < NB; u += TS::kThreads) L.cnt[u] = a.rowptr[u + 1] - a.rowptr[u];
        __syncthreads();
        for (int u = t; u < NB; u += TS::kThreads) {
            const int c = L.cnt[u];
            int rank = 0;
            for (int v = 0; v < NB; ++v) {
                const int cv = L.cnt[v];
                rank += (cv > c) | ((cv == c) & (v < u));
            }
            if (rank == tn) L.sel[0] = u;
            if (NBR == 2 && rank == NB - 1 - tn) L.sel[NBR - 1] = u;
        }
        __syncthreads();
#pragma unroll
        for (int b = 0; b < NBR; ++b) br[b] = __builtin_amdgcn_readfirstlane(L.sel[b]);
    }

    // Operands in device group order: the group-g main-plane tile of X rows
    // m0.. is xrows * 64 contiguous bytes at (g M + m0) 64, that of block row
    // br 8 KB at (g N + 128 br) 64, and R block p is 8 KB.  These loads
    // go through a resource spanning exactly that tile (offsets in the vector
    // operand only), so X rows past xrows fail the range check and read zero;
    // the tail-plane loads use the whole-operand resource with such rows moved
    // past its end.
    const uint32_t xrows = (uint32_t)min(TM, M - m0);
    const uint32_t xbytes = xrows * (uint32_t)kRow;
    const uint32_t tail0 = (uint32_t)G * (uint32_t)M * (uint32_t)kRow;

    // CSR walks of the tile's NBR block rows, from the first entry at or after
    // gb.  They read through the constant address space so they stay in scalar
    // registers (scalar loads do not count against the vector-memory counter
    // the pipeline waits on).  nk[b] is the group of block row b's next block
    // (INT_MAX: none), loaded one entry ahead so no group waits for it.
    const cint32_t* res_kb = (const cint32_t*)(a.res_kb);
    int rp[NBR], re[NBR], nk[NBR];
#pragma unroll
    for (int b = 0; b < NBR; ++b) {
        rp[b] = re[b] = 0;
        nk[b] = 0x7fffffff;
        if (a.rowptr) {
            const cint32_t* rowptr = (const cint32_t*)(a.rowptr);
            rp[b] = rowptr[br[b]];
            re[b] = rowptr[br[b] + 1];
            while (rp[b] < re[b] && res_kb[rp[b]] < gb) ++rp[b];
            if (rp[b] < re[b]) nk[b] = res_kb[rp[b]];
        }
    }

    // Loads.  The WAVES_N waves with wm == 0 (the loaders, ld = wn) fetch
    // everything; they are the ones that reach the group's barrier first (the
    // older waves win issue), so the issue cost lands where there is slack.
    // Loader ld fills the 1 KB blocks (16 rows each) 4 ld .. 4 ld + 3 of the X
    // main-plane and W tiles, the tail-plane blocks 2 ld and 2 ld + 1 (block b:
    // the 16 bytes of quarters 2 jp, 2 jp + 1 of rows 64 kb + l, jp = b / (TM / 64),
    // kb = b % (TM / 64); in LDS the tail tile is [quarter pair][row]),
    // and of the residual tiles of the block rows flattened (block 8 br + j is
    // block j of block row br), i.e. blocks 4 (ld & 1) .. + 3 of block row
    // ld / 2, when that block row has a block at the group; and its scale
    // share: loaders ld < NBR the weight scales of block row ld, loaders
    // NBR .. 2 NBR - 1 the residual scales of block row ld - NBR (256 B each).
    // Lane l takes row 16 b + l / 4 and physical chunk l % 4, i.e. logical
    // chunk (l % 4) ^ swz(row) of that row, so each load instruction reads
    // 1 KB of whole 64-byte rows, contiguous.
    static_assert(TM == 64 * WAVES_N && TN == 64 * WAVES_N && 8 * NBR == 4 * WAVES_N,
                  "four X, W and R blocks per loader");
    static_assert(TM / 32 == 2 * WAVES_N, "two tail-plane blocks per loader");
    const bool loader = wm == 0;
    const int ld = wn, lbr = ld >> 1;
    // lane offsets of the first of the loader's four blocks (the swizzle of
    // row 16 b + l / 4 is (l / 8) % 4 for every b, so block k is 1024 k on)
    const uint32_t vt = (uint32_t)(64 * ld + (lane >> 2)) * kRow + (((lane & 3) ^ ((lane >> 3) & 3)) << 4);
    const uint32_t vr = (uint32_t)(64 * (ld & 1) + (lane >> 2)) * kRow + (((lane & 3) ^ ((lane >> 3) & 3)) << 4);
    // tail blocks: quarter pair tq[k], rows trow[k] + l (lane offsets past the
    // end for rows from M on)
    constexpr int kRowBlocks = TM / 64;                     // 64-row blocks of the tail tile per quarter pair
    int tq[2], trow[2];
    uint32_t vtl[2];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const int b = 2 * ld + k;
        tq[k] = b / kRowBlocks;
        trow[k] = 64 * (b % kRowBlocks);
        vtl[k] = ((uint32_t)(trow[k] + lane) * 32u + 16u * (uint32_t)tq[k]) | (m0 + trow[k] + lane < M ? 0u : kPastEnd);
    }

    // Loads of group g into `slot` (issued by the loaders right after the
    // barrier inside the dense pass of group g - 2; past the last group they
    // read nothing: zero-size resources, offsets past the end).  p[b] is block
    // row b's residual block at g (-1: none).
    struct Plan {
        i32x4 xr, wr, sc;                    // resources
        uint32_t x, w, s, xt[2];             // LDS destinations
        uint32_t xto[2];                     // tail-plane block offsets (uniform; past the end: read nothing)
        bool has_s;
    };
    auto plan = [&](int g, int slot, int (&p)[NBR]) -> Plan {
        const bool live = g < ge;
        const int gl = live ? g : 0;
        Plan P;
        P.xr = buf_desc(a.Xq + piece_offset(M, m0, gl), live ? xbytes : 0u);
        P.wr = buf_desc(a.Wq + piece_offset(N, kTB * br[lbr], gl), live ? (uint32_t)kTile : 0u);
        P.x = lds_addr(&L.x[slot][(4 * ld) * 1024]);
        P.w = lds_addr(&L.w[slot][(4 * ld) * 1024]);
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            P.xt[k] = lds_addr(&L.xt[slot][tq[k]][trow[k] * 16]);
            P.xto[k] = live ? tail0 + ((uint32_t)gl * (uint32_t)M + (uint32_t)m0) * 32u : kPastEnd;
        }
#pragma unroll
        for (int b = 0; b < NBR; ++b) {
            p[b] = -1;
            if (live && nk[b] == g) {
                p[b] = rp[b]++;
                nk[b] = rp[b] < re[b] ? res_kb[rp[b]] : 0x7fffffff;
            }
        }
        P.has_s = false;
        P.sc = buf_desc(a.Wq, 0u);
        P.s = 0;
        if constexpr (!RAW) {
            if (live && ld < NBR) {
                P.has_s = true;
                P.sc = buf_desc(a.s_w + wscale_index(N, kTB * br[ld], g), kTB * 2);
                P.s = lds_addr(&L.sw[slot][64 * ld]);
            }
        }
        return P;
    };
    // Residual loads of group g (blocks p) into residual slot rs, issued one
    // group ahead.
    struct RPlan {
        i32x4 rr, sc;
        uint32_t r, s;
        bool has_r, has_s;
    };
    auto rplan = [&](int rs, const int (&p)[NBR]) -> RPlan {
        RPlan P;
        const int pr = (NBR == 2 && lbr == 1) ? p[NBR - 1] : p[0];
        P.has_r = pr >= 0;
        P.rr = buf_desc(a.Rq + (int64_t)(pr >= 0 ? pr : 0) * kTile, (uint32_t)kTile);
        P.r = lds_addr(&L.r[rs][lbr][(4 * (ld & 1)) * 1024]);
        P.has_s = false;
        P.sc = buf_desc(a.Wq, 0u);
        P.s = 0;
        if constexpr (!RAW) {
            const int sb = ld - NBR;
            const int ps = (NBR == 2 && sb == 1) ? p[NBR - 1] : p[0];
            if (sb >= 0 && sb < NBR && ps >= 0) {
                P.has_s = true;
                P.sc = buf_desc(a.s_r + (int64_t)ps * kTB, kTB * 2);
                P.s = lds_addr(L.sr[rs][sb]);
            }
        }
        return P;
    };
    // the loads of a plan (loaders only; outside any MFMA block)
    auto issue = [&](const Plan& P) {
        if (!loader) return;
        dma16x4(P.xr, P.x, vt);
#pragma unroll
        for (int k = 0; k < 2; ++k) dma16s(a.rx, P.xt[k], vtl[k], P.xto[k]);
        dma16x4(P.wr, P.w, vr);                            // rows of block row lbr
        if (P.has_s) dma4(P.sc, P.s, (uint32_t)lane * 4);
    };
    auto issue_r = [&](const RPlan& P) {
        if (!loader) return;
        if (P.has_r) dma16x4(P.rr, P.r, vr);
        if (P.has_s) dma4(P.sc, P.s, (uint32_t)lane * 4);
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

    // The wave's rows wrow .. wrow + 16 WM - 1 and its column sub-tiles
    // c = 0 .. 3 at tile columns 16 (wn + WAVES_N c) .., interleaved so that
    // every wave has kCPerBR sub-tiles in each residual block row: a residual
    // block keeps all the waves busy, not only those of its block row.
    const int wrow = 16 * WM * wm;

    // LDS reads.  Every row and column this lane reads has the same swizzle
    // (rows wrow + 16 i + lrow, columns 16 (wn + WAVES_N c) + lrow: (row / 2) % 4
    // is (lrow / 2) % 4), so each read is a lane offset computed once plus a
    // constant (slot, sub-tile row i, sub-tile column c).
    // The lane offsets include the start of their array (each kept opaque to
    // the compiler, so that the constant that remains is below the 64 KB of
    // an LDS instruction's immediate offset).
    const uint32_t swz_l = (uint32_t)(lq ^ ((lrow >> 1) & 3)) << 4;
    auto lane_base = [](const void* array, uint32_t off) {
        uint32_t v = lds_addr(array) + off;
        asm volatile("" : "+v"(v));
        return v;
    };
    const uint32_t xo = lane_base(L.x, (uint32_t)(wrow + lrow) * kRow + swz_l);                   // + 1024 i
    const uint32_t to = lane_base(L.xt, (uint32_t)(lq >> 1) * (TM * 16) + (uint32_t)(wrow + lrow) * 16 +
                                            (uint32_t)(lq & 1) * 8);                           // + 256 i
    const uint32_t wo = lane_base(L.w, (uint32_t)(16 * wn + lrow) * kRow + swz_l);      // + 1024 WAVES_N c
    const uint32_t so = lane_base(L.sw, (uint32_t)(16 * wn + lrow) * 2);                // + 32 WAVES_N c
    const uint32_t ro = lane_base(L.r, (uint32_t)(16 * wn + lrow) * kRow + swz_l);
    const uint32_t sro = lane_base(L.sr, (uint32_t)(16 * wn + lrow) * 2);
    // the activation operand of sub-tile row i: main-plane chunk and tail
    auto a_main = [&](int slot, int i) { return lds_read16(xo + TM * kRow * slot + 1024 * i); };
    auto a_tail = [&](int slot, int i) { return lds_read8(to + TM * 32 * slot + 256 * i); };
    // a weight or residual scale as an fp32 register value (kept out of the
    // fma, whose mixed-precision form measured slower)
    auto scale_f32 = [](uint16_t bits) {
        float v = half_bits_to_float(bits);
        asm volatile("" : "+v"(v));
        return v;
    };

    // Operands of a group's dense pass that are read ahead, right after the
    // barrier that publishes the group (in the middle of the previous group's
    // dense pass): the wave's four W fragments (folded), their scales and its
    // first A fragment.  The pass then starts without waiting for LDS.
    struct Ahead {
        uint4 w[WN], a0;
        uint2 a0t;
        uint16_t s[WN];
    };
    auto read_ahead = [&](int slot, Ahead& H) {
#pragma unroll
        for (int c = 0; c < WN; ++c) {
            H.w[c] = lds_read16(wo + TN * kRow * slot + 1024 * WAVES_N * c);
            H.s[c] = RAW ? 0 : lds_read2(so + TN * 2 * slot + 32 * WAVES_N * c);
        }
        H.a0 = a_main(slot, 0);
        H.a0t = a_tail(slot, 0);
    };

    // One pass over the staged group S.  The dense pass (RES == 0) multiplies
    // all four sub-tiles with the W fragments (from H); in the middle of it
    // (MFMAs of the first half still running: the compiler places the wait
    // states of their results across the blocks of the load issue) it waits
    // for the loads in flight, meets the other waves (which frees the slots of
    // the previous group), has the loaders issue the loads of plans P and RP
    // and reads the next group's operands ahead into H.  A residual pass
    // multiplies the sub-tiles in the bit set RES (those of one block row) with
    // the R fragments of that block row from residual slot RS.  The fp32 path
    // accumulates scale x (group sum / 64); the factor 64 is applied once, in
    // the final epilogue (exact).
    constexpr int kSync = WM / 2;
    auto phase = [&](auto slot_c, auto res_c, Ahead& H, int rs, const Plan& P, const RPlan& RP) {
        constexpr int SL = decltype(slot_c)::value, SNEXT = SL == kStages - 1 ? 0 : SL + 1;
        constexpr int RES = decltype(res_c)::value;
        constexpr bool DENSE = RES == 0;
        constexpr int kBR = DENSE ? 0 : (RES >> kCPerBR ? 1 : 0);   // block row of a residual pass
        auto has = [](int c) { return DENSE || ((RES >> c) & 1); };
        i32x8 b[WN];
        float bs[WN];
#pragma unroll
        for (int c = 0; c < WN; ++c) {
            if (!has(c)) continue;
            if constexpr (DENSE) {
                b[c] = unfold_codes(H.w[c]);
                bs[c] = RAW ? 0.f : scale_f32(H.s[c]);
            } else {
                // row 16 (wn + WAVES_N c) + lrow - 128 kBR of the block row's R tile
                const int rc = 1024 * WAVES_N * c - kTile * kBR;
                b[c] = unfold_codes(lds_read16(ro + (uint32_t)(rs * NBR * kTile) + kBR * kTile + rc));
                bs[c] = RAW ? 0.f : scale_f32(lds_read2(sro + (uint32_t)(rs * NBR * kTB * 2) + kBR * kTB * 2 + rc / 32));
            }
        }
        // Software pipeline over the sub-tile rows: the activation operand of
        // row i + 1 is read before the MFMAs of row i are issued, and those
        // before the epilogue of row i - 1, so each result is read several
        // MFMAs after it was started (no wait states to fill).
        f32x4 tq[2][WN];
        auto a_row = [&](auto ic) -> i32x8 {
            constexpr int i = decltype(ic)::value;
            if constexpr (DENSE && i == 0) return act_operand(H.a0, H.a0t);
            else return act_operand(a_main(SL, i), a_tail(SL, i));
        };
        auto mfma_row = [&](auto ic, const i32x8 av) {
            constexpr int i = decltype(ic)::value;
#pragma unroll
            for (int c = 0; c < WN; ++c)
                if (has(c)) tq[i & 1][c] = mfma_codes(av, b[c], f32x4{0.f, 0.f, 0.f, 0.f});
        };
        auto epilogue_row = [&](auto ic) {
            constexpr int i = decltype(ic)::value;
#pragma unroll
            for (int c = 0; c < WN; ++c) {
                if (!has(c)) continue;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    if constexpr (!RAW) acc[i][c][r] = __builtin_fmaf(bs[c], tq[i & 1][c][r], acc[i][c][r]);
                    else if constexpr (DENSE) iacc[i][c][r] += (int)(tq[i & 1][c][r] * kCodeScale);   // exact
                    else racc[i][c][r] += (int)(tq[i & 1][c][r] * kCodeScale);
                }
            }
        };
        // Rows 0 .. WM - 1, software-pipelined.  The dense pass meets the
        // other waves after issuing the MFMAs of row kSync - 1 (its operand
        // for row kSync already read: the current slot is not touched by the
        // barrier), so those MFMAs run across the barrier, the loads and the
        // reads ahead, and row kSync's MFMAs can issue right after them.
        // Each row's sums are pinned right after its epilogue, which keeps
        // that epilogue in place (the compiler would otherwise sink it past
        // the barrier and the load issue).
        auto pin_row = [&](int i) {
#pragma unroll
            for (int c = 0; c < WN; ++c) {
                if (!has(c)) continue;
                if constexpr (!RAW) pin(acc[i][c]);
                else if constexpr (DENSE) pin(iacc[i][c]);
                else pin(racc[i][c]);
            }
        };
        // The activation operand is read two rows ahead (one row of MFMAs
        // and epilogue does not cover the LDS latency).
        i32x8 av = a_row(std::integral_constant<int, 0>{});
        i32x8 an = av;
        if constexpr (WM > 1) an = a_row(std::integral_constant<int, 1>{});
        static_for<WM>([&](auto ic) {
            constexpr int i = decltype(ic)::value;
            i32x8 ann = an;
            if constexpr (i + 2 < WM) ann = a_row(std::integral_constant<int, i + 2>{});
            mfma_row(std::integral_constant<int, i>{}, av);
            if constexpr (i > 0) {
                epilogue_row(std::integral_constant<int, i - 1>{});
                pin_row(i - 1);
            }
            if constexpr (DENSE && i == kSync - 1) {
                wait_loads_and_sync();      // the only loads in flight are those issued one group ago
                issue(P);
                issue_r(RP);
                read_ahead(SNEXT, H);
            }
            av = an;
            an = ann;
        });
        epilogue_row(std::integral_constant<int, WM - 1>{});
        pin_row(WM - 1);
    };

    // residual blocks of the current group and of the groups one and two
    // ahead (-1: none), per block row
    int p_cur[NBR], p_next[NBR], p_new[NBR];
    issue(plan(gb, 0, p_cur));
    issue_r(rplan(gb & 1, p_cur));
    const Plan P1 = plan(gb + 1, 1, p_next);
    issue(P1);
    constexpr int kBR0 = (1 << kCPerBR) - 1;                // sub-tiles of block row 0
    // group gb (and its residual tiles) have landed once no more than the
    // loads of group gb + 1 (ten, plus its weight scales) are in flight; the
    // barrier inside gb's dense pass waits for the rest
    wait_vm_and_sync(loader ? 10 + (P1.has_s ? 1 : 0) : 0);
    Ahead H;
    read_ahead(0, H);
    // Group g (ring slot SL, known at compile time: the loop below is unrolled
    // three times) holds its operands (published by the barrier inside the
    // previous dense pass), residual slot g & 1 its residual tiles, and H its
    // dense pass's first operands.  The dense pass issues the loads of group
    // g + 2 into the slot of group g - 1 and the residual loads of group g + 1
    // into the residual slot of group g - 1, both freed by its barrier; then a
    // residual pass per block row with a block at this group: every wave
    // multiplies its kCPerBR sub-tiles of that block row.  (Passes rather than
    // variants of the dense code: one code path per group keeps the
    // accumulators in fixed registers.)
    auto step = [&](auto slot_c, int g) {
        constexpr int SL = decltype(slot_c)::value, SFREE = (SL + 2) % kStages;
        const Plan P = plan(g + 2, SFREE, p_new);
        const RPlan RP = rplan((g + 1) & 1, p_next);
        const int rs = g & 1;
        phase(slot_c, std::integral_constant<int, 0>{}, H, rs, P, RP);
        if (p_cur[0] >= 0) phase(slot_c, std::integral_constant<int, kBR0>{}, H, rs, P, RP);
        if constexpr (NBR == 2)
            if (p_cur[1] >= 0) phase(slot_c, std::integral_constant<int, kBR0 << kCPerBR>{}, H, rs, P, RP);
#pragma unroll
        for (int b = 0; b < NBR; ++b) {
            p_cur[b] = p_next[b];
            p_next[b] = p_new[b];
        }
    };
    for (int g = gb; g < ge; g += kStages) {
        step(std::integral_constant<int, 0>{}, g);
        if (g + 1 < ge) step(std::integral_constant<int, 1>{}, g + 1);
        if (g + 2 < ge) step(std::integral_constant<int, 2>{}, g + 2);
    }
    // the X and W loads issued for the two groups past the end read nothing,
    // but they still write a ring slot: let them finish first
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

    // epilogue: lane holds rows 4 * (lane / 16) + r of each sub-tile, column
    // lane % 16; the fp32 sums are scale x (group sum / 64)
    if constexpr (!RAW && !SPLIT) {
        if (a.y16) {
            // fp16 Y through the ring's LDS: the tile, row-major (row r, local
            // column lc = 16 (wn + WAVES_N c) + lrow, i.e. block row br[lc / 128]),
            // its 16-byte chunks (8 columns) swizzled by chunk ^ 2 ((r / 4) % 4) so
            // the four row quarters a write covers hit distinct banks; then each
            // thread stores whole 16-byte row pieces (eight times fewer store
            // instructions than one fp16 value a lane, each covering whole lines)
            static_assert(sizeof(Ring) >= (size_t)TM * TN * 2, "the output tile fits the ring");
            uint8_t* ys = reinterpret_cast<uint8_t*>(&L);
            auto ys_off = [](int r, int lc) {
                return (uint32_t)r * (uint32_t)(TN * 2) + (uint32_t)((((lc >> 3) ^ (((r >> 2) & 3) << 1)) << 4) +
                                                                     ((lc & 7) << 1));
            };
            __syncthreads();                              // every wave is done with the ring
#pragma unroll
            for (int i = 0; i < WM; ++i) {
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int rl = wrow + 16 * i + 4 * lq + r;
                    const int m = m0 + rl;
                    const float sx = m < M ? half_bits_to_float(a.s_x[m]) * kCodeScale : 0.f;
#pragma unroll
                    for (int c = 0; c < WN; ++c)
                        *reinterpret_cast<uint16_t*>(ys + ys_off(rl, 16 * (wn + WAVES_N * c) + lrow)) =
                            float_to_half_bits(sx * acc[i][c][r]);
                }
            }
            __syncthreads();
            constexpr int kPiecesPerRow = TN / 8;
            const int rows = min(TM, M - m0);
            for (int q = t; q < rows * kPiecesPerRow; q += TS::kThreads) {
                const int rl = q / kPiecesPerRow, lc = 8 * (q % kPiecesPerRow);
                const int n = kTB * br[lc / kTB] + (lc & (kTB - 1));
                *reinterpret_cast<uint4*>(a.Y + (int64_t)(m0 + rl) * a.ldy + n) =
                    *reinterpret_cast<const uint4*>(ys + ys_off(rl, lc));
            }
            return;
        }
    }
#pragma unroll
    for (int i = 0; i < WM; ++i) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int m = m0 + wrow + 16 * i + 4 * lq + r;
            if (m >= M) continue;
            const float sx = (RAW || SPLIT) ? 0.f : half_bits_to_float(a.s_x[m]) * kCodeScale;
#pragma unroll
            for (int c = 0; c < WN; ++c) {
                const int n = kTB * br[c / kCPerBR] + ((16 * (wn + WAVES_N * c) + lrow) & (kTB - 1));
                if constexpr (RAW && SPLIT) {
                    // integer sums of a group range: added in any order, exact
                    atomicAdd(&a.Tb[(int64_t)m * N + n], iacc[i][c][r]);
                    atomicAdd(&a.Tr[(int64_t)m * N + n], racc[i][c][r]);
                } else if constexpr (RAW) {
                    a.Tb[(int64_t)m * N + n] = iacc[i][c][r];
                    a.Tr[(int64_t)m * N + n] = racc[i][c][r];
                } else if constexpr (SPLIT) {
                    part[((int64_t)blockIdx.y * M + m) * N + n] = acc[i][c][r] * kCodeScale;
                } else {
                    a.Y[(int64_t)m * a.ldy + n] = float_to_half_bits(sx * acc[i][c][r]);
                }
            }
        }
    }
}

#ifndef MQ_MEDIUM_TU
// Y[m, n] = fp16(s_x[m] * sum_{s < splits} part[s, m, n]), summed in split order.
__global__ __launch_bounds__(256) void reduce_splits_kernel(const float* __restrict__ part, int splits,
                                                            int M, int N, const uint16_t* __restrict__ s_x,
                                                            uint16_t* __restrict__ Y, int ldy) {
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t total = (int64_t)M * N;
    if (idx >= total) return;
    const int m = (int)(idx / N), n = (int)(idx % N);
    float v = 0.f;
    for (int s = 0; s < splits; ++s) v += part[s * total + idx];
    Y[(int64_t)m * ldy + n] = float_to_half_bits(half_bits_to_float(s_x[m]) * v);
}

// Zero-fills n int32 (the raw split-K sums are accumulated into them).
__global__ __launch_bounds__(256) void fill_zero_kernel(int32_t* __restrict__ p, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0;
}
#endif

// Split-K factor for the tiled kernel: doubled while the split grid still
// fits in one round of two workgroups per CU (at least 8 groups per split).
// Past one round only when the splits stay long (32 groups or more), where
// more, shorter workgroups pay for the partial round: 25600 -> 5120 at M = 512
// (160 tiles) 124 us with two splits, 108 with four; at shorter K the extra
// half round costs more (K = N = 4096 at M = 1536, 384 tiles: 55.7 us with two
// splits, 39.7 with none; 4096 -> 14336 at M = 512: 69 against 44.4 us).
static int tiled_splits(int M, int N, int K) {
    const int64_t tiles = (int64_t)((M + kTB - 1) / kTB) * (N / kTB);
    const int G = K / kGroup;
    int s = 1;
    while (G / (s * 2) >= 8 && (tiles * s * 2 <= 512 || (tiles * s < 512 && G / (s * 2) >= 32))) s *= 2;
    return s;
}

// --------------------------------------------------------------------------
// Decode kernel (M <= 32): a workgroup owns SPW adjacent 16-column strips
// (16 SPW <= 64 columns, inside one 128-row block row) and all M rows.  Its
// eight waves split the K groups into contiguous runs, and the block row's
// residual blocks into contiguous runs of its CSR entries (by entry, not by
// group: no search of the CSR, and hot block rows spread over all waves).
// Each wave streams its groups and then its blocks as one sequence of items
// through a ring of GD register stages (the loads of GD items in flight; the
// SPW strips of an item are adjacent 1 KB pieces of Wq or of the block).
// Partial sums are added through LDS in wave order (deterministic).  A stage
// holding an item issues a fixed number of loads; a stage past the last item
// issues none (loads at offsets past the resource, which read zeros, still
// cost nearly as much as real ones: issuing them measured up to 20 % slower).
// When the tiles outnumber a round of resident workgroups, each workgroup
// takes several in turn (PT), with one item stream running through them.
// --------------------------------------------------------------------------
// Fused activation quantisation (FQ): at most kFusedMaxM rows and
// kFusedCPT 16-element chunks per thread; the workgroup quantises the rows
// into LDS itself (same arithmetic as mq_quantize_act) instead of reading Xq.
constexpr int kFusedMaxM = 4, kFusedCPT = 4;
constexpr int kDecodeWaves = 8;

// Items in flight per wave: stages of WM X fragments, WN B fragments and
// their scales filling about 96 registers (measured: a deeper ring of the 64 x 64
// medium tile, 144 registers, ran slower).
template <int WM, int WN, bool RAW, bool A8 = false>
struct StreamDepth {
    static constexpr int kStageRegs = (A8 ? 12 : 6) * WM + 4 * WN + (WN == 4 ? 1 : WN);
    static constexpr int kBudget = 96;
    static constexpr int GD = kBudget / kStageRegs < 2 ? 2 : kBudget / kStageRegs > 6 ? 6 : kBudget / kStageRegs;
};

// The streaming kernel: eight waves = KS = 8 / (WGM WGN) splits of the K
// loop x a WGM x WGN grid of waves, each wave WM x WN sub-tiles of 16 x 16:
// a (16 WM WGM) x (16 WN WGN) output tile.  Decode: WM <= 2, WN = 1, 2 or 4
// (all M <= 32 rows, K over eight waves); medium M: WM = 2 or 4, WN = 4 (the
// whole 32 x 64 or 64 x 64 tile per wave, K over eight waves).
// The W4A4 activation operand is read in its stored operand form (main-plane
// chunk and tail), fused quantisation (FQ) unfolds its codes from LDS.
// A8 (the W4A8 variant): the activation operand is INT8, stored as an e4m3
// high plane and a folded 4-bit low plane (mq_quantize_act8); each product
// takes the low-plane MFMA and the fp8 x fp6 MFMA of the high plane chained
// on its result (both exact), the rest is unchanged.
template <int WM, int WN, int WGM, int WGN, bool RAW, bool FQ, bool A8 = false, bool XS = false, bool PT = false>
__global__ __launch_bounds__(64 * kDecodeWaves) void gemm_stream_kernel(GemmArgs a) {
    static_assert(WN * WGN == 1 || WN * WGN == 2 || WN * WGN == 4 || WN * WGN == 8,
                  "tile columns inside one block row");
    static_assert(!(FQ && RAW), "fused quantisation feeds the fp16 path");
    static_assert(!FQ || (WGM == 1 && WGN == 1), "fused quantisation: one tile of all rows");
    static_assert(!(FQ && A8), "fused quantisation is the W4A4 decode path");
    constexpr bool A4 = !FQ && !A8;                              // activations in operand form
    static_assert(!XS || (A4 && WGM == 1 && WGN == 1), "staged activations: the W4A4 decode tile");
    constexpr bool A4G = A4 && !XS;                              // ... read from memory per item
    constexpr int NW = kDecodeWaves, WG2 = WGM * WGN, KS = NW / WG2;
    static_assert(KS * WG2 == NW, "eight waves");
    constexpr int TM = 16 * WM * WGM, TN = 16 * WN * WGN;
    constexpr int SPW = WN;
    // PT (decode with fused quantisation or staged activations): the
    // workgroup takes the tiles blockIdx.x + k gridDim.x in turn (all in tile
    // row 0), quantising or staging the rows once for all of them
    static_assert(!PT || FQ || XS, "several tiles a workgroup: the decode tiles");
    constexpr int GD = StreamDepth<WM, WN, RAW, A8>::GD;
    constexpr bool kScaleShfl = SPW == 4;
    constexpr int kAcc = WM * SPW * 4;                           // sums per lane and accumulator
    // cross-wave partial sums red[wave][value][lane] (one accumulator per
    // round: raw mode adds the base and then the residual sums); FQ: packed
    // codes of the M rows (M x K/2 bytes, row-major) in dynamic LDS
    __shared__ __attribute__((aligned(16))) uint32_t red[NW][kAcc][64];
    extern __shared__ __attribute__((aligned(16))) uint8_t dyn[];
    __shared__ uint32_t amax_sh[kFusedMaxM];
    __shared__ uint16_t sx_sh[kFusedMaxM];
    uint8_t* xs = dyn;

    const int M = a.M, N = a.N, K = a.K;
    const int G = K / kGroup;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
    const int lrow = lane & 15, lq = lane >> 4;
    const int split = wave / WG2, wpos = wave % WG2, wm = wpos / WGN, wn = wpos % WGN;
    const int tiles_m = (M + TM - 1) / TM, tiles_n = N / TN;
    int tm, tn;
    tile_coords(blockIdx.x, tiles_m, tiles_n, tm, tn);
    const int m0 = tm * TM, n0 = tn * TN;
    const int nb = n0 / kGroup, roff = n0 % kGroup;
    const int mw = m0 + 16 * WM * wm;                            // the wave's first row
    const int nw = 16 * WN * wn;                                 // its first column inside the tile

    // this split's run of groups
    const int gper = G / KS, gextra = G % KS;
    const int gb = split * gper + min(split, gextra);
    const int ng = gper + (split < gextra ? 1 : 0);

    // this split's run of the block row's CSR entries (scalar loads through
    // the constant address space: off the vector-memory counter)
    const cint32_t* res_kb = (const cint32_t*)(a.res_kb);
    int pb = 0, ne = 0;
    // PT: the workgroup's ntw tiles (at most 64; every wave has at least one
    // group in each), lane k holding tile k's first column (vn0) and this
    // split's run of its block row's entries (vpb, vne); the wave's items
    // over all its tiles: nall
    int ntw = 1, vn0 = n0, vpb = 0, vne = 0, nall = 0;
    if constexpr (PT) {
        ntw = (tiles_n - (int)blockIdx.x + (int)gridDim.x - 1) / (int)gridDim.x;
        if (lane < ntw) {
            int tml, tnl;
            tile_coords((int)blockIdx.x + lane * (int)gridDim.x, tiles_m, tiles_n, tml, tnl);
            vn0 = tnl * TN;
            if (a.rowptr) {
                const int nbl = vn0 / kGroup;
                const int rp = a.rowptr[nbl], cnt = a.rowptr[nbl + 1] - rp;
                const int eper = cnt / KS, eextra = cnt % KS;
                vpb = rp + split * eper + min(split, eextra);
                vne = eper + (split < eextra ? 1 : 0);
            }
        }
        int sum = vne;
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o, 64);
        nall = __builtin_amdgcn_readfirstlane(sum) + ntw * ng;
        pb = __builtin_amdgcn_readlane(vpb, 0);
        ne = __builtin_amdgcn_readlane(vne, 0);
    } else if (a.rowptr) {
        const cint32_t* rowptr = (const cint32_t*)(a.rowptr);
        const int rp = rowptr[nb], cnt = rowptr[nb + 1] - rp;
        const int eper = cnt / KS, eextra = cnt % KS;
        pb = rp + split * eper + min(split, eextra);
        ne = eper + (split < eextra ? 1 : 0);
    }

    // whole-operand resources (32-bit offsets; launch() checks every operand < 2 GB)
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(FQ ? a.Wq : a.Xq, FQ ? 0u : a.xq_bytes);
    const uint32_t loff = (uint32_t)lrow * kGroupBytes + (uint32_t)lq * 16;   // lane's bytes of a 16-row piece

    // X fragment of rows 16 i .. 16 i + 15 at group g: from the quantised rows
    // in LDS (FQ; rows past M read 0) or from Xq (rows past M read 0)
    auto x_offset = [&](int g, int i) -> uint32_t {
        return ((uint32_t)g * (uint32_t)M + (uint32_t)mw + 16u * i) * kGroupBytes + loff;
    };
    // XS: the rows' operand bytes copied into LDS at the start, in the
    // layout of Xq except that the 16-byte chunk q of a main-plane row r sits
    // at chunk q ^ ((r / 4) % 4) (the 16 rows of a read then hit distinct
    // banks); rows from M on read row M - 1 (their outputs are not written)
    auto xs_main = [&](int g, int r, int q) -> uint32_t {
        return ((uint32_t)g * (uint32_t)M + (uint32_t)r) * 64u + ((uint32_t)(q ^ ((r >> 2) & 3)) << 4);
    };
    auto x_staged = [&](int g, int i) -> i32x8 {
        const int r = min(mw + 16 * i + lrow, M - 1);
        const uint4 mv = *reinterpret_cast<const uint4*>(&xs[xs_main(g, r, lq)]);
        const uint2 tv = *reinterpret_cast<const uint2*>(
            &xs[(uint32_t)G * (uint32_t)M * 64u + ((uint32_t)g * (uint32_t)M + (uint32_t)r) * 32u + (uint32_t)lq * 8u]);
        return act_operand(mv, tv);
    };
    auto x_lds = [&](int g, int i) -> uint4 {
        const int row = mw + 16 * i + lrow;
        uint4 v = make_uint4(0u, 0u, 0u, 0u);
        if (row < M) v = *reinterpret_cast<const uint4*>(&xs[(int64_t)row * (K / 2) + g * kGroupBytes + lq * 16]);
        return v;
    };

    f32x4 acc[WM][SPW];
    i32x4 iacc[WM][SPW], racc[WM][SPW];
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
        for (int s = 0; s < SPW; ++s) {
            acc[i][s] = f32x4{0.f, 0.f, 0.f, 0.f};
            iacc[i][s] = i32x4{0, 0, 0, 0};
            racc[i][s] = i32x4{0, 0, 0, 0};
        }
    auto pin_all = [&]() {
#pragma unroll
        for (int i = 0; i < WM; ++i)
#pragma unroll
            for (int s = 0; s < SPW; ++s) {
                if constexpr (RAW) { pin(iacc[i][s]); pin(racc[i][s]); }
                else pin(acc[i][s]);
            }
    };

    // One stream of items per wave: its dense groups (group gb + j, B = the
    // strips' W pieces, scales s_w), then its residual entries (block p at
    // group res_kb[p], B = the strips' R pieces, scales s_r), through one ring
    // of GD register stages, so the residual blocks continue the pipeline
    // without a bubble (64 x 64 tiles: the first entry has a stage of its own).
    struct Stage {
        uint4 x[WM], b[SPW];
        uint2 xt[A4G ? WM : 1];                          // A4 from memory: the operand's tail dwords
        uint4 xh[A8 ? WM : 1][2];                        // A8: the e4m3 high plane (32 bytes)
        // scales: four strips, one load (lane l: column row0 + l, handed out by
        // shuffles); fewer, one load per strip (column row0 + 16 s + lrow)
        uint16_t sc[kScaleShfl ? 1 : SPW];
        int g;
        bool res;
    };
    // A8: the low plane follows the M K bytes of the high plane; A4: the tail
    // plane follows the G M 64 bytes of the main plane
    const uint32_t lo_base = A8 ? (uint32_t)M * (uint32_t)K : 0u;
    const uint32_t tail0 = (uint32_t)G * (uint32_t)M * (uint32_t)kGroupBytes;
    // 64 x 64 tiles (four dense groups a wave at K = 4096, a two-stage ring):
    // the split's first residual entry goes through a stage of its own (Sr),
    // loaded in the prologue right after the ring's stages and multiplied
    // before the ring loop, so that a wave with one residual block beside its
    // dense groups needs no third round of the ring (K = N = 4096, M = 256:
    // 13.5 -> 13.0 us; decode and 32 x 64 tiles, whose rings already hold a
    // fifth item, measured slower with it).  The ring takes the dense groups
    // and the other entries: ring item j is group gb + j (j < ng) or entry
    // j - ng + R0.
    constexpr int R0 = (WM == 4 && WN == 4 && !A8) ? 1 : 0;
    static_assert(!(PT && R0), "decode tiles have no first-residual stage");
    const int nitems = PT ? nall : ng + (ne > R0 ? ne - R0 : 0);
    // groups of the first entry and of the ring's next entry (scalar; the
    // latter loaded one entry ahead)
    const int kb_first = (R0 && ne > 0) ? (int)res_kb[pb] : 0;
    int kb_next = (ne > R0) ? (int)res_kb[pb + R0] : 0;
    // activation rows from M on are read as zeros without touching memory
    // (decode tiles are mostly such rows)
    uint32_t xdead[WM];
#pragma unroll
    for (int i = 0; i < WM; ++i) xdead[i] = mw + 16 * i + lrow < M ? 0u : kPastEnd;
    // the loads of an item: group g, residual block p (res), of the tile at
    // columns n0 or (PT) tn[0]
    auto issue_item = [&](Stage& S, int g, bool res, int p, auto... tn) {
        S.g = g;
        S.res = res;
        if constexpr (!FQ && !XS) {
#pragma unroll
            for (int i = 0; i < WM; ++i) S.x[i] = bload16(rx, (lo_base + x_offset(g, i)) | xdead[i], 0);
        }
        if constexpr (A4G) {
#pragma unroll
            for (int i = 0; i < WM; ++i) {
                const uint32_t to = tail0 + ((uint32_t)g * (uint32_t)M + (uint32_t)(mw + 16 * i + lrow)) * 32u +
                                    (uint32_t)lq * 8u;
                const i32x2 v = __builtin_amdgcn_raw_buffer_load_b64(rx, to | xdead[i], 0, 0);
                S.xt[i] = make_uint2((uint32_t)v[0], (uint32_t)v[1]);
            }
        }
        if constexpr (A8) {
#pragma unroll
            for (int i = 0; i < WM; ++i) {
                const uint32_t ho = ((uint32_t)g * (uint32_t)M + (uint32_t)(mw + 16 * i + lrow)) * 128u + (uint32_t)lq * 32u;
                S.xh[i][0] = bload16(rx, ho | xdead[i], 0);
                S.xh[i][1] = bload16(rx, (ho + 16u) | xdead[i], 0);
            }
        }
        // resources built from the selected base (a select of scalars, not of
        // two descriptors, which the compiler would turn into branches)
        const bool use_r = res && a.Rq != nullptr;
        const __amdgpu_buffer_rsrc_t rb =
            make_rsrc(use_r ? (const void*)a.Rq : (const void*)a.Wq, use_r ? a.rq_bytes : a.wq_bytes);
        uint32_t row0;
        if constexpr (sizeof...(tn) > 0) {
            const int t0 = (tn, ...);
            row0 = (res ? (uint32_t)p * kGroup + (uint32_t)(t0 % kGroup) : (uint32_t)g * (uint32_t)N + (uint32_t)t0) +
                   (uint32_t)nw;
        } else {
            row0 = (res ? (uint32_t)p * kGroup + (uint32_t)roff : (uint32_t)g * (uint32_t)N + (uint32_t)n0) +
                   (uint32_t)nw;
        }
#pragma unroll
        for (int s = 0; s < SPW; ++s)
            S.b[s] = bload16(rb, (row0 + 16u * s) * kGroupBytes + loff, 0);
        if constexpr (!RAW) {
            const bool use_sr = res && a.s_r != nullptr;
            const __amdgpu_buffer_rsrc_t rs =
                make_rsrc(use_sr ? (const void*)a.s_r : (const void*)a.s_w, use_sr ? a.sr_bytes : a.sw_bytes);
            if constexpr (kScaleShfl) {
                S.sc[0] = __builtin_amdgcn_raw_buffer_load_b16(rs, (row0 + (uint32_t)lane) * 2u, 0, 0);
            } else {
#pragma unroll
                for (int s = 0; s < SPW; ++s)
                    S.sc[s] = __builtin_amdgcn_raw_buffer_load_b16(rs, (row0 + 16u * s + (uint32_t)lrow) * 2u,
                                                                   0, 0);
            }
        }
    };
    // (item j < nitems; no loads are issued past the last item)
    auto load_item = [&](Stage& S, int j) {
        const bool res = j >= ng;                        // uniform
        const int p = pb + (j - ng) + R0;
        int g = gb + j;
        if (res) {
            g = kb_next;
            if (j - ng + R0 + 1 < ne) kb_next = (int)res_kb[p + 1];
        }
        issue_item(S, g, res, p);
    };
    // PT: items are loaded in order, tile after tile; the cursor: tile lk
    // (columns ln0, entries lpb .. lpb + lne - 1), item lj of it
    int lk = 0, lj = 0, ln0 = n0, lpb = pb, lne = ne;
    auto load_next = [&](Stage& S) {
        if (lj == ng + lne) {
            ++lk;
            lj = 0;
            ln0 = __builtin_amdgcn_readlane(vn0, lk);
            lpb = __builtin_amdgcn_readlane(vpb, lk);
            lne = __builtin_amdgcn_readlane(vne, lk);
            kb_next = lne > 0 ? (int)res_kb[lpb] : 0;
        }
        const bool res = lj >= ng;                       // uniform
        const int p = lpb + (lj - ng);
        int g = gb + lj;
        if (res) {
            g = kb_next;
            if (lj - ng + 1 < lne) kb_next = (int)res_kb[p + 1];
        }
        issue_item(S, g, res, p, ln0);
        ++lj;
    };
    auto compute_item = [&](const Stage& S, auto res_c) {
        constexpr bool RES = decltype(res_c)::value;
        i32x8 av[WM], ah[A8 ? WM : 1];
#pragma unroll
        for (int i = 0; i < WM; ++i) {
            if constexpr (XS) av[i] = x_staged(S.g, i);
            else if constexpr (A4) av[i] = act_operand(S.x[i], S.xt[i]);
            else av[i] = unfold_codes(FQ ? x_lds(S.g, i) : S.x[i]);
        }
        if constexpr (A8) {
#pragma unroll
            for (int i = 0; i < WM; ++i)
                ah[i] = i32x8{(int)S.xh[i][0].x, (int)S.xh[i][0].y, (int)S.xh[i][0].z, (int)S.xh[i][0].w,
                              (int)S.xh[i][1].x, (int)S.xh[i][1].y, (int)S.xh[i][1].z, (int)S.xh[i][1].w};
        }
#pragma unroll
        for (int s = 0; s < SPW; ++s) {
            const i32x8 bv = unfold_codes(S.b[s]);
            // column 16 s + lrow's scale (x 64: at the end)
            uint16_t sb = 0;
            if constexpr (!RAW) sb = kScaleShfl ? (uint16_t)__shfl((int)S.sc[0], 16 * s + lrow, 64) : S.sc[s];
            const float sc = RAW ? 0.f : half_bits_to_float(sb);
#pragma unroll
            for (int i = 0; i < WM; ++i) {
                f32x4 t = mfma_codes(av[i], bv, f32x4{0.f, 0.f, 0.f, 0.f});
                if constexpr (A8) t = mfma_e4m3_codes(ah[i], bv, t);   // + the high plane: exact
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    if constexpr (!RAW) acc[i][s][r] = __builtin_fmaf(sc, t[r], acc[i][s][r]);
                    else if constexpr (RES) racc[i][s][r] += (int)(t[r] * kCodeScale);
                    else iacc[i][s][r] += (int)(t[r] * kCodeScale);   // exact integer
                }
            }
        }
        pin_all();
    };

    // FQ, part 1: this thread's chunks of X, loaded first so that they are
    // the first loads to land
    const int nxc = K / 16;
    uint4 xv[FQ ? kFusedCPT : 1][2];
    auto row_of = [&](int idx) { return (idx >= nxc) + (idx >= 2 * nxc) + (idx >= 3 * nxc); };
    if constexpr (FQ) {
        if (threadIdx.x < kFusedMaxM) amax_sh[threadIdx.x] = 0u;
#pragma unroll
        for (int i = 0; i < kFusedCPT; ++i) {
            const int idx = (int)threadIdx.x + i * 64 * NW;
            xv[i][0] = xv[i][1] = make_uint4(0, 0, 0, 0);
            if (idx < M * nxc) {
                const int m = row_of(idx), c = idx - m * nxc;
                const uint16_t* src = a.X + (int64_t)m * a.ldx + 16 * c;
                xv[i][0] = ldg16(reinterpret_cast<const uint8_t*>(src));
                xv[i][1] = ldg16(reinterpret_cast<const uint8_t*>(src + 8));
            }
        }
    }

    // XS, part 1: this thread's 16-byte chunks of Xq (up to kStageCPT),
    // loaded ahead of the ring
    constexpr int kStageCPT = 8;
    const int nxs = (int)(a.xq_bytes / 16u);
    uint4 xsv[XS ? kStageCPT : 1];
    if constexpr (XS) {
#pragma unroll
        for (int k = 0; k < kStageCPT; ++k) {
            const int idx = (int)threadIdx.x + k * 64 * NW;
            xsv[k] = bload16(rx, idx < nxs ? (uint32_t)idx * 16u : kPastEnd, 0);
        }
    }

    // (the scheduling barriers keep each stage's loads together and the
    // stages in ring order, so the wait for a stage counts exactly the
    // stages issued after it)
    Stage St[GD], Sr;                                   // Sr: used when R0 > 0
    static_for<GD>([&](auto dc) {
        constexpr int d = decltype(dc)::value;
        if (d < nitems) {
            if constexpr (PT) load_next(St[d]);
            else load_item(St[d], d);
        }
        __builtin_amdgcn_sched_barrier(0);
    });
    if constexpr (R0 > 0) {
        if (ne > 0) issue_item(Sr, kb_first, true, pb);
        __builtin_amdgcn_sched_barrier(0);
    }

    if constexpr (XS) {
        // XS, part 2: the chunks into LDS (main-plane chunks swizzled)
        const int nmain = G * M * 4;                       // main-plane chunks
#pragma unroll
        for (int k = 0; k < kStageCPT; ++k) {
            const int idx = (int)threadIdx.x + k * 64 * NW;
            if (idx < nxs) {
                uint32_t dst = (uint32_t)idx * 16u;
                if (idx < nmain) {
                    const int q = idx & 3, gr = idx >> 2, g = gr / M, r = gr - g * M;
                    dst = xs_main(g, r, q);
                }
                *reinterpret_cast<uint4*>(&xs[dst]) = xsv[k];
            }
        }
        __syncthreads();
    }

    if constexpr (FQ) {
        // FQ, part 2: row maxima across the workgroup (LDS atomic max on the
        // sign-cleared fp16 bits), scales, codes into LDS
        __syncthreads();                                   // amax_sh cleared
#pragma unroll
        for (int i = 0; i < kFusedCPT; ++i) {
            const int idx = (int)threadIdx.x + i * 64 * NW;
            if (idx < M * nxc) {
                const uint32_t c0m = chunk_absmax_bits(xv[i][0]), c1m = chunk_absmax_bits(xv[i][1]);
                atomicMax(&amax_sh[row_of(idx)], c0m > c1m ? c0m : c1m);
            }
        }
        __syncthreads();
        float sc[kFusedMaxM];
#pragma unroll
        for (int r = 0; r < kFusedMaxM; ++r) {
            const uint16_t sb = scale_bits_from_amax(half_bits_to_float((uint16_t)amax_sh[r]));
            sc[r] = half_bits_to_float(sb);
            if (threadIdx.x == 0) sx_sh[r] = sb;
        }
#pragma unroll
        for (int i = 0; i < kFusedCPT; ++i) {
            const int idx = (int)threadIdx.x + i * 64 * NW;
            if (idx < M * nxc) {
                const int m = row_of(idx), c = idx - m * nxc;
                const float s = m == 0 ? sc[0] : m == 1 ? sc[1] : m == 2 ? sc[2] : sc[3];
                *reinterpret_cast<uint2*>(&xs[(int64_t)m * (K / 2) + 8 * c]) =
                    quant_chunk(xv[i][0], xv[i][1], s, 1.0f / s);
            }
        }
        __syncthreads();
    }

    if (R0 > 0 && ne > 0) {
        if (RAW) compute_item(Sr, std::true_type{});
        else compute_item(Sr, std::false_type{});
    }
    // cross-wave reduction of the tile at columns tn0, splits added in split
    // order (deterministic), and its outputs
    constexpr int kRounds = RAW ? 2 : 1;
    auto reduce_store = [&](int tn0) {
#pragma unroll
        for (int round = 0; round < kRounds; ++round) {
            if (round > 0) __syncthreads();                     // the previous round is read
#pragma unroll
            for (int i = 0; i < WM; ++i)
#pragma unroll
                for (int s = 0; s < SPW; ++s)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int v = (i * SPW + s) * 4 + r;
                        uint32_t x;
                        if constexpr (RAW) x = (uint32_t)(round == 0 ? iacc[i][s][r] : racc[i][s][r]);
                        else x = __float_as_uint(acc[i][s][r]);
                        red[wave][v][lane] = x;
                    }
            __syncthreads();
            for (int e = threadIdx.x; e < WG2 * kAcc * 64; e += 64 * NW) {
                const int wp = e / (kAcc * 64), v = (e / 64) % kAcc, l = e % 64;
                const int is = v / 4, r = v % 4;
                const int i = is / SPW, s = is % SPW;
                const int m = m0 + 16 * (WM * (wp / WGN) + i) + 4 * (l >> 4) + r;
                const int n = tn0 + 16 * (WN * (wp % WGN) + s) + (l & 15);
                if (m >= M) continue;
                if constexpr (RAW) {
                    int32_t t = 0;
                    for (int k = 0; k < KS; ++k) t += (int32_t)red[k * WG2 + wp][v][l];
                    (round == 0 ? a.Tb : a.Tr)[(int64_t)m * N + n] = t;
                } else {
                    float sum = 0.f;
                    for (int k = 0; k < KS; ++k) sum += __uint_as_float(red[k * WG2 + wp][v][l]);
                    const uint16_t sxb = FQ ? sx_sh[m] : a.s_x[m];
                    a.Y[(int64_t)m * a.ldy + n] = float_to_half_bits(half_bits_to_float(sxb) * kCodeScale * sum);
                }
            }
        }
    };
    auto zero_acc = [&]() {
#pragma unroll
        for (int i = 0; i < WM; ++i)
#pragma unroll
            for (int s = 0; s < SPW; ++s) {
                acc[i][s] = f32x4{0.f, 0.f, 0.f, 0.f};
                iacc[i][s] = i32x4{0, 0, 0, 0};
                racc[i][s] = i32x4{0, 0, 0, 0};
            }
    };

    // PT: the tile being multiplied (ordinal ck, columns cn0) and its items
    // still to come (every wave has at least one item in each tile, so a tile
    // is complete when the next tile's first item comes up, and every wave
    // meets the same barriers)
    int ck = 0, cn0 = n0, cleft = ng + ne;
    for (int j0 = 0; j0 < nitems; j0 += GD) {
        static_for<GD>([&](auto dc) {
            constexpr int d = decltype(dc)::value;
            const int j = j0 + d;
            if (j < nitems) {
                if constexpr (PT) {
                    if (cleft == 0) {
                        reduce_store(cn0);
                        __syncthreads();                    // its partial sums are read
                        zero_acc();
                        ++ck;
                        cn0 = __builtin_amdgcn_readlane(vn0, ck);
                        cleft = ng + __builtin_amdgcn_readlane(vne, ck);
                    }
                    --cleft;
                }
                if (RAW && St[d].res) compute_item(St[d], std::true_type{});
                else compute_item(St[d], std::false_type{});
            }
            __builtin_amdgcn_sched_barrier(0);
            if (j + GD < nitems) {
                if constexpr (PT) load_next(St[d]);
                else load_item(St[d], j + GD);
            }
            __builtin_amdgcn_sched_barrier(0);
        });
    }
    reduce_store(cn0);
}

// --------------------------------------------------------------------------
// Host dispatch
// --------------------------------------------------------------------------
constexpr int kSkinnyMaxM = 32;
constexpr int kSkinnyAutoM = 32;   // AUTO picks the skinny kernel up to this M

// Strips per decode tile: two when that still gives every CU a workgroup (a
// tile's adjacent strips share DRAM pages and the block row's CSR entries),
// else one.  (Four measured no faster than two on the 5120 -> 25600 layer at
// one token, slightly slower.)
constexpr int kCUs = 256;
static int decode_spw(int N) {
    const int S = N / 16;
    if (S / 2 >= kCUs) return 2;
    return 1;
}
// at one row: two strips only while their tiles still fit in one round of
// two workgroups a CU (4096 -> 14336: 11.0 -> 9.6 us); on wider layers one
// strip, so that the workgroups that take several tiles stay balanced
// (8192 -> 28672: 28.5 -> 27.3 us)
static int decode_spw_one_row(int N) {
    return N / 32 <= 2 * kCUs ? decode_spw(N) : 1;
}

// Decode grids (fused quantisation or staged activations): one workgroup per
// tile while the tiles fit in one round of resident workgroups, else a
// round's worth (a multiple of eight, so a workgroup's tiles stay on its XCD)
// of PT workgroups, each quantising or staging the rows once and taking its
// tiles in turn with the next tile's loads in flight while it finishes the
// current one (fused quantisation, four rows, 8192 -> 28672: 38.7 -> 30.6 us,
// 5120 -> 25600: 26.3 -> 21.7 us; staged activations, 5120 -> 25600 at one
// and 16 rows: 18.55 -> 18.25 and 20.2 -> 19.6 us).  Every wave needs a group
// of each tile (K >= 8 x 128) and a workgroup at most 64 tiles (one a lane);
// 0: one workgroup per tile.
// Resident workgroups per CU of a decode kernel with this much dynamic LDS
// (the runtime's occupancy query, remembered per kernel and LDS size).
static int decode_occupancy(const void* kernel, size_t lds_bytes) {
    struct Entry {
        const void* kernel;
        size_t lds;
        int occ;
    };
    static std::mutex mutex;
    static Entry cache[64];
    static int used = 0;
    std::lock_guard<std::mutex> lock(mutex);
    for (int i = 0; i < used; ++i)
        if (cache[i].kernel == kernel && cache[i].lds == lds_bytes) return cache[i].occ;
    int occ = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kernel, 64 * kDecodeWaves, lds_bytes) != hipSuccess) {
        (void)hipGetLastError();    // a failed query must not surface as the launch's error
        return 1;
    }
    if (occ < 1) occ = 1;
    if (used < 64) cache[used++] = Entry{kernel, lds_bytes, occ};
    return occ;
}

static unsigned decode_grid(const void* kernel, size_t lds_bytes, int K, int64_t tiles) {
    if (tiles <= kCUs || K / kGroup < kDecodeWaves) return 0;     // one round whatever the occupancy
    const int64_t slots = (int64_t)decode_occupancy(kernel, lds_bytes) * kCUs;
    if (tiles <= slots) return 0;
    const int64_t per = (tiles + slots - 1) / slots;
    if (per > 64) return (unsigned)(((tiles + 63) / 64 + 7) / 8 * 8);
    return (unsigned)slots;
}

template <int WM, int WN, int WGM, int WGN, bool RAW, bool FQ, bool A8 = false, bool XS = false>
static void launch_stream(const GemmArgs& a, size_t xs_bytes, hipStream_t stream) {
    const int64_t tiles = (int64_t)((a.M + 16 * WM * WGM - 1) / (16 * WM * WGM)) * (a.N / (16 * WN * WGN));
    if constexpr (FQ || XS) {
        const auto pt = gemm_stream_kernel<WM, WN, WGM, WGN, RAW, FQ, A8, XS, true>;
        const unsigned grid = decode_grid(reinterpret_cast<const void*>(pt), xs_bytes, a.K, tiles);
        if (grid > 0) {
            hipLaunchKernelGGL(pt, dim3(grid), dim3(64 * kDecodeWaves), xs_bytes, stream, a);
            return;
        }
    }
    hipLaunchKernelGGL((gemm_stream_kernel<WM, WN, WGM, WGN, RAW, FQ, A8, XS>), dim3((unsigned)tiles),
                       dim3(64 * kDecodeWaves), xs_bytes, stream, a);
}

// The W4A4 medium tiles (64 x 64 when they give every CU one, else 32 x 64)
// are compiled in a translation unit of their own (medium_gemm.hip, which
// includes this file with MQ_MEDIUM_TU defined and nothing else of the
// library), built with the compiler's maximum-ILP scheduling strategy: the
// default one measured 5 % slower there (K = N = 4096, M = 256: 13.2 against
// 12.5 us), and that strategy measured slower on the tiled and decode kernels.
template <bool RAW>
void launch_medium_tiles(const GemmArgs& a, bool tile64, hipStream_t stream);
#ifdef MQ_MEDIUM_TU
template <bool RAW>
void launch_medium_tiles(const GemmArgs& a, bool tile64, hipStream_t stream) {
    if (tile64) launch_stream<4, 4, 1, 1, RAW, false>(a, 0, stream);
    else launch_stream<2, 4, 1, 1, RAW, false>(a, 0, stream);
}
template void launch_medium_tiles<false>(const GemmArgs&, bool, hipStream_t);
template void launch_medium_tiles<true>(const GemmArgs&, bool, hipStream_t);
}  // namespace mq
#else

// Decode: the activation rows are copied into LDS once per workgroup when
// they fit beside the partial-sum exchange (two workgroups a CU: 80 KB each;
// at most 8 chunks of 16 bytes a thread), so the items load only weights.
constexpr size_t kDecodeLdsBytes = 80 * 1024, kStageMaxBytes = 64 * 1024;
static size_t staged_act_bytes(const GemmArgs& a, int wm, int spw) {
    const size_t xb = (size_t)a.xq_bytes;
    const size_t red = (size_t)kDecodeWaves * wm * spw * 4 * 64 * 4;
    return (xb <= kStageMaxBytes && xb + red <= kDecodeLdsBytes) ? xb : 0;
}

template <int WM, int SPW, bool RAW, bool FQ>
static void launch_decode_spw(const GemmArgs& a, size_t xs_bytes, hipStream_t stream) {
    if constexpr (!FQ) {
        const size_t xb = staged_act_bytes(a, WM, SPW);
        if (xb > 0) return launch_stream<WM, SPW, 1, 1, RAW, false, false, true>(a, xb, stream);
    }
    launch_stream<WM, SPW, 1, 1, RAW, FQ>(a, xs_bytes, stream);
}

// xs_bytes: LDS for the quantised rows (fused quantisation), 0 otherwise
template <int WM, bool RAW, bool FQ>
static void launch_decode(const GemmArgs& a, int spw, size_t xs_bytes, hipStream_t stream) {
    if (spw >= 2) return launch_decode_spw<WM, 2, RAW, FQ>(a, xs_bytes, stream);
    launch_decode_spw<WM, 1, RAW, FQ>(a, xs_bytes, stream);
}

// 256 x 256 or 128 x 128 tiles, by the estimated number of rounds: the large
// tile runs one workgroup per CU, the 128 x 128 tile two, and a round of the
// latter measured about 0.66 of a round of the former (for a quarter of the
// work: 4096 -> 14336, 14336 -> 4096 and 4096 -> 24576 at M = 4096 / 8192).
// So the large tile wins whenever the small tiles would need more than one
// round (even when the large ones leave CUs idle: 5120 -> 5120 and
// 25600 -> 5120 at M = 2048, 160 tiles, were 9 and 11 % faster than 640 small
// tiles), and the small tile (with split-K when they are few) takes grids
// that fit in one round.
// (68 rather than the 66 measured: where two rounds of large tiles meet
// three of small ones, a near tie at 66, the large tiles measured faster on
// 5120 -> 25600 at M = 768, 117 against 127 us, 4096 -> 14336 at M = 1536,
// 102.5 against 107.6, 14336 -> 4096 at M = 6144 and 5120 -> 5120 at
// M = 4096, and slower only on K = N = 4096 at M = 5120, 100.5 against 94.7.)
constexpr int kLargeRoundPct = 100, kSmallRoundPct = 68;
static bool large_tiles_fit(int M, int N) {
    if (N % 256 != 0) return false;
    const int64_t tl = (int64_t)((M + 255) / 256) * (N / 256);
    const int64_t ts = (int64_t)((M + 127) / 128) * (N / 128);
    const int64_t rl = (tl + kCUs - 1) / kCUs, rs = (ts + 2 * kCUs - 1) / (2 * kCUs);
    return kLargeRoundPct * rl < kSmallRoundPct * rs;
}

// Buffer resource words (as buf_desc), built on the host.
static i32x4 host_buf_desc(const void* base, uint32_t bytes) {
    const uint64_t b = reinterpret_cast<uint64_t>(base);
    return i32x4{(int)(uint32_t)b, (int)((uint32_t)(b >> 32) & 0xFFFFu), (int)bytes, 0x00020000};
}

// AUTO takes the medium (streaming) kernel where the 128 x 128 tiles would
// be too few to give every CU two workgroups (the tiled kernel would split K
// and add the partial sums in a second launch), as long as its 64 x 64 tiles
// fit on the CUs in one round (one workgroup per CU: its partial-sum exchange
// takes most of the LDS), or in a few rounds at short K: four up to K = 4096,
// three and a half up to 8192 (5120 -> 25600 at M = 128, 3.1 rounds: 46.1 us
// against 56.2 split).  There the split and its reduction cost more than the
// extra rounds (K = N = 4096: M = 512 27.4 -> 20.3 us, M = 768 38.0 -> 29.0 us;
// 5120 -> 1024 at M = 2048 28.4 -> 22.7 us; 5120 -> 5120 at M = 512 41.6 ->
// 35.5 us), but not beyond (K = N = 4096 at M = 1280, five rounds: 38.6 us
// tiled against 44.9; 5120 -> 5120 at M = 768, four rounds, 46.0 against
// 47.5), and deeper K amortises them (14336 -> 4096 at M = 1024: 78 us split
// against 96 us medium).
constexpr int kMediumTargetWGs = 512;
static bool medium_preferred(int M, int N, int K) {
    const int64_t t128 = (int64_t)((M + kTB - 1) / kTB) * (N / kTB), t64 = (int64_t)((M + 63) / 64) * (N / 64);
    // (in half rounds)
    const int64_t half_rounds = K <= 4096 ? 8 : K <= 8192 ? 7 : 2;
    return t128 < kMediumTargetWGs && 2 * t64 <= half_rounds * kCUs;
}

// Byte sizes of the operands and buffer resources spanning each of them.
// Whole-operand resources take 32-bit offsets (and offsets from 2 GB up serve
// as "past the end"), so every operand must stay below 2 GB.
template <bool RAW>
static mq_status operand_resources(GemmArgs& a, bool a8 = false) {
    const uint64_t G = (uint64_t)(a.K / kGroup);
    const uint64_t sizes[5] = {G * a.M * (a8 ? 3 * kGroupBytes : kActGroupBytes), G * a.N * kGroupBytes,
                               (uint64_t)a.nnzb * kTB * kGroupBytes,
                               G * a.N * 2, (uint64_t)a.nnzb * kTB * 2};
    for (uint64_t b : sizes)
        if (b >= (1ull << 31)) return MQ_ERR_UNSUPPORTED_SHAPE;
    a.xq_bytes = (uint32_t)sizes[0];
    a.wq_bytes = (uint32_t)sizes[1];
    a.rq_bytes = (uint32_t)sizes[2];
    a.sw_bytes = RAW ? 0u : (uint32_t)sizes[3];
    a.sr_bytes = RAW ? 0u : (uint32_t)sizes[4];
    // a resource over an absent operand has a valid base and no bytes
    auto desc = [&](const void* p, uint32_t bytes) {
        return host_buf_desc(p ? p : (const void*)a.Wq, p ? bytes : 0u);
    };
    a.rx = desc(a.Xq, a.xq_bytes);
    a.rw = desc(a.Wq, a.wq_bytes);
    a.rr = desc(a.Rq, a.rq_bytes);
    a.rsw = desc(a.s_w, a.sw_bytes);
    a.rsr = desc(a.s_r, a.sr_bytes);
    return MQ_OK;
}

// The kernel family a launch takes: AUTO by shape, and the explicit choices
// that do not apply to the shape mapped to the tiled kernel.
static mq_variant resolve_variant(mq_variant variant, int M, int N, int K) {
    if (variant == MQ_VARIANT_AUTO)
        variant = M <= kSkinnyAutoM ? MQ_VARIANT_SKINNY
                  : large_tiles_fit(M, N) ? MQ_VARIANT_TILED_LARGE
                  : medium_preferred(M, N, K) ? MQ_VARIANT_MEDIUM : MQ_VARIANT_TILED;
    if (variant == MQ_VARIANT_SKINNY && M > kSkinnyMaxM) variant = MQ_VARIANT_TILED;
    if (variant == MQ_VARIANT_TILED_LARGE && N % 256 != 0) variant = MQ_VARIANT_TILED;
    return variant;
}

template <bool RAW>
static mq_status launch(mq_variant variant, const GemmArgs& args, void* workspace, size_t ws_bytes,
                        hipStream_t stream) {
    GemmArgs a = args;
    const mq_status rs = operand_resources<RAW>(a);
    if (rs != MQ_OK) return rs;
    a.y16 = (!RAW && a.Y && mq_host::aligned(a.Y, 16)) ? 1 : 0;
    variant = resolve_variant(variant, a.M, a.N, a.K);
    if (variant == MQ_VARIANT_MEDIUM) {
        // one workgroup per CU (its ring takes most of the LDS): 64-row tiles
        // when they alone give every CU one, else 32-row ones
        const int64_t t64 = (int64_t)((a.M + 63) / 64) * (a.N / 64);
        const int64_t t32 = (int64_t)((a.M + 31) / 32) * (a.N / 64);
        if (t32 > 0x7fffffff) return MQ_ERR_UNSUPPORTED_SHAPE;
        launch_medium_tiles<RAW>(a, t64 >= kCUs, stream);
    } else if (variant == MQ_VARIANT_TILED_LARGE) {
        using TS = TileShape<8, 4>;
        const int64_t tiles = (int64_t)((a.M + TS::kTM - 1) / TS::kTM) * (a.N / TS::kTN);
        if (tiles > 0x7fffffff) return MQ_ERR_UNSUPPORTED_SHAPE;
        a.rank_rows = tiles <= (int64_t)kCUs * TS::kPerCU;
        hipLaunchKernelGGL((gemm_tiled_kernel<8, 4, RAW, false>), dim3((unsigned)tiles), dim3(TS::kThreads), 0,
                           stream, a, 0, (float*)nullptr);
    } else if (variant == MQ_VARIANT_SKINNY) {
        if (a.M <= 16) launch_decode<1, RAW, false>(a, a.M == 1 ? decode_spw_one_row(a.N) : decode_spw(a.N), 0, stream);
        else launch_decode<2, RAW, false>(a, decode_spw(a.N), 0, stream);
    } else {
        const int64_t tiles = (int64_t)((a.M + kTB - 1) / kTB) * (a.N / kTB);
        if (tiles > 0x7fffffff) return MQ_ERR_UNSUPPORTED_SHAPE;
        const int splits = tiled_splits(a.M, a.N, a.K);
        a.rank_rows = tiles * splits <= (int64_t)kCUs * TileShape<4, 2>::kPerCU;
        if (splits == 1) {
            hipLaunchKernelGGL((gemm_tiled_kernel<4, 2, RAW, false>), dim3((unsigned)tiles),
                               dim3(TileShape<4, 2>::kThreads), 0, stream, a, 0, (float*)nullptr);
        } else if constexpr (RAW) {
            // raw sums: every split adds its exact integer partial sums into Tb, Tr
            const int64_t total = (int64_t)a.M * a.N;
            hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, stream,
                               a.Tb, total);
            hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, stream,
                               a.Tr, total);
            const int G = a.K / kGroup;
            const int gps = (G + splits - 1) / splits;
            hipLaunchKernelGGL((gemm_tiled_kernel<4, 2, RAW, true>), dim3((unsigned)tiles, splits),
                               dim3(TileShape<4, 2>::kThreads), 0, stream, a, gps, (float*)nullptr);
        } else {
            if (!workspace || ws_bytes < (size_t)splits * a.M * a.N * sizeof(float)) return MQ_ERR_WORKSPACE;
            const int G = a.K / kGroup;
            const int gps = (G + splits - 1) / splits;
            float* part = static_cast<float*>(workspace);
            hipLaunchKernelGGL((gemm_tiled_kernel<4, 2, RAW, true>), dim3((unsigned)tiles, splits),
                               dim3(TileShape<4, 2>::kThreads), 0, stream, a, gps, part);
            mq_status st = mq_host::launch_status();
            if (st != MQ_OK) return st;
            const int64_t total = (int64_t)a.M * a.N;
            hipLaunchKernelGGL(reduce_splits_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, stream,
                               part, splits, a.M, a.N, a.s_x, a.Y, a.ldy);
        }
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
    if (M <= 0 || !mq_host::shape_ok(N, K)) return 0;
    const int splits = tiled_splits(M, N, K);
    return splits > 1 ? (size_t)splits * M * N * sizeof(float) : 0;
}

extern "C" mq_status mq_fused_gemm_plan(int M, int N, int K, int* variant, int* splits) {
    if (!variant || !splits || M < 1 || M > (1 << 24)) return MQ_ERR_INVALID_ARG;
    if (!mq_host::shape_ok(N, K)) return MQ_ERR_UNSUPPORTED_SHAPE;
    const mq_variant v = resolve_variant(MQ_VARIANT_AUTO, M, N, K);
    *variant = (int)v;
    *splits = v == MQ_VARIANT_TILED ? tiled_splits(M, N, K) : 1;
    return MQ_OK;
}

extern "C" mq_status mq_fused_gemm_variant(mq_variant variant, int M, int N, int K,
                                           const uint8_t* Xq, const void* s_x,
                                           const uint8_t* Wq, const void* s_w,
                                           const int32_t* res_rowptr, const int32_t* res_kb, int nnzb,
                                           const uint8_t* Rq, const void* s_r,
                                           void* Y, int ldy,
                                           void* workspace, size_t ws_bytes, hipStream_t stream) {
    (void)workspace;
    if (variant < MQ_VARIANT_AUTO || variant > MQ_VARIANT_MEDIUM) return MQ_ERR_INVALID_ARG;
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
    a.nnzb = nnzb;
    return launch<false>(variant, a, workspace, ws_bytes, stream);
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
    if (variant < MQ_VARIANT_AUTO || variant > MQ_VARIANT_MEDIUM) return MQ_ERR_INVALID_ARG;
    mq_status st = check_common(M, N, K, Xq, Wq, res_rowptr, res_kb, nnzb, Rq);
    if (st != MQ_OK) return st;
    if (M == 0) return MQ_OK;
    if (!Tb || !Tr) return MQ_ERR_INVALID_ARG;
    if (!mq_host::aligned(Tb, 4) || !mq_host::aligned(Tr, 4)) return MQ_ERR_MISALIGNED;
    GemmArgs a{M, N, K, Xq, nullptr, Wq, nullptr, nnzb > 0 ? res_rowptr : nullptr, res_kb, Rq,
               nullptr, nullptr, 0, Tb, Tr};
    a.nnzb = nnzb;
    return launch<true>(variant, a, nullptr, 0, stream);
}

// ---------------------------------------------------------------------------
// W4A8 (per-token INT8 activations): the streaming kernels for every M --
// decode tiles up to 32 rows, 64 x 64 tiles (32 x 64 when those are fewer
// than the CUs) above.
// ---------------------------------------------------------------------------
template <bool RAW>
static mq_status launch_a8(GemmArgs a, hipStream_t stream) {
    const mq_status rs = operand_resources<RAW>(a, true);
    if (rs != MQ_OK) return rs;
    if (a.M <= 16) {
        const int spw = decode_spw(a.N);
        if (spw == 2) launch_stream<1, 2, 1, 1, RAW, false, true>(a, 0, stream);
        else launch_stream<1, 1, 1, 1, RAW, false, true>(a, 0, stream);
    } else if (a.M <= 32) {
        if (decode_spw(a.N) >= 2) launch_stream<2, 2, 1, 1, RAW, false, true>(a, 0, stream);
        else launch_stream<2, 1, 1, 1, RAW, false, true>(a, 0, stream);
    } else {
        const int64_t t64 = (int64_t)((a.M + 63) / 64) * (a.N / 64);
        const int64_t t32 = (int64_t)((a.M + 31) / 32) * (a.N / 64);
        if (t32 > 0x7fffffff) return MQ_ERR_UNSUPPORTED_SHAPE;
        if (t64 >= kCUs) launch_stream<4, 4, 1, 1, RAW, false, true>(a, 0, stream);
        else launch_stream<2, 4, 1, 1, RAW, false, true>(a, 0, stream);
    }
    return mq_host::launch_status();
}

extern "C" mq_status mq_fused_gemm_a8(int M, int N, int K,
                                      const uint8_t* Xq8, const void* s_x,
                                      const uint8_t* Wq, const void* s_w,
                                      const int32_t* res_rowptr, const int32_t* res_kb, int nnzb,
                                      const uint8_t* Rq, const void* s_r,
                                      void* Y, int ldy, hipStream_t stream) {
    mq_status st = check_common(M, N, K, Xq8, Wq, res_rowptr, res_kb, nnzb, Rq);
    if (st != MQ_OK) return st;
    if (ldy < N || ldy % 8 != 0) return MQ_ERR_UNSUPPORTED_SHAPE;
    if (M == 0) return MQ_OK;
    if (!s_x || !s_w || !Y || (nnzb > 0 && !s_r)) return MQ_ERR_INVALID_ARG;
    if (!mq_host::aligned(s_x, 2) || !mq_host::aligned(s_w, 2) || !mq_host::aligned(Y, 2) ||
        (s_r && !mq_host::aligned(s_r, 2)))
        return MQ_ERR_MISALIGNED;
    GemmArgs a{M, N, K, Xq8, static_cast<const uint16_t*>(s_x), Wq, static_cast<const uint16_t*>(s_w),
               nnzb > 0 ? res_rowptr : nullptr, res_kb, Rq, static_cast<const uint16_t*>(s_r),
               static_cast<uint16_t*>(Y), ldy, nullptr, nullptr};
    a.nnzb = nnzb;
    return launch_a8<false>(a, stream);
}

extern "C" mq_status mq_fused_gemm_a8_acc_i32(int M, int N, int K,
                                              const uint8_t* Xq8,
                                              const uint8_t* Wq,
                                              const int32_t* res_rowptr, const int32_t* res_kb, int nnzb,
                                              const uint8_t* Rq,
                                              int32_t* Tb, int32_t* Tr, hipStream_t stream) {
    mq_status st = check_common(M, N, K, Xq8, Wq, res_rowptr, res_kb, nnzb, Rq);
    if (st != MQ_OK) return st;
    if (M == 0) return MQ_OK;
    if (!Tb || !Tr) return MQ_ERR_INVALID_ARG;
    if (!mq_host::aligned(Tb, 4) || !mq_host::aligned(Tr, 4)) return MQ_ERR_MISALIGNED;
    GemmArgs a{M, N, K, Xq8, nullptr, Wq, nullptr, nnzb > 0 ? res_rowptr : nullptr, res_kb, Rq,
               nullptr, nullptr, 0, Tb, Tr};
    a.nnzb = nnzb;
    return launch_a8<true>(a, stream);
}

// ---------------------------------------------------------------------------
// Whole layer from fp16 activations
// ---------------------------------------------------------------------------
static bool fused_decode_ok(int M, int K) {
    return M >= 1 && M <= kFusedMaxM && (int64_t)M * (K / 16) <= (int64_t)kFusedCPT * 64 * 8 &&
           (int64_t)M * (K / 2) <= 64 * 1024;
}

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

extern "C" size_t mq_linear_workspace_size(int M, int N, int K) {
    if (M <= 0 || !mq_host::shape_ok(N, K) || fused_decode_ok(M, K)) return 0;
    return align256(mq_fused_gemm_workspace_size(M, N, K)) + align256((size_t)M * (K / 4) * 3) +
           align256((size_t)2 * M);
}

static mq_status linear_impl(int M, int N, int K, const void* X, int ldx,
                             const uint8_t* Wq, const void* s_w,
                             const int32_t* res_rowptr, const int32_t* res_kb, int nnzb,
                             const uint8_t* Rq, const void* s_r,
                             void* Y, int ldy,
                             void* workspace, size_t ws_bytes, hipStream_t stream) {
    mq_status st = check_common(M, N, K, static_cast<const uint8_t*>(X), Wq, res_rowptr, res_kb, nnzb, Rq);
    if (st != MQ_OK) return st;
    if (ldx < K || ldx % 8 != 0 || ldy < N || ldy % 8 != 0) return MQ_ERR_UNSUPPORTED_SHAPE;
    const size_t need = mq_linear_workspace_size(M, N, K);
    if (ws_bytes < need) return MQ_ERR_WORKSPACE;
    if (M == 0) return MQ_OK;
    if (!s_w || !Y || (nnzb > 0 && !s_r) || (need > 0 && !workspace)) return MQ_ERR_INVALID_ARG;
    if (!mq_host::aligned(s_w, 2) || !mq_host::aligned(Y, 2) || (s_r && !mq_host::aligned(s_r, 2)) ||
        (workspace && !mq_host::aligned(workspace, 16)))
        return MQ_ERR_MISALIGNED;
    if (fused_decode_ok(M, K)) {
        GemmArgs a{M, N, K, nullptr, nullptr, Wq, static_cast<const uint16_t*>(s_w),
                   nnzb > 0 ? res_rowptr : nullptr, res_kb, Rq, static_cast<const uint16_t*>(s_r),
                   static_cast<uint16_t*>(Y), ldy, nullptr, nullptr, static_cast<const uint16_t*>(X), ldx};
        a.nnzb = nnzb;
        st = operand_resources<false>(a);
        if (st != MQ_OK) return st;
        // (at four rows two strips measured faster than one on the wide
        // layers, where one row takes one: 5120 -> 25600 19.9 -> 19.1 us)
        launch_decode<1, false, true>(a, M == 1 ? decode_spw_one_row(N) : decode_spw(N), (size_t)M * (K / 2), stream);
        return mq_host::launch_status();
    }
    // quantise into the workspace, then the fused GEMM
    uint8_t* ws = static_cast<uint8_t*>(workspace);
    const size_t gws = mq_fused_gemm_workspace_size(M, N, K);
    uint8_t* Xq = ws + align256(gws);
    void* sx = Xq + align256((size_t)M * (K / 4) * 3);
    st = mq_quantize_act(X, M, K, ldx, Xq, sx, stream);
    if (st != MQ_OK) return st;
    return mq_fused_gemm(M, N, K, Xq, sx, Wq, s_w, res_rowptr, res_kb, nnzb, Rq, s_r, Y, ldy,
                         gws > 0 ? ws : nullptr, gws, stream);
}

extern "C" mq_status mq_linear(int M, int N, int K, const void* X, int ldx,
                               const uint8_t* Wq, const void* s_w,
                               const int32_t* res_rowptr, const int32_t* res_kb, int nnzb,
                               const uint8_t* Rq, const void* s_r,
                               void* Y, int ldy,
                               void* workspace, size_t ws_bytes, hipStream_t stream) {
    return linear_impl(M, N, K, X, ldx, Wq, s_w, res_rowptr, res_kb, nnzb, Rq, s_r, Y, ldy, workspace, ws_bytes,
                       stream);
}

// ---------------------------------------------------------------------------
// Scratch-free whole layer: mq_linear's workspace (the quantised rows, their
// scales and any split-K partial sums) in a file-scope device array instead
// of caller memory, for callers that cannot allocate.  Every GPU the library
// runs on holds its own copy until the process ends; calls on one GPU share
// it.  Nothing in it needs clearing: each call writes every byte it reads.
// ---------------------------------------------------------------------------
constexpr size_t kScratchBytes = (size_t)128 << 20;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mutex;
static void* g_scratch_ptr[kMaxDevices];

// this device's address of the scratch array (looked up once per device,
// with the device current); nullptr on failure
static void* device_scratch() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
        g_scratch_ptr[dev] = p;
    }
    return g_scratch_ptr[dev];
}

extern "C" size_t mq_scratch_bytes(void) { return kScratchBytes; }

extern "C" mq_status mq_linear_noalloc(int M, int N, int K, const void* X, int ldx,
                                       const uint8_t* Wq, const void* s_w,
                                       const int32_t* res_rowptr, const int32_t* res_kb, int nnzb,
                                       const uint8_t* Rq, const void* s_r,
                                       void* Y, int ldy, hipStream_t stream) {
    const size_t need = mq_linear_workspace_size(M, N, K);
    if (need > kScratchBytes) return MQ_ERR_SCRATCH_LIMIT;
    void* ws = nullptr;
    if (need > 0) {
        ws = device_scratch();
        if (!ws) return MQ_ERR_HIP;
    }
    return linear_impl(M, N, K, X, ldx, Wq, s_w, res_rowptr, res_kb, nnzb, Rq, s_r, Y, ldy, ws, need, stream);
}
#endif  // MQ_MEDIUM_TU
