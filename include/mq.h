/*
 * mq.h -- C ABI of libmq: MosaicQuant's fused W4A4 + sparse-residual linear
 * layer for AMD Instinct MI355X (gfx950).
 *
 * The layer (arXiv 2606.15652, Section 3 Eq. (4), Alg. 1 last step) is
 *
 *     Y = dequant(Xq Wq^T) + dequant(Xq (M_S (.) Rq)^T)
 *
 * with a dense 4-bit base weight Wq (one fp16 scale per output row per
 * 128-long group along K), a 4-bit residual Rq present only on a selected set
 * S of 128x128 weight blocks (one fp16 scale per row inside each block), and
 * per-token 4-bit activations Xq (one fp16 scale per row).  Both weight terms
 * are consumed by one kernel; residual MACs run inside the dense K-loop.
 *
 * Conventions shared by every call
 * --------------------------------
 * - Pointers are DEVICE pointers owned by the caller unless stated; the
 *   library keeps no pointer after a call returns and allocates nothing.
 * - Calls are asynchronous on `stream` (0 = the null stream).  On error
 *   nothing is launched and an mq_status < 0 is returned; no call throws.
 * - fp16 arrays are IEEE binary16 passed as `void*` / `const void*`.
 * - Shapes: K and N are multiples of 128 with 128 <= K <= 2^20 and
 *   128 <= N <= 2^24; 0 <= M <= 2^24 (M == 0 is a no-op).
 * - Packed 4-bit weight codes (Wq, Rq): codes q in [-7, 7], 4 bits each, a row
 *   of K codes taking K/2 bytes as K/16 chunks of 8 bytes; chunk c holds codes
 *   16c .. 16c+15.  Code e of a chunk is the 6-bit sign-magnitude field
 *   f_e = 32 [q < 0] + |q| at bit 6e of a 96-bit word O = (o0, o1, o2) of
 *   32-bit words; bits 6e+3 and 6e+4 of every field are zero.  The zero bits
 *   of o0 (ZA = 0x18618618) and of o1 (ZB = 0x86186186) together cover every
 *   bit o2 can use, and the chunk stores the little-endian words
 *       P0 = o0 | (o2 & ZA),   P1 = o1 | (o2 & ZB).
 *   Every byte pattern is a valid chunk (a sign bit with magnitude 0 is the
 *   code 0).  The layout lets the GEMM feed the codes, unchanged in value, to
 *   the fp6 (e2m3) matrix instruction of CDNA4 with four bit operations per
 *   chunk; the paper fixes no bit layout (Section 4.2 fuses layout packing
 *   with quantisation).
 * - Group order of packed weight rows (Wq [N rows]): a row's K/2 bytes are
 *   K/128 pieces of 64 bytes (one 128-code group each), stored group-major:
 *   piece (row n, group g) sits at byte (g N + n) 64.  Every 128-row x
 *   128-code tile is then one contiguous run of bytes, and the tiles of
 *   neighbouring row blocks are neighbours.
 * - Activation codes Xq [M rows] (codes in [-7, 7]) are stored in the
 *   operand form of the fp6 matrix instruction, so the GEMM reads them with
 *   no bit work: 3K/4 bytes a row.  For row r, group g (G = K/128 groups)
 *   and quarter j = 0..3 (codes k = 128 g + 32 j + e, e = 0..31), the fields
 *   f_e above, unfolded, form the 192-bit word F = sum_e f_e 2^(6e), six
 *   little-endian 32-bit words d0..d5:
 *       d0..d3 at byte (g M + r) 64 + 16 j               (main plane),
 *       d4, d5 at byte G M 64 + (g M + r) 32 + 8 j       (tail plane).
 *   The bits 6e+3, 6e+4 of every field must be zero (mq_quantize_act and
 *   mq_repack_act write them so); other patterns give unspecified outputs.
 * - Weight scales s_w are stored [K/128][N]: s_w of (row n, group g) at
 *   element g N + n.
 * - Code operand pointers (Xq, Wq, Rq) must be 16-byte aligned; fp16
 *   pointers 2-byte aligned; int32 pointers 4-byte aligned; fp32/fp64 arrays
 *   naturally aligned.  Violations return MQ_ERR_MISALIGNED.
 * - Canonical interchange layout (mq_repack_*, mq_unpack_*): one
 *   two's-complement 4-bit code per nibble, two per byte, the code of the
 *   even k in the low nibble, a row of K codes as K/2 bytes in k order; Wq
 *   [N][K/2], Xq [M][K/2], Rq [nnzb][128][64]; weight scales s_w [N][K/128].
 *   A caller holding codes in that layout converts them once with
 *   mq_repack_weights / mq_repack_act; every other call takes the library
 *   layout above.
 * - Inputs must be finite.  Outputs must not alias inputs.
 * - Thread safety: every call may be made concurrently from several host
 *   threads.  The only global state is the per-device address of the
 *   scratch array of mq_linear_noalloc, set once per device under a lock.
 */
#ifndef MQ_H
#define MQ_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum mq_status {
    MQ_OK = 0,
    MQ_ERR_INVALID_ARG = -1,       /* null pointer, negative size, bad budget  */
    MQ_ERR_UNSUPPORTED_SHAPE = -2, /* K or N not a positive multiple of 128,
                                      leading dimension too small / unaligned  */
    MQ_ERR_MISALIGNED = -3,        /* pointer alignment rule violated          */
    MQ_ERR_WORKSPACE = -4,         /* workspace smaller than required          */
    MQ_ERR_HIP = -5,               /* the HIP runtime reported a launch error  */
    MQ_ERR_SCRATCH_LIMIT = -6      /* a scratch-free call needs more scratch than
                                      the library holds (mq_scratch_bytes)      */
} mq_status;

/* Kernel family selection (testing and A/B timing).  AUTO picks by M. */
typedef enum mq_variant {
    MQ_VARIANT_AUTO = 0,
    MQ_VARIANT_SKINNY = 1,   /* decode: split-K over the waves of a workgroup  */
    MQ_VARIANT_TILED = 2,    /* prefill: 128 x 128 output tiles, K-loop of groups */
    MQ_VARIANT_TILED_LARGE = 3, /* prefill: 256 x 256 output tiles (N % 256 == 0,
                                   else as TILED); AUTO takes it when
                                   128 x 128 tiles would need more than one
                                   round of two per CU                       */
    MQ_VARIANT_MEDIUM = 4       /* 32 or 64 x 64 output tiles; AUTO takes it
                                   when 128 x 128 tiles would be too few to
                                   fill the chip and the 64 x 64 tiles fit in
                                   one round (or in five, up to K = 8192)    */
} mq_variant;

/* Static string naming a status code.  Never NULL. */
const char* mq_status_string(mq_status s);

/* Library ABI version (major * 100 + minor). */
int mq_version(void);

/* ======================================================================== */
/* Hot path                                                                  */
/* ======================================================================== */

/*
 * Per-token symmetric INT4 activation quantisation (Section 2, Eq. (1), one
 * scale per token; fused with code packing as in Section 4.2 "Kernel
 * Fusion"):
 *     a = max_k |X[m,k]|,  s_x[m] = fp16_rn(fp32(a) / 7),
 *     Xq[m,k] = clamp(round_half_even(X[m,k] / s_x[m]), -7, 7)  (0 if s == 0)
 *   X   : fp16 [M, ldx] row-major, ldx >= K, ldx % 8 == 0, 16-byte aligned.
 *   Xq  : out, uint8 [M, 3K/4] codes in the activation operand layout (above).
 *   s_x : out, fp16 [M].
 */
mq_status mq_quantize_act(const void* X, int M, int K, int ldx,
                          uint8_t* Xq, void* s_x, hipStream_t stream);

/* Bytes of workspace mq_fused_gemm needs for this shape (0: none). */
size_t mq_fused_gemm_workspace_size(int M, int N, int K);

/*
 * The kernel family mq_fused_gemm (AUTO) takes for an M x N x K layer, from
 * the shape alone (host logic; no device call, callable without a GPU):
 *   *variant : an mq_variant value (MQ_VARIANT_SKINNY, _TILED, _TILED_LARGE
 *              or _MEDIUM);
 *   *splits  : K splits of the 128 x 128 tiled kernel (whose partial sums go
 *              through the workspace), 1 for the other families.
 * MQ_ERR_INVALID_ARG for null outputs or M outside [1, 2^24],
 * MQ_ERR_UNSUPPORTED_SHAPE for N, K that mq_fused_gemm does not accept
 * (multiples of 128, K <= 2^20, N <= 2^24).
 */
mq_status mq_fused_gemm_plan(int M, int N, int K, int* variant, int* splits);

/*
 * Fused dense + sparse-residual W4A4 GEMM (Section 3 Eq. (4) with Eq. (2)'s
 * scale factorisation per group; Section 4.2 "Kernel Fusion" and
 * "Overlapped pipeline"):
 *     A_b[m,n,g] = sum_{k in g} Xq[m,k] Wq[n,k]
 *     A_r[m,n,g] = sum_{k in g} Xq[m,k] Rq[p][n%128][k%128]   if (n/128,g) in S
 *     Y[m,n] = fp16( s_x[m] * sum_g ( s_w[n,g] A_b + s_r[p][n%128] A_r ) )
 *   Xq, s_x          : uint8 [M, 3K/4] operand layout, fp16 [M] (from mq_quantize_act)
 *   Wq, s_w          : uint8 [N, K/2] group order, fp16 [K/128, N]
 *   res_rowptr       : int32 [N/128 + 1], CSR over 128-row block rows;
 *                      res_rowptr[0] == 0, res_rowptr[N/128] == nnzb.
 *   res_kb           : int32 [nnzb], block column (group) of each selected
 *                      block, strictly ascending within a block row.
 *   Rq, s_r          : uint8 [nnzb, 128, 64], fp16 [nnzb, 128]; block p holds
 *                      rows n = 128*nb + r, columns k = 128*res_kb[p] + c.
 *   nnzb == 0        : res_kb, Rq, s_r (and res_rowptr) may be NULL.
 *   Y, ldy           : out, fp16 [M, ldy], ldy >= N, ldy % 8 == 0.
 *   workspace        : >= mq_fused_gemm_workspace_size(M, N, K) bytes (may be
 *                      NULL when that is 0).
 * The CSR's contents are trusted (checked only by the test-suite): a kb
 * outside [0, K/128) or an unsorted row gives undefined results.
 */
mq_status mq_fused_gemm(int M, int N, int K,
                        const uint8_t* Xq, const void* s_x,
                        const uint8_t* Wq, const void* s_w,
                        const int32_t* res_rowptr, const int32_t* res_kb, int nnzb,
                        const uint8_t* Rq, const void* s_r,
                        void* Y, int ldy,
                        void* workspace, size_t ws_bytes, hipStream_t stream);

/* mq_fused_gemm with an explicit kernel family. */
mq_status mq_fused_gemm_variant(mq_variant variant, int M, int N, int K,
                                const uint8_t* Xq, const void* s_x,
                                const uint8_t* Wq, const void* s_w,
                                const int32_t* res_rowptr, const int32_t* res_kb, int nnzb,
                                const uint8_t* Rq, const void* s_r,
                                void* Y, int ldy,
                                void* workspace, size_t ws_bytes, hipStream_t stream);

/*
 * Same main loop (same kernel family, tiles and split-K ranges as the fp16
 * call), raw integer epilogue (for bit-exact testing):
 *     Tb[m,n] = sum_g A_b[m,n,g],   Tr[m,n] = sum_g A_r[m,n,g]
 *   Tb, Tr : out, int32 [M, N] row-major.  Exact: |Tb|, |Tr| <= 49 K < 2^31
 *            for every supported K.  Where the fp16 call splits K over
 *            workgroups, the splits' integer sums are added atomically into
 *            Tb, Tr (cleared first; integer addition is exact in any order).
 */
mq_status mq_fused_gemm_acc_i32(mq_variant variant, int M, int N, int K,
                                const uint8_t* Xq,
                                const uint8_t* Wq,
                                const int32_t* res_rowptr, const int32_t* res_kb, int nnzb,
                                const uint8_t* Rq,
                                int32_t* Tb, int32_t* Tr, hipStream_t stream);

/*
 * The whole layer from fp16 activations: mq_quantize_act followed by
 * mq_fused_gemm, with the same results bit for bit (Section 4.2 "Kernel
 * Fusion": quantisation fused into the GEMM).  For decode-sized inputs
 * (M <= 4, M * K <= 32768) one kernel does both: every workgroup quantises the
 * activation rows into LDS itself, which saves a launch.  Otherwise the
 * activations are quantised into the workspace first.
 *   X, ldx   : fp16 [M, ldx], ldx >= K, ldx % 8 == 0, 16-byte aligned.
 *   others   : as for mq_fused_gemm.
 *   workspace: >= mq_linear_workspace_size(M, N, K) bytes, 16-byte aligned
 *              (may be NULL when that is 0).
 */
size_t mq_linear_workspace_size(int M, int N, int K);
mq_status mq_linear(int M, int N, int K, const void* X, int ldx,
                    const uint8_t* Wq, const void* s_w,
                    const int32_t* res_rowptr, const int32_t* res_kb, int nnzb,
                    const uint8_t* Rq, const void* s_r,
                    void* Y, int ldy,
                    void* workspace, size_t ws_bytes, hipStream_t stream);

/* ======================================================================== */
/* W4A8 variant (per-token INT8 activations)                                 */
/* ======================================================================== */

/*
 * Per-token symmetric INT8 activation quantisation (the W4A8 setting of the
 * paper's appendix "Implementation Details": per-token dynamic activation
 * quantisation; Eq. (1) with q_max = 127):
 *     s_x[m] = fp16_rn(fp32(max_k |X[m,k]|) / 127),
 *     x = clamp(round_half_even(X[m,k] / s_x[m]), -127, 127)   (0 if s == 0)
 *   X   : fp16 [M, ldx], as for mq_quantize_act.
 *   Xq8 : out, uint8 [M * K * 3 / 2] in the library's A8 layout: each code as
 *         x = 8 h + l, h = floor(x / 8) in [-16, 15], l in [0, 7]; bytes
 *         [0, M K): the fp8 e4m3 byte of h, piece (row m, group g) of 128
 *         bytes at (g M + m) 128, its 16-code chunk c (codes 16c .. 16c+15 of
 *         the group, in k order) at byte 32 (c mod 4) + 16 (c div 4) of the
 *         piece (the operand order of the matrix instruction); [M K, 3 M K / 2):
 *         the codes l as 4-bit codes in the W4A4 layout (folded chunks,
 *         group order).  16-byte aligned.
 *   s_x : out, fp16 [M].
 */
mq_status mq_quantize_act8(const void* X, int M, int K, int ldx,
                           uint8_t* Xq8, void* s_x, hipStream_t stream);

/*
 * W4A8 layer: as mq_fused_gemm (same weights, residual blocks, epilogue of
 * Section 3 Eq. (4) and Eq. (2)) with INT8 activation codes Xq8 (layout of
 * mq_quantize_act8).  Exact integer group sums (|sum| <= 127 * 7 * 128).
 * Every M runs on the streaming kernels (no workspace).
 */
mq_status mq_fused_gemm_a8(int M, int N, int K,
                           const uint8_t* Xq8, const void* s_x,
                           const uint8_t* Wq, const void* s_w,
                           const int32_t* res_rowptr, const int32_t* res_kb, int nnzb,
                           const uint8_t* Rq, const void* s_r,
                           void* Y, int ldy, hipStream_t stream);

/* Raw integer sums of the W4A8 layer (testing): Tb, Tr int32 [M, N];
 * |Tb|, |Tr| <= 889 K < 2^31. */
mq_status mq_fused_gemm_a8_acc_i32(int M, int N, int K,
                                   const uint8_t* Xq8,
                                   const uint8_t* Wq,
                                   const int32_t* res_rowptr, const int32_t* res_kb, int nnzb,
                                   const uint8_t* Rq,
                                   int32_t* Tb, int32_t* Tr, hipStream_t stream);

/* INT8 codes: canonical int8 rows Xc [M, ldq] (ldq >= K, ldq % 16 == 0,
 * 16-byte aligned) <-> the A8 layout.  -128 (outside the method's range) is
 * stored as -127 and counted into the optional device counter n_invalid. */
mq_status mq_repack_act8(int M, int K, const int8_t* Xc, int ldq, uint8_t* Xq8,
                         int32_t* n_invalid, hipStream_t stream);
mq_status mq_unpack_act8(int M, int K, const uint8_t* Xq8, int8_t* Xc, int ldq,
                         hipStream_t stream);

/*
 * Comparison baseline: the unfused pipeline the fused kernel replaces
 * (Section 4.2 "Kernel Fusion", Fig. 3; Appendix "Kernel Profile"), three
 * launches on `stream`:
 *   1. the dense W4A4 GEMM (mq_fused_gemm with no residual blocks) -> fp16 Y;
 *   2. a block-sparse residual GEMM that reads Xq again from memory and
 *      writes fp32 partial sums P[m,n] = sum_g s_r[p][n%128] A_r[m,n,g] into
 *      the workspace (block rows with residual blocks only);
 *   3. a reduce-add Y[m,n] <- fp16(f32(Y[m,n]) + s_x[m] P[m,n]) on those
 *      block rows.
 * Same operands, layouts and checks as mq_fused_gemm; Y is rounded to fp16
 * twice on block rows with residual blocks (within the output bar).
 *   workspace : >= mq_unfused_workspace_size(M, N, K) bytes, 16-byte aligned
 *               (never NULL for M > 0).  N/128 <= 65535.
 */
size_t mq_unfused_workspace_size(int M, int N, int K);
mq_status mq_unfused_gemm(int M, int N, int K,
                          const uint8_t* Xq, const void* s_x,
                          const uint8_t* Wq, const void* s_w,
                          const int32_t* res_rowptr, const int32_t* res_kb, int nnzb,
                          const uint8_t* Rq, const void* s_r,
                          void* Y, int ldy,
                          void* workspace, size_t ws_bytes, hipStream_t stream);

/* ======================================================================== */
/* Layout conversion (offline; canonical <-> library layout)                 */
/* ======================================================================== */

/*
 * Canonical int4 weights -> library layout (the paper fixes no bit layout;
 * Section 4.2 fuses layout packing with quantisation).  The method's codes
 * lie in [-7, 7] (Eq. (1) with q_max = 7): a nibble of -8 (0x8) is stored as
 * -7 and counted.
 *   Wq_c      : uint8 [N, K/2] canonical nibbles, 8-byte aligned.
 *   s_w_c     : fp16 [N, K/128] (may be NULL together with s_w: no scales).
 *   Rq_c      : uint8 [nnzb, 128, 64] canonical nibbles (block p, row r,
 *               column c = code k of the block's 128), 8-byte aligned.
 *   Wq, s_w, Rq : out, library layout (Wq group order, s_w [K/128][N],
 *               Rq [nnzb, 128, 64] folded), 16-byte aligned packed outputs.
 *   n_invalid : optional int32 device counter; the number of -8 nibbles is
 *               added to it (atomically; the caller clears it).
 * The residual scales s_r and the CSR need no conversion.
 */
mq_status mq_repack_weights(int N, int K, const uint8_t* Wq_c, const void* s_w_c, int nnzb,
                            const uint8_t* Rq_c, uint8_t* Wq, void* s_w, uint8_t* Rq,
                            int32_t* n_invalid, hipStream_t stream);

/* Library layout -> canonical (the inverse of mq_repack_weights); pointer
 * rules mirrored (library side 16-byte aligned). */
mq_status mq_unpack_weights(int N, int K, const uint8_t* Wq, const void* s_w, int nnzb,
                            const uint8_t* Rq, uint8_t* Wq_c, void* s_w_c, uint8_t* Rq_c,
                            hipStream_t stream);

/*
 * Canonical int4 activation codes -> the library's activation operand layout, e.g. for
 * codes quantised elsewhere; -8 handled as for mq_repack_weights.
 *   Xq_c : uint8 [M, ldq] canonical rows (ldq >= K/2, ldq % 8 == 0), 8-byte aligned.
 *   Xq   : out, uint8 [M, 3K/4] activation operand layout, 16-byte aligned.
 */
mq_status mq_repack_act(int M, int K, const uint8_t* Xq_c, int ldq, uint8_t* Xq,
                        int32_t* n_invalid, hipStream_t stream);

/* Library-layout activation codes (as mq_quantize_act writes them) ->
 * canonical rows Xq_c [M, ldq]. */
mq_status mq_unpack_act(int M, int K, const uint8_t* Xq, uint8_t* Xq_c, int ldq,
                        hipStream_t stream);

/*
 * mq_linear without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  The workspace mq_linear would take (the
 * quantised rows, their scales, split-K partial sums) lives in a file-scope
 * device array of mq_scratch_bytes() bytes (128 MiB) that the library holds on
 * every GPU it runs on until the process ends.  The call allocates nothing.
 *   Same operands, results and checks as mq_linear.
 *   Returns MQ_ERR_SCRATCH_LIMIT, launching nothing, when
 *   mq_linear_workspace_size(M, N, K) > mq_scratch_bytes().
 *   Calls on one GPU share its array: calls that overlap in time on one GPU
 *   (other streams, other host threads) race and must be serialised by the
 *   caller.  Each call writes every scratch byte it reads; nothing needs
 *   clearing between calls.
 */
size_t mq_scratch_bytes(void);
mq_status mq_linear_noalloc(int M, int N, int K, const void* X, int ldx,
                            const uint8_t* Wq, const void* s_w,
                            const int32_t* res_rowptr, const int32_t* res_kb, int nnzb,
                            const uint8_t* Rq, const void* s_r,
                            void* Y, int ldy, hipStream_t stream);

/* ======================================================================== */
/* Offline weight preparation (not on the timed path)                        */
/* ======================================================================== */

/*
 * Dense 4-bit base and residual-norm block scores (Section 2 Eq. (1) per
 * (row, 128-group); residual R = W - Q(W) of Section 3 Eq. (4); block
 * criterion ||R_B||_F^2 of Section 3, Observation 2):
 *     s_w[n,g] = fp16_rn(fp32(max_{k in g} |W[n,k]|) / 7),
 *     Wq[n,k]  = clamp(round_half_even(W[n,k] / s_w[n,g]), -7, 7),
 *     R[n,k]   = W[n,k] - s_w[n,g] Wq[n,k]                    (fp32),
 *     score[nb,kb] = sum over the 128x128 block of R^2         (fp64).
 *   W     : fp32 [N, ldw], ldw >= K, ldw % 4 == 0, 16-byte aligned.
 *   Wq    : out, uint8 [N, K/2] group order;  s_w : out, fp16 [K/128, N].
 *   score : out, fp64 [N/128, K/128] (may be NULL to skip scoring).
 */
mq_status mq_quantize_weight(const float* W, int N, int K, int ldw,
                             uint8_t* Wq, void* s_w, double* score,
                             hipStream_t stream);

/*
 * Diagonal Hessian estimate h_j = (2/T) sum_t X[t,j]^2 from T calibration
 * tokens (Alg. 1, second step; Section 4.1).
 *   X : fp16 [T, ldx];  h : out, fp64 [K].
 */
mq_status mq_hessian_diag(const void* X, int T, int K, int ldx, double* h,
                          hipStream_t stream);

/*
 * Delta-Hessian block score (Alg. 1; Section 4.1):
 *     S_B = [ sum_B h_j R_ij^2 - sum_B h_j (R_ij - Q(R)_ij)^2 ]_+
 * with Q(R) the block's 4-bit residual (one scale per block row, as
 * mq_quantize_residual produces it) and R rebuilt from W, s_w and Wq.
 *   score : out, fp64 [N/128, K/128].
 */
mq_status mq_block_scores_dhessian(const float* W, int N, int K, int ldw,
                                   const uint8_t* Wq, const void* s_w,
                                   const double* h, double* score,
                                   hipStream_t stream);

/*
 * Top-K block selection and block mask in CSR form (Alg. 1, TopK and mask
 * steps): the nnzb blocks with the largest score are selected, ties broken by
 * the lower linear index nb * KB + kb.
 *   score      : fp64 [NB, KB]  (NB = N/128, KB = K/128), finite.
 *   res_rowptr : out, int32 [NB + 1];  res_kb : out, int32 [nnzb].
 * Requires 0 <= nnzb <= NB * KB.
 */
mq_status mq_select_blocks(const double* score, int NB, int KB, int nnzb,
                           int32_t* res_rowptr, int32_t* res_kb,
                           hipStream_t stream);

/*
 * Sparse 4-bit residual on the selected blocks (Section 3 Eq. (4); Alg. 1
 * last step), one fp16 scale per row inside each block (Eq. (1)):
 *     R = W - s_w Wq;  s_r[p][r] = fp16_rn(fp32(max_c |R|) / 7);
 *     Rq[p][r][c] = clamp(round_half_even(R / s_r), -7, 7)
 *   W, Wq, s_w : as for mq_quantize_weight (same W).
 *   CSR        : as for mq_fused_gemm.
 *   Rq, s_r    : out, uint8 [nnzb, 128, 64], fp16 [nnzb, 128].
 */
mq_status mq_quantize_residual(const float* W, int N, int K, int ldw,
                               const uint8_t* Wq, const void* s_w,
                               const int32_t* res_rowptr, const int32_t* res_kb,
                               int nnzb, uint8_t* Rq, void* s_r,
                               hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* MQ_H */
