/*
 * CPU oracle for MosaicQuant's fused W4A4 + sparse-residual linear layer.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the GPU library links, includes or
 * calls this file; only the test-suite, the smoke check and the CPU-baseline
 * leg of the benchmark load it.  It shares no code, header, table or constant
 * generator with the HIP path.
 *
 * Plain, slow, obviously-correct C.  Every function follows one passage of the
 * paper (arXiv 2606.15652, "MosaicQuant / ZipperEngine"):
 *
 *   Section 2, Eq. (1)   uniform symmetric quantisation, Q = round(X / s),
 *                        s = max|X| / q_max; dequantised value s * Q.
 *   Section 2, Eq. (2)   quantised linear layer X W ~ s_X s_W Q_X Q_W.
 *   Section 3, Eq. (4)   X W ~ Q(X) Q(W) + Q(X) Q(R), R = W - Q(W).
 *   Section 3 (Obs. 2)   residual-norm block criterion ||R_B||_F^2.
 *   Section 4.1, Alg. 1  Delta-Hessian score S_B, top-K selection, block mask,
 *                        W_MQ = Q(W) + M_S (.) Q(R).
 *
 * Readings of points the paper leaves open (each one is also listed, with its
 * reason, in the design notes):
 *   q_max = 7 (symmetric signed 4-bit, -8 never produced, clamp kept);
 *   round() = round half to even; the quotient x / s is the correctly rounded
 *   fp32 quotient by the stored fp16 scale; s = fp16_rn(fp32(max|x|) / 7);
 *   an all-zero vector (or a scale that rounds to 0) gives s = 0, q = 0;
 *   weights: one fp16 scale per output row per 128-long group along K;
 *   activations: one fp16 scale per token (row) over all K;
 *   residual: 128x128 blocks aligned with the groups, one fp16 scale per row
 *   inside each selected block;
 *   top-K ties: lower linear block index (nb * KB + kb) wins;
 *   W4A8 (appendix "Implementation Details": per-token dynamic activation
 *   quantisation): the same quantiser with q_max = 127, codes in [-127, 127];
 *   packed layout (the paper fixes no bit layout; its Section 4.2 fuses the
 *   layout packing with quantisation): 4 bits per code in 8-byte chunks of
 *   16 codes, sign-magnitude, folded as described at pack_chunk() below.
 *
 * Floating point: quantisation decisions are taken in fp32 (the precision the
 * GPU kernels use, so both sides decide every code identically); scores and
 * the output epilogue are fp64; integer dot products are exact (int64).
 * Build: gcc -O3 -fno-fast-math -ffp-contract=off -fopenmp -shared -fPIC.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_BLOCK 128   /* group length along K == residual block edge */

/* Threads the parallel loops below use (for reporting CPU timings). */
int orc_num_threads(void) { return omp_get_max_threads(); }
#define ORC_QMAX 7

/* ------------------------------------------------------------------------ */
/* IEEE binary16 <-> binary32, written from the format's definition.         */
/* ------------------------------------------------------------------------ */

/* Round a float to the nearest binary16 value (ties to even); return bits. */
uint16_t orc_f32_to_f16(float xf)
{
    uint16_t sign = signbit(xf) ? 0x8000u : 0u;
    double x = fabs((double)xf);
    if (isnan(xf)) return 0x7E00u;
    /* largest finite half is 65504; values >= 65520 round to infinity */
    if (x >= 65520.0) return (uint16_t)(sign | 0x7C00u);
    if (x == 0.0) return sign;
    /* quantum (unit in the last place) of the binade x falls in */
    int e;
    frexp(x, &e);                 /* x = f * 2^e, f in [0.5, 1) */
    int unbiased = e - 1;         /* x in [2^unbiased, 2^(unbiased+1)) */
    double quantum = unbiased < -14 ? ldexp(1.0, -24) : ldexp(1.0, unbiased - 10);
    double n = rint(x / quantum); /* exact division (power of two), RN-even */
    double v = n * quantum;       /* the rounded value, representable in half */
    if (v >= 65520.0) return (uint16_t)(sign | 0x7C00u);
    if (v < ldexp(1.0, -14)) {    /* subnormal (or rounded up to min normal) */
        uint32_t m = (uint32_t)(v / ldexp(1.0, -24));
        return (uint16_t)(sign | m);  /* m == 1024 encodes the min normal */
    }
    frexp(v, &e);
    unbiased = e - 1;
    uint32_t mant = (uint32_t)((v / ldexp(1.0, unbiased) - 1.0) * 1024.0);
    return (uint16_t)(sign | ((uint32_t)(unbiased + 15) << 10) | mant);
}

float orc_f16_to_f32(uint16_t h)
{
    int s = (h >> 15) & 1, ex = (h >> 10) & 0x1F, m = h & 0x3FF;
    double v;
    if (ex == 0x1F) v = m ? NAN : INFINITY;
    else if (ex == 0) v = ldexp((double)m, -24);
    else v = ldexp(1.0 + m / 1024.0, ex - 15);
    return (float)(s ? -v : v);
}

void orc_f32_to_f16_array(const float* x, uint16_t* h, int64_t n)
{
    for (int64_t i = 0; i < n; ++i) h[i] = orc_f32_to_f16(x[i]);
}

void orc_f16_to_f32_array(const uint16_t* h, float* x, int64_t n)
{
    for (int64_t i = 0; i < n; ++i) x[i] = orc_f16_to_f32(h[i]);
}

/* ------------------------------------------------------------------------ */
/* Eq. (1): symmetric b-bit quantisation of one vector, q_max = 2^(b-1) - 1. */
/* ------------------------------------------------------------------------ */

/* Quantise v[0..n) (stride 1) with q_max = qmax.  Writes the fp16 scale bits
 * and the codes. */
static void quant_sym(const float* v, int n, int qmax, uint16_t* s_bits, int8_t* q)
{
    float amax = 0.0f;
    for (int i = 0; i < n; ++i) {
        float a = fabsf(v[i]);
        if (a > amax) amax = a;
    }
    float ratio = amax / (float)qmax;         /* fp32, correctly rounded */
    uint16_t sb = orc_f32_to_f16(ratio);
    float s = orc_f16_to_f32(sb);
    *s_bits = sb;
    for (int i = 0; i < n; ++i) {
        if (s == 0.0f) { q[i] = 0; continue; }
        float r = rintf(v[i] / s);            /* fp32 quotient, ties to even */
        if (r > qmax) r = (float)qmax;
        if (r < -qmax) r = (float)-qmax;
        q[i] = (int8_t)r;
    }
}

/* the 4-bit quantiser of the method (q_max = 7) */
static void quant_sym4(const float* v, int n, uint16_t* s_bits, int8_t* q)
{
    quant_sym(v, n, ORC_QMAX, s_bits, q);
}

/* ------------------------------------------------------------------------ */
/* Packed layout of 4-bit codes.                                             */
/*                                                                           */
/* A row of K codes is K/16 chunks of 8 bytes; chunk c holds codes           */
/* k = 16c .. 16c + 15.  Code e of a chunk (|q| <= 7) becomes the 6-bit field */
/*     f_e = 32 * [q < 0] + |q|                                              */
/* at bit 6e of a 96-bit word O (bits 6e+3 and 6e+4 stay zero).  Writing     */
/* O = o0 + 2^32 o1 + 2^64 o2, let ZA (ZB) be the always-zero bits of o0     */
/* (o1); ZA and ZB are disjoint and together cover every bit of o2 that can  */
/* be non-zero, so the chunk stores the two little-endian 32-bit words       */
/*     P0 = o0 | (o2 & ZA),   P1 = o1 | (o2 & ZB)                            */
/* and o2 = (P0 & ZA) | (P1 & ZB) comes back from them.  Every 8-byte        */
/* pattern decodes to 16 codes in [-7, 7] (a set sign bit with magnitude 0   */
/* is the code 0).                                                           */
/* ------------------------------------------------------------------------ */

/* always-zero bits of word w (0, 1, 2) of O, derived from the field layout */
static uint32_t zero_bits(int w)
{
    uint32_t z = 0;
    for (int e = 0; e < 16; ++e)
        for (int b = 3; b <= 4; ++b) {
            int bit = 6 * e + b;
            if (bit / 32 == w) z |= 1u << (bit % 32);
        }
    return z;
}

static uint32_t rd32(const uint8_t* p)
{
    return (uint32_t)p[0] | ((uint32_t)p[1] << 8) | ((uint32_t)p[2] << 16) | ((uint32_t)p[3] << 24);
}

static void wr32(uint8_t* p, uint32_t v)
{
    p[0] = (uint8_t)v; p[1] = (uint8_t)(v >> 8); p[2] = (uint8_t)(v >> 16); p[3] = (uint8_t)(v >> 24);
}

/* 16 codes -> 8 bytes */
static void pack_chunk(const int8_t* q, uint8_t* out)
{
    uint32_t o[3] = {0, 0, 0};
    for (int e = 0; e < 16; ++e) {
        int mag = q[e] < 0 ? -q[e] : q[e];
        uint32_t f = (uint32_t)((q[e] < 0 ? 32 : 0) + mag);
        for (int b = 0; b < 6; ++b)
            if (f & (1u << b)) {
                int bit = 6 * e + b;
                o[bit / 32] |= 1u << (bit % 32);
            }
    }
    wr32(out, o[0] | (o[2] & zero_bits(0)));
    wr32(out + 4, o[1] | (o[2] & zero_bits(1)));
}

/* 8 bytes -> 16 codes */
static void unpack_chunk(const uint8_t* ch, int8_t* q)
{
    uint32_t p0 = rd32(ch), p1 = rd32(ch + 4);
    uint32_t za = zero_bits(0), zb = zero_bits(1);
    uint32_t o[3] = {p0 & ~za, p1 & ~zb, (p0 & za) | (p1 & zb)};
    for (int e = 0; e < 16; ++e) {
        uint32_t f = 0;
        for (int b = 0; b < 6; ++b) {
            int bit = 6 * e + b;
            if (o[bit / 32] & (1u << (bit % 32))) f |= 1u << b;
        }
        int mag = (int)(f & 7u);
        q[e] = (int8_t)((f & 32u) ? -mag : mag);
    }
}

/* signed value of code k of a packed row */
static int unpack_code(const uint8_t* row, int k)
{
    int8_t q[16];
    unpack_chunk(row + (k / 16) * 8, q);
    return q[k % 16];
}

/* packed bytes (K/2) -> codes of a row */
static void unpack_row(const uint8_t* packed, int K, int8_t* out)
{
    for (int c = 0; c < K / 16; ++c) unpack_chunk(packed + 8 * c, out + 16 * c);
}

/* codes of a row (K a multiple of 16) -> packed bytes (K/2) */
static void pack_row(const int8_t* q, int K, uint8_t* out)
{
    for (int c = 0; c < K / 16; ++c) pack_chunk(q + 16 * c, out + 8 * c);
}

int orc_unpack_code(const uint8_t* row, int k) { return unpack_code(row, k); }
void orc_pack_codes(const int8_t* q, int rows, int K, uint8_t* out)
{
    for (int r = 0; r < rows; ++r) pack_row(q + (int64_t)r * K, K, out + (int64_t)r * (K / 2));
}
void orc_unpack_codes(const uint8_t* packed, int rows, int K, int8_t* out)
{
    for (int r = 0; r < rows; ++r) unpack_row(packed + (int64_t)r * (K / 2), K, out + (int64_t)r * K);
}

/* ------------------------------------------------------------------------ */
/* Activation operand layout (the form the library's quantiser writes): for  */
/* row r, 128-code group g and quarter j (codes k = 128 g + 32 j + e,         */
/* e = 0 .. 31), the 6-bit fields f_e of the packed layout (not folded) form */
/* the 192-bit word F = sum_e f_e 2^(6e), six little-endian 32-bit words     */
/* d0 .. d5.  With G = K / 128 groups and M rows:                            */
/*   d0 .. d3 at byte (g M + r) 64 + 16 j          (main plane), and        */
/*   d4, d5   at byte G M 64 + (g M + r) 32 + 8 j   (tail plane).            */
/* 3K/4 bytes per row.  The fields' exponent bits (6e+3, 6e+4) are zero.     */
/* ------------------------------------------------------------------------ */
static uint64_t act6_main(int M, int r, int g, int j) { return ((uint64_t)g * M + r) * 64 + 16 * (uint64_t)j; }
static uint64_t act6_tail(int M, int G, int r, int g, int j)
{
    return (uint64_t)G * M * 64 + ((uint64_t)g * M + r) * 32 + 8 * (uint64_t)j;
}

void orc_pack_act6(const int8_t* q, int M, int K, uint8_t* out)
{
    int G = K / 128;
    for (int r = 0; r < M; ++r)
        for (int g = 0; g < G; ++g)
            for (int j = 0; j < 4; ++j) {
                uint32_t d[6] = {0, 0, 0, 0, 0, 0};
                for (int e = 0; e < 32; ++e) {
                    int v = q[(int64_t)r * K + 128 * g + 32 * j + e];
                    uint32_t f = (uint32_t)((v < 0 ? 32 : 0) + (v < 0 ? -v : v));
                    for (int b = 0; b < 6; ++b)
                        if (f & (1u << b)) {
                            int bit = 6 * e + b;
                            d[bit / 32] |= 1u << (bit % 32);
                        }
                }
                uint8_t* mp = out + act6_main(M, r, g, j);
                for (int w = 0; w < 4; ++w) wr32(mp + 4 * w, d[w]);
                uint8_t* tp = out + act6_tail(M, G, r, g, j);
                wr32(tp, d[4]);
                wr32(tp + 4, d[5]);
            }
}

/* the inverse; returns the number of fields with a non-zero exponent bit
 * (such a field is not a code) */
int64_t orc_unpack_act6(const uint8_t* in, int M, int K, int8_t* q)
{
    int G = K / 128;
    int64_t bad = 0;
    for (int r = 0; r < M; ++r)
        for (int g = 0; g < G; ++g)
            for (int j = 0; j < 4; ++j) {
                uint32_t d[6];
                const uint8_t* mp = in + act6_main(M, r, g, j);
                const uint8_t* tp = in + act6_tail(M, G, r, g, j);
                for (int w = 0; w < 4; ++w) d[w] = rd32(mp + 4 * w);
                d[4] = rd32(tp);
                d[5] = rd32(tp + 4);
                for (int e = 0; e < 32; ++e) {
                    uint32_t f = 0;
                    for (int b = 0; b < 6; ++b) {
                        int bit = 6 * e + b;
                        if (d[bit / 32] & (1u << (bit % 32))) f |= 1u << b;
                    }
                    if (f & 24u) ++bad;
                    int mag = (int)(f & 7u);
                    q[(int64_t)r * K + 128 * g + 32 * j + e] = (int8_t)((f & 32u) ? -mag : mag);
                }
            }
    return bad;
}

/* ------------------------------------------------------------------------ */
/* Canonical nibble layout (the interchange format of the library's          */
/* boundary): one 4-bit two's-complement code per nibble, two per byte, the  */
/* even k in the low nibble, rows of K/2 bytes in k order.  A nibble holds   */
/* -8 .. 7; the method's codes are -7 .. 7 (Eq. (1) with q_max = 7).         */
/* ------------------------------------------------------------------------ */
void orc_pack_nibbles(const int8_t* q, int rows, int K, uint8_t* out)
{
    for (int64_t i = 0; i < (int64_t)rows * (K / 2); ++i) {
        int lo = q[2 * i], hi = q[2 * i + 1];
        out[i] = (uint8_t)(((unsigned)lo & 0xFu) | (((unsigned)hi & 0xFu) << 4));
    }
}

void orc_unpack_nibbles(const uint8_t* in, int rows, int K, int8_t* q)
{
    for (int64_t i = 0; i < (int64_t)rows * (K / 2); ++i) {
        int lo = in[i] & 0xF, hi = in[i] >> 4;
        q[2 * i] = (int8_t)(lo >= 8 ? lo - 16 : lo);
        q[2 * i + 1] = (int8_t)(hi >= 8 ? hi - 16 : hi);
    }
}

/* ------------------------------------------------------------------------ */
/* Per-token activation quantisation (Eq. 1 applied row by row).             */
/* ------------------------------------------------------------------------ */
void orc_quantize_act(const uint16_t* X, int M, int K, int ldx,
                      uint8_t* Xq, uint16_t* s_x)
{
    #pragma omp parallel for schedule(static)
    for (int m = 0; m < M; ++m) {
        float* v = (float*)malloc(sizeof(float) * (size_t)K);
        int8_t* q = (int8_t*)malloc((size_t)K);
        for (int k = 0; k < K; ++k) v[k] = orc_f16_to_f32(X[(int64_t)m * ldx + k]);
        quant_sym4(v, K, &s_x[m], q);
        pack_row(q, K, Xq + (int64_t)m * (K / 2));
        free(v);
        free(q);
    }
}

/* Per-token symmetric INT8 activation quantisation (the W4A8 setting of the
 * appendix "Implementation Details": per-token dynamic activation
 * quantisation; Eq. (1) with q_max = 127, -128 never produced).  Codes are
 * plain int8 [M, K] row-major. */
void orc_quantize_act8(const uint16_t* X, int M, int K, int ldx,
                       int8_t* Xq8, uint16_t* s_x)
{
    #pragma omp parallel for schedule(static)
    for (int m = 0; m < M; ++m) {
        float* v = (float*)malloc(sizeof(float) * (size_t)K);
        for (int k = 0; k < K; ++k) v[k] = orc_f16_to_f32(X[(int64_t)m * ldx + k]);
        quant_sym(v, K, 127, &s_x[m], Xq8 + (int64_t)m * K);
        free(v);
    }
}

/* ------------------------------------------------------------------------ */
/* Dense 4-bit base Q(W) and residual R = W - Q(W) (Eq. 4; Alg. 1 first     */
/* step).  Groups of 128 along K, one scale per (row, group).                */
/* ------------------------------------------------------------------------ */
void orc_quantize_weight(const float* W, int N, int K,
                         uint8_t* Wq, uint16_t* s_w, float* R)
{
    const int G = K / ORC_BLOCK;
    #pragma omp parallel for schedule(static)
    for (int n = 0; n < N; ++n) {
        int8_t q[ORC_BLOCK];
        for (int g = 0; g < G; ++g) {
            const float* v = W + (int64_t)n * K + (int64_t)g * ORC_BLOCK;
            uint16_t sb;
            quant_sym4(v, ORC_BLOCK, &sb, q);
            s_w[(int64_t)n * G + g] = sb;
            float s = orc_f16_to_f32(sb);
            pack_row(q, ORC_BLOCK, Wq + (int64_t)n * (K / 2) + (int64_t)g * (ORC_BLOCK / 2));
            if (R) {
                float* r = R + (int64_t)n * K + (int64_t)g * ORC_BLOCK;
                for (int i = 0; i < ORC_BLOCK; ++i) {
                    float deq = s * (float)q[i];    /* exact in fp32 */
                    r[i] = v[i] - deq;              /* one rounding */
                }
            }
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Block scores.                                                             */
/* ------------------------------------------------------------------------ */

/* Residual-norm criterion (Section 3, Observation 2): ||R_B||_F^2, summed in
 * fp64 over the block in row-major order. score is [NB, KB] row-major. */
void orc_block_scores_frob(const float* R, int N, int K, double* score)
{
    const int NB = N / ORC_BLOCK, KB = K / ORC_BLOCK;
    #pragma omp parallel for schedule(static)
    for (int b = 0; b < NB * KB; ++b) {
        int nb = b / KB, kb = b % KB;
        double acc = 0.0;
        for (int r = 0; r < ORC_BLOCK; ++r)
            for (int c = 0; c < ORC_BLOCK; ++c) {
                double x = R[(int64_t)(nb * ORC_BLOCK + r) * K + kb * ORC_BLOCK + c];
                acc += x * x;
            }
        score[b] = acc;
    }
}

/* Diagonal Hessian estimate h_j = (2/T) sum_t X[t,j]^2 over T calibration
 * tokens (Alg. 1 second step; Section 4.1).  X is fp16 bits [T, K]. */
void orc_hessian_diag(const uint16_t* X, int T, int K, double* h)
{
    for (int j = 0; j < K; ++j) {
        double acc = 0.0;
        for (int t = 0; t < T; ++t) {
            double x = orc_f16_to_f32(X[(int64_t)t * K + j]);
            acc += x * x;
        }
        h[j] = 2.0 / (double)T * acc;
    }
}

/* Delta-Hessian score (Alg. 1; Section 4.1):
 *   S_B = [ sum_B h_j R_ij^2 - sum_B h_j (R_ij - Q(R)_ij)^2 ]_+
 * where Q(R) is the block's 4-bit residual with one scale per block row
 * (the same quantiser the selected blocks later receive). */
void orc_block_scores_dhessian(const float* R, int N, int K, const double* h,
                               double* score)
{
    const int NB = N / ORC_BLOCK, KB = K / ORC_BLOCK;
    #pragma omp parallel for schedule(static)
    for (int b = 0; b < NB * KB; ++b) {
        int nb = b / KB, kb = b % KB;
        double before = 0.0, after = 0.0;
        int8_t q[ORC_BLOCK];
        for (int r = 0; r < ORC_BLOCK; ++r) {
            const float* v = R + (int64_t)(nb * ORC_BLOCK + r) * K + kb * ORC_BLOCK;
            uint16_t sb;
            quant_sym4(v, ORC_BLOCK, &sb, q);
            double s = orc_f16_to_f32(sb);
            for (int c = 0; c < ORC_BLOCK; ++c) {
                double hj = h[kb * ORC_BLOCK + c];
                double rv = v[c];
                double e = rv - s * (double)q[c];
                before += hj * rv * rv;
                after += hj * e * e;
            }
        }
        double d = before - after;
        score[b] = d > 0.0 ? d : 0.0;
    }
}

/* ------------------------------------------------------------------------ */
/* Top-K selection (Alg. 1) and block mask in CSR form.                      */
/* ------------------------------------------------------------------------ */
static const double* g_sort_scores;
static int cmp_desc(const void* a, const void* b)
{
    int i = *(const int*)a, j = *(const int*)b;
    double si = g_sort_scores[i], sj = g_sort_scores[j];
    if (si > sj) return -1;
    if (si < sj) return 1;
    return (i > j) - (i < j);        /* tie: lower linear index first */
}

/* Select the nnzb highest-scoring blocks.  Output: CSR over block rows,
 * rowptr [NB+1], kb [nnzb] ascending within each row; also mask [NB*KB]
 * (1 = selected) if non-null.  Returns 0, or -1 on bad nnzb. */
int orc_select_topk(const double* score, int NB, int KB, int nnzb,
                    int32_t* rowptr, int32_t* kb_out, uint8_t* mask)
{
    int nblk = NB * KB;
    if (nnzb < 0 || nnzb > nblk) return -1;
    int* order = (int*)malloc(sizeof(int) * (size_t)(nblk > 0 ? nblk : 1));
    uint8_t* sel = (uint8_t*)calloc((size_t)(nblk > 0 ? nblk : 1), 1);
    for (int i = 0; i < nblk; ++i) order[i] = i;
    g_sort_scores = score;
    qsort(order, (size_t)nblk, sizeof(int), cmp_desc);
    for (int i = 0; i < nnzb; ++i) sel[order[i]] = 1;
    int p = 0;
    rowptr[0] = 0;
    for (int nb = 0; nb < NB; ++nb) {
        for (int kb = 0; kb < KB; ++kb)
            if (sel[nb * KB + kb]) kb_out[p++] = kb;
        rowptr[nb + 1] = p;
    }
    if (mask) memcpy(mask, sel, (size_t)nblk);
    free(order);
    free(sel);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Sparse 4-bit residual M_S (.) Q(R) on the selected blocks (Eq. 4; Alg. 1  */
/* last step).  Rq is block-major [nnzb][128 rows][64 bytes]; s_r [nnzb][128]*/
/* ------------------------------------------------------------------------ */
void orc_quantize_residual(const float* R, int N, int K,
                           const int32_t* rowptr, const int32_t* kb_idx, int nnzb,
                           uint8_t* Rq, uint16_t* s_r)
{
    const int NB = N / ORC_BLOCK;
    (void)nnzb;
    for (int nb = 0; nb < NB; ++nb) {
        for (int p = rowptr[nb]; p < rowptr[nb + 1]; ++p) {
            int kb = kb_idx[p];
            int8_t q[ORC_BLOCK];
            for (int r = 0; r < ORC_BLOCK; ++r) {
                const float* v = R + (int64_t)(nb * ORC_BLOCK + r) * K + kb * ORC_BLOCK;
                quant_sym4(v, ORC_BLOCK, &s_r[(int64_t)p * ORC_BLOCK + r], q);
                pack_row(q, ORC_BLOCK, Rq + ((int64_t)p * ORC_BLOCK + r) * (ORC_BLOCK / 2));
            }
        }
    }
}

/* ------------------------------------------------------------------------ */
/* The linear layer itself (Eq. 2 and Eq. 4):                                */
/*   A_b[m,n,g] = sum_{k in g} Xq[m,k] Wq[n,k]                               */
/*   A_r[m,n,g] = sum_{k in g} Xq[m,k] Rq[p][n%128][k%128]   (selected only) */
/*   Tb = sum_g A_b,  Tr = sum_g A_r                        (exact, int64)   */
/*   Y[m,n] = s_x[m] * sum_g ( s_w[n,g] A_b + [sel] s_r[p][n%128] A_r )      */
/* with the fp16 scales widened exactly and the sum taken in fp64.           */
/* ------------------------------------------------------------------------ */
typedef struct {
    int M, N, K, G, NB;
    const uint8_t *Xq, *Wq, *Rq;
    double *sx, *sw, *sr;    /* the fp16 scales, widened exactly */
    int32_t* pmap;           /* [NB*G]: residual block index p or -1 */
} orc_layer;

static void layer_init(orc_layer* L, int M, int N, int K,
                       const uint8_t* Xq, const uint16_t* s_x,
                       const uint8_t* Wq, const uint16_t* s_w,
                       const int32_t* rowptr, const int32_t* kb_idx,
                       const uint8_t* Rq, const uint16_t* s_r)
{
    L->M = M; L->N = N; L->K = K; L->G = K / ORC_BLOCK; L->NB = N / ORC_BLOCK;
    L->Xq = Xq; L->Wq = Wq; L->Rq = Rq;
    L->pmap = (int32_t*)malloc(sizeof(int32_t) * (size_t)L->NB * L->G);
    for (int i = 0; i < L->NB * L->G; ++i) L->pmap[i] = -1;
    int nnzb = 0;
    if (rowptr) {
        for (int nb = 0; nb < L->NB; ++nb)
            for (int p = rowptr[nb]; p < rowptr[nb + 1]; ++p)
                L->pmap[nb * L->G + kb_idx[p]] = p;
        nnzb = rowptr[L->NB];
    }
    L->sx = (double*)malloc(sizeof(double) * (size_t)(M > 0 ? M : 1));
    L->sw = (double*)malloc(sizeof(double) * (size_t)N * L->G);
    L->sr = (double*)malloc(sizeof(double) * (size_t)(nnzb > 0 ? nnzb : 1) * ORC_BLOCK);
    for (int m = 0; m < M; ++m) L->sx[m] = orc_f16_to_f32(s_x[m]);
    for (int64_t i = 0; i < (int64_t)N * L->G; ++i) L->sw[i] = orc_f16_to_f32(s_w[i]);
    for (int64_t i = 0; i < (int64_t)nnzb * ORC_BLOCK; ++i) L->sr[i] = orc_f16_to_f32(s_r[i]);
}

static void layer_free(orc_layer* L)
{
    free(L->pmap); free(L->sx); free(L->sw); free(L->sr);
}

/* One output element.  xrow/wrow are the unpacked int8 codes of the row. */
static void layer_elem(const orc_layer* L, const int8_t* xrow, const int8_t* wrow,
                       int m, int n, int64_t* tb, int64_t* tr, double* y)
{
    const int K = L->K;
    int64_t Tb = 0, Tr = 0;
    double acc = 0.0;
    for (int g = 0; g < L->G; ++g) {
        int64_t ab = 0;
        for (int k = g * ORC_BLOCK; k < (g + 1) * ORC_BLOCK; ++k)
            ab += (int64_t)xrow[k] * wrow[k];
        Tb += ab;
        acc += L->sw[(int64_t)n * L->G + g] * (double)ab;
        int p = L->pmap[(n / ORC_BLOCK) * L->G + g];
        if (p >= 0) {
            const uint8_t* rrow = L->Rq + ((int64_t)p * ORC_BLOCK + n % ORC_BLOCK) * (ORC_BLOCK / 2);
            int8_t rc[ORC_BLOCK];
            unpack_row(rrow, ORC_BLOCK, rc);
            int64_t ar = 0;
            for (int c = 0; c < ORC_BLOCK; ++c)
                ar += (int64_t)xrow[g * ORC_BLOCK + c] * rc[c];
            Tr += ar;
            acc += L->sr[(int64_t)p * ORC_BLOCK + n % ORC_BLOCK] * (double)ar;
        }
    }
    (void)K;
    *tb = Tb;
    *tr = Tr;
    *y = L->sx[m] * acc;
}


/* Full layer: Tb, Tr, Y64 are [M, N] row-major (any may be NULL).
 * Returns the number of entries of Tb or Tr outside the int32 range. */
int64_t orc_linear(int M, int N, int K,
                   const uint8_t* Xq, const uint16_t* s_x,
                   const uint8_t* Wq, const uint16_t* s_w,
                   const int32_t* rowptr, const int32_t* kb_idx, int nnzb,
                   const uint8_t* Rq, const uint16_t* s_r,
                   int64_t* Tb, int64_t* Tr, double* Y64)
{
    orc_layer L;
    layer_init(&L, M, N, K, Xq, s_x, Wq, s_w, nnzb > 0 ? rowptr : NULL, kb_idx, Rq, s_r);
    int8_t* wun = (int8_t*)malloc((size_t)N * K);
    #pragma omp parallel for schedule(static)
    for (int n = 0; n < N; ++n) unpack_row(Wq + (int64_t)n * (K / 2), K, wun + (int64_t)n * K);
    int64_t overflow = 0;
    #pragma omp parallel for schedule(dynamic, 1) reduction(+ : overflow)
    for (int m = 0; m < M; ++m) {
        int8_t* xrow = (int8_t*)malloc((size_t)K);
        unpack_row(Xq + (int64_t)m * (K / 2), K, xrow);
        for (int n = 0; n < N; ++n) {
            int64_t tb, tr;
            double y;
            layer_elem(&L, xrow, wun + (int64_t)n * K, m, n, &tb, &tr, &y);
            if (tb > INT32_MAX || tb < INT32_MIN || tr > INT32_MAX || tr < INT32_MIN) ++overflow;
            int64_t o = (int64_t)m * N + n;
            if (Tb) Tb[o] = tb;
            if (Tr) Tr[o] = tr;
            if (Y64) Y64[o] = y;
        }
        free(xrow);
    }
    free(wun);
    layer_free(&L);
    return overflow;
}

/* Selected outputs only: (ms[i], ns[i]) for i < ns_count. */
int64_t orc_linear_sampled(int M, int N, int K,
                           const uint8_t* Xq, const uint16_t* s_x,
                           const uint8_t* Wq, const uint16_t* s_w,
                           const int32_t* rowptr, const int32_t* kb_idx, int nnzb,
                           const uint8_t* Rq, const uint16_t* s_r,
                           int64_t count, const int32_t* ms, const int32_t* ns,
                           int64_t* Tb, int64_t* Tr, double* Y64)
{
    orc_layer L;
    layer_init(&L, M, N, K, Xq, s_x, Wq, s_w, nnzb > 0 ? rowptr : NULL, kb_idx, Rq, s_r);
    int64_t overflow = 0;
    #pragma omp parallel for schedule(dynamic, 16) reduction(+ : overflow)
    for (int64_t i = 0; i < count; ++i) {
        int8_t* xrow = (int8_t*)malloc((size_t)K);
        int8_t* wrow = (int8_t*)malloc((size_t)K);
        unpack_row(Xq + (int64_t)ms[i] * (K / 2), K, xrow);
        unpack_row(Wq + (int64_t)ns[i] * (K / 2), K, wrow);
        int64_t tb, tr;
        double y;
        layer_elem(&L, xrow, wrow, ms[i], ns[i], &tb, &tr, &y);
        if (tb > INT32_MAX || tb < INT32_MIN || tr > INT32_MAX || tr < INT32_MIN) ++overflow;
        if (Tb) Tb[i] = tb;
        if (Tr) Tr[i] = tr;
        if (Y64) Y64[i] = y;
        free(xrow);
        free(wrow);
    }
    layer_free(&L);
    return overflow;
}

/* W4A8 layer: as orc_linear, with the activations given as int8 codes
 * [M, K] (orc_quantize_act8) instead of packed 4-bit rows.  The group sums
 * and the epilogue are those of Eq. (4) and Eq. (2) unchanged. */
int64_t orc_linear_a8(int M, int N, int K,
                      const int8_t* Xq8, const uint16_t* s_x,
                      const uint8_t* Wq, const uint16_t* s_w,
                      const int32_t* rowptr, const int32_t* kb_idx, int nnzb,
                      const uint8_t* Rq, const uint16_t* s_r,
                      int64_t* Tb, int64_t* Tr, double* Y64)
{
    orc_layer L;
    layer_init(&L, M, N, K, NULL, s_x, Wq, s_w, nnzb > 0 ? rowptr : NULL, kb_idx, Rq, s_r);
    int8_t* wun = (int8_t*)malloc((size_t)N * K);
    #pragma omp parallel for schedule(static)
    for (int n = 0; n < N; ++n) unpack_row(Wq + (int64_t)n * (K / 2), K, wun + (int64_t)n * K);
    int64_t overflow = 0;
    #pragma omp parallel for schedule(dynamic, 1) reduction(+ : overflow)
    for (int m = 0; m < M; ++m) {
        const int8_t* xrow = Xq8 + (int64_t)m * K;
        for (int n = 0; n < N; ++n) {
            int64_t tb, tr;
            double y;
            layer_elem(&L, xrow, wun + (int64_t)n * K, m, n, &tb, &tr, &y);
            if (tb > INT32_MAX || tb < INT32_MIN || tr > INT32_MAX || tr < INT32_MIN) ++overflow;
            int64_t o = (int64_t)m * N + n;
            if (Tb) Tb[o] = tb;
            if (Tr) Tr[o] = tr;
            if (Y64) Y64[o] = y;
        }
    }
    free(wun);
    layer_free(&L);
    return overflow;
}

/* Selected outputs of the W4A8 layer: (ms[i], ns[i]) for i < count. */
int64_t orc_linear_a8_sampled(int M, int N, int K,
                              const int8_t* Xq8, const uint16_t* s_x,
                              const uint8_t* Wq, const uint16_t* s_w,
                              const int32_t* rowptr, const int32_t* kb_idx, int nnzb,
                              const uint8_t* Rq, const uint16_t* s_r,
                              int64_t count, const int32_t* ms, const int32_t* ns,
                              int64_t* Tb, int64_t* Tr, double* Y64)
{
    orc_layer L;
    layer_init(&L, M, N, K, NULL, s_x, Wq, s_w, nnzb > 0 ? rowptr : NULL, kb_idx, Rq, s_r);
    int64_t overflow = 0;
    #pragma omp parallel for schedule(dynamic, 16) reduction(+ : overflow)
    for (int64_t i = 0; i < count; ++i) {
        int8_t* wrow = (int8_t*)malloc((size_t)K);
        unpack_row(Wq + (int64_t)ns[i] * (K / 2), K, wrow);
        int64_t tb, tr;
        double y;
        layer_elem(&L, Xq8 + (int64_t)ms[i] * K, wrow, ms[i], ns[i], &tb, &tr, &y);
        if (tb > INT32_MAX || tb < INT32_MIN || tr > INT32_MAX || tr < INT32_MIN) ++overflow;
        if (Tb) Tb[i] = tb;
        if (Tr) Tr[i] = tr;
        if (Y64) Y64[i] = y;
        free(wrow);
    }
    layer_free(&L);
    return overflow;
}
