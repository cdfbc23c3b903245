/*
 * vc_oracle.c -- CPU oracle for the 8-bit VC-Attention forward (V-Smooth + ExpCast-FP8).
 *
 * TEST INFRASTRUCTURE. This file is the independent reference that the GPU library is checked
 * against. Only the test-suite, the smoke check and the benchmark's CPU-baseline leg may load it;
 * the product path never does. It shares no code, header or table with the HIP library.
 *
 * Style: plain scalar C, one obvious loop per definition, no blocking or fusion beyond what the
 * method itself prescribes. Floating point follows the method where the method fixes a decision
 * in fp32 (quantization scales and codes, the ExpCast-FP8 multiply-add of Sec. 3.3); every
 * accumulation that only feeds the tolerance-checked output is done in fp64. Build with
 * -ffp-contract=off and without fast-math so that every fp32 operation written here is exactly
 * one IEEE-754 rounding (fmaf where a fused multiply-add is meant).
 *
 * Paper references: Sec. 3.1 (online softmax, eq. tiled-low-bit-attention), Sec. 3.2 (V-Smooth:
 * eq. kv-reordering, eq. block-demeaning, eq. optimal-value-mean, eq. vc-online-update),
 * Sec. 3.3 (ExpCast-FP8, eq. direct-fp8), Sec. 3.4 and Appendix B (fused preprocessing operand
 * by operand), Appendix D (Proposition 1).
 *
 * Where the paper leaves a detail open, the reading taken here is the one listed in the
 * design notes of the repository ("readings" table); each such spot is marked READING below.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define D 128          /* head dimension; the whole method is stated at d = 128 */
#define BLK 128        /* hardware block B_v = 128 rows (Sec. 3.2) */
#define NPAIR 64       /* rotary channel pairs */

/* ------------------------------------------------------------------------------------------ */
/* Scalar formats                                                                             */
/* ------------------------------------------------------------------------------------------ */

float or_bf16_to_f32(uint16_t h)
{
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

/* bf16 round-to-nearest-even of an fp32 value (NaN kept quiet). */
uint16_t or_f32_to_bf16(float f)
{
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40);
    uint32_t lsb = (u >> 16) & 1u;
    u += 0x7fffu + lsb;
    return (uint16_t)(u >> 16);
}

/* OCP E4M3 (e4m3fn) decode, straight from the definition quoted in Sec. 3.3:
 * exponent field e (4 bits, bias 7), mantissa field m (3 bits); e > 0 encodes 2^(e-7)(1+m/8),
 * e = 0 encodes the subnormal 2^(-6) m/8; 0x7f and 0xff are NaN (no infinities). */
double or_e4m3_decode(uint8_t b)
{
    int e = (b >> 3) & 15, m = b & 7;
    double s = (b & 0x80) ? -1.0 : 1.0;
    if (e == 15 && m == 7) return NAN;
    if (e == 0) return s * ldexp(m / 8.0, -6);
    return s * ldexp(1.0 + m / 8.0, e - 7);
}

/* Sorted table of the 127 non-negative finite E4M3 values, code c <-> value (codes 0..126). */
static double g_e4m3_pos[127];
static int g_e4m3_init = 0;
static void e4m3_table(void)
{
    if (g_e4m3_init) return;
    for (int c = 0; c < 127; ++c) g_e4m3_pos[c] = or_e4m3_decode((uint8_t)c);
    g_e4m3_init = 1;
}

/* E4M3 encode: nearest representable value, ties to the even code (code parity is mantissa
 * parity), saturating to +-448 (code 0x7e) beyond the largest finite value. NaN -> 0x7f.
 * The search is a binary search over the sorted table above; no bit tricks. */
uint8_t or_e4m3_encode(float x)
{
    e4m3_table();
    if (isnan(x)) return 0x7f;
    uint8_t sign = signbit(x) ? 0x80 : 0x00;
    double a = fabs((double)x);
    if (a >= 448.0) return sign | 0x7e;
    int lo = 0, hi = 126;                 /* invariant: pos[lo] <= a < pos[hi] */
    while (hi - lo > 1) {
        int mid = (lo + hi) / 2;
        if (g_e4m3_pos[mid] <= a) lo = mid; else hi = mid;
    }
    double dlo = a - g_e4m3_pos[lo], dhi = g_e4m3_pos[hi] - a;
    int c;
    if (dlo < dhi) c = lo;
    else if (dhi < dlo) c = hi;
    else c = (lo % 2 == 0) ? lo : hi;
    return sign | (uint8_t)c;
}

/* ------------------------------------------------------------------------------------------ */
/* ExpCast-FP8 (Sec. 3.3, eq. direct-fp8)                                                     */
/* ------------------------------------------------------------------------------------------ */

/* The byte written for a log2-domain score u <= 0 with the row maximum scaled to 2^8:
 * clip to [0,120] of the round-to-nearest-even of 8(u+8) + 56 + beta, evaluated in fp32. */
int or_expcast_code_u(float u, float beta)
{
    float c = 8.0f * (u + 8.0f) + 56.0f + beta;
    float r = rintf(c);
    if (r < 0.0f) r = 0.0f;
    if (r > 120.0f) r = 120.0f;
    return (int)r;
}

/* The same map inside the attention loop. The score s of a query and a key (the int32 dot
 * product of the INT8 codes, or the fp32 score of the MXFP4 product) times a is in log2 units (a
 * folds the block scales, 1/sqrt(d), log2(e) and, with the Hadamard rotation, 1/128). With
 * running maximum m', u = s a - m', so 8(u+8)+56+beta = 8a*s + (120 + beta - 8m'): one fused
 * multiply-add in fp32.
 * READING: the multiply-add is fmaf(s, 8a, fl(fl(120+beta) - 8m')); 8a and 8m' are exact. */
int or_expcast_code_s(float s, float a, float m_new, float beta)
{
    float cst = 120.0f + beta;
    float bias = cst - 8.0f * m_new;
    float c = fmaf(s, 8.0f * a, bias);
    float r = rintf(c);
    if (r < 0.0f) r = 0.0f;
    if (r > 120.0f) r = 120.0f;
    return (int)r;
}
int or_expcast_code_acc(int32_t acc, float a, float m_new, float beta)
{
    return or_expcast_code_s((float)acc, a, m_new, beta);  /* |acc| < 2^24: exact */
}

/* The conventional path the paper compares against: exponentiate in fp32, scale by 2^8, cast
 * to E4M3 (Sec. 3.3, first listing). exp2 is evaluated in fp64 and rounded once to fp32. */
int or_exp_then_cast_code_s(float s, float a, float m_new)
{
    float t = s * a;
    float u = t - m_new;
    float p = (float)exp2((double)u);
    return (int)or_e4m3_encode(p * 256.0f);
}
int or_exp_then_cast_code_acc(int32_t acc, float a, float m_new)
{
    return or_exp_then_cast_code_s((float)acc, a, m_new);
}

/* ------------------------------------------------------------------------------------------ */
/* Rotary embedding over the (t, h, w) grid                                                   */
/* ------------------------------------------------------------------------------------------ */

/* READING (the paper fuses RoPE but never writes it out): 3-axis rotary embedding on
 * interleaved channel pairs (2i, 2i+1). Pairs 0..21 rotate with the frame index, 22..42 with
 * the row index, 43..63 with the column index; within an axis of d_a channels (44, 42, 42) pair
 * j turns by pos * theta^(-2j/d_a), theta = 10000.
 * Tables: row r of a (F+Ht+Wd) x 64 table is a position along one axis (rows 0..F-1 frames,
 * F..F+Ht-1 grid rows, F+Ht..F+Ht+Wd-1 grid columns); column i holds cos/sin of pair i's angle
 * when pair i belongs to that axis, and 1/0 otherwise. Angles in fp64, rounded once to fp32. */
static int pair_axis(int i) { return i < 22 ? 0 : (i < 43 ? 1 : 2); }
static int axis_first_pair(int a) { return a == 0 ? 0 : (a == 1 ? 22 : 43); }
static int axis_channels(int a) { return a == 0 ? 44 : 42; }

void or_rope_tables(int F, int Ht, int Wd, double theta, float *cos_t, float *sin_t)
{
    int rows = F + Ht + Wd;
    for (int r = 0; r < rows; ++r) {
        int axis = r < F ? 0 : (r < F + Ht ? 1 : 2);
        int pos = axis == 0 ? r : (axis == 1 ? r - F : r - F - Ht);
        for (int i = 0; i < NPAIR; ++i) {
            if (pair_axis(i) != axis) { cos_t[r * NPAIR + i] = 1.0f; sin_t[r * NPAIR + i] = 0.0f; continue; }
            int j = i - axis_first_pair(axis);
            double inv_freq = pow(theta, -(2.0 * j) / (double)axis_channels(axis));
            double ang = (double)pos * inv_freq;
            cos_t[r * NPAIR + i] = (float)cos(ang);
            sin_t[r * NPAIR + i] = (float)sin(ang);
        }
    }
}

/* Token n of the flattened latent grid: n = (f * Ht + y) * Wd + x. */
static void token_pos(int n, int Ht, int Wd, int *f, int *y, int *x)
{
    *x = n % Wd;
    *y = (n / Wd) % Ht;
    *f = n / (Wd * Ht);
}

/* Rotate one 128-channel row of token n in place:
 * y0 = fmaf(x0, c, -(x1*s)), y1 = fmaf(x0, s, x1*c)  (READING: this evaluation order). */
static void rope_row(float *x, int n, int F, int Ht, int Wd, const float *cos_t, const float *sin_t)
{
    int f, y, w;
    token_pos(n, Ht, Wd, &f, &y, &w);
    for (int i = 0; i < NPAIR; ++i) {
        int axis = pair_axis(i);
        int r = axis == 0 ? f : (axis == 1 ? F + y : F + Ht + w);
        float c = cos_t[r * NPAIR + i], s = sin_t[r * NPAIR + i];
        float x0 = x[2 * i], x1 = x[2 * i + 1];
        float p = x1 * s, q = x1 * c;
        x[2 * i] = fmaf(x0, c, -p);
        x[2 * i + 1] = fmaf(x0, s, q);
    }
}

/* ------------------------------------------------------------------------------------------ */
/* Hadamard rotation of Q and K (Sec. 3.4 / Appendix B)                                       */
/* ------------------------------------------------------------------------------------------ */

/* READING: Sylvester Hadamard H_128 (no random signs), unnormalised, applied as a fast
 * Walsh-Hadamard transform with stages h = 1, 2, 4, ..., 64 in this order, each butterfly
 * (a, b) -> (a + b, a - b) rounded in fp32. H H^T = 128 I, so (QH)(KH)^T = 128 QK^T and the
 * 1/128 is folded into the score scale. */
void or_fwht128(float *x)
{
    for (int h = 1; h < D; h <<= 1)
        for (int i = 0; i < D; ++i)
            if ((i & h) == 0) {
                float a = x[i], b = x[i + h];
                x[i] = a + b;
                x[i + h] = a - b;
            }
}

/* ------------------------------------------------------------------------------------------ */
/* Per-block symmetric INT8 quantizer for Q and K (Sec. 3.1 operand model)                    */
/* ------------------------------------------------------------------------------------------ */

/* READING: one fp32 scale per 128-row block, scale = amax/127, code = rint(x * (127/amax)),
 * clamped to [-127, 127]; amax over the valid rows only; an all-zero block gets scale 1 and
 * zero codes; rows past the valid count (padding) get zero codes. */
static void quant_block_i8(const float *x, int valid, int8_t *codes, float *scale)
{
    float amax = 0.0f;
    for (int r = 0; r < valid; ++r)
        for (int c = 0; c < D; ++c) {
            float v = fabsf(x[r * D + c]);
            if (v > amax) amax = v;
        }
    memset(codes, 0, (size_t)BLK * D);
    if (amax == 0.0f) { *scale = 1.0f; return; }
    float inv = 127.0f / amax;
    *scale = amax / 127.0f;
    for (int r = 0; r < valid; ++r)
        for (int c = 0; c < D; ++c) {
            float q = rintf(x[r * D + c] * inv);
            if (q > 127.0f) q = 127.0f;
            if (q < -127.0f) q = -127.0f;
            codes[r * D + c] = (int8_t)q;
        }
}

/* ------------------------------------------------------------------------------------------ */
/* MXFP4 quantizer for Q and K (the 4-bit variant: OCP microscaling, 32-element blocks)        */
/* ------------------------------------------------------------------------------------------ */

/* FP4 E2M1 element of the OCP MX formats: sign bit 3, exponent field bits 2..1 (bias 1),
 * mantissa bit 0. Exponent field 0 encodes the subnormal m/2, otherwise 2^(e-1) (1 + m/2):
 * magnitudes 0, 0.5, 1, 1.5, 2, 3, 4, 6. No infinities or NaN. */
double or_fp4_decode(uint8_t c)
{
    const int s = (c >> 3) & 1, e = (c >> 1) & 3, m = c & 1;
    const double mag = e == 0 ? 0.5 * m : ldexp(1.0 + 0.5 * m, e - 1);
    return s ? -mag : mag;
}

/* Nearest E2M1 value, ties to the code with mantissa bit 0, saturating at magnitude 6.
 * READING: a value whose magnitude rounds to 0 gets the code +0 (0x0). The search runs over the
 * 8 magnitudes in increasing order. */
uint8_t or_fp4_encode(float x)
{
    const double a = fabs((double)x);
    int best = 0;
    double bd = fabs(a - or_fp4_decode(0));
    for (int c = 1; c < 8; ++c) {
        const double d = fabs(a - or_fp4_decode((uint8_t)c));
        if (d < bd || (d == bd && (c & 1) == 0)) { bd = d; best = c; }
    }
    if (a > 6.0) best = 7;
    return (uint8_t)(best == 0 ? 0 : ((x < 0.0f ? 8 : 0) | best));
}

/* One block of 32 consecutive channels of a row. READING (OCP MX shared-scale rule): with amax
 * the block's largest magnitude, the shared exponent is X = floor(log2(amax)) - 2 (2 is the
 * largest E2M1 exponent), clamped to [-127, 127], stored as the E8M0 byte X + 127; each element
 * is or_fp4_encode(x * 2^-X) (the scaling is exact). An all-zero block gets the byte 127 and
 * zero codes. */
void or_mx_block(const float *x, uint8_t *codes, uint8_t *scale)
{
    float amax = 0.0f;
    for (int c = 0; c < 32; ++c)
        if (fabsf(x[c]) > amax) amax = fabsf(x[c]);
    if (amax == 0.0f) {
        *scale = 127;
        memset(codes, 0, 32);
        return;
    }
    int E;
    frexpf(amax, &E);  /* amax = f 2^E, f in [0.5, 1): floor(log2(amax)) = E - 1 */
    int X = E - 1 - 2;
    if (X < -127) X = -127;
    if (X > 127) X = 127;
    *scale = (uint8_t)(X + 127);
    for (int c = 0; c < 32; ++c) codes[c] = or_fp4_encode(ldexpf(x[c], -X));
}

/* Rows of a 128-row block: four MX blocks per valid row; padded rows get zero codes and the
 * scale byte 127. codes: one E2M1 code per byte [128 x 128]; scales [128 x 4]. */
static void quant_block_mx(const float *x, int valid, uint8_t *codes, uint8_t *scales)
{
    memset(codes, 0, (size_t)BLK * D);
    memset(scales, 127, (size_t)BLK * 4);
    for (int r = 0; r < valid; ++r)
        for (int b = 0; b < 4; ++b) or_mx_block(&x[r * D + 32 * b], &codes[r * D + 32 * b], &scales[r * 4 + b]);
}

/* FP8 Q/K (READING: the FP8-QK variant of Sec. 4.5 for matrix units without INT8): symmetric
 * OCP E4M3 codes per 128-row block, like the INT8 quantizer with 448 (the largest finite E4M3
 * value) in place of 127: scale = amax / 448, code = E4M3 nearest-even encoding of
 * fl(x * fl(448 / amax)) (at most 448 up to one rounding, so the encoder's saturation decides
 * nothing), with every code of zero magnitude stored as +0 (READING: the sign of an exact zero
 * after the rotation depends on the order of its additions, which the method does not fix);
 * all-zero block: scale 1, codes 0; padded rows: code 0. */
static void quant_block_f8(const float *x, int valid, uint8_t *codes, float *scale)
{
    float amax = 0.0f;
    for (int r = 0; r < valid; ++r)
        for (int c = 0; c < D; ++c) {
            float v = fabsf(x[r * D + c]);
            if (v > amax) amax = v;
        }
    memset(codes, 0, (size_t)BLK * D);
    if (amax == 0.0f) { *scale = 1.0f; return; }
    float inv = 448.0f / amax;
    *scale = amax / 448.0f;
    for (int r = 0; r < valid; ++r)
        for (int c = 0; c < D; ++c) {
            uint8_t b = or_e4m3_encode(x[r * D + c] * inv);
            codes[r * D + c] = (b & 0x7f) ? b : 0;
        }
}

/* The score of one query row against one key row from their MX codes, exact (fp64):
 * sum over the four blocks of 2^(Xq + Xk) times the block's dot product of the decoded elements. */
double or_mx_score(const uint8_t *q, const uint8_t *qs, const uint8_t *k, const uint8_t *ks)
{
    double s = 0.0;
    for (int b = 0; b < 4; ++b) {
        double dot = 0.0;
        for (int c = 32 * b; c < 32 * b + 32; ++c) dot += or_fp4_decode(q[c]) * or_fp4_decode(k[c]);
        s += ldexp(dot, ((int)qs[b] - 127) + ((int)ks[b] - 127));
    }
    return s;
}

/* ------------------------------------------------------------------------------------------ */
/* Preprocessing of one (batch, head): Q, K, V -> codes, scales, means (Sec. 3.4, App. B)     */
/* ------------------------------------------------------------------------------------------ */

enum { OR_QK_INT8 = 0, OR_QK_FP8 = 1, OR_QK_MXFP4 = 2 };

typedef struct {
    int32_t N, F, Ht, Wd;
    int32_t rope, hadamard, smooth_k, smooth_v;
    int32_t qk_fmt;  /* OR_QK_INT8, OR_QK_FP8 or OR_QK_MXFP4 */
} or_prep_cfg;

/* Inputs: Q, K, V as bf16 bit patterns [N x 128] in token order; perm (K/V gather, NULL =
 * identity); q_perm (Q gather, NULL = identity); RoPE tables (ignored when rope = 0).
 * Outputs, with T = ceil(N/128) and Np = 128 T:
 *   q_codes int8 [Np x 128], q_scale [T]          (query order, or q_perm order)
 *   k_codes int8 [Np x 128], k_scale [T]          (permuted order K' = K[perm])
 *   k_mean  fp32 [128]                            (zeros when smooth_k = 0)
 *   v_codes E4M3 bytes [Np x 128], v_scale [128]  (permuted order, residual after demeaning)
 *   v_mean  bf16 bits [T x 128]                   (zeros when smooth_v = 0)
 * With qk_fmt = OR_QK_FP8 q_codes / k_codes hold E4M3 bytes (same layout, scales amax/448).
 * With qk_fmt = OR_QK_MXFP4 the Q and K rows are quantized by MX blocks instead (the INT8
 * outputs are not written): q_mx, k_mx one E2M1 code per byte [Np x 128], q_mxs, k_mxs E8M0
 * scale bytes [Np x 4].
 * Returns 0, or -1 on allocation failure. */
int or_prep_head(const or_prep_cfg *cfg, const uint16_t *Q, const uint16_t *K, const uint16_t *V,
                 const int32_t *perm, const int32_t *q_perm, const float *cos_t, const float *sin_t,
                 int8_t *q_codes, float *q_scale, int8_t *k_codes, float *k_scale, float *k_mean,
                 uint8_t *v_codes, float *v_scale, uint16_t *v_mean,
                 uint8_t *q_mx, uint8_t *q_mxs, uint8_t *k_mx, uint8_t *k_mxs)
{
    const int mx = cfg->qk_fmt == OR_QK_MXFP4;
    const int N = cfg->N, T = (N + BLK - 1) / BLK, Np = T * BLK;
    float *xq = calloc((size_t)Np * D, sizeof(float));
    float *kr = calloc((size_t)N * D, sizeof(float));
    float *xk = calloc((size_t)Np * D, sizeof(float));
    float *xv = calloc((size_t)Np * D, sizeof(float));
    float *res = calloc((size_t)Np * D, sizeof(float));
    if (!xq || !kr || !xk || !xv || !res) { free(xq); free(kr); free(xk); free(xv); free(res); return -1; }

    /* Q: gather (optional), RoPE at the token's own grid position, Hadamard. */
    for (int r = 0; r < N; ++r) {
        int n = q_perm ? q_perm[r] : r;
        for (int c = 0; c < D; ++c) xq[r * D + c] = or_bf16_to_f32(Q[(size_t)n * D + c]);
        if (cfg->rope) rope_row(&xq[r * D], n, cfg->F, cfg->Ht, cfg->Wd, cos_t, sin_t);
        if (cfg->hadamard) or_fwht128(&xq[r * D]);
    }
    for (int j = 0; j < T; ++j) {
        int valid = N - j * BLK < BLK ? N - j * BLK : BLK;
        if (mx)
            quant_block_mx(&xq[(size_t)j * BLK * D], valid, &q_mx[(size_t)j * BLK * D], &q_mxs[(size_t)j * BLK * 4]);
        else if (cfg->qk_fmt == OR_QK_FP8)
            quant_block_f8(&xq[(size_t)j * BLK * D], valid, (uint8_t *)&q_codes[(size_t)j * BLK * D], &q_scale[j]);
        else
            quant_block_i8(&xq[(size_t)j * BLK * D], valid, &q_codes[(size_t)j * BLK * D], &q_scale[j]);
    }

    /* K: RoPE in token order. */
    for (int n = 0; n < N; ++n) {
        for (int c = 0; c < D; ++c) kr[(size_t)n * D + c] = or_bf16_to_f32(K[(size_t)n * D + c]);
        if (cfg->rope) rope_row(&kr[(size_t)n * D], n, cfg->F, cfg->Ht, cfg->Wd, cos_t, sin_t);
    }
    /* Key channel mean over the N tokens (softmax-invariant shift, Sec. 2 / App. B).
     * READING: fp32 sums in a fixed order: per original-order 128-token block a sequential sum
     * from 0 over its rows, then a sequential sum of the block sums, then one division by N;
     * the mean is subtracted before the Hadamard rotation (H is linear, so this equals
     * subtracting the rotated mean afterwards). */
    for (int c = 0; c < D; ++c) k_mean[c] = 0.0f;
    if (cfg->smooth_k) {
        for (int c = 0; c < D; ++c) {
            float tot = 0.0f;
            for (int j = 0; j < T; ++j) {
                int valid = N - j * BLK < BLK ? N - j * BLK : BLK;
                float part = 0.0f;
                for (int r = 0; r < valid; ++r) part += kr[(size_t)(j * BLK + r) * D + c];
                tot += part;
            }
            k_mean[c] = tot / (float)N;
        }
        for (int n = 0; n < N; ++n)
            for (int c = 0; c < D; ++c) kr[(size_t)n * D + c] = kr[(size_t)n * D + c] - k_mean[c];
    }
    /* K' = K[perm] (eq. kv-reordering), then Hadamard, then per-block INT8. */
    for (int r = 0; r < N; ++r) {
        int n = perm ? perm[r] : r;
        memcpy(&xk[(size_t)r * D], &kr[(size_t)n * D], D * sizeof(float));
        if (cfg->hadamard) or_fwht128(&xk[(size_t)r * D]);
    }
    for (int j = 0; j < T; ++j) {
        int valid = N - j * BLK < BLK ? N - j * BLK : BLK;
        if (mx)
            quant_block_mx(&xk[(size_t)j * BLK * D], valid, &k_mx[(size_t)j * BLK * D], &k_mxs[(size_t)j * BLK * 4]);
        else if (cfg->qk_fmt == OR_QK_FP8)
            quant_block_f8(&xk[(size_t)j * BLK * D], valid, (uint8_t *)&k_codes[(size_t)j * BLK * D], &k_scale[j]);
        else
            quant_block_i8(&xk[(size_t)j * BLK * D], valid, &k_codes[(size_t)j * BLK * D], &k_scale[j]);
    }

    /* V' = V[perm]; block means and residuals (eq. block-demeaning). */
    for (int r = 0; r < N; ++r) {
        int n = perm ? perm[r] : r;
        for (int c = 0; c < D; ++c) xv[(size_t)r * D + c] = or_bf16_to_f32(V[(size_t)n * D + c]);
    }
    for (int j = 0; j < T; ++j) {
        int valid = N - j * BLK < BLK ? N - j * BLK : BLK;
        for (int c = 0; c < D; ++c) {
            float mu = 0.0f;
            if (cfg->smooth_v) {
                /* READING: fp32 sequential sum over the block's valid rows, one division by the
                 * valid count, stored as bf16 (the 16-bit mean of Sec. 3.2); the residual uses
                 * the stored (rounded) mean, so residual + mean reproduces V' exactly. */
                float s = 0.0f;
                for (int r = 0; r < valid; ++r) s += xv[(size_t)(j * BLK + r) * D + c];
                uint16_t mb = or_f32_to_bf16(s / (float)valid);
                v_mean[(size_t)j * D + c] = mb;
                mu = or_bf16_to_f32(mb);
            } else {
                v_mean[(size_t)j * D + c] = 0;
            }
            for (int r = 0; r < valid; ++r)
                res[(size_t)(j * BLK + r) * D + c] = xv[(size_t)(j * BLK + r) * D + c] - mu;
        }
    }
    /* Per-channel E4M3 residual quantizer (Sec. 3.2 / App. B): READING: one scale per channel
     * over all N tokens of the head, scale = amax/448, code = E4M3(RNE, saturating) of
     * residual * (448/amax); an all-zero channel gets scale 1; padded rows get code 0. */
    memset(v_codes, 0, (size_t)Np * D);
    for (int c = 0; c < D; ++c) {
        float amax = 0.0f;
        for (int r = 0; r < N; ++r) {
            float v = fabsf(res[(size_t)r * D + c]);
            if (v > amax) amax = v;
        }
        if (amax == 0.0f) { v_scale[c] = 1.0f; continue; }
        float inv = 448.0f / amax;
        v_scale[c] = amax / 448.0f;
        for (int r = 0; r < N; ++r) v_codes[(size_t)r * D + c] = or_e4m3_encode(res[(size_t)r * D + c] * inv);
    }
    free(xq); free(kr); free(xk); free(xv); free(res);
    return 0;
}

/* ------------------------------------------------------------------------------------------ */
/* Attention on the prepared operands (Sec. 3.1 eq. tiled-low-bit-attention, Sec. 3.2         */
/* eq. vc-online-update, Sec. 3.3 eq. direct-fp8)                                             */
/* ------------------------------------------------------------------------------------------ */

enum { OR_P_EXPCAST = 0, OR_P_EXP_THEN_CAST = 1 };

typedef struct {
    int32_t N, hadamard, smooth_v, p_mode;
    float sm_scale, beta;
    int32_t qk_fmt;  /* OR_QK_INT8, OR_QK_FP8 or OR_QK_MXFP4 */
} or_attn_cfg;

/* Score scale in log2 units for one (query block, key block) pair:
 * a = fl(fl(sq * sk) * kappa), kappa = fp32(sm_scale * log2(e) / (hadamard ? 128 : 1)). */
static float score_kappa(const or_attn_cfg *cfg)
{
    double k = (double)cfg->sm_scale * 1.4426950408889634074;
    if (cfg->hadamard) k /= 128.0;
    return (float)k;
}

/* One query row against all key tiles, tiles of 128 keys taken in ascending order.
 * READING: the running maximum is the exact one of eq. tiled-low-bit-attention, updated once
 * per 128-key tile (no deferred rescaling), computed as max(m, fl(M*a)) with M the int32 row
 * maximum of the tile (rounding is monotone, so this is the maximum of fl(acc*a)). Padded key
 * columns are excluded from the maximum and get P = 0. The probability row sum r is the sum of
 * the decoded low-bit P (the normaliser accumulates exactly what multiplies V). A, l and alpha
 * are fp64. The block mean enters as r * (mu / s_V) in the code units of the residual
 * (App. B), so one final multiply by s_V returns value units. */
static void attn_row(const or_attn_cfg *cfg, int i, const int8_t *qc, const float *qs,
                     const int8_t *kc, const float *ks, const uint8_t *vc, const float *vs,
                     const uint16_t *vm, const uint8_t *qm, const uint8_t *qms, const uint8_t *km,
                     const uint8_t *kms, double *out, uint8_t *codes_out)
{
    const int N = cfg->N, T = (N + BLK - 1) / BLK;
    const int mx = cfg->qk_fmt == OR_QK_MXFP4;
    const float kappa = score_kappa(cfg);
    const float sq = mx ? 1.0f : qs[i / BLK];
    const int8_t *q = &qc[(size_t)i * D];
    double A[D], pv[D], mu_code[D];
    double l = 0.0;
    float m = -INFINITY;
    float sc[BLK];
    for (int c = 0; c < D; ++c) A[c] = 0.0;
    for (int j = 0; j < T; ++j) {
        const int valid = N - j * BLK < BLK ? N - j * BLK : BLK;
        /* INT8: s = the exact int32 dot product of the codes, a = fl(fl(s_q s_k) kappa);
         * MXFP4 (READING): s = the exact score of the MX codes rounded once to fp32 (the block
         * scales are inside s), a = kappa. */
        const float a = mx ? kappa : (sq * ks[j]) * kappa;
        float M = -INFINITY;
        for (int s = 0; s < valid; ++s) {
            const size_t key = (size_t)(j * BLK + s);
            float v;
            if (mx) {
                v = (float)or_mx_score(&qm[(size_t)i * D], &qms[(size_t)i * 4], &km[key * D], &kms[key * 4]);
            } else if (cfg->qk_fmt == OR_QK_FP8) {
                /* FP8 (READING): the exact dot product of the decoded E4M3 codes (exact in fp64:
                 * every product has 8 significant bits within a span of 2^-18 .. 2^17) rounded
                 * once to fp32; a = fl(fl(s_q s_k) kappa) as for INT8 */
                const uint8_t *qb = (const uint8_t *)q, *kb = (const uint8_t *)&kc[key * D];
                double dot = 0.0;
                for (int c = 0; c < D; ++c) dot += or_e4m3_decode(qb[c]) * or_e4m3_decode(kb[c]);
                v = (float)dot;
            } else {
                const int8_t *k = &kc[key * D];
                int32_t dot = 0;
                for (int c = 0; c < D; ++c) dot += (int32_t)q[c] * (int32_t)k[c];
                v = (float)dot;  /* |dot| <= 128 * 127^2 < 2^24: exact */
            }
            sc[s] = v;
            if (v > M) M = v;
        }
        float tmax = M * a;
        float m_new = m > tmax ? m : tmax;
        double alpha = (m == -INFINITY) ? 0.0 : exp2((double)m - (double)m_new);
        double r = 0.0;
        for (int c = 0; c < D; ++c) pv[c] = 0.0;
        for (int s = 0; s < valid; ++s) {
            int code = cfg->p_mode == OR_P_EXPCAST ? or_expcast_code_s(sc[s], a, m_new, cfg->beta)
                                                   : or_exp_then_cast_code_s(sc[s], a, m_new);
            if (codes_out) codes_out[j * BLK + s] = (uint8_t)code;
            double p = or_e4m3_decode((uint8_t)code);
            if (p == 0.0) continue;
            r += p;
            const uint8_t *v = &vc[(size_t)(j * BLK + s) * D];
            for (int c = 0; c < D; ++c) pv[c] += p * or_e4m3_decode(v[c]);
        }
        for (int c = 0; c < D; ++c)
            mu_code[c] = cfg->smooth_v ? (double)or_bf16_to_f32(vm[(size_t)j * D + c]) / (double)vs[c] : 0.0;
        for (int c = 0; c < D; ++c) A[c] = alpha * A[c] + pv[c] + r * mu_code[c];
        l = alpha * l + r;
        m = m_new;
    }
    for (int c = 0; c < D; ++c) out[c] = A[c] * (double)vs[c] / l;
}

/* Selected query rows (indices into the prepared query order) of one head. out: [n_rows x 128]
 * fp64, before the final bf16 rounding. Rows run in parallel; each row is independent. */
void or_attn_head(const or_attn_cfg *cfg, const int8_t *q_codes, const float *q_scale,
                  const int8_t *k_codes, const float *k_scale, const uint8_t *v_codes,
                  const float *v_scale, const uint16_t *v_mean, int n_rows, const int32_t *rows,
                  double *out, const uint8_t *q_mx, const uint8_t *q_mxs, const uint8_t *k_mx,
                  const uint8_t *k_mxs)
{
#pragma omp parallel for schedule(dynamic, 1)
    for (int t = 0; t < n_rows; ++t)
        attn_row(cfg, rows[t], q_codes, q_scale, k_codes, k_scale, v_codes, v_scale, v_mean,
                 q_mx, q_mxs, k_mx, k_mxs, &out[(size_t)t * D], NULL);
}

/* The 8-bit probability codes the recurrence forms for the selected query rows: codes_out
 * [n_rows x 128 T] (key order of the prepared K', padded keys 0), each tile's codes taken at that
 * tile's running maximum. Same arguments as or_attn_head otherwise (out may be scratch). */
void or_attn_head_codes(const or_attn_cfg *cfg, const int8_t *q_codes, const float *q_scale,
                        const int8_t *k_codes, const float *k_scale, const uint8_t *v_codes,
                        const float *v_scale, const uint16_t *v_mean, int n_rows, const int32_t *rows,
                        double *out, const uint8_t *q_mx, const uint8_t *q_mxs, const uint8_t *k_mx,
                        const uint8_t *k_mxs, uint8_t *codes_out)
{
    const int T = (cfg->N + BLK - 1) / BLK;
    memset(codes_out, 0, (size_t)n_rows * T * BLK);
#pragma omp parallel for schedule(dynamic, 1)
    for (int t = 0; t < n_rows; ++t)
        attn_row(cfg, rows[t], q_codes, q_scale, k_codes, k_scale, v_codes, v_scale, v_mean,
                 q_mx, q_mxs, k_mx, k_mxs, &out[(size_t)t * D], &codes_out[(size_t)t * T * BLK]);
}

/* The same online recurrence on full-precision operands (no quantizer, exact exponential):
 * scores s = q.k * sm_scale in fp64 from already rotated fp64 rows, P~ = exp(s - m') per
 * 128-key tile, block means mu_j of V' (fp64) restored through r * mu_j. Used only to pin the
 * recurrence (eq. tiled-low-bit-attention with eq. vc-online-update) against direct softmax. */
void or_attn_tiled_f64(int N, const double *Qf, const double *Kf, const double *Vf, double sm_scale,
                       int smooth_v, int n_rows, const int32_t *rows, double *out)
{
    const int T = (N + BLK - 1) / BLK;
    double *mu = calloc((size_t)T * D, sizeof(double));
    for (int j = 0; j < T && smooth_v; ++j) {
        int valid = N - j * BLK < BLK ? N - j * BLK : BLK;
        for (int c = 0; c < D; ++c) {
            double s = 0.0;
            for (int r = 0; r < valid; ++r) s += Vf[(size_t)(j * BLK + r) * D + c];
            mu[(size_t)j * D + c] = s / valid;
        }
    }
#pragma omp parallel for schedule(dynamic, 1)
    for (int t = 0; t < n_rows; ++t) {
        const int i = rows[t];
        double A[D], sc[BLK], l = 0.0, m = -INFINITY;
        for (int c = 0; c < D; ++c) A[c] = 0.0;
        for (int j = 0; j < T; ++j) {
            int valid = N - j * BLK < BLK ? N - j * BLK : BLK;
            double M = -INFINITY;
            for (int s = 0; s < valid; ++s) {
                double dot = 0.0;
                for (int c = 0; c < D; ++c) dot += Qf[(size_t)i * D + c] * Kf[(size_t)(j * BLK + s) * D + c];
                sc[s] = dot * sm_scale;
                if (sc[s] > M) M = sc[s];
            }
            double m_new = m > M ? m : M;
            double alpha = (m == -INFINITY) ? 0.0 : exp(m - m_new);
            double r = 0.0, pv[D];
            for (int c = 0; c < D; ++c) pv[c] = 0.0;
            for (int s = 0; s < valid; ++s) {
                double p = exp(sc[s] - m_new);
                r += p;
                for (int c = 0; c < D; ++c)
                    pv[c] += p * (Vf[(size_t)(j * BLK + s) * D + c] - mu[(size_t)j * D + c]);
            }
            for (int c = 0; c < D; ++c) A[c] = alpha * A[c] + pv[c] + r * mu[(size_t)j * D + c];
            l = alpha * l + r;
            m = m_new;
        }
        for (int c = 0; c < D; ++c) out[(size_t)t * D + c] = A[c] / l;
    }
    free(mu);
}

/* Exact attention in fp64 from the bf16 inputs: O = softmax(Q K^T / sqrt(d)) V (Sec. 3.1),
 * the accuracy reference for the whole low-bit pipeline. RoPE (when rope = 1) is applied in
 * fp64 with fp64 angles, independent of the fp32 tables. Rows are query token indices. */
static void rope_row_f64(double *x, int n, int Ht, int Wd, double theta)
{
    int f, y, w;
    token_pos(n, Ht, Wd, &f, &y, &w);
    for (int i = 0; i < NPAIR; ++i) {
        int axis = pair_axis(i);
        int pos = axis == 0 ? f : (axis == 1 ? y : w);
        int j = i - axis_first_pair(axis);
        double ang = (double)pos * pow(theta, -(2.0 * j) / (double)axis_channels(axis));
        double c = cos(ang), s = sin(ang), x0 = x[2 * i], x1 = x[2 * i + 1];
        x[2 * i] = x0 * c - x1 * s;
        x[2 * i + 1] = x0 * s + x1 * c;
    }
}

void or_ref_attn_head(int N, int F, int Ht, int Wd, int rope, double sm_scale, const uint16_t *Q,
                      const uint16_t *K, const uint16_t *V, int n_rows, const int32_t *rows,
                      double *out)
{
    (void)F;
    double *kf = malloc((size_t)N * D * sizeof(double));
    for (int n = 0; n < N; ++n) {
        for (int c = 0; c < D; ++c) kf[(size_t)n * D + c] = or_bf16_to_f32(K[(size_t)n * D + c]);
        if (rope) rope_row_f64(&kf[(size_t)n * D], n, Ht, Wd, 10000.0);
    }
#pragma omp parallel for schedule(dynamic, 1)
    for (int t = 0; t < n_rows; ++t) {
        int i = rows[t];
        double q[D], o[D];
        double *s = malloc((size_t)N * sizeof(double));
        for (int c = 0; c < D; ++c) q[c] = or_bf16_to_f32(Q[(size_t)i * D + c]);
        if (rope) rope_row_f64(q, i, Ht, Wd, 10000.0);
        double mx = -INFINITY;
        for (int n = 0; n < N; ++n) {
            double dot = 0.0;
            for (int c = 0; c < D; ++c) dot += q[c] * kf[(size_t)n * D + c];
            s[n] = dot * sm_scale;
            if (s[n] > mx) mx = s[n];
        }
        double den = 0.0;
        for (int c = 0; c < D; ++c) o[c] = 0.0;
        for (int n = 0; n < N; ++n) {
            double p = exp(s[n] - mx);
            den += p;
            for (int c = 0; c < D; ++c) o[c] += p * (double)or_bf16_to_f32(V[(size_t)n * D + c]);
        }
        for (int c = 0; c < D; ++c) out[(size_t)t * D + c] = o[c] / den;
        free(s);
    }
    free(kf);
}

/* Apply the rotary embedding (fp32 tables) to every row of one head: exposed so that tests can
 * pin the rotation on its own (norm preservation, relative-position property). */
void or_rope_apply(int N, int F, int Ht, int Wd, const float *cos_t, const float *sin_t, float *x)
{
    for (int n = 0; n < N; ++n) rope_row(&x[(size_t)n * D], n, F, Ht, Wd, cos_t, sin_t);
}

/* ------------------------------------------------------------------------------------------ */
/* Value-guided grouping (Sec. 3.2 "Value-guided permutation")                                */
/* ------------------------------------------------------------------------------------------ */

enum { OR_GROUP_IDENTITY = 0, OR_GROUP_CUBE = 1, OR_GROUP_KMEANS = 2 };

typedef struct {
    int32_t N, F, Ht, Wd;
    int32_t mode, k, iters, warm_start;
    int32_t cube_t, cube_h, cube_w;
} or_group_cfg;

/* Round-half-to-even of num / den for den > 0, in exact integer arithmetic. */
static int32_t div_rne(int64_t num, int64_t den)
{
    int64_t q = num / den, rem = num % den;
    if (rem < 0) { q -= 1; rem += den; }          /* floor division: 0 <= rem < den */
    if (2 * rem > den || (2 * rem == den && (q & 1))) q += 1;
    return (int32_t)q;
}

/* Stable counting sort of labels in [0, nlab): perm lists token indices by label ascending,
 * original index ascending within a label (READING: argsort is taken stable). */
static void stable_sort_labels(int N, const int32_t *z, int nlab, int32_t *perm, int32_t *inv)
{
    int64_t *start = calloc((size_t)nlab + 1, sizeof(int64_t));
    for (int n = 0; n < N; ++n) start[z[n] + 1]++;
    for (int k = 0; k < nlab; ++k) start[k + 1] += start[k];
    for (int n = 0; n < N; ++n) perm[start[z[n]]++] = n;
    if (inv) for (int r = 0; r < N; ++r) inv[perm[r]] = r;
    free(start);
}

/* READING of the online k-means: Lloyd iterations at inference time on per-head INT8 codes of
 * V (scale = amax/127 over the whole head, code = rint(v * 127/amax)), squared-L2 distance
 * evaluated exactly in int32 as |C_k|^2 - 2 x.C_k with ties to the smallest k, centroids
 * updated to the round-half-even integer mean of their members (an empty cluster keeps its
 * centroid). Cold start: centroid k is token floor((2k+1)N/(2K)) (evenly spaced along the grid
 * raster); warm start: the caller's fp32 centroids requantized with this head's scale.
 * Labels are those of the last assignment; returned centroids are code * scale in fp32.
 * CUBE: label = raster index of the (cube_t x cube_h x cube_w) cube holding the token (the
 * static cube order of Sec. 3.2); IDENTITY: label 0. perm = stable sort of labels. */
int or_group_head(const or_group_cfg *cfg, const uint16_t *V, const float *cent_in,
                  int32_t *labels, int32_t *perm, int32_t *inv_perm, float *cent_out)
{
    const int N = cfg->N, K = cfg->k;
    if (cfg->mode == OR_GROUP_IDENTITY) {
        for (int n = 0; n < N; ++n) { labels[n] = 0; perm[n] = n; if (inv_perm) inv_perm[n] = n; }
        return 0;
    }
    if (cfg->mode == OR_GROUP_CUBE) {
        int nh = (cfg->Ht + cfg->cube_h - 1) / cfg->cube_h, nw = (cfg->Wd + cfg->cube_w - 1) / cfg->cube_w;
        int nf = (cfg->F + cfg->cube_t - 1) / cfg->cube_t;
        for (int n = 0; n < N; ++n) {
            int f, y, x;
            token_pos(n, cfg->Ht, cfg->Wd, &f, &y, &x);
            labels[n] = ((f / cfg->cube_t) * nh + y / cfg->cube_h) * nw + x / cfg->cube_w;
        }
        stable_sort_labels(N, labels, nf * nh * nw, perm, inv_perm);
        return 0;
    }
    /* KMEANS */
    int8_t *x = malloc((size_t)N * D);
    int32_t *C = malloc((size_t)K * D * sizeof(int32_t));
    int64_t *S = malloc((size_t)K * D * sizeof(int64_t));
    int64_t *cnt = malloc((size_t)K * sizeof(int64_t));
    int64_t *nrm = malloc((size_t)K * sizeof(int64_t));
    if (!x || !C || !S || !cnt || !nrm) { free(x); free(C); free(S); free(cnt); free(nrm); return -1; }
    float amax = 0.0f;
    for (size_t e = 0; e < (size_t)N * D; ++e) {
        float v = fabsf(or_bf16_to_f32(V[e]));
        if (v > amax) amax = v;
    }
    float scale = amax > 0.0f ? amax / 127.0f : 1.0f;
    float inv = amax > 0.0f ? 127.0f / amax : 0.0f;
    for (size_t e = 0; e < (size_t)N * D; ++e) {
        float q = rintf(or_bf16_to_f32(V[e]) * inv);
        if (q > 127.0f) q = 127.0f;
        if (q < -127.0f) q = -127.0f;
        x[e] = (int8_t)q;
    }
    for (int k = 0; k < K; ++k)
        for (int c = 0; c < D; ++c) {
            if (cfg->warm_start) {
                float q = rintf(cent_in[(size_t)k * D + c] * inv);
                if (q > 127.0f) q = 127.0f;
                if (q < -127.0f) q = -127.0f;
                C[(size_t)k * D + c] = (int32_t)q;
            } else {
                int64_t n0 = ((int64_t)(2 * k + 1) * N) / (2 * (int64_t)K);
                C[(size_t)k * D + c] = x[(size_t)n0 * D + c];
            }
        }
    for (int it = 0; it < cfg->iters; ++it) {
        for (int k = 0; k < K; ++k) {
            int64_t s = 0;
            for (int c = 0; c < D; ++c) s += (int64_t)C[(size_t)k * D + c] * C[(size_t)k * D + c];
            nrm[k] = s;
        }
        for (int n = 0; n < N; ++n) {
            int best = 0;
            int64_t bd = 0;
            for (int k = 0; k < K; ++k) {
                int64_t dot = 0;
                for (int c = 0; c < D; ++c) dot += (int64_t)x[(size_t)n * D + c] * C[(size_t)k * D + c];
                int64_t dist = nrm[k] - 2 * dot;
                if (k == 0 || dist < bd) { bd = dist; best = k; }
            }
            labels[n] = best;
        }
        memset(S, 0, (size_t)K * D * sizeof(int64_t));
        memset(cnt, 0, (size_t)K * sizeof(int64_t));
        for (int n = 0; n < N; ++n) {
            cnt[labels[n]]++;
            for (int c = 0; c < D; ++c) S[(size_t)labels[n] * D + c] += x[(size_t)n * D + c];
        }
        for (int k = 0; k < K; ++k)
            if (cnt[k] > 0)
                for (int c = 0; c < D; ++c) C[(size_t)k * D + c] = div_rne(S[(size_t)k * D + c], cnt[k]);
    }
    if (cfg->iters == 0)                     /* no Lloyd round: labels from one assignment */
        for (int n = 0; n < N; ++n) {
            int best = 0;
            int64_t bd = 0;
            for (int k = 0; k < K; ++k) {
                int64_t dot = 0, nk = 0;
                for (int c = 0; c < D; ++c) {
                    dot += (int64_t)x[(size_t)n * D + c] * C[(size_t)k * D + c];
                    nk += (int64_t)C[(size_t)k * D + c] * C[(size_t)k * D + c];
                }
                int64_t dist = nk - 2 * dot;
                if (k == 0 || dist < bd) { bd = dist; best = k; }
            }
            labels[n] = best;
        }
    if (cent_out)
        for (int k = 0; k < K; ++k)
            for (int c = 0; c < D; ++c) cent_out[(size_t)k * D + c] = (float)C[(size_t)k * D + c] * scale;
    stable_sort_labels(N, labels, K, perm, inv_perm);
    free(x); free(C); free(S); free(cnt); free(nrm);
    return 0;
}

/* Per-head INT8 view of V used by the grouping (exposed so tests can brute-force assignments). */
void or_group_codes(int N, const uint16_t *V, int8_t *x, float *scale_out)
{
    float amax = 0.0f;
    for (size_t e = 0; e < (size_t)N * D; ++e) {
        float v = fabsf(or_bf16_to_f32(V[e]));
        if (v > amax) amax = v;
    }
    float inv = amax > 0.0f ? 127.0f / amax : 0.0f;
    *scale_out = amax > 0.0f ? amax / 127.0f : 1.0f;
    for (size_t e = 0; e < (size_t)N * D; ++e) {
        float q = rintf(or_bf16_to_f32(V[e]) * inv);
        if (q > 127.0f) q = 127.0f;
        if (q < -127.0f) q = -127.0f;
        x[e] = (int8_t)q;
    }
}

/* ------------------------------------------------------------------------------------------ */
/* Batched entry points: loop over (batch, head), heads in parallel                           */
/* ------------------------------------------------------------------------------------------ */

int or_prep(int BH, const or_prep_cfg *cfg, const uint16_t *Q, const uint16_t *K, const uint16_t *V,
            const int32_t *perm, const int32_t *q_perm, const float *cos_t, const float *sin_t,
            int8_t *q_codes, float *q_scale, int8_t *k_codes, float *k_scale, float *k_mean,
            uint8_t *v_codes, float *v_scale, uint16_t *v_mean,
            uint8_t *q_mx, uint8_t *q_mxs, uint8_t *k_mx, uint8_t *k_mxs)
{
    const size_t N = (size_t)cfg->N, T = (N + BLK - 1) / BLK, Np = T * BLK;
    const int mx = cfg->qk_fmt == OR_QK_MXFP4;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad)
    for (int h = 0; h < BH; ++h) {
        int rc = or_prep_head(cfg, Q + h * N * D, K + h * N * D, V + h * N * D,
                              perm ? perm + h * N : NULL, q_perm ? q_perm + h * N : NULL, cos_t, sin_t,
                              q_codes + h * Np * D, q_scale + h * T, k_codes + h * Np * D, k_scale + h * T,
                              k_mean + h * D, v_codes + h * Np * D, v_scale + h * D, v_mean + h * T * D,
                              mx ? q_mx + h * Np * D : NULL, mx ? q_mxs + h * Np * 4 : NULL,
                              mx ? k_mx + h * Np * D : NULL, mx ? k_mxs + h * Np * 4 : NULL);
        bad |= (rc != 0);
    }
    return bad ? -1 : 0;
}

int or_group(int BH, const or_group_cfg *cfg, const uint16_t *V, const float *cent_in, int32_t *labels,
             int32_t *perm, int32_t *inv_perm, float *cent_out)
{
    const size_t N = (size_t)cfg->N, K = (size_t)(cfg->k > 0 ? cfg->k : 1);
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad)
    for (int h = 0; h < BH; ++h) {
        int rc = or_group_head(cfg, V + h * N * D, cent_in ? cent_in + h * K * D : NULL, labels + h * N,
                               perm + h * N, inv_perm ? inv_perm + h * N : NULL,
                               cent_out ? cent_out + h * K * D : NULL);
        bad |= (rc != 0);
    }
    return bad ? -1 : 0;
}

/* Elementwise helpers over arrays (for tests). */
void or_e4m3_encode_array(int n, const float *x, uint8_t *out)
{
    for (int i = 0; i < n; ++i) out[i] = or_e4m3_encode(x[i]);
}
void or_fp4_encode_array(int n, const float *x, uint8_t *out)
{
    for (int i = 0; i < n; ++i) out[i] = or_fp4_encode(x[i]);
}
void or_mx_blocks(int n_blocks, const float *x, uint8_t *codes, uint8_t *scales)
{
    for (int b = 0; b < n_blocks; ++b) or_mx_block(&x[32 * b], &codes[32 * b], &scales[b]);
}
void or_e4m3_decode_array(int n, const uint8_t *b, double *out)
{
    for (int i = 0; i < n; ++i) out[i] = or_e4m3_decode(b[i]);
}
void or_expcast_u_array(int n, const float *u, float beta, int32_t *out)
{
    for (int i = 0; i < n; ++i) out[i] = or_expcast_code_u(u[i], beta);
}
void or_fwht_rows(int n, float *x)
{
    for (int i = 0; i < n; ++i) or_fwht128(&x[(size_t)i * D]);
}
void or_bf16_round_array(int n, const float *x, uint16_t *out)
{
    for (int i = 0; i < n; ++i) out[i] = or_f32_to_bf16(x[i]);
}
