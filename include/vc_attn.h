/*
 * vc_attn.h -- C ABI of the MI355X (gfx950) 8-bit VC-Attention forward.
 *
 * The method (VC-Attention, "Value Smoothing and Softmax Casting for Low-bit Attention"):
 *   - V-Smooth (Sec. 3.2): per (batch, head), group the value tokens by k-means, sort K and V
 *     rows by cluster (Q keeps its order, eq. kv-reordering), subtract one bf16 mean per block
 *     of 128 permuted rows (eq. block-demeaning) and quantize only the residual to E4M3 with a
 *     per-channel scale; the mean is restored inside the online softmax (eq. vc-online-update).
 *   - ExpCast-FP8 (Sec. 3.3): the E4M3 byte of every probability is written directly by one
 *     fused multiply-add of its log2-domain score, clip(RNE(8(u+8) + 56 + beta), 0, 120)
 *     (eq. direct-fp8), instead of an fp32 exponential followed by a cast.
 *   - Fused preprocessing (Sec. 3.4, Appendix B): RoPE, key centering, the gather by the
 *     permutation, the Q/K Hadamard rotation, block means and the quantizers are fused into
 *     the passes that produce the low-bit operands.
 *
 * Problem statement (Sec. 3.1): non-causal self-attention O = softmax(Q K^T / sqrt(d)) V over N
 * tokens flattened from a frames x rows x cols latent grid, n = (f * Ht + y) * Wd + x, head
 * dimension d = 128, with low-bit operands X_q = s_X * X_hat.
 *
 * Conventions for every entry point:
 *   - Tensor arguments are DEVICE pointers to contiguous memory, 16-byte aligned, owned by the
 *     caller. The library allocates nothing per call and keeps no device state between calls;
 *     the grouping state reused across calls (permutation, centroids) lives in caller buffers.
 *   - `stream` is a hipStream_t passed as void* (NULL: the default stream). All work is
 *     enqueued asynchronously on it; no entry point synchronizes the device.
 *   - Arguments are validated on the host before anything is enqueued. On any error nothing is
 *     launched and a vc_status other than VC_OK is returned. VC_ERR_HIP means a launch failed;
 *     vc_last_hip_error() then returns the hipError_t (thread-local). Faults inside kernels
 *     surface at the caller's next synchronization of the stream.
 *   - Permutation arguments must hold a permutation of [0, N) per (batch, head). Kernels clamp
 *     out-of-range entries into [0, N) (memory-safe), but the result is then unspecified.
 *   - Entry points are reentrant: concurrent calls are safe on distinct buffers.
 *
 * Tensor shapes use T = ceil(N / 128) blocks and Np = 128 T padded rows.
 */
#ifndef VC_ATTN_H
#define VC_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    VC_OK = 0,
    VC_ERR_NULL = 1,        /* a required pointer is NULL */
    VC_ERR_SHAPE = 2,       /* d != 128, N != F*Ht*Wd, a non-positive size, or sizes too large */
    VC_ERR_UNSUPPORTED = 3, /* an option value outside the documented set */
    VC_ERR_WORKSPACE = 4,   /* workspace NULL or smaller than vc_attn_workspace_size() */
    VC_ERR_ALIGN = 5,       /* a tensor pointer not 16-byte aligned */
    VC_ERR_HIP = 6,         /* a HIP launch or runtime call failed (see vc_last_hip_error) */
    VC_ERR_INTERNAL = 7
} vc_status;

/* Problem shape. Requires d == 128, N == F * Ht * Wd, B, H, N >= 1, B * H * Np * 128 < 2^31. */
typedef struct {
    int32_t B, H, N, d;
    int32_t F, Ht, Wd;      /* latent grid: frames, rows, cols */
} vc_shape;

enum { VC_QK_INT8 = 0,      /* per-128-row-block symmetric INT8 Q and K */
       VC_QK_FP8 = 1,       /* per-128-row-block symmetric OCP E4M3 Q and K (Sec. 4.5) */
       VC_QK_MXFP4 = 2 };   /* OCP MX FP4 (E2M1) Q and K, one E8M0 scale per 32 channels of a row */
enum { VC_P_EXPCAST = 0, VC_P_EXP_THEN_CAST = 1 };

/* Options of the low-bit path.
 *   qk_fmt   : VC_QK_INT8 (the method's 8-bit path), VC_QK_FP8 (Q and K as E4M3 codes per 128-row
 *              block, scale amax/448, nearest-even, codes of zero magnitude stored as +0: the
 *              configuration of Sec. 4.5 for matrix units without INT8; the scores come out of
 *              the FP8 matrix product in fp32) or VC_QK_MXFP4 (the 4-bit variant: Q and K
 *              quantized after the Hadamard rotation by 32-channel blocks, shared exponent
 *              floor(log2(amax)) - 2, elements rounded to the nearest E2M1 value with ties to the
 *              even code and saturation at 6; the scores come out of the scaled FP4 matrix
 *              product in fp32; P and V stay 8-bit).
 *   p_mode   : VC_P_EXPCAST (ExpCast-FP8, eq. direct-fp8) or VC_P_EXP_THEN_CAST (fp32 exp2,
 *              scale by 2^8, E4M3 round-to-nearest-even cast: the conventional path).
 *   rope     : 1 = apply the 3-axis rotary embedding in the preprocessing (pairs 0..21 turn with
 *              the frame, 22..42 with the row, 43..63 with the column; tables below);
 *              0 = inputs are already rotated.
 *   hadamard : 1 = rotate Q and K rows by the 128-point Sylvester Hadamard matrix (unnormalised;
 *              the 1/128 enters the score scale).
 *   smooth_k : 1 = subtract the key channel mean (over the N tokens) before quantizing K.
 *   smooth_v : 1 = V-Smooth block demeaning (means restored in the attention kernel);
 *              0 = plain per-channel E4M3 V.
 *   sm_scale : softmax scale, >= 0 with sm_scale * log2(e) finite in fp32 (VC_ERR_UNSUPPORTED
 *              otherwise); 0 selects 1/sqrt(d).
 *   beta     : ExpCast-FP8 centring constant (the method uses -0.35), -1 <= beta <= 0
 *              (VC_ERR_UNSUPPORTED otherwise). Sec. 3.3 derives the shift from the rounding
 *              error range [-0.689, 0]; inside [-1, 0] the row maximum's code stays in
 *              [119, 120], so no code overflows the clip of eq. direct-fp8 and no row sum is 0.
 * Each flag must be 0 or 1. */
typedef struct {
    int32_t qk_fmt;
    int32_t p_mode;
    int32_t rope, hadamard, smooth_k, smooth_v;
    float sm_scale;
    float beta;
} vc_opts;

enum { VC_GROUP_IDENTITY = 0, VC_GROUP_CUBE = 1, VC_GROUP_KMEANS = 2 };

/* Grouping options (Sec. 3.2 "Value-guided permutation").
 *   mode       : VC_GROUP_IDENTITY (perm = 0..N-1), VC_GROUP_CUBE (static cubes of cube[0]
 *                frames x cube[1] rows x cube[2] cols in raster order, tokens in raster order
 *                inside a cube), VC_GROUP_KMEANS (Lloyd k-means on per-head INT8 codes of V,
 *                squared-L2, ties to the smallest cluster; labels sorted stably).
 *   k          : clusters, 1 <= k <= min(N, 64) (VC_ERR_UNSUPPORTED otherwise).
 *   iters      : Lloyd rounds (assign + update), 0 <= iters <= 64.
 *   warm_start : 1 = initialise from `centroids` (value units, previous call's output);
 *                0 = centroid c starts at token floor((2c+1) N / (2k)).
 *   cube       : cube extents for VC_GROUP_CUBE, each >= 1. */
typedef struct {
    int32_t mode, k, iters, warm_start;
    int32_t cube[3];
} vc_group_opts;

/* Low-bit operands written by vc_attn_prep and read by vc_attn_forward (caller-owned device
 * buffers). Physical layouts of the code tensors are tiled for the matrix instructions:
 *
 *   q, k : int8, B*H*Np*128 bytes. Per (b, h) and 128-row block j, the 16384 bytes of the block
 *          are ordered [rb 4][dc 4][dh 2][r 32][e 16]: byte (row, ch) of the block, with
 *          rb = row/32, r = row%32, dc = ch/32, dh = (ch%32)/16, e = ch%16, sits at
 *          ((rb*4 + dc)*2 + dh)*512 + r*16 + e. q rows are in query order (q_perm order when a
 *          q_perm is given); k rows in permuted order K' = K[perm]. Padded rows hold 0.
 *   q_scale, k_scale : fp32 [B, H, T], one scale per 128-row block (code * scale = value).
 *   With qk_fmt = VC_QK_FP8 instead:
 *   q, k : E4M3 bytes, B*H*Np*128 bytes. Per (b, h) and 128-row block j, the 16384 bytes are
 *          ordered [rb 4][m 2][h 2][half 2][r 32][e 16]: byte (row, ch) sits at
 *          ((((rb*2 + m)*2 + h)*2 + half)*32 + r)*16 + e with rb = row/32, r = row%32, m = ch/64,
 *          h = (ch%64)/32, half = (ch%32)/16, e = ch%16 (lane h*32 + r of the FP8 32x32x64
 *          product holds channels 64m + 32h .. + 31 of one row as two 16-byte halves).
 *          q_scale, k_scale as for INT8 (amax/448).
 *   With qk_fmt = VC_QK_MXFP4 instead:
 *   q, k : packed E2M1 codes, B*H*Np*64 bytes. Per (b, h) and 128-row block j, the 8192 bytes are
 *          ordered [rb 4][m 2][h 2][r 32][16 bytes]: channel ch of row `row` is the nibble
 *          ch % 2 (0 = low) of byte ((rb*2 + m)*2 + h)*512 + r*16 + (ch % 32)/2 with rb = row/32,
 *          r = row%32, m = ch/64, h = (ch%64)/32 (lane h*32 + r of the scaled matrix product
 *          holds one 32-channel block of one row). Padded rows hold 0.
 *   q_mx_scale, k_mx_scale : E8M0 bytes (value 2^(byte - 127)), B*H*Np*4 bytes. Per (b, h) and
 *          block j, the 512 bytes are ordered [lane 64][rb 4][m 2]: the scale of row 32*rb + r,
 *          channels 64*m + 32*h .. + 31 sits at (h*32 + r)*8 + rb*2 + m. Padded rows hold 127.
 *   q_scale, k_scale are not used.
 *   k_mean : fp32 [B, H, 128], the key channel mean subtracted before quantizing (0 if off).
 *   v    : E4M3 (OCP e4m3fn) bytes of the demeaned residual, B*H*Np*128 bytes, permuted order.
 *          Per (b, h) and 128-row block, ordered [kc 2][db 4][kh 2][sh 2][c 32][t 16]: with
 *          db = ch/32, c = ch%32 and w = key%32, the byte of key row `key` and channel ch sits
 *          at ((((kc*4 + db)*2 + kh)*2 + sh)*32 + c)*16 + t where 2*kc + sh = key/32,
 *          kh = (w%8)/4 and t = 4*(w/8) + w%4 (channel-major 16-key groups, the order in which
 *          the attention kernel's probability registers hold the keys). Padded rows hold 0.
 *   v_scale: fp32 [B, H, 128], per-channel residual scale (code * scale = residual value).
 *   v_mean : bf16 bits [B, H, T, 128], the block means mu_j subtracted (0 if smooth_v = 0).
 */
typedef struct {
    int8_t *q;
    float *q_scale;
    int8_t *k;
    float *k_scale;
    float *k_mean;
    uint8_t *v;
    float *v_scale;
    uint16_t *v_mean;
    uint8_t *q_mx_scale;   /* VC_QK_MXFP4 only (may be NULL otherwise) */
    uint8_t *k_mx_scale;
} vc_prepped;

/* Fill *o with the method's defaults: INT8 QK, ExpCast-FP8, RoPE, Hadamard, key centering and
 * V-Smooth on, sm_scale 0 (1/sqrt(d)), beta -0.35. */
void vc_opts_default(vc_opts *o);

/* Fill *g with: KMEANS, k = 32, iters = 8, cold start, cube {4, 2, 16}. */
void vc_group_opts_default(vc_group_opts *g);

/* Bytes of device workspace needed by vc_attn_prep / vc_attn_group for this shape and options
 * (the larger of the two). Returns 0 if the shape or options are invalid. */
size_t vc_attn_workspace_size(const vc_shape *shape, const vc_opts *opts, const vc_group_opts *gopts);

/* HOST helper: rotary tables, written to host arrays cos_t/sin_t of (F + Ht + Wd) x 64 fp32.
 * Row r < F is frame r, F <= r < F+Ht grid row r-F, then grid column r-F-Ht. Column i holds the
 * cos/sin of pair i's angle pos * theta^(-2j/d_a) (j = i minus the axis' first pair; d_a = 44
 * for frames, 42 for rows and columns) when pair i belongs to that row's axis, else 1 / 0.
 * Angles are evaluated in fp64 and rounded once to fp32. Copy the tables to the device for
 * vc_attn_prep. Returns VC_ERR_NULL on NULL tables, VC_ERR_SHAPE for a non-positive extent, a
 * theta that is not finite and positive, or F + Ht + Wd >= 2^25 (the entry count must fit int). */
vc_status vc_rope_tables(int32_t F, int32_t Ht, int32_t Wd, double theta, float *cos_t, float *sin_t);

/* Value-guided grouping (Sec. 3.2, "Value-guided permutation"; grouping schedule Sec. 3.4).
 *   V         : bf16 bits [B, H, N, 128] (token order).
 *   centroids : fp32 [B, H, k, 128], value units. Read when warm_start = 1; always written
 *               (KMEANS) with the final centroids. May be NULL for IDENTITY / CUBE.
 *   labels    : int32 [B, H, N] cluster (KMEANS: of the last assignment; CUBE: cube index;
 *               IDENTITY: 0).
 *   perm      : int32 [B, H, N], perm[r] = token placed at row r (stable sort of labels).
 *   inv_perm  : int32 [B, H, N] or NULL; inv_perm[perm[r]] = r.
 *   ws        : device workspace of ws_bytes >= vc_attn_workspace_size(shape, NULL, gopts). */
vc_status vc_attn_group(const vc_shape *shape, const vc_group_opts *gopts, const uint16_t *V,
                        float *centroids, int32_t *labels, int32_t *perm, int32_t *inv_perm,
                        void *ws, size_t ws_bytes, void *stream);

/* Fused preprocessing (Sec. 3.4 and Appendix B): Q, K, V bf16 bits [B, H, N, 128] in token
 * order -> the low-bit operands in *out (layouts above).
 *   perm   : int32 [B, H, N] K/V gather (K' = K[perm], V' = V[perm]); NULL = identity.
 *   q_perm : int32 [B, H, N] optional query gather; NULL = query order (the method's case).
 *   rope_cos, rope_sin : device fp32 tables from vc_rope_tables (read only when opts->rope).
 *   ws     : device workspace of ws_bytes >= vc_attn_workspace_size(shape, opts, NULL).
 * Q is rotated at each token's own position, Hadamard-rotated and quantized per 128-row block;
 * K is rotated, centred by its channel mean, gathered, rotated by H and quantized per block; V
 * is gathered, demeaned per block (bf16 means) and quantized per channel to E4M3. */
vc_status vc_attn_prep(const vc_shape *shape, const vc_opts *opts, const uint16_t *Q,
                       const uint16_t *K, const uint16_t *V, const int32_t *perm,
                       const int32_t *q_perm, const float *rope_cos, const float *rope_sin,
                       const vc_prepped *out, void *ws, size_t ws_bytes, void *stream);

/* vc_attn_prep for callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation): the same kernels and results, with the
 * preprocessing workspace taken from a static device array of 32 MiB that the library holds on
 * each GPU it runs on until the process ends, instead of a caller buffer. The call itself allocates
 * nothing (no hipMalloc, no allocating library routine); the first call on a GPU looks up that
 * GPU's copy of the array. Arguments and errors as vc_attn_prep, without ws / ws_bytes; shapes
 * whose preprocessing workspace, vc_attn_workspace_size(shape, opts, NULL), exceeds 32 MiB
 * (33554432 bytes; B * H * ceil(N / 128) up to about 32000) return VC_ERR_WORKSPACE. Every call on
 * a GPU shares that GPU's array: calls that overlap in time on one GPU (different streams, or
 * different threads) race and must be serialized by the caller. */
vc_status vc_attn_prep_noalloc(const vc_shape *shape, const vc_opts *opts, const uint16_t *Q,
                               const uint16_t *K, const uint16_t *V, const int32_t *perm,
                               const int32_t *q_perm, const float *rope_cos, const float *rope_sin,
                               const vc_prepped *out, void *stream);

/* Attention kernel (Sec. 3.1 eq. tiled-low-bit-attention with Sec. 3.2 eq. vc-online-update and
 * Sec. 3.3 eq. direct-fp8): INT8 Q K'^T on the matrix cores, running row maximum per 128-key
 * tile (tiles in ascending order), 8-bit P (ExpCast-FP8 or exp-then-cast), FP8 P R_hat on the
 * matrix cores, block means restored through the probability row sum, O = A * s_V / l.
 *   in     : operands written by vc_attn_prep with the same shape and opts.
 *   q_perm : the q_perm given to vc_attn_prep (output row i is written to token q_perm[i]);
 *            NULL = query order.
 *   O      : bf16 bits [B, H, N, 128], token order.
 * Domain: with p_mode = VC_P_EXPCAST, a query row whose running maximum score in log2 units
 * (sm_scale * log2(e) * q.k of the quantized operands) reaches 2^27 in magnitude, i.e. softmax
 * logits beyond about 9.3e7, is outside the supported domain: its output row is written as NaN.
 * Every other row is the method's result (codes exactly those of eq. direct-fp8). */
vc_status vc_attn_forward(const vc_shape *shape, const vc_opts *opts, const vc_prepped *in,
                          const int32_t *q_perm, uint16_t *O, void *stream);

/* vc_attn_forward that also writes the 8-bit probability codes it forms (Sec. 3.3 eq.
 * direct-fp8 in ExpCast mode, the FP8 cast of the exponentials otherwise), for debugging and
 * parity checks; it waits for every tile copy in flight before each tile, so copies no longer
 * overlap the computation.
 *   p_codes       : device uint8 [B, H, N, 128 T] (T = ceil(N / 128)), 16-byte aligned,
 *                   caller-owned, fully overwritten. Row i is the prepared query i (before q_perm);
 *                   byte 128 t + s is key s of tile t of the prepared K', coded at the running
 *                   maximum after tile t; keys past N are 0.
 *   p_codes_bytes : size of the p_codes buffer; VC_ERR_WORKSPACE if below B*H*N*128*T.
 * Other arguments and errors as vc_attn_forward; VC_ERR_NULL if p_codes is NULL. */
vc_status vc_attn_forward_codes(const vc_shape *shape, const vc_opts *opts, const vc_prepped *in,
                                const int32_t *q_perm, uint16_t *O, uint8_t *p_codes,
                                size_t p_codes_bytes, void *stream);

/* The FP8 score product of the attention kernel (qk_fmt = VC_QK_FP8, Sec. 4.5), on caller data,
 * for checking its accumulation error: the kernel forms each 32 keys x 32 queries block of scores
 * with two chained E4M3 32x32x64 matrix instructions (channels 0..63, then 64..127, the first
 * result as the second's accumulator input), and this entry point runs that same instruction
 * sequence from the accumulator c_in:
 *   out[b][i][j] = c_in[b][i][j] + sum_{c < 128} e4m3(a[b][i][c]) * e4m3(bm[b][j][c]),
 * summed as the matrix unit sums (not an exact fp32 sum once the products span many binades).
 *   a, bm : device uint8 [n][32][128], E4M3 (OCP e4m3fn) bytes, row-major.
 *   c_in  : device fp32 [n][32][32], the accumulator input (zeros reproduce the kernel's scores).
 *   out   : device fp32 [n][32][32].
 * n >= 1 blocks (VC_ERR_SHAPE otherwise); the usual NULL / alignment checks. Not on the
 * attention path: it exists so that the error bound assumed for FP8 scores can be measured. */
vc_status vc_fp8_score_product(const uint8_t *a, const uint8_t *bm, const float *c_in, float *out, int32_t n,
                               void *stream);

/* Static description of a status code. */
const char *vc_status_str(vc_status s);

/* hipError_t behind the last VC_ERR_HIP returned on this thread (0 if none). */
int vc_last_hip_error(void);

#ifdef __cplusplus
}
#endif

#endif /* VC_ATTN_H */
