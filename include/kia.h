/*
 * kia.h -- C ABI of the MI355X (gfx950) K-interval attention library.
 *
 * The operator (Zhu, Hu, Kozlowski, "Pretraining Transformers with Quantized
 * Softmax in Attention"): causal scaled-dot-product attention whose
 * exponential is rebuilt from K+1 grid values e^{b_r} (Sec. 3, App. A).
 *   S = Q K^T / sqrt(d) in fp32; per row M = max s, m = min s over the valid
 *   keys; calibration MinMax (h = (M-m)/K, b_r = (1-r/K)(m-M)) or FWM
 *   (h = tau/K, b_r = -tau + r h, zero weight for s - M < -tau);
 *   reconstruction LERP (w^L = (1-t) e^{b_r} + t e^{b_{r+1}}) or Nearest
 *   (w^N = e^{b_l}, l = r + 1[t >= 1/2]); P = w / sum w; O = P V.
 *   Backward (App. B): the surrogate of Eq. (wste) or Eq. (pste), the LERP
 *   slope Delta, and (per the gradient mode) the calibration terms of
 *   Eq. (calgrad) and Eq. (full) on the argmax/argmin keys (ties split
 *   evenly).
 *
 * Conventions for every entry point:
 *   - Tensors are contiguous row-major [B, H, T, d] device buffers owned by
 *     the caller; pointers must be 16-byte aligned, `stats` 256-byte aligned.
 *   - d in {16, 32, 64, 128}; 1 <= K <= 64; B, H, T >= 1, T <= 65536,
 *     B*H*T*d < 2^31, and the statistics (see kia_stats_bytes_bf16o, about
 *     4*B*H*T^2 bytes causal and 8*B*H*T^2 otherwise for the two tile
 *     fields) at most KIA_MAX_STATS_BYTES (else KIA_ERR_SHAPE, also from
 *     kia_stats_bytes). The softmax scale is fixed to fl32(1/sqrt(d)) and a
 *     score is fl32(fl32(q.k) * scale) (the fp32 scores of App. A).
 *   - Determinism: the forward is bitwise repeatable. By default the
 *     backward is not: the row sums of every key block's score gradients
 *     (S_self, and cM under MinMax) are accumulated with float atomics, and
 *     so are the calibration terms and tie splits scattered onto the
 *     argmax/argmin keys of dK, so dQ and dK can differ in their last bits
 *     from run to run (within fp32 rounding); dV is repeatable unless a
 *     small grid is split (KIA_GRID_*). kia_set_deterministic(1) makes
 *     every backward reduction run in a fixed order, so that the backward
 *     too is bitwise repeatable.
 *   - calib: 0 MinMax, 1 FWM, 2 resolved (FWM and resolved need a finite
 *     tau > 0; tau ignored for MinMax).
 *     recon: 0 LERP, 1 Nearest (2-4: exponential weight functions, see
 *     KIA_RECON_SOFTMAX). ste: 0 Weight-STE (Eq. wste), 1 Prob-STE
 *     (Eq. pste); irrelevant for LERP. detach: the gradient mode (KIA_GRAD_*):
 *     0 full calibration gradient (Eq. full), 1 extrema detached (App. B,
 *     Detach), 2 max_only / 3 min_only: the self term plus the maximum's
 *     (resp. minimum's) channel only (appendix on the detached-gradient
 *     record, single-channel ablation; FWM has no minimum channel, so 2 is
 *     full and 3 is detach there), 4 detached with the P1 projection of
 *     each row onto the zero-sum subspace (its mean over the row's valid
 *     keys subtracted; App. B, Detach); the forward also takes 5,
 *     KIA_GRAD_NONE (no backward follows). causal: 1 key j is valid for query
 *     i iff j <= i; 0 every key is valid.
 *   - Index decisions (interval r, level l, FWM tail, the degenerate test
 *     M - m <= 1e-12) follow, on the fp32 scores, the fp64 expressions
 *       MinMax: u = (K * (s - m)) / (M - m)   FWM: a = (s - M) + tau,
 *               tail <=> a < 0, u = (K * a) / tau
 *     r = min(floor(u), K-1), t = u - r, l = r + 1[t >= 1/2].
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = default stream);
 *     nothing synchronizes, allocates or frees. All argument checks run on
 *     the host before any launch: a nonzero return means nothing was
 *     enqueued (except KIA_ERR_HIP, a launch failure).
 *   - Return 0 on success or a negative KIA_ERR_* code; kia_strerror names it.
 *   - Process-wide state: the launch-shape policy and the timing hook (set
 *     only by their own calls), a per-device cache of the CU count, and the
 *     per-device address of kia_attn_fwd_bwd_static's array. Apart from
 *     these, the entry points keep no state between calls, and calls on
 *     different streams and buffers may run concurrently.
 */
#ifndef KIA_H
#define KIA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KIA_OK 0
#define KIA_ERR_NULL (-1)    /* a required pointer is NULL */
#define KIA_ERR_SHAPE (-2)   /* B, H or T < 1, T > 65536, or size overflow */
#define KIA_MAX_STATS_BYTES (1ull << 37) /* 128 GiB: under half of one GPU's HBM */
#define KIA_ERR_HEADDIM (-3) /* d not in {16, 32, 64, 128} */
#define KIA_ERR_K (-4)       /* K not in [1, 64] */
#define KIA_ERR_ENUM (-5)    /* calib/recon/ste/detach (mode)/causal out of range */
#define KIA_ERR_TAU (-6)     /* FWM/resolved with tau <= 0 or not finite */
#define KIA_ERR_ALIGN (-7)   /* tensor not 16-byte or stats not 256-byte aligned */
#define KIA_ERR_HIP (-8)     /* HIP launch/runtime error */
#define KIA_ERR_SCRATCH (-9) /* statistics larger than KIA_STATIC_BYTES */

#define KIA_CALIB_MINMAX 0
#define KIA_CALIB_FWM 1
/* The tail-policy diagnostic "resolved" (appendix on the tail policy in the
 * MinMax -> FWM change): FWM's step h = tau/K and origin b_0 = -tau, the grid
 * continued below -tau with negative intervals (b_r = -tau + r h, r any
 * integer <= K-1), so no key is zeroed: u = (K * ((s - M) + tau)) / tau,
 * r = min(floor(u), K-1), t = u - r, l = r + 1[t >= 1/2]. Backward as FWM
 * (only the maximum's channel). Index decisions are exact while
 * |u| < 2^22 ((M - m) K / tau below about 4e6). Statistics also hold m, amin
 * and nmin. Debug codes: bit 15 valid, bit 14 l = r + 1, bits 0-13 r in
 * two's complement (clamped to -8192). */
#define KIA_CALIB_RESOLVED 2
#define KIA_RECON_LERP 0
#define KIA_RECON_NEAREST 1
/* Exponential weight functions of the baselines the paper compares with
 * (the same two passes, no grid; K, calib, tau and ste are not used and not
 * checked, and the bf16-input entry points reject them with KIA_ERR_ENUM):
 *   z = fl32(s - M) per valid key (M the row maximum);
 *   SOFTMAX (App. A, Softmax): w = e^z;
 *   BF16EXP (App. D, BF16-exp): w = bf16(e^{bf16(z)}) with both roundings
 *     to nearest even; backward through the casts and the bf16 exponential,
 *     dz = bf16(bf16(dL/dw) w);
 *   FP8EXP (App. D, FP8-rounded exp): w^exp = fl32(e^z), w = e4m3(w^exp)
 *     (float8_e4m3fn, nearest even; values below 2^-10 become 0); backward
 *     through the rounding as the identity with the fp32 exponential's
 *     derivative, dz = dL/dw w^exp.
 *   The exponential inside a rounding is the correctly rounded fp32 value
 *   (an fp64 exponential decides keys near a rounding midpoint).
 *   dL/dw_j = (g_j - <g>_P) / W; dS = dz plus, under the gradient modes
 *   that keep the maximum's channel (full, max_only), -sum_j dz_j on the
 *   argmax keys (split over ties): M stays on the gradient path of z.
 *   detach and min_only drop it, P1 projects the detached row. Statistics:
 *   M, amax, nmax, W (= WL) as for FWM; U holds the fp32 exponential. */
#define KIA_RECON_SOFTMAX 2
#define KIA_RECON_BF16EXP 3
#define KIA_RECON_FP8EXP 4
#define KIA_STE_WEIGHT 0
#define KIA_STE_PROB 1
#define KIA_GRAD_FULL 0
#define KIA_GRAD_DETACH 1
#define KIA_GRAD_MAX_ONLY 2
#define KIA_GRAD_MIN_ONLY 3
#define KIA_GRAD_DETACH_P1 4
/* Forward only (the forward's gradient mode when no backward will read its
 * stats, e.g. an evaluation or inference pass): the forward leaves out what
 * only the backward reads, O^L = P^L V of Prob-STE with Nearest (a third of
 * that forward's matrix work) and, on the fp32 entry points, the per-key
 * decisions its second pass would store in U. O and every per-row statistic
 * are the same as under the other modes. The backward entry points and
 * kia_attn_fwd_bwd_static reject it (KIA_ERR_ENUM, nothing enqueued); a
 * backward or kia_debug_codes_stored on stats that such a forward filled is
 * undefined (the Python binding refuses both). */
#define KIA_GRAD_NONE 5

/*
 * Per-row statistics kept from the forward for the backward (the row state
 * of App. A: extrema, tie sets, normalizers; App. B: O^L for Prob-STE).
 * `stats` is one caller-allocated device buffer of kia_stats_bytes() bytes,
 * a struct of arrays with R = B*H*T entries each, in this order:
 *   M (f32), m (f32), W (f32: the forward normalizer, W^N for Nearest and
 *   W^L for LERP), WL (f32: W^L), amax (i32: first argmax key), amin (i32:
 *   first argmin key), nmax (i32: number of keys equal to M), nmin (i32),
 *   then the backward's scratch: a 16-float record per row, and two f32 row
 *   sums; O^L = P^L V (f32, [R, d]; written for Nearest with Prob-STE only,
 *   present for every operator so that no offset depends on recon or ste);
 *   then the
 *   backward's dS scratch: B*H*n tiles of 32x32 f32 (4 KiB each) with
 *   n = q(q+1)/2 for causal and q*q otherwise, q = ceil(T/32) (about
 *   2*B*H*T^2 bytes causal, 4*B*H*T^2 otherwise); then U, tiles of the same
 *   shape and count: the forward's fp32 scores Q K^T of every (query, key)
 *   pair that its extrema pass computed, replaced by its second pass with
 *   the decided grid position u of the pair (the value the index decisions
 *   of the conventions above were taken from), so that the backward neither
 *   recomputes the scores nor the decisions; under FWM with Nearest, whose
 *   backward needs only the interval, the level bit and the tail, by one
 *   byte per key instead (1 + 2r + [t >= 1/2], 0 for the tail) in the first
 *   KiB of each tile. Element order inside a tile is the kernels' register
 *   order (internal). Last, the deterministic backward's scratch:
 *   max(2 * ceil(T/128), 4) * R f32 (kia_set_deterministic).
 * Each array starts at a 256-byte boundary (kia_stats_offset gives it).
 * m, amin and nmin are written for MinMax only (FWM uses only the maximum).
 * kia_attn_fwd writes the statistics and U; kia_attn_bwd reads them and uses
 * the scratch; calling the backward with flags other than the forward's
 * that filled `stats` is undefined.
 */
#define KIA_STAT_M 0
#define KIA_STAT_m 1
#define KIA_STAT_W 2
#define KIA_STAT_WL 3
#define KIA_STAT_AMAX 4
#define KIA_STAT_AMIN 5
#define KIA_STAT_NMAX 6
#define KIA_STAT_NMIN 7
#define KIA_STAT_ROWREC 8  /* 16 floats per row */
#define KIA_STAT_SSELF 9
#define KIA_STAT_CM 10
#define KIA_STAT_OL 11     /* R*d floats, written iff recon=Nearest, ste=Prob */
#define KIA_STAT_DS 12     /* backward dS scratch (tiles, see above) */
#define KIA_STAT_U 13      /* forward scores / decided positions (tiles) */
#define KIA_STAT_PART 14   /* deterministic backward: row-sum partials of each
                              128-key block, [2, ceil(T/128), R] fp32, then
                              the calibration records of its dK gather
                              ([R, 4]); max(2 ceil(T/128), 4) R floats */
#define KIA_STAT_ACC 15    /* bf16-output backward: fp32 dQ, dK, dV [3, R, d]
                              (kia_stats_bytes_bf16o; absent otherwise) */

/* Size in bytes of the stats buffer for this problem (0 on bad arguments).
 * recon takes every KIA_RECON_* value; the size and every offset depend on
 * B, H, T, d and causal only (recon and ste are validated, not used). */
int kia_stats_bytes(int B, int H, int T, int d, int recon, int ste,
                    int causal, size_t *bytes);

/* Byte offset of field `field` (KIA_STAT_*) inside the stats buffer. */
int kia_stats_offset(int B, int H, int T, int d, int recon, int ste,
                     int causal, int field, size_t *offset);

/*
 * Forward (Sec. 3 objects, calibration and reconstruction; App. A).
 * In: q, k, v [B,H,T,d] fp32. Out: o [B,H,T,d] fp32, stats (see above).
 * The output does not depend on `ste` or `detach` (strict hard forward
 * P = P^N for Nearest, App. fwd audits (iii)); both are accepted so that a
 * caller passes the same flags to both directions.
 */
int kia_attn_fwd(const float *q, const float *k, const float *v, float *o,
                 void *stats, int B, int H, int T, int d, int K, int calib,
                 float tau, int recon, int ste, int detach, int causal,
                 void *stream);

/*
 * Backward (App. B): gradients of a loss L with upstream dO = dL/dO.
 * In: q, k, v, o (the forward's output), dO [B,H,T,d] fp32; stats as filled
 * by kia_attn_fwd with the same arguments (its scratch is overwritten).
 * Out: dq, dk, dv [B,H,T,d] fp32 (fully overwritten).
 *   g_j = dO_i . v_j; gamma_j = (g_j - <g>_{P^X}) / W^X with X the hard
 *   point for Nearest + Weight-STE, the LERP point otherwise;
 *   dS_ij = gamma_j Delta_j (+ the Eq. full terms the mode keeps; P1
 *   subtracts the row mean of the detached dS);
 *   dV = P^T dO (forward P), dQ = scale dS K, dK = scale dS^T Q.
 */
int kia_attn_bwd(const float *q, const float *k, const float *v,
                 const float *o, const float *dO, void *stats, float *dq,
                 float *dk, float *dv, int B, int H, int T, int d, int K,
                 int calib, float tau, int recon, int ste, int detach,
                 int causal, void *stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight training or serving loops, harnesses that forbid
 * allocation): kia_attn_fwd followed by kia_attn_bwd in one call, with the
 * statistics kept in a device array the library owns instead of a
 * caller-allocated `stats` (KIA_STATIC_BYTES per GPU, held from the first
 * call on that GPU until the process ends). The caller passes the inputs
 * q, k, v, dO and the outputs o, dq, dk, dv ([B,H,T,d] fp32, as in
 * kia_attn_fwd / kia_attn_bwd, whose arguments, checks and results these
 * are); nothing is allocated or freed. Problems whose statistics exceed
 * KIA_STATIC_BYTES (kia_stats_bytes) return KIA_ERR_SCRATCH before any
 * launch: 128 MiB holds the paper's micro-batch-1 attention calls (B1 H12
 * and B1 H24 at T = 1024, d = 64). Every call on one GPU uses that GPU's
 * single array, so calls that overlap on one GPU (concurrent streams or
 * threads) race; calls in one stream order are safe, each overwrites what
 * the last one left.
 */
#define KIA_STATIC_BYTES (128u << 20)
int kia_attn_fwd_bwd_static(const float *q, const float *k, const float *v,
                            const float *dO, float *o, float *dq, float *dk,
                            float *dv, int B, int H, int T, int d, int K,
                            int calib, float tau, int recon, int ste,
                            int detach, int causal, void *stream);

/*
 * bf16-input variant (the 1B-scale workload's bf16 inputs with fp32
 * accumulation). q, k, v and dO are bf16 bit patterns (uint16_t, the upper
 * half of the fp32 encoding); o, stats, dq, dk, dv and every argument
 * check, convention and statistics field are as in kia_attn_fwd and
 * kia_attn_bwd. Every product runs on the bf16 MFMA with fp32 accumulation:
 * Q K^T and dO V^T take the inputs exactly (a score is the fp32 sum of
 * exact bf16 x bf16 products, in the order of the bf16 score sub-tile, so
 * it can differ from the fp32 path's in the last bits); P V, O^L, P^T dO,
 * dS^T Q and dS K round their fp32 operand P (the forward weight), w^L or
 * dS to bf16 (relative error <= 2^-9 per element). Scores, extrema, index
 * decisions, grid weights, normalizers W and W^L, and the backward's row
 * sums stay fp32. Mixing the variants on one `stats` is undefined.
 */
int kia_attn_fwd_bf16(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                      float *o, void *stats, int B, int H, int T, int d,
                      int K, int calib, float tau, int recon, int ste,
                      int detach, int causal, void *stream);
int kia_attn_bwd_bf16(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                      const float *o, const uint16_t *dO, void *stats,
                      float *dq, float *dk, float *dv, int B, int H, int T,
                      int d, int K, int calib, float tau, int recon, int ste,
                      int detach, int causal, void *stream);

/*
 * bf16-output variant (the paper's models run in bf16 autocast around the
 * attention operator: Protocol details, "Training." and "Numerics and
 * hardware."): the bf16-input variant with o, dq, dk and dv as bf16 bit
 * patterns (uint16_t), each the round-to-nearest-even of the fp32 value the
 * kernels accumulate (one rounding per element). Everything else,
 * including the argument checks, the statistics and O^L, is as in
 * kia_attn_fwd_bf16 / kia_attn_bwd_bf16, except: the backward's D = dO . O
 * (Weight-STE, LERP) takes the bf16 O it is given, and its stats buffer
 * needs kia_stats_bytes_bf16o bytes, whose last field (KIA_STAT_ACC) holds
 * the fp32 dQ and dK accumulators (the calibration terms, tie splits and the
 * P1 projection add into them after the main kernels) and, when a small
 * grid splits the main kernel's query ranges (whose parts add up), dV's.
 * A stats buffer of that size also serves the other entry points.
 */
int kia_stats_bytes_bf16o(int B, int H, int T, int d, int recon, int ste,
                          int causal, size_t *bytes);
int kia_attn_fwd_bf16o(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                       uint16_t *o, void *stats, int B, int H, int T, int d,
                       int K, int calib, float tau, int recon, int ste,
                       int detach, int causal, void *stream);
int kia_attn_bwd_bf16o(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                       const uint16_t *o, const uint16_t *dO, void *stats,
                       uint16_t *dq, uint16_t *dk, uint16_t *dv, int B, int H,
                       int T, int d, int K, int calib, float tau, int recon,
                       int ste, int detach, int causal, void *stream);

/*
 * Index codes of every (query, key) pair, computed by the same device code
 * as the forward from the same scores (for bit-exact index tests).
 * In: q, k, and stats filled by kia_attn_fwd with the same arguments.
 * Out: codes [B,H,T,T] uint16 (device): bits 0-5 interval r, bits 6-12
 * nearest level l, bit 13 FWM tail, bit 14 valid key, bit 15 degenerate
 * MinMax row; r = l = 0 on tail and degenerate keys, 0 for invalid keys.
 * For the exponential weight functions: bit 15 valid key, bits 0-14 the
 * weight's bf16 bit pattern (BF16EXP) or its E4M3 byte (FP8EXP), 0 for
 * SOFTMAX; 0 for invalid keys.
 */
int kia_debug_codes(const float *q, const float *k, const void *stats,
                    uint16_t *codes, int B, int H, int T, int d, int K,
                    int calib, float tau, int recon, int causal, void *stream);
/* The same for the bf16-input variant (bf16 score sub-tile). */
int kia_debug_codes_bf16(const uint16_t *q, const uint16_t *k,
                         const void *stats, uint16_t *codes, int B, int H,
                         int T, int d, int K, int calib, float tau, int recon,
                         int causal, void *stream);

/*
 * Code words of the decisions the forward stored for the backward (stats
 * field U: the positions u that the second pass decided and the backward
 * reads; for an exponential weight function its stored fp32 exponential),
 * decoded without recomputing any score, so that an index test checks the
 * product's own decisions and U's tile addressing. Call after kia_attn_fwd
 * or kia_attn_fwd_bf16 with the same B..causal (ste selects the stats
 * layout; the backward leaves U unchanged, so a call after kia_attn_bwd
 * gives the same words). Out: codes [B,H,T,T] uint16 (device, caller-owned,
 * 16-byte aligned), the format of kia_debug_codes; 0 for keys that are not
 * valid. Same argument checks as kia_attn_fwd; KIA_ERR_SHAPE if B*H*T*T
 * overflows.
 */
int kia_debug_codes_stored(const void *stats, uint16_t *codes, int B, int H,
                           int T, int d, int K, int calib, float tau,
                           int recon, int ste, int causal, void *stream);

/*
 * The fp32 scores s = fl32(fl32(q.k) * fl32(1/sqrt(d))) of every (query,
 * key) pair, from the canonical score sub-tile that the forward's extrema
 * pass evaluates (bit-identical to the scores every decision of
 * kia_attn_fwd resp. kia_attn_fwd_bf16 is taken on; App. A: the operator
 * acts on the fp32 score rows). For tests that hand the oracle the
 * kernels' own scores. Out: scores [B,H,T,T] f32 (device, caller-owned,
 * 16-byte aligned), 0 for keys that are not valid (j > i when causal).
 */
int kia_debug_scores(const float *q, const float *k, float *scores, int B,
                     int H, int T, int d, int causal, void *stream);
int kia_debug_scores_bf16(const uint16_t *q, const uint16_t *k, float *scores,
                          int B, int H, int T, int d, int causal,
                          void *stream);

/*
 * Score-gradient decomposition (appendix on the detached-gradient record,
 * local gradient decomposition: g_full = g_self + g_M + g_m). Call after
 * kia_attn_bwd (input_bf16 = 0) or kia_attn_bwd_bf16 (input_bf16 = 1) with
 * the same B..causal and the gradient mode 0, 2 or 3 (the modes that
 * compute both channels' row sums); nothing else may have touched `stats`.
 * Out (device, caller-owned): g_self [B,H,T,T] f32, the detached dS_ij =
 * gamma_j Delta_j of App. B as the backward computed it (bf16-rounded for
 * the bf16 variant), zero on keys that are not valid; cM, cm [B,H,T] f32,
 * the row sums sum_j gamma_j dw_j/dM and sum_j gamma_j dw_j/dm (0 on
 * degenerate rows; FWM: cM = -sum_j dS_ij, cm = 0). g_M adds cM/nmax on each
 * key whose score equals M (amax and its ties, see stats), g_m adds cm/nmin
 * on each key equal to m.
 */
int kia_debug_score_grad(const void *stats, int input_bf16, float *g_self,
                         float *cM, float *cm, int B, int H, int T, int d,
                         int calib, int recon, int ste, int causal, void *stream);

/*
 * Geometry probe (Sec. 2 and the appendix paragraph on the geometry probe):
 * per-row statistics of the operator's fp32 scores and of its distortion of
 * them. Call after kia_attn_fwd with the same B..causal on `stats` (its M,
 * m and W are used; nothing is written to it). MinMax or FWM calibration
 * with LERP or Nearest reconstruction (others: KIA_ERR_ENUM); fp32 inputs.
 * Out: out [B,H,T,KIA_GEO_COUNT] f32 (device, caller-owned); per row i over
 * its valid keys, with z = s - M and P^E the softmax of the row's scores:
 *   SPAN M - m; H the native width ((M - m)/K MinMax, tau/K FWM);
 *   ZQ001 the 0.1% quantile of z (sorted, linear interpolation at
 *   (n - 1)/1000); QNORM |q_i|, KNORM |k_i|; ENTROPY -sum P^E ln P^E;
 *   FRAC6 the fraction of keys with z < -6; TOPMASS the P^E mass on keys in
 *   the top level (Nearest, l = K) or top interval (LERP, r = K-1);
 *   EFFB exp H(q), q_b the P^E mass of bucket b (the level l for Nearest,
 *   the interval r for LERP, one bucket for the FWM tail; degenerate MinMax
 *   rows have one bucket); TV 1/2 sum_j |P_j - P^E_j| with P the forward's
 *   probabilities. The paper averages rows i >= 1; row 0 is reported too.
 */
#define KIA_GEO_SPAN 0
#define KIA_GEO_H 1
#define KIA_GEO_ZQ001 2
#define KIA_GEO_QNORM 3
#define KIA_GEO_KNORM 4
#define KIA_GEO_ENTROPY 5
#define KIA_GEO_FRAC6 6
#define KIA_GEO_TOPMASS 7
#define KIA_GEO_EFFB 8
#define KIA_GEO_TV 9
#define KIA_GEO_COUNT 10
int kia_geometry_probe(const float *q, const float *k, const void *stats,
                       float *out, int B, int H, int T, int d, int K,
                       int calib, float tau, int recon, int causal,
                       void *stream);

/*
 * Matrix-core peak probe (a measurement aid for the roofline, not part of
 * the operator): `workgroups` workgroups of four waves each run `iters`
 * rounds of four independent fp32 v_mfma_f32_32x32x2_f32 (4096 flops each)
 * on register operands, so a launch executes
 * workgroups x 4 x iters x 4 x 4096 flops; the caller times it (e.g. with
 * events on `stream`) for the chip's sustained fp32 matrix rate. out
 * (device, caller-owned, 8-byte aligned, 4 uint64) receives workgroup 0's
 * first wave's shader clock counter (s_memtime) before and after its loop,
 * then the 100 MHz constant-rate counter (s_memrealtime) before and after:
 * (out[1] - out[0]) / (out[3] - out[2]) x 100 MHz is the shader clock under
 * this load. workgroups and iters in [1, 2^20] (else KIA_ERR_SHAPE); NULL out:
 * KIA_ERR_NULL; misaligned out: KIA_ERR_ALIGN. Recorded by the timing hook
 * as "kia_mfma_probe".
 */
int kia_mfma_peak_probe(unsigned long long *out, int workgroups, int iters, void *stream);

/*
 * Measurement hook for benchmarks. kia_timing_enable(1) clears the record
 * and from then on brackets every kernel the library launches with two
 * hipEvents recorded on that launch's stream (events are created per
 * launch; at most 65536 launches are recorded). kia_timing_read waits for
 * the recorded events of the kernels called `name` ("kia_fwd",
 * "kia_bwd_pre", "kia_bwd_main", "kia_bwd_dq", "kia_bwd_ties",
 * "kia_bwd_p1", "kia_cast_bf16", "kia_codes", "kia_codes_stored", "kia_scores",
 * "kia_score_grad", "kia_geometry",
 * "kia_mfma_probe") and returns their summed duration in ms and their count
 * (in the deterministic backward, "kia_bwd_main" also counts its row-sum
 * pass and "kia_bwd_dq" its calibration gather).
 * kia_timing_enable(0) stops recording and frees the events. Process-wide
 * state, not thread-safe; the kernels' results do not depend on it.
 */
int kia_timing_enable(int on);
int kia_timing_read(const char *name, double *total_ms, int *launches);

/*
 * Launch-shape policy (process-wide, not thread-safe; affects later calls).
 * KIA_GRID_AUTO (default) picks per call: when a problem's natural grid
 * leaves the CUs short of work (micro-batch-1 shapes), the kernels split it
 * -- the fp32 forward takes one 32-row group with four key quarters per
 * workgroup (d <= 64; eight key parts in 8-wave workgroups when there are
 * fewer 64-row blocks than CUs) instead of two row groups with two key
 * halves, the backward's main kernel (fp32 and bf16 inputs) splits each key
 * block's query range over several workgroups (dK, dV added atomically) and
 * the fp32 dQ kernel each group of query tiles' keys over several pieces
 * (dQ added atomically). KIA_GRID_WIDE never splits;
 * KIA_GRID_SPLIT always does (the forward's four key quarters, the
 * backward's splits in at least two parts). The policies compute the same decisions,
 * extrema and codes; O, W and the gradients differ only in fp32 summation
 * order (neither backward is bitwise repeatable: see Determinism above).
 * Returns KIA_ERR_ENUM for another value.
 */
#define KIA_GRID_AUTO 0
#define KIA_GRID_WIDE 1
#define KIA_GRID_SPLIT 2
int kia_set_grid_policy(int policy);

/*
 * Deterministic backward (process-wide, not thread-safe; affects later
 * calls). on = 1: every reduction of the backward runs in a fixed order, so
 * that repeated calls on the same inputs give bitwise equal dQ, dK, dV (the
 * forward always does):
 *   - the main kernel's query ranges and the dQ kernel's keys are not split
 *     (the unsplit launch shapes of KIA_GRID_WIDE, whatever the policy);
 *   - each 128-key block writes its row sums of the score gradients into
 *     KIA_STAT_PART, which a pass adds up in key-block order;
 *   - the calibration terms of rows with unique extrema are gathered per
 *     key, in row order, instead of scattered onto dK (the dQ kernel leaves
 *     one record per row in KIA_STAT_PART for that);
 *   - the rows with tied extrema of one (b, h) slice are taken by a single
 *     wave, in row order.
 * The results differ from those of on = 0 only in fp32 summation order.
 * on = 0 (default) restores the atomic reductions. Returns KIA_ERR_ENUM
 * for another value.
 */
int kia_set_deterministic(int on);

/* Human-readable text for a return code (static storage). */
const char *kia_strerror(int code);

#ifdef __cplusplus
}
#endif

#endif /* KIA_H */
