/*
 * kia_oracle.c -- plain fp64 CPU oracle of causal K-interval attention.
 *
 * TEST INFRASTRUCTURE. Only tests/, __graft_entry__.smoke() and the
 * cpu_baseline leg of bench.py may load or call this library. The product
 * path (paper_2609_33591_amd/) never does, and this file shares no code,
 * header, table or helper with it.
 *
 * What it follows (Zhu, Hu, Kozlowski, "Pretraining Transformers with
 * Quantized Softmax in Attention"):
 *   - Sec. 3 "Objects and calibration", "Reconstruction", Eq. (calgrad),
 *     Eq. (full), Eq. (wste), Eq. (pste);
 *   - App. A "Operator definitions and edge cases" and Table S (tab:edge);
 *   - App. B "Gradient derivations" (normalization Jacobian, LERP own-score
 *     slope, full calibration gradient, detach, Weight-STE, Prob-STE, FWM);
 *   - App. A "Softmax" and App. D "Reduced-precision exponential baselines"
 *     (BF16-exp, FP8-rounded exp with the fp32 exponential's backward);
 *   - the appendix on the tail policy in the MinMax -> FWM change: the
 *     "resolved" grid (FWM step and origin, continued below -tau);
 *   - Sec. 2 and the appendix paragraph on the geometry probe (per-row
 *     statistics of the scores and of the operator's distortion).
 *
 * Everything is computed in fp64 after the scores. Scores are the paper's
 * fp32 scores (App. A: the operator acts on a row of fp32 scores
 * S = Q K^T / sqrt(d_h)); with round_scores=1 the oracle forms them as
 * fl32( fl32(q.k) * fl32(1/sqrt(d)) ), with round_scores=0 it keeps the fp64
 * value q.k * (1/sqrt(d)) (used by the finite-difference pins).
 *
 * Index decisions (interval r, nearest level l, FWM tail) are taken on the
 * given scores by one correctly rounded fp64 division each:
 *   MinMax: u = (K * (s - m)) / (M - m)
 *   FWM:    a = (s - M) + tau,  tail <=> a < 0,  u = (K * a) / tau
 *   resolved: u = (K * ((s - M) + tau)) / tau, no tail, r = min(floor(u), K-1)
 * which is (z - z_min)/h resp. (z + tau)/h of App. A rewritten so that an
 * exact grid point or midpoint of fp32 scores lands exactly on the integer
 * or half-integer (a reading of the paper's real-arithmetic formulas).
 *
 * Build: gcc -O2 -std=c11 -fopenmp -ffp-contract=off -shared -fPIC
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define KIO_CALIB_MINMAX 0
#define KIO_CALIB_FWM 1
/* App. tail-policy decomposition, "resolved": FWM's step tau/K and origin
 * -tau, the grid continued below -tau with negative indices, no zero tail. */
#define KIO_CALIB_RESOLVED 2
#define KIO_RECON_LERP 0
#define KIO_RECON_NEAREST 1
/* App. A (operator definitions, Softmax) and App. D (reduced-precision
 * exponential baselines): exact softmax, BF16-exp, FP8 (E4M3)-rounded exp.
 * These ignore K, the calibration and the STE choice. */
#define KIO_RECON_SOFTMAX 2
#define KIO_RECON_BF16EXP 3
#define KIO_RECON_FP8EXP 4
#define KIO_STE_WEIGHT 0
#define KIO_STE_PROB 1
#define KIO_GRAD_FULL 0
#define KIO_GRAD_DETACH 1
#define KIO_GRAD_MAX_ONLY 2
#define KIO_GRAD_MIN_ONLY 3
#define KIO_GRAD_DETACH_P1 4

/* App. A: degenerate branch iff M - m <= eps, eps = 1e-12. */
#define KIO_DEGEN_EPS 1e-12

/* Per-row record exported to Python (doubles, KIO_ROWINFO entries). */
#define KIO_ROWINFO 16
enum {
  RI_M = 0, RI_m, RI_AMAX, RI_NMAX, RI_AMIN, RI_NMIN, RI_DEGEN, RI_H,
  RI_WN, RI_WL, RI_W, RI_CM, RI_Cm, RI_SSELF, RI_NVALID, RI_SPARE
};

typedef struct {
  double M, m;
  int amax, nmax, amin, nmin;
  int degen;
  double h;     /* interval width */
  double zmin;  /* z_lo: lowest grid point b_0 in z = s - M coordinates */
  double WN, WL, W;
} row_state;

/* ---------------------------------------------------------------------- */
/* Row forward: calibration, index, reconstruction, normalization.        */
/* ---------------------------------------------------------------------- */

/*
 * Row extrema and their tie sets (App. A: amax/amin over the causal-valid
 * keys; Table tab:edge: ties are kept as sets, first index and size here).
 */
static void row_extrema(int n, const double *s, row_state *st) {
  st->M = s[0];
  st->m = s[0];
  for (int j = 1; j < n; ++j) {
    if (s[j] > st->M) st->M = s[j];
    if (s[j] < st->m) st->m = s[j];
  }
  st->amax = -1; st->nmax = 0; st->amin = -1; st->nmin = 0;
  for (int j = 0; j < n; ++j) {
    if (s[j] == st->M) { if (st->amax < 0) st->amax = j; st->nmax++; }
    if (s[j] == st->m) { if (st->amin < 0) st->amin = j; st->nmin++; }
  }
}

/*
 * Grid value e^{b_r}, b_r = (1 - r/K) z_lo with z_lo = m - M (MinMax, Sec. 3:
 * b_r = (1 - r/K)(m - M)) or z_lo = -tau (FWM: b_r = -tau + r tau/K). This
 * form makes b_K = 0 and b_0 = z_lo exact.
 */
static double grid_exp(const row_state *st, int K, int r) {
  return exp((1.0 - (double)r / (double)K) * st->zmin);
}

/* ---------------------------------------------------------------------- */
/* Exponential weight functions (softmax and the reduced-precision        */
/* baselines).                                                             */
/* ---------------------------------------------------------------------- */

static int is_exp_mode(int recon) {
  return recon == KIO_RECON_SOFTMAX || recon == KIO_RECON_BF16EXP ||
         recon == KIO_RECON_FP8EXP;
}

static uint32_t f32_bits(float x) { uint32_t b; memcpy(&b, &x, 4); return b; }
static float f32_of(uint32_t b) { float x; memcpy(&x, &b, 4); return x; }

/*
 * bfloat16 rounding of x: x is first rounded to fp32 (the weights and
 * gradients of the reduced-precision path are fp32 tensors before the cast),
 * then to the nearer of the two bfloat16 values that bracket it (fp32 bit
 * patterns with the low 16 bits cleared, towards and away from zero), ties
 * to the one with an even last kept bit.
 */
static double bf16_round(double x) {
  float f = (float)x;
  uint32_t b = f32_bits(f);
  uint32_t lo = b & 0xFFFF0000u;
  if (lo == b) return (double)f;
  float vlo = f32_of(lo), vhi = f32_of(lo + 0x10000u);
  double dlo = fabs((double)f - (double)vlo), dhi = fabs((double)vhi - (double)f);
  if (dlo < dhi) return (double)vlo;
  if (dhi < dlo) return (double)vhi;
  return ((lo >> 16) & 1u) ? (double)vhi : (double)vlo;
}

/* Value of the float8_e4m3fn code c in [0, 0x7E]: 4 exponent bits (bias 7),
 * 3 mantissa bits, subnormals m * 2^-9 (0x7F is NaN, not used). */
static double e4m3_value(int c) {
  int e = c >> 3, m = c & 7;
  if (e == 0) return ldexp((double)m, -9);
  return ldexp(1.0 + (double)m / 8.0, e - 7);
}

/* Nearest non-negative E4M3 value to x >= 0 by exhaustive search over the
 * codes, ties to the even code (round to nearest even). Returns the code. */
static int e4m3_round(double x, double *val) {
  int best = 0;
  double bd = fabs(x);
  for (int c = 1; c <= 0x7E; ++c) {
    double d = fabs(x - e4m3_value(c));
    if (d < bd || (d == bd && (c & 1) == 0)) { bd = d; best = c; }
  }
  *val = e4m3_value(best);
  return best;
}

/*
 * Weight of one key from its fp32 shift z = s - M (z <= 0):
 *   softmax:  w = e^z (App. A, Softmax);
 *   BF16-exp: w = bf16(e^{bf16(z)}), the input rounded before the
 *             exponential and the result rounded after it;
 *   FP8-exp:  w^exp = fp32(e^z), w = e4m3(w^exp).
 * wE receives the value whose derivative the backward uses (e^z, w, w^exp);
 * code the quantized weight's bit pattern (bf16 bits or the E4M3 byte; 0 for
 * softmax).
 */
static void exp_weight(float z, int recon, double *w, double *wE, int *code) {
  *code = 0;
  if (recon == KIO_RECON_SOFTMAX) {
    *w = exp((double)z);
    *wE = *w;
  } else if (recon == KIO_RECON_BF16EXP) {
    double zb = bf16_round((double)z);
    *w = bf16_round(exp(zb));
    *wE = *w;
    *code = (int)(f32_bits((float)*w) >> 16);
  } else {
    double we = (double)(float)exp((double)z);
    *code = e4m3_round(we, w);
    *wE = we;
  }
}

/*
 * Forward of one row under an exponential weight function. z_j is the fp32
 * difference s_j - M of the fp32 scores (App. A: z_j = s_j - M); the row
 * maximum's key has z = 0 and weight 1, so W >= 1. Outputs: u[j] = z_j,
 * wL[j] = wN[j] = w_j, t[j] = wE_j (the arrays of the K-interval path, so
 * that the attention loops stay shared).
 */
static void exp_row_forward(int n, const double *s, int recon, row_state *st,
                            double *u, double *t, double *wL, double *wN) {
  row_extrema(n, s, st);
  st->degen = 0;
  st->h = 0.0;
  st->zmin = 0.0;
  st->WN = 0.0;
  float M32 = (float)st->M;
  for (int j = 0; j < n; ++j) {
    float z = (float)s[j] - M32;
    double w, wE;
    int code;
    exp_weight(z, recon, &w, &wE, &code);
    u[j] = (double)z;
    t[j] = wE;
    wL[j] = w;
    wN[j] = w;
    st->WN += w;
  }
  st->WL = st->WN;
  st->W = st->WN;
}

/*
 * dL/ds of one row under an exponential weight function, given
 * g_j = dL/dP_j. With P = w / W (normalization at the forward weights),
 * dL/dw_j = (g_j - sum_i P_i g_i) / W. Then
 *   softmax:  dz_j = dL/dw_j * e^{z_j};
 *   BF16-exp: the backward of the casts and of the bf16 exponential:
 *             dz_j = bf16( bf16(dL/dw_j) * w_j );
 *   FP8-exp:  identity through the rounding, fp32 exponential's derivative:
 *             dz_j = dL/dw_j * w^exp_j.
 * The row maximum stays on the gradient path (z = s - M): the max channel
 * is cM = -sum_j dz_j on the argmax keys (added by row_scatter), so every
 * row of dS sums to zero. cm = 0 (no minimum).
 */
static void exp_row_backward(int n, const double *g, int recon,
                             const row_state *st, const double *wE,
                             const double *w, double *dS, double *cM_out,
                             double *sself_out) {
  double gbar = 0.0;
  for (int j = 0; j < n; ++j) gbar += (w[j] / st->W) * g[j];
  double sself = 0.0;
  for (int j = 0; j < n; ++j) {
    double dw = (g[j] - gbar) / st->W;
    double dz;
    if (recon == KIO_RECON_BF16EXP)
      dz = bf16_round(bf16_round(dw) * w[j]);
    else
      dz = dw * wE[j];
    dS[j] = dz;
    sself += dz;
  }
  *cM_out = -sself;
  *sself_out = sself;
}

/*
 * One row of K-interval weights. Inputs: n valid scores s[0..n-1]. Outputs
 * per key: r (interval), l (nearest level), tail flag, u = r + t, t, w^L,
 * w^N; the row state (extrema, h, W^N, W^L, forward W).
 */
static void row_forward(int n, const double *s, int K, int calib, double tau,
                        int recon, row_state *st, int *r, int *l, int *tail,
                        double *u, double *t, double *wL, double *wN) {
  if (is_exp_mode(recon)) {
    for (int j = 0; j < n; ++j) { r[j] = 0; l[j] = 0; tail[j] = 0; }
    exp_row_forward(n, s, recon, st, u, t, wL, wN);
    return;
  }
  row_extrema(n, s, st);
  st->degen = 0;
  if (calib == KIO_CALIB_MINMAX) {
    double span = st->M - st->m;
    /* Degenerate branch (App. A, tab:edge): weights 1, P uniform. */
    if (span <= KIO_DEGEN_EPS) {
      st->degen = 1;
      st->h = 1.0; /* h_safe */
      st->zmin = 0.0;
    } else {
      st->h = span / (double)K;
      st->zmin = st->m - st->M;
    }
  } else {
    st->h = tau / (double)K;
    st->zmin = -tau;
  }
  st->WN = 0.0; st->WL = 0.0;
  for (int j = 0; j < n; ++j) {
    tail[j] = 0;
    if (st->degen) {
      r[j] = 0; l[j] = 0; u[j] = 0.0; t[j] = 0.0;
      wL[j] = 1.0; wN[j] = 1.0;
    } else {
      double uj;
      if (calib == KIO_CALIB_MINMAX) {
        uj = ((double)K * (s[j] - st->m)) / (st->M - st->m);
      } else if (calib == KIO_CALIB_RESOLVED) {
        /* every key on the FWM grid, u < 0 below the window */
        uj = ((double)K * ((s[j] - st->M) + tau)) / tau;
      } else {
        double a = (s[j] - st->M) + tau;
        if (a < 0.0) {
          /* FWM zero tail: w = 0 below the window (Sec. 3, App. A). */
          tail[j] = 1;
          r[j] = 0; l[j] = 0; u[j] = 0.0; t[j] = 0.0;
          wL[j] = 0.0; wN[j] = 0.0;
          continue;
        }
        uj = ((double)K * a) / tau;
      }
      /* r = clip(floor(u), 0, K-1); t = u - r in [0,1] (App. A). The
       * resolved grid has no lower end: r = min(floor(u), K-1). */
      int rj = (int)floor(uj);
      if (rj < 0 && calib != KIO_CALIB_RESOLVED) rj = 0;
      if (rj > K - 1) rj = K - 1;
      double tj = uj - (double)rj;
      if (tj < 0.0) tj = 0.0;
      if (tj > 1.0) tj = 1.0;
      /* Nearest: l = r + 1[t >= 1/2], midpoint rounds up (tab:edge). */
      int lj = rj + (tj >= 0.5 ? 1 : 0);
      r[j] = rj; l[j] = lj; u[j] = uj; t[j] = tj;
      double Er = grid_exp(st, K, rj), Er1 = grid_exp(st, K, rj + 1);
      wL[j] = (1.0 - tj) * Er + tj * Er1;   /* LERP */
      wN[j] = grid_exp(st, K, lj);             /* Nearest */
    }
    st->WN += wN[j];
    st->WL += wL[j];
  }
  st->W = (recon == KIO_RECON_NEAREST) ? st->WN : st->WL;
}

/* ---------------------------------------------------------------------- */
/* Row backward: surrogate Jacobian plus calibration terms.                */
/* ---------------------------------------------------------------------- */

/*
 * dL/ds for one row given g_j = dL/dP_j (App. B).
 *  gamma_j = (g_j - sum_i P^X_i g_i) / W^X, X = hard point (Weight-STE with
 *  Nearest, Eq. wste) or LERP point (LERP, and Prob-STE, Eq. pste).
 *  dS_j = gamma_j Delta_j, Delta_j = (e^{b_{r+1}} - e^{b_r}) / h;
 *  full gradient adds sum_j gamma_j dw_j/dM on the argmax keys and
 *  sum_j gamma_j dw_j/dm on the argmin keys, split evenly among ties
 *  (Eq. full, Eq. calgrad; FWM: dw/dM = -Delta, no m term). Detach keeps
 *  gamma_j Delta_j only. Degenerate MinMax rows: zero gradient (tab:edge).
 *
 *  Gradient modes (`grad`): 0 full; 1 detach; 2 max_only and 3 min_only
 *  keep the self term and one extremum channel only (appendix on the
 *  detached-gradient record: single-channel ablation and local gradient
 *  decomposition, g_max_only = g_self + g_M, g_min_only = g_self + g_m;
 *  FWM has no minimum channel); 4 detach with the P1
 *  projection of each row onto the zero-sum subspace, g'_j = g_j minus the
 *  mean of g over the row's valid keys (App. B, Detach).
 */
static void row_backward(int n, const double *g, int K, int calib, int recon,
                         int ste, int grad, const row_state *st,
                         const int *r, const int *tail, const double *u,
                         const double *t, const double *wL, const double *wN,
                         double *dS, double *cM_out, double *cm_out,
                         double *sself_out) {
  (void)grad; /* the mode acts in row_scatter: the self term is shared */
  *cM_out = 0.0; *cm_out = 0.0; *sself_out = 0.0;
  if (is_exp_mode(recon)) {
    exp_row_backward(n, g, recon, st, t, wL, dS, cM_out, sself_out);
    return;
  }
  if (st->degen) {
    for (int j = 0; j < n; ++j) dS[j] = 0.0;
    return;
  }
  int hard_point = (recon == KIO_RECON_NEAREST && ste == KIO_STE_WEIGHT);
  const double *wX = hard_point ? wN : wL;
  double WX = hard_point ? st->WN : st->WL;
  double gbar = 0.0;   /* <g>_{P^X} */
  for (int j = 0; j < n; ++j) gbar += (wX[j] / WX) * g[j];
  double cM = 0.0, cm = 0.0, sself = 0.0;
  for (int j = 0; j < n; ++j) {
    if (tail[j]) { dS[j] = 0.0; continue; }
    double gamma = (g[j] - gbar) / WX;
    double Er = grid_exp(st, K, r[j]), Er1 = grid_exp(st, K, r[j] + 1);
    double delta = (Er1 - Er) / st->h;
    dS[j] = gamma * delta;
    sself += dS[j];
    if (calib == KIO_CALIB_MINMAX) {
      double rho = (r[j] + t[j]) / (double)K;
      double X = ((1.0 - t[j]) * r[j] * Er + t[j] * (r[j] + 1) * Er1) / (double)K;
      double dwdM = -wL[j] - delta * rho + X;
      double dwdm = -delta * (1.0 - rho) + wL[j] - X;
      cM += gamma * dwdM;
      cm += gamma * dwdm;
    } else {
      cM += -gamma * delta;
    }
    (void)u;
  }
  *cM_out = cM; *cm_out = cm; *sself_out = sself;
}

/* Adds the calibration terms of Eq. (full) kept by the gradient mode onto
 * the argmax/argmin keys; mode 4 projects the detached row (P1). */
static void row_scatter(int n, const double *s, int calib, int grad,
                        const row_state *st, double cM, double cm, double *dS) {
  if (grad == KIO_GRAD_DETACH_P1) {
    double mean = 0.0;
    for (int j = 0; j < n; ++j) mean += dS[j];
    mean /= (double)n;
    for (int j = 0; j < n; ++j) dS[j] -= mean;
    return;
  }
  if (st->degen || grad == KIO_GRAD_DETACH) return;
  int keepM = grad == KIO_GRAD_FULL || grad == KIO_GRAD_MAX_ONLY;
  int keepm = calib == KIO_CALIB_MINMAX &&
              (grad == KIO_GRAD_FULL || grad == KIO_GRAD_MIN_ONLY);
  double inM = keepM ? cM / (double)st->nmax : 0.0;
  double inm = keepm ? cm / (double)st->nmin : 0.0;
  for (int j = 0; j < n; ++j) {
    if (keepM && s[j] == st->M) dS[j] += inM;
    if (keepm && s[j] == st->m) dS[j] += inm;
  }
}

/* ---------------------------------------------------------------------- */
/* Exported row-level entry point (used by the pins).                     */
/* ---------------------------------------------------------------------- */

static void fill_rowinfo(const row_state *st, int n, double cM, double cm,
                         double sself, double *info) {
  for (int k = 0; k < KIO_ROWINFO; ++k) info[k] = 0.0;
  info[RI_M] = st->M; info[RI_m] = st->m;
  info[RI_AMAX] = st->amax; info[RI_NMAX] = st->nmax;
  info[RI_AMIN] = st->amin; info[RI_NMIN] = st->nmin;
  info[RI_DEGEN] = st->degen; info[RI_H] = st->h;
  info[RI_WN] = st->WN; info[RI_WL] = st->WL; info[RI_W] = st->W;
  info[RI_CM] = cM; info[RI_Cm] = cm; info[RI_SSELF] = sself;
  info[RI_NVALID] = n;
}

/*
 * kio_row: forward (and, if g != NULL, backward) of one row of n scores.
 * Outputs (each may be NULL except where noted): P (forward probabilities),
 * wL, wN, r, l, tail, u, dS (needs g), info[KIO_ROWINFO].
 * Returns 0, or -1 on bad arguments.
 */
int kio_row(int n, const double *s, const double *g, int K, int calib,
            double tau, int recon, int ste, int grad, double *P,
            double *wL_out, double *wN_out, int32_t *r_out, int32_t *l_out,
            int32_t *tail_out, double *u_out, double *dS, double *info) {
  if (n <= 0 || s == NULL || K < 1) return -1;
  if (recon < 0 || recon > KIO_RECON_FP8EXP) return -1;
  if (calib < KIO_CALIB_MINMAX || calib > KIO_CALIB_RESOLVED) return -1;
  if (calib != KIO_CALIB_MINMAX && !(tau > 0.0) && !is_exp_mode(recon)) return -1;
  int *r = malloc(sizeof(int) * n), *l = malloc(sizeof(int) * n);
  int *tail = malloc(sizeof(int) * n);
  double *u = malloc(sizeof(double) * n), *t = malloc(sizeof(double) * n);
  double *wL = malloc(sizeof(double) * n), *wN = malloc(sizeof(double) * n);
  double *ds = malloc(sizeof(double) * n);
  row_state st;
  row_forward(n, s, K, calib, tau, recon, &st, r, l, tail, u, t, wL, wN);
  const double *w = (recon == KIO_RECON_NEAREST) ? wN : wL;
  double cM = 0.0, cm = 0.0, sself = 0.0;
  if (g != NULL) {
    row_backward(n, g, K, calib, recon, ste, grad, &st, r, tail, u, t, wL,
                 wN, ds, &cM, &cm, &sself);
    row_scatter(n, s, is_exp_mode(recon) ? KIO_CALIB_FWM : calib, grad, &st, cM,
                cm, ds);
  }
  for (int j = 0; j < n; ++j) {
    if (P) P[j] = w[j] / st.W;
    if (wL_out) wL_out[j] = wL[j];
    if (wN_out) wN_out[j] = wN[j];
    if (r_out) r_out[j] = r[j];
    if (l_out) l_out[j] = l[j];
    if (tail_out) tail_out[j] = tail[j];
    if (u_out) u_out[j] = u[j];
    if (dS && g) dS[j] = ds[j];
  }
  if (info) fill_rowinfo(&st, n, cM, cm, sself, info);
  free(r); free(l); free(tail); free(u); free(t); free(wL); free(wN); free(ds);
  return 0;
}

/* ---------------------------------------------------------------------- */
/* Attention level: S = Q K^T / sqrt(d), O = P V, and the backward.        */
/* ---------------------------------------------------------------------- */

/* Score of query row qi against key row kj (App. A: fp32 scores). */
static double score(const double *qi, const double *kj, int d, double scale,
                    int round_scores) {
  double acc = 0.0;
  for (int c = 0; c < d; ++c) acc += qi[c] * kj[c];
  if (round_scores) {
    float a32 = (float)acc;
    float s32 = a32 * (float)scale;
    return (double)s32;
  }
  return acc * scale;
}

static double score_scale(int d, int round_scores) {
  double sc = 1.0 / sqrt((double)d);
  if (round_scores) sc = (double)(float)sc;
  return sc;
}

/*
 * Code of one key for the index parity tests: bits 0-5 r, bits 6-12 l,
 * bit 13 tail, bit 14 valid, bit 15 degenerate row (r = l = 0 on tail and
 * degenerate keys; 0 for future keys).
 */
static uint16_t key_code(int valid, int degen, int tail, int r, int l) {
  if (!valid) return 0;
  uint16_t c = (uint16_t)(1u << 14);
  if (degen) return (uint16_t)(c | (1u << 15));
  if (tail) return (uint16_t)(c | (1u << 13));
  return (uint16_t)(c | (uint16_t)r | (uint16_t)(l << 6));
}

typedef struct {
  int B, H, T, d, K, calib, recon, ste, grad, causal, round_scores;
  double tau;
} attn_cfg;

/* Score s_ij of row i: the caller's fp32 score (given-scores mode: App. A
 * defines the operator on a row of fp32 scores, so the scores a kernel
 * computed can be handed over as they are), or formed from q_i, k_j. */
static double row_score(const attn_cfg *c, const float *given, const double *qi,
                        const double *kj, int i, int j, double scale) {
  if (given) return (double)given[(size_t)i * c->T + j];
  return score(qi, kj, c->d, scale, c->round_scores);
}

/*
 * Forward of one (b,h) slice. o [T,d]; ol [T,d] or NULL (O^L = P^L V);
 * info [T,KIO_ROWINFO] or NULL; codes [T,T] or NULL.
 */
static void attn_fwd_slice(const attn_cfg *c, const double *q, const double *k,
                           const double *v, const float *given, double *o,
                           double *ol, double *info, uint16_t *codes,
                           int row_lo, int row_hi) {
  int T = c->T, d = c->d;
  double scale = score_scale(d, c->round_scores);
  double *s = malloc(sizeof(double) * T), *u = malloc(sizeof(double) * T);
  double *t = malloc(sizeof(double) * T), *wL = malloc(sizeof(double) * T);
  double *wN = malloc(sizeof(double) * T);
  int *r = malloc(sizeof(int) * T), *l = malloc(sizeof(int) * T);
  int *tail = malloc(sizeof(int) * T);
  for (int i = row_lo; i < row_hi; ++i) {
    int n = c->causal ? i + 1 : T;
    for (int j = 0; j < n; ++j)
      s[j] = row_score(c, given, q + (size_t)i * d, k + (size_t)j * d, i, j, scale);
    row_state st;
    row_forward(n, s, c->K, c->calib, c->tau, c->recon, &st, r, l, tail, u, t,
                wL, wN);
    const double *w = (c->recon == KIO_RECON_NEAREST) ? wN : wL;
    for (int e = 0; e < d; ++e) {
      double acc = 0.0, accL = 0.0;
      for (int j = 0; j < n; ++j) {
        acc += (w[j] / st.W) * v[(size_t)j * d + e];
        accL += (wL[j] / st.WL) * v[(size_t)j * d + e];
      }
      o[(size_t)i * d + e] = acc;
      if (ol) ol[(size_t)i * d + e] = accL;
    }
    if (info) fill_rowinfo(&st, n, 0.0, 0.0, 0.0, info + (size_t)i * KIO_ROWINFO);
    if (codes && is_exp_mode(c->recon)) {
      /* quantized weight codes: bit 15 valid, bits 0-14 the bf16 pattern or
       * the E4M3 byte of w (w <= 1 keeps bit 14 clear) */
      for (int j = 0; j < T; ++j) {
        uint16_t cj = 0;
        if (j < n) {
          double w, wE;
          int code;
          exp_weight((float)u[j], c->recon, &w, &wE, &code);
          cj = (uint16_t)(0x8000u | (unsigned)code);
        }
        codes[(size_t)i * T + j] = cj;
      }
    } else if (codes && c->calib == KIO_CALIB_RESOLVED) {
      /* resolved grid (negative intervals): bit 15 valid, bit 14 l = r + 1,
       * bits 0-13 r in two's complement, clamped to [-8192, 8191] */
      for (int j = 0; j < T; ++j) {
        uint16_t cj = 0;
        if (j < n) {
          int rr = r[j] < -8192 ? -8192 : r[j];
          cj = (uint16_t)(0x8000u | (unsigned)((l[j] - r[j]) << 14) |
                          ((unsigned)rr & 0x3FFFu));
        }
        codes[(size_t)i * T + j] = cj;
      }
    } else if (codes) {
      for (int j = 0; j < T; ++j) {
        int valid = j < n;
        codes[(size_t)i * T + j] =
            key_code(valid, st.degen, valid ? tail[j] : 0, valid ? r[j] : 0,
                     valid ? l[j] : 0);
      }
    }
  }
  free(s); free(u); free(t); free(wL); free(wN); free(r); free(l); free(tail);
}

/*
 * Backward of rows [row_lo, row_hi) of one (b,h) slice (App. B):
 * g_j = dO_i . v_j; dV_j += P_j dO_i with the forward P; dQ_i = scale
 * sum_j dS_ij k_j; dK_j += scale dS_ij q_i. dk/dv are accumulated into the
 * given buffers (zeroed by the caller); dS [T,T] or NULL receives the full
 * dL/ds; info as in the forward plus cM, cm, S_self.
 */
static void attn_bwd_rows(const attn_cfg *c, const double *q, const double *k,
                          const double *v, const double *dO, const float *given,
                          double *dq, double *dk, double *dv, double *dS_out,
                          double *info, int row_lo, int row_hi) {
  int T = c->T, d = c->d;
  double scale = score_scale(d, c->round_scores);
  double *s = malloc(sizeof(double) * T), *u = malloc(sizeof(double) * T);
  double *t = malloc(sizeof(double) * T), *wL = malloc(sizeof(double) * T);
  double *wN = malloc(sizeof(double) * T), *g = malloc(sizeof(double) * T);
  double *ds = malloc(sizeof(double) * T);
  int *r = malloc(sizeof(int) * T), *l = malloc(sizeof(int) * T);
  int *tail = malloc(sizeof(int) * T);
  for (int i = row_lo; i < row_hi; ++i) {
    int n = c->causal ? i + 1 : T;
    const double *qi = q + (size_t)i * d, *doi = dO + (size_t)i * d;
    for (int j = 0; j < n; ++j)
      s[j] = row_score(c, given, qi, k + (size_t)j * d, i, j, scale);
    row_state st;
    row_forward(n, s, c->K, c->calib, c->tau, c->recon, &st, r, l, tail, u, t,
                wL, wN);
    for (int j = 0; j < n; ++j) {
      double acc = 0.0;
      for (int e = 0; e < d; ++e) acc += doi[e] * v[(size_t)j * d + e];
      g[j] = acc;
    }
    double cM, cm, sself;
    row_backward(n, g, c->K, c->calib, c->recon, c->ste, c->grad, &st, r,
                 tail, u, t, wL, wN, ds, &cM, &cm, &sself);
    row_scatter(n, s, is_exp_mode(c->recon) ? KIO_CALIB_FWM : c->calib, c->grad,
                &st, cM, cm, ds);
    const double *w = (c->recon == KIO_RECON_NEAREST) ? wN : wL;
    for (int e = 0; e < d; ++e) {
      double acc = 0.0;
      for (int j = 0; j < n; ++j) acc += ds[j] * k[(size_t)j * d + e];
      dq[(size_t)i * d + e] = scale * acc;
    }
    for (int j = 0; j < n; ++j) {
      double pj = w[j] / st.W;
      for (int e = 0; e < d; ++e) {
        dv[(size_t)j * d + e] += pj * doi[e];
        dk[(size_t)j * d + e] += scale * ds[j] * qi[e];
      }
    }
    if (dS_out) {
      for (int j = 0; j < T; ++j) dS_out[(size_t)i * T + j] = j < n ? ds[j] : 0.0;
    }
    if (info) fill_rowinfo(&st, n, cM, cm, sself, info + (size_t)i * KIO_ROWINFO);
  }
  free(s); free(u); free(t); free(wL); free(wN); free(g); free(ds);
  free(r); free(l); free(tail);
}

static int check_cfg(const attn_cfg *c) {
  if (c->B <= 0 || c->H <= 0 || c->T <= 0 || c->d <= 0 || c->K < 1) return -1;
  if (c->calib < KIO_CALIB_MINMAX || c->calib > KIO_CALIB_RESOLVED) return -1;
  if (c->recon < 0 || c->recon > KIO_RECON_FP8EXP) return -1;
  if (c->calib != KIO_CALIB_MINMAX && !(c->tau > 0.0) && !is_exp_mode(c->recon))
    return -1;
  return 0;
}

/*
 * kio_attn_fwd: q,k,v [B,H,T,d] fp64 -> o [B,H,T,d]; ol (O^L) may be NULL;
 * info [B,H,T,KIO_ROWINFO] may be NULL; codes [B,H,T,T] may be NULL.
 * slice_lo/slice_hi restrict the work to (b,h) slices [lo,hi) of B*H (the
 * outputs of the other slices are left untouched). given [B,H,T,T] fp32
 * scores or NULL (see row_score). Parallel over rows.
 */
int kio_attn_fwd(const double *q, const double *k, const double *v, double *o,
                 double *ol, double *info, uint16_t *codes, int B, int H,
                 int T, int d, int K, int calib, double tau, int recon,
                 int causal, int round_scores, int slice_lo, int slice_hi,
                 const float *given) {
  attn_cfg c = {B, H, T, d, K, calib, recon, 0, 0, causal, round_scores, tau};
  if (check_cfg(&c)) return -1;
  if (slice_lo < 0) slice_lo = 0;
  if (slice_hi > B * H || slice_hi <= 0) slice_hi = B * H;
  const int RB = 16; /* rows per task */
  int nrb = (T + RB - 1) / RB;
  long ntask = (long)(slice_hi - slice_lo) * nrb;
#pragma omp parallel for schedule(dynamic, 1)
  for (long task = 0; task < ntask; ++task) {
    int sl = slice_lo + (int)(task / nrb);
    int rb = (int)(task % nrb);
    size_t off = (size_t)sl * T * d;
    attn_fwd_slice(&c, q + off, k + off, v + off,
                   given ? given + (size_t)sl * T * T : NULL, o + off, ol ? ol + off : NULL,
                   info ? info + (size_t)sl * T * KIO_ROWINFO : NULL,
                   codes ? codes + (size_t)sl * T * T : NULL, rb * RB,
                   (rb + 1) * RB < T ? (rb + 1) * RB : T);
  }
  return 0;
}

/*
 * kio_attn_bwd: gradients of L = sum(dO * O) w.r.t. q, k, v (fp64, [B,H,T,d]).
 * dS [B,H,T,T] and info [B,H,T,KIO_ROWINFO] may be NULL. Work on (b,h)
 * slices [slice_lo, slice_hi): parallel over slices when there are at least
 * as many slices as threads, otherwise over the rows of each slice with
 * per-thread dK/dV accumulators summed at the end. given as in
 * kio_attn_fwd.
 */
int kio_attn_bwd(const double *q, const double *k, const double *v,
                 const double *dO, double *dq, double *dk, double *dv,
                 double *dS, double *info, int B, int H, int T, int d, int K,
                 int calib, double tau, int recon, int ste, int grad,
                 int causal, int round_scores, int slice_lo, int slice_hi,
                 const float *given) {
  attn_cfg c = {B, H, T, d, K, calib, recon, ste, grad, causal, round_scores, tau};
  if (check_cfg(&c)) return -1;
  if (slice_lo < 0) slice_lo = 0;
  if (slice_hi > B * H || slice_hi <= 0) slice_hi = B * H;
  int nthr = omp_get_max_threads();
  if (slice_hi - slice_lo >= nthr) {
#pragma omp parallel for schedule(dynamic, 1)
    for (int sl = slice_lo; sl < slice_hi; ++sl) {
      size_t off = (size_t)sl * T * d;
      memset(dk + off, 0, sizeof(double) * (size_t)T * d);
      memset(dv + off, 0, sizeof(double) * (size_t)T * d);
      attn_bwd_rows(&c, q + off, k + off, v + off, dO + off,
                    given ? given + (size_t)sl * T * T : NULL, dq + off, dk + off,
                    dv + off, dS ? dS + (size_t)sl * T * T : NULL,
                    info ? info + (size_t)sl * T * KIO_ROWINFO : NULL, 0, T);
    }
    return 0;
  }
  const int RB = 8;  /* rows per task */
  for (int sl = slice_lo; sl < slice_hi; ++sl) {
    size_t off = (size_t)sl * T * d;
    memset(dk + off, 0, sizeof(double) * (size_t)T * d);
    memset(dv + off, 0, sizeof(double) * (size_t)T * d);
#pragma omp parallel
    {
      double *pk = calloc((size_t)T * d, sizeof(double));
      double *pv = calloc((size_t)T * d, sizeof(double));
#pragma omp for schedule(dynamic, 1)
      for (int rb = 0; rb < (T + RB - 1) / RB; ++rb) {
        int hi = (rb + 1) * RB < T ? (rb + 1) * RB : T;
        attn_bwd_rows(&c, q + off, k + off, v + off, dO + off,
                      given ? given + (size_t)sl * T * T : NULL, dq + off, pk, pv,
                      dS ? dS + (size_t)sl * T * T : NULL,
                      info ? info + (size_t)sl * T * KIO_ROWINFO : NULL, rb * RB, hi);
      }
#pragma omp critical
      {
        for (size_t e = 0; e < (size_t)T * d; ++e) {
          dk[off + e] += pk[e];
          dv[off + e] += pv[e];
        }
      }
      free(pk);
      free(pv);
    }
  }
  return 0;
}

int kio_rowinfo_len(void) { return KIO_ROWINFO; }

/* Threads the OpenMP runtime uses for the parallel loops above. */
int kio_max_threads(void) { return omp_get_max_threads(); }

/* ---------------------------------------------------------------------- */
/* Geometry probe (App. geometry-probe paragraph; Sec. 2 geometry probe).  */
/* ---------------------------------------------------------------------- */

#define KIO_GEO_COUNT 10
enum {
  GEO_SPAN = 0, GEO_H, GEO_ZQ, GEO_QNORM, GEO_KNORM, GEO_ENTROPY, GEO_FRAC6,
  GEO_TOPMASS, GEO_EFFB, GEO_TV
};

static int cmp_double(const void *a, const void *b) {
  double x = *(const double *)a, y = *(const double *)b;
  return (x > y) - (x < y);
}

/*
 * Per-row statistics of the probe, from the operator's own fp32 scores of
 * row i (valid keys j <= i, or all keys when not causal):
 *   span M - m; native width h ((M - m)/K under MinMax, tau/K under FWM);
 *   the 0.1% quantile of z = s - M over the row (sorted z, linear
 *   interpolation at position (n - 1) * 0.001); the norms of q_i and k_i;
 *   the entropy -sum P^E log P^E of the softmax P^E of the row's scores; the
 *   fraction of keys with z < -6; the top-bucket mass, the softmax mass on
 *   the keys in the operator's top level (Nearest: l = K) or top interval
 *   (LERP: r = K - 1); the effective bucket count exp H(q), q_b = sum of
 *   P^E over the keys of bucket b (the operator's level l for Nearest, its
 *   interval r for LERP, and one bucket for the FWM tail); and the total
 *   variation 1/2 sum_j |P^native_j - P^E_j| between the operator's forward
 *   probabilities and the softmax.
 * out [B,H,T,KIO_GEO_COUNT]. MinMax or FWM calibration, LERP or Nearest.
 */
int kio_geometry(const double *q, const double *k, double *out, int B, int H,
                 int T, int d, int K, int calib, double tau, int recon,
                 int causal) {
  if (B < 1 || H < 1 || T < 1 || d < 1 || K < 1) return -1;
  if (calib != KIO_CALIB_MINMAX && calib != KIO_CALIB_FWM) return -1;
  if (recon != KIO_RECON_LERP && recon != KIO_RECON_NEAREST) return -1;
  if (calib == KIO_CALIB_FWM && !(tau > 0.0)) return -1;
  double scale = score_scale(d, 1);
  long nrow = (long)B * H * T;
#pragma omp parallel
  {
    double *s = malloc(sizeof(double) * T), *u = malloc(sizeof(double) * T);
    double *t = malloc(sizeof(double) * T), *wL = malloc(sizeof(double) * T);
    double *wN = malloc(sizeof(double) * T), *z = malloc(sizeof(double) * T);
    double *pe = malloc(sizeof(double) * T);
    double *bucket = malloc(sizeof(double) * (K + 2));
    int *r = malloc(sizeof(int) * T), *l = malloc(sizeof(int) * T);
    int *tail = malloc(sizeof(int) * T);
#pragma omp for schedule(dynamic, 16)
    for (long row = 0; row < nrow; ++row) {
      int sl = (int)(row / T), i = (int)(row % T);
      const double *qs = q + (size_t)sl * T * d, *ks = k + (size_t)sl * T * d;
      int n = causal ? i + 1 : T;
      for (int j = 0; j < n; ++j)
        s[j] = score(qs + (size_t)i * d, ks + (size_t)j * d, d, scale, 1);
      row_state st;
      row_forward(n, s, K, calib, tau, recon, &st, r, l, tail, u, t, wL, wN);
      const double *w = (recon == KIO_RECON_NEAREST) ? wN : wL;
      double *o = out + (size_t)row * KIO_GEO_COUNT;
      o[GEO_SPAN] = st.M - st.m;
      o[GEO_H] = calib == KIO_CALIB_MINMAX ? (st.M - st.m) / (double)K : tau / (double)K;
      /* softmax of the row */
      double WE = 0.0;
      for (int j = 0; j < n; ++j) {
        z[j] = s[j] - st.M;
        pe[j] = exp(z[j]);
        WE += pe[j];
      }
      double H = 0.0, frac = 0.0, top = 0.0, tv = 0.0;
      for (int b = 0; b < K + 2; ++b) bucket[b] = 0.0;
      for (int j = 0; j < n; ++j) {
        pe[j] /= WE;
        if (pe[j] > 0.0) H -= pe[j] * log(pe[j]);
        if (z[j] < -6.0) frac += 1.0;
        int b = tail[j] ? K + 1 : (recon == KIO_RECON_NEAREST ? l[j] : r[j]);
        bucket[b] += pe[j];
        if (!tail[j] && (recon == KIO_RECON_NEAREST ? l[j] == K : r[j] == K - 1))
          top += pe[j];
        tv += fabs(w[j] / st.W - pe[j]);
      }
      double Hq = 0.0;
      for (int b = 0; b < K + 2; ++b)
        if (bucket[b] > 0.0) Hq -= bucket[b] * log(bucket[b]);
      o[GEO_ENTROPY] = H;
      o[GEO_FRAC6] = frac / (double)n;
      o[GEO_TOPMASS] = top;
      o[GEO_EFFB] = exp(Hq);
      o[GEO_TV] = 0.5 * tv;
      /* 0.1% quantile of z: sorted, linear interpolation */
      qsort(z, (size_t)n, sizeof(double), cmp_double);
      double pos = (double)(n - 1) * 0.001;
      int lo = (int)floor(pos);
      int hi = lo + 1 < n ? lo + 1 : lo;
      o[GEO_ZQ] = z[lo] + (pos - (double)lo) * (z[hi] - z[lo]);
      double qq = 0.0, kk = 0.0;
      for (int c = 0; c < d; ++c) {
        qq += qs[(size_t)i * d + c] * qs[(size_t)i * d + c];
        kk += ks[(size_t)i * d + c] * ks[(size_t)i * d + c];
      }
      o[GEO_QNORM] = sqrt(qq);
      o[GEO_KNORM] = sqrt(kk);
    }
    free(s); free(u); free(t); free(wL); free(wN); free(z); free(pe); free(bucket);
    free(r); free(l); free(tail);
  }
  return 0;
}

/*
 * kio_expw: the exponential weight function on n given fp32 shifts z
 * (recon 2 softmax, 3 BF16-exp, 4 FP8-exp). w[i], wE[i] and code[i] as in
 * exp_weight(); any output may be NULL. Returns 0, or -1 on bad arguments.
 */
int kio_expw(int n, const float *z, int recon, double *w, double *wE,
             int32_t *code) {
  if (n < 0 || z == NULL || !is_exp_mode(recon)) return -1;
  for (int i = 0; i < n; ++i) {
    double a, b;
    int c;
    exp_weight(z[i], recon, &a, &b, &c);
    if (w) w[i] = a;
    if (wE) wE[i] = b;
    if (code) code[i] = c;
  }
  return 0;
}
