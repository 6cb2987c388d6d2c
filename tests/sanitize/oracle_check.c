/*
 * Sanitizer driver for the fp64 oracle (test infrastructure): built together
 * with oracle/kia_oracle.c under AddressSanitizer and UndefinedBehavior-
 * Sanitizer (host code only) and run by tests/test_sanitizers_host.py. It
 * calls every exported entry point on small inputs over every calibration,
 * weight function, surrogate, gradient mode and causal setting (ragged
 * lengths, single-key rows, constant rows, given scores) and checks that the
 * results are finite and that each forward row of P sums to 1.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int kio_row(int n, const double *s, const double *g, int K, int calib, double tau, int recon,
            int ste, int grad, double *P, double *wL, double *wN, int32_t *r, int32_t *l,
            int32_t *tail, double *u, double *dS, double *info);
int kio_attn_fwd(const double *q, const double *k, const double *v, double *o, double *ol,
                 double *info, uint16_t *codes, int B, int H, int T, int d, int K, int calib,
                 double tau, int recon, int causal, int round_scores, int slice_lo,
                 int slice_hi, const float *given);
int kio_attn_bwd(const double *q, const double *k, const double *v, const double *dO,
                 double *dq, double *dk, double *dv, double *dS, double *info, int B, int H,
                 int T, int d, int K, int calib, double tau, int recon, int ste, int grad,
                 int causal, int round_scores, int slice_lo, int slice_hi, const float *given);
int kio_geometry(const double *q, const double *k, double *out, int B, int H, int T, int d,
                 int K, int calib, double tau, int recon, int causal);
int kio_expw(int n, const float *z, int recon, double *w, double *wE, int32_t *code);
int kio_max_threads(void);

static uint64_t state = 12345;
static double uniform(void) {  /* 64-bit LCG, top 53 bits */
  state = state * 6364136223846793005ull + 1442695040888963407ull;
  return (double)(state >> 11) * (1.0 / 9007199254740992.0);
}
static double normal(void) {
  double a = uniform() + 1e-300, b = uniform();
  return sqrt(-2.0 * log(a)) * cos(6.283185307179586 * b);
}

static int fails = 0;
#define CHECK(c, msg)                                      \
  do {                                                     \
    if (!(c)) {                                            \
      fprintf(stderr, "check failed: %s (%s)\n", msg, #c); \
      ++fails;                                             \
    }                                                      \
  } while (0)

static int finite_all(const double *x, size_t n) {
  for (size_t i = 0; i < n; ++i)
    if (!isfinite(x[i])) return 0;
  return 1;
}

int main(void) {
  CHECK(kio_max_threads() >= 1, "threads");
  /* rows */
  for (int n = 1; n <= 40; n += 13) {
    double *s = malloc(sizeof(double) * n), *g = malloc(sizeof(double) * n);
    double *P = malloc(sizeof(double) * n), *wL = malloc(sizeof(double) * n);
    double *wN = malloc(sizeof(double) * n), *u = malloc(sizeof(double) * n);
    double *dS = malloc(sizeof(double) * n), info[16];
    int32_t *r = malloc(sizeof(int32_t) * n), *l = malloc(sizeof(int32_t) * n);
    int32_t *tl = malloc(sizeof(int32_t) * n);
    for (int shape = 0; shape < 3; ++shape) {
      for (int j = 0; j < n; ++j) {
        s[j] = shape == 0 ? (double)(float)(3.0 * normal()) : (shape == 1 ? 0.5 : (j % 2) * 1e-13);
        g[j] = normal();
      }
      for (int calib = 0; calib < 3; ++calib)
        for (int recon = 0; recon < 5; ++recon)
          for (int ste = 0; ste < 2; ++ste)
            for (int grad = 0; grad < 5; ++grad)
              for (int K = 1; K <= 16; K *= 4) {
                int rc = kio_row(n, s, g, K, calib, 6.0, recon, ste, grad, P, wL, wN, r, l, tl,
                                 u, dS, info);
                CHECK(rc == 0, "kio_row");
                double sum = 0.0;
                for (int j = 0; j < n; ++j) sum += P[j];
                CHECK(fabs(sum - 1.0) < 1e-12, "row sums to 1");
                CHECK(finite_all(dS, n) && finite_all(P, n), "row finite");
              }
    }
    CHECK(kio_row(n, s, g, 0, 0, 6.0, 0, 0, 0, P, wL, wN, r, l, tl, u, dS, info) != 0,
          "K = 0 rejected");
    free(s); free(g); free(P); free(wL); free(wN); free(u); free(dS); free(r); free(l); free(tl);
  }
  /* attention: ragged T, every head size class, given scores */
  const int B = 1, H = 2, T = 37, d = 16;
  size_t nx = (size_t)B * H * T * d, ns = (size_t)B * H * T * T;
  double *q = malloc(sizeof(double) * nx), *k = malloc(sizeof(double) * nx);
  double *v = malloc(sizeof(double) * nx), *dO = malloc(sizeof(double) * nx);
  double *o = malloc(sizeof(double) * nx), *ol = malloc(sizeof(double) * nx);
  double *dq = malloc(sizeof(double) * nx), *dk = malloc(sizeof(double) * nx);
  double *dv = malloc(sizeof(double) * nx), *dS = malloc(sizeof(double) * ns);
  double *info = malloc(sizeof(double) * B * H * T * 16), *geo = malloc(sizeof(double) * B * H * T * 10);
  uint16_t *codes = malloc(sizeof(uint16_t) * ns);
  float *given = malloc(sizeof(float) * ns);
  for (size_t i = 0; i < nx; ++i) {
    q[i] = 2.0 * normal(); k[i] = normal(); v[i] = normal(); dO[i] = normal();
  }
  for (size_t i = 0; i < ns; ++i) given[i] = (float)(4.0 * normal());
  for (int causal = 0; causal < 2; ++causal)
    for (int calib = 0; calib < 3; ++calib)
      for (int recon = 0; recon < 5; ++recon)
        for (int gv = 0; gv < 2; ++gv) {
          const float *gs = gv ? given : NULL;
          CHECK(kio_attn_fwd(q, k, v, o, ol, info, codes, B, H, T, d, 4, calib, 8.0, recon,
                             causal, 1, 0, B * H, gs) == 0, "fwd");
          CHECK(finite_all(o, nx) && finite_all(ol, nx), "fwd finite");
          for (int grad = 0; grad < 5; ++grad) {
            CHECK(kio_attn_bwd(q, k, v, dO, dq, dk, dv, dS, info, B, H, T, d, 4, calib, 8.0,
                               recon, grad & 1, grad, causal, 1, 0, B * H, gs) == 0, "bwd");
            CHECK(finite_all(dq, nx) && finite_all(dk, nx) && finite_all(dv, nx), "bwd finite");
          }
          if (calib < 2 && recon < 2)
            CHECK(kio_geometry(q, k, geo, B, H, T, d, 4, calib, 8.0, recon, causal) == 0, "geo");
        }
  /* one slice only (the row-parallel backward with per-thread partials) */
  CHECK(kio_attn_bwd(q, k, v, dO, dq, dk, dv, NULL, NULL, B, H, T, d, 4, 0, 8.0, 0, 0, 0, 1, 0,
                     1, 2, NULL) == 0, "bwd slice");
  CHECK(kio_attn_fwd(q, k, v, o, NULL, NULL, NULL, B, H, T, d, 0, 0, 8.0, 0, 1, 1, 0, 1,
                     NULL) != 0, "fwd rejects K = 0");
  float z[64];
  double w[64], wE[64];
  int32_t code[64];
  for (int i = 0; i < 64; ++i) z[i] = -(float)i * 0.75f;
  for (int recon = 2; recon < 5; ++recon)
    CHECK(kio_expw(64, z, recon, w, wE, code) == 0 && finite_all(w, 64), "expw");
  CHECK(kio_expw(64, z, 0, w, wE, code) != 0, "expw rejects a grid recon");
  free(q); free(k); free(v); free(dO); free(o); free(ol); free(dq); free(dk); free(dv);
  free(dS); free(info); free(geo); free(codes); free(given);
  if (fails) {
    fprintf(stderr, "%d checks failed\n", fails);
    return 1;
  }
  printf("oracle sanitizer run: ok\n");
  return 0;
}
