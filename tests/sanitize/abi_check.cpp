// Sanitizer driver for the C ABI's host code (test infrastructure): linked
// with a host-sanitized build of paper_2609_33591_amd/csrc/kia_abi.hip and
// run by tests/test_sanitizers_host.py on a machine without a GPU. It covers
// the stats layout (sizes and offsets of every field, causal and not, with
// and without the bf16-output accumulators) and every argument check of
// every entry point: each call here is refused on the host before any HIP
// call, so no device is needed.
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "kia.h"

static int fails = 0;
#define CHECK(c)                                         \
  do {                                                   \
    if (!(c)) {                                          \
      fprintf(stderr, "check failed line %d: %s\n", __LINE__, #c); \
      ++fails;                                           \
    }                                                    \
  } while (0)

int main() {
  // layout
  const int shapes[][4] = {{1, 1, 1, 16}, {2, 3, 100, 64}, {1, 12, 1024, 64}, {3, 1, 77, 32},
                           {1, 2, 130, 128}, {1, 1, 65536, 16}};
  for (auto &sh : shapes)
    for (int causal = 0; causal < 2; ++causal)
      for (int recon = 0; recon < 5; ++recon)
        for (int ste = 0; ste < 2; ++ste) {
          size_t bytes = 0, big = 0, prev = 0;
          CHECK(kia_stats_bytes(sh[0], sh[1], sh[2], sh[3], recon, ste, causal, &bytes) == KIA_OK);
          CHECK(kia_stats_bytes_bf16o(sh[0], sh[1], sh[2], sh[3], recon, ste, causal, &big) ==
                KIA_OK);
          CHECK(big > bytes);
          for (int f = 0; f <= KIA_STAT_ACC; ++f) {
            size_t off = 1;
            CHECK(kia_stats_offset(sh[0], sh[1], sh[2], sh[3], recon, ste, causal, f, &off) ==
                  KIA_OK);
            CHECK(off % 256 == 0 && off >= prev && off <= bytes);
            prev = off;
          }
        }
  size_t b = 7;
  CHECK(kia_stats_bytes(0, 1, 1, 16, 0, 0, 1, &b) == KIA_ERR_SHAPE && b == 0);
  CHECK(kia_stats_bytes(1, 1, 65537, 16, 0, 0, 1, &b) == KIA_ERR_SHAPE);
  CHECK(kia_stats_bytes(65536, 65536, 65536, 128, 0, 0, 1, &b) == KIA_ERR_SHAPE);
  CHECK(kia_stats_bytes(1, 1, 1, 24, 0, 0, 1, &b) == KIA_ERR_HEADDIM);
  CHECK(kia_stats_bytes(1, 1, 1, 16, 5, 0, 1, &b) == KIA_ERR_ENUM);
  CHECK(kia_stats_bytes(1, 1, 1, 16, 0, 0, 1, nullptr) == KIA_ERR_NULL);
  CHECK(kia_stats_offset(1, 1, 1, 16, 0, 0, 1, KIA_STAT_ACC + 1, &b) == KIA_ERR_ENUM);
  CHECK(kia_stats_offset(1, 1, 1, 16, 0, 0, 1, -1, &b) == KIA_ERR_ENUM);

  // argument checks (all refused before any HIP call)
  alignas(256) static float buf[64];
  float *p = buf;
  uint16_t *h = reinterpret_cast<uint16_t *>(buf);
  float *mis = reinterpret_cast<float *>(reinterpret_cast<char *>(buf) + 4);
  void *st = buf, *stmis = reinterpret_cast<char *>(buf) + 16;
  const int B = 1, H = 1, T = 64, d = 16;
  struct Bad { int B, T, d, K, calib; float tau; int recon, ste, det, causal, rc; };
  const Bad bad[] = {{0, T, d, 4, 0, 8.f, 0, 0, 0, 1, KIA_ERR_SHAPE},
                     {B, 0, d, 4, 0, 8.f, 0, 0, 0, 1, KIA_ERR_SHAPE},
                     {B, T, 48, 4, 0, 8.f, 0, 0, 0, 1, KIA_ERR_HEADDIM},
                     {B, T, d, 0, 0, 8.f, 0, 0, 0, 1, KIA_ERR_K},
                     {B, T, d, 65, 0, 8.f, 0, 0, 0, 1, KIA_ERR_K},
                     {B, T, d, 4, 3, 8.f, 0, 0, 0, 1, KIA_ERR_ENUM},
                     {B, T, d, 4, 1, 0.f, 0, 0, 0, 1, KIA_ERR_TAU},
                     {B, T, d, 4, 2, -1.f, 1, 0, 0, 1, KIA_ERR_TAU},
                     {B, T, d, 4, 0, 8.f, 7, 0, 0, 1, KIA_ERR_ENUM},
                     {B, T, d, 4, 0, 8.f, 1, 2, 0, 1, KIA_ERR_ENUM},
                     {B, T, d, 4, 0, 8.f, 1, 0, 6, 1, KIA_ERR_ENUM},
                     {B, T, d, 4, 0, 8.f, 1, 0, 0, 2, KIA_ERR_ENUM}};
  for (const Bad &a : bad) {
    CHECK(kia_attn_fwd(p, p, p, p, st, a.B, H, a.T, a.d, a.K, a.calib, a.tau, a.recon, a.ste,
                       a.det, a.causal, nullptr) == a.rc);
    CHECK(kia_attn_bwd(p, p, p, p, p, st, p, p, p, a.B, H, a.T, a.d, a.K, a.calib, a.tau,
                       a.recon, a.ste, a.det, a.causal, nullptr) == a.rc);
    CHECK(kia_attn_fwd_bf16(h, h, h, p, st, a.B, H, a.T, a.d, a.K, a.calib, a.tau, a.recon,
                            a.ste, a.det, a.causal, nullptr) == a.rc);
    CHECK(kia_attn_bwd_bf16o(h, h, h, h, h, st, h, h, h, a.B, H, a.T, a.d, a.K, a.calib, a.tau,
                             a.recon, a.ste, a.det, a.causal, nullptr) == a.rc);
    CHECK(kia_attn_fwd_bwd_static(p, p, p, p, p, p, p, p, a.B, H, a.T, a.d, a.K, a.calib, a.tau,
                                  a.recon, a.ste, a.det, a.causal, nullptr) == a.rc);
    if (a.det == 0)  // the stored-codes export has no gradient mode
      CHECK(kia_debug_codes_stored(st, h, a.B, H, a.T, a.d, a.K, a.calib, a.tau, a.recon, a.ste,
                                   a.causal, nullptr) == a.rc);
  }
  CHECK(kia_attn_fwd(nullptr, p, p, p, st, B, H, T, d, 4, 0, 8.f, 0, 0, 0, 1, nullptr) ==
        KIA_ERR_NULL);
  // forward only (KIA_GRAD_NONE): the forward's checks pass, every backward refuses it
  CHECK(kia_attn_fwd(nullptr, p, p, p, st, B, H, T, d, 4, 1, 8.f, 1, 1, KIA_GRAD_NONE, 1,
                     nullptr) == KIA_ERR_NULL);
  CHECK(kia_attn_bwd(p, p, p, p, p, st, p, p, p, B, H, T, d, 4, 1, 8.f, 1, 1, KIA_GRAD_NONE, 1,
                     nullptr) == KIA_ERR_ENUM);
  CHECK(kia_attn_bwd_bf16(h, h, h, p, h, st, p, p, p, B, H, T, d, 4, 1, 8.f, 1, 1,
                          KIA_GRAD_NONE, 1, nullptr) == KIA_ERR_ENUM);
  CHECK(kia_attn_bwd_bf16o(h, h, h, h, h, st, h, h, h, B, H, T, d, 4, 1, 8.f, 1, 1,
                           KIA_GRAD_NONE, 1, nullptr) == KIA_ERR_ENUM);
  CHECK(kia_attn_fwd_bwd_static(p, p, p, p, p, p, p, p, B, H, T, d, 4, 1, 8.f, 1, 1,
                                KIA_GRAD_NONE, 1, nullptr) == KIA_ERR_ENUM);
  CHECK(kia_attn_bwd(p, p, p, p, p, st, p, nullptr, p, B, H, T, d, 4, 0, 8.f, 0, 0, 0, 1,
                     nullptr) == KIA_ERR_NULL);
  CHECK(kia_attn_fwd(p, p, mis, p, st, B, H, T, d, 4, 0, 8.f, 0, 0, 0, 1, nullptr) ==
        KIA_ERR_ALIGN);
  CHECK(kia_attn_fwd(p, p, p, p, stmis, B, H, T, d, 4, 0, 8.f, 0, 0, 0, 1, nullptr) ==
        KIA_ERR_ALIGN);
  CHECK(kia_attn_fwd_bf16(h, h, h, p, st, B, H, T, d, 4, 1, 8.f, 2, 0, 0, 1, nullptr) ==
        KIA_ERR_ENUM);  // exponential weight functions: fp32 inputs only
  CHECK(kia_attn_fwd_bf16o(h, h, h, nullptr, st, B, H, T, d, 4, 0, 8.f, 0, 0, 0, 1, nullptr) ==
        KIA_ERR_NULL);
  CHECK(kia_attn_bwd_bf16o(h, h, h, h, h, st, h, nullptr, h, B, H, T, d, 4, 0, 8.f, 0, 0, 0, 1,
                           nullptr) == KIA_ERR_NULL);
  CHECK(kia_attn_fwd_bwd_static(p, p, p, p, p, p, p, p, 8, 12, 1024, 64, 4, 1, 8.f, 1, 1, 0, 1,
                                nullptr) == KIA_ERR_SCRATCH);
  CHECK(kia_debug_codes(p, p, st, h, B, H, T, d, 0, 0, 8.f, 0, 1, nullptr) == KIA_ERR_K);
  CHECK(kia_debug_codes_bf16(h, h, st, nullptr, B, H, T, d, 4, 0, 8.f, 0, 1, nullptr) ==
        KIA_ERR_NULL);
  CHECK(kia_debug_scores(p, p, p, B, H, T, 20, 1, nullptr) == KIA_ERR_HEADDIM);
  CHECK(kia_debug_scores_bf16(h, nullptr, p, B, H, T, d, 1, nullptr) == KIA_ERR_NULL);
  CHECK(kia_debug_score_grad(st, 2, p, p, p, B, H, T, d, 0, 0, 0, 1, nullptr) == KIA_ERR_ENUM);
  CHECK(kia_geometry_probe(p, p, st, p, B, H, T, d, 4, 2, 8.f, 0, 1, nullptr) == KIA_ERR_ENUM);
  CHECK(kia_mfma_peak_probe(nullptr, 1, 1, nullptr) == KIA_ERR_NULL);
  CHECK(kia_mfma_peak_probe(reinterpret_cast<unsigned long long *>(buf), 0, 1, nullptr) ==
        KIA_ERR_SHAPE);
  CHECK(kia_set_grid_policy(3) == KIA_ERR_ENUM);
  CHECK(kia_set_grid_policy(KIA_GRID_AUTO) == KIA_OK);
  CHECK(kia_set_deterministic(2) == KIA_ERR_ENUM);
  CHECK(kia_set_deterministic(1) == KIA_OK && kia_set_deterministic(0) == KIA_OK);
  for (int c = -12; c <= 1; ++c) CHECK(kia_strerror(c) != nullptr && strlen(kia_strerror(c)) > 0);
  CHECK(kia_timing_enable(1) == KIA_OK && kia_timing_enable(0) == KIA_OK);
  double ms = -1;
  int n = -1;
  CHECK(kia_timing_read("kia_fwd", &ms, &n) == KIA_OK && n == 0 && ms == 0.0);
  CHECK(kia_timing_read(nullptr, &ms, &n) == KIA_ERR_NULL);
  if (fails) {
    fprintf(stderr, "%d checks failed\n", fails);
    return 1;
  }
  printf("abi host sanitizer run: ok\n");
  return 0;
}
