// kia_device.hpp -- device building blocks shared by every K-interval
// attention kernel for gfx950 (CDNA4, wave64, fp32 MFMA 32x32x2).
//
// Canonical score sub-tile. Every kernel that needs a score s_ij computes it
// with score_tile(): a 32-key x 32-query block of S^T accumulated by
// v_mfma_f32_32x32x2_f32 over d in one fixed order, with the key block and
// the query block aligned to multiples of 32. The A operand is K (rows =
// keys), the B operand Q (columns = queries). Lane l (half h = l/32) feeds,
// at k-step s, K[key0 + l%32][h*d/2 + s] and Q[query0 + l%32][h*d/2 + s].
// Output register r of lane l holds S^T[key0 + krel(r, h)][query0 + l%32]
// with krel(r, h) = 8*(r/4) + 4*h + r%4. Same operands, same instruction
// sequence, same lane/register position: the fp32 score of a pair is
// bit-identical in the forward's two passes, the backward and the tie path,
// which the exact extremum ties and index decisions rely on.
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

namespace kia {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

enum { CAL_MINMAX = 0, CAL_FWM = 1 };
enum { REC_LERP = 0, REC_NEAREST = 1 };
enum { STE_WEIGHT = 0, STE_PROB = 1 };

// Row record written by the backward's preprocessing (16 floats per row).
enum {
  RR_ALPHA = 0, RR_BETA, RR_MARGIN2, RR_HL, RR_B1L, RR_EMH, RR_DCOEF,
  RR_INVWF, RR_INVWX, RR_NEGDXW, RR_M, RR_m, RR_FLAGS, RR_COUNT = 16
};

// Device view of the caller's stats buffer (layout documented in kia.h).
struct Stats {
  float *M, *m, *W, *WL;
  int *amax, *amin, *nmax, *nmin;
  float *rowrec;  // [R][RR_COUNT]
  float *sself, *cM;
  float *OL;      // [R][d] or nullptr
  float *dS;      // backward scratch: dS_self in 32x32 tiles, 1024 floats each
};

__device__ __forceinline__ f32x16 mfma32(float a, float b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

// Column blocks of the PV-type products are 32 wide: d = 16 is padded to
// 32 zero columns in LDS and never stored.
template <int D> struct Dims {
  static constexpr int DP = D < 32 ? 32 : D;  // padded width
  static constexpr int NC = DP / 32;          // 32-wide column blocks
  static constexpr int DS = DP + 4;           // LDS row stride (floats)
  static constexpr int FWD_WAVES_PER_EU = D <= 64 ? 2 : 1;
};

__device__ __forceinline__ int krel(int r, int half) {
  return 8 * (r >> 2) + 4 * half + (r & 3);
}

// S^T sub-tile: kop[s], qop[s] as described above; returns raw q.k sums.
template <int D>
__device__ __forceinline__ f32x16 score_tile(const float (&kop)[D / 2],
                                             const float (&qop)[D / 2]) {
  f32x16 acc;
#pragma unroll
  for (int e = 0; e < 16; ++e) acc[e] = 0.f;
#pragma unroll
  for (int s = 0; s < D / 2; ++s) acc = mfma32(kop[s], qop[s], acc);
  return acc;
}

// Per-row constants of the fast index/weight evaluation.
//   u_fast = fma(acc, alpha, beta) approximates u (MinMax (K(s-m))/(M-m),
//   FWM K(s-M+tau)/tau) within margin2/2 (worst-case rounding bound x8);
//   E_{r+1} = exp2(r*hl + b1l) = e^{b_{r+1}}, E_r = E_{r+1} * emh (emh =
//   e^{-h}), Delta_r = E_{r+1} * dcoef (dcoef = (1 - e^{-h})/h).
// Degenerate MinMax rows (M - m <= 1e-12, App. A) map every key to u = K
// with all weights 1 and Delta = 0.
struct RowConst {
  float alpha, beta, margin2, hl, b1l, emh, dcoef;
  bool degen;
};

__device__ inline RowConst row_const(float M, float m, int K, int calib,
                                     float tau, float scale) {
  RowConst rc;
  const double Kd = (double)K;
  const double LOG2E = 1.4426950408889634074;
  double h, zlo;
  rc.degen = false;
  if (calib == CAL_MINMAX) {
    const double span = (double)M - (double)m;
    if (span <= 1e-12) {
      rc.degen = true;
      rc.alpha = 0.f; rc.beta = (float)K; rc.margin2 = 0.f;
      rc.hl = 0.f; rc.b1l = 0.f; rc.emh = 1.f; rc.dcoef = 0.f;
      return rc;
    }
    const double c = Kd / span;
    rc.alpha = (float)(c * (double)scale);
    rc.beta = (float)(-(double)m * c);
    const double A = fmax(fabs((double)M), fabs((double)m));
    rc.margin2 = (float)ldexp(3.0 * c * A + Kd, -20);
    h = span / Kd;
    zlo = (double)m - (double)M;
  } else {
    const double t = (double)tau;
    const double c = Kd / t;
    rc.alpha = (float)(c * (double)scale);
    rc.beta = (float)(Kd - (double)M * c);
    const double A = fabs((double)M) + t;
    rc.margin2 = (float)ldexp(3.0 * c * A + 2.0 * Kd, -20);
    h = t / Kd;
    zlo = -t;
  }
  rc.hl = (float)(h * LOG2E);
  rc.b1l = (float)((zlo + h) * LOG2E);
  rc.emh = (float)exp(-h);
  rc.dcoef = (float)(-expm1(-h) / h);
  return rc;
}

// Exact index decision on the fp32 score s (fp64 expressions of kia.h).
__device__ __forceinline__ void exact_decision(float s, float M, float m, int K,
                                            int calib, float tau, float &rf,
                                            int &up, int &tail) {
#pragma clang fp contract(off)
  double u;
  tail = 0;
  if (calib == CAL_MINMAX) {
    u = ((double)K * ((double)s - (double)m)) / ((double)M - (double)m);
  } else {
    const double a = ((double)s - (double)M) + (double)tau;
    if (a < 0.0) {
      tail = 1; rf = 0.f; up = 0;
      return;
    }
    u = ((double)K * a) / (double)tau;
  }
  double r = floor(u);
  if (r < 0.0) r = 0.0;
  if (r > (double)(K - 1)) r = (double)(K - 1);
  double t = u - r;
  if (t < 0.0) t = 0.0;
  if (t > 1.0) t = 1.0;
  rf = (float)r;
  up = t >= 0.5 ? 1 : 0;
}

// Index decisions of the 16 keys a lane holds in one score sub-tile.
// acc: raw sums; outputs per register: rf (interval, as float), t (position
// in the interval), up (l = r + up), tail (FWM cut). Keys whose fast u lies
// within the rounding margin of an interior integer/half-integer are decided
// by exact_decision(), one key per lane per round (rare; ~1e-5 of keys).
struct Decided {
  float rf[16], t[16];
  uint32_t up, tail;  // bit r
};

__device__ __forceinline__ void decide16(const f32x16 &acc, const RowConst &rc,
                                         float M, float m, int K, int calib,
                                         float tau, float scale, Decided &dd) {
  const float Kf = (float)K;
  const float lo = (calib == CAL_FWM) ? 0.f : 1.f;
  const float hi = 2.f * Kf - 1.f;
  uint32_t amb = 0;
  dd.up = 0; dd.tail = 0;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const float u = fmaf(acc[r], rc.alpha, rc.beta);
    const float v2 = u + u;
    const float n = rintf(v2);
    const bool a = (fabsf(v2 - n) <= rc.margin2) & (n >= lo) & (n <= hi);
    amb |= (a ? 1u : 0u) << r;
    const float rf = fminf(fmaxf(floorf(u), 0.f), Kf - 1.f);
    dd.rf[r] = rf;
    const float t = fminf(fmaxf(u - rf, 0.f), 1.f);
    dd.up |= (t >= 0.5f ? 1u : 0u) << r;
    dd.tail |= (((calib == CAL_FWM) & (u < 0.f)) ? 1u : 0u) << r;
  }
  while (__any(amb != 0)) {
    const int r0 = amb ? __builtin_ctz(amb) : 0;
    float x = acc[0];
#pragma unroll
    for (int r = 1; r < 16; ++r) x = (r0 == r) ? acc[r] : x;
    float rf; int up, tl;
    exact_decision(x * scale, M, m, K, calib, tau, rf, up, tl);
    if (amb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) dd.rf[r] = (r0 == r) ? rf : dd.rf[r];
      dd.up = (dd.up & ~(1u << r0)) | ((uint32_t)up << r0);
      dd.tail = (dd.tail & ~(1u << r0)) | ((uint32_t)tl << r0);
      amb &= amb - 1u;
    }
  }
#pragma unroll
  for (int r = 0; r < 16; ++r)
    dd.t[r] = fminf(fmaxf(fmaf(acc[r], rc.alpha, rc.beta) - dd.rf[r], 0.f), 1.f);
}

// e^{b_{r+1}} = 2^(r*hl + b1l): the raw v_exp_f32 (arguments are <= 0;
// results below the normal range flush to 0, which only drops weights
// below 1e-38 relative to the row maximum's weight 1).
__device__ __forceinline__ float grid_upper(float rf, const RowConst &rc) {
  return __builtin_amdgcn_exp2f(fmaf(rf, rc.hl, rc.b1l));
}

// Workgroup barrier ordering LDS only: outstanding global stores and
// atomics are not waited for.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Tile index of the dS scratch (32x32 sub-tiles, causal: kt <= qt only).
__host__ __device__ inline size_t ds_tiles_per_slice(int nq, int causal) {
  return causal ? (size_t)nq * (nq + 1) / 2 : (size_t)nq * nq;
}
__device__ __forceinline__ size_t ds_tile(int bh, int qt, int kt, int nq,
                                          int causal) {
  const size_t in = causal ? (size_t)qt * (qt + 1) / 2 + kt : (size_t)qt * nq + kt;
  return (size_t)bh * ds_tiles_per_slice(nq, causal) + in;
}

// Stats view from the caller's buffer (offsets as kia_stats_offset()).
__host__ __device__ inline size_t align256(size_t x) {
  return (x + 255) & ~(size_t)255;
}

}  // namespace kia
