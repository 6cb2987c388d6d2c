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
// bit-identical wherever it is computed (the forward's extrema pass, whose
// tiles the second pass and the backward reuse, the tie path and the debug
// codes), which the exact extremum ties and index decisions rely on.
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

namespace kia {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// CAL_RESOLVED: the tail-policy diagnostic (FWM's step tau/K and origin -tau,
// the grid continued below -tau with negative intervals, no zero tail)
enum { CAL_MINMAX = 0, CAL_FWM = 1, CAL_RESOLVED = 2 };
// K-interval reconstructions, then the exponential weight functions of the
// baselines: exact softmax (App. A) and the reduced-precision exponentials
// BF16-exp and FP8 (E4M3)-rounded exp (App. D). The latter three use only
// the row maximum (z = s - M) and no grid.
enum { REC_LERP = 0, REC_NEAREST = 1, REC_SOFTMAX = 2, REC_BF16EXP = 3, REC_FP8EXP = 4 };
__host__ __device__ constexpr bool is_exp_rec(int r) { return r >= REC_SOFTMAX; }
enum { STE_WEIGHT = 0, STE_PROB = 1 };

// Row record written by the backward's preprocessing (16 floats per row).
// RR_B1LW = b1l - log2 W: exp2(r hl + b1lw) = e^{b_{r+1}} / W, so the forward
// probability comes out of the exponential directly; RR_C1, RR_C0: gamma
// Delta = (g c1 + c0) e^{b_{r+1}} / W with c1 = dcoef W / W^X and
// c0 = -dcoef W D^X / W^X.
enum {
  RR_ALPHA = 0, RR_BETA, RR_MARGIN2, RR_HL, RR_B1L, RR_EMH, RR_DCOEF,
  RR_INVWF, RR_INVWX, RR_NEGDXW, RR_M, RR_m, RR_FLAGS, RR_B1LW, RR_C1, RR_C0,
  RR_COUNT = 16
};

// Device view of the caller's stats buffer (layout documented in kia.h).
struct Stats {
  float *M, *m, *W, *WL;
  int *amax, *amin, *nmax, *nmin;
  float *rowrec;  // [R][RR_COUNT]
  float *sself, *cM;
  float *OL;      // [R][d] or nullptr
  float *dS;      // backward scratch: dS in 32x32 tiles, 1024 floats each
  float *U;       // forward -> backward: raw scores, then decided u, same tiles
  float *part;    // deterministic backward: row-sum partials [2][ceil(T/128)][R],
                  // then the calibration records [R][4] of the dK gather
};

// Deterministic backward: a row's calibration record for the dK gather, as
// the dQ kernel's epilogue decides it: {argmax key or -1, scale cM, argmin
// key or -1, scale cm} (-1: the row is not one with unique extrema, or the
// channel is not taken).
__device__ __forceinline__ void put_calib_record(float *part, size_t ridx, bool ok, bool minmax,
                                                 int am, int an, float fM, float fm) {
  reinterpret_cast<f32x4 *>(part)[ridx] =
      f32x4{ok ? (float)am : -1.f, fM, (ok && minmax) ? (float)an : -1.f, fm};
}

// The row sums of one 128-key block's score gradients (S_self, and cM under
// MinMax): added atomically, or, in the deterministic backward, stored as
// the block's partial for a sum in key-block order.
template <typename A>
__device__ __forceinline__ void put_row_sums(const A &a, int kb, size_t ridx, float s,
                                             float mm, bool minmax) {
  if (a.det) {
    const size_t R = (size_t)a.BH * a.T;
    const int nkb = (a.T + 127) / 128;
    a.st.part[(size_t)kb * R + ridx] = s;
    if (minmax) a.st.part[(size_t)(nkb + kb) * R + ridx] = mm;
  } else {
    atomicAdd(a.st.sself + ridx, s);
    if (minmax) atomicAdd(a.st.cM + ridx, mm);
  }
}

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

// Folds one score sub-tile into a lane's running extremum X with its first
// key index ax and its count cx. sv holds the lane's 16 scores, invalid keys
// set to -inf (maximum) or +inf (minimum); a lane's keys grow with r and
// the tiles come in increasing key order, so the first index of a tie is
// the one already held. One tile extremum, then one sweep for the count and
// the first position of it.
template <bool MAX>
__device__ __forceinline__ void tile_extremum(const float (&sv)[16], int js, int half,
                                              float &X, int &ax, int &cx) {
  float tm = sv[0];
#pragma unroll
  for (int r = 1; r < 16; ++r) tm = MAX ? fmaxf(tm, sv[r]) : fminf(tm, sv[r]);
  int tc = 0, tf = 0;
#pragma unroll
  for (int r = 15; r >= 0; --r) {
    const bool e = sv[r] == tm;
    tc += e ? 1 : 0;
    tf = e ? r : tf;
  }
  const bool some = MAX ? (tm != -INFINITY) : (tm != INFINITY);  // a valid key
  const bool take = some & (MAX ? (tm > X) : (tm < X));
  const bool tie = some & (tm == X);
  ax = take ? js + krel(tf, half) : ax;
  cx = take ? tc : (tie ? cx + tc : cx);
  X = take ? tm : X;
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
    // FWM decides window keys only (|s| <= |M| + tau); the resolved grid
    // decides every key, down to m, where |u| reaches c (M - m) + K
    const double A = calib == CAL_RESOLVED
                         ? fmax(fabs((double)M), fabs((double)m)) + t + ((double)M - (double)m)
                         : fabs((double)M) + t;
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

// The grid constants the backward uses (hl, b1l, emh, dcoef of RowConst),
// in fp32 except the degenerate test, which must be the forward's
// (fp64 span <= 1e-12). A few ulp from row_const's fp64-derived values.
__device__ inline void grid_consts(float M, float m, int K, int calib, float tau,
                                   float &hl, float &b1l, float &emh, float &dcoef,
                                   bool &degen) {
  const float LOG2E = 1.44269504f;
  float h, zlo;
  degen = false;
  if (calib == CAL_MINMAX) {
    if ((double)M - (double)m <= 1e-12) {
      degen = true;
      hl = 0.f; b1l = 0.f; emh = 1.f; dcoef = 0.f;
      return;
    }
    zlo = m - M;
    h = -zlo / (float)K;
  } else {
    zlo = -tau;
    h = tau / (float)K;
  }
  hl = h * LOG2E;
  b1l = (zlo + h) * LOG2E;
  emh = expf(-h);
  dcoef = -expm1f(-h) / h;
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
  } else if (calib == CAL_RESOLVED) {
    u = ((double)K * (((double)s - (double)M) + (double)tau)) / (double)tau;
  } else {
    const double a = ((double)s - (double)M) + (double)tau;
    if (a < 0.0) {
      tail = 1; rf = 0.f; up = 0;
      return;
    }
    u = ((double)K * a) / (double)tau;
  }
  double r = floor(u);
  if (r < 0.0 && calib != CAL_RESOLVED) r = 0.0;  // the resolved grid has no lower end
  if (r > (double)(K - 1)) r = (double)(K - 1);
  double t = u - r;
  if (t < 0.0) t = 0.0;
  if (t > 1.0) t = 1.0;
  rf = (float)r;
  up = t >= 0.5 ? 1 : 0;
}

// Index decisions of the 16 keys a lane holds in one score sub-tile, kept
// as one fp32 position u per key (r, t, l and the FWM tail are re-derived
// from u by key_of()). Fast path: u = fma(acc, alpha, beta). A key whose u
// lies within the rounding margin of an interior integer/half-integer
// (~1e-5 of keys) is decided by exact_decision() and its u is clamped into
// the interval of that decision (one key per lane per round), so that
// key_of() reproduces the exact decision and t stays within the margin.
template <int CALIB>
__device__ __forceinline__ bool is_ambiguous(float u, float margin2, float hi) {
  const float v2 = u + u;
  // boundaries 2u = n: MinMax 1 <= n <= 2K-1 (u = 0 is the argmin itself),
  // FWM and resolved n <= 2K-1 (FWM: the cut u = 0 and above; keys far in
  // the FWM tail near a negative half-integer only take the exact path).
  // Clamping 2u into [3/4, 2K - 3/4] keeps every such n and puts 2u = 0 and
  // 2u = 2K (the extrema themselves) a quarter away from any integer.
  const float c = CALIB == CAL_MINMAX ? __builtin_amdgcn_fmed3f(v2, 0.75f, hi + 0.25f)
                                      : fminf(v2, hi + 0.25f);
  return fabsf(c - rintf(c)) <= margin2;
}

// A float strictly below the boundary x (a multiple of 1/2 of either sign),
// within two ulp of it (2^-24 below x = 0).
__device__ __forceinline__ float below(float x) {
  return x - fmaxf(fabsf(x) * 0x1p-23f, 0x1p-24f);
}

template <int CALIB>
__device__ __forceinline__ void fix_ambiguous(const f32x16 &acc, const RowConst &rc,
                                           float M, float m, int K, float tau,
                                           float scale, float (&u)[16]) {
  const float Kf = (float)K, hi = 2.f * Kf - 1.f;
  uint32_t amb = 0;
#pragma unroll
  for (int r = 0; r < 16; ++r)
    amb |= (is_ambiguous<CALIB>(u[r], rc.margin2, hi) ? 1u : 0u) << r;
  while (__any(amb != 0)) {
    const int r0 = amb ? __builtin_ctz(amb) : 0;
    float x = acc[0], uu = u[0];
#pragma unroll
    for (int r = 1; r < 16; ++r) {
      x = (r0 == r) ? acc[r] : x;
      uu = (r0 == r) ? u[r] : uu;
    }
    float rf; int up, tl;
    exact_decision(x * scale, M, m, K, CALIB, tau, rf, up, tl);
    float lo = rf + (up ? 0.5f : 0.f);
    float hv = (up && rf == Kf - 1.f) ? Kf : below(rf + (up ? 1.f : 0.5f));
    const float uf = tl ? -1.f : fminf(fmaxf(uu, lo), hv);
    if (amb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) u[r] = (r0 == r) ? uf : u[r];
      amb &= amb - 1u;
    }
  }
}

template <int CALIB>
__device__ __forceinline__ void decide_u(const f32x16 &acc, const RowConst &rc,
                                         float M, float m, int K, float tau,
                                         float scale, float (&u)[16]) {
  const float hi = 2.f * (float)K - 1.f;
  bool any = false;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    u[r] = fmaf(acc[r], rc.alpha, rc.beta);
    any |= is_ambiguous<CALIB>(u[r], rc.margin2, hi);
  }
  if (__any(any)) fix_ambiguous<CALIB>(acc, rc, M, m, K, tau, scale, u);
}

// Interval r (as float), position t, level bit and FWM tail of a key from u.
struct KeyDec {
  float rf, t;
  bool up, tail;
};
template <int CALIB>
__device__ __forceinline__ KeyDec key_of(float u, float Kf) {
  KeyDec k;
  const float fl = floorf(u);
  // MinMax: u can round a hair below 0 at the argmin; FWM keys below 0 are
  // the tail (zero weight) and the resolved grid has no lower end
  k.rf = fminf(CALIB == CAL_MINMAX ? fmaxf(fl, 0.f) : fl, Kf - 1.f);
  k.t = fminf(fmaxf(u - k.rf, 0.f), 1.f);
  k.up = k.t >= 0.5f;
  k.tail = (CALIB == CAL_FWM) && (u < 0.f);
  return k;
}

// Stored decisions in compact form. Under FWM with Nearest the backward
// needs of a key only its interval r, its level bit [t >= 1/2] and the tail
// (P^N and gamma Delta_r take no t, and FWM has no minimum channel), so the
// second pass keeps one byte per key, 1 + 2r + [t >= 1/2] for a window key
// and 0 for the tail, in the first KiB of the pair's U tile (lane l's 16
// keys at bytes 16 l + r, r the register) instead of the fp32 position u.
template <int CALIB, int RECON>
__host__ __device__ constexpr bool compact_codes() {
  return CALIB == CAL_FWM && RECON == REC_NEAREST;
}

// The byte of a decided key (exact small integer as a float): tail keys
// (FWM: rf <= -1) give a value <= 0, stored as 0.
__device__ __forceinline__ float code_value(const KeyDec &kd) {
  return fmaxf(fmaf(kd.rf, 2.f, kd.up ? 2.f : 1.f), 0.f);
}

// Register r's byte into the lane's four code words (packed as the keys
// are decided, so that only four words stay live).
// v_cvt_pk_u8_f32 converts and inserts one byte; the values are exact
// integers in [0, 2K], so its rounding and saturation do not matter.
__device__ __forceinline__ void code_put(uint32_t (&w)[4], int r, const KeyDec &kd) {
  w[r >> 2] = __builtin_amdgcn_cvt_pk_u8_f32(code_value(kd), r & 3, (r & 3) ? w[r >> 2] : 0u);
}

// The lane's 16 bytes of the tile (one 16-byte store).
__device__ __forceinline__ void codes_store(float *tile, int lane, const uint32_t (&w)[4]) {
  *reinterpret_cast<uint4 *>(reinterpret_cast<char *>(tile) + 16 * lane) =
      make_uint4(w[0], w[1], w[2], w[3]);
}

__device__ __forceinline__ uint4 codes_load(const float *tile, int lane) {
  return *reinterpret_cast<const uint4 *>(reinterpret_cast<const char *>(tile) + 16 * lane);
}

// Interval, level bit and tail of register r from the lane's code words
// (t is 1 for the upper level and 0 otherwise: Nearest uses no more).
__device__ __forceinline__ KeyDec key_of_code(const uint4 &w, int r) {
  const uint32_t word = r < 4 ? w.x : (r < 8 ? w.y : (r < 12 ? w.z : w.w));
  const float cf = (float)((word >> (8 * (r & 3))) & 0xFFu);
  const float h = fmaf(cf, 0.5f, -0.5f);  // r + up / 2
  KeyDec k;
  k.rf = floorf(h);
  k.up = h - k.rf > 0.25f;
  k.t = k.up ? 1.f : 0.f;
  k.tail = cf < 0.5f;
  return k;
}

// e^{b_{r+1}} = 2^(r*hl + b1l): the raw v_exp_f32 (arguments are <= 0;
// results below the normal range flush to 0, which only drops weights
// below 1e-38 relative to the row maximum's weight 1).
__device__ __forceinline__ float grid_upper(float rf, const RowConst &rc) {
  return __builtin_amdgcn_exp2f(fmaf(rf, rc.hl, rc.b1l));
}

// ---- exponential weight functions (softmax, BF16-exp, FP8-exp) ----------
// The shift of a key from the row maximum, z = fl32(s - M) with the fp32
// score s = fl32(acc * scale): two roundings, never contracted into an fma.
__device__ __forceinline__ float score_shift(float acc, float scale, float M) {
#pragma clang fp contract(off)
  const float s = acc * scale;
  return s - M;
}

// fp32 -> bfloat16, round to nearest even, as the fp32 value with the low
// 16 bits clear (finite inputs).
__device__ __forceinline__ float bf16_rne(float x) {
  uint32_t b = __float_as_uint(x);
  b += 0x7FFFu + ((b >> 16) & 1u);
  return __uint_as_float(b & 0xFFFF0000u);
}

// Two fp32 values as one word of two bf16 (round to nearest even; a in the
// low half).
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  return (__float_as_uint(bf16_rne(a)) >> 16) | (__float_as_uint(bf16_rne(b)) & 0xFFFF0000u);
}

// Non-negative fp32 x (<= 448) -> float8_e4m3fn, round to nearest even.
// Below 2^-6 the grid is m * 2^-9 (subnormal codes m = 0..7; m = 8 is the
// smallest normal 2^-6, code 0x08); above, 3 mantissa bits with exponent
// bias 7. Returns the value; `code` receives the E4M3 byte.
__device__ __forceinline__ float e4m3_rne(float x, uint32_t &code) {
  if (x < 0x1p-6f) {
    const float m = rintf(x * 512.f);
    code = (uint32_t)m;
    return m * 0x1p-9f;
  }
  uint32_t b = __float_as_uint(x);
  b += 0x7FFFFu + ((b >> 20) & 1u);
  b &= 0xFFF00000u;
  code = (((b >> 23) - 120u) << 3) | ((b >> 20) & 7u);
  return __uint_as_float(b);
}

// Is the fp32 exponential e within the error of the fast expf() (a few
// ulp; the test window is 16 ulp) of a rounding midpoint of the target
// format? Then the rounding is decided on the correctly rounded value
// fl32(exp(x)) from the fp64 exponential instead. BF16-exp also sends
// results below the normal range there (their bf16 codes are subnormal).
template <int RECON>
__device__ __forceinline__ bool exp_near_tie(float e) {
  if constexpr (RECON == REC_BF16EXP) {
    const uint32_t lo = __float_as_uint(e) & 0xFFFFu;
    return (lo - 0x7FF0u <= 0x20u) | (e < 0x1p-126f);
  } else if constexpr (RECON == REC_FP8EXP) {
    if (e < 0x1p-6f) {
      const float y = e * 512.f;
      return fabsf(y - floorf(y) - 0.5f) <= 0x1p-16f;
    }
    const uint32_t m = __float_as_uint(e) & 0xFFFFFu;
    return m - 0x7FFF0u <= 0x20u;
  } else {
    return false;
  }
}

// Argument of the exponential: z, or bf16(z) for BF16-exp.
template <int RECON>
__device__ __forceinline__ float exp_arg(float z) {
  return RECON == REC_BF16EXP ? bf16_rne(z) : z;
}

// The fp32 exponentials e_r = fl32(exp(arg(z_r))) of the 16 keys a lane
// holds, as the weight function rounds them: fast expf(), and the fp64
// exponential for keys near a rounding midpoint (one key per lane per
// round, so the slow path runs once per round for the whole wave).
template <int RECON>
__device__ __forceinline__ void exp_tile(const float (&z)[16], float (&e)[16]) {
  uint32_t amb = 0;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    e[r] = expf(exp_arg<RECON>(z[r]));
    amb |= (exp_near_tie<RECON>(e[r]) ? 1u : 0u) << r;
  }
  if constexpr (RECON != REC_SOFTMAX) {
    while (__any(amb != 0)) {
      const int r0 = amb ? __builtin_ctz(amb) : 0;
      float x = z[0];
#pragma unroll
      for (int r = 1; r < 16; ++r) x = (r0 == r) ? z[r] : x;
      const float ex = (float)exp((double)exp_arg<RECON>(x));
      if (amb) {
#pragma unroll
        for (int r = 0; r < 16; ++r) e[r] = (r0 == r) ? ex : e[r];
        amb &= amb - 1u;
      }
    }
  }
}

// Forward weight from the stored fp32 exponential (the value U keeps for
// the backward): softmax w = e, BF16-exp w = bf16(e) (stored already
// rounded), FP8-exp w = e4m3(e).
template <int RECON>
__device__ __forceinline__ float exp_weight_of(float e) {
  if constexpr (RECON == REC_FP8EXP) {
    uint32_t c;
    return e4m3_rne(e, c);
  } else if constexpr (RECON == REC_BF16EXP) {
    return bf16_rne(e);
  } else {
    return e;
  }
}

// Workgroup barrier ordering LDS only: outstanding global stores and
// atomics are not waited for.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Work of the dQ product: query group g of qg tiles (query tiles qg g ..
// qg g + qg - 1) needs the 64-key chunks below 32 qg (g + 1) (causal) or all
// of them; cut into pieces of at most `piece` chunks (piece 0: one piece).
__host__ __device__ inline int dq_chunks(int g, int T, int causal, int qg) {
  const int all = (T + 63) / 64;
  const int need = (qg * (g + 1) + 1) / 2;
  return causal ? (need < all ? need : all) : all;
}
__host__ __device__ inline int dq_pieces(int g, int T, int causal, int piece, int qg) {
  return piece > 0 ? (dq_chunks(g, T, causal, qg) + piece - 1) / piece : 1;
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

// Element (lane l, register r) of a 32x32 fp32 tile of the scratch fields
// (dS, U) sits at (r / 4) * 256 + 4 l + r % 4: the g-th 16-byte access of
// all 64 lanes covers one contiguous KiB.
__device__ __forceinline__ void tile_load(const float *tile, int lane, float (&v)[16]) {
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const f32x4 x = *reinterpret_cast<const f32x4 *>(tile + 256 * g + 4 * lane);
    v[4 * g] = x[0]; v[4 * g + 1] = x[1]; v[4 * g + 2] = x[2]; v[4 * g + 3] = x[3];
  }
}
__device__ __forceinline__ void tile_store(float *tile, int lane, const float (&v)[16]) {
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const f32x4 x = {v[4 * g], v[4 * g + 1], v[4 * g + 2], v[4 * g + 3]};
    *reinterpret_cast<f32x4 *>(tile + 256 * g + 4 * lane) = x;
  }
}

// ---- buffer loads of row blocks ---------------------------------------------
// A buffer resource over rows [r0, rend) of a row-major [*, D] fp32 array:
// loads at byte offsets at or past its end read as zeros (the hardware's
// range check), so ragged tails need no address clamping or masking on the
// vector units.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t row_rsrc(const float *base, int r0,
                                                          int rend, int D) {
  const int rb = min(r0, rend);
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(base) + (size_t)rb * D,
                                           (short)0, (rend - rb) * D * 4, 0x00020000);
}
__device__ __forceinline__ f32x4 buffer_f32x4(__amdgpu_buffer_rsrc_t rs, uint32_t voff) {
  return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, voff, 0, 0));
}
// Byte offset of 16-byte vector idx of a row block (DP / 4 vectors a row);
// padded columns (c >= D) point past the end of any buffer.
template <int D> __device__ __forceinline__ uint32_t row_vec_offset(int idx) {
  constexpr int DP = Dims<D>::DP;
  const int r = idx / (DP / 4), c4 = idx % (DP / 4);
  return c4 * 4 < D ? (uint32_t)(r * D + c4 * 4) * 4u : 0x80000000u;
}

// ---- gradient modes (the backward's `detach` argument) ---------------------
// 0 full (Eq. full), 1 detach, 2 max_only / 3 min_only (one extremum
// channel; appendix on the detached-gradient record), 4 detach with the P1
// zero-sum projection (App. B, Detach).
enum { GRAD_FULL = 0, GRAD_DETACH = 1, GRAD_MAX_ONLY = 2, GRAD_MIN_ONLY = 3, GRAD_P1 = 4 };
// the extremum channels' row sums (cM, cm) are needed
__host__ __device__ inline bool grad_channels(int g) {
  return g == GRAD_FULL || g == GRAD_MAX_ONLY || g == GRAD_MIN_ONLY;
}
__host__ __device__ inline bool grad_keep_max(int g) { return g == GRAD_FULL || g == GRAD_MAX_ONLY; }
__host__ __device__ inline bool grad_keep_min(int g) { return g == GRAD_FULL || g == GRAD_MIN_ONLY; }

// ---- bf16 inputs ---------------------------------------------------------
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ float bf2f(uint32_t bits16) {
  return __uint_as_float(bits16 << 16);
}
// four consecutive inputs as fp32 (bf16 -> fp32 is exact)
__device__ __forceinline__ f32x4 load4(const float *p) {
  return *reinterpret_cast<const f32x4 *>(p);
}
__device__ __forceinline__ f32x4 load4(const uint16_t *p) {
  const uint2 x = *reinterpret_cast<const uint2 *>(p);
  const f32x4 r = {bf2f(x.x & 0xffffu), bf2f(x.x >> 16), bf2f(x.y & 0xffffu), bf2f(x.y >> 16)};
  return r;
}
__device__ __forceinline__ float load1(const float *p) { return *p; }
__device__ __forceinline__ float load1(const uint16_t *p) { return bf2f(*p); }

// v_mfma_f32_32x32x16_bf16: lane l feeds A[l%32][8(l/32) + e] and
// B[8(l/32) + e][l%32], e = 0..7; the output layout is the one of mfma32.
__device__ __forceinline__ f32x16 mfma16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ bf16x8 as_bf16x8(uint4 x) {
  return __builtin_bit_cast(bf16x8, x);
}
__device__ __forceinline__ bf16x8 to_bf16x8(const float *v) {
  bf16x8 r;
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = (__bf16)v[e];
  return r;
}

// Canonical bf16 score sub-tile: S^T with A = K, B = Q; lane l (half h)
// feeds K[key0 + l%32][16s + 8h + e] and Q[query0 + l%32][16s + 8h + e] at
// k-step s. Output register r of lane l holds S^T[key0 + krel(r, h)]
// [query0 + l%32] (as score_tile). Every bf16 kernel computes a pair's
// score with this sub-tile, so it is bit-identical wherever it is computed.
template <int D>
__device__ __forceinline__ f32x16 score_tile16(const bf16x8 (&kop)[D / 16],
                                               const bf16x8 (&qop)[D / 16]) {
  f32x16 acc;
#pragma unroll
  for (int e = 0; e < 16; ++e) acc[e] = 0.f;
#pragma unroll
  for (int s = 0; s < D / 16; ++s) acc = mfma16(kop[s], qop[s], acc);
  return acc;
}
// the lane's operand of one 32-row tile of a [T, D] bf16 slice (row clamped
// into the slice; rows at or beyond T read as zero)
template <int D>
__device__ __forceinline__ void load_rows16(const uint16_t *slice, int row, int T, int half,
                                            bf16x8 (&op)[D / 16]) {
  const bool ok = row < T;
  const uint16_t *src = slice + (size_t)(ok ? row : 0) * D + 8 * half;
#pragma unroll
  for (int s = 0; s < D / 16; ++s) {
    uint4 x = *reinterpret_cast<const uint4 *>(src + 16 * s);
    if (!ok) x = make_uint4(0, 0, 0, 0);
    op[s] = as_bf16x8(x);
  }
}

// Stats view from the caller's buffer (offsets as kia_stats_offset()).
__host__ __device__ inline size_t align256(size_t x) {
  return (x + 255) & ~(size_t)255;
}

}  // namespace kia
