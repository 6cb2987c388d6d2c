// kia_fwd.hip -- forward of causal K-interval attention on gfx950.
//
// One workgroup = 4 waves = 64 query rows of one (b, h): two row groups of
// 32 rows times two key halves. Each wave keeps its 32 Q rows in registers
// as the B operand of the canonical score sub-tile. Keys stream through LDS
// in chunks of 64 (one 32-key tile per key half); the waves of a row group
// take alternate tiles, so the longest rows' work is split over two waves.
// Grids too small to fill the chip (KP = 4) take one row group of 32 rows
// with four key quarters instead: chunks of 128 keys, every fourth tile per
// wave, twice the workgroups; the smallest grids (KP = 8) take eight key
// parts in workgroups of 8 waves (chunks of 256 keys).
//
// Pass 1 (row extrema, App. A: amax/amin over the valid keys): score
//   sub-tiles, stored to the stats field U, and per-lane running max/min
//   with first index and tie count, merged across the two lanes that share
//   a row, then across the key parts through LDS (max, then smallest
//   index, tie counts added).
// Pass 2 (Sec. 3 reconstruction and normalization): the grid depends on the
//   extrema, so the wave reads its stored score tiles back (one ahead): per
//   key the interval/level decision, whose decided position u replaces the
//   score in U for the backward, w^L and w^N from e^{b_{r+1}} (one exp2 per
//   key), the row sums
//   W^N, W^L, and O += w V on fp32 MFMA with the weight registers as the B
//   operand (no data movement). Prob-STE with Nearest also accumulates
//   O^L = w^L V for the backward. The weights are absolute once the extrema
//   are known, so the key parts' partial sums simply add (through LDS);
//   O = (sum w v) / W at the end: W >= 1 because the argmax key has weight
//   e^0 = 1, so no online rescaling.
// Exponential weight functions (softmax, BF16-exp, FP8-exp; App. A, App. D)
//   take the same two passes with the maximum only: pass 2 forms z = s - M,
//   the fp32 exponential as the weight function rounds it (kept in U in
//   place of the score) and the weight, with no grid.
#include <type_traits>

#include "kia_device.hpp"
#include "kia_kernels.hpp"

namespace kia {

constexpr int FWD_TK = 32;   // keys per tile (one MFMA sub-tile)
constexpr int CODES_BM = 128;
constexpr int CODES_BN = 64;

template <int D>
__device__ __forceinline__ void load_tile_lds(float *dst, const float *src,
                                              int j0, int T, int tid) {
  // rows j0 .. j0+CODES_BN-1 of a [T, D] slice into dst[CODES_BN][DS]; zero
  // beyond T and beyond D so that masked products never meet garbage
  // (0 * NaN).
  constexpr int DP = Dims<D>::DP, DS = Dims<D>::DS;
  constexpr int V4 = CODES_BN * DP / 4;
#pragma unroll
  for (int e = tid; e < V4; e += 256) {
    const int row = e / (DP / 4), c4 = e % (DP / 4);
    f32x4 val = {0.f, 0.f, 0.f, 0.f};
    if (j0 + row < T && c4 * 4 < D)
      val = *reinterpret_cast<const f32x4 *>(src + (size_t)(j0 + row) * D + c4 * 4);
    *reinterpret_cast<f32x4 *>(dst + row * DS + c4 * 4) = val;
  }
}

// Next-chunk register prefetch of a [ROWS, D] slice of K or V by NT
// threads, through buffer loads: each NT-thread pass gets a buffer resource
// that starts at its first row and ends at row T, so rows past T (and padded
// columns) read as zeros.
template <int D, int ROWS, int NT = 256> struct TileFetch {
  static constexpr int DP = Dims<D>::DP, DS = Dims<D>::DS;
  static constexpr int V4 = ROWS * DP / 4;   // 16-byte vectors per chunk
  static constexpr int PF = V4 / NT;         // passes of NT threads
  static constexpr int RPP = NT / (DP / 4);  // rows per pass
  static_assert(V4 % NT == 0, "whole passes");
  f32x4 x[PF];
  __device__ __forceinline__ void fetch(const float *src, int j0, int T, uint32_t voff) {
#pragma unroll
    for (int e = 0; e < PF; ++e) x[e] = buffer_f32x4(row_rsrc(src, j0 + e * RPP, T, D), voff);
  }
  __device__ __forceinline__ void stash(float *dst, int tid) const {
#pragma unroll
    for (int e = 0; e < PF; ++e) {
      const int idx = tid + NT * e;
      const int r = idx / (DP / 4), c4 = idx % (DP / 4);
      *reinterpret_cast<f32x4 *>(dst + r * DS + c4 * 4) = x[e];
    }
  }
};

// Running (extremum, first index, count) merge; `b` is the later part.
template <bool MAX>
__device__ __forceinline__ void merge_ext(float &M, int &a, int &c, float M2, int a2, int c2) {
  const bool take = MAX ? (M2 > M) : (M2 < M);
  const bool tie = M2 == M;
  a = take ? a2 : (tie ? min(a, a2) : a);
  c = take ? c2 : (tie ? c + c2 : c);
  M = take ? M2 : M;
}

template <int D, int CALIB, int RECON, bool OL, int KP>
__global__ __launch_bounds__(KP == 8 ? 512 : 256, Dims<D>::FWD_WAVES_PER_EU) void fwd_kernel(FwdArgs a) {
  constexpr int DS = Dims<D>::DS, NC = Dims<D>::NC;
  // MinMax and the resolved grid need the row minimum (resolved: for the
  // rounding margin of its far keys only)
  constexpr bool TRACKMIN = CALIB != CAL_FWM, NEAREST = RECON == REC_NEAREST;
  constexpr bool EXPW = is_exp_rec(RECON);
  static_assert(!EXPW || (CALIB == CAL_FWM && !OL), "exp weights use the maximum only");
  // per-lane values a wave of key part > 0 hands to part 0 at the end
  constexpr int NRED = NC * 16 * (OL ? 2 : 1) + 2;
  // KP key parts times RG row groups of 32 rows; a chunk holds one 32-key
  // tile per key part
  static_assert(KP == 2 || KP == 4 || KP == 8, "key parts");
  constexpr int RG = KP == 8 ? 1 : 4 / KP, BM = 32 * RG, CHK = FWD_TK * KP;
  constexpr int NT = 64 * RG * KP;  // threads: one wave per (row group, key part)
  static_assert((KP - 1) * RG * 64 * NRED <= 2 * CHK * DS, "reduction buffer");
  // K chunks (pass 1) and V chunks (pass 2) share one double buffer: the
  // passes are separated by the extrema merge's workgroup barrier. Half the
  // LDS of separate buffers, so twice the workgroups fit on a CU.
  __shared__ __attribute__((aligned(16))) float CH[2][CHK * DS];
  __shared__ int Xc[RG][KP][6][32];  // pass-1 partials [row group][key part][field][row]

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, half = lane >> 5, l32 = lane & 31;
  const int pr = wave % RG, kh = wave / RG;  // row group, key part
  const int T = a.T;
  const int nqb = (T + BM - 1) / BM;
  // heaviest (last) query blocks first; (b,h) fastest
  const int bh = blockIdx.x % a.BH;
  const int qb = nqb - 1 - (int)(blockIdx.x / a.BH);
  const int i0 = qb * BM;
  const int iw = i0 + pr * 32;
  const int row = iw + l32;
  const size_t slice = (size_t)bh * T * D;
  const float *qs = a.q + slice, *ks = a.k + slice, *vs = a.v + slice;
  const float Kf = (float)a.K;
  // key j is valid for this lane's row iff j <= jlim; a tile starting at js
  // holds a valid key for some row of the wave iff js <= wlim
  const int jlim = a.causal ? min(row, T - 1) : T - 1;
  const int wlim = iw >= T ? -1 : (a.causal ? min(iw + 31, T - 1) : T - 1);
  // every key j <= wmin is valid for every row of the wave
  const int wmin = a.causal ? min(iw, T - 1) : T - 1;

  float qop[D / 2];
  {
    const int rr = row < T ? row : T - 1;
    const float *src = qs + (size_t)rr * D + half * (D / 2);
#pragma unroll
    for (int s = 0; s < D / 2; s += 4) {
      f32x4 x = *reinterpret_cast<const f32x4 *>(src + s);
      qop[s] = x[0]; qop[s + 1] = x[1]; qop[s + 2] = x[2]; qop[s + 3] = x[3];
    }
  }

  const int kend = a.causal ? min(T, i0 + BM) : T;
  const int nstep = (kend + CHK - 1) / CHK;
  const int toff = kh * FWD_TK * DS;  // this wave's tile inside a chunk
  const uint32_t foff = row_vec_offset<D>(tid);  // this thread's vector in a pass

  auto load_kop = [&](const float *Kb, float (&kop)[D / 2]) {
    const float *kr = Kb + l32 * DS + half * (D / 2);
#pragma unroll
    for (int s = 0; s < D / 2; s += 4) {
      f32x4 x = *reinterpret_cast<const f32x4 *>(kr + s);
      kop[s] = x[0]; kop[s + 1] = x[1]; kop[s + 2] = x[2]; kop[s + 3] = x[3];
    }
  };

  // chunks whose tile of this wave holds a valid key: p < npw
  const int npw = wlim < kh * FWD_TK ? 0 : min(nstep, (wlim - kh * FWD_TK) / CHK + 1);
  // this wave's score tiles in U (tile of chunk p at + (KP p + kh) * 1024;
  // the tiles of one query tile are consecutive in both layouts)
  float *Ut = a.st.U + ds_tile(bh, iw / 32, kh, (T + 31) / 32, a.causal) * 1024;

  // chunk prefetch registers: K chunks in pass 1, then V chunks in pass 2
  // (V chunk 0 is fetched during the last K step and stashed in CH[0] once
  // pass 1's last step has ended)
  TileFetch<D, CHK, NT> fch;

  // ---------------- pass 1: scores, extrema, first index, tie counts -----
  float Mx = -INFINITY, Mn = INFINITY;
  int ax = 0x7fffffff, an = 0x7fffffff, cx = 0, cn = 0;
  {
    fch.fetch(ks, 0, T, foff);
    fch.stash(CH[0], tid);
    lds_barrier();
    for (int p = 0; p < nstep; ++p) {
      // the next K chunk; after the last one, pass 2's first V chunk
      const bool more = p + 1 < nstep;
      fch.fetch(more ? ks : vs, more ? (p + 1) * CHK : 0, T, foff);
      if (p < npw) {
        const int js = p * CHK + kh * FWD_TK;
        float kop[D / 2];
        load_kop(CH[p & 1] + toff, kop);
        const f32x16 acc = score_tile<D>(kop, qop);
        {
          float sv[16];
#pragma unroll
          for (int r = 0; r < 16; ++r) sv[r] = acc[r];
          tile_store(Ut + (size_t)p * (KP * 1024), lane, sv);
        }
        float sx[16];
        if (js + FWD_TK - 1 <= wmin) {
          // interior tile: every key is valid for every row of the wave
#pragma unroll
          for (int r = 0; r < 16; ++r) sx[r] = acc[r] * a.scale;
          tile_extremum<true>(sx, js, half, Mx, ax, cx);
          if constexpr (TRACKMIN) tile_extremum<false>(sx, js, half, Mn, an, cn);
        } else {
          float sn[16];
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const float sc = acc[r] * a.scale;
            const bool valid = js + krel(r, half) <= jlim;
            sx[r] = valid ? sc : -INFINITY;
            sn[r] = valid ? sc : INFINITY;
          }
          tile_extremum<true>(sx, js, half, Mx, ax, cx);
          if constexpr (TRACKMIN) tile_extremum<false>(sn, js, half, Mn, an, cn);
        }
      }
      fch.stash(CH[(p + 1) & 1], tid);
      lds_barrier();
    }
    // the last step stashed V chunk 0 in CH[nstep & 1]; pass 2 wants CH[0]
    if (nstep & 1) fch.stash(CH[0], tid);
  }
  merge_ext<true>(Mx, ax, cx, __shfl_xor(Mx, 32), __shfl_xor(ax, 32), __shfl_xor(cx, 32));
  if constexpr (TRACKMIN)
    merge_ext<false>(Mn, an, cn, __shfl_xor(Mn, 32), __shfl_xor(an, 32), __shfl_xor(cn, 32));
  // key parts: every wave of a row group merges the parts in the same order
  if (half == 0) {
    int *x = &Xc[pr][kh][0][l32];
    x[0] = __float_as_int(Mx); x[32] = ax; x[64] = cx;
    x[96] = __float_as_int(Mn); x[128] = an; x[160] = cn;
  }
  __syncthreads();
  {
    const int *x0 = &Xc[pr][0][0][l32];
    Mx = __int_as_float(x0[0]); ax = x0[32]; cx = x0[64];
    if constexpr (TRACKMIN) { Mn = __int_as_float(x0[96]); an = x0[128]; cn = x0[160]; }
#pragma unroll
    for (int q = 1; q < KP; ++q) {
      const int *x1 = &Xc[pr][q][0][l32];
      merge_ext<true>(Mx, ax, cx, __int_as_float(x1[0]), x1[32], x1[64]);
      if constexpr (TRACKMIN)
        merge_ext<false>(Mn, an, cn, __int_as_float(x1[96]), x1[128], x1[160]);
    }
  }
  const size_t ridx = (size_t)bh * T + row;
  if (kh == 0 && half == 0 && row < T) {
    a.st.M[ridx] = Mx;
    a.st.amax[ridx] = ax;
    a.st.nmax[ridx] = cx;
    if constexpr (TRACKMIN) {
      a.st.m[ridx] = Mn;
      a.st.amin[ridx] = an;
      a.st.nmin[ridx] = cn;
    }
  }
  if constexpr (!TRACKMIN) Mn = Mx;  // unused by FWM
  RowConst rc{};
  if constexpr (!EXPW) rc = row_const(Mx, Mn, a.K, CALIB, a.tau, a.scale);

  // ---------------- pass 2: reconstruct, normalize, O = P V ---------------
  // The wave's own score tiles come back from U (one tile ahead, in two
  // fixed register sets); each is replaced there by its decided positions.
  f32x16 oacc[NC], olacc[OL ? NC : 1];
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) oacc[c][e] = 0.f;
  if constexpr (OL) {
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int e = 0; e < 16; ++e) olacc[c][e] = 0.f;
  }
  float WN = 0.f, WLs = 0.f;
  auto load_s = [&](int p, f32x16 &S) {
    float sv[16];
    tile_load(Ut + (size_t)p * (KP * 1024), lane, sv);
#pragma unroll
    for (int r = 0; r < 16; ++r) S[r] = sv[r];
  };
  auto tile = [&](int p, const f32x16 &S, auto masked_tag) {
    constexpr bool MASKED = decltype(masked_tag)::value;
    const int js = p * CHK + kh * FWD_TK;
    float w[16], wl[16];
    float tWN = 0.f, tWL = 0.f;  // sub-tile sums first: shorter running sums
    if constexpr (EXPW) {
      // z = s - M, the fp32 exponential as the weight function rounds it
      // (kept in U for the backward; bf16-rounded already for BF16-exp),
      // and the weight
      float z[16], e[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) z[r] = score_shift(S[r], a.scale, Mx);
      exp_tile<RECON>(z, e);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        if constexpr (RECON == REC_BF16EXP) e[r] = bf16_rne(e[r]);
        const bool valid = js + krel(r, half) <= jlim;
        w[r] = valid ? exp_weight_of<RECON>(e[r]) : 0.f;
        tWN += w[r];
      }
      if (a.keep) tile_store(Ut + (size_t)p * (KP * 1024), lane, e);
      tWL = tWN;
    } else {
    float u[16];
    uint32_t cw[4];
    decide_u<CALIB>(S, rc, Mx, Mn, a.K, a.tau, a.scale, u);
    if constexpr (!compact_codes<CALIB, RECON>())
      if (a.keep) tile_store(Ut + (size_t)p * (KP * 1024), lane, u);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const KeyDec kd = key_of<CALIB>(u[r], Kf);
      if constexpr (compact_codes<CALIB, RECON>()) code_put(cw, r, kd);
      float Eu;
      if constexpr (MASKED) {
        Eu = grid_upper(kd.rf, rc);
      } else {
        // interior tile: only the FWM tail is zero, through e^{-inf} = 0
        const float arg = fmaf(kd.rf, rc.hl, rc.b1l);
        Eu = __builtin_amdgcn_exp2f(kd.tail ? -INFINITY : arg);
      }
      const float El = Eu * rc.emh;
      float wL = fmaf(kd.t, Eu - El, El);
      float wN = kd.up ? Eu : El;
      if constexpr (MASKED) {
        const bool valid = (js + krel(r, half) <= jlim) & !kd.tail;
        wL = valid ? wL : 0.f;
        wN = valid ? wN : 0.f;
      }
      tWL += wL;
      wl[r] = wL;
      if constexpr (NEAREST) {
        tWN += wN;
        w[r] = wN;
      } else {
        w[r] = wL;
      }
    }
    if constexpr (compact_codes<CALIB, RECON>())
      if (a.keep) codes_store(Ut + (size_t)p * (KP * 1024), lane, cw);
    }
    WN += tWN;
    WLs += tWL;
    const float *Vb = CH[p & 1] + toff;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const float *vr = Vb + c * 32 + l32;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float vop = vr[krel(r, half) * DS];
        oacc[c] = mfma32(vop, w[r], oacc[c]);
        if constexpr (OL) olacc[c] = mfma32(vop, wl[r], olacc[c]);
      }
    }
  };
  {
    // V chunk 0 is in CH[0] already (ordered by the extrema merge's barrier)
    f32x16 SA, SB;
    if (npw > 0) load_s(0, SA);
    // tiles below the wave's first row are interior (no causal mask)
    auto run = [&](int p, const f32x16 &S) {
      if (p * CHK + kh * FWD_TK + FWD_TK - 1 <= wmin)
        tile(p, S, std::integral_constant<bool, false>{});
      else
        tile(p, S, std::integral_constant<bool, true>{});
    };
    for (int p = 0; p < nstep; p += 2) {
      fch.fetch(vs, min(p + 1, nstep - 1) * CHK, T, foff);
      if (p + 1 < npw) load_s(p + 1, SB);
      if (p < npw) run(p, SA);
      fch.stash(CH[(p + 1) & 1], tid);
      lds_barrier();
      if (p + 1 >= nstep) break;
      fch.fetch(vs, min(p + 2, nstep - 1) * CHK, T, foff);
      if (p + 2 < npw) load_s(p + 2, SA);
      if (p + 1 < npw) run(p + 1, SB);
      fch.stash(CH[p & 1], tid);
      lds_barrier();
    }
  }
  WN += __shfl_xor(WN, 32);
  WLs += __shfl_xor(WLs, 32);
  // key parts 1.. hand their partial sums to key part 0, which adds them in
  // part order (chunk buffers are free: the last step ended with a barrier)
  float *red = &CH[0][0] + pr * (KP - 1) * 64 * NRED + lane;
  if (kh > 0) {
    float *rk = red + (kh - 1) * 64 * NRED;
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        rk[(c * 16 + e) * 64] = oacc[c][e];
        if constexpr (OL) rk[((NC + c) * 16 + e) * 64] = olacc[c][e];
      }
    rk[(NRED - 2) * 64] = WN;
    rk[(NRED - 1) * 64] = WLs;
  }
  __syncthreads();
  if (kh > 0) return;
#pragma unroll 1
  for (int q = 0; q < KP - 1; ++q) {
    const float *rk = red + q * 64 * NRED;
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        oacc[c][e] += rk[(c * 16 + e) * 64];
        if constexpr (OL) olacc[c][e] += rk[((NC + c) * 16 + e) * 64];
      }
    WN += rk[(NRED - 2) * 64];
    WLs += rk[(NRED - 1) * 64];
  }
  const float W = NEAREST ? WN : WLs;
  if (half == 0 && row < T) {
    a.st.W[ridx] = W;
    a.st.WL[ridx] = WLs;
  }
  if (row < T) {
    const float inv = 1.f / W, invl = 1.f / WLs;
    float *orow = a.o + slice + (size_t)row * D;
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int n = c * 32 + 8 * g + 4 * half;
        if (n >= D) continue;
        f32x4 x = {oacc[c][4 * g] * inv, oacc[c][4 * g + 1] * inv,
                   oacc[c][4 * g + 2] * inv, oacc[c][4 * g + 3] * inv};
        *reinterpret_cast<f32x4 *>(orow + n) = x;
        if constexpr (OL) {
          f32x4 y = {olacc[c][4 * g] * invl, olacc[c][4 * g + 1] * invl,
                     olacc[c][4 * g + 2] * invl, olacc[c][4 * g + 3] * invl};
          *reinterpret_cast<f32x4 *>(a.st.OL + ridx * D + n) = y;
        }
      }
  }
}

// Debug codes: the same score sub-tiles, decide_u() and key_of() as pass 2
// (REC = REC_LERP stands for both K-interval reconstructions); for an
// exponential weight function (REC >= REC_SOFTMAX) the quantized weight's
// code from the same score_shift() and exp_tile() as pass 2.
template <int D, int CALIB, int REC, typename TI>
__global__ __launch_bounds__(256) void codes_kernel(CodesArgsT<TI> a) {
  constexpr bool EXPW = is_exp_rec(REC);
  constexpr bool B16 = sizeof(TI) == 2;
  constexpr int DS = Dims<D>::DS;
  __shared__ __attribute__((aligned(16))) float Ks[CODES_BN * DS];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, half = lane >> 5, l32 = lane & 31;
  const int T = a.T;
  const int nqb = (T + CODES_BM - 1) / CODES_BM;
  const int bh = blockIdx.x % a.BH;
  const int qb = nqb - 1 - (int)(blockIdx.x / a.BH);
  const int i0 = qb * CODES_BM, iw = i0 + wave * 32, row = iw + l32;
  const size_t slice = (size_t)bh * T * D;
  const float Kf = (float)a.K;
  float qop[D / 2];
  bf16x8 qop16[D / 16];
  if constexpr (B16) {
    load_rows16<D>(a.q + slice, row < T ? row : T - 1, T, half, qop16);
  } else {
    const int rr = row < T ? row : T - 1;
    const float *src = a.q + slice + (size_t)rr * D + half * (D / 2);
#pragma unroll
    for (int s = 0; s < D / 2; s += 4) {
      f32x4 x = *reinterpret_cast<const f32x4 *>(src + s);
      qop[s] = x[0]; qop[s + 1] = x[1]; qop[s + 2] = x[2]; qop[s + 3] = x[3];
    }
  }
  const size_t ridx = (size_t)bh * T + (row < T ? row : T - 1);
  const float Mx = a.st.M[ridx];
  const float Mn = CALIB != CAL_FWM ? a.st.m[ridx] : Mx;
  RowConst rc{};
  if constexpr (!EXPW) rc = row_const(Mx, Mn, a.K, CALIB, a.tau, a.scale);
  const int kend = a.causal ? min(T, i0 + CODES_BM) : T;
  const int ntiles = (T + CODES_BN - 1) / CODES_BN;
  for (int t = 0; t < ntiles; ++t) {
    const int j0 = t * CODES_BN;
    __syncthreads();
    if constexpr (!B16) load_tile_lds<D>(Ks, a.k + slice, j0, T, tid);
    __syncthreads();
#pragma unroll
    for (int sub = 0; sub < CODES_BN / 32; ++sub) {
      const int js = j0 + sub * 32;
      if (js >= T) continue;
      uint16_t code[16];
      if (js >= kend || (a.causal && js > iw + 31)) {
#pragma unroll
        for (int r = 0; r < 16; ++r) code[r] = 0;
      } else {
        f32x16 acc;
        if constexpr (B16) {
          bf16x8 kop16[D / 16];
          load_rows16<D>(a.k + slice, js + l32, T, half, kop16);
          acc = score_tile16<D>(kop16, qop16);
        } else {
          float kop[D / 2];
          const float *kr = Ks + (sub * 32 + l32) * DS + half * (D / 2);
#pragma unroll
          for (int s = 0; s < D / 2; s += 4) {
            f32x4 x = *reinterpret_cast<const f32x4 *>(kr + s);
            kop[s] = x[0]; kop[s + 1] = x[1]; kop[s + 2] = x[2]; kop[s + 3] = x[3];
          }
          acc = score_tile<D>(kop, qop);
        }
        if constexpr (EXPW) {
          // bit 15 valid; bits 0-14 the bf16 pattern (BF16-exp) or the E4M3
          // byte (FP8-exp) of the weight, 0 for softmax (w <= 1: bit 14 clear)
          float z[16], e[16];
#pragma unroll
          for (int r = 0; r < 16; ++r) z[r] = score_shift(acc[r], a.scale, Mx);
          exp_tile<REC>(z, e);
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int j = js + krel(r, half);
            const bool valid = (j < T) & (!a.causal | (j <= row));
            uint32_t c = 0;
            if constexpr (REC == REC_BF16EXP) c = __float_as_uint(bf16_rne(e[r])) >> 16;
            if constexpr (REC == REC_FP8EXP) e4m3_rne(e[r], c);
            code[r] = valid ? (uint16_t)(0x8000u | c) : (uint16_t)0;
          }
        } else {
        float u[16];
        decide_u<CALIB>(acc, rc, Mx, Mn, a.K, a.tau, a.scale, u);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int j = js + krel(r, half);
          const bool valid = (j < T) & (!a.causal | (j <= row));
          const KeyDec kd = key_of<CALIB>(u[r], Kf);
          uint16_t c = 0;
          if (valid && CALIB == CAL_RESOLVED) {
            // bit 15 valid, bit 14 l = r + 1, bits 0-13 r (two's complement,
            // clamped to [-8192, 8191])
            const int rr = (int)fmaxf(kd.rf, -8192.f);
            c = (uint16_t)(0x8000u | (kd.up ? 0x4000u : 0u) | ((uint32_t)rr & 0x3FFFu));
          } else if (valid) {
            c = (uint16_t)(1u << 14);
            if (rc.degen) c |= (uint16_t)(1u << 15);
            else if (kd.tail) c |= (uint16_t)(1u << 13);
            else {
              const int rr = (int)kd.rf;
              const int ll = rr + (kd.up ? 1 : 0);
              c |= (uint16_t)(rr | (ll << 6));
            }
          }
          code[r] = c;
        }
        }
      }
      if (row < T) {
        uint16_t *dst = a.codes + ((size_t)bh * T + row) * T;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int j = js + krel(r, half);
          if (j < T) dst[j] = code[r];
        }
      }
    }
  }
}

// Code words of the decisions the forward stored in U (the positions u
// that pass 2 wrote and the backward reads; for an exponential weight
// function the fp32 exponential): the same format as codes_kernel, with no
// score recomputed. One wave per (b,h, 32-query tile) over all key tiles;
// codes of keys that are not valid (and of unstored tiles) are 0.
template <int CALIB, int REC>
__global__ __launch_bounds__(256) void stored_codes_kernel(StoredCodesArgs a) {
  constexpr bool EXPW = is_exp_rec(REC);
  constexpr bool COMPACT = compact_codes<CALIB, REC>();
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, half = lane >> 5, l32 = lane & 31;
  const int T = a.T;
  const int nq = (T + 31) / 32;
  const size_t gw = (size_t)blockIdx.x * 4 + wave;
  if (gw >= (size_t)a.BH * nq) return;
  const int bh = (int)(gw / nq), qt = (int)(gw % nq);
  const int i = qt * 32 + l32;
  const float Kf = (float)a.K;
  bool degen = false;
  if (CALIB == CAL_MINMAX && i < T) {
    const size_t ridx = (size_t)bh * T + i;
    degen = (double)a.st.M[ridx] - (double)a.st.m[ridx] <= 1e-12;
  }
  for (int kt = 0; kt < nq; ++kt) {
    const bool stored = !a.causal || kt <= qt;
    float u[16];
    uint4 cw = make_uint4(0, 0, 0, 0);
    const float *tile = a.st.U + ds_tile(bh, qt, kt, nq, a.causal) * 1024;
    if (stored) {
      if constexpr (COMPACT) cw = codes_load(tile, lane);
      else tile_load(tile, lane, u);
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int j = kt * 32 + krel(r, half);
      if (i >= T || j >= T) continue;
      const bool valid = stored & (!a.causal | (j <= i));
      uint32_t c = 0;
      if (valid && COMPACT) {
        const KeyDec kd = key_of_code(cw, r);
        c = 1u << 14;
        if (kd.tail) c |= 1u << 13;
        else {
          const int rr = (int)kd.rf;
          c |= (uint32_t)(rr | ((rr + (kd.up ? 1 : 0)) << 6));
        }
      } else if (valid && EXPW) {
        if constexpr (REC == REC_BF16EXP) c = __float_as_uint(bf16_rne(u[r])) >> 16;
        if constexpr (REC == REC_FP8EXP) e4m3_rne(u[r], c);
        c |= 0x8000u;
      } else if (valid) {
        const KeyDec kd = key_of<CALIB>(u[r], Kf);
        if (CALIB == CAL_RESOLVED) {
          const int rr = (int)fmaxf(kd.rf, -8192.f);
          c = 0x8000u | (kd.up ? 0x4000u : 0u) | ((uint32_t)rr & 0x3FFFu);
        } else {
          c = 1u << 14;
          if (degen) c |= 1u << 15;
          else if (kd.tail) c |= 1u << 13;
          else {
            const int rr = (int)kd.rf;
            c |= (uint32_t)(rr | ((rr + (kd.up ? 1 : 0)) << 6));
          }
        }
      }
      a.codes[((size_t)bh * T + i) * T + j] = (uint16_t)c;
    }
  }
}

// The canonical fp32 scores s = fl32(acc * scale) of every pair (the values
// the forward's extrema pass stored and every decision is taken on), 0 for
// keys that are not valid. Same sub-tile and operand loads as codes_kernel.
template <int D, typename TI>
__global__ __launch_bounds__(256) void scores_kernel(ScoresArgsT<TI> a) {
  constexpr bool B16 = sizeof(TI) == 2;
  constexpr int DS = Dims<D>::DS;
  __shared__ __attribute__((aligned(16))) float Ks[CODES_BN * DS];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, half = lane >> 5, l32 = lane & 31;
  const int T = a.T;
  const int nqb = (T + CODES_BM - 1) / CODES_BM;
  const int bh = blockIdx.x % a.BH;
  const int qb = nqb - 1 - (int)(blockIdx.x / a.BH);
  const int i0 = qb * CODES_BM, iw = i0 + wave * 32, row = iw + l32;
  const size_t slice = (size_t)bh * T * D;
  float qop[D / 2];
  bf16x8 qop16[D / 16];
  if constexpr (B16) {
    load_rows16<D>(a.q + slice, row < T ? row : T - 1, T, half, qop16);
  } else {
    const int rr = row < T ? row : T - 1;
    const float *src = a.q + slice + (size_t)rr * D + half * (D / 2);
#pragma unroll
    for (int s = 0; s < D / 2; s += 4) {
      f32x4 x = *reinterpret_cast<const f32x4 *>(src + s);
      qop[s] = x[0]; qop[s + 1] = x[1]; qop[s + 2] = x[2]; qop[s + 3] = x[3];
    }
  }
  const int ntiles = (T + CODES_BN - 1) / CODES_BN;
  for (int t = 0; t < ntiles; ++t) {
    const int j0 = t * CODES_BN;
    __syncthreads();
    if constexpr (!B16) load_tile_lds<D>(Ks, a.k + slice, j0, T, tid);
    __syncthreads();
#pragma unroll
    for (int sub = 0; sub < CODES_BN / 32; ++sub) {
      const int js = j0 + sub * 32;
      if (js >= T) continue;
      f32x16 acc;
      if constexpr (B16) {
        bf16x8 kop16[D / 16];
        load_rows16<D>(a.k + slice, js + l32, T, half, kop16);
        acc = score_tile16<D>(kop16, qop16);
      } else {
        float kop[D / 2];
        const float *kr = Ks + (sub * 32 + l32) * DS + half * (D / 2);
#pragma unroll
        for (int s = 0; s < D / 2; s += 4) {
          f32x4 x = *reinterpret_cast<const f32x4 *>(kr + s);
          kop[s] = x[0]; kop[s + 1] = x[1]; kop[s + 2] = x[2]; kop[s + 3] = x[3];
        }
        acc = score_tile<D>(kop, qop);
      }
      if (row < T) {
        float *dst = a.scores + ((size_t)bh * T + row) * T;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int j = js + krel(r, half);
          if (j < T) dst[j] = (!a.causal | (j <= row)) ? acc[r] * a.scale : 0.f;
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Geometry probe (the paper's per-row score statistics): one wave per 32
// query rows, four waves per workgroup, keys streamed through LDS in tiles of
// 64 as in codes_kernel, scores from the canonical sub-tile and decisions
// from decide_u()/key_of(), so M, the levels and the native weights are the
// forward's own. Pass A: softmax sums W_E = sum e^z and sum e^z z, the count
// of z < -6 (decided in fp64), the top-bucket mass, the bucket masses (LDS
// float atomics, [row][K + 2]: levels/intervals 0..K, the FWM tail K + 1),
// the row minimum and the LQ smallest scores of each lane (sorted insertion).
// Pass B: TV = 1/2 sum |w / W - e^z / W_E| with the forward's W.
constexpr int GEO_COUNT = 10;

template <int D, int CALIB, int RECON, int LQ>
__global__ __launch_bounds__(256) void geometry_kernel(GeoArgs a) {
  constexpr int DS = Dims<D>::DS;
  constexpr bool NEAREST = RECON == REC_NEAREST;
  __shared__ __attribute__((aligned(16))) float Ks[CODES_BN * DS];
  __shared__ float bucket[CODES_BM * 66];  // [row][K + 2], K <= 64
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, half = lane >> 5, l32 = lane & 31;
  const int T = a.T, K = a.K, NB = a.K + 2;
  const int nqb = (T + CODES_BM - 1) / CODES_BM;
  const int bh = blockIdx.x % a.BH;
  const int qb = nqb - 1 - (int)(blockIdx.x / a.BH);
  const int i0 = qb * CODES_BM, iw = i0 + wave * 32, row = iw + l32;
  const int lrow = wave * 32 + l32;
  const size_t slice = (size_t)bh * T * D;
  const float Kf = (float)K;
  for (int e = tid; e < CODES_BM * NB; e += 256) bucket[e] = 0.f;
  float qop[D / 2];
  float qss = 0.f, kss = 0.f;
  {
    const int rr = row < T ? row : T - 1;
    const float *src = a.q + slice + (size_t)rr * D + half * (D / 2);
    const float *ksrc = a.k + slice + (size_t)rr * D + half * (D / 2);
#pragma unroll
    for (int c = 0; c < D / 2; c += 4) {
      const f32x4 x = *reinterpret_cast<const f32x4 *>(src + c);
      const f32x4 y = *reinterpret_cast<const f32x4 *>(ksrc + c);
      qop[c] = x[0]; qop[c + 1] = x[1]; qop[c + 2] = x[2]; qop[c + 3] = x[3];
      qss += x[0] * x[0] + x[1] * x[1] + x[2] * x[2] + x[3] * x[3];
      kss += y[0] * y[0] + y[1] * y[1] + y[2] * y[2] + y[3] * y[3];
    }
  }
  const size_t ridx = (size_t)bh * T + (row < T ? row : T - 1);
  const float M = a.st.M[ridx];
  const float Mn = CALIB == CAL_MINMAX ? a.st.m[ridx] : M;
  const float W = a.st.W[ridx];
  const RowConst rc = row_const(M, Mn, K, CALIB, a.tau, a.scale);
  const int kend = a.causal ? min(T, i0 + CODES_BM) : T;
  const int ntiles = (kend + CODES_BN - 1) / CODES_BN;
  const int jlim = row < T ? (a.causal ? row : T - 1) : -1;

  // native weight and bucket of one key from its decided position
  auto native = [&](float u, float &w, int &b, bool &top) {
    const KeyDec kd = key_of<CALIB>(u, Kf);
    const float Eu = grid_upper(kd.rf, rc);
    const float El = Eu * rc.emh;
    const float wl = fmaf(kd.t, Eu - El, El);
    w = kd.tail ? 0.f : (NEAREST ? (kd.up ? Eu : El) : wl);
    const int lev = (int)kd.rf + (NEAREST && kd.up ? 1 : 0);
    b = kd.tail ? K + 1 : lev;
    top = !kd.tail && (NEAREST ? lev == K : (int)kd.rf == K - 1);
    if (rc.degen) { w = 1.f; b = 0; top = false; }  // App. A: weights 1, r = l = 0
  };

  float WE = 0.f, A = 0.f, topE = 0.f, smin = INFINITY, tv = 0.f;
  int cnt6 = 0;
  float low[LQ];
#pragma unroll
  for (int e = 0; e < LQ; ++e) low[e] = INFINITY;
  for (int pass = 0; pass < 2; ++pass) {
    float WEt = 0.f;
    if (pass == 1) WEt = WE;
    for (int t = 0; t < ntiles; ++t) {
      const int j0 = t * CODES_BN;
      __syncthreads();
      load_tile_lds<D>(Ks, a.k + slice, j0, T, tid);
      __syncthreads();
#pragma unroll
      for (int sub = 0; sub < CODES_BN / 32; ++sub) {
        const int js = j0 + sub * 32;
        if (js >= T || (a.causal && js > iw + 31)) continue;  // wave-uniform
        float kop[D / 2];
        const float *kr = Ks + (sub * 32 + l32) * DS + half * (D / 2);
#pragma unroll
        for (int c = 0; c < D / 2; c += 4) {
          const f32x4 x = *reinterpret_cast<const f32x4 *>(kr + c);
          kop[c] = x[0]; kop[c + 1] = x[1]; kop[c + 2] = x[2]; kop[c + 3] = x[3];
        }
        const f32x16 acc = score_tile<D>(kop, qop);
        float u[16];
        decide_u<CALIB>(acc, rc, M, Mn, K, a.tau, a.scale, u);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int j = js + krel(r, half);
          const bool valid = j <= jlim;
          const float sc = acc[r] * a.scale;
          const float z = score_shift(acc[r], a.scale, M);
          const float e = valid ? expf(z) : 0.f;
          float w; int b; bool top;
          native(u[r], w, b, top);
          if (pass == 0) {
            WE += e;
            A += e * z;
            topE += top ? e : 0.f;
            cnt6 += (valid && (double)sc - (double)M < -6.0) ? 1 : 0;
            if (valid) {
              smin = fminf(smin, sc);
              atomicAdd(&bucket[lrow * NB + b], e);
              if (sc < low[LQ - 1]) {
                float x = sc;
#pragma unroll
                for (int e2 = 0; e2 < LQ; ++e2) {
                  const float lo = fminf(low[e2], x);
                  x = fmaxf(low[e2], x);
                  low[e2] = lo;
                }
              }
            }
          } else if (valid) {
            tv += fabsf(w / W - e / WEt);
          }
        }
      }
    }
    if (pass == 0) WE += __shfl_xor(WE, 32);
  }
  A += __shfl_xor(A, 32);
  topE += __shfl_xor(topE, 32);
  cnt6 += __shfl_xor(cnt6, 32);
  smin = fminf(smin, __shfl_xor(smin, 32));
  tv += __shfl_xor(tv, 32);
  qss += __shfl_xor(qss, 32);
  kss += __shfl_xor(kss, 32);
  // the partner half's smallest scores merged into this lane's list (read
  // in full first: both halves merge at once)
  float other[LQ];
#pragma unroll
  for (int e = 0; e < LQ; ++e) other[e] = __shfl_xor(low[e], 32);
#pragma unroll
  for (int e = 0; e < LQ; ++e) {
    float x = other[e];
#pragma unroll
    for (int e2 = 0; e2 < LQ; ++e2) {
      const float lo = fminf(low[e2], x);
      x = fmaxf(low[e2], x);
      low[e2] = lo;
    }
  }
  __syncthreads();
  if (half == 1 || row >= T) return;
  const int n = a.causal ? row + 1 : T;
  float Hq = 0.f;
  for (int b = 0; b < NB; ++b) {
    const float mb = bucket[lrow * NB + b];
    Hq += mb > 0.f ? mb * logf(mb) : 0.f;
  }
  const float lWE = logf(WE);
  // 0.1% quantile of z: linear interpolation at (n - 1) * 0.001 between
  // the order statistics lo and lo + 1 of the row's scores
  const double pos = (double)(n - 1) * 0.001;
  const int lo = (int)floor(pos), hi = lo + 1 < n ? lo + 1 : lo;
  float slo = low[0], shi = low[0];
#pragma unroll
  for (int e = 1; e < LQ; ++e) {
    slo = e == lo ? low[e] : slo;
    shi = e == hi ? low[e] : shi;
  }
  const double zlo = (double)slo - (double)M, zhi = (double)shi - (double)M;
  float *o = a.out + ((size_t)bh * T + row) * GEO_COUNT;
  const float span = M - smin;
  o[0] = span;
  o[1] = CALIB == CAL_MINMAX ? span / Kf : a.tau / Kf;
  o[2] = (float)(zlo + (pos - (double)lo) * (zhi - zlo));
  o[3] = sqrtf(qss);
  o[4] = sqrtf(kss);
  o[5] = lWE - A / WE;
  o[6] = (float)cnt6 / (float)n;
  o[7] = topE / WE;
  o[8] = expf(lWE - Hq / WE);
  o[9] = 0.5f * tv;
}

#define KIA_GEO_INST(D)                                                        \
  template __global__ void geometry_kernel<D, CAL_MINMAX, REC_LERP, 3>(GeoArgs);     \
  template __global__ void geometry_kernel<D, CAL_MINMAX, REC_NEAREST, 3>(GeoArgs);  \
  template __global__ void geometry_kernel<D, CAL_FWM, REC_LERP, 3>(GeoArgs);        \
  template __global__ void geometry_kernel<D, CAL_FWM, REC_NEAREST, 3>(GeoArgs);     \
  template __global__ void geometry_kernel<D, CAL_MINMAX, REC_LERP, 12>(GeoArgs);    \
  template __global__ void geometry_kernel<D, CAL_MINMAX, REC_NEAREST, 12>(GeoArgs); \
  template __global__ void geometry_kernel<D, CAL_FWM, REC_LERP, 12>(GeoArgs);       \
  template __global__ void geometry_kernel<D, CAL_FWM, REC_NEAREST, 12>(GeoArgs);    \
  template __global__ void geometry_kernel<D, CAL_MINMAX, REC_LERP, 67>(GeoArgs);    \
  template __global__ void geometry_kernel<D, CAL_MINMAX, REC_NEAREST, 67>(GeoArgs); \
  template __global__ void geometry_kernel<D, CAL_FWM, REC_LERP, 67>(GeoArgs);       \
  template __global__ void geometry_kernel<D, CAL_FWM, REC_NEAREST, 67>(GeoArgs);
KIA_GEO_INST(16)
KIA_GEO_INST(32)
KIA_GEO_INST(64)
KIA_GEO_INST(128)

// ---------------------------------------------------------------------------
// Matrix-core peak probe (a measurement aid, not part of the operator): four
// independent accumulator chains of v_mfma_f32_32x32x2_f32 on register
// operands, `iters` rounds per wave. Workgroup 0's first wave records the
// shader clock counter and the 100 MHz constant-rate counter around its loop.
__global__ __launch_bounds__(256) void mfma_probe_kernel(unsigned long long *out, int iters) {
  const int lane = threadIdx.x & 63;
  const float x = 0.001f * (float)lane, y = 1.f - 0.0005f * (float)lane;
  f32x16 c0, c1, c2, c3;
#pragma unroll
  for (int e = 0; e < 16; ++e) c0[e] = c1[e] = c2[e] = c3[e] = 0.f;
  __builtin_amdgcn_sched_barrier(0);
  const unsigned long long t0 = __builtin_amdgcn_s_memtime();
  const unsigned long long r0 = __builtin_amdgcn_s_memrealtime();
  __builtin_amdgcn_sched_barrier(0);
  for (int i = 0; i < iters; ++i) {
    c0 = mfma32(x, y, c0);
    c1 = mfma32(y, x, c1);
    c2 = mfma32(x, x, c2);
    c3 = mfma32(y, y, c3);
  }
  __builtin_amdgcn_sched_barrier(0);
  float sum = 0.f;
#pragma unroll
  for (int e = 0; e < 16; ++e) sum += c0[e] + c1[e] + c2[e] + c3[e];
  const unsigned long long t1 = __builtin_amdgcn_s_memtime();
  const unsigned long long r1 = __builtin_amdgcn_s_memrealtime();
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    out[0] = t0; out[1] = t1; out[2] = r0; out[3] = r1;
  }
  if (sum == -1.f) out[0] = 0;  // never true (all products are >= 0): keeps the chains live
}

#define KIA_FWD_KP(D, KP)                                                        \
  template __global__ void fwd_kernel<D, CAL_MINMAX, REC_LERP, false, KP>(FwdArgs);     \
  template __global__ void fwd_kernel<D, CAL_MINMAX, REC_NEAREST, false, KP>(FwdArgs);  \
  template __global__ void fwd_kernel<D, CAL_MINMAX, REC_NEAREST, true, KP>(FwdArgs);   \
  template __global__ void fwd_kernel<D, CAL_FWM, REC_LERP, false, KP>(FwdArgs);        \
  template __global__ void fwd_kernel<D, CAL_FWM, REC_NEAREST, false, KP>(FwdArgs);     \
  template __global__ void fwd_kernel<D, CAL_FWM, REC_NEAREST, true, KP>(FwdArgs);      \
  template __global__ void fwd_kernel<D, CAL_RESOLVED, REC_LERP, false, KP>(FwdArgs);   \
  template __global__ void fwd_kernel<D, CAL_RESOLVED, REC_NEAREST, false, KP>(FwdArgs);\
  template __global__ void fwd_kernel<D, CAL_RESOLVED, REC_NEAREST, true, KP>(FwdArgs); \
  template __global__ void fwd_kernel<D, CAL_FWM, REC_SOFTMAX, false, KP>(FwdArgs);     \
  template __global__ void fwd_kernel<D, CAL_FWM, REC_BF16EXP, false, KP>(FwdArgs);     \
  template __global__ void fwd_kernel<D, CAL_FWM, REC_FP8EXP, false, KP>(FwdArgs);
#define KIA_CODES_INST(D)                                                               \
  template __global__ void codes_kernel<D, CAL_MINMAX, REC_LERP, float>(CodesArgs);     \
  template __global__ void codes_kernel<D, CAL_FWM, REC_LERP, float>(CodesArgs);        \
  template __global__ void codes_kernel<D, CAL_RESOLVED, REC_LERP, float>(CodesArgs);   \
  template __global__ void codes_kernel<D, CAL_FWM, REC_SOFTMAX, float>(CodesArgs);     \
  template __global__ void codes_kernel<D, CAL_FWM, REC_BF16EXP, float>(CodesArgs);     \
  template __global__ void codes_kernel<D, CAL_FWM, REC_FP8EXP, float>(CodesArgs);      \
  template __global__ void codes_kernel<D, CAL_MINMAX, REC_LERP, uint16_t>(CodesArgs16);\
  template __global__ void codes_kernel<D, CAL_FWM, REC_LERP, uint16_t>(CodesArgs16);   \
  template __global__ void codes_kernel<D, CAL_RESOLVED, REC_LERP, uint16_t>(CodesArgs16);
KIA_FWD_KP(16, 2)
KIA_FWD_KP(32, 2)
KIA_FWD_KP(64, 2)
KIA_FWD_KP(128, 2)
// one row group and four (eight) key parts for grids too small to fill the chip
KIA_FWD_KP(16, 4)
KIA_FWD_KP(32, 4)
KIA_FWD_KP(64, 4)
KIA_FWD_KP(16, 8)
KIA_FWD_KP(32, 8)
KIA_FWD_KP(64, 8)
KIA_CODES_INST(16)
KIA_CODES_INST(32)
KIA_CODES_INST(64)
KIA_CODES_INST(128)
template __global__ void stored_codes_kernel<CAL_MINMAX, REC_LERP>(StoredCodesArgs);
template __global__ void stored_codes_kernel<CAL_FWM, REC_LERP>(StoredCodesArgs);
template __global__ void stored_codes_kernel<CAL_FWM, REC_NEAREST>(StoredCodesArgs);
template __global__ void stored_codes_kernel<CAL_RESOLVED, REC_LERP>(StoredCodesArgs);
template __global__ void stored_codes_kernel<CAL_FWM, REC_SOFTMAX>(StoredCodesArgs);
template __global__ void stored_codes_kernel<CAL_FWM, REC_BF16EXP>(StoredCodesArgs);
template __global__ void stored_codes_kernel<CAL_FWM, REC_FP8EXP>(StoredCodesArgs);
#define KIA_SCORES_INST(D)                                                  \
  template __global__ void scores_kernel<D, float>(ScoresArgsT<float>);     \
  template __global__ void scores_kernel<D, uint16_t>(ScoresArgsT<uint16_t>);
KIA_SCORES_INST(16)
KIA_SCORES_INST(32)
KIA_SCORES_INST(64)
KIA_SCORES_INST(128)

}  // namespace kia
