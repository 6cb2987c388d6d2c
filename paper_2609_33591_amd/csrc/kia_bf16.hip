// kia_bf16.hip -- the bf16-input variant of the forward and backward on
// gfx950: q, k, v and dO are bf16, every product runs on the bf16 MFMA
// (v_mfma_f32_32x32x16_bf16) with fp32 accumulation, and everything else
// (scores, extrema, index decisions, weights, normalizers, gradients of the
// scores, outputs) is fp32 as in the fp32 path. The computed operands of
// the second products (weights, dS) are rounded to bf16 for the MFMA.
//
// The kernels mirror the fp32 ones (kia_fwd.hip, kia_bwd.hip): same
// workgroup shapes and stats fields (the forward stores the score tiles in
// U and replaces them by the decided positions u, which the backward reads;
// recomputing the scores in the second pass is cheap on the bf16 MFMA but
// its extra staging registers cost more than the tile traffic at d = 128).
// The dS scratch holds bf16 (2 KiB per tile), the dQ product's operand
// precision. They also differ in the operand staging. A 32x32x16 MFMA takes 8 consecutive k-slots per lane
// half; in the products whose k index is a key (P V, dS K), a lane's own
// weight (or dS) registers r = 8t .. 8t+7 are the k-slots, that is the keys
// krel(8t + e, h), so V and K are staged transposed in LDS and a lane reads
// its 8 operands as two 8-byte runs of 4 consecutive keys. In the products
// whose k index is a query (P^T dO, dS^T Q), P and dS go through the
// wave-private transpose of the fp32 path and dO, Q are staged transposed.
#include <type_traits>

#include "kia_device.hpp"
#include "kia_kernels.hpp"

namespace kia {

constexpr int H16_CH = 64;  // keys per streamed chunk
constexpr int H16_TS = 68;  // row stride (bf16) of a transposed 64-key chunk
constexpr int H16_QT = 40;  // row stride (bf16) of a transposed 32-query tile
constexpr int H16_XS = 40;  // wave-private transpose row stride (bf16)
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));

template <int D> struct Dims16 {
  static constexpr int NC = D >= 32 ? D / 32 : 1;  // 32-column output blocks
  static constexpr int RS = D + 8;                  // row-major LDS row (bf16)
};

__device__ __forceinline__ bf16x8 pair_bf16x8(uint2 lo, uint2 hi) {
  return as_bf16x8(make_uint4(lo.x, lo.y, hi.x, hi.y));
}

// Register prefetch of a [ROWS, D] bf16 slice by NT threads in blocks of 4
// rows x 8 columns (one 16-byte load per row). The loads are unconditional
// (clamped rows) and masked when stashed into LDS, row-major or transposed.
template <int D, int ROWS, int NT> struct Blocks16 {
  static constexpr int CB = D / 8;
  static constexpr int NB = (ROWS / 4) * CB;
  static constexpr int PB = (NB + NT - 1) / NT;
  uint4 x[PB][4];
  uint32_t ok;
  __device__ __forceinline__ void fetch(const uint16_t *slice, int j0, int T, int tid) {
    ok = 0;
#pragma unroll
    for (int e = 0; e < PB; ++e) {
      const int b = tid + NT * e;
      const bool bv = b < NB;
      const int rb = bv ? b / CB : 0, cb = bv ? b % CB : 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = j0 + 4 * rb + i;
        const bool v = bv & (row < T);
        ok |= (v ? 1u : 0u) << (4 * e + i);
        x[e][i] = *reinterpret_cast<const uint4 *>(slice + (size_t)(v ? row : 0) * D + 8 * cb);
      }
    }
  }
  template <int RSTRIDE>
  __device__ __forceinline__ void stash_rows(uint16_t *dst, int tid) const {
#pragma unroll
    for (int e = 0; e < PB; ++e) {
      const int b = tid + NT * e;
      if (b < NB) {
        const int rb = b / CB, cb = b % CB;
#pragma unroll
        for (int i = 0; i < 4; ++i)
          *reinterpret_cast<uint4 *>(dst + (4 * rb + i) * RSTRIDE + 8 * cb) =
              ((ok >> (4 * e + i)) & 1u) ? x[e][i] : make_uint4(0, 0, 0, 0);
      }
    }
  }
  // column 8cb + c of the block's 4 rows -> dst[(8cb + c) * TSTRIDE + 4rb ..]
  template <int TSTRIDE>
  __device__ __forceinline__ void stash_cols(uint16_t *dst, int tid) const {
#pragma unroll
    for (int e = 0; e < PB; ++e) {
      const int b = tid + NT * e;
      if (b < NB) {
        const int rb = b / CB, cb = b % CB;
        uint32_t w[4][4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const uint4 v = ((ok >> (4 * e + i)) & 1u) ? x[e][i] : make_uint4(0, 0, 0, 0);
          w[i][0] = v.x; w[i][1] = v.y; w[i][2] = v.z; w[i][3] = v.w;
        }
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          const int dw = c >> 1;
          uint32_t p01, p23;
          if (c & 1) {
            p01 = (w[0][dw] >> 16) | (w[1][dw] & 0xffff0000u);
            p23 = (w[2][dw] >> 16) | (w[3][dw] & 0xffff0000u);
          } else {
            p01 = (w[0][dw] & 0xffffu) | (w[1][dw] << 16);
            p23 = (w[2][dw] & 0xffffu) | (w[3][dw] << 16);
          }
          *reinterpret_cast<uint2 *>(dst + (8 * cb + c) * TSTRIDE + 4 * rb) = make_uint2(p01, p23);
        }
      }
    }
  }
};

// ---------------------------------------------------------------------------
// Forward: one workgroup = 4 waves = 64 query rows = 2 row groups x 2 key
// halves, as fwd_kernel; K chunks row-major (score sub-tile A operand), V
// chunks transposed (P V A operand).
template <int D, int CALIB, int RECON, bool OL>
__global__ __launch_bounds__(256, 2) void fwd16_kernel(FwdArgs16 a) {
  constexpr int NC = Dims16<D>::NC, RS = Dims16<D>::RS;
  // MinMax and the resolved grid need the row minimum (resolved: for the
  // rounding margin of its far keys only)
  constexpr bool TRACKMIN = CALIB != CAL_FWM, NEAREST = RECON == REC_NEAREST;
  constexpr int NRED = NC * 16 * (OL ? 2 : 1) + 2;
  constexpr int KBUF = H16_CH * RS;  // bf16 per K chunk
  constexpr int VBUF = D * H16_TS;   // bf16 per transposed V chunk
  constexpr int STAGE = 2 * KBUF + 2 * VBUF;
  constexpr int RED = 2 * 64 * NRED * 2;  // reduction floats, in bf16 units
  constexpr int SM = STAGE > RED ? STAGE : RED;
  __shared__ __attribute__((aligned(16))) uint16_t smem[SM];
  __shared__ int Xc[2][2][6][32];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, half = lane >> 5, l32 = lane & 31;
  const int pr = wave & 1, kh = wave >> 1;
  const int T = a.T;
  const int nqb = (T + 63) / 64;
  const int bh = blockIdx.x % a.BH;
  const int qb = nqb - 1 - (int)(blockIdx.x / a.BH);
  const int i0 = qb * 64;
  const int iw = i0 + pr * 32;
  const int row = iw + l32;
  const size_t slice = (size_t)bh * T * D;
  const uint16_t *qs = a.q + slice, *ks = a.k + slice, *vs = a.v + slice;
  const float Kf = (float)a.K;
  const int jlim = a.causal ? min(row, T - 1) : T - 1;
  const int wlim = iw >= T ? -1 : (a.causal ? min(iw + 31, T - 1) : T - 1);
  // every key j <= wmin is valid for every row of the wave
  const int wmin = a.causal ? min(iw, T - 1) : T - 1;
  const int kend = a.causal ? min(T, i0 + 64) : T;
  const int nstep = (kend + H16_CH - 1) / H16_CH;
  const int npw = wlim < kh * 32 ? 0 : min(nstep, (wlim - kh * 32) / H16_CH + 1);
  float *Ut = a.st.U + ds_tile(bh, iw / 32, kh, (T + 31) / 32, a.causal) * 1024;

  bf16x8 qop[D / 16];
  load_rows16<D>(qs, row < T ? row : T - 1, T, half, qop);

  // ---------------- pass 1: scores, extrema, first index, tie counts -----
  float Mx = -INFINITY, Mn = INFINITY;
  int ax = 0x7fffffff, an = 0x7fffffff, cx = 0, cn = 0;
  {
    Blocks16<D, H16_CH, 256> fk;
    fk.fetch(ks, 0, T, tid);
    fk.template stash_rows<RS>(smem, tid);
    lds_barrier();
    for (int p = 0; p < nstep; ++p) {
      fk.fetch(ks, min(p + 1, nstep - 1) * H16_CH, T, tid);
      if (p < npw) {
        const int js = p * H16_CH + kh * 32;
        const uint16_t *kr = smem + (p & 1) * KBUF + (kh * 32 + l32) * RS + 8 * half;
        bf16x8 kop[D / 16];
#pragma unroll
        for (int s = 0; s < D / 16; ++s) kop[s] = as_bf16x8(*reinterpret_cast<const uint4 *>(kr + 16 * s));
        const f32x16 acc = score_tile16<D>(kop, qop);
        {
          float sv[16];
#pragma unroll
          for (int r = 0; r < 16; ++r) sv[r] = acc[r];
          tile_store(Ut + (size_t)p * 2048, lane, sv);
        }
        float sx[16];
        if (js + 31 <= wmin) {
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
      fk.template stash_rows<RS>(smem + ((p + 1) & 1) * KBUF, tid);
      lds_barrier();
    }
  }
  auto merge = [](bool mx, float &M, int &ai, int &c, float M2, int a2, int c2) {
    const bool take = mx ? (M2 > M) : (M2 < M);
    const bool tie = M2 == M;
    ai = take ? a2 : (tie ? min(ai, a2) : ai);
    c = take ? c2 : (tie ? c + c2 : c);
    M = take ? M2 : M;
  };
  merge(true, Mx, ax, cx, __shfl_xor(Mx, 32), __shfl_xor(ax, 32), __shfl_xor(cx, 32));
  if constexpr (TRACKMIN)
    merge(false, Mn, an, cn, __shfl_xor(Mn, 32), __shfl_xor(an, 32), __shfl_xor(cn, 32));
  if (half == 0) {
    int *x = &Xc[pr][kh][0][l32];
    x[0] = __float_as_int(Mx); x[32] = ax; x[64] = cx;
    x[96] = __float_as_int(Mn); x[128] = an; x[160] = cn;
  }
  __syncthreads();
  {
    const int *x0 = &Xc[pr][0][0][l32], *x1 = &Xc[pr][1][0][l32];
    Mx = __int_as_float(x0[0]); ax = x0[32]; cx = x0[64];
    merge(true, Mx, ax, cx, __int_as_float(x1[0]), x1[32], x1[64]);
    if constexpr (TRACKMIN) {
      Mn = __int_as_float(x0[96]); an = x0[128]; cn = x0[160];
      merge(false, Mn, an, cn, __int_as_float(x1[96]), x1[128], x1[160]);
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
  if constexpr (!TRACKMIN) Mn = Mx;
  const RowConst rc = row_const(Mx, Mn, a.K, CALIB, a.tau, a.scale);

  // ---------------- pass 2: reconstruct, normalize, O = P V ---------------
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
  uint16_t *Vt = smem + 2 * KBUF;
  auto load_s = [&](int p, f32x16 &S) {
    float sv[16];
    tile_load(Ut + (size_t)p * 2048, lane, sv);
#pragma unroll
    for (int r = 0; r < 16; ++r) S[r] = sv[r];
  };
  auto tile = [&](int p, const f32x16 &S, auto masked_tag) {
    constexpr bool MASKED = decltype(masked_tag)::value;
    constexpr bool COMPACT = compact_codes<CALIB, RECON>();
    float u[16];
    uint32_t cw[4];
    decide_u<CALIB>(S, rc, Mx, Mn, a.K, a.tau, a.scale, u);
    if constexpr (!COMPACT) tile_store(Ut + (size_t)p * 2048, lane, u);
    const int js = p * H16_CH + kh * 32;
    float w[16], wl[16];
    float tWN = 0.f, tWL = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const KeyDec kd = key_of<CALIB>(u[r], Kf);
      if constexpr (COMPACT) code_put(cw, r, kd);
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
    if constexpr (COMPACT) codes_store(Ut + (size_t)p * 2048, lane, cw);
    WN += tWN;
    WLs += tWL;
    const uint16_t *Vb = Vt + (p & 1) * VBUF + kh * 32 + 4 * half;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const bf16x8 bw = to_bf16x8(&w[8 * t]);
      bf16x8 bl;
      if constexpr (OL) bl = to_bf16x8(&wl[8 * t]);
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const int col = 32 * c + l32;
        const uint16_t *vr = Vb + (col < D ? col : 0) * H16_TS + 16 * t;
        uint2 lo = *reinterpret_cast<const uint2 *>(vr);
        uint2 hi = *reinterpret_cast<const uint2 *>(vr + 8);
        if (col >= D) { lo = make_uint2(0, 0); hi = lo; }
        const bf16x8 av = pair_bf16x8(lo, hi);
        oacc[c] = mfma16(av, bw, oacc[c]);
        if constexpr (OL) olacc[c] = mfma16(av, bl, olacc[c]);
      }
    }
  };
  {
    Blocks16<D, H16_CH, 256> fv;
    fv.fetch(vs, 0, T, tid);
    fv.template stash_cols<H16_TS>(Vt, tid);
    f32x16 SA, SB;
    if (npw > 0) load_s(0, SA);
    // tiles below the wave's first row are interior (no causal mask)
    auto run = [&](int p, const f32x16 &S) {
      if (p * H16_CH + kh * 32 + 31 <= wmin)
        tile(p, S, std::integral_constant<bool, false>{});
      else
        tile(p, S, std::integral_constant<bool, true>{});
    };
    lds_barrier();
    for (int p = 0; p < nstep; p += 2) {
      fv.fetch(vs, min(p + 1, nstep - 1) * H16_CH, T, tid);
      if (p + 1 < npw) load_s(p + 1, SB);
      if (p < npw) run(p, SA);
      fv.template stash_cols<H16_TS>(Vt + ((p + 1) & 1) * VBUF, tid);
      lds_barrier();
      if (p + 1 >= nstep) break;
      fv.fetch(vs, min(p + 2, nstep - 1) * H16_CH, T, tid);
      if (p + 2 < npw) load_s(p + 2, SA);
      if (p + 1 < npw) run(p + 1, SB);
      fv.template stash_cols<H16_TS>(Vt + (p & 1) * VBUF, tid);
      lds_barrier();
    }
  }
  WN += __shfl_xor(WN, 32);
  WLs += __shfl_xor(WLs, 32);
  float *red = reinterpret_cast<float *>(smem) + pr * 64 * NRED + lane;
  if (kh == 1) {
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        red[(c * 16 + e) * 64] = oacc[c][e];
        if constexpr (OL) red[((NC + c) * 16 + e) * 64] = olacc[c][e];
      }
    red[(NRED - 2) * 64] = WN;
    red[(NRED - 1) * 64] = WLs;
  }
  __syncthreads();
  if (kh == 1) return;
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      oacc[c][e] += red[(c * 16 + e) * 64];
      if constexpr (OL) olacc[c][e] += red[((NC + c) * 16 + e) * 64];
    }
  WN += red[(NRED - 2) * 64];
  WLs += red[(NRED - 1) * 64];
  const float W = NEAREST ? WN : WLs;
  if (half == 0 && row < T) {
    a.st.W[ridx] = W;
    a.st.WL[ridx] = WLs;
  }
  if (row < T) {
    const float inv = 1.f / W, invl = 1.f / WLs;
    float *orow = a.o + slice + (size_t)row * D;
    uint16_t *orow16 = a.o16 + slice + (size_t)row * D;
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int n = c * 32 + 8 * g + 4 * half;
        if (n >= D) continue;
        f32x4 x = {oacc[c][4 * g] * inv, oacc[c][4 * g + 1] * inv,
                   oacc[c][4 * g + 2] * inv, oacc[c][4 * g + 3] * inv};
        if (a.o16)
          *reinterpret_cast<uint2 *>(orow16 + n) =
              make_uint2(pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]));
        else
          *reinterpret_cast<f32x4 *>(orow + n) = x;
        if constexpr (OL) {
          f32x4 y = {olacc[c][4 * g] * invl, olacc[c][4 * g + 1] * invl,
                     olacc[c][4 * g + 2] * invl, olacc[c][4 * g + 3] * invl};
          *reinterpret_cast<f32x4 *>(a.st.OL + ridx * D + n) = y;
        }
      }
  }
}

// ---------------------------------------------------------------------------
// Backward main (bf16 inputs): KV-major as bwd_main_shared_kernel, 8 waves
// in two groups of 4 taking alternate 32-query tiles; 128 keys per
// workgroup with V row-major in LDS (dP^T A operand); per group the query
// tile's dO row-major (dP^T B operand) and transposed (dV B operand) and Q
// transposed (dK B operand).
template <int D, int CALIB, int RECON, bool SPLIT>
__global__ __launch_bounds__(512, 1) void bwd16_main_kernel(BwdArgs16 a) {
  constexpr int NC = Dims16<D>::NC, RS = Dims16<D>::RS;
  constexpr int VR = 128 * RS;           // bf16: V rows of the workgroup
  constexpr int DOR = 32 * RS;           // bf16: dO rows of a query tile
  constexpr int TT = D * H16_QT;         // bf16: a transposed query tile
  constexpr int GRP = DOR + 2 * TT;      // bf16 per group: dO rows, dO^T, Q^T
  constexpr int XW = 8 * 32 * H16_XS;    // bf16: wave-private transposes
  constexpr int STAGE_B = 2 * (VR + 2 * GRP + XW);      // bytes
  constexpr int RED_B = 4 * NC * 16 * 64 * 4;           // bytes: one of dV/dK of group 1
  constexpr int SMB = STAGE_B > RED_B ? STAGE_B : RED_B;
  __shared__ __attribute__((aligned(16))) unsigned char smem[SMB];
  __shared__ __attribute__((aligned(16))) float Rec[2][32 * RR_COUNT];
  __shared__ float Part[2][4 * 32 * 2];
  uint16_t *Vr = reinterpret_cast<uint16_t *>(smem);
  uint16_t *G0 = Vr + VR;
  uint16_t *Xt = G0 + 2 * GRP;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, half = lane >> 5, l32 = lane & 31;
  const int grp = wave >> 2, wk = wave & 3, gtid = tid & 255;
  const int T = a.T;
  const int nq = (T + 31) / 32;
  // key block (ascending: the longest causal key blocks first) and the part
  // of its query range (qsplit parts of nearly equal tile counts)
  const int qsplit = SPLIT ? a.qsplit : 1;
  const int kb = (int)(blockIdx.x / a.BH) / qsplit;
  const int qpart = (int)(blockIdx.x / a.BH) % qsplit;
  const int bh = blockIdx.x % a.BH;
  const int j0 = kb * 128;
  const int jw = j0 + 32 * wk;
  const size_t slice = (size_t)bh * T * D;
  const uint16_t *qs = a.q + slice, *vs = a.v + slice, *dos = a.dO + slice;
  constexpr bool minmax = CALIB == CAL_MINMAX;
  constexpr bool nearest = RECON == REC_NEAREST;
  const bool want_cm = minmax & grad_channels(a.grad);
  const float invK = 1.f / (float)a.K, Kf = (float)a.K;
  uint16_t *dOr = G0 + grp * GRP, *dOt = dOr + DOR, *Qt = dOt + TT;

  {
    Blocks16<D, 128, 512> fvv;
    fvv.fetch(vs, j0, T, tid);
    fvv.template stash_rows<RS>(Vr, tid);
  }

  f32x16 dva[NC], dka[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) { dva[c][e] = 0.f; dka[c][e] = 0.f; }

  Blocks16<D, 32, 256> fq, fd;
  f32x4 prr;
  uint32_t prok;
  auto fetch = [&](int i0) {
    fq.fetch(qs, i0, T, gtid);
    fd.fetch(dos, i0, T, gtid);
    const int r = (gtid / (RR_COUNT / 4)) % 32, c4 = gtid % (RR_COUNT / 4);
    const bool ok = (gtid < 32 * RR_COUNT / 4) & (i0 + r < T);
    prok = ok ? 1u : 0u;
    const size_t rix = (size_t)bh * T + (ok ? i0 + r : 0);
    prr = *reinterpret_cast<const f32x4 *>(a.st.rowrec + rix * RR_COUNT + c4 * 4);
  };
  auto stash = [&]() {
    fq.template stash_cols<H16_QT>(Qt, gtid);
    fd.template stash_rows<RS>(dOr, gtid);
    fd.template stash_cols<H16_QT>(dOt, gtid);
    if (gtid < 32 * RR_COUNT / 4) {
      const f32x4 pad = {0.f, (gtid % (RR_COUNT / 4)) == 0 ? (float)a.K : 0.f, 0.f, 0.f};
      *reinterpret_cast<f32x4 *>(&Rec[grp][gtid * 4]) = prok ? prr : pad;
    }
  };

  const int q0 = a.causal ? j0 : 0;
  const int ntall = (T - q0 + 31) / 32;
  const int tb = ntall * qpart / qsplit, te = ntall * (qpart + 1) / qsplit;
  const int qstart = q0 + tb * 32;
  const int nt = te - tb;
  const int npair = (nt + 1) / 2;
  uint16_t *Xw = Xt + wave * 32 * H16_XS;
  if (grp < nt) fetch(qstart + grp * 32);
  for (int it = 0; it < npair; ++it) {
    const int t = 2 * it + grp;
    const int i0 = qstart + t * 32;
    if (t < nt) stash();
    lds_barrier();
    if (t + 2 < nt) fetch(i0 + 64);

    float ps = 0.f, pm = 0.f;
    const bool active = (t < nt) & (jw < T) & !(a.causal & (jw > i0 + 31));
    if (active) {
      // the forward's decided positions (one byte per key under FWM with
      // Nearest)
      constexpr bool COMPACT = compact_codes<CALIB, RECON>();
      float u[16];
      uint4 cw;
      {
        const float *ut = a.st.U + ds_tile(bh, i0 / 32, jw / 32, nq, a.causal) * 1024;
        if constexpr (COMPACT) cw = codes_load(ut, lane);
        else tile_load(ut, lane, u);
      }
      f32x16 G;
#pragma unroll
      for (int e = 0; e < 16; ++e) G[e] = 0.f;
      {
        const uint16_t *vr = Vr + (32 * wk + l32) * RS + 8 * half;
        const uint16_t *dr = dOr + l32 * RS + 8 * half;
#pragma unroll
        for (int s = 0; s < D / 16; ++s)
          G = mfma16(as_bf16x8(*reinterpret_cast<const uint4 *>(vr + 16 * s)),
                     as_bf16x8(*reinterpret_cast<const uint4 *>(dr + 16 * s)), G);
      }
      const float *rr = Rec[grp] + l32 * RR_COUNT;
      const f32x4 r0 = *reinterpret_cast<const f32x4 *>(rr);
      const f32x4 r1 = *reinterpret_cast<const f32x4 *>(rr + 4);
      const f32x4 r2 = *reinterpret_cast<const f32x4 *>(rr + 8);
      const f32x4 r3 = *reinterpret_cast<const f32x4 *>(rr + 12);
      RowConst rc;
      rc.alpha = r0[0]; rc.beta = r0[1]; rc.margin2 = r0[2]; rc.hl = r0[3];
      rc.b1l = r1[0]; rc.emh = r1[1]; rc.dcoef = r1[2];
      rc.degen = r3[0] != 0.f;
      const float invWf = r1[3], invWX = r2[0], negDXW = r2[1];
      const int i = i0 + l32;
      const int jlim = i < T ? (a.causal ? i : T - 1) : -1;
      float P[16], dS[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        KeyDec kd;
        if constexpr (COMPACT) kd = key_of_code(cw, r);
        else kd = key_of<CALIB>(u[r], Kf);
        const bool valid = (jw + krel(r, half) <= jlim) & !kd.tail;
        const float Eu = grid_upper(kd.rf, rc);
        const float El = Eu * rc.emh;
        const float wL = fmaf(kd.t, Eu - El, El);
        const float wf = nearest ? (kd.up ? Eu : El) : wL;
        const float gamma = fmaf(G[r], invWX, negDXW);
        const float Delta = Eu * rc.dcoef;
        P[r] = valid ? wf * invWf : 0.f;
        dS[r] = valid ? gamma * Delta : 0.f;
        ps += dS[r];
        if (want_cm) {
          const float uc = kd.rf + kd.t;
          const float X = fmaf(kd.rf, wL, kd.t * Eu) * invK;
          const float dM = X - wL - Delta * uc * invK;
          pm += valid ? gamma * dM : 0.f;
        }
      }
      {
        // dS rounded to bf16 (the dQ product's operand), 2 KiB per tile:
        // element (lane l, register r) at (r/8)*512 + 8l + r%8
        uint16_t *dst = reinterpret_cast<uint16_t *>(a.st.dS) +
                        ds_tile(bh, i0 / 32, jw / 32, nq, a.causal) * 1024 + 8 * lane;
#pragma unroll
        for (int t2 = 0; t2 < 2; ++t2)
          *reinterpret_cast<bf16x8 *>(dst + 512 * t2) = to_bf16x8(&dS[8 * t2]);
      }
      // dV += P^T dO, dK += dS^T Q: k-slots are the queries 16t + 8h + e;
      // the operand goes through the wave's private LDS tile rounded to bf16
      auto transposed_product = [&](const float (&X)[16], const uint16_t *Bt, f32x16 (&acc)[NC]) {
#pragma unroll
        for (int r = 0; r < 16; ++r)
          Xw[krel(r, half) * H16_XS + l32] = __builtin_bit_cast(uint16_t, (__bf16)X[r]);
#pragma unroll
        for (int t2 = 0; t2 < 2; ++t2) {
          // read as a vector of the stored element type (a uint4 read may be
          // moved above the 16-bit stores it does not alias by type)
          const bf16x8 av = __builtin_bit_cast(
              bf16x8, *reinterpret_cast<const u16x8 *>(Xw + l32 * H16_XS + 16 * t2 + 8 * half));
#pragma unroll
          for (int c = 0; c < NC; ++c) {
            const int col = 32 * c + l32;
            uint4 bv = *reinterpret_cast<const uint4 *>(Bt + (col < D ? col : 0) * H16_QT + 16 * t2 + 8 * half);
            if (col >= D) bv = make_uint4(0, 0, 0, 0);
            acc[c] = mfma16(av, as_bf16x8(bv), acc[c]);
          }
        }
      };
      transposed_product(P, dOt, dva);
      transposed_product(dS, Qt, dka);
    }
    ps += __shfl_xor(ps, 32);
    pm += __shfl_xor(pm, 32);
    if (half == 0) {
      Part[grp][(wk * 32 + l32) * 2] = ps;
      Part[grp][(wk * 32 + l32) * 2 + 1] = pm;
    }
    lds_barrier();
    if (a.grad != GRAD_DETACH && wk == 0 && lane < 32 && t < nt && i0 + lane < T) {
      float sv = 0.f, mm = 0.f;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        sv += Part[grp][(w * 32 + lane) * 2];
        mm += Part[grp][(w * 32 + lane) * 2 + 1];
      }
      const size_t ridx = (size_t)bh * T + i0 + lane;
      put_row_sums(a, kb, ridx, sv, mm, minmax);
    }
  }
  // sum the two groups' dV, then dK (group 1 -> LDS -> group 0), and store;
  // the buffer overlaps V and the tiles: a workgroup with an empty query
  // part (only a split range has one) ran no iteration, whose barriers would
  // have seen its V stash land, so it waits here
  if (SPLIT && nt == 0) __syncthreads();
  float *red = reinterpret_cast<float *>(smem) + (size_t)wk * (NC * 16 * 64) + lane;
#pragma unroll
  for (int which = 0; which < 2; ++which) {
    f32x16 (&acc)[NC] = which == 0 ? dva : dka;
    if (grp == 1) {
#pragma unroll
      for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r) red[(c * 16 + r) * 64] = acc[c][r];
    }
    __syncthreads();
    if (grp == 0) {
#pragma unroll
      for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int j = jw + krel(r, half);
          const int col = 32 * c + l32;
          const float v = acc[c][r] + red[(c * 16 + r) * 64];
          if (j < T && col < D) {
            const size_t e = slice + (size_t)j * D + col;
            if constexpr (SPLIT) {  // parts of the query range add up (zeroed by bwd_pre)
              if (which == 1) atomicAdd(a.dk + e, a.scale * v);
              else atomicAdd(a.dv + e, v);
            } else if (which == 1) a.dk[e] = a.scale * v;
            else if (a.dv16) a.dv16[e] = (uint16_t)(__float_as_uint(bf16_rne(v)) >> 16);
            else a.dv[e] = v;
          }
        }
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// dQ (bf16 inputs) = scale * (dS K + calibration terms): as bwd_dq_kernel,
// with each 64-key chunk of K staged transposed in bf16 and the fp32 dS
// tiles (stored in bf16 by bwd16_main_kernel) as the A operand.
template <int D>
__global__ __launch_bounds__(512) void bwd16_dq_kernel(BwdArgs16 a) {
  constexpr int NC = Dims16<D>::NC;
  constexpr int KT = D * H16_TS;  // bf16 per transposed chunk
  constexpr int STAGE_B = 2 * KT * 2;
  constexpr int RED_B = 4 * NC * 16 * 64 * 4;
  constexpr int SMB = STAGE_B > RED_B ? STAGE_B : RED_B;
  __shared__ __attribute__((aligned(16))) unsigned char smem[SMB];
  uint16_t *Kt = reinterpret_cast<uint16_t *>(smem);

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, half = lane >> 5, l32 = lane & 31;
  const int pq = wave & 3, kh = wave >> 2;
  const int T = a.T;
  const int nq = (T + 31) / 32;
  const int npq = (nq + 3) / 4;
  const int bh = blockIdx.x % a.BH;
  const int g = npq - 1 - (int)(blockIdx.x / a.BH);
  const int qt = 4 * g + pq;
  const bool live = qt < nq;
  const int qtc = live ? qt : nq - 1;
  const size_t slice = (size_t)bh * T * D;
  const uint16_t *ks = a.k + slice;
  const int kend = a.causal ? min(T, (4 * g + 4) * 32) : T;
  const int nstep = (kend + 63) / 64;
  const int ktmine = a.causal ? qtc : nq - 1;
  const int npw = !live || ktmine < kh ? 0 : min(nstep, (ktmine - kh) / 2 + 1);
  const bool minmax = a.calib == CAL_MINMAX;

  f32x16 acc[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[c][e] = 0.f;

  Blocks16<D, 64, 512> kA, kB;
  uint4 dA[2], dB[2];
  auto fetch = [&](int p, Blocks16<D, 64, 512> &kx, uint4 (&dx)[2]) {
    kx.fetch(ks, p * 64, T, tid);
    const int kt = min(2 * p + kh, ktmine);
    // the bf16 dS tile of bwd16_main_kernel
    const uint16_t *src = reinterpret_cast<const uint16_t *>(a.st.dS) +
                          ds_tile(bh, qtc, kt, nq, a.causal) * 1024 + 8 * lane;
#pragma unroll
    for (int t = 0; t < 2; ++t) dx[t] = *reinterpret_cast<const uint4 *>(src + 512 * t);
  };
  auto mma = [&](int buf, const uint4 (&dx)[2]) {
    const uint16_t *kb = Kt + buf * KT + kh * 32 + 4 * half;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const bf16x8 av = as_bf16x8(dx[t]);
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const int col = 32 * c + l32;
        const uint16_t *kr = kb + (col < D ? col : 0) * H16_TS + 16 * t;
        uint2 lo = *reinterpret_cast<const uint2 *>(kr);
        uint2 hi = *reinterpret_cast<const uint2 *>(kr + 8);
        if (col >= D) { lo = make_uint2(0, 0); hi = lo; }
        acc[c] = mfma16(av, pair_bf16x8(lo, hi), acc[c]);
      }
    }
  };
  fetch(0, kA, dA);
  kA.template stash_cols<H16_TS>(Kt, tid);
  fetch(min(1, nstep - 1), kB, dB);
  lds_barrier();
  for (int p = 0; p < nstep; p += 2) {
    if (p < npw) mma(0, dA);
    kB.template stash_cols<H16_TS>(Kt + KT, tid);
    fetch(min(p + 2, nstep - 1), kA, dA);
    lds_barrier();
    if (p + 1 >= nstep) break;
    if (p + 1 < npw) mma(1, dB);
    kA.template stash_cols<H16_TS>(Kt, tid);
    fetch(min(p + 3, nstep - 1), kB, dB);
    lds_barrier();
  }
  {
    float *red = reinterpret_cast<float *>(smem) + pq * (NC * 16 * 64) + lane;
    if (kh == 1) {
#pragma unroll
      for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int e = 0; e < 16; ++e) red[(c * 16 + e) * 64] = acc[c][e];
    }
    __syncthreads();
    if (kh == 0) {
#pragma unroll
      for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[c][e] += red[(c * 16 + e) * 64];
    }
  }
  if (!live) return;  // no barrier below

  // calibration terms of rows with unique extrema (lanes 0..31: one row each)
  const int row = qt * 32 + l32;
  const size_t ridx = (size_t)bh * T + (row < T ? row : T - 1);
  bool ok = false;
  float cMt = 0.f, cm = 0.f;
  int am = 0, an = 0;
  if (grad_channels(a.grad) && row < T && a.st.rowrec[ridx * RR_COUNT + RR_FLAGS] == 0.f) {
    const int nmax = a.st.nmax[ridx];
    const int nmin = minmax ? a.st.nmin[ridx] : 1;
    ok = (nmax == 1) & (nmin == 1);
    const float ss = a.st.sself[ridx];
    cMt = minmax ? a.st.cM[ridx] : -ss;
    cm = minmax ? -(ss + cMt) : 0.f;
    if (!grad_keep_max(a.grad)) cMt = 0.f;
    if (!grad_keep_min(a.grad)) cm = 0.f;
    am = a.st.amax[ridx];
    an = minmax ? a.st.amin[ridx] : am;
  }
  if (!ok) { cMt = 0.f; cm = 0.f; am = 0; an = 0; }
  if (kh == 0) {
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int src = krel(e, half);
      const float fM = __shfl(cMt, src), fm = __shfl(cm, src);
      const int iam = __shfl(am, src), ian = __shfl(an, src);
      const int qrow = qt * 32 + src;
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const int n = 32 * c + l32;
        const int nn = n < D ? n : 0;
        float v = acc[c][e];
        v = fmaf(fM, load1(ks + (size_t)iam * D + nn), v);
        v = fmaf(fm, load1(ks + (size_t)ian * D + nn), v);
        if (qrow < T && n < D) a.dq[slice + (size_t)qrow * D + n] = a.scale * v;
      }
    }
  }
  // scatter onto the argmax/argmin keys of dK (the deterministic backward
  // gathers these per key instead: one record per row for it)
  if (a.det && grad_channels(a.grad) && kh == 0 && half == 0 && row < T)
    put_calib_record(a.st.part, ridx, ok, minmax, am, an, cMt * a.scale, cm * a.scale);
  if (grad_channels(a.grad) && !a.det) {
    constexpr int NE = (D + 63) / 64;
    for (int rr0 = 16 * kh; rr0 < 16 * kh + 16; rr0 += 8) {
      float qv[8][NE];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int qrow = qt * 32 + rr0 + u;
#pragma unroll
        for (int x = 0; x < NE; ++x) {
          const int n = lane + 64 * x;
          const int qr = qrow < T ? qrow : T - 1, nn = n < D ? n : 0;
          qv[u][x] = load1(a.q + slice + (size_t)qr * D + nn);
        }
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int rr = rr0 + u;
        if (!__shfl(ok ? 1 : 0, rr)) continue;  // wave-uniform
        const float fM = __shfl(cMt, rr) * a.scale, fm = __shfl(cm, rr) * a.scale;
        const int iam = __shfl(am, rr), ian = __shfl(an, rr);
#pragma unroll
        for (int x = 0; x < NE; ++x) {
          const int n = lane + 64 * x;
          if (n < D) {
            atomicAdd(a.dk + slice + (size_t)iam * D + n, fM * qv[u][x]);
            if (minmax) atomicAdd(a.dk + slice + (size_t)ian * D + n, fm * qv[u][x]);
          }
        }
      }
    }
  }
}

#define KIA_B16_INST(D)                                                                  \
  template __global__ void fwd16_kernel<D, CAL_MINMAX, REC_LERP, false>(FwdArgs16);      \
  template __global__ void fwd16_kernel<D, CAL_MINMAX, REC_NEAREST, false>(FwdArgs16);   \
  template __global__ void fwd16_kernel<D, CAL_MINMAX, REC_NEAREST, true>(FwdArgs16);    \
  template __global__ void fwd16_kernel<D, CAL_FWM, REC_LERP, false>(FwdArgs16);         \
  template __global__ void fwd16_kernel<D, CAL_FWM, REC_NEAREST, false>(FwdArgs16);      \
  template __global__ void fwd16_kernel<D, CAL_FWM, REC_NEAREST, true>(FwdArgs16);       \
  template __global__ void fwd16_kernel<D, CAL_RESOLVED, REC_LERP, false>(FwdArgs16);    \
  template __global__ void fwd16_kernel<D, CAL_RESOLVED, REC_NEAREST, false>(FwdArgs16); \
  template __global__ void fwd16_kernel<D, CAL_RESOLVED, REC_NEAREST, true>(FwdArgs16);  \
  template __global__ void bwd16_main_kernel<D, CAL_RESOLVED, REC_LERP, false>(BwdArgs16);    \
  template __global__ void bwd16_main_kernel<D, CAL_RESOLVED, REC_LERP, true>(BwdArgs16);     \
  template __global__ void bwd16_main_kernel<D, CAL_RESOLVED, REC_NEAREST, false>(BwdArgs16); \
  template __global__ void bwd16_main_kernel<D, CAL_RESOLVED, REC_NEAREST, true>(BwdArgs16);  \
  template __global__ void bwd16_main_kernel<D, CAL_MINMAX, REC_LERP, false>(BwdArgs16);      \
  template __global__ void bwd16_main_kernel<D, CAL_MINMAX, REC_LERP, true>(BwdArgs16);       \
  template __global__ void bwd16_main_kernel<D, CAL_MINMAX, REC_NEAREST, false>(BwdArgs16);   \
  template __global__ void bwd16_main_kernel<D, CAL_MINMAX, REC_NEAREST, true>(BwdArgs16);    \
  template __global__ void bwd16_main_kernel<D, CAL_FWM, REC_LERP, false>(BwdArgs16);         \
  template __global__ void bwd16_main_kernel<D, CAL_FWM, REC_LERP, true>(BwdArgs16);          \
  template __global__ void bwd16_main_kernel<D, CAL_FWM, REC_NEAREST, false>(BwdArgs16);      \
  template __global__ void bwd16_main_kernel<D, CAL_FWM, REC_NEAREST, true>(BwdArgs16);       \
  template __global__ void bwd16_dq_kernel<D>(BwdArgs16);
KIA_B16_INST(16)
KIA_B16_INST(32)
KIA_B16_INST(64)
KIA_B16_INST(128)

}  // namespace kia
