// kia_bwd.hip -- backward of causal K-interval attention on gfx950.
//
// Four launches on the caller's stream (App. B):
//  1. bwd_pre   per row: D^X = dO . O^X (O^X = O, or O^L for Prob-STE with
//               Nearest) and the row record (grid constants, 1/W, 1/W^X,
//               -D^X/W^X); zeroes the two row sums.
//  2. bwd_main  KV-major: one workgroup per 128 keys, 4 waves x 32 keys
//               keep their K and V rows in registers and stream 32-query
//               tiles (double-buffered in LDS, prefetched into registers
//               one tile ahead): S^T and dP^T on MFMA (the canonical
//               sub-tile, bit-identical to the forward), per key
//               gamma = (g - D^X)/W^X, Delta, dS = gamma Delta, the row sums
//               S_self = sum dS and (MinMax) sum gamma dw^L/dM
//               (Eq. calgrad); dV += P^T dO and dK += dS^T Q through a
//               wave-private LDS transpose; dS is written to a tiled fp32
//               scratch for the dQ product.
//  3. bwd_dq    Q-major: dQ = scale (dS K + calibration terms of the row):
//               Eq. (full) puts cM = sum_j gamma_j dw_j/dM on the argmax key
//               and cm = -(S_self + cM) (from Delta + dw/dM + dw/dm = 0) on
//               the argmin key; FWM has cM = -S_self. For rows with unique
//               extrema it also scatter-adds dK_amax += scale cM q_i and
//               dK_amin += scale cm q_i.
//  4. bwd_ties  (full gradient only) rows with tied extrema: recompute the
//               row's scores with the canonical sub-tile and split cM / cm
//               evenly over every key equal to M / m (edge-case table).
#include "kia_device.hpp"
#include "kia_kernels.hpp"

namespace kia {

constexpr int BKV = 128;  // keys per bwd_main workgroup
constexpr int BQ = 32;    // queries per streamed tile
constexpr int XS = 36;    // transpose buffer row stride (floats)

// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void bwd_pre_kernel(BwdArgs a) {
  constexpr int L = D / 4;  // lanes per row, one float4 each
  constexpr int RPB = 256 / L;
  const int tid = threadIdx.x;
  const int sub = tid % L;
  const size_t R = (size_t)a.BH * a.T;
  const size_t ridx = (size_t)blockIdx.x * RPB + tid / L;
  const bool live = ridx < R;
  const bool probN = (a.recon == REC_NEAREST) & (a.ste == STE_PROB);
  float dot = 0.f;
  if (live) {
    const float *ox = probN ? a.st.OL + ridx * D : a.o + ridx * D;
    const f32x4 x = *reinterpret_cast<const f32x4 *>(ox + sub * 4);
    const f32x4 y = *reinterpret_cast<const f32x4 *>(a.dO + ridx * D + sub * 4);
    dot = x[0] * y[0] + x[1] * y[1] + x[2] * y[2] + x[3] * y[3];
  }
#pragma unroll
  for (int off = L / 2; off > 0; off >>= 1) dot += __shfl_xor(dot, off);
  if (live && sub == 0) {
    const bool minmax = a.calib == CAL_MINMAX;
    const float M = a.st.M[ridx];
    const float m = minmax ? a.st.m[ridx] : M;
    const RowConst rc = row_const(M, m, a.K, a.calib, a.tau, a.scale);
    const float W = a.st.W[ridx];
    const float WX = probN ? a.st.WL[ridx] : W;
    const float invWX = 1.f / WX;
    f32x4 *rec = reinterpret_cast<f32x4 *>(a.st.rowrec + ridx * RR_COUNT);
    const f32x4 r0 = {rc.alpha, rc.beta, rc.margin2, rc.hl};
    const f32x4 r1 = {rc.b1l, rc.emh, rc.dcoef, 1.f / W};
    const f32x4 r2 = {invWX, -dot * invWX, M, m};
    const f32x4 r3 = {rc.degen ? 1.f : 0.f, 0.f, 0.f, 0.f};
    rec[0] = r0; rec[1] = r1; rec[2] = r2; rec[3] = r3;
    a.st.sself[ridx] = 0.f;
    a.st.cM[ridx] = 0.f;
  }
}

// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void bwd_main_kernel(BwdArgs a) {
  constexpr int NC = Dims<D>::NC, DS = Dims<D>::DS, DP = Dims<D>::DP;
  constexpr int QV4 = BQ * DP / 4;         // float4 per Q (or dO) tile
  constexpr int PF = (QV4 + 255) / 256;    // float4 per thread and tensor
  __shared__ __attribute__((aligned(16))) float Qs[2][BQ * DS];
  __shared__ __attribute__((aligned(16))) float dOs[2][BQ * DS];
  __shared__ __attribute__((aligned(16))) float Rec[2][BQ * RR_COUNT];
  __shared__ __attribute__((aligned(16))) float Xt[4 * 32 * XS];
  __shared__ float Part[2][4 * 32 * 2];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, half = lane >> 5, l32 = lane & 31;
  const int T = a.T;
  const int nq = (T + 31) / 32;
  const int kb = blockIdx.x / a.BH;  // ascending: the longest causal key blocks first
  const int bh = blockIdx.x % a.BH;
  const int j0 = kb * BKV;
  const int jw = j0 + 32 * wave;
  const size_t slice = (size_t)bh * T * D;
  const float *qs = a.q + slice, *ks = a.k + slice, *vs = a.v + slice,
              *dos = a.dO + slice;
  const bool minmax = a.calib == CAL_MINMAX;
  const bool nearest = a.recon == REC_NEAREST;
  const bool want_cm = minmax & !a.detach;
  const float invK = 1.f / (float)a.K;

  // this wave's 32 keys as A operands (canonical layout)
  float kop[D / 2], vop[D / 2];
  {
    const int key = jw + l32;
    const bool ok = key < T;
    const float *kr = ks + (size_t)(ok ? key : 0) * D + half * (D / 2);
    const float *vr = vs + (size_t)(ok ? key : 0) * D + half * (D / 2);
#pragma unroll
    for (int s = 0; s < D / 2; s += 4) {
      f32x4 x = *reinterpret_cast<const f32x4 *>(kr + s);
      f32x4 y = *reinterpret_cast<const f32x4 *>(vr + s);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        kop[s + e] = ok ? x[e] : 0.f;
        vop[s + e] = ok ? y[e] : 0.f;
      }
    }
  }

  f32x16 dva[NC], dka[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) { dva[c][e] = 0.f; dka[c][e] = 0.f; }

  // next-tile prefetch registers
  f32x4 pq[PF], pd[PF], pr;
  auto fetch = [&](int i0) {
#pragma unroll
    for (int e = 0; e < PF; ++e) {
      const int idx = tid + 256 * e;
      const int r = idx / (DP / 4), c4 = idx % (DP / 4);
      f32x4 x = {0.f, 0.f, 0.f, 0.f}, y = x;
      if (idx < QV4 && i0 + r < T && c4 * 4 < D) {
        x = *reinterpret_cast<const f32x4 *>(qs + (size_t)(i0 + r) * D + c4 * 4);
        y = *reinterpret_cast<const f32x4 *>(dos + (size_t)(i0 + r) * D + c4 * 4);
      }
      pq[e] = x;
      pd[e] = y;
    }
    pr = f32x4{0.f, 0.f, 0.f, 0.f};
    if (tid < BQ * RR_COUNT / 4) {
      const int r = tid / (RR_COUNT / 4), c4 = tid % (RR_COUNT / 4);
      if (i0 + r < T)
        pr = *reinterpret_cast<const f32x4 *>(a.st.rowrec + ((size_t)bh * T + i0 + r) * RR_COUNT + c4 * 4);
      else if (c4 == 0)
        pr[1] = (float)a.K;  // padding rows: u = K, never ambiguous
    }
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int e = 0; e < PF; ++e) {
      const int idx = tid + 256 * e;
      if (idx < QV4) {
        const int r = idx / (DP / 4), c4 = idx % (DP / 4);
        *reinterpret_cast<f32x4 *>(&Qs[buf][r * DS + c4 * 4]) = pq[e];
        *reinterpret_cast<f32x4 *>(&dOs[buf][r * DS + c4 * 4]) = pd[e];
      }
    }
    if (tid < BQ * RR_COUNT / 4) *reinterpret_cast<f32x4 *>(&Rec[buf][tid * 4]) = pr;
  };

  const int qstart = a.causal ? j0 : 0;
  const int nt = (T - qstart + BQ - 1) / BQ;
  float *Xw = Xt + wave * 32 * XS;
  fetch(qstart);
  stash(0);
  lds_barrier();
  for (int t = 0; t < nt; ++t) {
    const int buf = t & 1;
    const int i0 = qstart + t * BQ;
    if (t + 1 < nt) fetch(i0 + BQ);

    float ps = 0.f, pm = 0.f;
    const bool active = (jw < T) & !(a.causal & (jw > i0 + 31));
    if (active) {
      const float *Qb = Qs[buf], *dOb = dOs[buf];
      float qop[D / 2], dop[D / 2];
      {
        const float *qr = Qb + l32 * DS + half * (D / 2);
        const float *dr = dOb + l32 * DS + half * (D / 2);
#pragma unroll
        for (int s = 0; s < D / 2; s += 4) {
          f32x4 x = *reinterpret_cast<const f32x4 *>(qr + s);
          f32x4 y = *reinterpret_cast<const f32x4 *>(dr + s);
#pragma unroll
          for (int e = 0; e < 4; ++e) { qop[s + e] = x[e]; dop[s + e] = y[e]; }
        }
      }
      const f32x16 S = score_tile<D>(kop, qop);
      f32x16 G;
#pragma unroll
      for (int e = 0; e < 16; ++e) G[e] = 0.f;
#pragma unroll
      for (int s = 0; s < D / 2; ++s) G = mfma32(vop[s], dop[s], G);

      const float *rr = Rec[buf] + l32 * RR_COUNT;
      const f32x4 r0 = *reinterpret_cast<const f32x4 *>(rr);
      const f32x4 r1 = *reinterpret_cast<const f32x4 *>(rr + 4);
      const f32x4 r2 = *reinterpret_cast<const f32x4 *>(rr + 8);
      const f32x4 r3 = *reinterpret_cast<const f32x4 *>(rr + 12);
      RowConst rc;
      rc.alpha = r0[0]; rc.beta = r0[1]; rc.margin2 = r0[2]; rc.hl = r0[3];
      rc.b1l = r1[0]; rc.emh = r1[1]; rc.dcoef = r1[2];
      rc.degen = r3[0] != 0.f;
      const float invWf = r1[3], invWX = r2[0], negDXW = r2[1];
      const float M = r2[2], m = r2[3];
      Decided dd;
      decide16(S, rc, M, m, a.K, a.calib, a.tau, a.scale, dd);

      const int i = i0 + l32;
      float P[16], dS[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int j = jw + krel(r, half);
        const bool valid = (j < T) & (i < T) & (!a.causal | (j <= i)) &
                           !((dd.tail >> r) & 1u);
        const float Eu = grid_upper(dd.rf[r], rc);
        const float El = Eu * rc.emh;
        const float wL = fmaf(dd.t[r], Eu - El, El);
        const float wN = ((dd.up >> r) & 1u) ? Eu : El;
        const float wf = nearest ? wN : wL;
        const float gamma = fmaf(G[r], invWX, negDXW);
        const float Delta = Eu * rc.dcoef;
        P[r] = valid ? wf * invWf : 0.f;
        dS[r] = valid ? gamma * Delta : 0.f;
        ps += dS[r];
        if (want_cm) {
          // dw^L/dM = X - w^L - Delta u / K, X = (r w^L + t e^{b_{r+1}}) / K
          const float u = dd.rf[r] + dd.t[r];
          const float X = fmaf(dd.rf[r], wL, dd.t[r] * Eu) * invK;
          const float dM = X - wL - Delta * u * invK;
          pm += valid ? gamma * dM : 0.f;
        }
      }
      // dS tile to the scratch, lane-major (the dQ kernel's A operand)
      {
        float *dst = a.st.dS + ds_tile(bh, i0 / 32, jw / 32, nq, a.causal) * 1024 + lane * 16;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          f32x4 x = {dS[4 * g], dS[4 * g + 1], dS[4 * g + 2], dS[4 * g + 3]};
          *reinterpret_cast<f32x4 *>(dst + 4 * g) = x;
        }
      }
      // dV += P^T dO  (A = P transposed through LDS, B = dO rows)
#pragma unroll
      for (int r = 0; r < 16; ++r) Xw[krel(r, half) * XS + l32] = P[r];
      float at[16];
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 x = *reinterpret_cast<const f32x4 *>(Xw + l32 * XS + 16 * half + 4 * g);
        at[4 * g] = x[0]; at[4 * g + 1] = x[1]; at[4 * g + 2] = x[2]; at[4 * g + 3] = x[3];
      }
#pragma unroll
      for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int st = 0; st < 16; ++st)
          dva[c] = mfma32(at[st], dOb[(16 * half + st) * DS + 32 * c + l32], dva[c]);
      // dK += dS^T Q
#pragma unroll
      for (int r = 0; r < 16; ++r) Xw[krel(r, half) * XS + l32] = dS[r];
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 x = *reinterpret_cast<const f32x4 *>(Xw + l32 * XS + 16 * half + 4 * g);
        at[4 * g] = x[0]; at[4 * g + 1] = x[1]; at[4 * g + 2] = x[2]; at[4 * g + 3] = x[3];
      }
#pragma unroll
      for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int st = 0; st < 16; ++st)
          dka[c] = mfma32(at[st], Qb[(16 * half + st) * DS + 32 * c + l32], dka[c]);
    }
    ps += __shfl_xor(ps, 32);
    pm += __shfl_xor(pm, 32);
    if (half == 0) {
      Part[buf][(wave * 32 + l32) * 2] = ps;
      Part[buf][(wave * 32 + l32) * 2 + 1] = pm;
    }
    if (t + 1 < nt) stash(buf ^ 1);
    lds_barrier();
    if (!a.detach && tid < 32 && i0 + tid < T) {
      float s = 0.f, mm = 0.f;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        s += Part[buf][(w * 32 + tid) * 2];
        mm += Part[buf][(w * 32 + tid) * 2 + 1];
      }
      const size_t ridx = (size_t)bh * T + i0 + tid;
      atomicAdd(a.st.sself + ridx, s);
      if (minmax) atomicAdd(a.st.cM + ridx, mm);
    }
  }
  // write dV, dK (lane -> column, register -> key)
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int j = jw + krel(r, half);
      if (j < T && 32 * c + l32 < D) {
        a.dv[slice + (size_t)j * D + 32 * c + l32] = dva[c][r];
        a.dk[slice + (size_t)j * D + 32 * c + l32] = a.scale * dka[c][r];
      }
    }
}

// ---------------------------------------------------------------------------
// dQ = scale * (dS K + calibration terms), one wave per 32-query tile.
template <int D>
__global__ __launch_bounds__(256) void bwd_dq_kernel(BwdArgs a) {
  constexpr int NC = Dims<D>::NC, DS = Dims<D>::DS, DP = Dims<D>::DP;
  constexpr int KV4 = 32 * DP / 4 / 64;  // float4 per lane of one K sub-tile
  __shared__ __attribute__((aligned(16))) float Kw[4][2][32 * DS];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, half = lane >> 5, l32 = lane & 31;
  const int T = a.T;
  const int nq = (T + 31) / 32;
  const int ng = (nq + 3) / 4;
  const int bh = blockIdx.x % a.BH;
  const int g = ng - 1 - (int)(blockIdx.x / a.BH);  // heaviest query tiles first
  const int qt = 4 * g + wave;
  if (qt >= nq) return;  // whole wave; no workgroup barrier below
  const size_t slice = (size_t)bh * T * D;
  const float *ks = a.k + slice;
  const int ktmax = a.causal ? qt : nq - 1;
  const bool minmax = a.calib == CAL_MINMAX;

  f32x16 acc[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[c][e] = 0.f;

  f32x4 pk[KV4], pdS[4];
  auto fetch = [&](int kt) {
#pragma unroll
    for (int e = 0; e < KV4; ++e) {
      const int idx = lane + 64 * e;
      const int r = idx / (DP / 4), c4 = idx % (DP / 4);
      const int key = kt * 32 + r;
      f32x4 x = {0.f, 0.f, 0.f, 0.f};
      if (key < T && c4 * 4 < D) x = *reinterpret_cast<const f32x4 *>(ks + (size_t)key * D + c4 * 4);
      pk[e] = x;
    }
    const float *src = a.st.dS + ds_tile(bh, qt, kt, nq, a.causal) * 1024 + lane * 16;
#pragma unroll
    for (int e = 0; e < 4; ++e) pdS[e] = *reinterpret_cast<const f32x4 *>(src + 4 * e);
  };
  fetch(0);
  for (int kt = 0; kt <= ktmax; ++kt) {
    float *Kb = Kw[wave][kt & 1];
#pragma unroll
    for (int e = 0; e < KV4; ++e) {
      const int idx = lane + 64 * e;
      const int r = idx / (DP / 4), c4 = idx % (DP / 4);
      *reinterpret_cast<f32x4 *>(Kb + r * DS + c4 * 4) = pk[e];
    }
    float dsr[16];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      dsr[4 * e] = pdS[e][0]; dsr[4 * e + 1] = pdS[e][1];
      dsr[4 * e + 2] = pdS[e][2]; dsr[4 * e + 3] = pdS[e][3];
    }
    if (kt < ktmax) fetch(kt + 1);
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        acc[c] = mfma32(dsr[r], Kb[krel(r, half) * DS + 32 * c + l32], acc[c]);
  }

  // calibration terms of rows with unique extrema (lanes 0..31: one row each)
  const int row = qt * 32 + l32;
  const size_t ridx = (size_t)bh * T + (row < T ? row : T - 1);
  bool ok = false;
  float cMt = 0.f, cm = 0.f;
  int am = 0, an = 0;
  if (!a.detach && row < T && a.st.rowrec[ridx * RR_COUNT + RR_FLAGS] == 0.f) {
    const int nmax = a.st.nmax[ridx];
    const int nmin = minmax ? a.st.nmin[ridx] : 1;
    ok = (nmax == 1) & (nmin == 1);
    const float ss = a.st.sself[ridx];
    cMt = minmax ? a.st.cM[ridx] : -ss;
    cm = minmax ? -(ss + cMt) : 0.f;
    am = a.st.amax[ridx];
    an = minmax ? a.st.amin[ridx] : am;
  }
  if (!ok) { cMt = 0.f; cm = 0.f; am = 0; an = 0; }
  // dQ rows: register e holds query krel(e, half), lane column 32c + l32
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int src = krel(e, half);
    const float fM = __shfl(cMt, src), fm = __shfl(cm, src);
    const int iam = __shfl(am, src), ian = __shfl(an, src);
    const int qrow = qt * 32 + src;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int n = 32 * c + l32;
      if (qrow < T && n < D) {
        float v = acc[c][e];
        if (fM != 0.f) v = fmaf(fM, ks[(size_t)iam * D + n], v);
        if (fm != 0.f) v = fmaf(fm, ks[(size_t)ian * D + n], v);
        a.dq[slice + (size_t)qrow * D + n] = a.scale * v;
      }
    }
  }
  // scatter of the calibration terms onto the argmax/argmin keys of dK
  if (!a.detach) {
    for (int rr = 0; rr < 32; ++rr) {
      if (!__shfl(ok ? 1 : 0, rr)) continue;
      const float fM = __shfl(cMt, rr) * a.scale, fm = __shfl(cm, rr) * a.scale;
      const int iam = __shfl(am, rr), ian = __shfl(an, rr);
      const int qrow = qt * 32 + rr;
      for (int n = lane; n < D; n += 64) {
        const float qv = a.q[slice + (size_t)qrow * D + n];
        atomicAdd(a.dk + slice + (size_t)iam * D + n, fM * qv);
        if (minmax) atomicAdd(a.dk + slice + (size_t)ian * D + n, fm * qv);
      }
    }
  }
}

// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void bwd_ties_kernel(BwdArgs a) {
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, half = lane >> 5, l32 = lane & 31;
  const int T = a.T;
  const int nrb = (T + 31) / 32;
  const size_t gw = (size_t)blockIdx.x * 4 + wave;
  if (gw >= (size_t)a.BH * nrb) return;
  const int bh = (int)(gw / nrb), rb = (int)(gw % nrb);
  const int i = rb * 32 + l32;
  const bool minmax = a.calib == CAL_MINMAX;
  const size_t slice = (size_t)bh * T * D;
  const size_t ridx = (size_t)bh * T + (i < T ? i : T - 1);
  bool tierow = false;
  float M = 0.f, m = 0.f, coefM = 0.f, coefm = 0.f;
  if (i < T && a.st.rowrec[ridx * RR_COUNT + RR_FLAGS] == 0.f) {
    const int nmax = a.st.nmax[ridx];
    const int nmin = minmax ? a.st.nmin[ridx] : 1;
    tierow = (nmax > 1) | (nmin > 1);
    const float ss = a.st.sself[ridx];
    const float cMt = minmax ? a.st.cM[ridx] : -ss;
    const float cm = minmax ? -(ss + cMt) : 0.f;
    M = a.st.M[ridx];
    m = minmax ? a.st.m[ridx] : M;
    coefM = cMt / (float)nmax;
    coefm = cm / (float)nmin;
  }
  if (!__any(tierow)) return;
  float qop[D / 2];
  {
    const int rr = i < T ? i : T - 1;
    const float *src = a.q + slice + (size_t)rr * D + half * (D / 2);
#pragma unroll
    for (int s = 0; s < D / 2; s += 4) {
      f32x4 x = *reinterpret_cast<const f32x4 *>(src + s);
      qop[s] = x[0]; qop[s + 1] = x[1]; qop[s + 2] = x[2]; qop[s + 3] = x[3];
    }
  }
  const int kend = a.causal ? min(T, rb * 32 + 32) : T;
  for (int js = 0; js < kend; js += 32) {
    float kop[D / 2];
    {
      const int key = js + l32;
      const bool okk = key < T;
      const float *src = a.k + slice + (size_t)(okk ? key : 0) * D + half * (D / 2);
#pragma unroll
      for (int s = 0; s < D / 2; s += 4) {
        f32x4 x = *reinterpret_cast<const f32x4 *>(src + s);
#pragma unroll
        for (int e = 0; e < 4; ++e) kop[s + e] = okk ? x[e] : 0.f;
      }
    }
    const f32x16 acc = score_tile<D>(kop, qop);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int j = js + krel(r, half);
      const bool valid = tierow & (j < T) & (!a.causal | (j <= i));
      const float s = acc[r] * a.scale;
      const bool hitM = valid & (s == M);
      const bool hitm = valid & minmax & (s == m);
      const float coef = hitM ? coefM : (hitm ? coefm : 0.f);
      uint64_t mask = __ballot(hitM | hitm);
      while (mask) {
        const int src = __ffsll((unsigned long long)mask) - 1;
        mask &= mask - 1;
        const float cf = __shfl(coef, src) * a.scale;
        const int isrc = rb * 32 + (src & 31);
        const int jsrc = js + krel(r, src >> 5);
        for (int e = lane; e < D; e += 64) {
          atomicAdd(a.dq + slice + (size_t)isrc * D + e,
                    cf * a.k[slice + (size_t)jsrc * D + e]);
          atomicAdd(a.dk + slice + (size_t)jsrc * D + e,
                    cf * a.q[slice + (size_t)isrc * D + e]);
        }
      }
    }
  }
}

#define KIA_INST(D)                                      \
  template __global__ void bwd_pre_kernel<D>(BwdArgs);   \
  template __global__ void bwd_main_kernel<D>(BwdArgs);  \
  template __global__ void bwd_dq_kernel<D>(BwdArgs);    \
  template __global__ void bwd_ties_kernel<D>(BwdArgs);
KIA_INST(16)
KIA_INST(32)
KIA_INST(64)
KIA_INST(128)

}  // namespace kia
