// kia_bwd.hip -- backward of causal K-interval attention on gfx950.
//
// Four launches on the caller's stream (App. B):
//  1. bwd_pre   per row: D^X = dO . O^X (O^X = O, or O^L for Prob-STE with
//               Nearest), the row record (grid constants, 1/W, 1/W^X,
//               -D^X/W^X), zeroes dQ and the two row sums.
//  2. bwd_main  one workgroup per 128 keys; 4 waves x 32 keys each keep
//               their K and V rows in registers and stream 32-query tiles:
//               S^T and dP^T on MFMA (canonical sub-tile, bit-identical to
//               the forward), per key gamma = (g - D^X)/W^X, Delta, dS =
//               gamma Delta, the row sums S_self = sum dS and (MinMax)
//               sum gamma dw^L/dM (Eq. calgrad), then dV += P^T dO and
//               dK += dS^T Q through a wave-private LDS transpose, and
//               dQ += dS K reduced over the 4 waves in LDS, added to HBM
//               with one float atomic per element and tile.
//  3. bwd_calib (full gradient only) rows whose max (and MinMax min) is
//               unique: Eq. (full) puts cM = sum_j gamma_j dw_j/dM on the
//               argmax key and cm = -(S_self + cM) (from Delta + dw/dM +
//               dw/dm = 0) on the argmin key; FWM has cM = -S_self. Applied
//               as dQ_i += scale (cM k_amax + cm k_amin) and scatter-adds
//               dK_amax += scale cM q_i, dK_amin += scale cm q_i.
//  4. bwd_ties  (full gradient only) rows with tied extrema: recompute the
//               row's scores with the canonical sub-tile and split cM / cm
//               evenly over every key equal to M / m (edge-case table).
#include "kia_device.hpp"
#include "kia_kernels.hpp"

namespace kia {

constexpr int BKV = 128;  // keys per backward workgroup
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
    const f32x4 z = {0.f, 0.f, 0.f, 0.f};
    *reinterpret_cast<f32x4 *>(a.dq + ridx * D + sub * 4) = z;
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
  __shared__ __attribute__((aligned(16))) float Qs[BQ * DS];
  __shared__ __attribute__((aligned(16))) float dOs[BQ * DS];
  __shared__ __attribute__((aligned(16))) float Rec[BQ * RR_COUNT];
  __shared__ __attribute__((aligned(16))) float Kb[BKV * DS];
  __shared__ __attribute__((aligned(16))) float Xt[4 * 32 * XS];
  __shared__ __attribute__((aligned(16))) float dQr[BQ * DP];
  __shared__ float Part[4 * 32 * 2];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, half = lane >> 5, l32 = lane & 31;
  const int T = a.T;
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
  // K block row-major in LDS (B operand of dQ += dS K)
 for (int e = tid; e < BKV * DP / 4; e += 256) {
    const int r = e / (DP / 4), c4 = e % (DP / 4);
    f32x4 x = {0.f, 0.f, 0.f, 0.f};
    if (j0 + r < T && c4 * 4 < D) x = *reinterpret_cast<const f32x4 *>(ks + (size_t)(j0 + r) * D + c4 * 4);
    *reinterpret_cast<f32x4 *>(Kb + r * DS + c4 * 4) = x;
  }

  f32x16 dva[NC], dka[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) { dva[c][e] = 0.f; dka[c][e] = 0.f; }

  const int qstart = a.causal ? j0 : 0;
  float *Xw = Xt + wave * 32 * XS;
  for (int i0 = qstart; i0 < T; i0 += BQ) {
    __syncthreads();
    for (int e = tid; e < BQ * DP / 4; e += 256) {
      const int r = e / (DP / 4), c4 = e % (DP / 4);
      f32x4 x = {0.f, 0.f, 0.f, 0.f}, y = x;
      if (i0 + r < T && c4 * 4 < D) {
        x = *reinterpret_cast<const f32x4 *>(qs + (size_t)(i0 + r) * D + c4 * 4);
        y = *reinterpret_cast<const f32x4 *>(dos + (size_t)(i0 + r) * D + c4 * 4);
      }
      *reinterpret_cast<f32x4 *>(Qs + r * DS + c4 * 4) = x;
      *reinterpret_cast<f32x4 *>(dOs + r * DS + c4 * 4) = y;
    }
    for (int e = tid; e < BQ * RR_COUNT / 4; e += 256) {
      const int r = e / (RR_COUNT / 4), c4 = e % (RR_COUNT / 4);
      f32x4 x = {0.f, 0.f, 0.f, 0.f};
      if (i0 + r < T)
        x = *reinterpret_cast<const f32x4 *>(a.st.rowrec + ((size_t)bh * T + i0 + r) * RR_COUNT + c4 * 4);
      else if (c4 == 0)
        x[1] = (float)a.K;  // padding rows: u = K, never ambiguous
      *reinterpret_cast<f32x4 *>(Rec + r * RR_COUNT + c4 * 4) = x;
    }
    for (int e = tid; e < BQ * DP; e += 256) dQr[e] = 0.f;
    __syncthreads();

    float ps = 0.f, pm = 0.f;
    const bool active = (jw < T) & !(a.causal & (jw > i0 + 31));
    if (active) {
      float qop[D / 2], dop[D / 2];
      {
        const float *qr = Qs + l32 * DS + half * (D / 2);
        const float *dr = dOs + l32 * DS + half * (D / 2);
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

      const float *rr = Rec + l32 * RR_COUNT;
      RowConst rc;
      rc.alpha = rr[RR_ALPHA]; rc.beta = rr[RR_BETA]; rc.margin2 = rr[RR_MARGIN2];
      rc.hl = rr[RR_HL]; rc.b1l = rr[RR_B1L]; rc.emh = rr[RR_EMH];
      rc.dcoef = rr[RR_DCOEF]; rc.degen = rr[RR_FLAGS] != 0.f;
      const float invWf = rr[RR_INVWF], invWX = rr[RR_INVWX], negDXW = rr[RR_NEGDXW];
      const float M = rr[RR_M], m = rr[RR_m];
      Decided dd;
      decide16(S, rc, M, m, a.K, a.calib, a.tau, a.scale, dd);

      const int i = i0 + l32;
      float P[16], dS[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int j = jw + krel(r, half);
        const bool valid = (j < T) & (i < T) & (!a.causal | (j <= i)) &
                           !((dd.tail >> r) & 1u);
        const float Eu = exp2f(fmaf(dd.rf[r], rc.hl, rc.b1l));
        const float El = Eu * rc.emh;
        const float wL = fmaf(dd.t[r], Eu - El, El);
        const float wN = ((dd.up >> r) & 1u) ? Eu : El;
        const float wf = nearest ? wN : wL;
        const float gamma = fmaf(G[r], invWX, negDXW);
        const float Delta = Eu * rc.dcoef;
        const float ds = gamma * Delta;
        P[r] = valid ? wf * invWf : 0.f;
        dS[r] = valid ? ds : 0.f;
        ps += dS[r];
        if (want_cm) {
          // dw^L/dM = X - w^L - Delta u / K, X = (r w^L + t e^{b_{r+1}}) / K
          const float u = dd.rf[r] + dd.t[r];
          const float X = fmaf(dd.rf[r], wL, dd.t[r] * Eu) * invK;
          const float dM = X - wL - Delta * u * invK;
          pm += valid ? gamma * dM : 0.f;
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
          dva[c] = mfma32(at[st], dOs[(16 * half + st) * DS + 32 * c + l32], dva[c]);
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
          dka[c] = mfma32(at[st], Qs[(16 * half + st) * DS + 32 * c + l32], dka[c]);
      // dQ += dS K  (A = dS registers as they are, B = K block rows)
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        f32x16 qa;
#pragma unroll
        for (int e = 0; e < 16; ++e) qa[e] = 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r)
          qa = mfma32(dS[r], Kb[(32 * wave + krel(r, half)) * DS + 32 * c + l32], qa);
#pragma unroll
        for (int e = 0; e < 16; ++e)
          atomicAdd(&dQr[krel(e, half) * DP + 32 * c + l32], qa[e]);
      }
    }
    ps += __shfl_xor(ps, 32);
    pm += __shfl_xor(pm, 32);
    if (half == 0) {
      Part[(wave * 32 + l32) * 2] = ps;
      Part[(wave * 32 + l32) * 2 + 1] = pm;
    }
    __syncthreads();
    for (int e = tid; e < BQ * DP; e += 256) {
      const int r = i0 + e / DP, n = e % DP;
      if (r < T && n < D) atomicAdd(a.dq + slice + (size_t)r * D + n, a.scale * dQr[e]);
    }
    if (!a.detach && tid < 32 && i0 + tid < T) {
      float s = 0.f, mm = 0.f;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        s += Part[(w * 32 + tid) * 2];
        mm += Part[(w * 32 + tid) * 2 + 1];
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
__device__ __forceinline__ void atomic_add4(float *p, f32x4 v) {
  atomicAdd(p, v[0]); atomicAdd(p + 1, v[1]);
  atomicAdd(p + 2, v[2]); atomicAdd(p + 3, v[3]);
}

template <int D>
__global__ __launch_bounds__(256) void bwd_calib_kernel(BwdArgs a) {
  constexpr int L = D / 4;
  const size_t R = (size_t)a.BH * a.T;
  const size_t t = (size_t)blockIdx.x * 256 + threadIdx.x;
  const size_t ridx = t / L;
  const int c4 = (int)(t % L);
  if (ridx >= R) return;
  const bool minmax = a.calib == CAL_MINMAX;
  if (a.st.rowrec[ridx * RR_COUNT + RR_FLAGS] != 0.f) return;  // degenerate
  const int nmax = a.st.nmax[ridx];
  const int nmin = minmax ? a.st.nmin[ridx] : 1;
  if (nmax != 1 || nmin != 1) return;  // tied extrema: bwd_ties
  const float ss = a.st.sself[ridx];
  const float cMt = minmax ? a.st.cM[ridx] : -ss;
  const float cm = minmax ? -(ss + cMt) : 0.f;
  const size_t base = (ridx / a.T) * (size_t)a.T * D;
  const f32x4 qi = *reinterpret_cast<const f32x4 *>(a.q + ridx * D + c4 * 4);
  f32x4 dq4 = *reinterpret_cast<const f32x4 *>(a.dq + ridx * D + c4 * 4);
  const int am = a.st.amax[ridx];
  const f32x4 ka = *reinterpret_cast<const f32x4 *>(a.k + base + (size_t)am * D + c4 * 4);
  const float fM = a.scale * cMt;
  dq4 += fM * ka;
  atomic_add4(a.dk + base + (size_t)am * D + c4 * 4, fM * qi);
  if (minmax) {
    const int an = a.st.amin[ridx];
    const f32x4 kn = *reinterpret_cast<const f32x4 *>(a.k + base + (size_t)an * D + c4 * 4);
    const float fm = a.scale * cm;
    dq4 += fm * kn;
    atomic_add4(a.dk + base + (size_t)an * D + c4 * 4, fm * qi);
  }
  *reinterpret_cast<f32x4 *>(a.dq + ridx * D + c4 * 4) = dq4;
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
      const bool ok = key < T;
      const float *src = a.k + slice + (size_t)(ok ? key : 0) * D + half * (D / 2);
#pragma unroll
      for (int s = 0; s < D / 2; s += 4) {
        f32x4 x = *reinterpret_cast<const f32x4 *>(src + s);
#pragma unroll
        for (int e = 0; e < 4; ++e) kop[s + e] = ok ? x[e] : 0.f;
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
  template __global__ void bwd_calib_kernel<D>(BwdArgs); \
  template __global__ void bwd_ties_kernel<D>(BwdArgs);
KIA_INST(16)
KIA_INST(32)
KIA_INST(64)
KIA_INST(128)

}  // namespace kia
