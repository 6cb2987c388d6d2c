// kia_bwd.hip -- backward of causal K-interval attention on gfx950.
//
// Four launches on the caller's stream (App. B):
//  1. bwd_pre   per row: D^X = dO . O^X (O^X = O, or O^L for Prob-STE with
//               Nearest) and the row record (grid constants, 1/W, 1/W^X,
//               -D^X/W^X); zeroes the two row sums.
//  2. bwd_main  KV-major: one workgroup per 128 keys, waves of 32 keys
//               stream 32-query tiles (staged in LDS, prefetched into
//               registers one tile ahead). The scores are not recomputed:
//               each (query, key) tile's decided positions u come from the
//               forward (stats U), so the index decisions are the forward's
//               own. dP^T on MFMA, per key (weights from u)
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
// The exponential weight functions (softmax, BF16-exp, FP8-exp) run the
// same launches with the FWM calibration's bookkeeping: U holds each key's
// fp32 exponential, dS = dz of the weight function, and the maximum's
// channel cM = -S_self lands on the argmax keys (z = s - M keeps M on the
// gradient path).
#include "kia_device.hpp"
#include "kia_kernels.hpp"

namespace kia {

constexpr int BKV = 128;  // keys per bwd_main workgroup
constexpr int BQ = 32;    // queries per streamed tile
constexpr int XS = 36;    // transpose buffer row stride (floats)

// ---------------------------------------------------------------------------
template <int D, typename TI>
__global__ __launch_bounds__(256) void bwd_pre_kernel(BwdArgsT<TI> a) {
  constexpr int L = D / 4;  // lanes per row, one float4 each
  constexpr int RPB = 256 / L;
  const int tid = threadIdx.x;
  const int sub = tid % L;
  const size_t R = (size_t)a.BH * a.T;
  const size_t ridx = (size_t)blockIdx.x * RPB + tid / L;
  const bool live = ridx < R;
  const bool probN = (a.recon == REC_NEAREST) & (a.ste == STE_PROB);
  float dot = 0.f;
  if (live && a.dq_piece > 0) {  // the dQ pieces add into dQ
    const f32x4 z = {0.f, 0.f, 0.f, 0.f};
    *reinterpret_cast<f32x4 *>(a.dq + ridx * D + sub * 4) = z;
  }
  if (live && a.qsplit > 1) {  // the split main kernel adds into dK, dV
    const f32x4 z = {0.f, 0.f, 0.f, 0.f};
    *reinterpret_cast<f32x4 *>(a.dk + ridx * D + sub * 4) = z;
    *reinterpret_cast<f32x4 *>(a.dv + ridx * D + sub * 4) = z;
  }
  // every load up front, from a clamped row (one memory round trip; the
  // row statistics are the same address for the row's lanes)
  const size_t rr = live ? ridx : 0;
  const float *ox = probN ? a.st.OL + rr * D : a.o + rr * D;
  // the bf16-output variant's O is bf16 (O^L stays fp32 in stats)
  const f32x4 x = (a.o16 && !probN) ? load4(a.o16 + rr * D + sub * 4)
                                    : *reinterpret_cast<const f32x4 *>(ox + sub * 4);
  const f32x4 y = load4(a.dO + rr * D + sub * 4);
  const float M = a.st.M[rr];
  const float m = a.calib != CAL_FWM && a.recon < REC_SOFTMAX ? a.st.m[rr] : M;
  const float W = a.st.W[rr];
  const float WX = probN ? a.st.WL[rr] : W;
  if (live) dot = x[0] * y[0] + x[1] * y[1] + x[2] * y[2] + x[3] * y[3];
#pragma unroll
  for (int off = L / 2; off > 0; off >>= 1) dot += __shfl_xor(dot, off);
  if (live && sub == 0) {
    // the grid constants (the decision constants alpha, beta, margin are not
    // needed: the backward reads the forward's decided positions)
    RowConst rc{};  // unused by the exponential weight functions
    rc.emh = 1.f;
    if (a.recon < REC_SOFTMAX)
      grid_consts(M, m, a.K, a.calib, a.tau, rc.hl, rc.b1l, rc.emh, rc.dcoef, rc.degen);
    const float invWX = 1.f / WX;
    f32x4 *rec = reinterpret_cast<f32x4 *>(a.st.rowrec + ridx * RR_COUNT);
    const f32x4 r0 = {rc.alpha, rc.beta, rc.margin2, rc.hl};
    const f32x4 r1 = {rc.b1l, rc.emh, rc.dcoef, 1.f / W};
    const f32x4 r2 = {invWX, -dot * invWX, M, m};
    f32x4 r3 = {rc.degen ? 1.f : 0.f, 0.f, 0.f, 0.f};
    if (a.recon < REC_SOFTMAX) {
      const float dW = rc.dcoef * W;
      r3[1] = rc.b1l - __log2f(W);
      r3[2] = dW * invWX;
      r3[3] = -dW * dot * invWX;
    }
    rec[0] = r0; rec[1] = r1; rec[2] = r2; rec[3] = r3;
    a.st.sself[ridx] = 0.f;
    a.st.cM[ridx] = 0.f;
  }
}

// ---------------------------------------------------------------------------
template <int D, int CALIB, int RECON>
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
  // key block (ascending: the longest causal key blocks first) and the part
  // of its query range (qsplit parts of nearly equal tile counts)
  const int kb = (int)(blockIdx.x / a.BH) / a.qsplit;
  const int qpart = (int)(blockIdx.x / a.BH) % a.qsplit;
  const int bh = blockIdx.x % a.BH;
  const int j0 = kb * BKV;
  const int jw = j0 + 32 * wave;
  const size_t slice = (size_t)bh * T * D;
  const float *qs = a.q + slice, *vs = a.v + slice,
              *dos = a.dO + slice;
  constexpr bool minmax = CALIB == CAL_MINMAX;
  constexpr bool nearest = RECON == REC_NEAREST;
  constexpr bool EXPW = is_exp_rec(RECON);
  constexpr bool COMPACT = compact_codes<CALIB, RECON>();
  const bool want_cm = minmax & grad_channels(a.grad);
  const float invK = 1.f / (float)a.K, Kf = (float)a.K;

  // this wave's 32 keys of V as A operands (canonical layout)
  float vop[D / 2];
  {
    const int key = jw + l32;
    const bool ok = key < T;
    const float *vr = vs + (size_t)(ok ? key : 0) * D + half * (D / 2);
#pragma unroll
    for (int s = 0; s < D / 2; s += 4) {
      f32x4 y = *reinterpret_cast<const f32x4 *>(vr + s);
#pragma unroll
      for (int e = 0; e < 4; ++e) vop[s + e] = ok ? y[e] : 0.f;
    }
  }

  f32x16 dva[NC], dka[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) { dva[c][e] = 0.f; dka[c][e] = 0.f; }

  // next-tile prefetch registers: Q and dO rows through buffer loads (rows
  // past T and padded columns read as zeros; no branch around a load, so
  // the compiler does not wait for them before the compute); the row
  // records of rows past T are replaced by padding when stashed
  static_assert(QV4 % 256 == 0, "whole passes");
  const uint32_t qoff = row_vec_offset<D>(tid);
  f32x4 pq[PF], pd[PF], pr;
  bool rok;
  auto fetch = [&](int i0) {
#pragma unroll
    for (int e = 0; e < PF; ++e) {
      const int rb = i0 + e * (1024 / DP);  // 256 threads cover 1024 / DP rows
      pq[e] = buffer_f32x4(row_rsrc(qs, rb, T, D), qoff);
      pd[e] = buffer_f32x4(row_rsrc(dos, rb, T, D), qoff);
    }
    {
      const int r = (tid / (RR_COUNT / 4)) % BQ, c4 = tid % (RR_COUNT / 4);
      rok = (tid < BQ * RR_COUNT / 4) & (i0 + r < T);
      const size_t rix = (size_t)bh * T + (rok ? i0 + r : 0);
      pr = *reinterpret_cast<const f32x4 *>(a.st.rowrec + rix * RR_COUNT + c4 * 4);
    }
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int e = 0; e < PF; ++e) {
      const int idx = tid + 256 * e;
      const int r = idx / (DP / 4), c4 = idx % (DP / 4);
      *reinterpret_cast<f32x4 *>(&Qs[buf][r * DS + c4 * 4]) = pq[e];
      *reinterpret_cast<f32x4 *>(&dOs[buf][r * DS + c4 * 4]) = pd[e];
    }
    if (tid < BQ * RR_COUNT / 4) {
      // padding rows: u = K (beta = K), never ambiguous
      const f32x4 pad = {0.f, (tid % (RR_COUNT / 4)) == 0 ? (float)a.K : 0.f, 0.f, 0.f};
      *reinterpret_cast<f32x4 *>(&Rec[buf][tid * 4]) = rok ? pr : pad;
    }
  };

  const int q0 = a.causal ? j0 : 0;
  const int ntall = (T - q0 + BQ - 1) / BQ;
  const int tb = ntall * qpart / a.qsplit, te = ntall * (qpart + 1) / a.qsplit;
  const int qstart = q0 + tb * BQ;
  const int nt = te - tb;
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
      // the forward's decided positions of this (query, key) tile (one byte
      // per key under FWM with Nearest)
      float u[16];
      uint4 cw;
      {
        const float *ut = a.st.U + ds_tile(bh, i0 / 32, jw / 32, nq, a.causal) * 1024;
        if constexpr (COMPACT) cw = codes_load(ut, lane);
        else tile_load(ut, lane, u);
      }
      float dop[D / 2];
      {
        const float *dr = dOb + l32 * DS + half * (D / 2);
#pragma unroll
        for (int s = 0; s < D / 2; s += 4) {
          f32x4 y = *reinterpret_cast<const f32x4 *>(dr + s);
#pragma unroll
          for (int e = 0; e < 4; ++e) dop[s + e] = y[e];
        }
      }
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

      const int i = i0 + l32;
      // key j is valid for this lane's query i iff j <= jlim
      const int jlim = i < T ? (a.causal ? i : T - 1) : -1;
      float P[16], dS[16];
      if constexpr (EXPW) {
        // u holds the forward's fp32 exponential e (bf16-rounded for
        // BF16-exp); dz = gamma e (softmax; FP8-exp: the fp32
        // exponential's derivative through an identity rounding), BF16-exp
        // the backward of its casts, bf16(bf16(gamma) w)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const bool valid = jw + krel(r, half) <= jlim;
          const float e = u[r];
          const float wf = RECON == REC_FP8EXP ? exp_weight_of<RECON>(e) : e;
          const float gamma = fmaf(G[r], invWX, negDXW);
          const float dz = RECON == REC_BF16EXP ? bf16_rne(bf16_rne(gamma) * e) : gamma * e;
          P[r] = valid ? wf * invWf : 0.f;
          dS[r] = valid ? dz : 0.f;
          ps += dS[r];
        }
      } else {
        // e' = e^{b_{r+1}} / W from one exponential (RR_B1LW): P is e' or
        // e' e^{-h} (LERP: the chord between them), dS = (g c1 + c0) e'
        const float b1lw = r3[1], c1 = r3[2], c0 = r3[3];
        const float Wf = 1.f / invWf;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          KeyDec kd;
          if constexpr (COMPACT) kd = key_of_code(cw, r);
          else kd = key_of<CALIB>(u[r], Kf);
          const float Ep = __builtin_amdgcn_exp2f(fmaf(kd.rf, rc.hl, b1lw));
          const float Elp = Ep * rc.emh;
          const float wLp = fmaf(kd.t, Ep - Elp, Elp);
          const float Pr = nearest ? (kd.up ? Ep : Elp) : wLp;
          const bool valid = (jw + krel(r, half) <= jlim) & !kd.tail;
          P[r] = valid ? Pr : 0.f;
          dS[r] = valid ? fmaf(G[r], c1, c0) * Ep : 0.f;
          ps += dS[r];
          if (want_cm) {
            // dw^L/dM = X - w^L - Delta u / K, X = (r w^L + t e^{b_{r+1}}) / K,
            // on the unscaled weights
            const float Eu = Ep * Wf, wL = wLp * Wf;
            const float gamma = fmaf(G[r], invWX, negDXW);
            const float Delta = Eu * rc.dcoef;
            const float uc = kd.rf + kd.t;
            const float X = fmaf(kd.rf, wL, kd.t * Eu) * invK;
            const float dM = X - wL - Delta * uc * invK;
            pm += valid ? gamma * dM : 0.f;
          }
        }
      }
      // dS tile to the scratch, lane-major (the dQ kernel's A operand)
      {
        tile_store(a.st.dS + ds_tile(bh, i0 / 32, jw / 32, nq, a.causal) * 1024, lane, dS);
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
    if (a.grad != GRAD_DETACH && tid < 32 && i0 + tid < T) {
      float s = 0.f, mm = 0.f;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        s += Part[buf][(w * 32 + tid) * 2];
        mm += Part[buf][(w * 32 + tid) * 2 + 1];
      }
      const size_t ridx = (size_t)bh * T + i0 + tid;
      put_row_sums(a, kb, ridx, s, mm, minmax);
    }
  }
  // write dV, dK (lane -> column, register -> key)
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int j = jw + krel(r, half);
      if (j < T && 32 * c + l32 < D) {
        if (a.qsplit > 1) {
          atomicAdd(a.dv + slice + (size_t)j * D + 32 * c + l32, dva[c][r]);
          atomicAdd(a.dk + slice + (size_t)j * D + 32 * c + l32, a.scale * dka[c][r]);
        } else {
          a.dv[slice + (size_t)j * D + 32 * c + l32] = dva[c][r];
          a.dk[slice + (size_t)j * D + 32 * c + l32] = a.scale * dka[c][r];
        }
      }
    }
}

// ---------------------------------------------------------------------------
// bwd_main for d <= 64 at two waves per SIMD: 8 waves per workgroup in two
// groups of 4. The workgroup's 128 keys have V in LDS (read as the MFMA A
// operand), so a wave keeps only its dV/dK accumulators in registers.
// Group g takes the query tiles t = g, g+2, ...; each group has its own
// tile buffers, two of them (iteration parity), and prefetches its next tile
// into registers, so one workgroup barrier per iteration orders the stash
// before the reads and the reads of two iterations back before the stash.
// The row sums of a tile's dS are added up (and sent out) one iteration
// later, behind that same barrier. The two groups' partial dV/dK are summed
// through LDS at the end.
template <int D, int CALIB, int RECON>
__global__ __launch_bounds__(512, 2) void bwd_main_shared_kernel(BwdArgs a) {
  constexpr int NC = Dims<D>::NC, DS = Dims<D>::DS, DP = Dims<D>::DP;
  constexpr int QV4 = BQ * DP / 4;         // float4 per Q (or dO) tile
  constexpr int PF = (QV4 + 255) / 256;    // float4 per group thread and tensor
  // One LDS block: V of the workgroup's keys, the Q / dO tiles and row
  // records [group][parity], the wave-private transpose tiles and the row-sum
  // partials [group][parity]. After the loop its start holds the second
  // group's dV/dK for the final reduction (clear of the partials).
  constexpr int KVF = BKV * DS, QT = BQ * DS, RT = BQ * RR_COUNT, PT = 4 * 32 * 2;
  constexpr int OFF_Q = KVF, OFF_DO = OFF_Q + 4 * QT, OFF_REC = OFF_DO + 4 * QT;
  constexpr int OFF_X = OFF_REC + 4 * RT, OFF_PART = OFF_X + 8 * 32 * XS;
  constexpr int LDS_FLOATS = OFF_PART + 4 * PT;
  static_assert(OFF_PART >= 4 * NC * 16 * 64 * 2, "reduction buffer");
  __shared__ __attribute__((aligned(16))) float L[LDS_FLOATS];
  float *Vb = L, *Xt = L + OFF_X;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, half = lane >> 5, l32 = lane & 31;
  // key tile wk of the wave: group 1 takes the tiles in reverse order, so
  // that the two waves sharing a SIMD (waves w and w + 4) own key tiles wk
  // and 3 - wk, and the tiles idle on the causal diagonal (the high ones of a
  // key block's first query tiles) never leave both waves of a SIMD idle
  const int grp = wave >> 2, wk = grp ? 3 - (wave & 3) : (wave & 3), gtid = tid & 255;
  const int T = a.T;
  const int nq = (T + 31) / 32;
  // key block (ascending: the longest causal key blocks first) and the part
  // of its query range (qsplit parts of nearly equal tile counts)
  const int kb = (int)(blockIdx.x / a.BH) / a.qsplit;
  const int qpart = (int)(blockIdx.x / a.BH) % a.qsplit;
  const int bh = blockIdx.x % a.BH;
  const int j0 = kb * BKV;
  const int jw = j0 + 32 * wk;
  const size_t slice = (size_t)bh * T * D;
  const float *qs = a.q + slice, *vs = a.v + slice,
              *dos = a.dO + slice;
  constexpr bool minmax = CALIB == CAL_MINMAX;
  constexpr bool nearest = RECON == REC_NEAREST;
  constexpr bool EXPW = is_exp_rec(RECON);
  constexpr bool COMPACT = compact_codes<CALIB, RECON>();
  const bool want_cm = minmax & grad_channels(a.grad);
  const float invK = 1.f / (float)a.K, Kf = (float)a.K;

  // V of the workgroup's keys: buffer loads issued first (keys past T and
  // padded columns read as zeros), stashed after the first tile's fetch is
  // in flight
  constexpr int VL = BKV * DP / 4 / 512;  // 16-byte vectors per thread
  static_assert(BKV * DP / 4 % 512 == 0, "whole passes");
  f32x4 vpre[VL];
  {
    const uint32_t voff = row_vec_offset<D>(tid);
#pragma unroll
    for (int e = 0; e < VL; ++e)
      vpre[e] = buffer_f32x4(row_rsrc(vs, j0 + e * (2048 / DP), T, D), voff);
  }
  auto stash_v = [&]() {
#pragma unroll
    for (int e = 0; e < VL; ++e) {
      const int idx = tid + 512 * e;
      const int r = idx / (DP / 4), c4 = idx % (DP / 4);
      *reinterpret_cast<f32x4 *>(Vb + r * DS + c4 * 4) = vpre[e];
    }
  };

  f32x16 dva[NC], dka[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) { dva[c][e] = 0.f; dka[c][e] = 0.f; }

  // Q and dO rows through buffer loads (rows past T and padded columns read
  // as zeros); row records past T replaced by padding when stashed
  static_assert(QV4 % 256 == 0, "whole passes");
  const uint32_t qoff = row_vec_offset<D>(gtid);
  f32x4 pq[PF], pd[PF], pr;
  bool rok;
  auto fetch = [&](int i0) {
#pragma unroll
    for (int e = 0; e < PF; ++e) {
      const int rb = i0 + e * (1024 / DP);  // 256 threads cover 1024 / DP rows
      pq[e] = buffer_f32x4(row_rsrc(qs, rb, T, D), qoff);
      pd[e] = buffer_f32x4(row_rsrc(dos, rb, T, D), qoff);
    }
    {
      const int r = (gtid / (RR_COUNT / 4)) % BQ, c4 = gtid % (RR_COUNT / 4);
      rok = (gtid < BQ * RR_COUNT / 4) & (i0 + r < T);
      const size_t rix = (size_t)bh * T + (rok ? i0 + r : 0);
      pr = *reinterpret_cast<const f32x4 *>(a.st.rowrec + rix * RR_COUNT + c4 * 4);
    }
  };
  auto stash = [&](int buf) {
    float *Qd = L + OFF_Q + (2 * grp + buf) * QT, *dOd = L + OFF_DO + (2 * grp + buf) * QT;
#pragma unroll
    for (int e = 0; e < PF; ++e) {
      const int idx = gtid + 256 * e;
      const int r = idx / (DP / 4), c4 = idx % (DP / 4);
      *reinterpret_cast<f32x4 *>(Qd + r * DS + c4 * 4) = pq[e];
      *reinterpret_cast<f32x4 *>(dOd + r * DS + c4 * 4) = pd[e];
    }
    if (gtid < BQ * RR_COUNT / 4) {
      // padding rows: u = K (beta = K), never ambiguous
      const f32x4 pad = {0.f, (gtid % (RR_COUNT / 4)) == 0 ? (float)a.K : 0.f, 0.f, 0.f};
      *reinterpret_cast<f32x4 *>(L + OFF_REC + (2 * grp + buf) * RT + gtid * 4) = rok ? pr : pad;
    }
  };

  const int q0 = a.causal ? j0 : 0;
  const int ntall = (T - q0 + BQ - 1) / BQ;
  const int tb = ntall * qpart / a.qsplit, te = ntall * (qpart + 1) / a.qsplit;
  const int qstart = q0 + tb * BQ;
  const int nt = te - tb;
  const int npair = (nt + 1) / 2;
  float *Xw = Xt + wave * 32 * XS;
  // row sums of iteration itp's tile: the four waves' partials, then one
  // atomic per row
  auto flush = [&](int itp) {
    const int tp = 2 * itp + grp, ip = qstart + tp * BQ;
    if (a.grad != GRAD_DETACH && wk == 0 && lane < 32 && tp < nt && ip + lane < T) {
      const float *pp = L + OFF_PART + (2 * grp + (itp & 1)) * PT;
      float sv = 0.f, mm = 0.f;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        sv += pp[(w * 32 + lane) * 2];
        mm += pp[(w * 32 + lane) * 2 + 1];
      }
      const size_t ridx = (size_t)bh * T + ip + lane;
      put_row_sums(a, kb, ridx, sv, mm, minmax);
    }
  };
  // the forward's decided positions of the wave's (query, key) tile, loaded
  // at the end of the group's previous tile (behind its barrier wait and
  // stash); the tile index is clamped into the stored tiles, so the load
  // needs no branch (its data is unused for an inactive tile)
  auto u_tile = [&](int tt) -> const float * {
    const int qt = min((qstart + tt * BQ) / 32, nq - 1);
    const int kt = min(jw / 32, a.causal ? qt : nq - 1);
    return a.st.U + ds_tile(bh, qt, kt, nq, a.causal) * 1024;
  };
  float u[16];
  uint4 cw;
  auto load_u = [&](int tt) {
    if constexpr (COMPACT) cw = codes_load(u_tile(tt), lane);
    else tile_load(u_tile(tt), lane, u);
  };
  if (grp < nt) fetch(qstart + grp * BQ);
  load_u(grp);  // behind the fetch, which the stash waits for
  stash_v();
  for (int it = 0; it < npair; ++it) {
    const int t = 2 * it + grp, buf = it & 1;
    const int i0 = qstart + t * BQ;
    if (t < nt) stash(buf);
    lds_barrier();
    if (it > 0) flush(it - 1);
    if (t + 2 < nt) fetch(i0 + 2 * BQ);

    float ps = 0.f, pm = 0.f;
    const bool active = (t < nt) & (jw < T) & !(a.causal & (jw > i0 + 31));
    if (active) {
      const float *Qb = L + OFF_Q + (2 * grp + buf) * QT;
      const float *dOb = L + OFF_DO + (2 * grp + buf) * QT;
      const float *vr = Vb + (32 * wk + l32) * DS + half * (D / 2);
      const float *dr = dOb + l32 * DS + half * (D / 2);
      f32x16 G;
#pragma unroll
      for (int e = 0; e < 16; ++e) G[e] = 0.f;
#pragma unroll
      for (int s = 0; s < D / 2; s += 4) {
        const f32x4 x = *reinterpret_cast<const f32x4 *>(vr + s);
        const f32x4 y = *reinterpret_cast<const f32x4 *>(dr + s);
#pragma unroll
        for (int e = 0; e < 4; ++e) G = mfma32(x[e], y[e], G);
      }

      const float *rr = L + OFF_REC + (2 * grp + buf) * RT + l32 * RR_COUNT;
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
      // key j is valid for this lane's query i iff j <= jlim
      const int jlim = i < T ? (a.causal ? i : T - 1) : -1;
      float P[16], dS[16];
      if constexpr (EXPW) {
        // u holds the forward's fp32 exponential e (bf16-rounded for
        // BF16-exp); dz = gamma e (softmax; FP8-exp: the fp32
        // exponential's derivative through an identity rounding), BF16-exp
        // the backward of its casts, bf16(bf16(gamma) w)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const bool valid = jw + krel(r, half) <= jlim;
          const float e = u[r];
          const float wf = RECON == REC_FP8EXP ? exp_weight_of<RECON>(e) : e;
          const float gamma = fmaf(G[r], invWX, negDXW);
          const float dz = RECON == REC_BF16EXP ? bf16_rne(bf16_rne(gamma) * e) : gamma * e;
          P[r] = valid ? wf * invWf : 0.f;
          dS[r] = valid ? dz : 0.f;
          ps += dS[r];
        }
      } else {
        // e' = e^{b_{r+1}} / W from one exponential (RR_B1LW): P is e' or
        // e' e^{-h} (LERP: the chord between them), dS = (g c1 + c0) e'
        const float b1lw = r3[1], c1 = r3[2], c0 = r3[3];
        const float Wf = 1.f / invWf;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          KeyDec kd;
          if constexpr (COMPACT) kd = key_of_code(cw, r);
          else kd = key_of<CALIB>(u[r], Kf);
          const float Ep = __builtin_amdgcn_exp2f(fmaf(kd.rf, rc.hl, b1lw));
          const float Elp = Ep * rc.emh;
          const float wLp = fmaf(kd.t, Ep - Elp, Elp);
          const float Pr = nearest ? (kd.up ? Ep : Elp) : wLp;
          const bool valid = (jw + krel(r, half) <= jlim) & !kd.tail;
          P[r] = valid ? Pr : 0.f;
          dS[r] = valid ? fmaf(G[r], c1, c0) * Ep : 0.f;
          ps += dS[r];
          if (want_cm) {
            // dw^L/dM = X - w^L - Delta u / K, X = (r w^L + t e^{b_{r+1}}) / K,
            // on the unscaled weights
            const float Eu = Ep * Wf, wL = wLp * Wf;
            const float gamma = fmaf(G[r], invWX, negDXW);
            const float Delta = Eu * rc.dcoef;
            const float uc = kd.rf + kd.t;
            const float X = fmaf(kd.rf, wL, kd.t * Eu) * invK;
            const float dM = X - wL - Delta * uc * invK;
            pm += valid ? gamma * dM : 0.f;
          }
        }
      }
      {
        tile_store(a.st.dS + ds_tile(bh, i0 / 32, jw / 32, nq, a.causal) * 1024, lane, dS);
      }
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
    load_u(t + 2);  // the group's next tile
    ps += __shfl_xor(ps, 32);
    pm += __shfl_xor(pm, 32);
    if (half == 0) {
      float *pp = L + OFF_PART + (2 * grp + buf) * PT;
      pp[(wk * 32 + l32) * 2] = ps;
      pp[(wk * 32 + l32) * 2 + 1] = pm;
    }
  }
  // sum the two groups' dV/dK (group 1 -> LDS -> group 0) and store; the
  // buffer overlaps V and the tiles, so wait for every wave (a workgroup
  // with an empty query part runs no loop iteration and its V stash may
  // still be landing); the last tile's row sums go out behind that barrier
  float *red = L + (size_t)wk * (NC * 16 * 64 * 2);
  lds_barrier();
  if (npair > 0) flush(npair - 1);
  if (grp == 1) {
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        red[((c * 16 + r) * 2) * 64 + lane] = dva[c][r];
        red[((c * 16 + r) * 2 + 1) * 64 + lane] = dka[c][r];
      }
  }
  lds_barrier();
  if (grp == 0) {
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int j = jw + krel(r, half);
        const float dvv = dva[c][r] + red[((c * 16 + r) * 2) * 64 + lane];
        const float dkv = dka[c][r] + red[((c * 16 + r) * 2 + 1) * 64 + lane];
        if (j < T && 32 * c + l32 < D) {
          if (a.qsplit > 1) {
            atomicAdd(a.dv + slice + (size_t)j * D + 32 * c + l32, dvv);
            atomicAdd(a.dk + slice + (size_t)j * D + 32 * c + l32, a.scale * dkv);
          } else {
            a.dv[slice + (size_t)j * D + 32 * c + l32] = dvv;
            a.dk[slice + (size_t)j * D + 32 * c + l32] = a.scale * dkv;
          }
        }
      }
  }
}

// ---------------------------------------------------------------------------
// dQ = scale * (dS K + calibration terms). One workgroup = 2 QG waves = QG
// consecutive 32-query tiles of one (b,h) times two key halves (QG = 2 for
// d <= 64, 4 for d = 128): keys stream in chunks of 64 (one 32-key tile per
// half), staged transposed in LDS (K^T, row stride DQ_KTS) so that the four
// consecutive keys a lane needs for four MFMA steps are one 16-byte read.
// Each wave streams its own dS tiles in two fixed register sets (loop
// unrolled by two), one step ahead; a K chunk is fetched into the single K
// register set right after the previous chunk's stash. The key halves'
// partial sums are added through LDS before the calibration epilogue.
constexpr int DQ_KTS = 68;

template <int D, int QG>
__global__ __launch_bounds__(128 * QG) void bwd_dq_kernel(BwdArgs a) {
  constexpr int NC = Dims<D>::NC, DP = Dims<D>::DP;
  constexpr int NT = 128 * QG;      // threads: QG query tiles x 2 key halves
  constexpr int CV4 = 64 * DP / 4;  // float4 of one 64-key chunk
  constexpr int KF = CV4 / NT;      // per thread
  static_assert(KF * NT == CV4, "chunk split");
  static_assert(QG * NC * 16 * 64 <= 2 * DP * DQ_KTS, "reduction buffer");
  __shared__ __attribute__((aligned(16))) float KtT[2][DP * DQ_KTS];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, half = lane >> 5, l32 = lane & 31;
  // query tile pq of the QG and key half kh; key half 1 takes the query
  // tiles in reverse order, so that (QG = 4) the two waves of a SIMD (w and
  // w + 4) own query tiles pq and 3 - pq and their causal key ranges add up
  // alike
  const int kh = wave / QG, pq = kh ? QG - 1 - (wave % QG) : (wave % QG);
  const int T = a.T;
  const int nq = (T + 31) / 32;
  const int npq = (nq + QG - 1) / QG;
  const int bh = blockIdx.x % a.BH;
  // work item -> query group g (heaviest first) and its key piece sp
  int item = (int)(blockIdx.x / a.BH), g = npq - 1;
  while (item >= dq_pieces(g, T, a.causal, a.dq_piece, QG))
    item -= dq_pieces(g--, T, a.causal, a.dq_piece, QG);
  const int sp = item;
  const int nch = dq_chunks(g, T, a.causal, QG);
  const int c0 = a.dq_piece > 0 ? sp * a.dq_piece : 0;
  const int c1 = a.dq_piece > 0 ? min(nch, c0 + a.dq_piece) : nch;
  const int qt = QG * g + pq;
  const bool live = qt < nq;
  const int qtc = live ? qt : nq - 1;
  const size_t slice = (size_t)bh * T * D;
  const float *ks = a.k + slice + (size_t)c0 * 64 * D;  // the piece's first key
  const int nstep = c1 - c0;  // chunks of the piece
  const int ktmine = a.causal ? qtc : nq - 1;  // this wave's last key tile
  // this wave's tile of the piece's chunk p is kt = 2 (c0 + p) + kh; it is
  // used iff p < npw
  const int npw = !live || ktmine < kh ? 0 : max(0, min(c1, (ktmine - kh) / 2 + 1) - c0);
  const int Tp = T - c0 * 64;  // keys from the piece's first key on
  const bool minmax = a.calib == CAL_MINMAX;

  f32x16 acc[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[c][e] = 0.f;

  // K chunks through buffer loads: keys at or past Tp and padded columns
  // read as zeros
  // (one register set for K: a chunk is fetched right after the previous
  // one is stashed, one MFMA step before its own stash)
  f32x4 kX[KF], dA[4], dB[4];
  const uint32_t koff = row_vec_offset<D>(tid);
  auto fetch_k = [&](int p) {
#pragma unroll
    for (int e = 0; e < KF; ++e)
      kX[e] = buffer_f32x4(row_rsrc(ks, p * 64 + e * (4 * NT / DP), Tp, D), koff);
  };
  auto fetch_d = [&](int p, f32x4 (&dx)[4]) {
    const int kt = min(2 * (c0 + p) + kh, ktmine);  // past this wave's row: unused
    const float *src = a.st.dS + ds_tile(bh, qtc, kt, nq, a.causal) * 1024 + 4 * lane;
#pragma unroll
    for (int e = 0; e < 4; ++e) dx[e] = *reinterpret_cast<const f32x4 *>(src + 256 * e);
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int e = 0; e < KF; ++e) {
      const int idx = tid + NT * e;
      const int r = idx / (DP / 4), c4 = idx % (DP / 4);
      // row d = 4 c4 + i holds key r at column r ^ sw(d): the 4-key groups
      // of a row are permuted by sw(d) = 4 ((d >> 3) & 7), so that the
      // lanes of a stash (16 rows d, 4 keys) fall in distinct banks
      float *dst = &KtT[buf][(4 * c4) * DQ_KTS + (r ^ (((c4 >> 1) & 7) << 2))];
#pragma unroll
      for (int i = 0; i < 4; ++i) dst[i * DQ_KTS] = kX[e][i];
    }
  };
  auto mma = [&](int buf, const f32x4 (&dx)[4]) {
    const float *kb = KtT[buf] + l32 * DQ_KTS;
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        // keys kh*32 + krel(4 g4 + i, half), i = 0..3: consecutive, the 4-key
        // group 8 kh + 2 g4 + half of row d = 32 c + l32, permuted as stashed
        const int grp4 = (8 * kh + 2 * g4 + half) ^ (((32 * c + l32) >> 3) & 7);
        const f32x4 bk = *reinterpret_cast<const f32x4 *>(kb + c * 32 * DQ_KTS + 4 * grp4);
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[c] = mfma32(dx[g4][i], bk[i], acc[c]);
      }
  };
  // prologue: chunk 0 in LDS buffer 0 with dA; chunk 1's dS tile in dB and
  // its K behind the first stash. Fetches and stashes run on every step
  // (chunk index clamped; surplus chunks are never used) so that the number
  // of loads in flight is the same on every path and the compiler's waits
  // stay one step behind.
  fetch_k(0);
  fetch_d(0, dA);
  fetch_d(min(1, nstep - 1), dB);
  // the calibration epilogue's row statistics (lanes 0..31: one row each)
  // and the q rows of its dK scatter, loaded behind the first two chunks'
  // fetches (so the first stash does not wait for them) and landing during
  // the key loop (every stats field exists for every calibration)
  constexpr int NE = (D + 63) / 64;
  const int row = qt * 32 + l32;
  const size_t ridx = (size_t)bh * T + (row < T ? row : T - 1);
  const float rflag = a.st.rowrec[ridx * RR_COUNT + RR_FLAGS];
  const int rnmax = a.st.nmax[ridx], rnmin = a.st.nmin[ridx];
  const float rss = a.st.sself[ridx], rcM = a.st.cM[ridx];
  const int ramax = a.st.amax[ridx], ramin = a.st.amin[ridx];
  float qv[16][NE];  // rows qt*32 + 16 kh + u of q, column lane + 64 x
  auto load_qv = [&]() {
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int qrow = qt * 32 + 16 * kh + u;
      const int qr = qrow < T ? qrow : T - 1;
#pragma unroll
      for (int x = 0; x < NE; ++x) {
        const int n = lane + 64 * x;
        qv[u][x] = a.q[slice + (size_t)qr * D + (n < D ? n : 0)];
      }
    }
  };
  // (d = 128: the 32 more registers would cost the key loop; loaded at the end)
  if constexpr (NE == 1) load_qv();
  stash(0);
  fetch_k(min(1, nstep - 1));
  lds_barrier();
  for (int p = 0; p < nstep; p += 2) {
    if (p < npw) mma(0, dA);
    stash(1);
    fetch_k(min(p + 2, nstep - 1));
    fetch_d(min(p + 2, nstep - 1), dA);
    lds_barrier();
    if (p + 1 >= nstep) break;
    if (p + 1 < npw) mma(1, dB);
    stash(0);
    fetch_k(min(p + 3, nstep - 1));
    fetch_d(min(p + 3, nstep - 1), dB);
    lds_barrier();
  }
  // key half 1 hands its partial sums to key half 0 (the chunk buffers are
  // free: the last step ended with a barrier)
  {
    float *red = &KtT[0][0] + pq * (NC * 16 * 64) + lane;
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
  bool ok = false;
  float cMt = 0.f, cm = 0.f;
  int am = 0, an = 0;
  if (sp == 0 && grad_channels(a.grad) && row < T && rflag == 0.f) {
    const int nmin = minmax ? rnmin : 1;
    ok = (rnmax == 1) & (nmin == 1);
    cMt = minmax ? rcM : -rss;
    cm = minmax ? -(rss + cMt) : 0.f;
    if (!grad_keep_max(a.grad)) cMt = 0.f;
    if (!grad_keep_min(a.grad)) cm = 0.f;
    am = ramax;
    an = minmax ? ramin : am;
  }
  if (!ok) { cMt = 0.f; cm = 0.f; am = 0; an = 0; }
  // dQ rows (key half 0): register e holds query krel(e, half), lane column
  // 32c + l32. The k rows of the calibration terms are gathered for EB rows
  // at a time before their dQ stores (stores to dq could alias k, so a load
  // after a store waits for it: one memory round trip per batch, not per
  // row); the argmin term exists for MinMax only (cm = 0 otherwise)
  constexpr int EB = D <= 32 ? 16 : (D == 64 ? 8 : 4);
  if (kh == 0) {
#pragma unroll
  for (int e0 = 0; e0 < 16; e0 += EB) {
    float kM[EB][NC], km[EB][NC];
#pragma unroll
    for (int b = 0; b < EB; ++b) {
      const int src = krel(e0 + b, half);
      const int iam = __shfl(am, src), ian = __shfl(an, src);
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const int n = 32 * c + l32;
        const int nn = n < D ? n : 0;
        kM[b][c] = a.k[slice + (size_t)iam * D + nn];
        km[b][c] = minmax ? a.k[slice + (size_t)ian * D + nn] : 0.f;
      }
    }
#pragma unroll
    for (int b = 0; b < EB; ++b) {
      const int e = e0 + b;
      const int src = krel(e, half);
      const float fM = __shfl(cMt, src), fm = __shfl(cm, src);
      const int qrow = qt * 32 + src;
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const int n = 32 * c + l32;
        float v = acc[c][e];
        v = fmaf(fM, kM[b][c], v);
        v = fmaf(fm, km[b][c], v);
        if (qrow < T && n < D) {
          if (a.dq_piece > 0) atomicAdd(a.dq + slice + (size_t)qrow * D + n, a.scale * v);
          else a.dq[slice + (size_t)qrow * D + n] = a.scale * v;
        }
      }
    }
  }
  }
  // scatter of the calibration terms onto the argmax/argmin keys of dK
  // (each key half takes 16 rows, their q preloaded; piece 0 only)
  // the deterministic backward gathers these per key instead: one record
  // per row for it
  if (a.det && grad_channels(a.grad) && kh == 0 && half == 0 && row < T)
    put_calib_record(a.st.part, ridx, ok, minmax, am, an, cMt * a.scale, cm * a.scale);
  if constexpr (NE > 1) load_qv();
  if (sp == 0 && grad_channels(a.grad) && !a.det) {
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int rr = 16 * kh + u;
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

// ---------------------------------------------------------------------------
// Rows with tied extrema of one 32-row block rb of slice bh, by one wave.
template <int D, typename TI>
__device__ __forceinline__ void tie_rows(const BwdArgsT<TI> &a, int bh, int rb, int lane) {
  const int half = lane >> 5, l32 = lane & 31;
  const int T = a.T;
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
    coefM = grad_keep_max(a.grad) ? cMt / (float)nmax : 0.f;
    coefm = grad_keep_min(a.grad) ? cm / (float)nmin : 0.f;
  }
  if (!__any(tierow)) return;
  // the row's scores with the canonical sub-tile of the input type
  auto tile_scores = [&](int js) -> f32x16 {
    if constexpr (sizeof(TI) == 2) {
      bf16x8 qop[D / 16], kop[D / 16];
      load_rows16<D>(a.q + slice, i < T ? i : T - 1, T, half, qop);
      load_rows16<D>(a.k + slice, js + l32, T, half, kop);
      return score_tile16<D>(kop, qop);
    } else {
      float qop[D / 2], kop[D / 2];
      const int rr = i < T ? i : T - 1;
      const int key = js + l32;
      const bool okk = key < T;
      const float *qs = a.q + slice + (size_t)rr * D + half * (D / 2);
      const float *ksrc = a.k + slice + (size_t)(okk ? key : 0) * D + half * (D / 2);
#pragma unroll
      for (int s = 0; s < D / 2; s += 4) {
        const f32x4 x = *reinterpret_cast<const f32x4 *>(qs + s);
        const f32x4 y = *reinterpret_cast<const f32x4 *>(ksrc + s);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          qop[s + e] = x[e];
          kop[s + e] = okk ? y[e] : 0.f;
        }
      }
      return score_tile<D>(kop, qop);
    }
  };
  const int kend = a.causal ? min(T, rb * 32 + 32) : T;
  for (int js = 0; js < kend; js += 32) {
    const f32x16 acc = tile_scores(js);
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
          const float dqv = cf * load1(a.k + slice + (size_t)jsrc * D + e);
          const float dkv = cf * load1(a.q + slice + (size_t)isrc * D + e);
          if (a.det) {
            // one wave per slice: element e is always this lane's, in order
            a.dq[slice + (size_t)isrc * D + e] += dqv;
            a.dk[slice + (size_t)jsrc * D + e] += dkv;
          } else {
            atomicAdd(a.dq + slice + (size_t)isrc * D + e, dqv);
            atomicAdd(a.dk + slice + (size_t)jsrc * D + e, dkv);
          }
        }
      }
    }
  }
}

// Ties: one wave per 32-row block, or in the deterministic backward one wave
// per (b, h) slice taking its row blocks in order (so that each dK row of the
// slice receives its tie terms from one wave, in a fixed order).
template <int D, typename TI>
__global__ __launch_bounds__(256) void bwd_ties_kernel(BwdArgsT<TI> a) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nrb = (a.T + 31) / 32;
  const size_t gw = (size_t)blockIdx.x * 4 + wave;
  if (a.det) {
    if (gw >= (size_t)a.BH) return;
    // which row blocks hold a tied row: 256 rows per round of loads
    const int T = a.T, bh = (int)gw;
    const bool minmax = a.calib == CAL_MINMAX;
    for (int r0 = 0; r0 < T; r0 += 256) {
      bool tie[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int i = r0 + 64 * c + lane;
        const size_t ridx = (size_t)bh * T + (i < T ? i : T - 1);
        const int nmin = minmax ? a.st.nmin[ridx] : 1;
        tie[c] = (i < T) & ((a.st.nmax[ridx] > 1) | (nmin > 1)) &
                 (a.st.rowrec[ridx * RR_COUNT + RR_FLAGS] == 0.f);
      }
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const uint64_t m = __ballot(tie[c]);
        const int rb = (r0 + 64 * c) / 32;
        if (m & 0xffffffffull) tie_rows<D, TI>(a, bh, rb, lane);
        if (m >> 32) tie_rows<D, TI>(a, bh, rb + 1, lane);
      }
    }
  } else {
    if (gw >= (size_t)a.BH * nrb) return;
    tie_rows<D, TI>(a, (int)(gw / nrb), (int)(gw % nrb), lane);
  }
}

// Deterministic backward: S_self (and cM under MinMax) of every row as the
// sum of its key blocks' partials, in key-block order (causal: the blocks
// at or below the row's own).
template <typename TI>
__global__ __launch_bounds__(256) void row_sums_kernel(BwdArgsT<TI> a) {
  const size_t R = (size_t)a.BH * a.T;
  const size_t ridx = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (ridx >= R) return;
  const int i = (int)(ridx % (size_t)a.T);
  const int nkb = (a.T + 127) / 128;
  const int kend = a.causal ? i / 128 + 1 : nkb;
  const bool minmax = a.calib == CAL_MINMAX;
  float s = 0.f, mm = 0.f;
  for (int kb = 0; kb < kend; ++kb) {
    s += a.st.part[(size_t)kb * R + ridx];
    if (minmax) mm += a.st.part[(size_t)(nkb + kb) * R + ridx];
  }
  a.st.sself[ridx] = s;
  if (minmax) a.st.cM[ridx] = mm;
}

// Deterministic backward: the calibration terms of the rows with unique
// extrema (the ones bwd_dq scatters otherwise), gathered onto dK. bwd_dq
// leaves one record per row in st.part (put_calib_record); one wave per 32
// keys of a slice scans the records in row order (causal: from its first
// key on), collects scale cM_i q_i on key amax_i and scale cm_i q_i on key
// amin_i in LDS, then adds each key's sum to its dK row.
template <int D, typename TI, int NW>
__global__ __launch_bounds__(64 * NW) void calib_gather_kernel(BwdArgsT<TI> a) {
  constexpr int NE = (D + 63) / 64;
  constexpr int GB = 16;  // hit rows whose q rows are loaded together
  // NW waves: wave w takes the 256-row rounds w, w + NW, ... and the keys
  // 32 w / NW onwards of the final sum
  __shared__ float acc[NW][32 * D];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int T = a.T, nkt = (T + 31) / 32;
  const int bh = blockIdx.x / nkt, j0 = (blockIdx.x % nkt) * 32;
  const size_t slice = (size_t)bh * T * D;
  const f32x4 *rec = reinterpret_cast<const f32x4 *>(a.st.part) + (size_t)bh * T;
  float *accw = acc[w];
  for (int e = lane; e < 32 * D; e += 64) accw[e] = 0.f;
  __syncthreads();
  const int ibeg = a.causal ? j0 : 0;
  for (int r0 = ibeg + 256 * w; r0 < T; r0 += 256 * NW) {
    // the records of 256 rows in one round of loads
    f32x4 rc[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int i = r0 + 64 * c + lane;
      rc[c] = rec[i < T ? i : T - 1];
      if (i >= T) rc[c] = f32x4{-1.f, 0.f, -1.f, 0.f};
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int kMl = (int)rc[c][0] - j0, kml = (int)rc[c][2] - j0;
      const bool hM = rc[c][0] >= 0.f && kMl >= 0 && kMl < 32;
      const bool hm = rc[c][2] >= 0.f && kml >= 0 && kml < 32;
      uint64_t mask = __ballot(hM | hm);
      const int i0 = r0 + 64 * c;
      // the hit rows in order, GB at a time: their q rows are loaded
      // together, then added one after the other
      while (mask) {
        int src[GB];
#pragma unroll
        for (int b = 0; b < GB; ++b) {
          src[b] = mask ? __ffsll((unsigned long long)mask) - 1 : -1;
          mask &= mask ? mask - 1 : 0;
        }
        // (unconditional loads from clamped addresses, so that they are all
        // in flight together; unused slots are zeroed after)
        float qv[GB][NE];
#pragma unroll
        for (int b = 0; b < GB; ++b) {
          const TI *qr = a.q + slice + (size_t)(i0 + (src[b] >= 0 ? src[b] : 0)) * D;
#pragma unroll
          for (int x = 0; x < NE; ++x) {
            const int n = lane + 64 * x;
            const float t = load1(qr + (n < D ? n : 0));
            qv[b][x] = (src[b] >= 0 && n < D) ? t : 0.f;
          }
        }
        // per channel, the batch's consecutive hits on one key are summed in
        // registers (in row order) and that run added to the key's LDS row
        // once: keys that hold the argmax of many rows do not serialize on
        // one LDS address
#pragma unroll
        for (int ch = 0; ch < 2; ++ch) {
          const int kl = ch == 0 ? (hM ? kMl : -1) : (hm ? kml : -1);
          const float fl = rc[c][ch == 0 ? 1 : 3];
          int cur = -1;
          float run[NE];
#pragma unroll
          for (int x = 0; x < NE; ++x) run[x] = 0.f;
#pragma unroll
          for (int b = 0; b < GB; ++b) {
            if (src[b] < 0) break;  // wave-uniform
            const int key = __shfl(kl, src[b]);
            if (key < 0) continue;
            const float f = __shfl(fl, src[b]);
            if (key != cur) {
              if (cur >= 0) {
#pragma unroll
                for (int x = 0; x < NE; ++x)
                  if (lane + 64 * x < D) accw[cur * D + lane + 64 * x] += run[x];
              }
              cur = key;
#pragma unroll
              for (int x = 0; x < NE; ++x) run[x] = 0.f;
            }
#pragma unroll
            for (int x = 0; x < NE; ++x) run[x] = fmaf(f, qv[b][x], run[x]);
          }
          if (cur >= 0) {
#pragma unroll
            for (int x = 0; x < NE; ++x)
              if (lane + 64 * x < D) accw[cur * D + lane + 64 * x] += run[x];
          }
        }
      }
    }
  }
  __syncthreads();
  // the waves' sums in wave order onto the dK rows; wave w takes KPW keys
  // (their rows loaded together, then stored)
  constexpr int KPW = 32 / NW;
  float dk[KPW][NE];
#pragma unroll
  for (int t = 0; t < KPW; ++t)
#pragma unroll
    for (int x = 0; x < NE; ++x) {
      const int n = lane + 64 * x;
      const int j = j0 + KPW * w + t < T ? j0 + KPW * w + t : T - 1;
      dk[t][x] = a.dk[slice + (size_t)j * D + (n < D ? n : 0)];
    }
#pragma unroll
  for (int t = 0; t < KPW; ++t)
#pragma unroll
    for (int x = 0; x < NE; ++x) {
      const int n = lane + 64 * x, jj = KPW * w + t;
      if ((j0 + jj < T) & (n < D)) {
        float sum = acc[0][jj * D + n];
#pragma unroll
        for (int v = 1; v < NW; ++v) sum += acc[v][jj * D + n];
        a.dk[slice + (size_t)(j0 + jj) * D + n] = dk[t][x] + sum;
      }
    }
}

// ---------------------------------------------------------------------------
// P1 (App. B, Detach): each detached row of dS minus its mean over the row's
// n_i valid keys, applied to dQ and dK as rank-1 corrections,
//   dQ_i -= scale * mean_i * sum_{j valid for i} k_j
//   dK_j -= scale * sum_{i: j valid for i} mean_i q_i,   mean_i = S_self_i / n_i
// (dV has no calibration term). One workgroup per (b,h) and 64 columns:
// four row segments scan in parallel and are combined through LDS.
template <int D, typename TI>
__global__ __launch_bounds__(256) void bwd_p1_kernel(BwdArgsT<TI> a) {
  constexpr int NCB = (D + 63) / 64;
  __shared__ float part[2][4][64];
  const int tid = threadIdx.x, cl = tid & 63, seg = tid >> 6;
  const int bh = blockIdx.x / NCB, cb = blockIdx.x % NCB;
  const int col = cb * 64 + cl;
  const bool cok = col < D;
  const int T = a.T;
  const int L = (T + 3) / 4;
  const int r0 = min(T, seg * L), r1 = min(T, r0 + L);
  const size_t slice = (size_t)bh * T * D;
  const float *ss = a.st.sself + (size_t)bh * T;
  auto mean = [&](int i) { return ss[i] / (float)(a.causal ? i + 1 : T); };
  const int cc = cok ? col : 0;
  float ks = 0.f, qs = 0.f;
  for (int i = r0; i < r1; ++i) {
    ks += load1(a.k + slice + (size_t)i * D + cc);
    qs += mean(i) * load1(a.q + slice + (size_t)i * D + cc);
  }
  part[0][seg][cl] = ks;
  part[1][seg][cl] = qs;
  __syncthreads();
  float kpre = 0.f, qsuf = 0.f, ktot = 0.f, qtot = 0.f;
#pragma unroll
  for (int s2 = 0; s2 < 4; ++s2) {
    const float kk = part[0][s2][cl], qq = part[1][s2][cl];
    ktot += kk;
    qtot += qq;
    if (s2 < seg) kpre += kk;
    if (s2 > seg) qsuf += qq;
  }
  if (!cok) return;
  for (int i = r0; i < r1; ++i) {
    kpre += load1(a.k + slice + (size_t)i * D + col);
    a.dq[slice + (size_t)i * D + col] -= a.scale * mean(i) * (a.causal ? kpre : ktot);
  }
  for (int j = r1 - 1; j >= r0; --j) {
    qsuf += mean(j) * load1(a.q + slice + (size_t)j * D + col);
    a.dk[slice + (size_t)j * D + col] -= a.scale * (a.causal ? qsuf : qtot);
  }
}

// ---------------------------------------------------------------------------
// bf16-output variant: the fp32 dQ, dK accumulators rounded once to bf16
// (nearest even), 8 elements per thread (n8 groups of 8).
__global__ __launch_bounds__(256) void cast_bf16_kernel(const float *src, uint16_t *dst,
                                                       size_t n8) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n8) return;
  const f32x4 x = *reinterpret_cast<const f32x4 *>(src + 8 * i);
  const f32x4 y = *reinterpret_cast<const f32x4 *>(src + 8 * i + 4);
  *reinterpret_cast<uint4 *>(dst + 8 * i) =
      make_uint4(pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]), pack_bf16x2(y[0], y[1]),
                 pack_bf16x2(y[2], y[3]));
}

// ---------------------------------------------------------------------------
// Score-gradient decomposition export: g_self dense from the dS scratch
// (fp32 tiles, or bf16 tiles of the bf16 variant) and the row sums of the
// two extremum channels. One wave per (b,h, 32-query tile).
__global__ __launch_bounds__(256) void score_grad_kernel(GradArgs a) {
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, half = lane >> 5, l32 = lane & 31;
  const int T = a.T;
  const int nq = (T + 31) / 32;
  const size_t gw = (size_t)blockIdx.x * 4 + wave;
  if (gw >= (size_t)a.BH * nq) return;
  const int bh = (int)(gw / nq), qt = (int)(gw % nq);
  const int i = qt * 32 + l32;
  const bool minmax = a.calib == CAL_MINMAX;
  if (half == 0 && i < T) {
    const size_t ridx = (size_t)bh * T + i;
    const bool degen = a.st.rowrec[ridx * RR_COUNT + RR_FLAGS] != 0.f;
    const float s = a.st.sself[ridx];
    const float cMv = degen ? 0.f : (minmax ? a.st.cM[ridx] : -s);
    a.cM[ridx] = cMv;
    a.cm[ridx] = (degen || !minmax) ? 0.f : -(s + cMv);
  }
  for (int kt = 0; kt < nq; ++kt) {
    const bool stored = !a.causal || kt <= qt;
    float v[16];
    if (stored) {
      const size_t tile = ds_tile(bh, qt, kt, nq, a.causal) * 1024;
      if (a.bf16) {
        const uint16_t *src = reinterpret_cast<const uint16_t *>(a.st.dS) + tile + 8 * lane;
#pragma unroll
        for (int r = 0; r < 16; ++r) v[r] = bf2f(src[512 * (r / 8) + r % 8]);
      } else {
        tile_load(a.st.dS + tile, lane, v);
      }
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int j = kt * 32 + krel(r, half);
      if (i < T && j < T)
        a.g_self[((size_t)bh * T + i) * T + j] =
            (stored && (!a.causal || j <= i)) ? v[r] : 0.f;
    }
  }
}

#define KIA_MAIN_INST(KERNEL, D)                                        \
  template __global__ void KERNEL<D, CAL_MINMAX, REC_LERP>(BwdArgs);    \
  template __global__ void KERNEL<D, CAL_MINMAX, REC_NEAREST>(BwdArgs); \
  template __global__ void KERNEL<D, CAL_FWM, REC_LERP>(BwdArgs);       \
  template __global__ void KERNEL<D, CAL_FWM, REC_NEAREST>(BwdArgs);    \
  template __global__ void KERNEL<D, CAL_RESOLVED, REC_LERP>(BwdArgs);    \
  template __global__ void KERNEL<D, CAL_RESOLVED, REC_NEAREST>(BwdArgs); \
  template __global__ void KERNEL<D, CAL_FWM, REC_SOFTMAX>(BwdArgs);    \
  template __global__ void KERNEL<D, CAL_FWM, REC_BF16EXP>(BwdArgs);    \
  template __global__ void KERNEL<D, CAL_FWM, REC_FP8EXP>(BwdArgs);
KIA_MAIN_INST(bwd_main_shared_kernel, 16)
KIA_MAIN_INST(bwd_main_shared_kernel, 32)
KIA_MAIN_INST(bwd_main_shared_kernel, 64)
KIA_MAIN_INST(bwd_main_kernel, 128)

#define KIA_INST(D)                                                       \
  template __global__ void bwd_pre_kernel<D, float>(BwdArgs);             \
  template __global__ void bwd_pre_kernel<D, uint16_t>(BwdArgs16);        \
  template __global__ void bwd_dq_kernel<D, dq_tiles(D)>(BwdArgs);        \
  template __global__ void bwd_ties_kernel<D, float>(BwdArgs);            \
  template __global__ void bwd_ties_kernel<D, uint16_t>(BwdArgs16);     \
  template __global__ void bwd_p1_kernel<D, float>(BwdArgs);              \
  template __global__ void bwd_p1_kernel<D, uint16_t>(BwdArgs16);        \
  template __global__ void calib_gather_kernel<D, float, 1>(BwdArgs);     \
  template __global__ void calib_gather_kernel<D, float, 4>(BwdArgs);     \
  template __global__ void calib_gather_kernel<D, uint16_t, 1>(BwdArgs16); \
  template __global__ void calib_gather_kernel<D, uint16_t, 4>(BwdArgs16);
KIA_INST(16)
KIA_INST(32)
KIA_INST(64)
KIA_INST(128)

template __global__ void row_sums_kernel<float>(BwdArgs);
template __global__ void row_sums_kernel<uint16_t>(BwdArgs16);

}  // namespace kia
