// kia_abi.hip -- extern "C" entry points of libkia (declared in include/kia.h).
// Host side only: argument validation (before any launch), the stats layout,
// kernel selection by head dimension, and launches on the caller's stream.
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "kia.h"
#include "kia_kernels.hpp"

namespace {

using namespace kia;

constexpr int NFIELD = 16;  // KIA_STAT_ACC last (size 0 unless the bf16-output layout)

bool need_ol(int recon, int ste) {
  return recon == KIA_RECON_NEAREST && ste == KIA_STE_PROB;
}

// Byte size of each stats field (KIA_STAT_* order).
size_t field_bytes(int B, int H, int T, int d, int recon, int ste, int causal,
                   int field) {
  const size_t R = (size_t)B * H * T;
  switch (field) {
    case KIA_STAT_ROWREC: return R * RR_COUNT * sizeof(float);
    // present for every operator, so that no field's offset depends on
    // recon or ste (only Nearest with Prob-STE writes it)
    case KIA_STAT_OL: return R * (size_t)d * sizeof(float);
    case KIA_STAT_DS:
    case KIA_STAT_U:
      return (size_t)B * H * ds_tiles_per_slice((T + 31) / 32, causal) * 1024 * sizeof(float);
    // (also the calibration records of the deterministic gather: 4 per row)
    case KIA_STAT_PART:
      return std::max<size_t>(2 * (size_t)((T + 127) / 128), 4) * R * sizeof(float);
    case KIA_STAT_ACC: return 0;  // only in kia_stats_bytes_bf16o
    default: return R * 4;
  }
}

size_t field_offset(int B, int H, int T, int d, int recon, int ste, int causal,
                    int field) {
  size_t off = 0;
  for (int f = 0; f < field; ++f)
    off += align256(field_bytes(B, H, T, d, recon, ste, causal, f));
  return off;
}

int check_shape(int B, int H, int T, int d) {
  if (B < 1 || H < 1 || T < 1 || T > 65536) return KIA_ERR_SHAPE;
  if (d != 16 && d != 32 && d != 64 && d != 128) return KIA_ERR_HEADDIM;
  const long double n = (long double)B * H * T * d;
  if (n >= 2147483648.0L) return KIA_ERR_SHAPE;
  return KIA_OK;
}

bool recon_ok(int recon) { return recon >= KIA_RECON_LERP && recon <= KIA_RECON_FP8EXP; }

// The statistics (bf16-output accumulators included) must fit in
// KIA_MAX_STATS_BYTES: the two tile fields grow as T^2.
int check_size(int B, int H, int T, int d, int causal) {
  const size_t bytes = field_offset(B, H, T, d, 0, 0, causal, NFIELD) +
                       align256((size_t)3 * B * H * T * d * sizeof(float));
  return bytes > (size_t)KIA_MAX_STATS_BYTES ? KIA_ERR_SHAPE : KIA_OK;
}

int check_args(int B, int H, int T, int d, int K, int calib, float tau,
               int recon, int ste, int detach, int causal) {
  int rc = check_shape(B, H, T, d);
  if (rc) return rc;
  if (is_exp_rec(recon)) {
    // exponential weight functions: K, calib, tau and ste are not used
    if (!recon_ok(recon) || detach < GRAD_FULL || detach > KIA_GRAD_NONE ||
        (causal != 0 && causal != 1))
      return KIA_ERR_ENUM;
    return check_size(B, H, T, d, causal);
  }
  if (K < 1 || K > 64) return KIA_ERR_K;
  if (calib < KIA_CALIB_MINMAX || calib > KIA_CALIB_RESOLVED || (recon != 0 && recon != 1) ||
      (ste != 0 && ste != 1) || detach < GRAD_FULL || detach > KIA_GRAD_NONE ||
      (causal != 0 && causal != 1))
    return KIA_ERR_ENUM;
  if (calib != KIA_CALIB_MINMAX && !(tau > 0.f && isfinite(tau))) return KIA_ERR_TAU;
  return check_size(B, H, T, d, causal);
}

bool al16(const void *p) { return ((uintptr_t)p & 15u) == 0; }
bool al256(const void *p) { return ((uintptr_t)p & 255u) == 0; }

Stats make_stats(void *base, int B, int H, int T, int d, int recon, int ste,
                 int causal) {
  const bool ol = need_ol(recon, ste);
  char *b = static_cast<char *>(base);
  auto at = [&](int f) { return b + field_offset(B, H, T, d, recon, ste, causal, f); };
  Stats s;
  s.M = (float *)at(KIA_STAT_M);
  s.m = (float *)at(KIA_STAT_m);
  s.W = (float *)at(KIA_STAT_W);
  s.WL = (float *)at(KIA_STAT_WL);
  s.amax = (int *)at(KIA_STAT_AMAX);
  s.amin = (int *)at(KIA_STAT_AMIN);
  s.nmax = (int *)at(KIA_STAT_NMAX);
  s.nmin = (int *)at(KIA_STAT_NMIN);
  s.rowrec = (float *)at(KIA_STAT_ROWREC);
  s.sself = (float *)at(KIA_STAT_SSELF);
  s.cM = (float *)at(KIA_STAT_CM);
  s.OL = ol ? (float *)at(KIA_STAT_OL) : nullptr;
  s.dS = (float *)at(KIA_STAT_DS);
  s.U = (float *)at(KIA_STAT_U);
  s.part = (float *)at(KIA_STAT_PART);
  return s;
}

float softmax_scale(int d) { return (float)(1.0 / sqrt((double)d)); }

int g_grid = KIA_GRID_AUTO;  // kia_set_grid_policy
int g_det = 0;               // kia_set_deterministic

// Compute units of the current device (queried once per device).
int device_cus() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cached[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        n <= 0)
      n = 256;
    cached[dev] = n;
  }
  return cached[dev];
}

// ---- launch timing hook (kia_timing_enable / kia_timing_read) -----------
struct TimedLaunch {
  const char *name;
  hipEvent_t start, stop;
};
bool g_timing = false;
std::vector<TimedLaunch> g_launches;

void clear_launches() {
  for (auto &t : g_launches) {
    hipEventDestroy(t.start);
    hipEventDestroy(t.stop);
  }
  g_launches.clear();
}

// Runs `launch` (one kernel launch on stream s); when timing is on, brackets
// it with two events recorded on the same stream.
template <class F>
void timed(const char *name, hipStream_t s, F launch) {
  if (!g_timing || g_launches.size() >= 65536) {
    launch();
    return;
  }
  TimedLaunch t{name, nullptr, nullptr};
  if (hipEventCreate(&t.start) != hipSuccess || hipEventCreate(&t.stop) != hipSuccess) {
    launch();
    return;
  }
  hipEventRecord(t.start, s);
  launch();
  hipEventRecord(t.stop, s);
  g_launches.push_back(t);
}

int launched() {
  return hipGetLastError() == hipSuccess ? KIA_OK : KIA_ERR_HIP;
}

template <int D, int CALIB, int KP>
void launch_fwd_k(const FwdArgs &a, hipStream_t s) {
  const int bm = KP == 2 ? 64 : 32;  // two row groups of 32 rows, or one
  const dim3 grid(a.BH * ((a.T + bm - 1) / bm)), block(KP == 8 ? 512 : 256);
  if (a.recon == KIA_RECON_SOFTMAX)
    hipLaunchKernelGGL((fwd_kernel<D, CAL_FWM, REC_SOFTMAX, false, KP>), grid, block, 0, s, a);
  else if (a.recon == KIA_RECON_BF16EXP)
    hipLaunchKernelGGL((fwd_kernel<D, CAL_FWM, REC_BF16EXP, false, KP>), grid, block, 0, s, a);
  else if (a.recon == KIA_RECON_FP8EXP)
    hipLaunchKernelGGL((fwd_kernel<D, CAL_FWM, REC_FP8EXP, false, KP>), grid, block, 0, s, a);
  else if (a.recon == KIA_RECON_LERP)
    hipLaunchKernelGGL((fwd_kernel<D, CALIB, REC_LERP, false, KP>), grid, block, 0, s, a);
  else if (a.st.OL)
    hipLaunchKernelGGL((fwd_kernel<D, CALIB, REC_NEAREST, true, KP>), grid, block, 0, s, a);
  else
    hipLaunchKernelGGL((fwd_kernel<D, CALIB, REC_NEAREST, false, KP>), grid, block, 0, s, a);
}

// Two row groups x two key halves, unless the 64-row grid leaves CUs short
// of two workgroups: then one row group x four key quarters (twice the
// workgroups, half the keys per wave on the longest rows), or, with fewer
// 64-row blocks than CUs, one row group x eight key parts (8-wave
// workgroups, a quarter of the keys per wave).
template <int D, int CALIB>
void launch_fwd_c(const FwdArgs &a, hipStream_t s) {
  if constexpr (D <= 64) {
    const long blocks = (long)a.BH * ((a.T + 63) / 64);
    if (g_grid == KIA_GRID_AUTO && blocks < device_cus()) {
      launch_fwd_k<D, CALIB, 8>(a, s);
      return;
    }
    if (g_grid == KIA_GRID_SPLIT || (g_grid == KIA_GRID_AUTO && blocks < 2L * device_cus())) {
      launch_fwd_k<D, CALIB, 4>(a, s);
      return;
    }
  }
  launch_fwd_k<D, CALIB, 2>(a, s);
}

template <int D>
void launch_fwd(const FwdArgs &a, hipStream_t s) {
  timed("kia_fwd", s, [&] {
    if (a.calib == KIA_CALIB_MINMAX) launch_fwd_c<D, CAL_MINMAX>(a, s);
    else if (a.calib == KIA_CALIB_RESOLVED) launch_fwd_c<D, CAL_RESOLVED>(a, s);
    else launch_fwd_c<D, CAL_FWM>(a, s);
  });
}

template <int D, typename TI>
void launch_codes(const CodesArgsT<TI> &a, int recon, hipStream_t s) {
  const dim3 grid(a.BH * ((a.T + 127) / 128)), block(256);
  timed("kia_codes", s, [&] {
    if constexpr (sizeof(TI) == 4) {
      if (recon == KIA_RECON_SOFTMAX) {
        hipLaunchKernelGGL((codes_kernel<D, CAL_FWM, REC_SOFTMAX, TI>), grid, block, 0, s, a);
        return;
      }
      if (recon == KIA_RECON_BF16EXP) {
        hipLaunchKernelGGL((codes_kernel<D, CAL_FWM, REC_BF16EXP, TI>), grid, block, 0, s, a);
        return;
      }
      if (recon == KIA_RECON_FP8EXP) {
        hipLaunchKernelGGL((codes_kernel<D, CAL_FWM, REC_FP8EXP, TI>), grid, block, 0, s, a);
        return;
      }
    }
    if (a.calib == KIA_CALIB_MINMAX)
      hipLaunchKernelGGL((codes_kernel<D, CAL_MINMAX, REC_LERP, TI>), grid, block, 0, s, a);
    else if (a.calib == KIA_CALIB_RESOLVED)
      hipLaunchKernelGGL((codes_kernel<D, CAL_RESOLVED, REC_LERP, TI>), grid, block, 0, s, a);
    else
      hipLaunchKernelGGL((codes_kernel<D, CAL_FWM, REC_LERP, TI>), grid, block, 0, s, a);
  });
}

// ---- bf16 inputs ----------------------------------------------------------
template <int D, int CALIB>
void launch_fwd16_c(const FwdArgs16 &a, hipStream_t s) {
  const dim3 grid(a.BH * ((a.T + 63) / 64)), block(256);
  if (a.recon == KIA_RECON_LERP)
    hipLaunchKernelGGL((fwd16_kernel<D, CALIB, REC_LERP, false>), grid, block, 0, s, a);
  else if (a.st.OL)
    hipLaunchKernelGGL((fwd16_kernel<D, CALIB, REC_NEAREST, true>), grid, block, 0, s, a);
  else
    hipLaunchKernelGGL((fwd16_kernel<D, CALIB, REC_NEAREST, false>), grid, block, 0, s, a);
}

template <int D>
void launch_fwd16(const FwdArgs16 &a, hipStream_t s) {
  timed("kia_fwd", s, [&] {
    if (a.calib == KIA_CALIB_MINMAX) launch_fwd16_c<D, CAL_MINMAX>(a, s);
    else if (a.calib == KIA_CALIB_RESOLVED) launch_fwd16_c<D, CAL_RESOLVED>(a, s);
    else launch_fwd16_c<D, CAL_FWM>(a, s);
  });
}

template <int D, int CALIB, int RECON>
void launch_main16(const BwdArgs16 &a, int nkb, hipStream_t s) {
  // the query-range split as its own instantiation: the unsplit kernel keeps
  // plain stores in its epilogue
  if (a.qsplit > 1)
    hipLaunchKernelGGL((bwd16_main_kernel<D, CALIB, RECON, true>), dim3(a.BH * nkb), dim3(512), 0, s, a);
  else
    hipLaunchKernelGGL((bwd16_main_kernel<D, CALIB, RECON, false>), dim3(a.BH * nkb), dim3(512), 0, s, a);
}

template <int D, int CALIB, int RECON>
void launch_main(const BwdArgs &a, int nkb, hipStream_t s) {
  // d <= 64: eight waves share one K/V block; d = 128: four waves, K/V in registers
  if constexpr (D <= 64)
    hipLaunchKernelGGL((bwd_main_shared_kernel<D, CALIB, RECON>), dim3(a.BH * nkb), dim3(512), 0, s, a);
  else
    hipLaunchKernelGGL((bwd_main_kernel<D, CALIB, RECON>), dim3(a.BH * nkb), dim3(256), 0, s, a);
}

// The backward's four launches; TI selects the fp32 or the bf16-input
// main and dQ kernels (pre-pass and tie path are shared templates).
template <int D, typename TI>
void launch_bwd(const BwdArgsT<TI> &a, hipStream_t s) {
  constexpr bool B16 = sizeof(TI) == 2;
  const size_t R = (size_t)a.BH * a.T;
  const size_t rpb = 256 / (D / 4);
  timed("kia_bwd_pre", s, [&] {
    hipLaunchKernelGGL((bwd_pre_kernel<D, TI>), dim3((unsigned)((R + rpb - 1) / rpb)),
                       dim3(256), 0, s, a);
  });
  const int nkb = (a.T + 127) / 128 * a.qsplit;
  timed("kia_bwd_main", s, [&] {
    if constexpr (B16) {
      if (a.calib == KIA_CALIB_MINMAX) {
        if (a.recon == KIA_RECON_LERP) launch_main16<D, CAL_MINMAX, REC_LERP>(a, nkb, s);
        else launch_main16<D, CAL_MINMAX, REC_NEAREST>(a, nkb, s);
      } else if (a.calib == KIA_CALIB_RESOLVED) {
        if (a.recon == KIA_RECON_LERP) launch_main16<D, CAL_RESOLVED, REC_LERP>(a, nkb, s);
        else launch_main16<D, CAL_RESOLVED, REC_NEAREST>(a, nkb, s);
      } else {
        if (a.recon == KIA_RECON_LERP) launch_main16<D, CAL_FWM, REC_LERP>(a, nkb, s);
        else launch_main16<D, CAL_FWM, REC_NEAREST>(a, nkb, s);
      }
    } else if (a.recon == KIA_RECON_SOFTMAX) {
      launch_main<D, CAL_FWM, REC_SOFTMAX>(a, nkb, s);
    } else if (a.recon == KIA_RECON_BF16EXP) {
      launch_main<D, CAL_FWM, REC_BF16EXP>(a, nkb, s);
    } else if (a.recon == KIA_RECON_FP8EXP) {
      launch_main<D, CAL_FWM, REC_FP8EXP>(a, nkb, s);
    } else {
      if (a.calib == KIA_CALIB_MINMAX) {
        if (a.recon == KIA_RECON_LERP) launch_main<D, CAL_MINMAX, REC_LERP>(a, nkb, s);
        else launch_main<D, CAL_MINMAX, REC_NEAREST>(a, nkb, s);
      } else if (a.calib == KIA_CALIB_RESOLVED) {
        if (a.recon == KIA_RECON_LERP) launch_main<D, CAL_RESOLVED, REC_LERP>(a, nkb, s);
        else launch_main<D, CAL_RESOLVED, REC_NEAREST>(a, nkb, s);
      } else {
        if (a.recon == KIA_RECON_LERP) launch_main<D, CAL_FWM, REC_LERP>(a, nkb, s);
        else launch_main<D, CAL_FWM, REC_NEAREST>(a, nkb, s);
      }
    }
  });
  // deterministic backward: the key blocks' row-sum partials added up in
  // order (timed with the main kernel)
  if (a.det && a.grad != GRAD_DETACH) {
    timed("kia_bwd_main", s, [&] {
      hipLaunchKernelGGL(row_sums_kernel<TI>, dim3((unsigned)((R + 255) / 256)), dim3(256), 0,
                         s, a);
    });
  }
  const int nq = (a.T + 31) / 32;
  timed("kia_bwd_dq", s, [&] {
    if constexpr (B16) {
      hipLaunchKernelGGL(bwd16_dq_kernel<D>, dim3(a.BH * ((nq + 3) / 4)), dim3(512), 0, s, a);
    } else {
      constexpr int QG = dq_tiles(D);
      int items = 0;
      for (int g = 0; g < (nq + QG - 1) / QG; ++g)
        items += dq_pieces(g, a.T, a.causal, a.dq_piece, QG);
      hipLaunchKernelGGL((bwd_dq_kernel<D, QG>), dim3(a.BH * items), dim3(128 * QG), 0, s, a);
    }
    // deterministic backward: the unique extrema's calibration terms
    // gathered onto dK per 32 keys (bwd_dq leaves them out)
    // (four waves per 32 keys when the scans are long or the grid is
    // small, one otherwise: the four waves' 4x LDS halves the residency)
    if (a.det && grad_channels(a.grad)) {
      if (a.T >= 4096 || a.BH * nq < 8 * device_cus())
        hipLaunchKernelGGL((calib_gather_kernel<D, TI, 4>), dim3(a.BH * nq), dim3(256), 0, s, a);
      else
        hipLaunchKernelGGL((calib_gather_kernel<D, TI, 1>), dim3(a.BH * nq), dim3(64), 0, s, a);
    }
  });
  if (grad_channels(a.grad)) {
    // one wave per 32-row block, or per slice in the deterministic backward
    const size_t nw = a.det ? (size_t)a.BH : (size_t)a.BH * ((a.T + 31) / 32);
    timed("kia_bwd_ties", s, [&] {
      hipLaunchKernelGGL((bwd_ties_kernel<D, TI>), dim3((unsigned)((nw + 3) / 4)),
                         dim3(256), 0, s, a);
    });
  }
  if (a.grad == GRAD_P1) {
    timed("kia_bwd_p1", s, [&] {
      hipLaunchKernelGGL((bwd_p1_kernel<D, TI>), dim3(a.BH * ((D + 63) / 64)), dim3(256), 0,
                         s, a);
    });
  }
}

}  // namespace

extern "C" int kia_stats_bytes(int B, int H, int T, int d, int recon, int ste,
                               int causal, size_t *bytes) {
  if (!bytes) return KIA_ERR_NULL;
  *bytes = 0;
  int rc = check_shape(B, H, T, d);
  if (rc) return rc;
  if (!recon_ok(recon) || (ste != 0 && ste != 1) || (causal != 0 && causal != 1))
    return KIA_ERR_ENUM;
  rc = check_size(B, H, T, d, causal);
  if (rc) return rc;
  *bytes = field_offset(B, H, T, d, recon, ste, causal, NFIELD);
  return KIA_OK;
}

extern "C" int kia_stats_offset(int B, int H, int T, int d, int recon, int ste,
                                int causal, int field, size_t *offset) {
  if (!offset) return KIA_ERR_NULL;
  *offset = 0;
  int rc = check_shape(B, H, T, d);
  if (rc) return rc;
  if (!recon_ok(recon) || (ste != 0 && ste != 1) || (causal != 0 && causal != 1) ||
      field < 0 || field >= NFIELD)
    return KIA_ERR_ENUM;
  rc = check_size(B, H, T, d, causal);
  if (rc) return rc;
  *offset = field_offset(B, H, T, d, recon, ste, causal, field);
  return KIA_OK;
}

namespace {

// Outputs of the bf16-output variant (bf16 bits), or none.
struct Bf16Out {
  uint16_t *o = nullptr, *dq = nullptr, *dk = nullptr, *dv = nullptr;
};

size_t acc_offset(int B, int H, int T, int d, int causal) {
  return field_offset(B, H, T, d, 0, 0, causal, KIA_STAT_ACC);
}

template <typename TI>
int attn_fwd(const TI *q, const TI *k, const TI *v, float *o, void *stats, int B, int H, int T,
             int d, int K, int calib, float tau, int recon, int ste, int detach, int causal,
             void *stream, const Bf16Out *bo = nullptr) {
  int rc = check_args(B, H, T, d, K, calib, tau, recon, ste, detach, causal);
  if (rc) return rc;
  if (sizeof(TI) == 2 && is_exp_rec(recon)) return KIA_ERR_ENUM;  // fp32 inputs only
  if (bo) o = reinterpret_cast<float *>(bo->o);  // never written as fp32
  if (!q || !k || !v || !o || !stats) return KIA_ERR_NULL;
  if (!al16(q) || !al16(k) || !al16(v) || !al16(o) || !al256(stats))
    return KIA_ERR_ALIGN;
  FwdArgsT<TI> a;
  a.q = q; a.k = k; a.v = v; a.o = o;
  if (bo) a.o16 = bo->o;
  a.st = make_stats(stats, B, H, T, d, recon, ste, causal);
  if (detach == KIA_GRAD_NONE) {  // only the backward reads O^L and the stored decisions
    a.st.OL = nullptr;
    a.keep = 0;
  }
  a.BH = B * H; a.T = T; a.K = K; a.calib = calib; a.recon = recon;
  a.causal = causal; a.tau = calib != KIA_CALIB_MINMAX ? tau : 0.f;
  if (is_exp_rec(recon)) { a.calib = CAL_FWM; a.tau = 0.f; a.K = 1; }  // maximum only
  a.scale = softmax_scale(d);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if constexpr (sizeof(TI) == 2) {
    switch (d) {
      case 16: launch_fwd16<16>(a, s); break;
      case 32: launch_fwd16<32>(a, s); break;
      case 64: launch_fwd16<64>(a, s); break;
      default: launch_fwd16<128>(a, s); break;
    }
  } else {
    switch (d) {
      case 16: launch_fwd<16>(a, s); break;
      case 32: launch_fwd<32>(a, s); break;
      case 64: launch_fwd<64>(a, s); break;
      default: launch_fwd<128>(a, s); break;
    }
  }
  return launched();
}

template <typename TI>
int attn_bwd(const TI *q, const TI *k, const TI *v, const float *o, const TI *dO,
             void *stats, float *dq, float *dk, float *dv, int B, int H, int T, int d, int K,
             int calib, float tau, int recon, int ste, int detach, int causal,
             void *stream, const Bf16Out *bo = nullptr) {
  int rc = check_args(B, H, T, d, K, calib, tau, recon, ste, detach, causal);
  if (rc) return rc;
  if (detach == KIA_GRAD_NONE) return KIA_ERR_ENUM;  // forward only
  if (sizeof(TI) == 2 && is_exp_rec(recon)) return KIA_ERR_ENUM;  // fp32 inputs only
  if (bo) {
    // bf16 outputs: dQ and dK accumulate in fp32 in the stats field ACC
    // (rounded once at the end), dV is written as bf16 by the main kernel
    o = reinterpret_cast<const float *>(bo->o);
    dv = reinterpret_cast<float *>(bo->dv);
    if (!bo->dq || !bo->dk || !stats) return KIA_ERR_NULL;
    if (!al16(bo->dq) || !al16(bo->dk) || !al256(stats)) return KIA_ERR_ALIGN;
    dq = reinterpret_cast<float *>(static_cast<char *>(stats) + acc_offset(B, H, T, d, causal));
    dk = dq + (size_t)B * H * T * d;
    // dV as bf16 straight from the main kernel, or (split main kernel, whose
    // parts add up atomically) through the third fp32 accumulator
    if (!bo->dv) return KIA_ERR_NULL;
    dv = dk + (size_t)B * H * T * d;
  }
  if (!q || !k || !v || !o || !dO || !stats || !dq || !dk || !dv)
    return KIA_ERR_NULL;
  if (!al16(q) || !al16(k) || !al16(v) || !al16(o) || !al16(dO) ||
      !al16(dq) || !al16(dk) || !al16(dv) || !al256(stats))
    return KIA_ERR_ALIGN;
  BwdArgsT<TI> a;
  a.q = q; a.k = k; a.v = v; a.o = o; a.dO = dO;
  a.dq = dq; a.dk = dk; a.dv = dv;
  if (bo) a.o16 = bo->o;
  a.st = make_stats(stats, B, H, T, d, recon, ste, causal);
  a.BH = B * H; a.T = T; a.K = K; a.calib = calib; a.recon = recon;
  a.ste = ste; a.grad = detach; a.causal = causal;
  // small grids (the paper's micro-batch-1 calls): split the query range of
  // each key block of the main kernel into about 1.5 workgroups per CU
  // (one fits per CU; measured best against 1, 2 and 3 per CU: the split
  // parts pay their V load and their atomic dK/dV epilogue each)
  a.qsplit = 1;
  a.dq_piece = 0;
  if (g_grid != KIA_GRID_WIDE) {
    const bool force = g_grid == KIA_GRID_SPLIT;
    const int cus = device_cus();
    const int blocks = B * H * ((T + 127) / 128);
    if (blocks < cus || force)
      a.qsplit = std::min(8, std::max(force ? 2 : 1, (3 * cus + blocks) / (2 * blocks)));
  }
  if (sizeof(TI) == 4 && g_grid != KIA_GRID_WIDE) {
    const bool force = g_grid == KIA_GRID_SPLIT;
    const int cus = device_cus();
    // dQ (fp32 inputs): groups of dq_tiles(d) query tiles; when they do not
    // fill the chip, cut their keys into pieces so that there are about two
    // pieces per CU
    const int qg = dq_tiles(d);
    const int npq = (T + 32 * qg - 1) / (32 * qg);
    if (B * H * npq < cus || force) {
      long chunks = 0;
      for (int g = 0; g < npq; ++g) chunks += dq_chunks(g, T, causal, qg);
      chunks *= (long)B * H;
      a.dq_piece = (int)std::max(2L, (chunks + 2L * cus - 1) / (2L * cus));
    }
  }
  // the deterministic backward takes the unsplit launch shapes
  if (g_det) { a.qsplit = 1; a.dq_piece = 0; a.det = 1; }
  if (bo && a.qsplit == 1) a.dv16 = bo->dv;
  a.tau = calib != KIA_CALIB_MINMAX ? tau : 0.f;
  if (is_exp_rec(recon)) { a.calib = CAL_FWM; a.tau = 0.f; a.K = 1; a.ste = STE_WEIGHT; }
  a.scale = softmax_scale(d);
  hipStream_t s = static_cast<hipStream_t>(stream);
  switch (d) {
    case 16: launch_bwd<16, TI>(a, s); break;
    case 32: launch_bwd<32, TI>(a, s); break;
    case 64: launch_bwd<64, TI>(a, s); break;
    default: launch_bwd<128, TI>(a, s); break;
  }
  if (bo) {
    const size_t n8 = (size_t)B * H * T * d / 8;
    timed("kia_cast_bf16", s, [&] {
      const dim3 grid((unsigned)((n8 + 255) / 256)), block(256);
      hipLaunchKernelGGL(cast_bf16_kernel, grid, block, 0, s, dq, bo->dq, n8);
      hipLaunchKernelGGL(cast_bf16_kernel, grid, block, 0, s, dk, bo->dk, n8);
      if (!a.dv16) hipLaunchKernelGGL(cast_bf16_kernel, grid, block, 0, s, dv, bo->dv, n8);
    });
  }
  return launched();
}

template <typename TI>
int debug_codes(const TI *q, const TI *k, const void *stats, uint16_t *codes, int B, int H,
                int T, int d, int K, int calib, float tau, int recon, int causal,
                void *stream) {
  int rc = check_args(B, H, T, d, K, calib, tau, recon, 0, 0, causal);
  if (rc) return rc;
  if (sizeof(TI) == 2 && is_exp_rec(recon)) return KIA_ERR_ENUM;  // fp32 inputs only
  if (!q || !k || !stats || !codes) return KIA_ERR_NULL;
  if (!al16(q) || !al16(k) || !al256(stats)) return KIA_ERR_ALIGN;
  CodesArgsT<TI> a;
  a.q = q; a.k = k;
  a.st = make_stats(const_cast<void *>(stats), B, H, T, d, recon, 0, causal);
  a.codes = codes;
  a.BH = B * H; a.T = T; a.K = K; a.calib = calib; a.causal = causal;
  a.tau = calib != KIA_CALIB_MINMAX ? tau : 0.f;
  if (is_exp_rec(recon)) { a.calib = CAL_FWM; a.tau = 0.f; a.K = 1; }
  a.scale = softmax_scale(d);
  hipStream_t s = static_cast<hipStream_t>(stream);
  switch (d) {
    case 16: launch_codes<16, TI>(a, recon, s); break;
    case 32: launch_codes<32, TI>(a, recon, s); break;
    case 64: launch_codes<64, TI>(a, recon, s); break;
    default: launch_codes<128, TI>(a, recon, s); break;
  }
  return launched();
}

}  // namespace

extern "C" int kia_attn_fwd(const float *q, const float *k, const float *v,
                            float *o, void *stats, int B, int H, int T, int d,
                            int K, int calib, float tau, int recon, int ste,
                            int detach, int causal, void *stream) {
  return attn_fwd(q, k, v, o, stats, B, H, T, d, K, calib, tau, recon, ste, detach, causal,
                  stream);
}

extern "C" int kia_attn_bwd(const float *q, const float *k, const float *v,
                            const float *o, const float *dO, void *stats,
                            float *dq, float *dk, float *dv, int B, int H,
                            int T, int d, int K, int calib, float tau,
                            int recon, int ste, int detach, int causal,
                            void *stream) {
  return attn_bwd(q, k, v, o, dO, stats, dq, dk, dv, B, H, T, d, K, calib, tau, recon, ste,
                  detach, causal, stream);
}

// ---- static scratch of kia_attn_fwd_bwd_static ---------------------------
// The statistics of the no-allocation entry point live in this array; every
// GPU the library runs on holds its own copy until the process ends. In host
// code `scratch` only names the symbol: its device address on the current
// GPU comes from hipGetSymbolAddress, taken once per device (scratch_base).
static __device__ __align__(256) unsigned char scratch[KIA_STATIC_BYTES];

namespace {
std::mutex g_scratch_mu;
void *g_scratch_ptr[64] = {};

int scratch_base(void **out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return KIA_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return KIA_ERR_HIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return KIA_OK;
}
}  // namespace

extern "C" int kia_attn_fwd_bwd_static(const float *q, const float *k, const float *v,
                                       const float *dO, float *o, float *dq, float *dk,
                                       float *dv, int B, int H, int T, int d, int K,
                                       int calib, float tau, int recon, int ste, int detach,
                                       int causal, void *stream) {
  int rc = check_args(B, H, T, d, K, calib, tau, recon, ste, detach, causal);
  if (rc) return rc;
  if (detach == KIA_GRAD_NONE) return KIA_ERR_ENUM;  // its backward needs the forward's state
  if (!q || !k || !v || !dO || !o || !dq || !dk || !dv) return KIA_ERR_NULL;
  if (!al16(q) || !al16(k) || !al16(v) || !al16(dO) || !al16(o) || !al16(dq) || !al16(dk) ||
      !al16(dv))
    return KIA_ERR_ALIGN;
  if (field_offset(B, H, T, d, recon, ste, causal, NFIELD) > (size_t)KIA_STATIC_BYTES)
    return KIA_ERR_SCRATCH;
  void *base = nullptr;
  rc = scratch_base(&base);
  if (rc) return rc;
  rc = attn_fwd(q, k, v, o, base, B, H, T, d, K, calib, tau, recon, ste, detach, causal,
                stream);
  if (rc) return rc;
  return attn_bwd(q, k, v, o, dO, base, dq, dk, dv, B, H, T, d, K, calib, tau, recon, ste,
                  detach, causal, stream);
}

extern "C" int kia_debug_codes(const float *q, const float *k,
                               const void *stats, uint16_t *codes, int B,
                               int H, int T, int d, int K, int calib,
                               float tau, int recon, int causal,
                               void *stream) {
  return debug_codes(q, k, stats, codes, B, H, T, d, K, calib, tau, recon, causal, stream);
}

extern "C" int kia_attn_fwd_bf16(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                                 float *o, void *stats, int B, int H, int T, int d,
                                 int K, int calib, float tau, int recon, int ste,
                                 int detach, int causal, void *stream) {
  return attn_fwd(q, k, v, o, stats, B, H, T, d, K, calib, tau, recon, ste, detach, causal,
                  stream);
}

extern "C" int kia_attn_bwd_bf16(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                                 const float *o, const uint16_t *dO, void *stats,
                                 float *dq, float *dk, float *dv, int B, int H,
                                 int T, int d, int K, int calib, float tau,
                                 int recon, int ste, int detach, int causal,
                                 void *stream) {
  return attn_bwd(q, k, v, o, dO, stats, dq, dk, dv, B, H, T, d, K, calib, tau, recon, ste,
                  detach, causal, stream);
}

extern "C" int kia_stats_bytes_bf16o(int B, int H, int T, int d, int recon, int ste,
                                     int causal, size_t *bytes) {
  int rc = kia_stats_bytes(B, H, T, d, recon, ste, causal, bytes);
  if (rc) return rc;
  *bytes = acc_offset(B, H, T, d, causal) + align256((size_t)3 * B * H * T * d * sizeof(float));
  return KIA_OK;
}

extern "C" int kia_attn_fwd_bf16o(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                                  uint16_t *o, void *stats, int B, int H, int T, int d, int K,
                                  int calib, float tau, int recon, int ste, int detach,
                                  int causal, void *stream) {
  Bf16Out bo;
  bo.o = o;
  return attn_fwd(q, k, v, nullptr, stats, B, H, T, d, K, calib, tau, recon, ste, detach,
                  causal, stream, &bo);
}

extern "C" int kia_attn_bwd_bf16o(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                                  const uint16_t *o, const uint16_t *dO, void *stats,
                                  uint16_t *dq, uint16_t *dk, uint16_t *dv, int B, int H, int T,
                                  int d, int K, int calib, float tau, int recon, int ste,
                                  int detach, int causal, void *stream) {
  Bf16Out bo;
  bo.o = const_cast<uint16_t *>(o);
  bo.dq = dq; bo.dk = dk; bo.dv = dv;
  return attn_bwd(q, k, v, nullptr, dO, stats, nullptr, nullptr, nullptr, B, H, T, d, K, calib,
                  tau, recon, ste, detach, causal, stream, &bo);
}

extern "C" int kia_debug_codes_bf16(const uint16_t *q, const uint16_t *k,
                                    const void *stats, uint16_t *codes, int B,
                                    int H, int T, int d, int K, int calib,
                                    float tau, int recon, int causal,
                                    void *stream) {
  return debug_codes(q, k, stats, codes, B, H, T, d, K, calib, tau, recon, causal, stream);
}

extern "C" int kia_debug_codes_stored(const void *stats, uint16_t *codes, int B, int H,
                                      int T, int d, int K, int calib, float tau, int recon,
                                      int ste, int causal, void *stream) {
  int rc = check_args(B, H, T, d, K, calib, tau, recon, ste, 0, causal);
  if (rc) return rc;
  if (!stats || !codes) return KIA_ERR_NULL;
  if (!al256(stats) || !al16(codes)) return KIA_ERR_ALIGN;
  if ((long double)B * H * T * T >= 9.2e18L) return KIA_ERR_SHAPE;
  StoredCodesArgs a;
  a.st = make_stats(const_cast<void *>(stats), B, H, T, d, recon, ste, causal);
  a.codes = codes;
  a.BH = B * H; a.T = T; a.K = K; a.causal = causal;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const size_t nw = (size_t)a.BH * ((T + 31) / 32);
  const dim3 grid((unsigned)((nw + 3) / 4)), block(256);
  timed("kia_codes_stored", s, [&] {
    if (recon == KIA_RECON_SOFTMAX)
      hipLaunchKernelGGL((stored_codes_kernel<CAL_FWM, REC_SOFTMAX>), grid, block, 0, s, a);
    else if (recon == KIA_RECON_BF16EXP)
      hipLaunchKernelGGL((stored_codes_kernel<CAL_FWM, REC_BF16EXP>), grid, block, 0, s, a);
    else if (recon == KIA_RECON_FP8EXP)
      hipLaunchKernelGGL((stored_codes_kernel<CAL_FWM, REC_FP8EXP>), grid, block, 0, s, a);
    else if (calib == KIA_CALIB_MINMAX)
      hipLaunchKernelGGL((stored_codes_kernel<CAL_MINMAX, REC_LERP>), grid, block, 0, s, a);
    else if (calib == KIA_CALIB_RESOLVED)
      hipLaunchKernelGGL((stored_codes_kernel<CAL_RESOLVED, REC_LERP>), grid, block, 0, s, a);
    else if (recon == KIA_RECON_NEAREST)  // compact one-byte codes
      hipLaunchKernelGGL((stored_codes_kernel<CAL_FWM, REC_NEAREST>), grid, block, 0, s, a);
    else
      hipLaunchKernelGGL((stored_codes_kernel<CAL_FWM, REC_LERP>), grid, block, 0, s, a);
  });
  return launched();
}

namespace {
template <typename TI>
int debug_scores(const TI *q, const TI *k, float *scores, int B, int H, int T, int d,
                 int causal, void *stream) {
  int rc = check_shape(B, H, T, d);
  if (rc) return rc;
  if (causal != 0 && causal != 1) return KIA_ERR_ENUM;
  if (!q || !k || !scores) return KIA_ERR_NULL;
  if (!al16(q) || !al16(k) || !al16(scores)) return KIA_ERR_ALIGN;
  if ((long double)B * H * T * T >= 9.2e18L) return KIA_ERR_SHAPE;
  ScoresArgsT<TI> a;
  a.q = q; a.k = k; a.scores = scores;
  a.BH = B * H; a.T = T; a.causal = causal;
  a.scale = softmax_scale(d);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const dim3 grid(a.BH * ((T + 127) / 128)), block(256);
  timed("kia_scores", s, [&] {
    switch (d) {
      case 16: hipLaunchKernelGGL((scores_kernel<16, TI>), grid, block, 0, s, a); break;
      case 32: hipLaunchKernelGGL((scores_kernel<32, TI>), grid, block, 0, s, a); break;
      case 64: hipLaunchKernelGGL((scores_kernel<64, TI>), grid, block, 0, s, a); break;
      default: hipLaunchKernelGGL((scores_kernel<128, TI>), grid, block, 0, s, a); break;
    }
  });
  return launched();
}
}  // namespace

extern "C" int kia_debug_scores(const float *q, const float *k, float *scores, int B, int H,
                                int T, int d, int causal, void *stream) {
  return debug_scores(q, k, scores, B, H, T, d, causal, stream);
}

extern "C" int kia_debug_scores_bf16(const uint16_t *q, const uint16_t *k, float *scores,
                                     int B, int H, int T, int d, int causal, void *stream) {
  return debug_scores(q, k, scores, B, H, T, d, causal, stream);
}

extern "C" int kia_debug_score_grad(const void *stats, int input_bf16, float *g_self,
                                    float *cM, float *cm, int B, int H, int T, int d,
                                    int calib, int recon, int ste, int causal,
                                    void *stream) {
  int rc = check_shape(B, H, T, d);
  if (rc) return rc;
  if (calib < KIA_CALIB_MINMAX || calib > KIA_CALIB_RESOLVED || !recon_ok(recon) ||
      (ste != 0 && ste != 1) ||
      (causal != 0 && causal != 1) || (input_bf16 != 0 && input_bf16 != 1) ||
      (input_bf16 && is_exp_rec(recon)))
    return KIA_ERR_ENUM;
  if (is_exp_rec(recon)) calib = KIA_CALIB_FWM;  // maximum only
  if (!stats || !g_self || !cM || !cm) return KIA_ERR_NULL;
  if (!al256(stats) || !al16(g_self) || !al16(cM) || !al16(cm)) return KIA_ERR_ALIGN;
  if ((long double)B * H * T * T >= 9.2e18L) return KIA_ERR_SHAPE;
  GradArgs a;
  a.st = make_stats(const_cast<void *>(stats), B, H, T, d, recon, ste, causal);
  a.g_self = g_self; a.cM = cM; a.cm = cm;
  a.BH = B * H; a.T = T; a.calib = calib; a.causal = causal; a.bf16 = input_bf16;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const size_t nw = (size_t)a.BH * ((T + 31) / 32);
  timed("kia_score_grad", s, [&] {
    hipLaunchKernelGGL(score_grad_kernel, dim3((unsigned)((nw + 3) / 4)), dim3(256), 0, s, a);
  });
  return launched();
}

namespace {
template <int D, int CALIB, int RECON>
void launch_geo_c(const GeoArgs &a, hipStream_t s) {
  const dim3 grid(a.BH * ((a.T + 127) / 128)), block(256);
  // the quantile needs the order statistics floor((T-1)/1000) and the next
  const int need = (a.T - 1) / 1000 + 2;
  if (need <= 3)
    hipLaunchKernelGGL((geometry_kernel<D, CALIB, RECON, 3>), grid, block, 0, s, a);
  else if (need <= 12)
    hipLaunchKernelGGL((geometry_kernel<D, CALIB, RECON, 12>), grid, block, 0, s, a);
  else
    hipLaunchKernelGGL((geometry_kernel<D, CALIB, RECON, 67>), grid, block, 0, s, a);
}

template <int D>
void launch_geo(const GeoArgs &a, int calib, int recon, hipStream_t s) {
  timed("kia_geometry", s, [&] {
    if (calib == KIA_CALIB_MINMAX) {
      if (recon == KIA_RECON_LERP) launch_geo_c<D, CAL_MINMAX, REC_LERP>(a, s);
      else launch_geo_c<D, CAL_MINMAX, REC_NEAREST>(a, s);
    } else {
      if (recon == KIA_RECON_LERP) launch_geo_c<D, CAL_FWM, REC_LERP>(a, s);
      else launch_geo_c<D, CAL_FWM, REC_NEAREST>(a, s);
    }
  });
}
}  // namespace

extern "C" int kia_geometry_probe(const float *q, const float *k, const void *stats,
                                  float *out, int B, int H, int T, int d, int K,
                                  int calib, float tau, int recon, int causal,
                                  void *stream) {
  int rc = check_args(B, H, T, d, K, calib, tau, recon, 0, 0, causal);
  if (rc) return rc;
  if (calib == KIA_CALIB_RESOLVED || is_exp_rec(recon)) return KIA_ERR_ENUM;
  if (!q || !k || !stats || !out) return KIA_ERR_NULL;
  if (!al16(q) || !al16(k) || !al16(out) || !al256(stats)) return KIA_ERR_ALIGN;
  GeoArgs a;
  a.q = q; a.k = k;
  a.st = make_stats(const_cast<void *>(stats), B, H, T, d, recon, 0, causal);
  a.out = out;
  a.BH = B * H; a.T = T; a.K = K; a.causal = causal;
  a.tau = calib == KIA_CALIB_FWM ? tau : 0.f;
  a.scale = softmax_scale(d);
  hipStream_t s = static_cast<hipStream_t>(stream);
  switch (d) {
    case 16: launch_geo<16>(a, calib, recon, s); break;
    case 32: launch_geo<32>(a, calib, recon, s); break;
    case 64: launch_geo<64>(a, calib, recon, s); break;
    default: launch_geo<128>(a, calib, recon, s); break;
  }
  return launched();
}

extern "C" int kia_mfma_peak_probe(unsigned long long *out, int workgroups, int iters,
                                   void *stream) {
  if (!out) return KIA_ERR_NULL;
  if ((reinterpret_cast<uintptr_t>(out) & 7) != 0) return KIA_ERR_ALIGN;
  if (workgroups < 1 || workgroups > (1 << 20) || iters < 1 || iters > (1 << 20))
    return KIA_ERR_SHAPE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  timed("kia_mfma_probe", s, [&] {
    hipLaunchKernelGGL(mfma_probe_kernel, dim3(workgroups), dim3(256), 0, s, out, iters);
  });
  return launched();
}

extern "C" int kia_set_deterministic(int on) {
  if (on != 0 && on != 1) return KIA_ERR_ENUM;
  g_det = on;
  return KIA_OK;
}

extern "C" int kia_set_grid_policy(int policy) {
  if (policy != KIA_GRID_AUTO && policy != KIA_GRID_WIDE && policy != KIA_GRID_SPLIT)
    return KIA_ERR_ENUM;
  g_grid = policy;
  return KIA_OK;
}

extern "C" int kia_timing_enable(int on) {
  clear_launches();
  g_timing = on != 0;
  return KIA_OK;
}

extern "C" int kia_timing_read(const char *name, double *total_ms,
                               int *launches) {
  if (!name || !total_ms || !launches) return KIA_ERR_NULL;
  *total_ms = 0.0;
  *launches = 0;
  for (auto &t : g_launches) {
    if (strcmp(t.name, name) != 0) continue;
    if (hipEventSynchronize(t.stop) != hipSuccess) return KIA_ERR_HIP;
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, t.start, t.stop) != hipSuccess) return KIA_ERR_HIP;
    *total_ms += ms;
    *launches += 1;
  }
  return KIA_OK;
}

extern "C" const char *kia_strerror(int code) {
  switch (code) {
    case KIA_OK: return "success";
    case KIA_ERR_NULL: return "a required pointer is NULL";
    case KIA_ERR_SHAPE: return "B, H or T out of range, or tensor size overflow";
    case KIA_ERR_HEADDIM: return "head dimension d must be 16, 32, 64 or 128";
    case KIA_ERR_K: return "K must lie in [1, 64]";
    case KIA_ERR_ENUM: return "calib/recon/ste/detach (gradient mode)/causal/field out of range";
    case KIA_ERR_TAU: return "FWM needs a finite tau > 0";
    case KIA_ERR_ALIGN: return "tensors must be 16-byte and stats 256-byte aligned";
    case KIA_ERR_HIP: return "HIP kernel launch failed";
    case KIA_ERR_SCRATCH:
      return "the problem's statistics exceed the static scratch of kia_attn_fwd_bwd_static "
             "(KIA_STATIC_BYTES)";
    default: return "unknown error code";
  }
}
