// kia_kernels.hpp -- argument blocks and kernel declarations shared between
// the host entry points (kia_abi.hip) and the kernel sources.
#pragma once

#include "kia_device.hpp"

namespace kia {

// TI: element type of the inputs q, k, v, dO (float, or uint16_t holding
// bf16 bits); outputs and statistics are fp32 either way.
template <typename TI> struct FwdArgsT {
  const TI *q, *k, *v;
  float *o;
  Stats st;
  int BH, T, K, calib, recon, causal;
  float tau, scale;
  uint16_t *o16 = nullptr;  // bf16-output variant: O as bf16 here instead of o
  // 0 (forward only): the fp32 second pass stores no decisions in U (the
  // bf16 forward stores them regardless: the branch costs its d = 128
  // instance ~500 B of spills per lane)
  int keep = 1;
};

template <typename TI> struct CodesArgsT {
  const TI *q, *k;
  Stats st;
  uint16_t *codes;
  int BH, T, K, calib, causal;
  float tau, scale;
};

template <typename TI> struct BwdArgsT {
  const TI *q, *k, *v;
  const float *o;
  const TI *dO;
  float *dq, *dk, *dv;
  Stats st;
  int BH, T, K, calib, recon, ste, grad, causal;  // grad: GRAD_* mode
  // qsplit > 1: each key block's query range is split over qsplit workgroups
  // of bwd_main, which add their dK/dV into dk/dv (zeroed by bwd_pre)
  int qsplit;
  // dq_piece > 0: bwd_dq cuts each query group's 64-key chunks into pieces
  // of at most dq_piece chunks, which add into dq (zeroed by bwd_pre)
  int dq_piece;
  // 1: every reduction in a fixed order (kia_set_deterministic): row sums
  // through st.part, calibration terms gathered per key, ties one wave per
  // slice; qsplit = 1 and dq_piece = 0
  int det = 0;
  float tau, scale;
  // bf16-output variant: the forward's O read as bf16 from o16 (instead of
  // o) and dV written as bf16 to dv16 (instead of dv); dq and dk then point
  // at the fp32 accumulators in stats, which cast_bf16_kernel rounds at the end
  const uint16_t *o16 = nullptr;
  uint16_t *dv16 = nullptr;
};

using FwdArgs = FwdArgsT<float>;
using CodesArgs = CodesArgsT<float>;
using BwdArgs = BwdArgsT<float>;
using FwdArgs16 = FwdArgsT<uint16_t>;
using CodesArgs16 = CodesArgsT<uint16_t>;
using BwdArgs16 = BwdArgsT<uint16_t>;

template <int D, int CALIB, int RECON, bool OL, int KP> __global__ void fwd_kernel(FwdArgs a);
template <int D, int CALIB, int REC, typename TI> __global__ void codes_kernel(CodesArgsT<TI> a);
// test exports: the code words of the decisions stored in U (no score
// recomputation), and the canonical fp32 score sub-tiles
struct StoredCodesArgs {
  Stats st;
  uint16_t *codes;
  int BH, T, K, causal;
};
template <int CALIB, int REC> __global__ void stored_codes_kernel(StoredCodesArgs a);
template <typename TI> struct ScoresArgsT {
  const TI *q, *k;
  float *scores;
  int BH, T, causal;
  float scale;
};
template <int D, typename TI> __global__ void scores_kernel(ScoresArgsT<TI> a);
template <int D, typename TI> __global__ void bwd_pre_kernel(BwdArgsT<TI> a);
template <int D, int CALIB, int RECON> __global__ void bwd_main_kernel(BwdArgs a);
template <int D, int CALIB, int RECON> __global__ void bwd_main_shared_kernel(BwdArgs a);
// query tiles per bwd_dq workgroup (x 2 key halves = its waves): two for
// d <= 64 (smaller workgroups, four per CU, balance the causal groups
// better), four for d = 128 (where the larger K chunk per thread would cost)
constexpr int dq_tiles(int d) { return d <= 64 ? 2 : 4; }
template <int D, int QG> __global__ void bwd_dq_kernel(BwdArgs a);
template <int D, typename TI> __global__ void bwd_ties_kernel(BwdArgsT<TI> a);
template <int D, typename TI> __global__ void bwd_p1_kernel(BwdArgsT<TI> a);
// deterministic backward: row sums from the key blocks' partials; the
// calibration terms of rows with unique extrema gathered onto dK per key
template <typename TI> __global__ void row_sums_kernel(BwdArgsT<TI> a);
template <int D, typename TI, int NW> __global__ void calib_gather_kernel(BwdArgsT<TI> a);
__global__ void cast_bf16_kernel(const float *src, uint16_t *dst, size_t n8);
struct GradArgs {
  Stats st;
  float *g_self, *cM, *cm;
  int BH, T, calib, causal, bf16;
};
__global__ void score_grad_kernel(GradArgs a);
struct GeoArgs {
  const float *q, *k;
  Stats st;
  float *out;  // [BH, T, 10]
  int BH, T, K, causal;
  float tau, scale;
};
template <int D, int CALIB, int RECON, int LQ> __global__ void geometry_kernel(GeoArgs a);
__global__ void mfma_probe_kernel(unsigned long long *out, int iters);
// bf16-input kernels (kia_bf16.hip)
template <int D, int CALIB, int RECON, bool OL> __global__ void fwd16_kernel(FwdArgs16 a);
template <int D, int CALIB, int RECON, bool SPLIT> __global__ void bwd16_main_kernel(BwdArgs16 a);
template <int D> __global__ void bwd16_dq_kernel(BwdArgs16 a);

}  // namespace kia
