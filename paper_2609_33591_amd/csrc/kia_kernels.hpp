// kia_kernels.hpp -- argument blocks and kernel declarations shared between
// the host entry points (kia_abi.hip) and the kernel sources.
#pragma once

#include "kia_device.hpp"

namespace kia {

struct FwdArgs {
  const float *q, *k, *v;
  float *o;
  Stats st;
  int BH, T, K, calib, recon, causal;
  float tau, scale;
};

struct CodesArgs {
  const float *q, *k;
  Stats st;
  uint16_t *codes;
  int BH, T, K, calib, causal;
  float tau, scale;
};

struct BwdArgs {
  const float *q, *k, *v, *o, *dO;
  float *dq, *dk, *dv;
  Stats st;
  int BH, T, K, calib, recon, ste, detach, causal;
  float tau, scale;
};

template <int D, int CALIB, int RECON, bool OL> __global__ void fwd_kernel(FwdArgs a);
template <int D, int CALIB> __global__ void codes_kernel(CodesArgs a);
template <int D> __global__ void bwd_pre_kernel(BwdArgs a);
template <int D, int CALIB, int RECON> __global__ void bwd_main_kernel(BwdArgs a);
template <int D, int CALIB, int RECON> __global__ void bwd_main_shared_kernel(BwdArgs a);
template <int D> __global__ void bwd_dq_kernel(BwdArgs a);
template <int D> __global__ void bwd_ties_kernel(BwdArgs a);

}  // namespace kia
