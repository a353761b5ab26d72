// Internal launch interface between the C ABI layer and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vitattn {

struct FwdArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  float* o;
  float* lse;
  int BH, N, d;
  float scale;
  hipStream_t stream;
};

struct BwdArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const float* o;
  const uint16_t* dout;
  const float* lse;
  float* dq;
  float* dk;
  float* dv;
  float* drow;  // workspace: D = rowsum(dO o O), [BH][N]
  int BH, N, d;
  float scale;
  hipStream_t stream;
};

hipError_t launch_fwd(const FwdArgs& a);
// Backward stages; launch_bwd runs all three in order.
hipError_t launch_bwd_rowdot(const BwdArgs& a);
hipError_t launch_bwd_dkdv(const BwdArgs& a);
hipError_t launch_bwd_dq(const BwdArgs& a);
hipError_t launch_bwd(const BwdArgs& a);

}  // namespace vitattn
