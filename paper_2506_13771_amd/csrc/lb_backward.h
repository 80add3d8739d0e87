// Internal declarations of the layer backward (quantization-aware training)
// and the prefill stages it reuses.
#pragma once

#include "lb_internal.h"

namespace lb {

// Prefill stage 1 without the latent scale: z [T][2][r] (fp32, token-major)
// of a.x through a.V and a.g (a.d_in inputs); a.ws holds the split partial
// sums (>= latent_workspace_bytes(T, d_in, r)).
hipError_t launch_stage1_sums(const ForwardArgs& a, float* z, hipStream_t stream);
// launch_stage1_sums of two inputs of one token count, rank and dtypes
// (a0.ws and a1.ws distinct), with one launch for both split sums.
hipError_t launch_stage1_sums2(const ForwardArgs& a0, float* z0, const ForwardArgs& a1, float* z1,
                               hipStream_t stream);
// Prefill stage 2 from w = l (.) src, src [T][2][r] fp32, through a.U, a.h
// and a.l into a.y (dtype a.act_dt, a.d_out outputs); a.ws holds the w terms
// (>= from_latent_workspace_bytes(T, r)).
hipError_t launch_stage2_scaled(const ForwardArgs& a, const float* src, hipStream_t stream);

struct BackwardArgs {
  const void* x;   // [T][d_in], act_dt
  const void* dy;  // [T][d_out], act_dt
  int act_dt, sc_dt;
  int T, d_in, d_out, r;
  const void* V[2];   // V signs, LB layout v1 role V (the forward's)
  const void* Ut[2];  // U signs packed with role V: M[k][i]
  const void* Vt[2];  // V signs packed with role U: M[j][k]
  const void* h[2];
  const void* g[2];
  const void* l[2];
  const float* U_lat[2];  // [d_out][r]
  const float* V_lat[2];  // [d_in][r]
  float* dU[2];
  float* dV[2];
  float* dh[2];
  float* dg[2];
  float* dl[2];
  void* dx;  // [T][d_in], act_dt, or null
  float kappa;
  void* ws;
  size_t ws_bytes;
};

bool backward_supports(int64_t T, int64_t d_in, int64_t d_out, int64_t r);
size_t backward_workspace_bytes(int T, int d_in, int d_out, int r);
// every size >= 1
hipError_t launch_backward(const BackwardArgs& b, hipStream_t stream);

}  // namespace lb
