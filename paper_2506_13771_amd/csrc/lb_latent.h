// Internal declarations of the one-launch latent kernel for a few tokens.
#pragma once

#include "lb_internal.h"

namespace lb {

constexpr int kLatentSmallMaxT = 4;  // tokens the one-launch latent kernel takes

bool latent_small_supports(int64_t T, int64_t d_in, int64_t r);
// the latent cache [T][2][r] (dtype lat_dt) of a.x at a.y, through a.V, a.g, a.l
hipError_t launch_latent_small(const ForwardArgs& a, int lat_dt, hipStream_t stream);

}  // namespace lb
