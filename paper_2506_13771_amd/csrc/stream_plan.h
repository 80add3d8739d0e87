// The plan of a streaming list forward (lb_list_*), shared by the look-up-table
// kernels (stream.hip) and the matrix-core kernels (stream_mma.hip): the
// per-linear descriptor the kernels read, and the header at the start of the
// workspace (the control block's words, with the error word at kCtrlError, and
// the fingerprint of the descriptors the plan was written for).
#pragma once

#include "lb_internal.h"

namespace lb {
namespace splan {

struct alignas(16) StreamLinear {
  const void* x;
  void* y;
  const void* U[2];
  const void* V[2];
  const void* h[2];
  const void* g[2];
  const void* l[2];
  float* part;  // [2][T][s1d][r] partial sums l (.) z of each run
  float* wlat;  // [2][T][r]      w = l (.) z
  int T, d_in, d_out, r;
  int s1d, bpr;
  uint32_t x_bytes, g_bytes, h_bytes, l_bytes, v_bytes, u_bytes;
};

// plan header: the control block's words (error word at kCtrlError), the
// fingerprint at words 4-5, the list length and the three work counts
constexpr int kHdrFp = 4;
constexpr int kHdrN = 6;
constexpr int kHdrCounts = 7;

// every kernel of a list first checks the plan against the call
__device__ __forceinline__ bool plan_ok(const uint32_t* hdr, uint64_t fp) {
  const uint64_t have = (static_cast<uint64_t>(hdr[kHdrFp + 1]) << 32) | hdr[kHdrFp];
  if (have == fp) return true;
  if (threadIdx.x == 0) __hip_atomic_fetch_or(const_cast<uint32_t*>(hdr) + kCtrlError, 2u, __ATOMIC_RELAXED,
                                              __HIP_MEMORY_SCOPE_AGENT);
  return false;
}

inline size_t align256(size_t b) { return (b + 255) / 256 * 256; }

inline int64_t packed_bytes64(int64_t n_out, int64_t n_red) {
  const int64_t w = n_red & 31;
  return 4 * (n_red >> 5) * n_out + (w == 0 ? 0 : (w <= 16 ? 2 : 4)) * n_out;
}

inline bool has_work(const ForwardArgs& a) { return a.T > 0 && a.d_in > 0 && a.d_out > 0 && a.r > 0; }

}  // namespace splan
}  // namespace lb
