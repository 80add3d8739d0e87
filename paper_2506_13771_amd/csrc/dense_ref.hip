// Checking path: dense effective weight from the packed buffers,
//   W[i][j] = sum_p h_p[i] g_p[j] sum_k s(U_p)[i][k] l_p[k] s(V_p)[j][k]
// (Sec. 3.1 Eq. w_primary_hat; Sec. 3.3 Eqs. res_approx_structure and
// final_weight_approx_res), fp32, ascending k.  Never on the forward path.
//
// A workgroup owns one output row i and 256 consecutive columns j.  The row's
// U words are staged in LDS; each thread walks k and reads the V word that
// holds bit (k, j) (threads of one 32-column block share it).
#include "lb_internal.h"

namespace lb {

namespace {

constexpr int kMaxRankWords = 512;  // r <= 16384 in this kernel

__global__ void __launch_bounds__(256) dense_ref_kernel(ForwardArgs a, float* __restrict__ W) {
  const int i = blockIdx.y;
  const int j = blockIdx.x * 256 + threadIdx.x;
  const int r = a.r;
  const int nw = nblocks32(r);
  __shared__ uint32_t urow[2][kMaxRankWords];
  for (int p = 0; p < 2; ++p) {
    const PackedView Uv{static_cast<const uint32_t*>(a.U[p]), a.d_out, r >> 5, r & 31};
    for (int kb = threadIdx.x; kb < nw; kb += 256) urow[p][kb] = load_word(Uv, kb, i);
  }
  __syncthreads();
  if (j >= a.d_in) return;
  float acc = 0.0f;
  for (int p = 0; p < 2; ++p) {
    const PackedView Vv{static_cast<const uint32_t*>(a.V[p]), r, a.d_in >> 5, a.d_in & 31};
    const int jb = j >> 5, jt = j & 31;
    float s = 0.0f;
    for (int k = 0; k < r; ++k) {
      const uint32_t ub = (urow[p][k >> 5] >> (k & 31)) & 1u;
      const uint32_t vb = (load_word(Vv, jb, k) >> jt) & 1u;
      const float lk = load_as_f32(a.l[p], k, a.sc_dt);
      s += (ub ^ vb) ? -lk : lk;
    }
    acc += load_as_f32(a.h[p], i, a.sc_dt) * s * load_as_f32(a.g[p], j, a.sc_dt);
  }
  W[static_cast<int64_t>(i) * a.d_in + j] = acc;
}

}  // namespace

hipError_t launch_dense_ref(const ForwardArgs& a, float* W, hipStream_t stream) {
  if (a.d_out == 0 || a.d_in == 0) return hipSuccess;
  if (nblocks32(a.r) > kMaxRankWords) return hipErrorInvalidValue;
  dim3 grid((a.d_in + 255) / 256, a.d_out);
  hipLaunchKernelGGL(dense_ref_kernel, grid, dim3(256), 0, stream, a, W);
  return hipGetLastError();
}

}  // namespace lb
