// Sign packing (Sec. 3.1, Eq. uv_sign) into LB layout v1, plus a zero-fill
// kernel for workspaces.
//
// One thread builds one 32-bit word (or one tail entry): bit t is set iff the
// element at reduction index 32 kb + t is negative (sign -1; +0, -0 and NaN give
// +1, NaNs are counted).  For LB_ROLE_V the reduction index runs down the rows
// of V, so consecutive threads (consecutive latent columns) read consecutive
// addresses of each row; for LB_ROLE_U it runs along a row of U, so each thread
// reads one contiguous 32-element run.
#include "lb_internal.h"

namespace lb {

namespace {

__device__ __forceinline__ bool is_neg_and_nan(const void* src, int64_t idx, int dt, int& nan) {
  float v = load_as_f32(src, idx, dt);
  nan += (v != v);
  return v < 0.0f;
}

__global__ void __launch_bounds__(256) pack_kernel(const void* __restrict__ src, int dt, int rows, int r, int role,
                                                  uint32_t* __restrict__ dst, int32_t* nan_count) {
  const int n_out = role == LB_ROLE_U ? rows : r;
  const int n_red = role == LB_ROLE_U ? r : rows;
  const int nb = n_red >> 5;
  const int w = n_red - 32 * nb;
  const int64_t n_full = static_cast<int64_t>(nb) * n_out;
  const int64_t n_items = n_full + (w ? n_out : 0);
  int nan = 0;
  for (int64_t item = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; item < n_items;
       item += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const bool tail = item >= n_full;
    const int kb = tail ? nb : static_cast<int>(item / n_out);
    const int o = tail ? static_cast<int>(item - n_full) : static_cast<int>(item - static_cast<int64_t>(kb) * n_out);
    const int width = tail ? w : 32;
    uint32_t word = 0;
    for (int t = 0; t < width; ++t) {
      const int q = 32 * kb + t;
      // element M[o][q] of the stage view, taken from src[rows][r]
      const int64_t idx = role == LB_ROLE_U ? static_cast<int64_t>(o) * r + q : static_cast<int64_t>(q) * r + o;
      word |= static_cast<uint32_t>(is_neg_and_nan(src, idx, dt, nan)) << t;
    }
    if (!tail) {
      dst[item] = word;
    } else if (w <= 16) {
      reinterpret_cast<uint16_t*>(dst + n_full)[o] = static_cast<uint16_t>(word);
    } else {
      dst[n_full + o] = word;
    }
  }
  if (nan_count && nan) atomicAdd(nan_count, nan);
}

// Zero n_words 32-bit words, then one trailing 16-bit half-word if `half_tail`.
__global__ void __launch_bounds__(256) fill_zero_kernel(uint32_t* __restrict__ p, int64_t n_words, int half_tail) {
  const int64_t i0 = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x;
  for (int64_t i = i0; i < n_words; i += static_cast<int64_t>(gridDim.x) * blockDim.x) p[i] = 0u;
  if (half_tail && i0 == 0) reinterpret_cast<uint16_t*>(p + n_words)[0] = 0;
}

__global__ void __launch_bounds__(256) zero_elems_kernel(void* __restrict__ p, int64_t n, int dt) {
  for (int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x)
    store_from_f32(p, i, dt, 0.0f);
}

}  // namespace

hipError_t launch_zero_elems(void* p, int64_t n, int dt, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  const int64_t blocks = (n + 255) / 256;
  const int grid = static_cast<int>(blocks < 8192 ? blocks : 8192);
  hipLaunchKernelGGL(zero_elems_kernel, dim3(grid), dim3(256), 0, stream, p, n, dt);
  return hipGetLastError();
}

hipError_t launch_pack(const void* src, int dt, int rows, int r, int role, void* dst, int32_t* nan_count,
                       hipStream_t stream) {
  const int n_out = role == LB_ROLE_U ? rows : r;
  const int n_red = role == LB_ROLE_U ? r : rows;
  const int64_t items = static_cast<int64_t>(nblocks32(n_red)) * n_out;
  if (items == 0) return hipSuccess;
  const int64_t blocks = (items + 255) / 256;
  const int grid = static_cast<int>(blocks < 65535 ? blocks : 65535);
  hipLaunchKernelGGL(pack_kernel, dim3(grid), dim3(256), 0, stream, src, dt, rows, r, role,
                     static_cast<uint32_t*>(dst), nan_count);
  return hipGetLastError();
}

hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t stream) {
  // bytes must be a multiple of 2 and p 4-byte aligned
  const int64_t n = static_cast<int64_t>(bytes / 4);
  const int half_tail = (bytes % 4) != 0;
  if (n == 0 && !half_tail) return hipSuccess;
  const int64_t blocks = (n + 255) / 256;
  const int grid = static_cast<int>(blocks < 1 ? 1 : (blocks < 8192 ? blocks : 8192));
  hipLaunchKernelGGL(fill_zero_kernel, dim3(grid), dim3(256), 0, stream, static_cast<uint32_t*>(p), n, half_tail);
  return hipGetLastError();
}

namespace {
__global__ void take_status_kernel(uint32_t* ctrl, int32_t* out) {
  const uint32_t v = __hip_atomic_exchange(ctrl + kCtrlError, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  *out = static_cast<int32_t>(v);
}
}  // namespace

hipError_t launch_take_status(uint32_t* ctrl, int32_t* out, hipStream_t stream) {
  hipLaunchKernelGGL(take_status_kernel, dim3(1), dim3(1), 0, stream, ctrl, out);
  return hipGetLastError();
}

}  // namespace lb
