// Internal declarations shared by the LittleBit HIP kernels and the C-ABI layer.
// Device helpers here implement the storage conventions of LB layout v1 and the
// dtype conversions; the method's arithmetic lives in the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>
#include <stdint.h>

#include "../../include/littlebit.h"

namespace lb {

constexpr int kDtF32 = LB_F32;
constexpr int kDtF16 = LB_F16;
constexpr int kDtBF16 = LB_BF16;

// ---------------------------------------------------------------------------
// dtype conversions (all exact widenings; one RNE narrowing at stores)
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf16_bits_to_f32(uint32_t u16) { return __uint_as_float(u16 << 16); }

__device__ __forceinline__ float f16_bits_to_f32(uint32_t u16) {
  return __half2float(__ushort_as_half(static_cast<unsigned short>(u16)));
}

__device__ __forceinline__ float load_as_f32(const void* p, int64_t i, int dt) {
  if (dt == kDtF32) return static_cast<const float*>(p)[i];
  const uint32_t u = static_cast<const uint16_t*>(p)[i];
  return dt == kDtBF16 ? bf16_bits_to_f32(u) : f16_bits_to_f32(u);
}

// fp32 -> bf16 bit pattern, round to nearest even; NaN stays NaN (quiet).
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  const uint32_t u = __float_as_uint(f);
  const uint32_t rne = (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
  return (u & 0x7fffffffu) > 0x7f800000u ? ((u >> 16) | 0x40u) : rne;  // a select, not a branch
}

__device__ __forceinline__ void store_from_f32(void* p, int64_t i, int dt, float v) {
  if (dt == kDtF32) {
    static_cast<float*>(p)[i] = v;
  } else if (dt == kDtBF16) {
    static_cast<uint16_t*>(p)[i] = static_cast<uint16_t>(f32_to_bf16_bits(v));
  } else {
    static_cast<__half*>(p)[i] = __float2half_rn(v);
  }
}

// ---------------------------------------------------------------------------
// LB layout v1 addressing: word kb of output o for a matrix with n_out outputs,
// nb full 32-bit blocks and a tail plane of width tailw (0, 1..16 -> uint16,
// 17..31 -> uint32).  kb == nb addresses the tail plane (zero-extended).
// ---------------------------------------------------------------------------
struct PackedView {
  const uint32_t* base;
  int n_out;
  int nb;     // full 32-bit blocks along the reduction dimension
  int tailw;  // width of the tail block (0 = none)
};

__device__ __forceinline__ uint32_t load_word(const PackedView& v, int kb, int o) {
  if (kb < v.nb) return v.base[static_cast<int64_t>(kb) * v.n_out + o];
  const char* t = reinterpret_cast<const char*>(v.base) + static_cast<int64_t>(4) * v.nb * v.n_out;
  if (v.tailw <= 16) return reinterpret_cast<const uint16_t*>(t)[o];
  return reinterpret_cast<const uint32_t*>(t)[o];
}

// Number of 32-bit blocks (including a tail block) along a reduction of length n.
__host__ __device__ __forceinline__ int nblocks32(int n) { return (n + 31) >> 5; }

// ---------------------------------------------------------------------------
// agent-scope synchronisation helpers (the L2s of the eight XCDs are not
// coherent with each other; agent-scope release/acquire orders them)
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t atomic_add_release(uint32_t* p, uint32_t v) {
  return __hip_atomic_fetch_add(p, v, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t atomic_add_relaxed(uint32_t* p, uint32_t v) {
  return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t atomic_load_relaxed(const uint32_t* p) {
  return __hip_atomic_load(const_cast<uint32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void atomic_store_relaxed(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void atomic_store_release(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void fence_acquire_agent() { __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent"); }
__device__ __forceinline__ void fence_release_agent() { __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent"); }

// Bounded spin: wait until *p >= target.  Returns false if the bound is hit
// (the caller then records an error instead of hanging the GPU).
__device__ __forceinline__ bool spin_until_at_least(const uint32_t* p, uint32_t target) {
  for (uint32_t it = 0; it < (1u << 22); ++it) {
    if (atomic_load_relaxed(p) >= target) return true;
    __builtin_amdgcn_s_sleep(2);
  }
  return false;
}

// ---------------------------------------------------------------------------
// workspace control block (fixed offsets at the start of every workspace)
// ---------------------------------------------------------------------------
constexpr int kCtrlEpoch = 0;      // decode: tag of the last completed call
constexpr int kCtrlDone = 1;       // decode: finished stage-2 workgroups of the running call
constexpr int kCtrlError = 2;      // set to nonzero if a bounded wait expired
constexpr int kCtrlWords = 64;
constexpr size_t kCtrlBytes = ((kCtrlWords * 4 + 255) / 256) * 256;

// ---------------------------------------------------------------------------
// kernel launchers (defined in the .hip files)
// ---------------------------------------------------------------------------
struct ForwardArgs {
  const void* x;
  int act_dt;
  int T, d_in, d_out, r;
  const void* U[2];
  const void* V[2];
  const void* h[2];
  const void* g[2];
  const void* l[2];
  int sc_dt;
  void* y;
  void* ws;
  size_t ws_bytes;
  // control block (epoch, done counter, error word) of the decode kernels'
  // call protocol; nullptr: the start of ws.  Every linear of a list launch
  // shares the control block at the start of the list's workspace, so that
  // tags stay unique per workspace whatever the list's layout.
  void* ctrl = nullptr;
};

// Look-up-table decode kernel geometry (pure function of the sizes; also sizes
// the workspace).
struct DecodeGeom {
  int nkt;     // 16-latent tiles per path
  int s1d;     // d_in runs per tile
  int bpr;     // 32-input blocks per run
  int n_s1;    // stage-1 workgroups
  int n_s2;    // stage-2 workgroups
  int direct;  // stage 2 reads every run's partial (else two-level sums)
  int tch;     // tokens per stage-2 chunk
  int wpl;     // stage 2: U words per lane and path (1, 2, 4 or 8)
  size_t smem_bytes, smem_bytes_elem;  // vector-load and element-wise variants
  size_t partial_off, partial_slots;
  size_t wbuf_off, wbuf_slots;
  size_t ws_bytes;
};
DecodeGeom decode_geometry(int T, int d_in, int d_out, int r);
bool decode_supports(int64_t T, int64_t d_in, int64_t d_out, int64_t r);
constexpr int kDecodeMaxTokens = 4;
constexpr int kDecodeMaxBatch = 16;  // linears per list launch of the look-up-table decode kernel
constexpr int kDecodeMaxRank = 1024;  // stage-2 tables of one token fit in LDS
// Workspace of lb_linear_forward_many: the list's control block, then one
// counter of finished stage-2 workgroups per member of a list launch, each in
// a 256-byte line of its own (atomics on one line serialise), then the slices.
constexpr size_t kListCtrStride = 256;
constexpr size_t kListHdrBytes = kCtrlBytes + kDecodeMaxBatch * kListCtrStride;

// Matrix-core decode kernel geometry.
struct MmaGeom {
  int nmf;    // 16-latent tiles per path
  int s1d;    // d_in runs per tile
  int bpr;    // 32-wide input blocks per run
  int n_s1;   // stage-1 workgroups
  int n_s2;   // stage-2 workgroups
  int direct;
  size_t smem_bytes;
  size_t partial_off, partial_slots;
  size_t wbuf_off, wbuf_slots;
  size_t ws_bytes;
};
constexpr int kMmaMaxTokens = 64;
constexpr int kMmaMaxRank = 832;  // U words of one row (both paths) held in registers in stage 2
MmaGeom decode_mma_geometry(int T, int d_in, int d_out, int r, int act_dt);
bool decode_mma_supports(int64_t T, int64_t d_in, int64_t d_out, int64_t r);

struct PrefillGeom {
  int nkb;           // 32-latent blocks per path
  int ns16;          // 16-latent subtiles per path
  int ms, n_lt;      // stage-1 subtiles per wave, latent tiles
  int n_tt;          // stage-1 token tiles (64 tokens)
  int ks, kb_per;    // stage-1 splits of d_in, 32-input steps per split
  int ns16p;         // stage-1 partial-sum subtile slots per path
  int n_un, n_og;    // stage-2 output units (128 outputs), output groups
  int n_tt2;         // stage-2 token tiles (64 tokens)
  int res;           // stage 2 holds every w fragment of its tile in LDS
  int kbc;           // stage-2 32-latent blocks per chunk when not resident
  size_t smem1, smem2;  // dynamic LDS of the two matrix-core stages
  size_t pbuf_off, pbuf_floats;
  size_t wterm_off, wterm_bytes;
  size_t ws_bytes;
};
PrefillGeom prefill_geometry(int T, int d_in, int d_out, int r);
bool prefill_supports(int64_t T, int64_t d_in, int64_t d_out, int64_t r);

hipError_t launch_pack(const void* src, int dt, int rows, int r, int role, void* dst, int32_t* nan_count,
                       hipStream_t stream);
hipError_t launch_decode(const ForwardArgs& a, const DecodeGeom& g, hipStream_t stream);
// n (1 .. kDecodeMaxBatch) independent linears of one activation and scale
// dtype, each with its own workspace slice in a[i].ws, in one launch
hipError_t launch_decode_batch(const ForwardArgs* a, int n, hipStream_t stream);
hipError_t launch_prefill(const ForwardArgs& a, const PrefillGeom& g, hipStream_t stream);
hipError_t launch_decode_mma(const ForwardArgs& a, const MmaGeom& g, hipStream_t stream);
// n (1 .. kDecodeMaxBatch) independent linears of one activation and scale
// dtype (T <= 64 each), each with its own workspace slice, in one launch per
// group of equal token tiles and load form
hipError_t launch_decode_mma_batch(const ForwardArgs* a, int n, hipStream_t stream);
// Latent cache [T][2][r] of dtype lat_dt.  launch_latent runs stage 1 of
// the prefill kernels on a.x and stores the cache at a.y; launch_from_latent
// reads the cache `lat` and runs stage 2 into a.y (dtype a.act_dt).  The
// workspaces hold the stage-1 partial sums / the w terms only.
bool latent_supports(int64_t T, int64_t d_in, int64_t r);
bool from_latent_supports(int64_t T, int64_t d_out, int64_t r);
size_t latent_workspace_bytes(int T, int d_in, int r);
size_t from_latent_workspace_bytes(int T, int r);
hipError_t launch_latent(const ForwardArgs& a, int lat_dt, hipStream_t stream);
hipError_t launch_from_latent(const ForwardArgs& a, const void* lat, int lat_dt, hipStream_t stream);
hipError_t launch_dense_ref(const ForwardArgs& a, float* W, hipStream_t stream);
// Streaming list forward (stream.hip, stream_mma.hip): three kinds of launch
// for the whole list, the plan (descriptors and work maps) in the workspace.
// Lists whose linears have at most 2 tokens use the look-up-table kernels,
// other lists (up to 64 tokens) the matrix-core kernels.
bool stream_supports(const ForwardArgs& a);
bool stream_list_supports(const ForwardArgs* a, int n);
bool stream_mma_supports(const ForwardArgs& a);
size_t stream_mma_workspace_bytes(const ForwardArgs* a, int n);
hipError_t stream_mma_init(const ForwardArgs* a, int n, uint64_t fingerprint, void* ws, hipStream_t stream);
hipError_t stream_mma_forward(const ForwardArgs* a, int n, uint64_t fingerprint, void* ws, hipStream_t stream);
size_t stream_workspace_bytes(const ForwardArgs* a, int n);
hipError_t stream_init(const ForwardArgs* a, int n, uint64_t fingerprint, void* ws, hipStream_t stream);
hipError_t stream_forward(const ForwardArgs* a, int n, uint64_t fingerprint, void* ws, hipStream_t stream);
// Dual-SVID conversion (svid.hip)
bool svid_supports(int64_t d_out, int64_t d_in, int64_t r, int64_t over);
size_t svid_workspace_bytes(int d_out, int d_in, int r, int over);
hipError_t launch_dual_svid(const void* W, int wdt, int d_out, int d_in, int r, int over, int iters, uint64_t seed,
                            const lb_svid_out* out, float* W_res, void* ws, hipStream_t stream);
hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t stream);
// *out = the error word of the control block at ctrl, which is then cleared
hipError_t launch_take_status(uint32_t* ctrl, int32_t* out, hipStream_t stream);
hipError_t launch_zero_elems(void* p, int64_t n, int dt, hipStream_t stream);

}  // namespace lb
