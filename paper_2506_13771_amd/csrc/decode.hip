// Decode kernel (small T): one launch computes
//   y[t][i] = sum_p h_p[i] sum_k U_p[i][k] l_p[k] z_p[t][k],
//   z_p[t][k] = sum_j V_p[j][k] g_p[j] x[t][j]
// for both paths (Proposition 1, Eq. proposition1; Sec. 3.3 Eq.
// final_weight_approx_res).  Signs are applied by flipping the IEEE sign bit of
// the fp32 operand (exact); accumulation is fp32.
//
// Launch structure (one grid, two roles, no host round trip):
//  * stage-1 workgroups hold the LOWEST block ids.  Each owns one path, a tile
//    of 16 latent columns and one of at most 8 runs of d_in.  Lane (kk, bs)
//    takes column k0 + kk and every 16th 32-wide block of the run, so the 16
//    lanes of a group read 64 contiguous bytes of V per step and accumulate in
//    registers; a fixed-order LDS reduction over the 16 groups ends the run.
//    The partial z goes to the workspace and an agent-scope counter is
//    incremented with release semantics.  Stage-1 workgroups never wait.
//  * stage-2 workgroups (higher ids, dispatched after every stage-1 workgroup
//    of their XCD) load their U words into registers first, then wait on the
//    counter (bounded spin), gather l (.) z with all partial loads in flight at
//    once (at most 8 partials per value, summed in a fixed order, so the result
//    is bitwise reproducible), and contract with U: KQ adjacent lanes share an
//    output row and split its words; a DPP butterfly joins them.  Both paths
//    are summed in fp32 and y is stored once.
//  * When T * r is large, the last-arriving stage-1 workgroup of each (path,
//    latent tile) first reduces that tile's partials ("two-level" mode), so
//    stage-2 workgroups read only the final l (.) z.
//  * The last stage-2 workgroup to finish resets every counter it used, so the
//    workspace needs no clearing between calls.
#include "lb_internal.h"

namespace lb {

namespace {

struct DecodeParams {
  const void* x;
  void* y;
  const void* U[2];
  const void* V[2];
  const void* h[2];
  const void* g[2];
  const void* l[2];
  uint32_t* ctrl;
  uint64_t* partial;  // [2][s1d][T][r] tagged partial z
  uint64_t* wbuf;     // [2][T][r] tagged l (.) z (two-level mode)
  int act_dt, sc_dt;
  int T, d_in, d_out, r;
  int nkt, bpw, s1d, n_s1;
  int kq_log2, rows2, n_s2, direct, tch;
};

constexpr int kThreads = 256;
constexpr int kKc = 16;        // latent columns per stage-1 tile
constexpr int kChunk = 16;     // 32-wide d_in blocks staged per stage-1 step
constexpr int kAStride = 36;   // LDS stride of one staged 32-wide block (bank spread)
constexpr int kMaxSplit = 8;   // d_in runs per latent tile (partials per z value)
constexpr int kPrefetch = 4;   // U words per path held in registers across the wait

__device__ __forceinline__ float flip(float v, uint32_t signmask) {
  return __uint_as_float(__float_as_uint(v) ^ signmask);
}

// Sum over the KQ lanes (adjacent, power of two <= 16) that share an output row.
__device__ __forceinline__ float row_sum(float v, int kq_log2) {
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));  // xor 1
  if (kq_log2 >= 2)
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false));  // xor 2
  if (kq_log2 >= 3) v += __shfl_xor(v, 4);
  if (kq_log2 >= 4) v += __shfl_xor(v, 8);
  return v;
}

// Tagged 64-bit slot: high word = call tag, low word = fp32 bits.  Written and
// read with relaxed agent-scope atomics, which are coherent across the XCDs'
// L2s without any cache writeback or invalidation.
__device__ __forceinline__ void put_slot(uint64_t* p, uint32_t tag, float v) {
  const uint64_t w = (static_cast<uint64_t>(tag) << 32) | __float_as_uint(v);
  __hip_atomic_store(p, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t get_slot(const uint64_t* p) {
  return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float slot_value(uint64_t w) { return __uint_as_float(static_cast<uint32_t>(w)); }
__device__ __forceinline__ bool slot_ready(uint64_t w, uint32_t tag) { return static_cast<uint32_t>(w >> 32) == tag; }

constexpr uint32_t kSpinLimit = 1u << 19;

// Sum of n (<= kMaxSplit) tagged slots spaced `stride` apart, waiting until every
// slot carries `tag`; summed in ascending slot order.  Returns false on timeout.
__device__ __forceinline__ bool gather_sum(const uint64_t* base, int64_t stride, int n, uint32_t tag, float& sum) {
  uint64_t v[kMaxSplit];
  for (uint32_t it = 0;; ++it) {
    bool ready = true;
#pragma unroll
    for (int c = 0; c < kMaxSplit; ++c) {
      v[c] = c < n ? get_slot(base + c * stride) : (static_cast<uint64_t>(tag) << 32);
      ready = ready && slot_ready(v[c], tag);
    }
    if (ready) break;
    if (it >= kSpinLimit) return false;
    __builtin_amdgcn_s_sleep(1);
  }
  float s = 0.0f;
#pragma unroll
  for (int c = 0; c < kMaxSplit; ++c)
    if (c < n) s += slot_value(v[c]);
  sum = s;
  return true;
}

template <int TM>
__device__ void stage1(const DecodeParams& P, int wg, float* smem, uint32_t tag) {
  const int per_path = P.nkt * P.s1d;
  const int p = wg / per_path;
  const int rem = wg - p * per_path;
  const int kt = rem / P.s1d;
  const int c = rem - kt * P.s1d;
  const int T = P.T, r = P.r, d_in = P.d_in;
  const int k0 = kt * kKc;
  const int kcn = min(kKc, r - k0);
  const int nbt = nblocks32(d_in);
  const int b0 = c * P.bpw;
  const int b1 = min(nbt, b0 + P.bpw);
  const int kk = threadIdx.x & (kKc - 1);
  const int bs = threadIdx.x >> 4;
  const bool col_ok = kk < kcn;
  const PackedView Vv{static_cast<const uint32_t*>(P.V[p]), r, d_in >> 5, d_in & 31};
  float* a_s = smem;  // [T][kChunk][kAStride]

  float acc[TM];
#pragma unroll
  for (int t = 0; t < TM; ++t) acc[t] = 0.0f;

  uint32_t word = (col_ok && b0 + bs < b1) ? load_word(Vv, b0 + bs, k0 + kk) : 0u;
  for (int cb = b0; cb < b1; cb += kChunk) {
    const int nblk = min(kChunk, b1 - cb);
    // stage a = x (.) g_p for this chunk (zero beyond d_in)
    for (int e = threadIdx.x; e < T * nblk * 32; e += kThreads) {
      const int t = e / (nblk * 32);
      const int jj = e - t * nblk * 32;
      const int j = cb * 32 + jj;
      float v = 0.0f;
      if (j < d_in)
        v = load_as_f32(P.x, static_cast<int64_t>(t) * d_in + j, P.act_dt) * load_as_f32(P.g[p], j, P.sc_dt);
      a_s[(t * kChunk + (jj >> 5)) * kAStride + (jj & 31)] = v;
    }
    __syncthreads();
    const uint32_t cur = word;
    const int nb_next = cb + kChunk + bs;
    word = (col_ok && nb_next < b1) ? load_word(Vv, nb_next, k0 + kk) : 0u;
    if (col_ok && bs < nblk) {
      const float* arow = a_s + bs * kAStride;
#pragma unroll
      for (int bit = 0; bit < 32; ++bit) {
        const uint32_t m = (cur << (31 - bit)) & 0x80000000u;
#pragma unroll
        for (int t = 0; t < TM; ++t)
          if (t < T) acc[t] += flip(arow[t * kChunk * kAStride + bit], m);
      }
    }
    __syncthreads();
  }

  // fixed-order reduction over the 16 block groups
  float* red = smem;  // [bs][T][kKc]
#pragma unroll
  for (int t = 0; t < TM; ++t)
    if (t < T) red[(bs * T + t) * kKc + kk] = acc[t];
  __syncthreads();
  uint64_t* slots = P.partial + static_cast<int64_t>(p * P.s1d) * T * r;  // [s1d][T][r]
  const bool reducer = !P.direct && c == P.s1d - 1;
  for (int e = threadIdx.x; e < T * kcn; e += kThreads) {
    const int t = e / kcn;
    const int k = e - t * kcn;
    float s = 0.0f;
    for (int g = 0; g < kThreads / kKc; ++g) s += red[(g * T + t) * kKc + k];
    const int64_t off = static_cast<int64_t>(t) * r + k0 + k;
    if (!reducer) {
      put_slot(slots + static_cast<int64_t>(c) * T * r + off, tag, s);
    } else {
      // two-level mode: the highest run of this latent tile (it only waits for
      // lower block ids) adds the other runs' partials in ascending order
      float others = 0.0f;
      const bool ok = gather_sum(slots + off, static_cast<int64_t>(T) * r, P.s1d - 1, tag, others);
      if (!ok) atomic_store_relaxed(P.ctrl + kCtrlError, 1u);
      const float z = ok ? others + s : __builtin_nanf("");
      put_slot(P.wbuf + static_cast<int64_t>(p) * T * r + off, tag, z * load_as_f32(P.l[p], k0 + k, P.sc_dt));
    }
  }
}

template <int TM>
__device__ void stage2(const DecodeParams& P, int q, float* smem, uint32_t tag) {
  const int tid = threadIdx.x;
  const int kq_log2 = P.kq_log2;
  const int KQ = 1 << kq_log2;
  const int rows_per_pass = kThreads >> kq_log2;
  const int rl = tid >> kq_log2;
  const int kq = tid & (KQ - 1);
  const int T = P.T, r = P.r, d_out = P.d_out;
  const int nw = nblocks32(r);
  const int rpad = 33 * nw;
  const int i_base = q * P.rows2;
  const int passes = P.rows2 / rows_per_pass;
  const PackedView Uv[2] = {{static_cast<const uint32_t*>(P.U[0]), d_out, r >> 5, r & 31},
                            {static_cast<const uint32_t*>(P.U[1]), d_out, r >> 5, r & 31}};
  float* w_s = smem;  // [2][tch][rpad], index 33 * kb + bit

  // the first row's U words, before any wait
  uint32_t pre[2][kPrefetch];
  const int i_first = i_base + rl;
#pragma unroll
  for (int p = 0; p < 2; ++p)
#pragma unroll
    for (int e = 0; e < kPrefetch; ++e) {
      const int kb = kq + KQ * e;
      pre[p][e] = (i_first < d_out && kb < nw) ? load_word(Uv[p], kb, i_first) : 0u;
    }

  bool ok = true;
  for (int t0 = 0; t0 < T; t0 += P.tch) {
    const int tn = min(P.tch, T - t0);
    // l (.) z for this token chunk (waiting on the tagged slots), zero-padded to whole words
    const int per_p = tn * 32 * nw;
    for (int e = tid; e < 2 * per_p; e += kThreads) {
      const int p = e / per_p;
      const int rem = e - p * per_p;
      const int t = rem / (32 * nw);
      const int k = rem - t * 32 * nw;
      float v = 0.0f;
      if (k < r) {
        const int64_t off = static_cast<int64_t>(t0 + t) * r + k;
        if (P.direct) {
          float z = 0.0f;
          const bool got = gather_sum(P.partial + static_cast<int64_t>(p * P.s1d) * T * r + off,
                                      static_cast<int64_t>(T) * r, P.s1d, tag, z);
          ok = ok && got;
          v = z * load_as_f32(P.l[p], k, P.sc_dt);
        } else {
          float wv = 0.0f;
          const bool got = gather_sum(P.wbuf + static_cast<int64_t>(p) * T * r + off, 0, 1, tag, wv);
          ok = ok && got;
          v = wv;
        }
      }
      w_s[(p * P.tch + t) * rpad + k + (k >> 5)] = v;
    }
    __syncthreads();

    for (int m = 0; m < passes; ++m) {
      const int i = i_base + rl + rows_per_pass * m;
      float acc[2][TM];
#pragma unroll
      for (int p = 0; p < 2; ++p)
#pragma unroll
        for (int t = 0; t < TM; ++t) acc[p][t] = 0.0f;
      if (i < d_out) {
        for (int e = 0; kq + KQ * e < nw; ++e) {
          const int kb = kq + KQ * e;
#pragma unroll
          for (int p = 0; p < 2; ++p) {
            const uint32_t word = (m == 0 && t0 == 0 && e < kPrefetch) ? pre[p][e < kPrefetch ? e : 0]
                                                                      : load_word(Uv[p], kb, i);
            const float* wrow = w_s + p * P.tch * rpad + 33 * kb;
#pragma unroll
            for (int bit = 0; bit < 32; ++bit) {
              const uint32_t msk = (word << (31 - bit)) & 0x80000000u;
#pragma unroll
              for (int t = 0; t < TM; ++t)
                if (t < tn) acc[p][t] += flip(wrow[t * rpad + bit], msk);
            }
          }
        }
      }
#pragma unroll
      for (int p = 0; p < 2; ++p)
#pragma unroll
        for (int t = 0; t < TM; ++t) acc[p][t] = row_sum(acc[p][t], kq_log2);
      if (kq == 0 && i < d_out) {
        const float h0 = load_as_f32(P.h[0], i, P.sc_dt);
        const float h1 = load_as_f32(P.h[1], i, P.sc_dt);
#pragma unroll
        for (int t = 0; t < TM; ++t)
          if (t < tn) store_from_f32(P.y, static_cast<int64_t>(t0 + t) * d_out + i, P.act_dt,
                                     h0 * acc[0][t] + h1 * acc[1][t]);
      }
    }
    __syncthreads();
  }
  if (!ok) atomic_store_relaxed(P.ctrl + kCtrlError, 1u);

  // every workgroup of this call has read the tag once all stage-2 workgroups are done:
  // the last one advances it for the next call
  __syncthreads();
  if (tid == 0) {
    const uint32_t old = atomic_add_relaxed(P.ctrl + kCtrlDone, 1u);
    if (old == static_cast<uint32_t>(P.n_s2 - 1)) {
      atomic_store_relaxed(P.ctrl + kCtrlDone, 0u);
      atomic_store_relaxed(P.ctrl + kCtrlEpoch, tag);
    }
  }
}

template <int TM>
__global__ void __launch_bounds__(kThreads) decode_kernel(DecodeParams P) {
  extern __shared__ float smem[];
  // this call's tag: one more than the epoch the previous call left behind
  const uint32_t tag = atomic_load_relaxed(P.ctrl + kCtrlEpoch) + 1u;
  const int wg = blockIdx.x;
  if (wg < P.n_s1)
    stage1<TM>(P, wg, smem, tag);
  else
    stage2<TM>(P, wg - P.n_s1, smem, tag);
}

size_t align256(size_t b) { return (b + 255) / 256 * 256; }

size_t decode_smem_bytes(const DecodeGeom& g, int T, int r) {
  const size_t s1a = static_cast<size_t>(T) * kChunk * kAStride;
  const size_t s1b = static_cast<size_t>(kThreads / kKc) * T * kKc;
  const size_t s2 = static_cast<size_t>(2) * g.tch * 33 * nblocks32(r);
  size_t m = s1a > s1b ? s1a : s1b;
  if (s2 > m) m = s2;
  return 4 * m;
}

}  // namespace

DecodeGeom decode_geometry(int T, int d_in, int d_out, int r) {
  DecodeGeom g{};
  constexpr int kLdsFloats = 12288;  // 48 KB of dynamic LDS for the stage-2 l (.) z tile
  g.kc = kKc;
  g.nkt = (r + kKc - 1) / kKc;
  const int nbt = nblocks32(d_in);
  int s1d = nbt / 16;
  if (s1d > kMaxSplit) s1d = kMaxSplit;
  if (s1d < 1) s1d = 1;
  g.bpw = nbt > 0 ? (nbt + s1d - 1) / s1d : 1;
  g.s1d = nbt > 0 ? (nbt + g.bpw - 1) / g.bpw : 0;
  g.n_s1 = 2 * g.nkt * g.s1d;
  g.direct = static_cast<int64_t>(2) * g.s1d * T * r <= 4096;
  // lanes per output row: enough to keep each lane's share of the row's words small
  const int nw = nblocks32(r);
  int kq_log2 = 2;
  while (kq_log2 < 4 && (nw >> kq_log2) > 2) ++kq_log2;
  g.kq_log2 = kq_log2;
  const int rows_per_pass = kThreads >> kq_log2;
  const int n_min = (d_out + rows_per_pass - 1) / rows_per_pass;
  const int passes = (n_min + 127) / 128;  // at most ~128 waiting workgroups
  g.rows2 = rows_per_pass * (passes > 0 ? passes : 1);
  g.n_s2 = (d_out + g.rows2 - 1) / g.rows2;
  const int rpad = 33 * nw;
  int tch = rpad > 0 ? kLdsFloats / (2 * rpad) : T;
  if (tch > T) tch = T;
  if (tch < 1) tch = 1;
  g.tch = tch;
  // tagged 8-byte slots
  g.partial_off = kCtrlBytes;
  g.partial_floats = static_cast<size_t>(2) * g.s1d * T * r;
  g.wbuf_off = g.partial_off + align256(8 * g.partial_floats);
  g.wbuf_floats = g.direct ? 0 : static_cast<size_t>(2) * T * r;
  g.ws_bytes = g.wbuf_off + align256(8 * g.wbuf_floats);
  return g;
}

hipError_t launch_decode(const ForwardArgs& a, const DecodeGeom& g, hipStream_t stream) {
  DecodeParams P{};
  P.x = a.x;
  P.y = a.y;
  for (int p = 0; p < 2; ++p) {
    P.U[p] = a.U[p];
    P.V[p] = a.V[p];
    P.h[p] = a.h[p];
    P.g[p] = a.g[p];
    P.l[p] = a.l[p];
  }
  char* ws = static_cast<char*>(a.ws);
  P.ctrl = reinterpret_cast<uint32_t*>(ws);
  P.partial = reinterpret_cast<uint64_t*>(ws + g.partial_off);
  P.wbuf = reinterpret_cast<uint64_t*>(ws + g.wbuf_off);
  P.act_dt = a.act_dt;
  P.sc_dt = a.sc_dt;
  P.T = a.T;
  P.d_in = a.d_in;
  P.d_out = a.d_out;
  P.r = a.r;
  P.nkt = g.nkt;
  P.bpw = g.bpw;
  P.s1d = g.s1d;
  P.n_s1 = g.n_s1;
  P.kq_log2 = g.kq_log2;
  P.rows2 = g.rows2;
  P.n_s2 = g.n_s2;
  P.direct = g.direct;
  P.tch = g.tch;
  const size_t smem = decode_smem_bytes(g, a.T, a.r);
  const dim3 grid(g.n_s1 + g.n_s2);
  const int T = a.T;
  if (T <= 1)
    hipLaunchKernelGGL(decode_kernel<1>, grid, dim3(kThreads), smem, stream, P);
  else if (T <= 2)
    hipLaunchKernelGGL(decode_kernel<2>, grid, dim3(kThreads), smem, stream, P);
  else if (T <= 4)
    hipLaunchKernelGGL(decode_kernel<4>, grid, dim3(kThreads), smem, stream, P);
  else if (T <= 8)
    hipLaunchKernelGGL(decode_kernel<8>, grid, dim3(kThreads), smem, stream, P);
  else
    hipLaunchKernelGGL(decode_kernel<16>, grid, dim3(kThreads), smem, stream, P);
  return hipGetLastError();
}

}  // namespace lb
