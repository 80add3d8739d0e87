// Device helpers shared by the single-launch forward kernels: tagged slots
// for the hand-off between workgroups, raw-bit loads that can all be issued
// before any is waited on, and conversions.
#pragma once
#include "lb_internal.h"

namespace lb {

// Polls of a tagged slot before a wait gives up and records an error.
constexpr uint32_t kSpinLimit = 1u << 19;

// ---------------------------------------------------------------------------
// tagged slots
// ---------------------------------------------------------------------------
__device__ __forceinline__ void put_slot(uint64_t* p, uint32_t tag, float v) {
  const uint64_t w = (static_cast<uint64_t>(tag) << 32) | __float_as_uint(v);
  __hip_atomic_store(p, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t get_slot(const uint64_t* p) {
  return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float slot_value(uint64_t w) { return __uint_as_float(static_cast<uint32_t>(w)); }
__device__ __forceinline__ bool slot_ready(uint64_t w, uint32_t tag) { return static_cast<uint32_t>(w >> 32) == tag; }

// Sum of n (<= MAXN) slots spaced `stride` apart, in ascending order, once
// every slot carries `tag` (used by the two-level reducers).
template <int MAXN>
__device__ __forceinline__ bool gather_sum(const uint64_t* base, int64_t stride, int n, uint32_t tag, float& sum) {
  uint64_t v[MAXN];
  bool ready = true;
#pragma unroll
  for (int c = 0; c < MAXN; ++c) {
    v[c] = c < n ? get_slot(base + c * stride) : (static_cast<uint64_t>(tag) << 32);
    ready = ready && slot_ready(v[c], tag);
  }
  for (uint32_t it = 0; !ready; ++it) {
    if (it >= kSpinLimit) return false;
    __builtin_amdgcn_s_sleep(1);
    ready = true;
#pragma unroll
    for (int c = 0; c < MAXN; ++c) {
      if (c < n && !slot_ready(v[c], tag)) v[c] = get_slot(base + c * stride);
      ready = ready && slot_ready(v[c], tag);
    }
  }
  float s = 0.0f;
#pragma unroll
  for (int c = 0; c < MAXN; ++c)
    if (c < n) s += slot_value(v[c]);
  sum = s;
  return true;
}

// ---------------------------------------------------------------------------
// loads and tables
// ---------------------------------------------------------------------------
// Element i of p (dtype DT) as fp32.  The dtype is a template parameter so
// that loads are straight-line code the compiler can batch.
template <int DT>
__device__ __forceinline__ float ld(const void* p, int64_t i) {
  if constexpr (DT == kDtF32) {
    return static_cast<const float*>(p)[i];
  } else {
    const uint32_t u = static_cast<const uint16_t*>(p)[i];
    return DT == kDtBF16 ? bf16_bits_to_f32(u) : f16_bits_to_f32(u);
  }
}

// Branch-free loads: the address is clamped to a valid element and the value
// selected afterwards, so no load sits inside a divergent branch (the compiler
// would wait for it before the branch rejoins, serialising the round trips).
template <int DT>
__device__ __forceinline__ float ld_or0(const void* p, int64_t i, bool ok) {
  const float v = ld<DT>(p, ok ? i : 0);
  return ok ? v : 0.0f;
}

// Raw bits of an element (fp32 bits, or a 16-bit value zero-extended), so that
// loads can be issued together and converted only after all are in flight.
template <int DT>
__device__ __forceinline__ uint32_t ld_bits(const void* p, int64_t i) {
  if constexpr (DT == kDtF32)
    return static_cast<const uint32_t*>(p)[i];
  else
    return static_cast<const uint16_t*>(p)[i];
}
template <int DT>
__device__ __forceinline__ float bits_to_f32(uint32_t u) {
  if constexpr (DT == kDtF32)
    return __uint_as_float(u);
  else if constexpr (DT == kDtBF16)
    return bf16_bits_to_f32(u);
  else
    return f16_bits_to_f32(u);
}

// Four consecutive elements p[i..i+3] as raw bits.  VEC: one 16-byte (fp32) or
// 8-byte (16-bit dtypes, two per dword) load, i a multiple of 4 and p aligned;
// otherwise four element loads, element e at p[i + e] if e < nvalid, else at
// p[0].  Element e is taken back with raw4_elem.
template <int DT, bool VEC>
__device__ __forceinline__ void ld4_bits(const void* p, int64_t i, int nvalid, uint32_t (&o)[4]) {
  if constexpr (VEC && DT == kDtF32) {
    const uint4 v = *reinterpret_cast<const uint4*>(static_cast<const uint32_t*>(p) + i);
    o[0] = v.x, o[1] = v.y, o[2] = v.z, o[3] = v.w;
  } else if constexpr (VEC) {
    const uint2 v = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(p) + i);
    o[0] = v.x, o[1] = v.y, o[2] = 0u, o[3] = 0u;
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = ld_bits<DT>(p, e < nvalid ? i + e : 0);
  }
}
template <int DT, bool VEC>
__device__ __forceinline__ float raw4_elem(const uint32_t (&o)[4], int e) {
  if constexpr (VEC && DT != kDtF32)
    return bits_to_f32<DT>((o[e >> 1] >> (16 * (e & 1))) & 0xffffu);
  else
    return bits_to_f32<DT>(o[e]);
}

// Make the compiler treat v as produced here: computations on v stay below
// this point (the hardware waits for v's load here, after the loads issued
// before it).
__device__ __forceinline__ void pin(uint32_t& v) { asm volatile("" : "+v"(v)); }
// The epoch word of the control block, read where it is written: the index
// goes through an opaque (and per-stage distinct) statement, so the compiler
// neither hoists the load out of its loop nor merges the two stages' loads
// into one before the branch (which would make a stage wait for it first).
template <int STAGE>
__device__ __forceinline__ uint32_t load_epoch(const uint32_t* ctrl) {
  int idx = kCtrlEpoch;
  asm volatile("; epoch load, stage %1" : "+s"(idx) : "i"(STAGE));
  return atomic_load_relaxed(ctrl + idx);
}

// Region A of a packed view (its full words) when it has any, else a word the
// kernel may read harmlessly (the control block): clamped full-word loads then
// stay in bounds even for a view whose whole buffer is a 2-byte tail plane.
__device__ __forceinline__ const uint32_t* full_words_or(const uint32_t* base, int nb, const uint32_t* fallback) {
  return nb > 0 ? base : fallback;
}

// Tail word of output row o of a packed view (0 if the view has none), as two
// 16-bit loads at clamped addresses; combined by tail_word after pinning.
__device__ __forceinline__ void ld_tail_bits(const uint32_t* base, int nb, int n_out, int tailw, int o, bool ok,
                                             uint32_t& lo, uint32_t& hi) {
  const uint16_t* h = reinterpret_cast<const uint16_t*>(base);
  const int64_t plane = static_cast<int64_t>(2) * nb * n_out;  // in 16-bit units
  const bool has = ok && tailw != 0;
  const int64_t e = tailw <= 16 ? o : static_cast<int64_t>(2) * o;
  lo = h[has ? plane + e : 0];
  hi = h[has && tailw > 16 ? plane + e + 1 : 0];
}
__device__ __forceinline__ uint32_t tail_word(uint32_t lo, uint32_t hi, int tailw) {
  return tailw > 16 ? (lo | (hi << 16)) : lo;
}

template <int DT>
__device__ __forceinline__ void st(void* p, int64_t i, float v) {
  if constexpr (DT == kDtF32) {
    static_cast<float*>(p)[i] = v;
  } else if constexpr (DT == kDtBF16) {
    static_cast<uint16_t*>(p)[i] = static_cast<uint16_t>(f32_to_bf16_bits(v));
  } else {
    // the fp32 value is formed first: without the pin the compiler may fold
    // the multiply that produced it into a mixed-precision fma that rounds
    // the exact product to f16 (a different result on fp32 ties)
    asm volatile("" : "+v"(v));
    static_cast<__half*>(p)[i] = __float2half_rn(v);
  }
}

// ---------------------------------------------------------------------------
// buffer loads: 32-bit byte offsets into a buffer of known size; a read past
// the end returns zero, so absent rows, columns and blocks need no clamping
// ---------------------------------------------------------------------------
typedef __amdgpu_buffer_rsrc_t rsrc_t;
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr uint32_t kOob = 0x7ffffff0u;  // a buffer offset past every buffer: loads return 0

__device__ __forceinline__ rsrc_t make_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), static_cast<short>(0), static_cast<int>(bytes),
                                           0x00020000);
}
// A buffer descriptor from a pointer and size the compiler cannot prove
// uniform (computed from block indices through 64-bit arithmetic): read back
// from the first lane, so the descriptor lives in scalar registers and the
// accesses need no per-lane descriptor loop.
__device__ __forceinline__ rsrc_t make_rsrc_uniform(const void* p, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(a));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(a >> 32));
  return make_rsrc(reinterpret_cast<const void*>((static_cast<uint64_t>(hi) << 32) | lo),
                   __builtin_amdgcn_readfirstlane(bytes));
}
// raw bits of element i (dtype DT) of a buffer; 0 past its end
template <int DT>
__device__ __forceinline__ uint32_t bload(rsrc_t r, uint32_t i, bool valid = true) {
  if constexpr (DT == kDtF32)
    return __builtin_amdgcn_raw_buffer_load_b32(r, valid ? i * 4u : kOob, 0, 0);
  else
    return static_cast<uint16_t>(__builtin_amdgcn_raw_buffer_load_b16(r, valid ? i * 2u : kOob, 0, 0));
}
// raw bits of elements i..i+3: one 16- or 8-byte load (VEC: i a multiple of 4,
// buffer aligned), else four element loads; taken back with raw4_elem
template <int DT, bool VEC>
__device__ __forceinline__ void bload4(rsrc_t r, uint32_t i, bool valid, uint32_t (&o)[4]) {
  if constexpr (VEC && DT == kDtF32) {
    const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, valid ? i * 4u : kOob, 0, 0);
    o[0] = v[0], o[1] = v[1], o[2] = v[2], o[3] = v[3];
  } else if constexpr (VEC) {
    const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(r, valid ? i * 2u : kOob, 0, 0);
    o[0] = v[0], o[1] = v[1], o[2] = 0u, o[3] = 0u;
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = bload<DT>(r, i + e, valid);
  }
}
// 16-bit element v of a bload4 group, raw bits
template <bool VEC>
__device__ __forceinline__ uint32_t raw16(const uint32_t (&o)[4], int v) {
  return VEC ? (o[v >> 1] >> (16 * (v & 1))) & 0xffffu : o[v];
}

// q = n / d for n < 2^20, 2 <= d < 2^12, with m = ceil(2^32 / d); m = 0 stands
// for d = 1
__device__ __forceinline__ uint32_t fast_div(uint32_t n, uint32_t m) { return m == 0 ? n : __umulhi(n, m); }

// ---------------------------------------------------------------------------
// matrix-core operands (v_mfma_f32_16x16x32_bf16).  Fragment layout: lane l
// holds row l % 16 of A (column l % 16 of B) at 8 reduction slots; register v
// of lane group gq = l / 16 holds the pair of reduction indices
// (4 gq + v, 4 gq + v + 16) of a 32-wide block (low, high half), the same
// relabelling of K for both operands, which puts bit 4 gq + v of a packed word
// (LB layout v1) at the bf16 sign of the low half and bit 4 gq + v + 16 at the
// high half with one shift and one mask.  The result lane holds rows
// 4 gq + e (e < 4) of column l % 16.
// ---------------------------------------------------------------------------
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

// exact bf16 terms of a value stored in dtype DT
template <int DT>
__host__ __device__ constexpr int nterms() {
  return DT == kDtF32 ? 3 : (DT == kDtF16 ? 2 : 1);
}
// v as N bf16 terms (bit patterns), each the leading 8 significant bits of
// what the previous terms left: exact when v has at most 8N significant bits
// (a bf16, f16 or fp32 value with N = its nterms)
template <int N>
__device__ __forceinline__ void split_exact(float v, uint32_t (&o)[N]) {
  float rem = v;
#pragma unroll
  for (int s = 0; s < N; ++s) {
    const uint32_t b = __float_as_uint(rem) & 0xffff0000u;
    o[s] = b >> 16;
    rem = rem - __uint_as_float(b);
  }
}
// v (any fp32) as N bf16 terms: leading bits, the last term rounded to nearest
template <int N>
__device__ __forceinline__ void split_round(float v, uint32_t (&o)[N]) {
  float rem = v;
#pragma unroll
  for (int s = 0; s < N - 1; ++s) {
    const uint32_t b = __float_as_uint(rem) & 0xffff0000u;
    o[s] = b >> 16;
    rem = rem - __uint_as_float(b);
  }
  o[N - 1] = f32_to_bf16_bits(rem);
}

__device__ __forceinline__ floatx4 mfma(u32x4 a, u32x4 b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0,
                                                 0, 0);
}

// signs of a packed word (this lane group's nibbles) on bf16 term pairs t[v]:
// the low half takes the sign of bit 4gq+v, the high half of bit 4gq+v+16
__device__ __forceinline__ u32x4 sign_terms(uint32_t word, int gq, const uint32_t (&t)[4]) {
  const uint32_t ws = word >> (4 * gq);
  u32x4 a;
#pragma unroll
  for (int v = 0; v < 4; ++v) a[v] = ((ws << (15 - v)) & 0x80008000u) ^ t[v];
  return a;
}

}  // namespace lb
