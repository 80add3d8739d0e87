// Prefill kernels (large T): the two binary contractions of Proposition 1
// (Eq. proposition1) as matrix-core products on gfx950.
//
//   stage 1:  w_p[t][k] = l_p[k] * sum_j (x[t][j] g_p[j]) s(V_p)[j][k]   (M=T, N=r,     K=d_in)
//   stage 2:  y[t][i]   = sum_p h_p[i] sum_k w_p[t][k] s(U_p)[i][k]      (M=T, N=d_out, K=r)
//
// Both paths are handled inside each workgroup.  The A operand (x (.) g_p, or
// w_p) is formed in fp32 and written to LDS as NSPLIT bf16 terms whose sum
// reproduces it: two terms (16 significant bits) for bf16/f16 activations,
// three (the full fp32 significand) for fp32 activations.
// The B operand is the sign matrix: each packed 32-bit word (32 consecutive
// reduction indices of one output column, LB layout v1) is expanded in
// registers to bf16 +-1 by moving its bits into the bf16 sign positions, so
// one word is exactly one K=32 B fragment of v_mfma_f32_16x16x32_bf16.  The
// K order inside a fragment is chosen so that this expansion is one shift and
// one and-or per register: register v of lane group gq holds reduction indices
// (4 gq + v, 4 gq + v + 16); the A operand is staged in the same order.
// Waves split the N dimension (each owns SPW 16-column subtiles and expands
// its own B fragments once per K step) and share the A tile through LDS, so a
// B fragment feeds 4 M-subtiles x NSPLIT MFMAs.
//
// Stage 1 splits the d_in reduction over `ks` workgroups per output tile.  The
// first workgroup of a tile to finish stores its tile; the others wait for its
// flag and add theirs with agent-scope float atomics; the last resets the
// tile's counters.  (The first finisher never waits, and every waiter waits
// for a workgroup that is already running, so the scheme cannot deadlock.)
#include "lb_internal.h"

namespace lb {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kBM = 64;              // tokens per M-tile (4 MFMA M-subtiles)
constexpr int kRowBytes = 80;        // LDS row: 32 bf16 + 16 bytes of bank padding
constexpr int kTileBytes = kBM * kRowBytes;

struct PrefillParams {
  const void* x;
  void* y;
  const void* U[2];
  const void* V[2];
  const void* h[2];
  const void* g[2];
  const void* l[2];
  uint32_t* ctrl;
  float* wbuf;  // [2][T][r] fp32
  int act_dt, sc_dt;
  int T, d_in, d_out, r;
  int n_mt, nnt, ks, kb_per;
};

// Expand one packed word into the B fragment of lane group gq (bf16 +-1).
__device__ __forceinline__ bf16x8 expand_signs(uint32_t word, int gq) {
  const uint32_t w = word >> (4 * gq);
  u32x4 v;
  v[0] = ((w << 15) & 0x80008000u) | 0x3F803F80u;
  v[1] = ((w << 14) & 0x80008000u) | 0x3F803F80u;
  v[2] = ((w << 13) & 0x80008000u) | 0x3F803F80u;
  v[3] = ((w << 12) & 0x80008000u) | 0x3F803F80u;
  return __builtin_bit_cast(bf16x8, v);
}

// Split an fp32 value into NSPLIT bf16 terms (round-to-nearest-even each).
template <int NSPLIT>
__device__ __forceinline__ void split_bf16(float v, uint32_t (&out)[NSPLIT]) {
  float rem = v;
#pragma unroll
  for (int s = 0; s < NSPLIT; ++s) {
    const uint32_t b = f32_to_bf16_bits(rem);
    out[s] = b;
    rem = rem - bf16_bits_to_f32(b);
  }
}

// Stage 8 values of one (row, lane group) item into the LDS A tiles.
// vals[v] pairs with vals[v + 4] (reduction indices 4gq+v and 4gq+v+16).
template <int NSPLIT>
__device__ __forceinline__ void stage_item(char* tile_base, int row, int gq, const float (&vals)[8]) {
  uint32_t lo[4][NSPLIT], hi[4][NSPLIT];
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    split_bf16<NSPLIT>(vals[v], lo[v]);
    split_bf16<NSPLIT>(vals[v + 4], hi[v]);
  }
#pragma unroll
  for (int s = 0; s < NSPLIT; ++s) {
    u32x4 pk;
#pragma unroll
    for (int v = 0; v < 4; ++v) pk[v] = lo[v][s] | (hi[v][s] << 16);
    *reinterpret_cast<u32x4*>(tile_base + s * kTileBytes + row * kRowBytes + 16 * gq) = pk;
  }
}

__device__ __forceinline__ bf16x8 load_afrag(const char* tile, int row, int gq) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(tile + row * kRowBytes + 16 * gq));
}

// ---------------------------------------------------------------------------
// stage 1
// ---------------------------------------------------------------------------
template <int NSPLIT, int SPW>
__global__ void __launch_bounds__(512) prefill_stage1(PrefillParams P) {
  extern __shared__ __attribute__((aligned(16))) char lds[];  // [2 paths][NSPLIT][64 rows][80 B]
  const int nthreads = blockDim.x;
  const int nw = nthreads >> 6;
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int n16 = lane & 15;
  const int gq = lane >> 4;
  const int tiles = P.n_mt * P.nnt;
  const int tile = blockIdx.x % tiles;
  const int ksi = blockIdx.x / tiles;
  const int mt = tile % P.n_mt;
  const int nt = tile / P.n_mt;
  const int m0 = mt * kBM;
  const int bn = nw * SPW * 16;
  const int n0 = nt * bn;
  const int T = P.T, d_in = P.d_in, r = P.r;
  const int nkb = nblocks32(d_in);
  const int kb0 = ksi * P.kb_per;
  const int kb1 = min(nkb, kb0 + P.kb_per);
  const PackedView Vv[2] = {{static_cast<const uint32_t*>(P.V[0]), r, d_in >> 5, d_in & 31},
                            {static_cast<const uint32_t*>(P.V[1]), r, d_in >> 5, d_in & 31}};

  floatx4 acc[2][4][SPW];
#pragma unroll
  for (int p = 0; p < 2; ++p)
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
      for (int s = 0; s < SPW; ++s) acc[p][mi][s] = floatx4{0.f, 0.f, 0.f, 0.f};

  for (int kb = kb0; kb < kb1; ++kb) {
    // A tiles: a_p[t][j] = x[t][j] g_p[j] for j in this 32-block
    for (int item = threadIdx.x; item < 2 * kBM * 4; item += nthreads) {
      const int p = item / (kBM * 4);
      const int rem = item - p * kBM * 4;
      const int row = rem >> 2;
      const int q = rem & 3;
      const int t = m0 + row;
      float vals[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int j = 32 * kb + 4 * q + (e & 3) + (e >> 2) * 16;
        float v = 0.0f;
        if (t < T && j < d_in)
          v = load_as_f32(P.x, static_cast<int64_t>(t) * d_in + j, P.act_dt) * load_as_f32(P.g[p], j, P.sc_dt);
        vals[e] = v;
      }
      stage_item<NSPLIT>(lds + p * NSPLIT * kTileBytes, row, q, vals);
    }
    // B fragments of this wave's subtiles
    bf16x8 bfrag[2][SPW];
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
      for (int s = 0; s < SPW; ++s) {
        const int col = n0 + (wave * SPW + s) * 16 + n16;
        const uint32_t word = col < r ? load_word(Vv[p], kb, col) : 0u;
        bfrag[p][s] = expand_signs(word, gq);
      }
    __syncthreads();
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
      for (int mi = 0; mi < 4; ++mi)
#pragma unroll
        for (int sp = 0; sp < NSPLIT; ++sp) {
          const bf16x8 af = load_afrag(lds + (p * NSPLIT + sp) * kTileBytes, mi * 16 + n16, gq);
#pragma unroll
          for (int s = 0; s < SPW; ++s)
            acc[p][mi][s] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, bfrag[p][s], acc[p][mi][s], 0, 0, 0);
        }
    __syncthreads();
  }

  // epilogue: scale by l and publish into w (first finisher stores, others add)
  __shared__ uint32_t s_role;  // 0 = first (store), 1 = adder, 2 = adder whose wait expired
  uint32_t* tc = P.ctrl + kCtrlTiles + 3 * tile;
  if (P.ks > 1) {
    if (threadIdx.x == 0) {
      const uint32_t old = atomic_add_relaxed(tc, 1u);
      uint32_t role = old == 0 ? 0u : 1u;
      if (role == 1) {
        if (!spin_until_at_least(tc + 1, 1u)) {
          atomic_store_relaxed(P.ctrl + kCtrlError, 1u);
          role = 2;
        }
      }
      s_role = role;
    }
    if (threadIdx.x == 0 && s_role != 0) fence_acquire_agent();
  } else if (threadIdx.x == 0) {
    s_role = 0;
  }
  __syncthreads();
  const uint32_t role = s_role;
  if (role != 2) {
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
      for (int s = 0; s < SPW; ++s) {
        const int col = n0 + (wave * SPW + s) * 16 + n16;
        if (col >= r) continue;
        const float lk = load_as_f32(P.l[p], col, P.sc_dt);
#pragma unroll
        for (int mi = 0; mi < 4; ++mi)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int t = m0 + mi * 16 + 4 * gq + e;
            if (t >= T) continue;
            float* dst = P.wbuf + (static_cast<int64_t>(p) * T + t) * r + col;
            const float v = acc[p][mi][s][e] * lk;
            if (role == 0)
              *dst = v;
            else
              __hip_atomic_fetch_add(dst, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          }
      }
  }
  if (P.ks > 1) {
    __syncthreads();
    if (threadIdx.x == 0) {
      if (role == 0) atomic_store_release(tc + 1, 1u);
      const uint32_t fin = atomic_add_relaxed(tc + 2, 1u);
      if (fin == static_cast<uint32_t>(P.ks - 1)) {
        atomic_store_relaxed(tc, 0u);
        atomic_store_relaxed(tc + 1, 0u);
        atomic_store_relaxed(tc + 2, 0u);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// stage 2
// ---------------------------------------------------------------------------
template <int NSPLIT, int SPW>
__global__ void __launch_bounds__(256) prefill_stage2(PrefillParams P) {
  extern __shared__ __attribute__((aligned(16))) char lds[];
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int n16 = lane & 15;
  const int gq = lane >> 4;
  const int mt = blockIdx.x % P.n_mt;
  const int nt = blockIdx.x / P.n_mt;
  const int m0 = mt * kBM;
  constexpr int kBN = 4 * SPW * 16;
  const int n0 = nt * kBN;
  const int T = P.T, r = P.r, d_out = P.d_out;
  const int nkb = nblocks32(r);
  const PackedView Uv[2] = {{static_cast<const uint32_t*>(P.U[0]), d_out, r >> 5, r & 31},
                            {static_cast<const uint32_t*>(P.U[1]), d_out, r >> 5, r & 31}};

  floatx4 acc[2][4][SPW];
#pragma unroll
  for (int p = 0; p < 2; ++p)
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
      for (int s = 0; s < SPW; ++s) acc[p][mi][s] = floatx4{0.f, 0.f, 0.f, 0.f};

  for (int kb = 0; kb < nkb; ++kb) {
    for (int item = threadIdx.x; item < 2 * kBM * 4; item += 256) {
      const int p = item / (kBM * 4);
      const int rem = item - p * kBM * 4;
      const int row = rem >> 2;
      const int q = rem & 3;
      const int t = m0 + row;
      float vals[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int k = 32 * kb + 4 * q + (e & 3) + (e >> 2) * 16;
        vals[e] = (t < T && k < r) ? P.wbuf[(static_cast<int64_t>(p) * T + t) * r + k] : 0.0f;
      }
      stage_item<NSPLIT>(lds + p * NSPLIT * kTileBytes, row, q, vals);
    }
    bf16x8 bfrag[2][SPW];
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
      for (int s = 0; s < SPW; ++s) {
        const int col = n0 + (wave * SPW + s) * 16 + n16;
        const uint32_t word = col < d_out ? load_word(Uv[p], kb, col) : 0u;
        bfrag[p][s] = expand_signs(word, gq);
      }
    __syncthreads();
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
      for (int mi = 0; mi < 4; ++mi)
#pragma unroll
        for (int sp = 0; sp < NSPLIT; ++sp) {
          const bf16x8 af = load_afrag(lds + (p * NSPLIT + sp) * kTileBytes, mi * 16 + n16, gq);
#pragma unroll
          for (int s = 0; s < SPW; ++s)
            acc[p][mi][s] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, bfrag[p][s], acc[p][mi][s], 0, 0, 0);
        }
    __syncthreads();
  }

#pragma unroll
  for (int s = 0; s < SPW; ++s) {
    const int col = n0 + (wave * SPW + s) * 16 + n16;
    if (col >= d_out) continue;
    const float h0 = load_as_f32(P.h[0], col, P.sc_dt);
    const float h1 = load_as_f32(P.h[1], col, P.sc_dt);
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int t = m0 + mi * 16 + 4 * gq + e;
        if (t >= T) continue;
        store_from_f32(P.y, static_cast<int64_t>(t) * d_out + col, P.act_dt,
                       h0 * acc[0][mi][s][e] + h1 * acc[1][mi][s][e]);
      }
  }
}

template <int NSPLIT>
hipError_t launch_nsplit(const PrefillParams& P, const PrefillGeom& g, hipStream_t stream) {
  const size_t smem = static_cast<size_t>(2) * NSPLIT * kTileBytes;
  const dim3 grid1(g.n_mt * g.s1_nnt * g.ks);
  const dim3 block1(64 * g.s1_nw);
  switch (g.s1_spw) {
    case 1: hipLaunchKernelGGL((prefill_stage1<NSPLIT, 1>), grid1, block1, smem, stream, P); break;
    case 2: hipLaunchKernelGGL((prefill_stage1<NSPLIT, 2>), grid1, block1, smem, stream, P); break;
    case 3: hipLaunchKernelGGL((prefill_stage1<NSPLIT, 3>), grid1, block1, smem, stream, P); break;
    default: hipLaunchKernelGGL((prefill_stage1<NSPLIT, 4>), grid1, block1, smem, stream, P); break;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  PrefillParams P2 = P;
  P2.nnt = g.s2_nnt;
  const dim3 grid2(g.n_mt * g.s2_nnt);
  if (g.s2_spw == 1)
    hipLaunchKernelGGL((prefill_stage2<NSPLIT, 1>), grid2, dim3(256), smem, stream, P2);
  else
    hipLaunchKernelGGL((prefill_stage2<NSPLIT, 2>), grid2, dim3(256), smem, stream, P2);
  return hipGetLastError();
}

size_t align256(size_t b) { return (b + 255) / 256 * 256; }

}  // namespace

PrefillGeom prefill_geometry(int T, int d_in, int d_out, int r) {
  PrefillGeom g{};
  g.bm = kBM;
  g.n_mt = (T + kBM - 1) / kBM;
  const int n_sub = (r + 15) / 16;
  if (n_sub <= 8) {
    g.s1_spw = 1;
    g.s1_nw = n_sub > 0 ? n_sub : 1;
  } else if (n_sub <= 16) {
    g.s1_spw = 2;
    g.s1_nw = (n_sub + 1) / 2;
  } else if (n_sub <= 24) {
    g.s1_spw = 3;
    g.s1_nw = (n_sub + 2) / 3;
  } else {
    g.s1_spw = 4;
    g.s1_nw = (n_sub + 3) / 4;
    if (g.s1_nw > 8) g.s1_nw = 8;
  }
  g.s1_bn = g.s1_nw * g.s1_spw * 16;
  g.s1_nnt = (r + g.s1_bn - 1) / g.s1_bn;
  if (g.s1_nnt < 1) g.s1_nnt = 1;
  const int nkb = nblocks32(d_in);
  const int tiles = g.n_mt * g.s1_nnt;
  int ks = tiles > 0 ? (512 + tiles - 1) / tiles : 1;
  int max_ks = nkb / 4;
  if (max_ks < 1) max_ks = 1;
  if (ks > max_ks) ks = max_ks;
  if (ks < 1) ks = 1;
  if (tiles > kCtrlMaxTiles) ks = 1;  // per-tile counters only exist for kCtrlMaxTiles tiles
  int kb_per = nkb > 0 ? (nkb + ks - 1) / ks : 1;
  ks = nkb > 0 ? (nkb + kb_per - 1) / kb_per : 1;
  g.ks = ks;
  g.s2_spw = 2;
  g.s2_bn = 128;
  g.s2_nnt = (d_out + 127) / 128;
  if (static_cast<int64_t>(g.n_mt) * g.s2_nnt < 256) {
    g.s2_spw = 1;
    g.s2_bn = 64;
    g.s2_nnt = (d_out + 63) / 64;
  }
  g.wbuf_off = kCtrlBytes;
  g.wbuf_floats = static_cast<size_t>(2) * T * r;
  g.ws_bytes = g.wbuf_off + align256(4 * g.wbuf_floats);
  return g;
}

hipError_t launch_prefill(const ForwardArgs& a, const PrefillGeom& g, hipStream_t stream) {
  PrefillParams P{};
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
  P.wbuf = reinterpret_cast<float*>(ws + g.wbuf_off);
  P.act_dt = a.act_dt;
  P.sc_dt = a.sc_dt;
  P.T = a.T;
  P.d_in = a.d_in;
  P.d_out = a.d_out;
  P.r = a.r;
  P.n_mt = g.n_mt;
  P.nnt = g.s1_nnt;
  P.ks = g.ks;
  const int nkb = nblocks32(a.d_in);
  P.kb_per = g.ks > 0 ? (nkb + g.ks - 1) / g.ks : nkb;
  if (a.act_dt == kDtF32) return launch_nsplit<3>(P, g, stream);
  return launch_nsplit<2>(P, g, stream);
}

}  // namespace lb
