// Prefill kernels (long token runs): the two binary contractions of
// Proposition 1 (Eq. proposition1) for both paths (Sec. 3.3, Eq.
// final_weight_approx_res) as matrix-core products on gfx950, in three
// launches.
//
//   P1:  z_p[t][k] = sum_j (s(V_p)[j][k] g_p[j]) x[t][j]           (M = latents, N = tokens, K = d_in)
//   P1b: w_p[t][k] = l_p[k] z_p[t][k], cut into bf16 terms
//   P2:  y[t][i]   = sum_p h_p[i] sum_k s(U_p)[i][k] w_p[t][k]    (M = outputs, N = tokens, K = r)
//
// P1.  The A operand is the sign of V_p XORed into the sign bits of exact
// bf16 terms of g_p (1 term for bf16, 2 for f16, 3 for fp32 scales), the B
// operand the exact bf16 terms of x (1, 2 or 3 by the activation dtype), so
// every product is exact and the matrix cores accumulate in fp32.  A
// workgroup owns 64 tokens (each A fragment feeds 4 token subtiles: the
// VALU work of cutting it stays below the matrix-core work) and a tile of up
// to 6 (path, 32-latent block) pairs -- all latents of both paths for r <= 96
// -- so x is read once per latent tile.  Its range of d_in is split over `ks`
// workgroups (about 256 workgroups in all); its 4 waves take interleaved
// 32-input steps with the next step's loads in flight, the g terms of its
// range are cut once into LDS, and the 4 waves are summed in LDS in a fixed
// order into the workgroup's partial sums.
// P1b.  Sums the ks partials in ascending order, scales by l and stores w as
// NW bf16 terms (2 for bf16/f16 outputs: 16 significant bits; 3 for fp32
// outputs: all 24), already laid out as B fragments of P2.  The launch
// boundaries order P1 -> P1b -> P2: no workgroup waits for another.
// P2.  A = the U signs as bf16 +-1 (exact), B = the w terms.  A workgroup owns
// 256 outputs x 64 tokens (a wave 64 x 64, 16 accumulator tiles per path).
// Per path it loads the w fragments, U words and row scales it needs straight
// into LDS (global-to-LDS loads, no registers), then runs its products from
// LDS; registers hold the accumulators only, so two workgroups share a CU and
// one's loads and stores overlap the other's products.  Both paths accumulate
// separately and y = h_0 acc_0 + h_1 acc_1 is rounded once.
//
// At 2048 tokens the matrix cores, not HBM, bound P1 and P2: each does
// 2 * T * 2r * d fp32-accumulated multiply-adds times the number of term pairs
// (2 for bf16 x with f16 scales in P1, 2 w terms in P2).
#include <atomic>

#include "device_common.h"

namespace lb {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr int kTok1 = 64;          // P1: tokens per workgroup (4 subtiles)
constexpr int kTn1 = 4;
constexpr int kMaxPairs = 6;       // P1: (path, latent block) pairs per tile
constexpr int kMaxKbPer = 128;     // P1: 32-input steps per workgroup (g terms held in LDS)
constexpr int kRedPairs = 2;       // P1: pairs summed across the waves per LDS round
constexpr int kTok2 = 64;          // P2: tokens per workgroup (4 subtiles)
constexpr int kTn2 = 4;
constexpr int kIm2 = 4;            // P2: 16-output subtiles per wave
constexpr int kOut2 = kWaves * kIm2 * 16;  // P2: outputs per workgroup
constexpr int kRing = 2;           // P1: steps of loads in flight per wave
constexpr int kMaxKbc = 8;         // P2: 32-latent blocks of one path staged per round (LDS: kMaxKbc * NW * 4 KB)
constexpr int kPbufItem = 8;       // P1 partial floats per (pair, token, lane group)
constexpr int kPbufPair = kTok1 * 4 * kPbufItem;

struct PrefillParams {
  const void* x;
  void* y;
  const void* U[2];
  const void* V[2];
  const void* h[2];
  const void* g[2];
  const void* l[2];
  float* pbuf;      // P1: [ks][tile][npt][64 tokens][4 lane groups][8] partial sums
  uint32_t* wterm;  // [2][NW][nkb][T][4 lane groups][4] w terms as B fragments
  int T, d_in, d_out, r;
  int nkb;          // 32-latent blocks per path
  int n_tt, n_lt;   // P1 token tiles, latent tiles
  int npt;          // P1 pairs per latent tile
  int ks, kb_per;   // P1 splits of d_in and 32-input steps per split
  int n_ot;         // P2 output tiles
  int kbc;          // P2 32-latent blocks staged in LDS per round
  int xvec, hvec, yvec;  // aligned vector access allowed for x / h / y
  uint32_t v_bytes, u_bytes, g_bytes, h_bytes, l_bytes, wt_bytes;
};

// Raw bits of x[row][j0 + v] and x[row][j0 + 16 + v] (v < 4): the inputs of one
// lane's slots in a 32-input step, always in the vector layout of bload4
// (16-bit elements two to a dword), whichever load form read them.
template <int ACT>
__device__ __forceinline__ void load_x8(rsrc_t xr, uint32_t e0, bool vec, uint32_t (&lo)[4], uint32_t (&hi)[4]) {
  if (vec) {
    bload4<ACT, true>(xr, e0, true, lo);
    bload4<ACT, true>(xr, e0 + 16, true, hi);
  } else {
    uint32_t a[4], b[4];
    bload4<ACT, false>(xr, e0, true, a);
    bload4<ACT, false>(xr, e0 + 16, true, b);
    if constexpr (ACT == kDtF32) {
#pragma unroll
      for (int v = 0; v < 4; ++v) lo[v] = a[v], hi[v] = b[v];
    } else {
      lo[0] = a[0] | (a[1] << 16), lo[1] = a[2] | (a[3] << 16), lo[2] = lo[3] = 0u;
      hi[0] = b[0] | (b[1] << 16), hi[1] = b[2] | (b[3] << 16), hi[2] = hi[3] = 0u;
    }
  }
}

// B fragment(s) of x: E exact bf16 terms.  MASK (the step that holds the end
// of d_in): inputs at or past jmax are zero (x past d_in is the next row).
template <int ACT, int E, bool MASK>
__device__ __forceinline__ void x_frag(const uint32_t (&lo)[4], const uint32_t (&hi)[4], int j0, int jmax,
                                       u32x4 (&B)[E]) {
  if constexpr (E == 1) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const uint32_t a = (!MASK || j0 + v < jmax) ? raw16<true>(lo, v) : 0u;
      const uint32_t b = (!MASK || j0 + 16 + v < jmax) ? raw16<true>(hi, v) : 0u;
      B[0][v] = a | (b << 16);
    }
  } else {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      uint32_t a[E], b[E];
      split_exact<E>((!MASK || j0 + v < jmax) ? raw4_elem<ACT, true>(lo, v) : 0.0f, a);
      split_exact<E>((!MASK || j0 + 16 + v < jmax) ? raw4_elem<ACT, true>(hi, v) : 0.0f, b);
#pragma unroll
      for (int e = 0; e < E; ++e) B[e][v] = a[e] | (b[e] << 16);
    }
  }
}

// Packed sign word of V_p for latent k at 32-input step kb (0 when k >= r).
__device__ __forceinline__ uint32_t v_word(rsrc_t vr, int kb, int k, int r, int nbv, int tailv, bool kok) {
  if (kb < nbv) return __builtin_amdgcn_raw_buffer_load_b32(vr, kok ? static_cast<uint32_t>(kb * r + k) * 4u : kOob, 0, 0);
  const uint32_t off = 4u * nbv * r + (tailv <= 16 ? 2u : 4u) * k;
  const uint32_t lo = __builtin_amdgcn_raw_buffer_load_b16(vr, kok ? off : kOob, 0, 0);
  const uint32_t hi = __builtin_amdgcn_raw_buffer_load_b16(vr, kok && tailv > 16 ? off + 2 : kOob, 0, 0);
  return (lo & 0xffffu) | (hi << 16);
}

// ---------------------------------------------------------------------------
// P1
// ---------------------------------------------------------------------------
template <int NPT, int ACT, int SC>
__global__ void __launch_bounds__(kThreads, 1) prefill_p1(PrefillParams P) {
  constexpr int G = nterms<SC>(), E = nterms<ACT>();
  extern __shared__ __attribute__((aligned(16))) char lds[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (scalar)
  const int n16 = lane & 15, gq = lane >> 4;
  const int tiles = P.n_tt * P.n_lt;
  const int ksi = blockIdx.x / tiles;
  const int tile = blockIdx.x - ksi * tiles;
  const int lt = tile / P.n_tt;
  const int tt = tile - lt * P.n_tt;
  const int T = P.T, d_in = P.d_in, r = P.r, nkb = P.nkb;
  const int t0 = tt * kTok1;
  const int q0 = lt * NPT;
  const int nq = min(NPT, 2 * nkb - q0);  // pairs of this tile
  const int nbv = d_in >> 5, tailv = d_in & 31, nbt = nblocks32(d_in);
  const int kbs = ksi * P.kb_per, kbe = min(nbt, kbs + P.kb_per), nk = kbe - kbs;
  const bool vec = P.xvec != 0;

  u32x4* gt = reinterpret_cast<u32x4*>(lds);  // g terms: [2][nk][4 lane groups][G]
  // x of this tile's tokens (a buffer from the tile's first row: reads past the
  // last token return zero)
  const int ex = ACT == kDtF32 ? 4 : 2;
  const int rows = min(kTok1, T - t0);
  const rsrc_t xr = make_rsrc_uniform(static_cast<const char*>(P.x) + static_cast<int64_t>(t0) * d_in * ex,
                                      static_cast<uint32_t>(rows * d_in * ex));
  const rsrc_t vr0 = make_rsrc(P.V[0], P.v_bytes), vr1 = make_rsrc(P.V[1], P.v_bytes);

  floatx4 acc[NPT][2][kTn1];
#pragma unroll
  for (int i = 0; i < NPT; ++i)
#pragma unroll
    for (int sb = 0; sb < 2; ++sb)
#pragma unroll
      for (int tn = 0; tn < kTn1; ++tn) acc[i][sb][tn] = floatx4{0.f, 0.f, 0.f, 0.f};

  // step loads: x slots of both token subtiles, the packed words of every pair
  // (pairs past the tile read zero words; their sums are never finalised)
  struct StepLoads {
    uint32_t xl[kTn1][4], xh[kTn1][4];
    uint32_t w[NPT][2];
  };
  // (a step past the range, valid == false, reads past every buffer: zeros,
  // with the same instructions, so the prefetch needs no branch)
  auto issue = [&](int kb, bool tail, bool valid, StepLoads& L) {
    const int j0 = 32 * kb + 4 * gq;
    const uint32_t xoff = valid ? static_cast<uint32_t>(n16 * d_in + j0) : (kOob >> 2);
#pragma unroll
    for (int tn = 0; tn < kTn1; ++tn)
      load_x8<ACT>(xr, xoff + (valid ? 16 * tn * d_in : 0), vec, L.xl[tn], L.xh[tn]);
#pragma unroll
    for (int i = 0; i < NPT; ++i) {
      const int q = q0 + i;
      const bool p1 = q >= nkb;
      const int kbl = q - (p1 ? nkb : 0);
#pragma unroll
      for (int sb = 0; sb < 2; ++sb) {
        const int k = 32 * kbl + 16 * sb + n16;
        const bool kok = valid && i < nq && k < r;
        if (!tail) {
          L.w[i][sb] = __builtin_amdgcn_raw_buffer_load_b32(p1 ? vr1 : vr0,
                                                            kok ? static_cast<uint32_t>(kb * r + k) * 4u : kOob, 0, 0);
        } else {
          // the tail block's word comes from the tail plane (16- or 32-bit entries)
          const uint32_t off = 4u * nbv * r + (tailv <= 16 ? 2u : 4u) * k;
          const uint32_t lo = __builtin_amdgcn_raw_buffer_load_b16(p1 ? vr1 : vr0, kok ? off : kOob, 0, 0);
          const uint32_t hi = __builtin_amdgcn_raw_buffer_load_b16(p1 ? vr1 : vr0, kok && tailv > 16 ? off + 2 : kOob, 0, 0);
          L.w[i][sb] = (lo & 0xffffu) | (hi << 16);
        }
      }
    }
  };
  auto compute = [&](int kb, bool tail, const StepLoads& L) {
    u32x4 B[kTn1][E];
#pragma unroll
    for (int tn = 0; tn < kTn1; ++tn) {
      if (tail)
        x_frag<ACT, E, true>(L.xl[tn], L.xh[tn], 32 * kb + 4 * gq, d_in, B[tn]);
      else
        x_frag<ACT, E, false>(L.xl[tn], L.xh[tn], 32 * kb + 4 * gq, d_in, B[tn]);
    }
#pragma unroll
    for (int i = 0; i < NPT; ++i) {
      const int p = q0 + i >= nkb ? 1 : 0;
      const u32x4* gp = gt + ((p * nk + (kb - kbs)) * 4 + gq) * G;
      u32x4 gv[G];
#pragma unroll
      for (int s = 0; s < G; ++s) gv[s] = gp[s];
#pragma unroll
      for (int sb = 0; sb < 2; ++sb) {
        const uint32_t ws = L.w[i][sb] >> (4 * gq);
        u32x4 msk;
#pragma unroll
        for (int v = 0; v < 4; ++v) msk[v] = (ws << (15 - v)) & 0x80008000u;
#pragma unroll
        for (int s = 0; s < G; ++s) {
          const u32x4 A = msk ^ gv[s];
#pragma unroll
          for (int tn = 0; tn < kTn1; ++tn)
#pragma unroll
            for (int e = 0; e < E; ++e) acc[i][sb][tn] = mfma(A, B[tn][e], acc[i][sb][tn]);
        }
      }
    }
  };
  // this wave's full steps kb(n) = kbs + wave + kWaves n, n < ns, through a
  // ring of kRing steps of loads in flight (ring slot n % kRing; a slot past
  // the last step reads zeros, with the same instructions); then the tail step
  const int kfe = min(kbe, nbv);
  const int kw0 = kbs + wave;
  const int ns = kw0 < kfe ? (kfe - kw0 + kWaves - 1) / kWaves : 0;
  StepLoads ring[kRing];
#pragma unroll
  for (int d2 = 0; d2 < kRing; ++d2) issue(kw0 + kWaves * d2, false, d2 < ns, ring[d2]);
  // g terms of both paths for this workgroup's steps, as A-operand register
  // pairs: gt[p][step][lane group][term] = 4 dwords
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    const rsrc_t gr = make_rsrc(p ? P.g[1] : P.g[0], P.g_bytes);
    for (int it = tid; it < nk * 4; it += kThreads) {
      const int kbl = it >> 2, g4 = it & 3;
      const uint32_t j0 = 32 * (kbs + kbl) + 4 * g4;
      uint32_t tl[4][G], th[4][G];
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        split_exact<G>(bits_to_f32<SC>(bload<SC>(gr, j0 + v)), tl[v]);
        split_exact<G>(bits_to_f32<SC>(bload<SC>(gr, j0 + 16 + v)), th[v]);
      }
#pragma unroll
      for (int s = 0; s < G; ++s) {
        u32x4 d;
#pragma unroll
        for (int v = 0; v < 4; ++v) d[v] = tl[v][s] | (th[v][s] << 16);
        gt[((p * nk + kbl) * 4 + g4) * G + s] = d;
      }
    }
  }
  __syncthreads();

  // whole rounds of the ring (every product unconditional: conditional
  // products would make the compiler copy accumulators), then the remainder
  int n0 = 0;
  for (; n0 + kRing <= ns; n0 += kRing) {
#pragma unroll
    for (int d2 = 0; d2 < kRing; ++d2) {
      const int n = n0 + d2;
      asm volatile("" ::: "memory");  // keep the ring's loads where they are issued
      compute(kw0 + kWaves * n, false, ring[d2]);
      issue(kw0 + kWaves * (n + kRing), false, n + kRing < ns, ring[d2]);
    }
  }
  static_assert(kRing == 2, "the remainder below handles one step");
  if (n0 < ns) compute(kw0 + kWaves * n0, false, ring[0]);
  if (tailv != 0 && nbv >= kbs && nbv < kbe && (nbv - kbs) % kWaves == wave) {
    StepLoads tl;
    issue(nbv, true, true, tl);
    compute(nbv, true, tl);
  }
  __syncthreads();  // the g terms are dead: the LDS is reused below

  // fixed-order sum over the 4 waves, kRedPairs pairs at a time, into this
  // workgroup's partial: pbuf[ks][tile][pair][token][lane group][8]
  float* red = reinterpret_cast<float*>(lds);  // [4 waves][kRedPairs][kTn1][64 lanes][8]
  float* part = P.pbuf + (static_cast<int64_t>(ksi) * tiles + tile) * NPT * kPbufPair;
#pragma unroll
  for (int c0 = 0; c0 < NPT; c0 += kRedPairs) {
#pragma unroll
    for (int il = 0; il < kRedPairs; ++il) {
      if (c0 + il < NPT) {
#pragma unroll
        for (int tn = 0; tn < kTn1; ++tn) {
          floatx4* d = reinterpret_cast<floatx4*>(red + (((wave * kRedPairs + il) * kTn1 + tn) * 64 + lane) * 8);
          d[0] = acc[c0 + il][0][tn];
          d[1] = acc[c0 + il][1][tn];
        }
      }
    }
    __syncthreads();
    for (int it = tid; it < kRedPairs * kTn1 * 64; it += kThreads) {
      const int il = it / (kTn1 * 64);
      const int tn = (it >> 6) % kTn1;
      const int ln = it & 63;
      if (c0 + il >= NPT) continue;
      floatx4 s0[kWaves], s1[kWaves];
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const floatx4* sp = reinterpret_cast<const floatx4*>(red + (((w * kRedPairs + il) * kTn1 + tn) * 64 + ln) * 8);
        s0[w] = sp[0];
        s1[w] = sp[1];
      }
      const int t = 16 * tn + (ln & 15), g4 = ln >> 4;
      floatx4* dst = reinterpret_cast<floatx4*>(part + (c0 + il) * kPbufPair + (t * 4 + g4) * kPbufItem);
      dst[0] = (s0[0] + s0[1]) + (s0[2] + s0[3]);
      dst[1] = (s1[0] + s1[1]) + (s1[2] + s1[3]);
    }
    __syncthreads();
  }

}

// ---------------------------------------------------------------------------
// P1b: w = l (.) (sum of the ks partials, ascending) as NW bf16 terms in P2's
// B-fragment layout wterm[p][term][kbl][t][lane group]; one thread per
// (token, pair, lane group)
// ---------------------------------------------------------------------------
template <int ACT, int SC>
__global__ void __launch_bounds__(kThreads) prefill_p1b(PrefillParams P) {
  constexpr int NW = ACT == kDtF32 ? 3 : 2;
  const int NPT = P.npt;
  const int nq2 = 2 * P.nkb;
  const int item = blockIdx.x * kThreads + threadIdx.x;
  if (item >= P.T * nq2 * 4) return;
  const int g4 = item & 3;
  const int rest = item >> 2;
  const int t = rest / nq2;
  const int q = rest - t * nq2;
  const int tile = (q / NPT) * P.n_tt + t / kTok1;
  const int tiles = P.n_tt * P.n_lt;
  const float* src = P.pbuf + (static_cast<int64_t>(tile) * NPT + q % NPT) * kPbufPair + ((t % kTok1) * 4 + g4) * kPbufItem;
  const int64_t kstride = static_cast<int64_t>(tiles) * NPT * kPbufPair;
  floatx4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = s0;
#pragma unroll 8
  for (int k2 = 0; k2 < P.ks; ++k2) {
    const floatx4* sp = reinterpret_cast<const floatx4*>(src + k2 * kstride);
    s0 += sp[0];
    s1 += sp[1];
  }
  const int p = q >= P.nkb ? 1 : 0;
  const int kbl = q - p * P.nkb;
  const int r = P.r;
  const rsrc_t lr = make_rsrc(p ? P.l[1] : P.l[0], P.l_bytes);
  uint32_t lo[NW][4], hi[NW][4];
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int k = 32 * kbl + 4 * g4 + v;
    const float w0 = s0[v] * bits_to_f32<SC>(bload<SC>(lr, k, k < r));
    const float w1 = s1[v] * bits_to_f32<SC>(bload<SC>(lr, k + 16, k + 16 < r));
    uint32_t a[NW], b[NW];
    split_round<NW>(k < r ? w0 : 0.0f, a);
    split_round<NW>(k + 16 < r ? w1 : 0.0f, b);
#pragma unroll
    for (int e = 0; e < NW; ++e) lo[e][v] = a[e], hi[e][v] = b[e];
  }
#pragma unroll
  for (int e = 0; e < NW; ++e) {
    u32x4 d;
#pragma unroll
    for (int v = 0; v < 4; ++v) d[v] = lo[e][v] | (hi[e][v] << 16);
    reinterpret_cast<u32x4*>(P.wterm)[((static_cast<int64_t>(p * NW + e) * P.nkb + kbl) * P.T + t) * 4 + g4] = d;
  }
}

// ---------------------------------------------------------------------------
// P2
// ---------------------------------------------------------------------------
// LDS of P2: w fragments [kbc][kTn2][NW][64 lanes] x 16 B and U words
// [4 waves][kbc][64] x 4 B
__host__ __device__ constexpr size_t p2_b_bytes(int kbc, int nw) { return static_cast<size_t>(kbc) * kTn2 * nw * 64 * 16; }
__host__ __device__ constexpr size_t p2_lds_bytes(int kbc, int nw) {
  return p2_b_bytes(kbc, nw) + static_cast<size_t>(kWaves) * kbc * 64 * 4;
}

typedef __attribute__((address_space(3))) void* lds_ptr;

template <int ACT, int SC>
__global__ void __launch_bounds__(kThreads, 2) prefill_p2(PrefillParams P) {
  constexpr int NW = ACT == kDtF32 ? 3 : 2;
  extern __shared__ __attribute__((aligned(16))) char lds[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (scalar)
  const int n16 = lane & 15, gq = lane >> 4;
  const int ot = blockIdx.x % P.n_ot;
  const int tt = blockIdx.x / P.n_ot;
  const int T = P.T, d_out = P.d_out, r = P.r, nkb = P.nkb, kbc = P.kbc;
  const int i0 = ot * kOut2 + wave * (kIm2 * 16);  // this wave's 64 outputs i0 .. i0 + 63
  const int t0 = tt * kTok2;
  const int nbu = r >> 5, tailu = r & 31;
  const rsrc_t wr = make_rsrc(P.wterm, P.wt_bytes);
  const rsrc_t ur[2] = {make_rsrc(P.U[0], P.u_bytes), make_rsrc(P.U[1], P.u_bytes)};  // compile-time path index
  const rsrc_t hr[2] = {make_rsrc(P.h[0], P.h_bytes), make_rsrc(P.h[1], P.h_bytes)};
  char* bl = lds;                                              // w fragments
  char* ul = bl + p2_b_bytes(kbc, NW);                         // U words
  const bool iok = i0 + lane < d_out;

  // row scales of this lane's outputs i0 + 16 im + 4 gq + e (raw; used at the
  // end).  (Global-to-LDS loads are used for 4- and 16-byte elements only.)
  uint32_t hb[2][kIm2][4];
#pragma unroll
  for (int pp = 0; pp < 2; ++pp)
#pragma unroll
    for (int im = 0; im < kIm2; ++im) {
      if (P.hvec)
        bload4<SC, true>(hr[pp], i0 + 16 * im + 4 * gq, true, hb[pp][im]);
      else
        bload4<SC, false>(hr[pp], i0 + 16 * im + 4 * gq, true, hb[pp][im]);
    }

  floatx4 acc[2][kIm2][kTn2];
#pragma unroll
  for (int pp = 0; pp < 2; ++pp)
#pragma unroll
    for (int im = 0; im < kIm2; ++im)
#pragma unroll
      for (int tn = 0; tn < kTn2; ++tn) acc[pp][im][tn] = floatx4{0.f, 0.f, 0.f, 0.f};

  const uint32_t ones[4] = {0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u};
#pragma unroll
  for (int pp = 0; pp < 2; ++pp) {
    for (int kb0 = 0; kb0 < nkb; kb0 += kbc) {
      const int nb = min(kbc, nkb - kb0);
      // one round of global-to-LDS loads: w fragment groups (one wave
      // instruction each: 64 lanes x 16 bytes, lane l's fragment at l * 16) ...
      const int ngroups = nb * kTn2 * NW;
      for (int gi = wave; gi < ngroups; gi += kWaves) {
        int rest = gi;
        const int e = rest % NW;
        rest /= NW;
        const int tn = rest % kTn2;
        const int kbl = rest / kTn2;
        const int t = t0 + 16 * tn + n16;
        const uint32_t off = static_cast<uint32_t>(
            ((static_cast<int64_t>(pp * NW + e) * nkb + kb0 + kbl) * T + t) * 4 + gq) * 16u;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(wr, (lds_ptr)(bl + gi * 1024), 16, t < T ? off : kOob, 0, 0, 0);
      }
      // ... and the U words of this wave's outputs (full words; the tail word
      // from the tail plane, 16- or 32-bit entries)
      for (int kbl = 0; kbl < nb; ++kbl) {
        const int kb = kb0 + kbl;
        if (kb < nbu) {
          __builtin_amdgcn_raw_ptr_buffer_load_lds(ur[pp], (lds_ptr)(ul + (wave * kbc + kbl) * 256), 4,
                                                   iok ? static_cast<uint32_t>(kb * d_out + i0 + lane) * 4u : kOob, 0,
                                                   0, 0);
        } else if (tailu > 16) {
          __builtin_amdgcn_raw_ptr_buffer_load_lds(ur[pp], (lds_ptr)(ul + (wave * kbc + kbl) * 256), 4,
                                                   iok ? 4u * nbu * d_out + 4u * (i0 + lane) : kOob, 0, 0, 0);
        }
      }
      // 16-bit tail words (the step past the full words, r % 32 in 1..16) in
      // registers
      uint32_t tw[kIm2];
      const bool has16 = tailu != 0 && tailu <= 16 && nbu >= kb0 && nbu < kb0 + nb;
#pragma unroll
      for (int im = 0; im < kIm2; ++im) {
        const int i = i0 + 16 * im + n16;
        tw[im] = __builtin_amdgcn_raw_buffer_load_b16(ur[pp], has16 && i < d_out ? 4u * nbu * d_out + 2u * i : kOob, 0,
                                                      0);
      }
      __builtin_amdgcn_s_waitcnt(0);  // global-to-LDS loads count as memory loads
      __syncthreads();
      // products from LDS
      for (int kbl = 0; kbl < nb; ++kbl) {
        const int kb = kb0 + kbl;
        const bool tail16 = kb >= nbu && tailu <= 16;
        u32x4 B[kTn2][NW];
#pragma unroll
        for (int tn = 0; tn < kTn2; ++tn)
#pragma unroll
          for (int e = 0; e < NW; ++e)
            B[tn][e] = reinterpret_cast<const u32x4*>(bl)[((kbl * kTn2 + tn) * NW + e) * 64 + lane];
#pragma unroll
        for (int im = 0; im < kIm2; ++im) {
          const uint32_t word = tail16 ? (tw[im] & 0xffffu)
                                       : reinterpret_cast<const uint32_t*>(ul)[(wave * kbc + kbl) * 64 + 16 * im + n16];
          const u32x4 A = sign_terms(word, gq, ones);
#pragma unroll
          for (int tn = 0; tn < kTn2; ++tn)
#pragma unroll
            for (int e = 0; e < NW; ++e) acc[pp][im][tn] = mfma(A, B[tn][e], acc[pp][im][tn]);
        }
      }
      __syncthreads();  // the next round reuses the LDS
    }
  }

  // y[t][i] = h_0[i] acc_0 + h_1[i] acc_1 for outputs i = i0 + 16 im + 4 gq + e
  // of token t = t0 + 16 tn + n16
  const int ey = ACT == kDtF32 ? 4 : 2;
  const rsrc_t yr = make_rsrc_uniform(static_cast<char*>(P.y) + static_cast<int64_t>(t0) * d_out * ey,
                                      static_cast<uint32_t>(min(kTok2, T - t0) * d_out * ey));
#pragma unroll
  for (int im = 0; im < kIm2; ++im) {
    const int ib = i0 + 16 * im + 4 * gq;
    float h0[4], h1[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      h0[e] = P.hvec ? raw4_elem<SC, true>(hb[0][im], e) : raw4_elem<SC, false>(hb[0][im], e);
      h1[e] = P.hvec ? raw4_elem<SC, true>(hb[1][im], e) : raw4_elem<SC, false>(hb[1][im], e);
    }
#pragma unroll
    for (int tn = 0; tn < kTn2; ++tn) {
      const int t = t0 + 16 * tn + n16;
      float v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = h0[e] * acc[0][im][tn][e] + h1[e] * acc[1][im][tn][e];
      const uint32_t base = static_cast<uint32_t>((t - t0) * d_out + ib);  // within the tile's rows
      if (P.yvec) {
        // whole groups of 4 outputs (d_out % 4 == 0); rows past T are past the buffer
        const bool ok = t < T && ib < d_out;
        if constexpr (ACT == kDtF32) {
          const u32x4 d = {__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]), __float_as_uint(v[3])};
          __builtin_amdgcn_raw_buffer_store_b128(d, yr, ok ? base * 4u : kOob, 0, 0);
        } else {
          uint32_t b[4];
#pragma unroll
          for (int e = 0; e < 4; ++e)
            b[e] = ACT == kDtBF16 ? f32_to_bf16_bits(v[e])
                                  : static_cast<uint32_t>(__half_as_ushort(__float2half_rn(v[e])));
          const u32x2 d = {b[0] | (b[1] << 16), b[2] | (b[3] << 16)};
          __builtin_amdgcn_raw_buffer_store_b64(d, yr, ok ? base * 2u : kOob, 0, 0);
        }
      } else if (t < T) {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (ib + e < d_out) st<ACT>(P.y, static_cast<int64_t>(t) * d_out + ib + e, v[e]);
      }
    }
  }
}

template <typename K>
hipError_t raise_lds_limit(K* fn, size_t bytes, std::atomic<size_t>& limit) {
  // more than the default dynamic LDS limit: raise the kernel's limit once per
  // size increase, so calls captured in a graph after an eager call of the
  // same shape make no attribute call
  if (bytes > limit.load()) {
    const hipError_t e =
        hipFuncSetAttribute(reinterpret_cast<const void*>(fn), hipFuncAttributeMaxDynamicSharedMemorySize,
                            static_cast<int>(bytes));
    if (e != hipSuccess) return e;
    limit.store(bytes);
  }
  return hipSuccess;
}

template <int NPT, int ACT, int SC>
hipError_t launch_p1(const PrefillParams& P, const PrefillGeom& g, hipStream_t stream) {
  static std::atomic<size_t> limit{65536};
  hipError_t e = raise_lds_limit(&prefill_p1<NPT, ACT, SC>, g.smem1, limit);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((prefill_p1<NPT, ACT, SC>), dim3(g.n_tt * g.n_lt * g.ks), dim3(kThreads), g.smem1, stream, P);
  return hipGetLastError();
}

template <int ACT, int SC>
hipError_t launch_both(const PrefillParams& P, const PrefillGeom& g, hipStream_t stream) {
  hipError_t e;
  switch (g.npt) {
    case 2: e = launch_p1<2, ACT, SC>(P, g, stream); break;
    case 4: e = launch_p1<4, ACT, SC>(P, g, stream); break;
    case 5: e = launch_p1<5, ACT, SC>(P, g, stream); break;
    default: e = launch_p1<kMaxPairs, ACT, SC>(P, g, stream); break;
  }
  if (e != hipSuccess) return e;
  const int items = P.T * 2 * P.nkb * 4;
  hipLaunchKernelGGL((prefill_p1b<ACT, SC>), dim3((items + kThreads - 1) / kThreads), dim3(kThreads), 0, stream, P);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  static std::atomic<size_t> limit{65536};
  const size_t smem2 = p2_lds_bytes(P.kbc, ACT == kDtF32 ? 3 : 2);
  if ((e = raise_lds_limit(&prefill_p2<ACT, SC>, smem2, limit)) != hipSuccess) return e;
  hipLaunchKernelGGL((prefill_p2<ACT, SC>), dim3(g.n_ot * g.n_tt2), dim3(kThreads), smem2, stream, P);
  return hipGetLastError();
}

template <int ACT>
hipError_t launch_act(const PrefillParams& P, int sc_dt, const PrefillGeom& g, hipStream_t stream) {
  switch (sc_dt) {
    case kDtF32: return launch_both<ACT, kDtF32>(P, g, stream);
    case kDtF16: return launch_both<ACT, kDtF16>(P, g, stream);
    default: return launch_both<ACT, kDtBF16>(P, g, stream);
  }
}

size_t align256(size_t b) { return (b + 255) / 256 * 256; }

int64_t packed_bytes(int64_t n_out, int64_t n_red) {
  const int64_t w = n_red & 31;
  return 4 * (n_red >> 5) * n_out + (w == 0 ? 0 : (w <= 16 ? 2 : 4)) * n_out;
}

}  // namespace

PrefillGeom prefill_geometry(int T, int d_in, int d_out, int r) {
  PrefillGeom g{};
  const int tt = T > 0 ? T : 1;
  g.nkb = nblocks32(r > 0 ? r : 1);
  const int npairs = 2 * g.nkb;
  // latent tiles of at most kMaxPairs pairs, as even as possible (2, 4, 5 or 6)
  g.n_lt = (npairs + kMaxPairs - 1) / kMaxPairs;
  g.npt = (npairs + g.n_lt - 1) / g.n_lt;
  if (g.npt == 3) g.npt = 4;
  g.n_tt = (tt + kTok1 - 1) / kTok1;
  const int nbt = nblocks32(d_in > 0 ? d_in : 1);
  const int tiles = g.n_tt * g.n_lt;
  // about 256 workgroups, every split at most kMaxKbPer steps, at least one
  // step per wave when the reduction is long enough
  int ks = (256 + tiles - 1) / tiles;
  if (ks > nbt / kWaves) ks = nbt / kWaves;
  const int ks_min = (nbt + kMaxKbPer - 1) / kMaxKbPer;
  if (ks < ks_min) ks = ks_min;
  if (ks < 1) ks = 1;
  g.kb_per = (nbt + ks - 1) / ks;
  g.ks = (nbt + g.kb_per - 1) / g.kb_per;
  g.n_ot = (d_out + kOut2 - 1) / kOut2;
  if (g.n_ot < 1) g.n_ot = 1;
  g.n_tt2 = (tt + kTok2 - 1) / kTok2;
  // P2 stages up to kMaxKbc 32-latent blocks of one path per round
  g.kbc = g.nkb < kMaxKbc ? g.nkb : kMaxKbc;
  // LDS of P1: the g terms (both paths, up to 3 terms) or the wave reduction
  const size_t gterm = static_cast<size_t>(2) * g.kb_per * 4 * 3 * 16;
  const size_t red = static_cast<size_t>(kWaves) * kRedPairs * kTn1 * 64 * 32;
  g.smem1 = gterm > red ? gterm : red;
  // workspace (nothing beyond the control block when there is nothing to compute)
  const bool work = T > 0 && d_in > 0 && r > 0;
  g.pbuf_off = kCtrlBytes;
  g.pbuf_floats = work ? static_cast<size_t>(g.ks) * tiles * g.npt * kPbufPair : 0;
  g.wterm_off = g.pbuf_off + align256(4 * g.pbuf_floats);
  g.wterm_bytes = work ? static_cast<size_t>(2) * 3 * g.nkb * T * 64 : 0;
  g.ws_bytes = g.wterm_off + align256(g.wterm_bytes);
  return g;
}

bool prefill_supports(int64_t T, int64_t d_in, int64_t d_out, int64_t r) {
  // 32-bit buffer offsets, and one arrival counter per P1 tile
  const int64_t lim = int64_t(1) << 31;
  const PrefillGeom g = prefill_geometry(static_cast<int>(T), static_cast<int>(d_in), static_cast<int>(d_out),
                                         static_cast<int>(r));
  return int64_t(kTok2) * d_out * 4 < lim && int64_t(kTok1) * d_in * 4 < lim && packed_bytes(d_out, r) < lim &&
         packed_bytes(r, d_in) < lim && static_cast<int64_t>(g.wterm_bytes) < lim &&
         (g.ks == 1 || static_cast<int64_t>(g.n_tt) * g.n_lt <= kCtrlMaxTiles);
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
  P.pbuf = reinterpret_cast<float*>(ws + g.pbuf_off);
  P.wterm = reinterpret_cast<uint32_t*>(ws + g.wterm_off);
  P.T = a.T;
  P.d_in = a.d_in;
  P.d_out = a.d_out;
  P.r = a.r;
  P.nkb = g.nkb;
  P.n_tt = g.n_tt;
  P.n_lt = g.n_lt;
  P.ks = g.ks;
  P.kb_per = g.kb_per;
  P.n_ot = g.n_ot;
  P.kbc = g.kbc;
  P.npt = g.npt;
  const int64_t ex = a.act_dt == kDtF32 ? 4 : 2, es = a.sc_dt == kDtF32 ? 4 : 2;
  P.xvec = (reinterpret_cast<uintptr_t>(a.x) % (4 * ex) == 0) && (a.d_in % 4 == 0);
  P.yvec = (reinterpret_cast<uintptr_t>(a.y) % (4 * ex) == 0) && (a.d_out % 4 == 0);
  // 4-element vector loads of h never straddle its end only when d_out % 4 == 0
  P.hvec = (reinterpret_cast<uintptr_t>(a.h[0]) % (4 * es) == 0) &&
           (reinterpret_cast<uintptr_t>(a.h[1]) % (4 * es) == 0) && (a.d_out % 4 == 0);
  P.v_bytes = static_cast<uint32_t>(packed_bytes(a.r, a.d_in));
  P.u_bytes = static_cast<uint32_t>(packed_bytes(a.d_out, a.r));
  P.g_bytes = static_cast<uint32_t>(a.d_in * es);
  P.h_bytes = static_cast<uint32_t>(a.d_out * es);
  P.l_bytes = static_cast<uint32_t>(a.r * es);
  const int nw = a.act_dt == kDtF32 ? 3 : 2;
  P.wt_bytes = static_cast<uint32_t>(static_cast<int64_t>(2) * nw * g.nkb * a.T * 64);
  switch (a.act_dt) {
    case kDtF32: return launch_act<kDtF32>(P, a.sc_dt, g, stream);
    case kDtF16: return launch_act<kDtF16>(P, a.sc_dt, g, stream);
    default: return launch_act<kDtBF16>(P, a.sc_dt, g, stream);
  }
}

}  // namespace lb
