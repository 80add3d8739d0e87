// Streaming list forward on the matrix cores, for lists with linears of up to
// 64 tokens (Proposition 1, Eq. proposition1; both paths summed as in Eq.
// final_weight_approx_res), in three kinds of launch whatever the list's
// length, with no workgroup waiting for another:
//   S1  one workgroup per (linear, path, group of MT tiles of 16 latents, run
//       of d_in): D[k][t] = sum_j (s(V_p[j][k]) g_p[j]) x[t][j] over the run
//       with v_mfma_f32_16x16x32_bf16; the bf16 terms of g and x of a 32-input
//       block are built once and serve every latent tile of the group; the 4
//       waves split the run's blocks and are summed in a fixed order; the
//       run's partial sums l (.) z go to the workspace (one launch per token
//       tile count, 1..4);
//   R   one thread per (linear, path, token, latent): w = l (.) z, the sum of
//       the runs' partials in ascending run order, cut into bf16 terms and
//       stored in the layout of stage 2's B operand;
//   S2  one workgroup per (linear, 128 output rows for up to 16 tokens, else
//       256): the rows' U signs in LDS, each 32-latent block's A operand built
//       once per row tile for every token tile, y = h_0 u_0 + h_1 u_1 rounded
//       once (one launch per token tile count).
// Operands as in the single-launch matrix-core kernel: g and x are cut into
// exact bf16 terms (1, 2 or 3 per value for bf16, f16, fp32), so every product
// is exact and the sums are fp32; w is cut into 2 bf16 terms (3 for fp32
// outputs), which carries 16 (24) significant bits into stage 2.
//
// Inputs of this path: x and g read as aligned groups of four (d_in a
// multiple of 4, x and g aligned to four elements).
#include <algorithm>
#include <cstring>
#include <vector>

#include "device_common.h"
#include "stream_plan.h"

namespace lb {

namespace {

using splan::align256;
using splan::has_work;
using splan::kHdrCounts;
using splan::kHdrFp;
using splan::kHdrN;
using splan::packed_bytes64;
using splan::plan_ok;
using splan::StreamLinear;

constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr int kMaxTok = 64;
constexpr int kMaxRank = 1024;
constexpr int kMaxRuns = 511;   // S1 map code: 9 bits of run
constexpr int kMaxGroups = 63;  // S1 map code: 6 bits of latent group

// latent tiles of a group and 32-input blocks of a run, by token tile count
__host__ __device__ constexpr int mt_of(int tt) { return tt == 1 ? 4 : (tt == 2 ? 8 : 6); }
__host__ __device__ constexpr int bpr_of(int tt) { return tt == 1 ? 16 : (tt == 2 ? 32 : 64); }
// blocks a wave loads per round
__host__ __device__ constexpr int ku_of(int tt) { return tt <= 2 ? 2 : 1; }

struct SmGeom {
  int tt, mt, ng, bpr, s1d;
};

SmGeom sm_geometry(const ForwardArgs& a) {
  SmGeom g{};
  g.tt = (a.T + 15) / 16;
  g.mt = mt_of(g.tt);
  const int nmf = (a.r + 15) / 16;
  g.ng = (nmf + g.mt - 1) / g.mt;
  const int nbt = nblocks32(a.d_in);
  g.bpr = bpr_of(g.tt);
  g.s1d = (nbt + g.bpr - 1) / g.bpr;
  return g;
}

// ---------------------------------------------------------------------------
// S1
// ---------------------------------------------------------------------------
template <int TT, int MT>
struct BlockLoads {
  uint32_t w[MT];
  uint32_t g[2][4];
  uint32_t x[TT][2][4];
};

// loads of block b (valid; else every load reads past the buffers: zeros);
// lane (n16, gq) reads the words of latents k0 + 16 m + n16 and x, g at
// inputs 32 b + 4 gq + 16 h + (0..3)
template <int TT, int MT, int ACT, int SC>
__device__ __forceinline__ void s1_load(rsrc_t vr, rsrc_t gr, rsrc_t xr, int b, bool valid, int k0, int n16, int gq,
                                        int r, int d_in, BlockLoads<TT, MT>& L) {
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    const int k = k0 + 16 * m + n16;
    L.w[m] = __builtin_amdgcn_raw_buffer_load_b32(vr, valid && k < r ? static_cast<uint32_t>(b * r + k) * 4u : kOob,
                                                  0, 0);
  }
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const uint32_t j0 = 32 * b + 4 * gq + 16 * h;
    bload4<SC, true>(gr, j0, valid, L.g[h]);
#pragma unroll
    for (int tt = 0; tt < TT; ++tt)
      bload4<ACT, true>(xr, static_cast<uint32_t>(16 * tt + n16) * d_in + j0, valid, L.x[tt][h]);
  }
}

// the tail block's word of latent k (tail plane of V_p's packing)
__device__ __forceinline__ uint32_t s1_tail_word(rsrc_t vr, int k, int r, int d_in, bool valid) {
  const int nbv = d_in >> 5, tailv = d_in & 31;
  const uint32_t plane = 4u * nbv * r;
  const bool ok = valid && k < r;
  const uint32_t off = tailv <= 16 ? plane + 2u * k : plane + 4u * k;
  const uint32_t lo = static_cast<uint16_t>(__builtin_amdgcn_raw_buffer_load_b16(vr, ok ? off : kOob, 0, 0));
  const uint32_t hi =
      static_cast<uint16_t>(__builtin_amdgcn_raw_buffer_load_b16(vr, ok && tailv > 16 ? off + 2 : kOob, 0, 0));
  return lo | (hi << 16);
}

// MASK: the tail block, whose x groups at inputs >= d_in belong to the next
// row and are zeroed (g reads zero there)
template <int TT, int MT, int ACT, int SC, bool MASK>
__device__ __forceinline__ void s1_block(const BlockLoads<TT, MT>& L, int b, int gq, int d_in,
                                         floatx4 (&acc)[MT][TT]) {
  constexpr int NG = nterms<SC>(), NX = nterms<ACT>();
  uint32_t gt[NG][4];
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    if constexpr (NG == 1) {
      gt[0][v] = raw16<true>(L.g[0], v) | (raw16<true>(L.g[1], v) << 16);
    } else {
      uint32_t lo[NG], hi[NG];
      split_exact<NG>(raw4_elem<SC, true>(L.g[0], v), lo);
      split_exact<NG>(raw4_elem<SC, true>(L.g[1], v), hi);
#pragma unroll
      for (int s = 0; s < NG; ++s) gt[s][v] = lo[s] | (hi[s] << 16);
    }
  }
  u32x4 X[TT][NX];
  const bool ok0 = !MASK || 32 * b + 4 * gq < d_in, ok1 = !MASK || 32 * b + 4 * gq + 16 < d_in;
#pragma unroll
  for (int tt = 0; tt < TT; ++tt)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      if constexpr (NX == 1) {
        X[tt][0][v] = (ok0 ? raw16<true>(L.x[tt][0], v) : 0u) | ((ok1 ? raw16<true>(L.x[tt][1], v) : 0u) << 16);
      } else {
        uint32_t lo[NX], hi[NX];
        split_exact<NX>(ok0 ? raw4_elem<ACT, true>(L.x[tt][0], v) : 0.0f, lo);
        split_exact<NX>(ok1 ? raw4_elem<ACT, true>(L.x[tt][1], v) : 0.0f, hi);
#pragma unroll
        for (int a = 0; a < NX; ++a) X[tt][a][v] = lo[a] | (hi[a] << 16);
      }
    }
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int s = 0; s < NG; ++s) {
      const u32x4 A = sign_terms(L.w[m], gq, gt[s]);
#pragma unroll
      for (int tt = 0; tt < TT; ++tt)
#pragma unroll
        for (int a = 0; a < NX; ++a) acc[m][tt] = mfma(A, X[tt][a], acc[m][tt]);
    }
}

template <int TT, int MT, int ACT, int SC>
__global__ void __launch_bounds__(kThreads) sm_s1_kernel(const uint32_t* __restrict__ hdr,
                                                         const StreamLinear* __restrict__ descs,
                                                         const uint32_t* __restrict__ map, uint64_t fp) {
  constexpr int KU = ku_of(TT);
  __shared__ floatx4 red[MT * TT * 64];
  if (!plan_ok(hdr, fp)) return;
  const uint32_t code = map[blockIdx.x];
  const StreamLinear& L = descs[code >> 16];
  const int p = (code >> 15) & 1, grp = (code >> 9) & 63, c = code & 511;
  const int T = L.T, r = L.r, d_in = L.d_in;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int n16 = lane & 15, gq = lane >> 4;
  const rsrc_t vr = make_rsrc_uniform(p ? L.V[1] : L.V[0], L.v_bytes);
  const rsrc_t gr = make_rsrc_uniform(p ? L.g[1] : L.g[0], L.g_bytes);
  const rsrc_t xr = make_rsrc_uniform(L.x, L.x_bytes);
  const int k0 = 16 * MT * grp;
  const int nbt = nblocks32(d_in), nbv = d_in >> 5;
  const int b0 = c * L.bpr;
  const int b1 = min(nbt, b0 + L.bpr);
  const int bf = min(b1, nbv);

  floatx4 acc[MT][TT];
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) acc[m][tt] = floatx4{0.f, 0.f, 0.f, 0.f};

  // the tail block (if this run holds it, block nbv) goes to wave 0, after its
  // full blocks (its loads are not held across the main loop)
  const bool tail = b1 > nbv && wave == 0;
  // full blocks: wave w takes blocks b0 + KU (w + 4 i) + u
  for (int rb = b0 + KU * wave; rb < bf; rb += KU * kWaves) {
    BlockLoads<TT, MT> Lb[KU];
#pragma unroll
    for (int u = 0; u < KU; ++u) s1_load<TT, MT, ACT, SC>(vr, gr, xr, rb + u, rb + u < bf, k0, n16, gq, r, d_in, Lb[u]);
#pragma unroll
    for (int u = 0; u < KU; ++u) s1_block<TT, MT, ACT, SC, false>(Lb[u], rb + u, gq, d_in, acc);
  }
  if (tail) {
    BlockLoads<TT, MT> LT;
    s1_load<TT, MT, ACT, SC>(vr, gr, xr, nbv, true, k0, n16, gq, r, d_in, LT);
#pragma unroll
    for (int m = 0; m < MT; ++m) LT.w[m] = s1_tail_word(vr, k0 + 16 * m + n16, r, d_in, true);
    s1_block<TT, MT, ACT, SC, true>(LT, nbv, gq, d_in, acc);
  }

  // fixed-order sum over the waves: w0 + (w1 + (w2 + w3))
  for (int w = kWaves - 1; w >= 1; --w) {
    if (wave == w) {
#pragma unroll
      for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int tt = 0; tt < TT; ++tt) {
          const int e = (m * TT + tt) * 64 + lane;
          red[e] = w == kWaves - 1 ? acc[m][tt] : acc[m][tt] + red[e];
        }
    }
    __syncthreads();
  }
  if (wave != 0) return;
  const rsrc_t lr = make_rsrc_uniform(p ? L.l[1] : L.l[0], L.l_bytes);
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    float lk[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) lk[e] = bits_to_f32<SC>(bload<SC>(lr, k0 + 16 * m + 4 * gq + e));
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
      const floatx4 s = acc[m][tt] + red[(m * TT + tt) * 64 + lane];
      const int t = 16 * tt + n16;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int k = k0 + 16 * m + 4 * gq + e;
        if (t < T && k < r) L.part[((static_cast<int64_t>(p) * T + t) * L.s1d + c) * r + k] = s[e] * lk[e];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// R: w = l (.) z, the runs' partial sums in ascending run order, written as NW
// bf16 terms straight into the matrix-core B fragments of stage 2: for path
// p, token tile tt, 32-latent block kb and term a, one u32x4 per lane, lane
// (n16, gq) register v holding the term of w at token 16 tt + n16 and latents
// 32 kb + 4 gq + v (low half) and + 16 (high half); tokens past T and latents
// past r are zero
// ---------------------------------------------------------------------------
__host__ __device__ constexpr int nw_of(int act) { return act == kDtF32 ? 3 : 2; }

__host__ __device__ inline size_t frag_bytes(int T, int r, int nw) {
  return static_cast<size_t>(2) * ((T + 15) / 16) * nblocks32(r) * nw * 1024;
}

template <int NW>
__global__ void __launch_bounds__(kThreads) sm_r_kernel(const uint32_t* __restrict__ hdr,
                                                        const StreamLinear* __restrict__ descs,
                                                        const uint32_t* __restrict__ map, uint64_t fp) {
  if (!plan_ok(hdr, fp)) return;
  const uint32_t code = map[blockIdx.x];
  const StreamLinear& L = descs[code >> 16];
  const int e = static_cast<int>(code & 0xffffu) * kThreads + threadIdx.x;
  const int T = L.T, r = L.r, s1d = L.s1d;
  const int tt_n = (T + 15) / 16, nkb = nblocks32(r), kp = 32 * nkb;
  const int per = 16 * tt_n * kp;  // padded (token, latent) slots of one path
  if (e >= 2 * per) return;
  const int p = e / per, rem = e - p * per;
  const int t = rem / kp, k = rem - t * kp;
  float w = 0.0f;
  if (t < T && k < r) {
    const float* src = L.part + (static_cast<int64_t>(p) * T + t) * s1d * r + k;
    int c = 0;
    for (; c + 8 <= s1d; c += 8) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = src[static_cast<int64_t>(c + u) * r];
#pragma unroll
      for (int u = 0; u < 8; ++u) w += v[u];
    }
    for (; c < s1d; ++c) w += src[static_cast<int64_t>(c) * r];
  }
  uint32_t terms[NW];
  split_round<NW>(w, terms);
  const int tt = t >> 4, n16 = t & 15, kb = k >> 5, kk = k & 31;
  const int half = kk >> 4, gq = (kk & 15) >> 2, v = kk & 3;
  uint16_t* frag = reinterpret_cast<uint16_t*>(L.wlat);
#pragma unroll
  for (int a = 0; a < NW; ++a) {
    const int64_t f = ((static_cast<int64_t>(p) * tt_n + tt) * nkb + kb) * NW + a;
    frag[((f * 64 + gq * 16 + n16) * 4 + v) * 2 + half] = static_cast<uint16_t>(terms[a]);
  }
}

// ---------------------------------------------------------------------------
// S2: the output rows of one linear, every token, both paths.  Wave w holds
// RB row tiles of 16 (local rows 16 (w + 4 b) + (0..15)) for every token tile;
// the A operand of a 32-latent block (the U signs, from LDS) is built once per
// row tile and serves every token tile.  The B fragments come from R.  (The
// A operands are what costs VALU time, so the waves split rows, not tokens.)
// ---------------------------------------------------------------------------
__host__ __device__ constexpr int rb_of(int tt) { return tt == 1 ? 2 : 4; }
// output rows of a stage-2 workgroup
__host__ __device__ constexpr int rw_of(int tt) { return 16 * kWaves * rb_of(tt); }
// U words per thread in flight while staging them in LDS
constexpr int kStage = 8;

template <int TT, int ACT, int SC>
__global__ void __launch_bounds__(kThreads) sm_s2_kernel(const uint32_t* __restrict__ hdr,
                                                         const StreamLinear* __restrict__ descs,
                                                         const uint32_t* __restrict__ map, uint64_t fp) {
  constexpr int NW = nw_of(ACT);
  constexpr int RB = rb_of(TT), RW = rw_of(TT);
  extern __shared__ uint32_t uwl[];  // [2][nkb][RW] U words of this workgroup's rows
  if (!plan_ok(hdr, fp)) return;
  const uint32_t code = map[blockIdx.x];
  const StreamLinear& L = descs[code >> 16];
  const int q = static_cast<int>(code & 0xffffu);
  const int T = L.T, r = L.r, d_out = L.d_out;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int n16 = lane & 15, gq = lane >> 4;
  const int nkb = nblocks32(r), nbu = r >> 5, tailu = r & 31;
  const int qrow0 = q * RW;

  // the rows' U words (rows past d_out and blocks past r read as zero): a
  // full word as one 32-bit load, the tail plane's as 16-bit halves; a few
  // words per thread in flight before they go to LDS
#pragma unroll
  for (int pp = 0; pp < 2; ++pp) {
    const rsrc_t ur = make_rsrc_uniform(pp ? L.U[1] : L.U[0], L.u_bytes);
    const uint32_t plane = 4u * nbu * d_out;
    for (int e0 = tid; e0 < nkb * RW; e0 += kStage * kThreads) {
      uint32_t wv[kStage];
#pragma unroll
      for (int u = 0; u < kStage; ++u) {
        const int e = e0 + u * kThreads;
        const int kb = e / RW, row = qrow0 + (e - kb * RW);
        const bool ok = e < nkb * RW && row < d_out;
        const bool full = ok && kb < nbu, tl = ok && kb == nbu && tailu != 0;
        const uint32_t toff = tailu <= 16 ? plane + 2u * row : plane + 4u * row;
        const uint32_t w = __builtin_amdgcn_raw_buffer_load_b32(
            ur, full ? static_cast<uint32_t>(kb * d_out + row) * 4u : kOob, 0, 0);
        const uint32_t lo = static_cast<uint16_t>(__builtin_amdgcn_raw_buffer_load_b16(ur, tl ? toff : kOob, 0, 0));
        const uint32_t hi = static_cast<uint16_t>(
            __builtin_amdgcn_raw_buffer_load_b16(ur, tl && tailu > 16 ? toff + 2 : kOob, 0, 0));
        wv[u] = w | lo | (hi << 16);
      }
#pragma unroll
      for (int u = 0; u < kStage; ++u) {
        const int e = e0 + u * kThreads;
        if (e < nkb * RW) uwl[pp * nkb * RW + e] = wv[u];
      }
    }
  }
  __syncthreads();
  const rsrc_t fr = make_rsrc_uniform(L.wlat, static_cast<uint32_t>(frag_bytes(T, r, NW)));
  const uint32_t ones[4] = {0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u};
  floatx4 yv[RB][TT];
#pragma unroll
  for (int pp = 0; pp < 2; ++pp) {
    floatx4 acc[RB][TT];
#pragma unroll
    for (int b = 0; b < RB; ++b)
#pragma unroll
      for (int j = 0; j < TT; ++j) acc[b][j] = floatx4{0.f, 0.f, 0.f, 0.f};
    const uint32_t* ucol = uwl + pp * nkb * RW + 16 * wave + n16;
    // byte offset of fragment (token tile j, block kb, term a) of this lane
    const uint32_t fbase = static_cast<uint32_t>(pp * TT * nkb * NW * 64 + lane) * 16u;
    for (int kb = 0; kb < nkb; ++kb) {
      u32x4 B[TT][NW];
#pragma unroll
      for (int j = 0; j < TT; ++j)
#pragma unroll
        for (int a = 0; a < NW; ++a)
          B[j][a] = __builtin_amdgcn_raw_buffer_load_b128(
              fr, fbase + static_cast<uint32_t>(((j * nkb + kb) * NW + a) * 64) * 16u, 0, 0);
#pragma unroll
      for (int b = 0; b < RB; ++b) {
        const u32x4 A = sign_terms(ucol[kb * RW + 16 * kWaves * b], gq, ones);
#pragma unroll
        for (int j = 0; j < TT; ++j)
#pragma unroll
          for (int a = 0; a < NW; ++a) acc[b][j] = mfma(A, B[j][a], acc[b][j]);
      }
    }
    // y = h_0 acc_0 + h_1 acc_1 at rows qrow0 + 16 (wave + 4 b) + 4 gq + e
    const rsrc_t hr = make_rsrc_uniform(pp ? L.h[1] : L.h[0], L.h_bytes);
#pragma unroll
    for (int b = 0; b < RB; ++b) {
      float hv[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) hv[e] = bits_to_f32<SC>(bload<SC>(hr, qrow0 + 16 * (wave + kWaves * b) + 4 * gq + e));
#pragma unroll
      for (int j = 0; j < TT; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float v = hv[e] * acc[b][j][e];
          yv[b][j][e] = pp == 0 ? v : yv[b][j][e] + v;
        }
    }
  }
#pragma unroll
  for (int b = 0; b < RB; ++b)
#pragma unroll
    for (int j = 0; j < TT; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int i = qrow0 + 16 * (wave + kWaves * b) + 4 * gq + e;
        const int t = 16 * j + n16;
        if (t < T && i < d_out) st<ACT>(L.y, static_cast<int64_t>(t) * d_out + i, yv[b][j][e]);
      }
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
size_t s2_smem_bytes(int nkb, int rw) { return 4u * 2u * nkb * rw; }

struct PlanLayout {
  int n1 = 0, nr = 0, n2 = 0;
  int n1_cls[5] = {0, 0, 0, 0, 0};  // S1 items of token-tile count <= k are map entries [0, n1_cls[k])
  int n2_cls[5] = {0, 0, 0, 0, 0};  // the same for S2 items
  int nkb_max = 1;
  size_t desc_off = 0, map1_off = 0, mapr_off = 0, map2_off = 0, data_off = 0, bytes = 0;
};

PlanLayout plan_layout(const ForwardArgs* a, int n) {
  PlanLayout P;
  size_t data = 0;
  for (int i = 0; i < n; ++i) {
    if (!has_work(a[i])) continue;
    const SmGeom g = sm_geometry(a[i]);
    const int rw = rw_of(g.tt);
    P.nkb_max = std::max(P.nkb_max, nblocks32(a[i].r));
    P.n1 += 2 * g.ng * g.s1d;
    P.n1_cls[g.tt] += 2 * g.ng * g.s1d;
    const int nr = static_cast<int>((2 * 16 * g.tt * 32 * nblocks32(a[i].r) + kThreads - 1) / kThreads);
    P.nr += nr;
    P.n2 += (a[i].d_out + rw - 1) / rw;
    P.n2_cls[g.tt] += (a[i].d_out + rw - 1) / rw;
    data += align256(sizeof(float) * 2 * a[i].T * g.s1d * a[i].r) +
            align256(frag_bytes(a[i].T, a[i].r, nw_of(a[i].act_dt)));
  }
  for (int k = 1; k < 5; ++k) {
    P.n1_cls[k] += P.n1_cls[k - 1];
    P.n2_cls[k] += P.n2_cls[k - 1];
  }
  P.desc_off = kCtrlBytes;
  P.map1_off = P.desc_off + align256(sizeof(StreamLinear) * static_cast<size_t>(n));
  P.mapr_off = P.map1_off + align256(4 * static_cast<size_t>(P.n1));
  P.map2_off = P.mapr_off + align256(4 * static_cast<size_t>(P.nr));
  P.data_off = P.map2_off + align256(4 * static_cast<size_t>(P.n2));
  P.bytes = P.data_off + data;
  return P;
}

template <int TT, int ACT, int SC>
void launch_s1(const char* b, const PlanLayout& P, uint64_t fp, hipStream_t stream) {
  const int n = P.n1_cls[TT] - P.n1_cls[TT - 1];
  if (n == 0) return;
  hipLaunchKernelGGL((sm_s1_kernel<TT, mt_of(TT), ACT, SC>), dim3(n), dim3(kThreads), 0, stream,
                     reinterpret_cast<const uint32_t*>(b), reinterpret_cast<const StreamLinear*>(b + P.desc_off),
                     reinterpret_cast<const uint32_t*>(b + P.map1_off) + P.n1_cls[TT - 1], fp);
}

template <int TT, int ACT, int SC>
void launch_s2(const char* b, const PlanLayout& P, uint64_t fp, hipStream_t stream) {
  const int n = P.n2_cls[TT] - P.n2_cls[TT - 1];
  if (n == 0) return;
  const size_t smem = s2_smem_bytes(P.nkb_max, rw_of(TT));
  if (smem > 65536)
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&sm_s2_kernel<TT, ACT, SC>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(smem));
  hipLaunchKernelGGL((sm_s2_kernel<TT, ACT, SC>), dim3(n), dim3(kThreads), smem, stream,
                     reinterpret_cast<const uint32_t*>(b), reinterpret_cast<const StreamLinear*>(b + P.desc_off),
                     reinterpret_cast<const uint32_t*>(b + P.map2_off) + P.n2_cls[TT - 1], fp);
}

template <int ACT, int SC>
void launch_all(const void* ws, const PlanLayout& P, uint64_t fp, hipStream_t stream) {
  const char* b = static_cast<const char*>(ws);
  launch_s1<1, ACT, SC>(b, P, fp, stream);
  launch_s1<2, ACT, SC>(b, P, fp, stream);
  launch_s1<3, ACT, SC>(b, P, fp, stream);
  launch_s1<4, ACT, SC>(b, P, fp, stream);
  hipLaunchKernelGGL((sm_r_kernel<nw_of(ACT)>), dim3(P.nr), dim3(kThreads), 0, stream,
                     reinterpret_cast<const uint32_t*>(b), reinterpret_cast<const StreamLinear*>(b + P.desc_off),
                     reinterpret_cast<const uint32_t*>(b + P.mapr_off), fp);
  launch_s2<1, ACT, SC>(b, P, fp, stream);
  launch_s2<2, ACT, SC>(b, P, fp, stream);
  launch_s2<3, ACT, SC>(b, P, fp, stream);
  launch_s2<4, ACT, SC>(b, P, fp, stream);
}

template <int ACT>
void launch_act(const void* ws, const PlanLayout& P, int sc_dt, uint64_t fp, hipStream_t stream) {
  switch (sc_dt) {
    case kDtF32: launch_all<ACT, kDtF32>(ws, P, fp, stream); break;
    case kDtF16: launch_all<ACT, kDtF16>(ws, P, fp, stream); break;
    default: launch_all<ACT, kDtBF16>(ws, P, fp, stream); break;
  }
}

}  // namespace

bool stream_mma_supports(const ForwardArgs& a) {
  if (!has_work(a)) return true;
  if (a.T > kMaxTok || a.r > kMaxRank) return false;
  const int64_t ex = a.act_dt == kDtF32 ? 4 : 2, es = a.sc_dt == kDtF32 ? 4 : 2;
  // x and g as aligned groups of four elements
  if (a.d_in % 4 != 0 || reinterpret_cast<uintptr_t>(a.x) % (4 * ex) != 0 ||
      reinterpret_cast<uintptr_t>(a.g[0]) % (4 * es) != 0 || reinterpret_cast<uintptr_t>(a.g[1]) % (4 * es) != 0)
    return false;
  // 32-bit buffer offsets: the (up to 16 ceil(T / 16)) token rows read, the packed signs
  const int64_t lim = int64_t(1) << 31;
  const int64_t rows = 16 * ((a.T + 15) / 16);
  if ((rows + 1) * a.d_in * ex >= lim || packed_bytes64(a.d_out, a.r) >= lim || packed_bytes64(a.r, a.d_in) >= lim)
    return false;
  const SmGeom g = sm_geometry(a);
  if (g.s1d > kMaxRuns || g.ng > kMaxGroups) return false;
  // map codes: 16 bits of work index per linear
  if (2 * 16 * g.tt * 32 * nblocks32(a.r) > 65535 * kThreads || a.d_out > 65535 * 64) return false;
  return true;
}

size_t stream_mma_workspace_bytes(const ForwardArgs* a, int n) { return plan_layout(a, n).bytes; }

hipError_t stream_mma_init(const ForwardArgs* a, int n, uint64_t fp, void* ws, hipStream_t stream) {
  const PlanLayout P = plan_layout(a, n);
  std::vector<char> host(P.data_off, 0);
  uint32_t* hdr = reinterpret_cast<uint32_t*>(host.data());
  hdr[kHdrFp] = static_cast<uint32_t>(fp);
  hdr[kHdrFp + 1] = static_cast<uint32_t>(fp >> 32);
  hdr[kHdrN] = static_cast<uint32_t>(n);
  hdr[kHdrCounts + 0] = static_cast<uint32_t>(P.n1);
  hdr[kHdrCounts + 1] = static_cast<uint32_t>(P.nr);
  hdr[kHdrCounts + 2] = static_cast<uint32_t>(P.n2);
  StreamLinear* D = reinterpret_cast<StreamLinear*>(host.data() + P.desc_off);
  uint32_t* m1 = reinterpret_cast<uint32_t*>(host.data() + P.map1_off);
  uint32_t* mr = reinterpret_cast<uint32_t*>(host.data() + P.mapr_off);
  uint32_t* m2 = reinterpret_cast<uint32_t*>(host.data() + P.map2_off);
  char* data = static_cast<char*>(ws) + P.data_off;
  int i1[4] = {P.n1_cls[0], P.n1_cls[1], P.n1_cls[2], P.n1_cls[3]}, ir = 0;
  int i2[4] = {P.n2_cls[0], P.n2_cls[1], P.n2_cls[2], P.n2_cls[3]};
  for (int i = 0; i < n; ++i) {
    StreamLinear& L = D[i];
    const ForwardArgs& f = a[i];
    L.x = f.x;
    L.y = f.y;
    for (int p = 0; p < 2; ++p) {
      L.U[p] = f.U[p];
      L.V[p] = f.V[p];
      L.h[p] = f.h[p];
      L.g[p] = f.g[p];
      L.l[p] = f.l[p];
    }
    L.T = f.T;
    L.d_in = f.d_in;
    L.d_out = f.d_out;
    L.r = f.r;
    if (!has_work(f)) continue;
    const SmGeom g = sm_geometry(f);
    L.s1d = g.s1d;
    L.bpr = g.bpr;
    const int64_t ex = f.act_dt == kDtF32 ? 4 : 2, es = f.sc_dt == kDtF32 ? 4 : 2;
    L.x_bytes = static_cast<uint32_t>(static_cast<int64_t>(f.T) * f.d_in * ex);
    L.g_bytes = static_cast<uint32_t>(f.d_in * es);
    L.h_bytes = static_cast<uint32_t>(f.d_out * es);
    L.l_bytes = static_cast<uint32_t>(f.r * es);
    L.v_bytes = static_cast<uint32_t>(packed_bytes64(f.r, f.d_in));
    L.u_bytes = static_cast<uint32_t>(packed_bytes64(f.d_out, f.r));
    L.part = reinterpret_cast<float*>(data);
    data += align256(sizeof(float) * 2 * f.T * g.s1d * f.r);
    L.wlat = reinterpret_cast<float*>(data);  // the B fragments of stage 2
    data += align256(frag_bytes(f.T, f.r, nw_of(f.act_dt)));
    // S1 and S2 items grouped by token-tile count (one launch each)
    for (int p = 0; p < 2; ++p)
      for (int gr = 0; gr < g.ng; ++gr)
        for (int c = 0; c < g.s1d; ++c)
          m1[i1[g.tt - 1]++] = (static_cast<uint32_t>(i) << 16) | (p << 15) | (gr << 9) | c;
    const int nrb = (2 * 16 * g.tt * 32 * nblocks32(f.r) + kThreads - 1) / kThreads;
    for (int j = 0; j < nrb; ++j) mr[ir++] = (static_cast<uint32_t>(i) << 16) | j;
    const int rw = rw_of(g.tt);
    const int nrow = (f.d_out + rw - 1) / rw;
    for (int j = 0; j < nrow; ++j) m2[i2[g.tt - 1]++] = (static_cast<uint32_t>(i) << 16) | j;
  }
  hipError_t e = hipMemcpyAsync(ws, host.data(), host.size(), hipMemcpyHostToDevice, stream);
  if (e != hipSuccess) return e;
  return hipStreamSynchronize(stream);
}

hipError_t stream_mma_forward(const ForwardArgs* a, int n, uint64_t fp, void* ws, hipStream_t stream) {
  const PlanLayout P = plan_layout(a, n);
  if (P.n1 == 0) return hipSuccess;
  int act = -1, sc = -1;
  for (int i = 0; i < n; ++i)
    if (has_work(a[i])) {
      act = a[i].act_dt;
      sc = a[i].sc_dt;
      break;
    }
  switch (act) {
    case kDtF32: launch_act<kDtF32>(ws, P, sc, fp, stream); break;
    case kDtF16: launch_act<kDtF16>(ws, P, sc, fp, stream); break;
    default: launch_act<kDtBF16>(ws, P, sc, fp, stream); break;
  }
  return hipGetLastError();
}

}  // namespace lb
