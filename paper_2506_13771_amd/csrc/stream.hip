// Streaming list forward for decode-sized linears (T <= 2 tokens): a list of
// independent LittleBit linears (Proposition 1, Eq. proposition1, both paths
// summed as in Eq. final_weight_approx_res) in three launches, whatever the
// list's length:
//   S1  one workgroup per (linear, path, run of d_in): the nibble tables of
//       a = g (.) x over the run are built once in LDS and serve every latent
//       of the linear; lane k of a wave reads the packed V words of latent
//       64 kt + k (256 bytes per wave and block, coalesced), and the run's
//       partial sums l (.) z go to the workspace;
//   R   one thread per (linear, path, token, latent): w = l (.) z, the sum of
//       the runs' partials in ascending run order;
//   S2  one workgroup per (linear, 256 output rows): tables over w, one lane
//       per output row, the row's U words of both paths, y = h_0 u_0 + h_1 u_1
//       rounded once.
// The linears are independent, so launch order is the only synchronisation:
// no workgroup waits for another, and the GPU stays busy across linears.
//
// Each result is bit-identical to the single-launch decode kernel's for the
// same linear: the d_in runs are that kernel's (decode_geometry), the tables
// and look-ups are the same code (lut_common.h), and every sum follows the
// same tree -- per latent, the 4 waves x 4 lane groups of the single kernel
// become 16 accumulators (wave w keeps the role of that kernel's wave w, and
// each lane holds the 4 lane groups' sequences for its own latent); per row,
// the 4 quad lanes' sequences over words q, q + 4, ... become 4 sequences in
// one lane.  Blocks past a run add +0 in the single kernel and are skipped
// here.  Both files are compiled without floating-point contraction.
//
// The list's descriptors and work maps live in the workspace (the "plan",
// written once by stream_init); every kernel first compares the plan's
// fingerprint with the one of the call and does nothing but set bit 1 of the
// error word if they differ.
#include <atomic>
#include <cstring>
#include <vector>

#include "lut_common.h"
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
using lut::build_table;
using lut::kBlk;
using lut::kChunk;
using lut::tree4;
using lut::word_sum_b;

constexpr int kThreads = 256;
constexpr int kMaxRunBlocks = 64;  // blocks of 32 inputs of one d_in run (tables of a run in LDS at once)
constexpr int kRpl = 2;                   // stage-2 output rows per lane
constexpr int kRowsS2 = kRpl * kThreads;  // stage-2 output rows per workgroup
constexpr int kMaxTokens = 2;
constexpr int kMaxRank = 1024;

// ---------------------------------------------------------------------------
// LDS addressing for the look-ups: a table set of one block is 512 bytes (8
// nibble tables of 16 floats), 256-byte aligned, so the address of entry n
// of table q is (block base) + 4 n + 64 q, with 4 n the byte taken out of a
// pre-shifted copy of the word (lut::word_sum_b) and 64 q the load's
// immediate offset.  v_perm_b32 forms (base with its low byte replaced by
// that byte) in one instruction; its selectors live in registers that the
// compiler cannot rematerialise (opaque_sel).
// ---------------------------------------------------------------------------
typedef __attribute__((address_space(3))) const float* lds_cfp;
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) const void*)p));
}
__device__ __forceinline__ float lds_f32(uint32_t addr) {
  return *reinterpret_cast<lds_cfp>(static_cast<uintptr_t>(addr));
}
__device__ __forceinline__ uint32_t opaque_sel(uint32_t v) {
  asm volatile("" : "+v"(v));
  return v;
}

// lut::word_sum_b for a table set at LDS byte address base (256-aligned):
// sel[j] = 0x07060500 | j keeps base's upper bytes and takes byte j of e / o.
__device__ __forceinline__ float word_sum_at(uint32_t base, uint32_t wk, const uint32_t (&sel)[4]) {
  const uint32_t e = (wk << 2) & 0x3C3C3C3Cu, o = (wk >> 2) & 0x3C3C3C3Cu;
  float v[8];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    v[2 * j] = lds_f32(__builtin_amdgcn_perm(base, e, sel[j]) + 64 * (2 * j));
    v[2 * j + 1] = lds_f32(__builtin_amdgcn_perm(base, o, sel[j]) + 64 * (2 * j + 1));
  }
  return ((v[0] + v[1]) + (v[2] + v[3])) + ((v[4] + v[5]) + (v[6] + v[7]));
}

// ---------------------------------------------------------------------------
// S1: partial sums of one run of d_in (at most MAXBLK blocks), every latent
// of one path.  The run is padded to MAXBLK blocks with zero tables: a word
// looked up in a zero table adds +0 or -0, which leaves every accumulator
// unchanged (an accumulator starts at +0 and never becomes -0), so the inner
// loop needs no test per block and stays one stretch of straight-line code
// in which the loads of the next tile are in flight while the current tile
// is summed.
// ---------------------------------------------------------------------------
template <int TM, int ACT, int SC, int MAXBLK, bool TAIL16, int NTALL>
__global__ void __launch_bounds__(kThreads) stream_s1_kernel(const uint32_t* __restrict__ hdr,
                                                             const StreamLinear* __restrict__ descs,
                                                             const uint32_t* __restrict__ map, uint64_t fp) {
  constexpr int kSet = 128;            // floats of one block's table set
  constexpr int kNch = MAXBLK / kChunk;  // 32-block chunks of a run
  constexpr int kWords = 8 * kNch;     // words of a tile per lane
  // LDS: the tables [TM][MAXBLK][kSet] (256-byte aligned), every wave's
  // partial sums of every tile [4][TM][rpad], the latent scales [r]
  extern __shared__ __attribute__((aligned(256))) float smem[];
  float* tbl = smem;
  if (!plan_ok(hdr, fp)) return;
  const uint32_t code = map[blockIdx.x];
  const int li = static_cast<int>(code >> 16), p = static_cast<int>((code >> 8) & 0xffu),
            c = static_cast<int>(code & 0xffu);
  const StreamLinear& L = descs[li];
  const int T = L.T, r = L.r, d_in = L.d_in;
  const int tid = threadIdx.x;
  const int nbv = d_in >> 5, tailv = d_in & 31, nbt = nblocks32(d_in);
  const int b0 = c * L.bpr, b1 = min(nbt, b0 + L.bpr), nblk = b1 - b0;
  // descriptors from the plan: read back from the first lane so that they
  // live in scalar registers (the compiler cannot prove them uniform)
  const rsrc_t vr = make_rsrc_uniform(p ? L.V[1] : L.V[0], L.v_bytes);
  const rsrc_t gr = make_rsrc_uniform(p ? L.g[1] : L.g[0], L.g_bytes);
  const rsrc_t xr = make_rsrc_uniform(L.x, L.x_bytes);
  const rsrc_t lr = make_rsrc_uniform(p ? L.l[1] : L.l[0], L.l_bytes);
  const int rpad = ((r + 63) >> 6) << 6;
  float* red = smem + TM * MAXBLK * kSet;  // [4 waves][TM][rpad]
  float* lsh = red + 4 * TM * rpad;        // [r]

  // wave w reads blocks 32 ch + 8 w + j (j = m + 4 u < 8) of each chunk ch
  // (the blocks the single kernel's wave w reads), lane k one latent of the
  // tile.  Words past the run or past r are loaded too and never matter
  // (zero tables, discarded latents); only a run that holds a 16-bit tail
  // block (a plane of 16-bit words after the full words; TAIL16, a launch of
  // its own) loads element-wise.
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const uint32_t plane = 4u * nbv * r;
  const int ntile = (r + 63) >> 6;
  auto load_tile = [&](int kt, uint32_t (&wd)[kWords]) {
    const int k = 64 * kt + lane;
    if constexpr (!TAIL16) {
      // a 17..31-bit tail plane holds 32-bit words at the full words' stride
#pragma unroll
      for (int ch = 0; ch < kNch; ++ch) {
        const uint32_t vo = static_cast<uint32_t>((b0 + 32 * ch + 8 * w) * r + k) * 4u;
#pragma unroll
        for (int j = 0; j < 8; ++j) wd[8 * ch + j] = __builtin_amdgcn_raw_buffer_load_b32(vr, vo, 4 * j * r, 0);
      }
      return;
    }
    const bool kok = k < r;
#pragma unroll
    for (int ch = 0; ch < kNch; ++ch)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int bi = 32 * ch + 8 * w + j;
        const int b = b0 + bi;
        const bool in = kok && bi < nblk;
        uint32_t v = __builtin_amdgcn_raw_buffer_load_b32(
            vr, in && b < nbv ? static_cast<uint32_t>(b * r + k) * 4u : kOob, 0, 0);
        const uint32_t lo = __builtin_amdgcn_raw_buffer_load_b16(vr, in && b == nbv ? plane + 2u * k : kOob, 0, 0);
        wd[8 * ch + j] = v | (lo & 0xffffu);
      }
  };
  // the g and x elements of the run's tables (and zero tables up to
  // MAXBLK: thread e builds table e % 8 of block e / 8) are loaded first, so
  // that the tables can be built while the words are still in flight
  // (vector-memory loads complete in issue order)
  static_assert((8 * MAXBLK) % kThreads == 0, "whole table items per thread");
  constexpr int kItems = 8 * MAXBLK / kThreads;
  uint32_t gb[kItems][4], xb[kItems][TM][4];
#pragma unroll
  for (int n = 0; n < kItems; ++n) {
    const int e = tid + kThreads * n;
    const int bi = e >> 3, q = e & 7;
    const int jb = 32 * (b0 + bi) + 4 * q;
    const bool in = bi < nblk;
    bload4<SC, false>(gr, jb, in, gb[n]);
#pragma unroll
    for (int t = 0; t < TM; ++t) bload4<ACT, false>(xr, t * d_in + jb, in && t < T, xb[n][t]);
  }
  // NTALL > 0 (every rank of the list <= 64 NTALL): every tile's words are
  // loaded at once, in flight while the tables are built; else two tiles'
  // words at a time
  constexpr int kBuf = NTALL > 0 ? NTALL : 2;
  uint32_t wbuf[kBuf][kWords];
  if constexpr (NTALL > 0) {
#pragma unroll
    for (int kt = 0; kt < NTALL; ++kt) load_tile(kt, wbuf[kt]);
  } else {
    load_tile(0, wbuf[0]);
  }
#pragma unroll
  for (int n = 0; n < kItems; ++n) {
    const int e = tid + kThreads * n;
    const int bi = e >> 3, q = e & 7;
    const int jb = 32 * (b0 + bi) + 4 * q;
#pragma unroll
    for (int t = 0; t < TM; ++t) {
      float a[4];
      lut::table_inputs<ACT, SC, false>(xb[n][t], gb[n], jb, d_in, tailv, a);
      lut::build_table_plain(tbl + (t * MAXBLK + bi) * kSet + 16 * q, a[0], a[1], a[2], a[3]);
    }
  }
  for (int k = tid; k < r; k += kThreads) lsh[k] = bits_to_f32<SC>(bload<SC>(lr, k));
  __syncthreads();

  uint32_t sel[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) sel[j] = opaque_sel(0x07060500u | static_cast<uint32_t>(j));
  const uint32_t tbase = lds_addr(tbl) + static_cast<uint32_t>(8 * w * kSet * 4);
  // one tile: the next tile's words are loaded first (past the last tile:
  // harmless loads that are never used), then this tile's are summed and the
  // wave's partial sums go to LDS; the two buffers alternate (a register copy
  // of a load's destination would wait for that load).  The waves never wait
  // for each other inside the loop.
  auto tile = [&](int kt, const uint32_t (&cw)[kWords], uint32_t (&nw_)[kWords]) {
    if constexpr (NTALL == 0) load_tile(kt + 1, nw_);
    float acc[4][TM];
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
      for (int t = 0; t < TM; ++t) acc[m][t] = 0.0f;
#pragma unroll
    for (int ch = 0; ch < kNch; ++ch)
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int m = 0; m < 4; ++m)
#pragma unroll
          for (int t = 0; t < TM; ++t)
            acc[m][t] += word_sum_at(tbase + static_cast<uint32_t>((t * MAXBLK + 32 * ch + m + 4 * u) * kSet * 4),
                                     cw[8 * ch + m + 4 * u], sel);
#pragma unroll
    for (int t = 0; t < TM; ++t)
      red[(w * TM + t) * rpad + 64 * kt + lane] = tree4(acc[0][t], acc[1][t], acc[2][t], acc[3][t]);
  };
  if constexpr (NTALL > 0) {
#pragma unroll
    for (int kt = 0; kt < NTALL; ++kt)
      if (kt < ntile) tile(kt, wbuf[kt], wbuf[kt]);
  } else {
    for (int kt = 0; kt < ntile; kt += 2) {
      tile(kt, wbuf[0], wbuf[1]);
      if (kt + 1 < ntile) tile(kt + 1, wbuf[1], wbuf[0]);
    }
  }
  __syncthreads();
  // the 4 waves' partial sums of each latent, scaled by l
  for (int e = tid; e < T * r; e += kThreads) {
    const int t = e / r, k = e - t * r;
    const float sv = tree4(red[(0 * TM + t) * rpad + k], red[(1 * TM + t) * rpad + k], red[(2 * TM + t) * rpad + k],
                           red[(3 * TM + t) * rpad + k]) *
                     lsh[k];
    L.part[((p * T + t) * L.s1d + c) * r + k] = sv;
  }
}

// ---------------------------------------------------------------------------
// R: w = l (.) z, the runs' partial sums in ascending run order
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(kThreads) stream_r_kernel(const uint32_t* __restrict__ hdr,
                                                            const StreamLinear* __restrict__ descs,
                                                            const uint32_t* __restrict__ map, uint64_t fp) {
  if (!plan_ok(hdr, fp)) return;
  const uint32_t code = map[blockIdx.x];
  const StreamLinear& L = descs[code >> 16];
  const int e = static_cast<int>(code & 0xffffu) * kThreads + threadIdx.x;
  const int r = L.r, s1d = L.s1d;
  if (e >= 2 * L.T * r) return;
  const int pt = e / r, k = e - pt * r;
  const float* src = L.part + static_cast<int64_t>(pt) * s1d * r + k;
  // every partial in flight at once, then the sum in ascending run order
  float v[lut::kMaxRuns];
#pragma unroll
  for (int cc = 0; cc < lut::kMaxRuns; ++cc) v[cc] = cc < s1d ? src[cc * r] : 0.0f;
  float w = 0.0f;
#pragma unroll
  for (int cc = 0; cc < lut::kMaxRuns; ++cc)
    if (cc < s1d) w += v[cc];
  L.wlat[e] = w;
}

// ---------------------------------------------------------------------------
// S2: kRowsS2 output rows of one linear (kRpl per lane), both paths
// ---------------------------------------------------------------------------
template <int TM, int ACT, int SC, int NWMAX>
__global__ void __launch_bounds__(kThreads) stream_s2_kernel(const uint32_t* __restrict__ hdr,
                                                             const StreamLinear* __restrict__ descs,
                                                             const uint32_t* __restrict__ map, uint64_t fp) {
  // static LDS: every table sits at a compile-time offset, so a look-up's
  // address is the byte taken from the word and the rest is the instruction's
  // immediate offset
  constexpr int kSet2 = 128;  // floats of one 32-latent block's table set
  __shared__ __attribute__((aligned(256))) float tb2[2 * TM * NWMAX * kSet2];
  if (!plan_ok(hdr, fp)) return;
  const uint32_t code = map[blockIdx.x];
  const StreamLinear& L = descs[code >> 16];
  const int T = L.T, r = L.r, d_out = L.d_out;
  const int tid = threadIdx.x;
  const int i0 = static_cast<int>(code & 0xffffu) * kRowsS2 + tid;  // rows i0 + kThreads * q
  const int nw = nblocks32(r), nbu = r >> 5, tailu = r & 31;

  // the latents this thread's tables are built from, loaded before the U
  // words so that the table build waits for them alone
  const int ngrp = 8 * nw;
  constexpr int kGrpMax = (2 * TM * 8 * NWMAX + kThreads - 1) / kThreads;
  float w4s[kGrpMax][4];
#pragma unroll
  for (int gi = 0; gi < kGrpMax; ++gi) {
    const int e = tid + kThreads * gi;
    const int pt = e / ngrp, grp = e - pt * ngrp;
    const int pp = pt / TM, t = pt - pp * TM;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int k = 4 * grp + j;
      const bool ok = e < 2 * TM * ngrp && t < T && k < r;
      w4s[gi][j] = ok ? L.wlat[(pp * T + t) * r + k] : 0.0f;
    }
  }

  // this lane's rows' U words of both paths, and their row scales
  uint32_t wd[kRpl][2][NWMAX], hb[kRpl][2];
  const uint32_t plane = 4u * nbu * d_out;
#pragma unroll
  for (int q = 0; q < kRpl; ++q) {
    const int i = i0 + kThreads * q;
    const bool iok = i < d_out;
#pragma unroll
    for (int pp = 0; pp < 2; ++pp) {
      const rsrc_t ur = make_rsrc_uniform(pp ? L.U[1] : L.U[0], L.u_bytes);
      const uint32_t vo = iok ? static_cast<uint32_t>(i) * 4u : kOob;
#pragma unroll
      for (int kb = 0; kb < NWMAX; ++kb) {
        if (kb < nbu) {
          wd[q][pp][kb] = __builtin_amdgcn_raw_buffer_load_b32(ur, vo, 4 * kb * d_out, 0);
        } else if (kb == nbu && tailu != 0) {
          const uint32_t off = plane + (tailu <= 16 ? 2u : 4u) * i;
          const uint32_t lo = __builtin_amdgcn_raw_buffer_load_b16(ur, iok ? off : kOob, 0, 0);
          const uint32_t hi = __builtin_amdgcn_raw_buffer_load_b16(ur, iok && tailu > 16 ? off + 2 : kOob, 0, 0);
          wd[q][pp][kb] = (lo & 0xffffu) | (hi << 16);
        } else {
          wd[q][pp][kb] = 0u;
        }
      }
      hb[q][pp] = bload<SC>(make_rsrc_uniform(pp ? L.h[1] : L.h[0], L.h_bytes), i, iok);
    }
  }

  // tables over groups of 4 latents of w (latents past r are 0)
#pragma unroll
  for (int gi = 0; gi < kGrpMax; ++gi) {
    const int e = tid + kThreads * gi;
    if (e < 2 * TM * ngrp) {
      const int pt = e / ngrp, grp = e - pt * ngrp;
      const int pp = pt / TM, t = pt - pp * TM;
      lut::build_table_plain(tb2 + ((pp * TM + t) * NWMAX + (grp >> 3)) * kSet2 + 16 * (grp & 7), w4s[gi][0],
                             w4s[gi][1], w4s[gi][2], w4s[gi][3]);
    }
  }
  __syncthreads();

  uint32_t sel[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) sel[j] = opaque_sel(0x07060500u | static_cast<uint32_t>(j));
  const uint32_t tbase = lds_addr(tb2);
#pragma unroll
  for (int t = 0; t < TM; ++t) {
    if (t >= T) break;
    // the single kernel's quad lane g sums words g, g + 4, ... in order
    float a[kRpl][2][4];
#pragma unroll
    for (int q = 0; q < kRpl; ++q)
#pragma unroll
      for (int pp = 0; pp < 2; ++pp)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) a[q][pp][g4] = 0.0f;
#pragma unroll
    for (int kb = 0; kb < NWMAX; ++kb) {
      if (kb < nw) {
#pragma unroll
        for (int pp = 0; pp < 2; ++pp) {
          const uint32_t tb = tbase + static_cast<uint32_t>(((pp * TM + t) * NWMAX + kb) * kSet2 * 4);
#pragma unroll
          for (int q = 0; q < kRpl; ++q) a[q][pp][kb & 3] += word_sum_at(tb, wd[q][pp][kb], sel);
        }
      }
    }
#pragma unroll
    for (int q = 0; q < kRpl; ++q) {
      const int i = i0 + kThreads * q;
      const float v = lut::row_value(bits_to_f32<SC>(hb[q][0]), tree4(a[q][0][0], a[q][0][1], a[q][0][2], a[q][0][3]),
                                     bits_to_f32<SC>(hb[q][1]), tree4(a[q][1][0], a[q][1][1], a[q][1][2], a[q][1][3]));
      if (i < d_out) st<ACT>(L.y, static_cast<int64_t>(t) * d_out + i, v);
    }
  }
}

// ---------------------------------------------------------------------------
// host side: plan layout, work counts and launches
// ---------------------------------------------------------------------------
// the S1 class of run c of a linear (see launch_s1)
int s1_class(const ForwardArgs& a, const DecodeGeom& g, int c) {
  const int nbt = nblocks32(a.d_in), nbv = a.d_in >> 5, tailv = a.d_in & 31;
  const int b1 = (c + 1) * g.bpr < nbt ? (c + 1) * g.bpr : nbt;
  const bool tail16 = tailv != 0 && tailv <= 16 && b1 > nbv;
  return (g.bpr <= kChunk ? 0 : 1) + (tail16 ? 2 : 0);
}

struct PlanLayout {
  int n1 = 0, nr = 0, n2 = 0;
  int n1_cls[5] = {0, 0, 0, 0, 0};  // S1 items of class < k are map entries [0, n1_cls[k]) (see launch_s1)
  int tm = 1, nwmax = 1, nblk_max = 1, rmax = 1;
  size_t desc_off = 0, map1_off = 0, mapr_off = 0, map2_off = 0, data_off = 0, bytes = 0;
};

PlanLayout plan_layout(const ForwardArgs* a, int n) {
  PlanLayout P;
  size_t data = 0;
  for (int i = 0; i < n; ++i) {
    if (!has_work(a[i])) continue;
    const DecodeGeom g = decode_geometry(a[i].T, a[i].d_in, a[i].d_out, a[i].r);
    P.n1 += 2 * g.s1d;
    for (int c = 0; c < g.s1d; ++c) P.n1_cls[s1_class(a[i], g, c) + 1] += 2;
    P.nr += (2 * a[i].T * a[i].r + kThreads - 1) / kThreads;
    P.n2 += (a[i].d_out + kRowsS2 - 1) / kRowsS2;
    P.tm = a[i].T > P.tm ? a[i].T : P.tm;
    P.nwmax = nblocks32(a[i].r) > P.nwmax ? nblocks32(a[i].r) : P.nwmax;
    P.rmax = a[i].r > P.rmax ? a[i].r : P.rmax;
    P.nblk_max = g.bpr > P.nblk_max ? g.bpr : P.nblk_max;
    data += align256(sizeof(float) * 2 * a[i].T * g.s1d * a[i].r) + align256(sizeof(float) * 2 * a[i].T * a[i].r);
  }
  for (int k = 1; k < 5; ++k) P.n1_cls[k] += P.n1_cls[k - 1];
  P.desc_off = kCtrlBytes;
  P.map1_off = P.desc_off + align256(sizeof(StreamLinear) * static_cast<size_t>(n));
  P.mapr_off = P.map1_off + align256(4 * static_cast<size_t>(P.n1));
  P.map2_off = P.mapr_off + align256(4 * static_cast<size_t>(P.nr));
  P.data_off = P.map2_off + align256(4 * static_cast<size_t>(P.n2));
  P.bytes = P.data_off + data;
  return P;
}

// S1 in up to four launches (independent of each other), one per class of
// items (the plan's S1 map lists them in this order): runs of at most 32
// blocks (half the LDS: twice the workgroups per CU) and of up to 64, each
// without and with a 16-bit tail block
template <int TM, int ACT, int SC, int MAXBLK, bool TAIL16, int NTALL>
void launch_s1_nt(const char* b, const PlanLayout& P, int cls, uint64_t fp, hipStream_t stream) {
  const int n = P.n1_cls[cls + 1] - P.n1_cls[cls];
  const int rpad = ((P.rmax + 63) / 64) * 64;
  const size_t smem = sizeof(float) * (TM * MAXBLK * 128 + 4 * TM * rpad + P.rmax);
  static std::atomic<size_t> limit{65536};
  if (smem > limit.load()) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&stream_s1_kernel<TM, ACT, SC, MAXBLK, TAIL16, NTALL>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(smem));
    limit.store(smem);
  }
  hipLaunchKernelGGL((stream_s1_kernel<TM, ACT, SC, MAXBLK, TAIL16, NTALL>), dim3(n), dim3(kThreads), smem, stream,
                     reinterpret_cast<const uint32_t*>(b), reinterpret_cast<const StreamLinear*>(b + P.desc_off),
                     reinterpret_cast<const uint32_t*>(b + P.map1_off) + P.n1_cls[cls], fp);
}
template <int TM, int ACT, int SC, int MAXBLK, bool TAIL16>
void launch_s1_class(const char* b, const PlanLayout& P, int cls, uint64_t fp, hipStream_t stream) {
  if (P.n1_cls[cls + 1] == P.n1_cls[cls]) return;
  // every tile's words in registers at once while the list's ranks allow
  // (5 tiles of 64 latents: r <= 320), else two tiles at a time
  if constexpr (TAIL16) {
    launch_s1_nt<TM, ACT, SC, MAXBLK, TAIL16, 0>(b, P, cls, fp, stream);
  } else {
    if (P.rmax <= 5 * 64)
      launch_s1_nt<TM, ACT, SC, MAXBLK, TAIL16, 5>(b, P, cls, fp, stream);
    else
      launch_s1_nt<TM, ACT, SC, MAXBLK, TAIL16, 0>(b, P, cls, fp, stream);
  }
}
template <int TM, int ACT, int SC>
void launch_s1(const void* ws, const PlanLayout& P, uint64_t fp, hipStream_t stream) {
  const char* b = static_cast<const char*>(ws);
  launch_s1_class<TM, ACT, SC, kChunk, false>(b, P, 0, fp, stream);
  launch_s1_class<TM, ACT, SC, kMaxRunBlocks, false>(b, P, 1, fp, stream);
  launch_s1_class<TM, ACT, SC, kChunk, true>(b, P, 2, fp, stream);
  launch_s1_class<TM, ACT, SC, kMaxRunBlocks, true>(b, P, 3, fp, stream);
}


template <int TM, int ACT, int SC, int NWMAX>
void launch_s2(const void* ws, const PlanLayout& P, uint64_t fp, hipStream_t stream) {
  const char* b = static_cast<const char*>(ws);
  hipLaunchKernelGGL((stream_s2_kernel<TM, ACT, SC, NWMAX>), dim3(P.n2), dim3(kThreads), 0, stream,
                     reinterpret_cast<const uint32_t*>(b), reinterpret_cast<const StreamLinear*>(b + P.desc_off),
                     reinterpret_cast<const uint32_t*>(b + P.map2_off), fp);
}

template <int TM, int ACT, int SC>
void launch_s2_nw(const void* ws, const PlanLayout& P, uint64_t fp, hipStream_t stream) {
  // the U words of a lane's rows stay in registers: the class of the list's
  // widest rank sets how many
  if (P.nwmax <= 4)
    launch_s2<TM, ACT, SC, 4>(ws, P, fp, stream);
  else if (P.nwmax <= 8)
    launch_s2<TM, ACT, SC, 8>(ws, P, fp, stream);
  else if (P.nwmax <= 12)
    launch_s2<TM, ACT, SC, 12>(ws, P, fp, stream);
  else if (P.nwmax <= 16)
    launch_s2<TM, ACT, SC, 16>(ws, P, fp, stream);
  else if (P.nwmax <= 24)
    launch_s2<TM, ACT, SC, 24>(ws, P, fp, stream);
  else
    launch_s2<TM, ACT, SC, 32>(ws, P, fp, stream);
}

template <int ACT, int SC>
void launch_all(const void* ws, const PlanLayout& P, uint64_t fp, hipStream_t stream) {
  const char* b = static_cast<const char*>(ws);
  if (P.tm <= 1)
    launch_s1<1, ACT, SC>(ws, P, fp, stream);
  else
    launch_s1<2, ACT, SC>(ws, P, fp, stream);
  hipLaunchKernelGGL(stream_r_kernel, dim3(P.nr), dim3(kThreads), 0, stream, reinterpret_cast<const uint32_t*>(b),
                     reinterpret_cast<const StreamLinear*>(b + P.desc_off),
                     reinterpret_cast<const uint32_t*>(b + P.mapr_off), fp);
  if (P.tm <= 1)
    launch_s2_nw<1, ACT, SC>(ws, P, fp, stream);
  else
    launch_s2_nw<2, ACT, SC>(ws, P, fp, stream);
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

namespace {

bool lut_supports(const ForwardArgs& a) {
  if (!has_work(a)) return true;
  if (a.T > kMaxTokens || a.r > kMaxRank || !decode_supports(a.T, a.d_in, a.d_out, a.r)) return false;
  if (a.d_out > 65535 * kRowsS2 || 2 * a.T * a.r > 65535 * kThreads) return false;
  const DecodeGeom g = decode_geometry(a.T, a.d_in, a.d_out, a.r);
  return g.bpr <= kMaxRunBlocks && g.s1d <= 255;
}

// a list with a linear of more than kMaxTokens tokens runs on the matrix cores
bool list_mma(const ForwardArgs* a, int n) {
  for (int i = 0; i < n; ++i)
    if (has_work(a[i]) && a[i].T > kMaxTokens) return true;
  return false;
}

}  // namespace

bool stream_supports(const ForwardArgs& a) { return lut_supports(a) || stream_mma_supports(a); }

bool stream_list_supports(const ForwardArgs* a, int n) {
  const bool mma = list_mma(a, n);
  for (int i = 0; i < n; ++i)
    if (!(mma ? stream_mma_supports(a[i]) : lut_supports(a[i]))) return false;
  return true;
}

size_t stream_workspace_bytes(const ForwardArgs* a, int n) {
  return list_mma(a, n) ? stream_mma_workspace_bytes(a, n) : plan_layout(a, n).bytes;
}

hipError_t stream_init(const ForwardArgs* a, int n, uint64_t fp, void* ws, hipStream_t stream) {
  if (list_mma(a, n)) return stream_mma_init(a, n, fp, ws, stream);
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
  int i1[4] = {P.n1_cls[0], P.n1_cls[1], P.n1_cls[2], P.n1_cls[3]}, ir = 0, i2 = 0;
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
    const DecodeGeom g = decode_geometry(f.T, f.d_in, f.d_out, f.r);
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
    L.wlat = reinterpret_cast<float*>(data);
    data += align256(sizeof(float) * 2 * f.T * f.r);
    // S1 items grouped by class (one launch each)
    for (int p = 0; p < 2; ++p)
      for (int c = 0; c < g.s1d; ++c) m1[i1[s1_class(f, g, c)]++] = (static_cast<uint32_t>(i) << 16) | (p << 8) | c;
    const int nrb = (2 * f.T * f.r + kThreads - 1) / kThreads;
    for (int j = 0; j < nrb; ++j) mr[ir++] = (static_cast<uint32_t>(i) << 16) | j;
    const int nrow = (f.d_out + kRowsS2 - 1) / kRowsS2;
    for (int j = 0; j < nrow; ++j) m2[i2++] = (static_cast<uint32_t>(i) << 16) | j;
  }
  hipError_t e = hipMemcpyAsync(ws, host.data(), host.size(), hipMemcpyHostToDevice, stream);
  if (e != hipSuccess) return e;
  return hipStreamSynchronize(stream);
}

hipError_t stream_forward(const ForwardArgs* a, int n, uint64_t fp, void* ws, hipStream_t stream) {
  if (list_mma(a, n)) return stream_mma_forward(a, n, fp, ws, stream);
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
