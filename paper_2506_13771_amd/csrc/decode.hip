// Decode kernel (T <= 4 tokens): one launch computes
//   y[t][i] = sum_p h_p[i] sum_k U_p[i][k] l_p[k] z_p[t][k],
//   z_p[t][k] = sum_j V_p[j][k] g_p[j] x[t][j]
// for both paths (Proposition 1, Eq. proposition1; Sec. 3.3 Eq.
// final_weight_approx_res).  Every product with a +-1 sign is exact and all
// sums are fp32.
//
// Sign application by look-up tables: for 4 consecutive reduction indices with
// values a0..a3, a 16-entry table holds every signed sum
// sum_i (bit i of m ? -a_i : +a_i).  A packed 32-bit word (LB layout v1: 32
// consecutive reduction indices of one output) is then 8 nibble look-ups
// instead of 32 sign flips.
//
// At decode sizes each SIMD runs one wave and a wave64 VALU instruction takes
// 4 cycles, so the time of a call is the length of its dependent chain of
// instructions and memory rounds.  The kernel is written for a short chain:
// fixed work per thread (one table and two packed words per stage-1 thread,
// one word per path and row quarter in stage 2), buffer loads (a read past a
// buffer returns zero, so ragged edges need no clamping or masking), 128-bit
// table writes, and one memory round per stage.
//
// Launch structure (one grid, two roles, no host round trip):
//  * stage-1 workgroups hold the LOWEST block ids.  Each owns one path, a tile
//    of 16 latent columns and one run of d_in, processed in chunks of 32
//    blocks of 32 inputs.  Thread tid builds the table of nibble tid % 8 of
//    block tid / 8 (one table per token); lane (kk, m) of wave w looks up the
//    words of column k0 + kk in blocks 8w + m and 8w + m + 4.  The 16 lanes of
//    a column are summed by shuffles (xor 16, xor 32) and the 4 waves in LDS,
//    in a fixed order.  The partial l (.) z of the run goes to the workspace
//    as tagged 64-bit slots (high word: this call's tag, low word: fp32
//    bits), written with relaxed agent-scope atomics, which reach the memory
//    side without any L2 writeback.
//  * stage-2 workgroups (higher ids, dispatched after every stage-1
//    workgroup of their XCD) load their U words and h first, then read the
//    slots with coherent agent-scope loads until every tag is current, sum
//    the partials of each latent in ascending run order while building tables
//    over groups of 4 latents, and contract with U: 4 adjacent lanes share an
//    output row (lane q takes the row's words q, q + 4, ...), a quad butterfly
//    joins them, and lane q stores token q.  Both paths are summed in fp32
//    and y is rounded once.
//  * When the partials are many (large T * r * runs), the highest run of each
//    latent tile first adds the other runs' partials ("two-level" mode), so
//    stage-2 workgroups read one slot per latent.
//  * Waits only ever target workgroups with lower block ids, which are
//    dispatched earlier on every XCD, so the grid cannot deadlock; every wait
//    is bounded and records an error word instead of hanging.
//  * The tag is one more than a per-workspace epoch word; the last stage-2
//    workgroup to finish (counted with one atomic per workgroup) stores it as
//    the new epoch, so consecutive calls, graph replays included, never
//    confuse each other's slots and the workspace needs no clearing.
#include <atomic>
#include <type_traits>

#include "lut_common.h"

namespace lb {

namespace {

using lut::build_table;
using lut::f32x4;
using lut::kBlk;
using lut::kChunk;
using lut::kKey;
using lut::kMaxRuns;
using lut::tsw;
using lut::word_sum;

constexpr int kThreads = 256;
constexpr int kKc = 16;                 // latent columns per stage-1 tile
constexpr int kKQ = 4;                  // stage 2: lanes per output row
constexpr int kRows2 = kThreads / kKQ;  // stage 2: output rows per workgroup
constexpr int kGather = 8;              // stage 2: slots a thread gathers per round
constexpr int kOwnRuns = 4;             // stage 2: runs up to which each table builder loads its own slots
constexpr int kDirectMaxSlots = kThreads * kGather;  // stage 2 reads every partial up to this many
constexpr size_t kLds2Max = 64 * 1024;  // stage-2 LDS budget per token chunk (bytes)

struct DecodeParams {
  const void* x;
  void* y;
  const void* U[2];
  const void* V[2];
  const void* h[2];
  const void* g[2];
  const void* l[2];
  uint32_t* ctrl;
  uint64_t* partial;  // [2][T][s1d][r] tagged partial l (.) z of each run
  uint64_t* wbuf;     // [2][T][r]      tagged l (.) z (two-level mode)
  int T, d_in, d_out, r;
  int nkt;     // 16-latent tiles per path
  int s1d;     // d_in runs per tile
  int bpr;     // 32-input blocks per run
  int n_s1;    // stage-1 workgroups (2 * nkt * s1d)
  int n_s2;    // stage-2 workgroups
  uint32_t* ctr;  // counter of this linear's finished stage-2 workgroups (in the control block, or a
                  // list launch's line of its own)
  int n_members;  // linears of the launch sharing the control block (1: a single call)
  int direct;  // stage 2 reads every run's partial (else the two-level sums)
  int tch;     // tokens per stage-2 chunk
  uint32_t magic_r;  // fast_div multiplier for r
  uint32_t x_bytes, g_bytes, l_bytes, h_bytes, v_bytes, u_bytes;
};

// ---------------------------------------------------------------------------
// stage 1
// ---------------------------------------------------------------------------
template <int TM, int ACT, int SC, bool VEC>
__device__ void stage1(const DecodeParams& P, int wg, float* smem) {
  const int per_path = P.nkt * P.s1d;
  const int p = wg >= per_path ? 1 : 0;
  const int rem = wg - p * per_path;
  const int kt = rem / P.s1d;
  const int c = rem - kt * P.s1d;
  const int T = P.T, r = P.r, d_in = P.d_in;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;  // wave index in a scalar
  const int kk = tid & 15, m = (tid >> 4) & 3;
  const int k = kt * kKc + kk;  // this lane's latent column
  const bool kok = k < r;
  const int nbv = d_in >> 5, tailv = d_in & 31;
  const int nbt = nblocks32(d_in);
  const int b0 = c * P.bpr, b1 = min(nbt, b0 + P.bpr);
  const int tb = tid >> 3, tq = tid & 7;  // builder: table tq of chunk block tb
  const rsrc_t vr = make_rsrc(p ? P.V[1] : P.V[0], P.v_bytes);
  const rsrc_t gr = make_rsrc(p ? P.g[1] : P.g[0], P.g_bytes);
  const rsrc_t xr = make_rsrc(P.x, P.x_bytes);
  float* tbl = smem;  // [TM][kChunk][kBlk]

  const uint32_t lbits = bload<SC>(make_rsrc(p ? P.l[1] : P.l[0], P.l_bytes), k, kok);
  uint32_t epoch = load_epoch<1>(P.ctrl);

  float acc[TM];
#pragma unroll
  for (int t = 0; t < TM; ++t) acc[t] = 0.0f;

  for (int cb = b0; cb < b1; cb += kChunk) {
    // this thread's table inputs: x of each token and g at inputs jb .. jb + 3
    const int jb = 32 * (cb + tb) + 4 * tq;
    const bool tok = cb + tb < b1;
    uint32_t gb[4], xb[TM][4];
    bload4<SC, VEC>(gr, jb, tok, gb);
#pragma unroll
    for (int t = 0; t < TM; ++t) bload4<ACT, VEC>(xr, t * d_in + jb, tok && t < T, xb[t]);
    // this lane's two packed words (blocks 8 wave + m and 8 wave + m + 4)
    uint32_t w[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int b = cb + 8 * wave + m + 4 * u;
      const bool full = kok && b < b1 && b < nbv;
      w[u] = __builtin_amdgcn_raw_buffer_load_b32(vr, full ? static_cast<uint32_t>(b * r + k) * 4u : kOob, 0, 0);
      if (tailv != 0) {
        // the tail block's word comes from the tail plane (16- or 32-bit entries)
        const bool tl = kok && b == nbv && b < b1;
        const uint32_t off = 4u * nbv * r + (tailv <= 16 ? 2u : 4u) * k;
        const uint32_t lo = __builtin_amdgcn_raw_buffer_load_b16(vr, tl ? off : kOob, 0, 0);
        const uint32_t hi = __builtin_amdgcn_raw_buffer_load_b16(vr, tl && tailv > 16 ? off + 2 : kOob, 0, 0);
        w[u] |= (lo & 0xffffu) | (hi << 16);
      }
    }
    // tables of a = x (.) g (zero past d_in and for absent tokens)
#pragma unroll
    for (int t = 0; t < TM; ++t) {
      float a[4];
      lut::table_inputs<ACT, SC, VEC>(xb[t], gb, jb, d_in, tailv, a);
      build_table(tbl + (t * kChunk + tb) * kBlk + 16 * tq, tq, a[0], a[1], a[2], a[3]);
    }
    __syncthreads();
    // look-ups (blocks past the run have zero words and zero tables)
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const uint32_t wk = w[u] ^ kKey;
      const float* tb8 = tbl + (8 * wave + m + 4 * u) * kBlk;
#pragma unroll
      for (int t = 0; t < TM; ++t) acc[t] += word_sum(tb8 + t * kChunk * kBlk, wk);
    }
    __syncthreads();
  }

  // fixed-order sum of the 16 lanes of each column: lanes kk + 16 m within a
  // wave by shuffles, then the 4 waves in LDS
  float* red = smem;  // [4 waves][TM][16]
#pragma unroll
  for (int t = 0; t < TM; ++t) {
    float v = acc[t];
    v += __shfl_xor(v, 16);
    v += __shfl_xor(v, 32);
    if (lane < 16) red[(wave * TM + t) * 16 + lane] = v;
  }
  pin(epoch);
  const uint32_t tag = epoch + 1u;  // this call's tag: one more than the epoch the previous call left
  __syncthreads();
  if (tid < 16 * TM) {
    const int t = tid >> 4;  // tid & 15 == kk: this thread loaded l of its own column
    const float s = lut::tree4(red[(0 * TM + t) * 16 + kk], red[(1 * TM + t) * 16 + kk],
                               red[(2 * TM + t) * 16 + kk], red[(3 * TM + t) * 16 + kk]) *
                    bits_to_f32<SC>(lbits);
    if (t < T && kok) {
      uint64_t* slots = P.partial + static_cast<int64_t>(p * T + t) * P.s1d * r + k;  // [p][t][run][k]
      if (P.direct || c != P.s1d - 1) {
        put_slot(slots + static_cast<int64_t>(c) * r, tag, s);
      } else {
        // two-level mode: the highest run of this tile (it only waits for lower
        // block ids) adds the other runs' partials in ascending order
        float others = 0.0f;
        const bool ok = gather_sum<kMaxRuns>(slots, r, P.s1d - 1, tag, others);
        if (!ok) atomic_store_relaxed(P.ctrl + kCtrlError, 1u);
        put_slot(P.wbuf + static_cast<int64_t>(p * T + t) * r + k, tag, ok ? others + s : __builtin_nanf(""));
      }
    }
  }
}

// ---------------------------------------------------------------------------
// stage 2
// ---------------------------------------------------------------------------
// Sum over the 4 lanes of a row (quad butterfly: xor 1, xor 2).
__device__ __forceinline__ float quad_sum(float v) {
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false));
  return v;
}

// RB blocks of kRows2 output rows per workgroup (list launches take several:
// the gathered partials and their tables serve every block)
template <int TM, int ACT, int SC, int WPL, int RB, bool OWN = false>
__device__ void stage2(const DecodeParams& P, int q2, float* smem) {
  const int tid = threadIdx.x;
  const int kq = tid & (kKQ - 1);
  const int T = P.T, r = P.r, d_out = P.d_out;
  int ir[RB];  // output row of each block
  bool iokr[RB];
#pragma unroll
  for (int b = 0; b < RB; ++b) {
    ir[b] = (q2 * RB + b) * kRows2 + (tid >> 2);
    iokr[b] = ir[b] < d_out;
  }
  const int nw = nblocks32(r), nbu = r >> 5, tailu = r & 31;
  const int nsrc = P.direct ? P.s1d : 1;
  const int R4 = (r + 3) & ~3;  // LDS row of the gathered partials (padded to 16 bytes)
  const int tch = P.tch;
  float* raw = smem;                         // [2][tch][nsrc][R4]
  float* tb2 = smem + 2 * tch * nsrc * R4;   // [2][tch][nw][kBlk]

  // prefetch: this lane's U words (words kq, kq + 4, ... of row i, as two 16-bit
  // halves so that full words and the tail word are the same loads) and h
  uint32_t wlo[RB][2][WPL], whi[RB][2][WPL], hb[RB][2];
  const uint32_t plane = 4u * nbu * d_out;
#pragma unroll
  for (int b = 0; b < RB; ++b) {
    const int i = ir[b];
    const bool iok = iokr[b];
    const uint32_t toff = plane + (tailu <= 16 ? 2u : 4u) * i;
#pragma unroll
    for (int pp = 0; pp < 2; ++pp) {
      const rsrc_t ur = make_rsrc(pp ? P.U[1] : P.U[0], P.u_bytes);
#pragma unroll
      for (int e = 0; e < WPL; ++e) {
        const int kb = kq + kKQ * e;
        const bool full = iok && kb < nbu, tl = iok && kb == nbu && tailu != 0;
        const uint32_t off = full ? static_cast<uint32_t>(kb * d_out + i) * 4u : (tl ? toff : kOob);
        wlo[b][pp][e] = __builtin_amdgcn_raw_buffer_load_b16(ur, off, 0, 0);
        whi[b][pp][e] =
            __builtin_amdgcn_raw_buffer_load_b16(ur, full || (tl && tailu > 16) ? off + 2 : kOob, 0, 0);
      }
      hb[b][pp] = bload<SC>(make_rsrc(pp ? P.h[1] : P.h[0], P.h_bytes), i, iok);
    }
  }
  uint32_t epoch = load_epoch<2>(P.ctrl);
  uint32_t tag = 0u, done_before = 0u;
  bool ok = true;

  // pre-computed split of the builders: row pt = tid / ngrp of 4-latent groups
  const int ngrp = 8 * nw;
  const int bpt = tid / ngrp, bgrp = tid - bpt * ngrp, bstep = kThreads / ngrp;

  // few enough builders for one pass, few runs: every builder thread loads
  // the slots of its own 4 latents itself (no LDS round trip or barrier
  // between the gather and the tables; the sums are the same)
  // (decided on the host: own_builders; OWN = false keeps this path out of the code)
  const bool own = OWN && P.direct && nsrc <= kOwnRuns && 2 * tch * ngrp <= kThreads;

  for (int t0 = 0; t0 < T; t0 += tch) {
    const int tn = min(tch, T - t0);
    if (own) {
      const bool bld = bpt < 2 * tn;
      const int pp = bpt >= tn ? 1 : 0;
      const int tl = bpt - pp * tn;
      const uint64_t* src = P.partial + (static_cast<int64_t>(pp * T + t0 + tl) * nsrc) * r;  // [run][k]
      const bool wave_bld = __builtin_amdgcn_readfirstlane(bpt) < 2 * tn;  // lane 0 builds if any lane does
      uint64_t sv[kOwnRuns][4];
      if (wave_bld) {
        // every load issued at once (a slot this thread does not need reads
        // the first slot of the buffer and is replaced below)
#pragma unroll
        for (int c = 0; c < kOwnRuns; ++c)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const bool need = bld && c < nsrc && 4 * bgrp + j < r;
            sv[c][j] = get_slot(need ? src + c * r + 4 * bgrp + j : P.partial);
          }
      }
      if (t0 == 0) {
        pin(epoch);
        tag = epoch + 1u;
        // count this workgroup as one that has read the epoch (the returned
        // count is used at the end)
        if (tid == 0) done_before = atomic_add_relaxed(P.ctr, 1u);
      }
      if (wave_bld) {
        // a slot not needed counts as ready with value +0 (a sum that starts
        // at +0 is unchanged by adding +0)
        const uint64_t none = static_cast<uint64_t>(tag) << 32;
#pragma unroll
        for (int c = 0; c < kOwnRuns; ++c)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            if (!(bld && c < nsrc && 4 * bgrp + j < r)) sv[c][j] = none;
        for (uint32_t it = 0;; ++it) {
          bool ready = true;
#pragma unroll
          for (int c = 0; c < kOwnRuns; ++c)
#pragma unroll
            for (int j = 0; j < 4; ++j) ready = ready && slot_ready(sv[c][j], tag);
          if (ready) break;
          if (it >= kSpinLimit) {
            ok = false;
            break;
          }
          __builtin_amdgcn_s_sleep(1);
#pragma unroll
          for (int c = 0; c < kOwnRuns; ++c)
#pragma unroll
            for (int j = 0; j < 4; ++j)
              if (!slot_ready(sv[c][j], tag)) sv[c][j] = get_slot(src + c * r + 4 * bgrp + j);
        }
        if (bld) {
          // l (.) z of the 4 latents: their partials in ascending run order (a
          // slot a timed-out wait never saw carrying this call's tag is NaN)
          float w4[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
          for (int c = 0; c < kOwnRuns; ++c)
#pragma unroll
            for (int j = 0; j < 4; ++j) w4[j] += slot_ready(sv[c][j], tag) ? slot_value(sv[c][j]) : __builtin_nanf("");
          build_table(tb2 + ((pp * tch + tl) * nw + (bgrp >> 3)) * kBlk + 16 * (bgrp & 7), bgrp & 7, w4[0], w4[1],
                      w4[2], w4[3]);
        }
      }
      __syncthreads();
    } else {
    // zero the padding of the gathered rows (latents r .. R4 - 1)
    if (R4 != r) {
      for (int e = tid; e < 2 * tch * nsrc * (R4 - r); e += kThreads) {
        const int row = e / (R4 - r);
        raw[row * R4 + r + (e - row * (R4 - r))] = 0.0f;
      }
    }
    // gather both paths' slots of tokens t0 .. t0 + tn - 1 (contiguous per
    // path): rounds of loads, then re-reads of any slot whose tag is not this
    // call's
    const int per_path = tn * nsrc * r;
    const int n = 2 * per_path;
    for (int e0 = 0; e0 < n; e0 += kThreads * kGather) {
      uint64_t sv[kGather];
      const uint64_t* src[kGather];
#pragma unroll
      for (int j = 0; j < kGather; ++j) {
        const int e = e0 + tid + kThreads * j;
        const int pp = e >= per_path ? 1 : 0;
        const int el = e - pp * per_path;
        src[j] = (P.direct ? P.partial + static_cast<int64_t>(pp * T + t0) * nsrc * r
                           : P.wbuf + static_cast<int64_t>(pp * T + t0) * r) + el;
        sv[j] = get_slot(e < n ? src[j] : P.partial);
      }
      if (t0 == 0 && e0 == 0) {
        pin(epoch);
        tag = epoch + 1u;
        // count this workgroup as one that has read the epoch (the returned
        // count is used at the end)
        if (tid == 0) done_before = atomic_add_relaxed(P.ctr, 1u);
      }
      for (uint32_t it = 0;; ++it) {
        bool ready = true;
#pragma unroll
        for (int j = 0; j < kGather; ++j) ready = ready && (e0 + tid + kThreads * j >= n || slot_ready(sv[j], tag));
        if (ready) break;
        if (it >= kSpinLimit) {
          ok = false;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
#pragma unroll
        for (int j = 0; j < kGather; ++j)
          if (e0 + tid + kThreads * j < n && !slot_ready(sv[j], tag)) sv[j] = get_slot(src[j]);
      }
#pragma unroll
      for (int j = 0; j < kGather; ++j) {
        const int e = e0 + tid + kThreads * j;
        if (e < n) {
          const int pp = e >= per_path ? 1 : 0;
          const int el = e - pp * per_path;
          const int row = static_cast<int>(fast_div(static_cast<uint32_t>(el), P.magic_r));  // tl * nsrc + run
          // a slot a timed-out wait never saw carrying this call's tag is NaN
          raw[(pp * tch * nsrc + row) * R4 + (el - row * r)] =
              slot_ready(sv[j], tag) ? slot_value(sv[j]) : __builtin_nanf("");
        }
      }
    }
    __syncthreads();
    // l (.) z of 4 latents = the sum of their partials (ascending run order),
    // then the nibble table over them
    for (int pt = bpt; bpt < bstep && pt < 2 * tn; pt += bstep) {
      const int pp = pt >= tn ? 1 : 0;
      const int tl = pt - pp * tn;
      f32x4 w4 = {0.0f, 0.0f, 0.0f, 0.0f};
      if (4 * bgrp < R4) {
        const float* rs = raw + ((pp * tch + tl) * nsrc) * R4 + 4 * bgrp;
        for (int cc = 0; cc < nsrc; ++cc) w4 += *reinterpret_cast<const f32x4*>(rs + cc * R4);
      }
      build_table(tb2 + ((pp * tch + tl) * nw + (bgrp >> 3)) * kBlk + 16 * (bgrp & 7), bgrp & 7, w4[0], w4[1],
                  w4[2], w4[3]);
    }
    __syncthreads();
    }
    // contraction of row i with both paths; lane kq covers words kq, kq + 4, ...
#pragma unroll
    for (int b = 0; b < RB; ++b) {
      float acc[2][TM];
#pragma unroll
      for (int pp = 0; pp < 2; ++pp)
#pragma unroll
        for (int t = 0; t < TM; ++t) acc[pp][t] = 0.0f;
#pragma unroll
      for (int pp = 0; pp < 2; ++pp)
#pragma unroll
        for (int e = 0; e < WPL; ++e) {
          const int kb = kq + kKQ * e;
          if (kb < nw) {
            const uint32_t wk = ((wlo[b][pp][e] & 0xffffu) | (whi[b][pp][e] << 16)) ^ kKey;
#pragma unroll
            for (int t = 0; t < TM; ++t)
              if (t < tn) acc[pp][t] += word_sum(tb2 + ((pp * tch + t) * nw + kb) * kBlk, wk);
          }
        }
      const float h0 = bits_to_f32<SC>(hb[b][0]), h1 = bits_to_f32<SC>(hb[b][1]);
#pragma unroll
      for (int t = 0; t < TM; ++t) {
        const float v = lut::row_value(h0, quad_sum(acc[0][t]), h1, quad_sum(acc[1][t]));
        if (iokr[b] && t < tn && kq == t) st<ACT>(P.y, static_cast<int64_t>(t0 + t) * d_out + ir[b], v);
      }
    }
    __syncthreads();  // the next token chunk reuses the LDS
  }
  if (!ok) atomic_store_relaxed(P.ctrl + kCtrlError, 1u);

  // The last stage-2 workgroup to count itself stores the tag as the epoch
  // for the next call.  Every workgroup of this call has read the epoch by
  // then: stage-2 workgroups counted themselves after reading it, and every
  // stage-1 workgroup published values carrying the tag, which this
  // workgroup has gathered (directly, or through the two-level reducers).
  // In a list launch each linear counts its workgroups on a word of its own
  // (one contended word for all of them would serialise the atomics), and the
  // last workgroup of each linear counts that linear on the shared word.
  if (tid == 0 && done_before == static_cast<uint32_t>(P.n_s2 - 1)) {
    atomic_store_relaxed(P.ctr, 0u);
    const bool last = P.n_members <= 1 ||
                      atomic_add_relaxed(P.ctrl + kCtrlDone, 1u) == static_cast<uint32_t>(P.n_members - 1);
    if (last) {
      if (P.n_members > 1) atomic_store_relaxed(P.ctrl + kCtrlDone, 0u);
      atomic_store_relaxed(P.ctrl + kCtrlEpoch, tag);
    }
  }
}

template <int TM, int ACT, int SC, bool VEC, int WPL, bool OWN>
__global__ void __launch_bounds__(kThreads, 2) decode_kernel(DecodeParams P) {
  extern __shared__ __attribute__((aligned(16))) float smem[];
  const int wg = blockIdx.x;
  if (wg < P.n_s1)
    stage1<TM, ACT, SC, VEC>(P, wg, smem);
  else
    stage2<TM, ACT, SC, WPL, 1, OWN>(P, wg - P.n_s1, smem);
}

// A list of independent linears in one launch: the stage-1 workgroups of
// every linear first (linear 0's, then linear 1's, ...), then the stage-2
// workgroups in the same order, so every wait still targets lower block ids.
// Each linear keeps its own workspace slice and call protocol; one
// instantiation serves all of them (TM, WPL: the largest of the list; VEC:
// only when every member is aligned; stage 2 masks the words a rank does
// not have).
// stage 2 of a list launch: blocks of kRows2 rows per workgroup (fewer for
// wide ranks, whose U words of several blocks would not stay in registers)
__host__ __device__ constexpr int batch_rows(int wpl) { return wpl <= 2 ? 4 : (wpl <= 4 ? 2 : 1); }
// ... for one-token lists only (the tables of more tokens leave no registers)
__host__ __device__ constexpr int list_rows(int tm, int wpl) { return tm == 1 ? batch_rows(wpl) : 1; }

// A list launch with more stage-1 workgroups than this goes out as two
// launches: every stage-1 workgroup first, in a kernel of its own, which needs
// far fewer registers than stage 2 (204 for a one-token list at four words per
// lane: 2 workgroups per CU), so that several times the workgroups per CU
// overlap their load latencies; then the stage-2 workgroups, whose waits then
// find every partial already published.
constexpr int kSplitMinS1 = 1024;

struct DecodeBatch {
  int n;
  int wg0;                      // list block id of this launch's first workgroup
  int s1_end[kDecodeMaxBatch];  // one past each linear's last stage-1 workgroup
  int s2_end[kDecodeMaxBatch];  // the same for stage 2, counted from the first stage-2 workgroup
  DecodeParams p[kDecodeMaxBatch];
};

template <int TM, int ACT, int SC, bool VEC, int WPL>
__global__ void __launch_bounds__(kThreads, 2) decode_batch_kernel(DecodeBatch B) {
  extern __shared__ __attribute__((aligned(16))) float smem[];
  const int wg = blockIdx.x + B.wg0;
  const int s1tot = B.s1_end[B.n - 1];
  if (wg < s1tot) {
    int i = 0;
    while (wg >= B.s1_end[i]) ++i;
    const DecodeParams P = B.p[i];
    stage1<TM, ACT, SC, VEC>(P, wg - (i ? B.s1_end[i - 1] : 0), smem);
  } else {
    const int w2 = wg - s1tot;
    int i = 0;
    while (w2 >= B.s2_end[i]) ++i;
    const DecodeParams P = B.p[i];
    stage2<TM, ACT, SC, WPL, list_rows(TM, WPL)>(P, w2 - (i ? B.s2_end[i - 1] : 0), smem);
  }
}

// the stage-1 workgroups of a list alone (grid: the list's stage-1 total)
template <int TM, int ACT, int SC, bool VEC>
__global__ void __launch_bounds__(kThreads) decode_batch_s1_kernel(DecodeBatch B) {
  extern __shared__ __attribute__((aligned(16))) float smem[];
  const int wg = blockIdx.x;
  int i = 0;
  while (wg >= B.s1_end[i]) ++i;
  const DecodeParams P = B.p[i];
  stage1<TM, ACT, SC, VEC>(P, wg - (i ? B.s1_end[i - 1] : 0), smem);
}

// whether stage 2 of a single call takes the path in which each table
// builder loads its own slots (the condition stage2 checks again)
inline bool own_builders(const DecodeParams& P) {
  const int nsrc = P.direct ? P.s1d : 1;
  return P.direct && nsrc <= kOwnRuns && 2 * P.tch * 8 * nblocks32(P.r) <= kThreads;
}

// one launch of the single-linear (DecodeParams) or list (DecodeBatch) kernel
template <int TM, int ACT, int SC, bool VEC, int WPL, typename A>
hipError_t launch_one(const A& args, dim3 grid, size_t smem, hipStream_t stream) {
  constexpr bool kOne = std::is_same<A, DecodeParams>::value;
  // more than the default dynamic LDS limit: raise the kernel's limit once per
  // size increase, so calls captured in a graph after an eager call of the
  // same shape make no attribute call
  static std::atomic<size_t> limit{65536};
  if (smem > limit.load()) {
    hipError_t e = hipSuccess;
    if constexpr (kOne) {
      e = hipFuncSetAttribute(reinterpret_cast<const void*>(&decode_kernel<TM, ACT, SC, VEC, WPL, false>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(smem));
      if (e == hipSuccess)
        e = hipFuncSetAttribute(reinterpret_cast<const void*>(&decode_kernel<TM, ACT, SC, VEC, WPL, true>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(smem));
    } else {
      e = hipFuncSetAttribute(reinterpret_cast<const void*>(&decode_batch_kernel<TM, ACT, SC, VEC, WPL>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(smem));
    }
    if (e != hipSuccess) return e;
    limit.store(smem);
  }
  if constexpr (kOne) {
    if (own_builders(args))
      hipLaunchKernelGGL((decode_kernel<TM, ACT, SC, VEC, WPL, true>), grid, dim3(kThreads), smem, stream, args);
    else
      hipLaunchKernelGGL((decode_kernel<TM, ACT, SC, VEC, WPL, false>), grid, dim3(kThreads), smem, stream, args);
  } else {
    const int s1 = args.s1_end[args.n - 1];
    if (s1 <= kSplitMinS1) {
      hipLaunchKernelGGL((decode_batch_kernel<TM, ACT, SC, VEC, WPL>), grid, dim3(kThreads), smem, stream, args);
    } else {
      // stage 1 alone: its tables of TM tokens are all the LDS it needs
      constexpr size_t smem1 = sizeof(float) * TM * kChunk * kBlk;
      static std::atomic<size_t> limit1{65536};
      if (smem1 > limit1.load()) {
        const hipError_t e =
            hipFuncSetAttribute(reinterpret_cast<const void*>(&decode_batch_s1_kernel<TM, ACT, SC, VEC>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(smem1));
        if (e != hipSuccess) return e;
        limit1.store(smem1);
      }
      hipLaunchKernelGGL((decode_batch_s1_kernel<TM, ACT, SC, VEC>), dim3(s1), dim3(kThreads), smem1, stream, args);
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess || static_cast<int>(grid.x) <= s1) return e;
      DecodeBatch b2 = args;
      b2.wg0 = s1;
      hipLaunchKernelGGL((decode_batch_kernel<TM, ACT, SC, VEC, WPL>), dim3(grid.x - s1), dim3(kThreads), smem, stream,
                         b2);
    }
  }
  return hipGetLastError();
}

template <int TM, int ACT, int SC, bool VEC, typename A>
hipError_t launch_wpl(const A& args, int wpl, dim3 grid, size_t smem, hipStream_t stream) {
  switch (wpl) {
    case 1: return launch_one<TM, ACT, SC, VEC, 1>(args, grid, smem, stream);
    case 2: return launch_one<TM, ACT, SC, VEC, 2>(args, grid, smem, stream);
    case 4: return launch_one<TM, ACT, SC, VEC, 4>(args, grid, smem, stream);
    default: return launch_one<TM, ACT, SC, VEC, 8>(args, grid, smem, stream);
  }
}

template <int ACT, int SC, typename A>
hipError_t launch_typed(const A& args, int T, bool vec, int wpl, dim3 grid, size_t smem, hipStream_t stream) {
  // x and g read as 4-element vectors when aligned (decided on the host); the
  // element-wise form is compiled for the widest token count only
  if (!vec) return launch_wpl<kDecodeMaxTokens, ACT, SC, false>(args, wpl, grid, smem, stream);
  if (T <= 1) return launch_wpl<1, ACT, SC, true>(args, wpl, grid, smem, stream);
  if (T <= 2) return launch_wpl<2, ACT, SC, true>(args, wpl, grid, smem, stream);
  return launch_wpl<4, ACT, SC, true>(args, wpl, grid, smem, stream);
}

template <int ACT, typename A>
hipError_t launch_act(const A& args, int T, int sc_dt, bool vec, int wpl, dim3 grid, size_t smem,
                      hipStream_t stream) {
  switch (sc_dt) {
    case kDtF32: return launch_typed<ACT, kDtF32>(args, T, vec, wpl, grid, smem, stream);
    case kDtF16: return launch_typed<ACT, kDtF16>(args, T, vec, wpl, grid, smem, stream);
    default: return launch_typed<ACT, kDtBF16>(args, T, vec, wpl, grid, smem, stream);
  }
}

template <typename A>
hipError_t launch_any(const A& args, int act_dt, int T, int sc_dt, bool vec, int wpl, dim3 grid, size_t smem,
                      hipStream_t stream) {
  switch (act_dt) {
    case kDtF32: return launch_act<kDtF32>(args, T, sc_dt, vec, wpl, grid, smem, stream);
    case kDtF16: return launch_act<kDtF16>(args, T, sc_dt, vec, wpl, grid, smem, stream);
    default: return launch_act<kDtBF16>(args, T, sc_dt, vec, wpl, grid, smem, stream);
  }
}

size_t align256(size_t b) { return (b + 255) / 256 * 256; }

int64_t packed_bytes(int64_t n_out, int64_t n_red) {
  const int64_t w = n_red & 31;
  return 4 * (n_red >> 5) * n_out + (w == 0 ? 0 : (w <= 16 ? 2 : 4)) * n_out;
}

size_t stage2_floats_per_token(int r, int nsrc) {
  const size_t R4 = (static_cast<size_t>(r) + 3) & ~static_cast<size_t>(3);
  return 2 * (static_cast<size_t>(nsrc) * R4 + static_cast<size_t>(nblocks32(r)) * kBlk);
}

int tm_of(int T) { return T <= 1 ? 1 : (T <= 2 ? 2 : 4); }

}  // namespace

DecodeGeom decode_geometry(int T, int d_in, int d_out, int r) {
  DecodeGeom g{};
  const int tt = T > 0 ? T : 1;
  g.nkt = (r + kKc - 1) / kKc;
  const int nbt = nblocks32(d_in);
  int s1d = (nbt + kChunk - 1) / kChunk;
  if (s1d > kMaxRuns) s1d = kMaxRuns;
  if (s1d < 1) s1d = 1;
  g.bpr = nbt > 0 ? (nbt + s1d - 1) / s1d : 1;
  g.s1d = nbt > 0 ? (nbt + g.bpr - 1) / g.bpr : 1;
  g.n_s1 = 2 * g.nkt * g.s1d;
  g.direct = g.s1d == 1 || static_cast<int64_t>(2) * tt * g.s1d * r <= kDirectMaxSlots;
  const int nsrc = g.direct ? g.s1d : 1;
  const size_t per_tok = stage2_floats_per_token(r, nsrc);
  int tch = per_tok > 0 ? static_cast<int>(kLds2Max / (4 * per_tok)) : tt;
  if (tch > tt) tch = tt;
  if (tch < 1) tch = 1;
  g.tch = tch;
  g.n_s2 = (d_out + kRows2 - 1) / kRows2;
  const int nw = nblocks32(r);
  g.wpl = nw <= kKQ ? 1 : (nw <= 2 * kKQ ? 2 : (nw <= 4 * kKQ ? 4 : 8));
  // LDS: stage-1 tables of tm_of(T) tokens (of kDecodeMaxTokens for the
  // element-wise variant, smem_bytes_elem), stage-2 gathered partials and tables
  const size_t s1 = static_cast<size_t>(4) * tm_of(tt) * kChunk * kBlk;
  const size_t s1e = static_cast<size_t>(4) * kDecodeMaxTokens * kChunk * kBlk;
  const size_t s2 = 4 * tch * per_tok;
  g.smem_bytes = s1 > s2 ? s1 : s2;
  g.smem_bytes_elem = s1e > s2 ? s1e : s2;
  g.partial_off = kCtrlBytes;
  g.partial_slots = static_cast<size_t>(2) * g.s1d * T * r;
  g.wbuf_off = g.partial_off + align256(8 * g.partial_slots);
  g.wbuf_slots = g.direct ? 0 : static_cast<size_t>(2) * T * r;
  g.ws_bytes = g.wbuf_off + align256(8 * g.wbuf_slots);
  return g;
}

bool decode_supports(int64_t T, int64_t d_in, int64_t d_out, int64_t r) {
  // buffer offsets are 32-bit: every operand stays below 2^31 bytes
  const int64_t lim = int64_t(1) << 31;
  return T <= kDecodeMaxTokens && r <= kDecodeMaxRank && T * d_in * 4 < lim && packed_bytes(d_out, r) < lim &&
         packed_bytes(r, d_in) < lim && d_out * 4 < lim && d_in * 4 < lim;
}

namespace {

// kernel parameters of one linear; returns whether x and g may be read as
// 4-element vectors
bool decode_params(const ForwardArgs& a, const DecodeGeom& g, DecodeParams& P) {
  P = DecodeParams{};
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
  P.ctrl = reinterpret_cast<uint32_t*>(a.ctrl ? a.ctrl : a.ws);
  P.partial = reinterpret_cast<uint64_t*>(ws + g.partial_off);
  P.wbuf = reinterpret_cast<uint64_t*>(ws + g.wbuf_off);
  P.T = a.T;
  P.d_in = a.d_in;
  P.d_out = a.d_out;
  P.r = a.r;
  P.nkt = g.nkt;
  P.s1d = g.s1d;
  P.bpr = g.bpr;
  P.n_s1 = g.n_s1;
  P.n_s2 = g.n_s2;
  P.ctr = P.ctrl + kCtrlDone;
  P.n_members = 1;
  P.direct = g.direct;
  P.tch = g.tch;
  P.magic_r = a.r > 1 ? static_cast<uint32_t>(((uint64_t(1) << 32) + a.r - 1) / a.r) : 0u;
  const int64_t ex = a.act_dt == kDtF32 ? 4 : 2, es = a.sc_dt == kDtF32 ? 4 : 2;
  P.x_bytes = static_cast<uint32_t>(static_cast<int64_t>(a.T) * a.d_in * ex);
  P.g_bytes = static_cast<uint32_t>(a.d_in * es);
  P.h_bytes = static_cast<uint32_t>(a.d_out * es);
  P.l_bytes = static_cast<uint32_t>(a.r * es);
  P.v_bytes = static_cast<uint32_t>(packed_bytes(a.r, a.d_in));
  P.u_bytes = static_cast<uint32_t>(packed_bytes(a.d_out, a.r));
  const uintptr_t xa = 4 * ex, ga = 4 * es;
  return (reinterpret_cast<uintptr_t>(a.x) % xa == 0) && (a.d_in % 4 == 0) &&
         (reinterpret_cast<uintptr_t>(a.g[0]) % ga == 0) && (reinterpret_cast<uintptr_t>(a.g[1]) % ga == 0);
}

}  // namespace

hipError_t launch_decode(const ForwardArgs& a, const DecodeGeom& g, hipStream_t stream) {
  DecodeParams P;
  const bool vec = decode_params(a, g, P);
  const dim3 grid(g.n_s1 + g.n_s2);
  const size_t smem = vec ? g.smem_bytes : g.smem_bytes_elem;
  return launch_any(P, a.act_dt, a.T, a.sc_dt, vec, g.wpl, grid, smem, stream);
}

hipError_t launch_decode_batch(const ForwardArgs* a, int n, hipStream_t stream) {
  if (n <= 0 || n > kDecodeMaxBatch) return hipErrorInvalidValue;
  DecodeBatch B{};
  B.n = n;
  bool vec = true;
  int T = 0, wpl = 1, s1 = 0, s2 = 0;
  size_t smem_vec = 0, smem_elem = 0;
  for (int i = 0; i < n; ++i) {
    if (a[i].act_dt != a[0].act_dt || a[i].sc_dt != a[0].sc_dt) return hipErrorInvalidValue;
    const DecodeGeom g = decode_geometry(a[i].T, a[i].d_in, a[i].d_out, a[i].r);
    vec = decode_params(a[i], g, B.p[i]) && vec;
    T = a[i].T > T ? a[i].T : T;
    wpl = g.wpl > wpl ? g.wpl : wpl;
    smem_vec = g.smem_bytes > smem_vec ? g.smem_bytes : smem_vec;
    smem_elem = g.smem_bytes_elem > smem_elem ? g.smem_bytes_elem : smem_elem;
    s1 += g.n_s1;
    B.s1_end[i] = s1;
  }
  // batch_rows row blocks per stage-2 workgroup (the list's widest rank
  // decides); the call protocol counts that many workgroups
  // the token count the launch instantiates (as launch_typed chooses it)
  const int tm = !vec ? kDecodeMaxTokens : (T <= 1 ? 1 : (T <= 2 ? 2 : 4));
  const int rb = list_rows(tm, wpl);
  for (int i = 0; i < n; ++i) {
    B.p[i].n_s2 = (B.p[i].n_s2 + rb - 1) / rb;
    s2 += B.p[i].n_s2;
    B.s2_end[i] = s2;
  }
  // members that share a control block end the call together: each counts
  // its stage-2 workgroups on a line of its own after the control block, the
  // last member to finish stores the epoch
  for (int i = 0; i < n; ++i) {
    int cnt = 0;
    for (int j = 0; j < n; ++j) cnt += B.p[j].ctrl == B.p[i].ctrl ? 1 : 0;
    if (cnt > 1) {
      B.p[i].ctr = reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(B.p[i].ctrl) + kCtrlBytes +
                                               kListCtrStride * static_cast<size_t>(i));
      B.p[i].n_members = cnt;
    }
  }
  return launch_any(B, a[0].act_dt, T, a[0].sc_dt, vec, wpl, dim3(s1 + s2), vec ? smem_vec : smem_elem, stream);
}

}  // namespace lb
