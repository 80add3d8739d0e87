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
// instead of 32 sign flips.  Tables are built in LDS, once per workgroup, for
// the activations of that workgroup's inputs.
//
// Launch structure (one grid, two roles, no host round trip, latency-first):
//  * stage-1 workgroups hold the LOWEST block ids.  Each owns one path, a tile
//    of 16 latent columns and one run of d_in.  All of its global loads (V
//    words, x, g, l) are issued before any is waited on.  Lane (kk, bs) takes
//    column k0 + kk and every 16th 32-wide block of the run; the 16 groups are
//    combined by cross-lane shuffles and a 4-way LDS sum in a fixed order.  The
//    partial l (.) z goes to the workspace as tagged 64-bit slots (high word:
//    this call's tag, low word: fp32 bits), written with relaxed agent-scope
//    atomics, which reach the memory side without any L2 writeback.
//  * stage-2 workgroups (higher ids, so dispatched after every stage-1
//    workgroup of their XCD) load their U words and h first, then read the
//    slots with coherent agent-scope loads until every tag is current, sum the
//    partials of each latent in a fixed order, build tables over groups of 4
//    latents and contract with U.  KQ adjacent lanes share an output row and
//    split its words; a butterfly joins them.  Both paths are summed in fp32
//    and y is stored once.
//  * When the partials are many (large T * r), the highest-id run of each
//    latent tile first adds the other runs' partials ("two-level" mode), so
//    stage-2 workgroups read one slot per latent.
//  * Waits only ever target workgroups with lower block ids, which are
//    dispatched earlier on every XCD, so the grid cannot deadlock; every wait
//    is bounded and records an error word instead of hanging.
//  * The tag is one more than a per-workspace epoch word; the last stage-2
//    workgroup to finish (counted with one atomic per workgroup) stores it as
//    the new epoch, so consecutive calls, graph replays included, never
//    confuse each other's slots and the workspace needs no clearing.
#include "device_common.h"

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
  uint64_t* partial;  // [2][T][s1d][r] tagged partial l (.) z
  uint64_t* wbuf;     // [2][T][r]      tagged l (.) z (two-level mode)
  int act_dt, sc_dt;
  int x_vec, g_vec;   // 4-element vector loads allowed for x / g
  int T, d_in, d_out, r;
  int nkt, bpw, s1d, n_s1, cb;
  int kq_log2, rows2, n_s2, direct, tch;
};

constexpr int kThreads = 256;
constexpr int kKc = 16;                 // latent columns per stage-1 tile
constexpr int kMaxSplit = 16;           // d_in runs per latent tile (partials per z value)
constexpr int kMaxWordsPerLane = 8;     // stage 1: V words a lane holds in registers per chunk
constexpr int kMaxGroupsPerThread = 3;  // stage 1: table groups a thread builds per chunk
constexpr int kRowWords = 2;            // stage 2: U words per row a lane holds (per path)
constexpr int kMaxPasses = 4;           // stage 2: rows per lane (2 for T > 2: register budget)
__host__ __device__ constexpr int max_passes(int tm) { return tm > 2 ? 2 : kMaxPasses; }
constexpr int kSlotsPerPath = 4;        // stage 2: slots a thread gathers per path in one round
constexpr int kLutBlock = 8 * 16 + 16;  // floats per 32-wide block of tables (padded: bank spread)
constexpr int kLdsFloats = 12288;       // 48 KB of dynamic LDS

// Nibble tables.  Block B of the table array holds the 8 tables (16 floats
// each, kLutBlock floats in all) of one 32-wide block of inputs; table q of
// block B is stored XOR-swizzled: entry m sits at position m ^ swz(B, q),
// swz(B, q) = (2 B + q / 4) mod 16.  A wave's builders (consecutive tables)
// then spread their writes over the LDS banks instead of hitting the same two
// (32-way conflicts unswizzled), and a lookup applies the same swizzle to the
// whole packed word with one XOR (word_key).
__device__ __forceinline__ int table_swizzle(int B, int q) { return (2 * B + (q >> 2)) & 15; }
__device__ __forceinline__ uint32_t word_key(int B) {
  return static_cast<uint32_t>((2 * B) & 15) * 0x11111111u ^ 0x11110000u;
}

// Table q of block B: entry m = sum_i (bit i of m ? -a_i : +a_i), built as
// (+-a0 +-a1) + (+-a2 +-a3), written at its swizzled position.
__device__ __forceinline__ void build_lut16(float a0, float a1, float a2, float a3, float* lut, int B, int q) {
  const float p01[4] = {a0 + a1, -a0 + a1, a0 - a1, -a0 - a1};
  const float p23[4] = {a2 + a3, -a2 + a3, a2 - a3, -a2 - a3};
  float* tb = lut + B * kLutBlock + 16 * q;
  const int sw = table_swizzle(B, q);
#pragma unroll
  for (int m = 0; m < 16; ++m) tb[m ^ sw] = p01[m & 3] + p23[m >> 2];
}

// Signed sum of one packed word against the 8 tables of block B (8
// independent reads, summed as a fixed tree).
__device__ __forceinline__ float word_dot(const float* lut, int B, uint32_t w) {
  const float* tb = lut + B * kLutBlock;
  const uint32_t k = w ^ word_key(B);
  float v[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) v[q] = tb[16 * q + ((k >> (4 * q)) & 15)];
  return ((v[0] + v[1]) + (v[2] + v[3])) + ((v[4] + v[5]) + (v[6] + v[7]));
}

// Sum over the KQ lanes (adjacent, power of two, 4..16) that share an output row.
__device__ __forceinline__ float row_sum(float v, int kq_log2) {
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));  // xor 1
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false));  // xor 2
  if (kq_log2 >= 3) v += __shfl_xor(v, 4);
  if (kq_log2 >= 4) v += __shfl_xor(v, 8);
  return v;
}

// ---------------------------------------------------------------------------
// stage 1
// ---------------------------------------------------------------------------
template <int TM, int ACT, int SC, bool VEC>
__device__ void stage1(const DecodeParams& P, int wg, float* smem) {
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
  const int tid = threadIdx.x;
  const int kk = tid & (kKc - 1);
  const int bs = tid >> 4;
  const bool col_ok = kk < kcn;
  const int CB = P.cb;
  // per-path pointers chosen by selects (no dynamic indexing into the parameters)
  const void* Vp = p ? P.V[1] : P.V[0];
  const void* gp = p ? P.g[1] : P.g[0];
  const void* lp = p ? P.l[1] : P.l[0];
  const uint32_t* Vw = static_cast<const uint32_t*>(Vp);
  const int nbv = d_in >> 5, tailv = d_in & 31;
  float* lut = smem;  // [T][CB][kLutBlock]

  uint32_t lk_bits = 0u;  // latent scale of this lane's column (raw)
  uint32_t epoch = 0u;    // the epoch left by the previous call (this call's tag is one more)
  float acc[TM];
#pragma unroll
  for (int t = 0; t < TM; ++t) acc[t] = 0.0f;

  for (int cb = b0; cb < b1; cb += CB) {
    const int nblk = min(CB, b1 - cb);
    const int ngroups = T * nblk * 8;
    // Every load of the chunk is issued before any value is used, at clamped
    // addresses, with validity applied afterwards: one memory round per chunk.
    // x and g by groups of 4 inputs (group e: token t, inputs j0..j0+3)
    uint32_t xr[kMaxGroupsPerThread][4], gr[kMaxGroupsPerThread][4];
#pragma unroll
    for (int gi = 0; gi < kMaxGroupsPerThread; ++gi) {
      const int e = tid + kThreads * gi;
      const int t = e / (nblk * 8);
      const int j0 = 32 * cb + 4 * (e - t * nblk * 8);  // 32 (cb + bl) + 4 q
      const int nvalid = e < ngroups ? min(4, d_in - j0) : 0;
      ld4_bits<ACT, VEC>(P.x, nvalid > 0 ? static_cast<int64_t>(t) * d_in + j0 : 0, nvalid, xr[gi]);
      ld4_bits<SC, VEC>(gp, nvalid > 0 ? j0 : 0, nvalid, gr[gi]);
    }
    // the latent scale (used once the partials, which carry l (.) z, are formed)
    lk_bits = ld_bits<SC>(lp, col_ok ? k0 + kk : 0);
    epoch = load_epoch<1>(P.ctrl);
    // the tail word of d_in (if this chunk holds the tail block)
    const int tail_bl = nbv - cb;  // local index of the tail block (when < nblk)
    uint32_t tlo, thi;
    ld_tail_bits(Vw, nbv, r, tailv, k0 + kk, col_ok && tail_bl < nblk, tlo, thi);
    // full V words
    const uint32_t* Vfull = full_words_or(Vw, nbv, P.ctrl);
    uint32_t words[kMaxWordsPerLane];
#pragma unroll
    for (int u = 0; u < kMaxWordsPerLane; ++u) {
      const int bl = bs + 16 * u;
      const bool ok = col_ok && bl < nblk && bl < tail_bl;
      words[u] = Vfull[ok ? static_cast<int64_t>(cb + bl) * r + k0 + kk : 0];
    }
    // keep the loads above and the uses of x, g and the tail below
    asm volatile("" ::: "memory");
#pragma unroll
    for (int gi = 0; gi < kMaxGroupsPerThread; ++gi)
#pragma unroll
      for (int i = 0; i < 4; ++i) pin(xr[gi][i]), pin(gr[gi][i]);
    pin(tlo), pin(thi);
    const uint32_t tailword = tail_word(tlo, thi, tailv);
    // nibble tables of a = x (.) g_p (zero beyond d_in)
#pragma unroll
    for (int gi = 0; gi < kMaxGroupsPerThread; ++gi) {
      const int e = tid + kThreads * gi;
      if (e < ngroups) {
        const int t = e / (nblk * 8);
        const int rem2 = e - t * nblk * 8;
        const int j0 = 32 * cb + 4 * rem2;
        float a[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
          a[i] = j0 + i < d_in ? raw4_elem<ACT, VEC>(xr[gi], i) * raw4_elem<SC, VEC>(gr[gi], i) : 0.0f;
        build_lut16(a[0], a[1], a[2], a[3], lut, t * CB + (rem2 >> 3), rem2 & 7);
      }
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kMaxWordsPerLane; ++u) {
      const int bl = bs + 16 * u;
      if (col_ok && bl < nblk) {
        const uint32_t w = bl == tail_bl ? tailword : words[u];
#pragma unroll
        for (int t = 0; t < TM; ++t)
          if (t < T) acc[t] += word_dot(lut, t * CB + bl, w);
      }
    }
    __syncthreads();
  }
  const float lk = bits_to_f32<SC>(lk_bits);
  // this call's tag: one more than the epoch the previous call left behind
  pin(epoch);
  const uint32_t tag = epoch + 1u;

  // fixed-order reduction over the 16 block groups: within a wave by shuffles
  // (groups 4w..4w+3 sit in lane bands of 16), then across the 4 waves in LDS
  float* red = smem;  // [4 waves][T][kKc]
#pragma unroll
  for (int t = 0; t < TM; ++t) {
    float v = col_ok ? acc[t] * lk : 0.0f;
    v += __shfl_xor(v, 16);
    v += __shfl_xor(v, 32);
    acc[t] = v;
  }
  if ((tid & 63) < kKc) {
#pragma unroll
    for (int t = 0; t < TM; ++t)
      if (t < T) red[((tid >> 6) * T + t) * kKc + kk] = acc[t];
  }
  __syncthreads();
  const bool reducer = !P.direct && c == P.s1d - 1;
  for (int e = tid; e < T * kcn; e += kThreads) {
    const int t = e / kcn;
    const int k = e - t * kcn;
    const float s = (red[(0 * T + t) * kKc + k] + red[(1 * T + t) * kKc + k]) +
                    (red[(2 * T + t) * kKc + k] + red[(3 * T + t) * kKc + k]);
    // slots of (p, t): [s1d][r]
    uint64_t* pt_slots = P.partial + (static_cast<int64_t>(p) * T + t) * P.s1d * r + k0 + k;
    if (!reducer) {
      put_slot(pt_slots + static_cast<int64_t>(c) * r, tag, s);
    } else {
      // two-level mode: the highest run of this latent tile (it only waits for
      // lower block ids) adds the other runs' partials in ascending order
      float others = 0.0f;
      const bool ok = gather_sum<kMaxSplit>(pt_slots, r, P.s1d - 1, tag, others);
      if (!ok) atomic_store_relaxed(P.ctrl + kCtrlError, 1u);
      put_slot(P.wbuf + (static_cast<int64_t>(p) * T + t) * r + k0 + k, tag, ok ? others + s : __builtin_nanf(""));
    }
  }
}

// ---------------------------------------------------------------------------
// stage 2
// ---------------------------------------------------------------------------
template <int TM, int ACT, int SC>
__device__ void stage2(const DecodeParams& P, int q, float* smem) {
  const int tid = threadIdx.x;
  const int kq_log2 = P.kq_log2;
  const int KQ = 1 << kq_log2;
  const int rows_per_pass = kThreads >> kq_log2;
  const int rl = tid >> kq_log2;
  const int kq = tid & (KQ - 1);
  const int T = P.T, r = P.r, d_out = P.d_out;
  const int nw = nblocks32(r);
  const int i_base = q * P.rows2 + rl;
  const int passes = P.rows2 / rows_per_pass;
  const int nsrc = P.direct ? P.s1d : 1;  // slots per latent value
  float* raw = smem;                                      // [2][tch][nsrc][r] slot values
  float* lut = smem + 2 * P.tch * nsrc * r;               // [2][tch][nw][kLutBlock]

  // every U word and row scale this lane will use, loaded (raw) before any
  // wait; they are combined once the first gather round is in flight
  constexpr int NP = max_passes(TM);
  // the epoch left by the previous call (this call's tag is one more)
  uint32_t epoch = load_epoch<2>(P.ctrl);
  uint32_t words[NP][2][kRowWords];
  uint32_t tlo[NP][2], thi[NP][2], hbits[NP][2];
  const int nbu = r >> 5;        // full words per row of U
  const int tailw = r & 31;      // width of the tail word (0: none)
#pragma unroll
  for (int m = 0; m < NP; ++m) {
    const int i = i_base + rows_per_pass * m;
    const bool live = m < passes && i < d_out;
#pragma unroll
    for (int pp = 0; pp < 2; ++pp) {
      const uint32_t* base = static_cast<const uint32_t*>(pp ? P.U[1] : P.U[0]);
      ld_tail_bits(base, nbu, d_out, tailw, i, live && kq == nbu % KQ, tlo[m][pp], thi[m][pp]);
#pragma unroll
      for (int e = 0; e < kRowWords; ++e) {
        const int kb = kq + KQ * e;
        const bool okf = live && kb < nbu;
        words[m][pp][e] = full_words_or(base, nbu, P.ctrl)[okf ? static_cast<int64_t>(kb) * d_out + i : 0];
      }
      hbits[m][pp] = ld_bits<SC>(pp ? P.h[1] : P.h[0], live ? i : 0);
    }
  }
  float hrow[NP][2];
  uint32_t tag = 0u, done_before = 0u;

  bool ok = true;
  for (int t0 = 0; t0 < T; t0 += P.tch) {
    const int tn = min(P.tch, T - t0);
    // gather this token chunk's slots: per path they are contiguous
    // ([t][nsrc][r]); one round of coherent loads, then re-reads of any slot
    // whose tag is not yet current
    const int per_path = tn * nsrc * r;
    const uint64_t* src[2];
#pragma unroll
    for (int pp = 0; pp < 2; ++pp)
      src[pp] = P.direct ? P.partial + (static_cast<int64_t>(pp) * T + t0) * nsrc * r
                         : P.wbuf + (static_cast<int64_t>(pp) * T + t0) * r;
    uint64_t sv[2][kSlotsPerPath];
#pragma unroll
    for (int pp = 0; pp < 2; ++pp)
#pragma unroll
      for (int j = 0; j < kSlotsPerPath; ++j) {
        const int e = tid + kThreads * j;
        sv[pp][j] = get_slot(src[pp] + (e < per_path ? e : 0));  // slots past the chunk are ignored
      }
    if (t0 == 0) {
      // the prefetched U words and row scales (their loads precede the gather)
      asm volatile("" ::: "memory");
      pin(epoch);
      tag = epoch + 1u;
      // count this workgroup as one that has read the epoch (issued once the
      // epoch has arrived; the returned count is used at the end)
      if (tid == 0) done_before = atomic_add_relaxed(P.ctrl + kCtrlDone, 1u);
#pragma unroll
      for (int m = 0; m < NP; ++m)
#pragma unroll
        for (int pp = 0; pp < 2; ++pp) {
          pin(tlo[m][pp]), pin(thi[m][pp]), pin(hbits[m][pp]);
#pragma unroll
          for (int e = 0; e < kRowWords; ++e) pin(words[m][pp][e]);
          const int i = i_base + rows_per_pass * m;
          const bool live = m < passes && i < d_out;
          // the word after a row's full words is its tail word (words past the row are never used)
#pragma unroll
          for (int e = 0; e < kRowWords; ++e)
            if (kq + KQ * e == nbu) words[m][pp][e] = tail_word(tlo[m][pp], thi[m][pp], tailw);
          hrow[m][pp] = live ? bits_to_f32<SC>(hbits[m][pp]) : 0.0f;
        }
    }
    for (uint32_t it = 0;; ++it) {
      bool ready = true;
#pragma unroll
      for (int pp = 0; pp < 2; ++pp)
#pragma unroll
        for (int j = 0; j < kSlotsPerPath; ++j)
          ready = ready && (tid + kThreads * j >= per_path || slot_ready(sv[pp][j], tag));
      if (ready) break;
      if (it >= kSpinLimit) {
        ok = false;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
#pragma unroll
      for (int pp = 0; pp < 2; ++pp)
#pragma unroll
        for (int j = 0; j < kSlotsPerPath; ++j)
          if (tid + kThreads * j < per_path && !slot_ready(sv[pp][j], tag))
            sv[pp][j] = get_slot(src[pp] + tid + kThreads * j);
    }
#pragma unroll
    for (int pp = 0; pp < 2; ++pp)
#pragma unroll
      for (int j = 0; j < kSlotsPerPath; ++j) {
        const int e = tid + kThreads * j;
        if (e < per_path) raw[pp * per_path + e] = slot_value(sv[pp][j]);
      }
    __syncthreads();
    // l (.) z = sum of the partials (ascending run order), then nibble tables
    // over groups of 4 latents
    for (int e = tid; e < 2 * tn * 8 * nw; e += kThreads) {
      const int pt = e / (8 * nw);
      const int gi = e - pt * 8 * nw;
      const float* rs = raw + pt * nsrc * r;
      float w[4] = {0.0f, 0.0f, 0.0f, 0.0f};
      for (int cc = 0; cc < nsrc; ++cc) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (4 * gi + i < r) w[i] += rs[cc * r + 4 * gi + i];
      }
      build_lut16(w[0], w[1], w[2], w[3], lut, pt * nw + (gi >> 3), gi & 7);
    }
    __syncthreads();

#pragma unroll
    for (int m = 0; m < NP; ++m) {
      if (m >= passes) break;
      const int i = i_base + rows_per_pass * m;
      float acc[2][TM];
#pragma unroll
      for (int pp = 0; pp < 2; ++pp)
#pragma unroll
        for (int t = 0; t < TM; ++t) acc[pp][t] = 0.0f;
#pragma unroll
      for (int e = 0; e < kRowWords; ++e) {
        const int kb = kq + KQ * e;
        if (kb < nw) {
#pragma unroll
          for (int pp = 0; pp < 2; ++pp)
#pragma unroll
            for (int t = 0; t < TM; ++t)
              if (t < tn) acc[pp][t] += word_dot(lut, (pp * tn + t) * nw + kb, words[m][pp][e]);
        }
      }
#pragma unroll
      for (int pp = 0; pp < 2; ++pp)
#pragma unroll
        for (int t = 0; t < TM; ++t) acc[pp][t] = row_sum(acc[pp][t], kq_log2);
      if (kq == 0 && i < d_out) {
#pragma unroll
        for (int t = 0; t < TM; ++t)
          if (t < tn)
            st<ACT>(P.y, static_cast<int64_t>(t0 + t) * d_out + i, hrow[m][0] * acc[0][t] + hrow[m][1] * acc[1][t]);
      }
    }
    __syncthreads();
  }
  if (!ok) atomic_store_relaxed(P.ctrl + kCtrlError, 1u);

  // The last stage-2 workgroup to count itself stores the tag as the epoch
  // for the next call.  Every workgroup of this call has read the epoch by
  // then: stage-2 workgroups counted themselves after reading it, and every
  // stage-1 workgroup published values carrying the tag, which this
  // workgroup has gathered (directly, or through the two-level reducers).
  if (tid == 0 && done_before == static_cast<uint32_t>(P.n_s2 - 1)) {
    atomic_store_relaxed(P.ctrl + kCtrlDone, 0u);
    atomic_store_relaxed(P.ctrl + kCtrlEpoch, tag);
  }
}

template <int TM, int ACT, int SC, bool VEC>
__global__ void __launch_bounds__(kThreads, 2) decode_kernel(DecodeParams P) {
  extern __shared__ float smem[];
  // each stage loads the epoch itself, together with its other loads
  const int wg = blockIdx.x;
  if (wg < P.n_s1)
    stage1<TM, ACT, SC, VEC>(P, wg, smem);
  else
    stage2<TM, ACT, SC>(P, wg - P.n_s1, smem);
}

template <int ACT, int SC>
hipError_t launch_typed(const DecodeParams& P, dim3 grid, size_t smem, hipStream_t stream) {
  // x and g read as 4-element vectors when aligned (decided on the host); the
  // element-wise form is compiled for the widest token count only
  if (!P.x_vec || !P.g_vec)
    hipLaunchKernelGGL((decode_kernel<kDecodeMaxTokens, ACT, SC, false>), grid, dim3(kThreads), smem, stream, P);
  else if (P.T <= 1)
    hipLaunchKernelGGL((decode_kernel<1, ACT, SC, true>), grid, dim3(kThreads), smem, stream, P);
  else if (P.T <= 2)
    hipLaunchKernelGGL((decode_kernel<2, ACT, SC, true>), grid, dim3(kThreads), smem, stream, P);
  else if (P.T <= 4)
    hipLaunchKernelGGL((decode_kernel<4, ACT, SC, true>), grid, dim3(kThreads), smem, stream, P);
  else
    return hipErrorInvalidValue;  // T <= kDecodeMaxTokens is checked by the caller
  return hipGetLastError();
}

template <int ACT>
hipError_t launch_act(const DecodeParams& P, dim3 grid, size_t smem, hipStream_t stream) {
  switch (P.sc_dt) {
    case kDtF32: return launch_typed<ACT, kDtF32>(P, grid, smem, stream);
    case kDtF16: return launch_typed<ACT, kDtF16>(P, grid, smem, stream);
    default: return launch_typed<ACT, kDtBF16>(P, grid, smem, stream);
  }
}

size_t align256(size_t b) { return (b + 255) / 256 * 256; }

size_t stage2_floats_per_token(int r, int nsrc) {
  const int nw = nblocks32(r);
  return static_cast<size_t>(2) * (static_cast<size_t>(nsrc) * r + static_cast<size_t>(nw) * kLutBlock);
}

size_t decode_smem_bytes(const DecodeGeom& g, int T, int r) {
  const size_t s1a = static_cast<size_t>(T) * g.cb * kLutBlock;
  const size_t s1b = static_cast<size_t>(4) * T * kKc;
  const size_t s2 = g.tch * stage2_floats_per_token(r, g.direct ? g.s1d : 1);
  size_t m = s1a > s1b ? s1a : s1b;
  if (s2 > m) m = s2;
  return 4 * m;
}

}  // namespace

DecodeGeom decode_geometry(int T, int d_in, int d_out, int r) {
  DecodeGeom g{};
  g.kc = kKc;
  g.nkt = (r + kKc - 1) / kKc;
  const int nbt = nblocks32(d_in);
  const int tt = T > 0 ? T : 1;
  const int nw = nblocks32(r);
  // blocks per staged chunk: bounded by the LDS tables, the table groups a
  // thread builds and the V words a lane holds
  int cb = kLdsFloats / (kLutBlock * tt);
  const int cb_groups = kThreads * kMaxGroupsPerThread / (8 * tt);
  if (cb > cb_groups) cb = cb_groups;
  if (cb > 16 * kMaxWordsPerLane) cb = 16 * kMaxWordsPerLane;
  if (cb < 1) cb = 1;
  // d_in runs: one staged chunk per workgroup when T is small, so that every
  // load of stage 1 is a single round; at most kMaxSplit partials per value
  int s1d = (nbt + cb - 1) / cb;
  if (s1d > kMaxSplit) s1d = kMaxSplit;
  if (s1d < 1) s1d = 1;
  g.bpw = nbt > 0 ? (nbt + s1d - 1) / s1d : 1;
  g.s1d = nbt > 0 ? (nbt + g.bpw - 1) / g.bpw : 0;
  if (cb > g.bpw) cb = g.bpw;
  g.cb = cb;
  g.n_s1 = 2 * g.nkt * g.s1d;
  // stage 2 reads every partial when one token's slots fit one gather round and
  // the LDS, else the two-level reducers' sums
  g.direct = (g.s1d * r <= kThreads * kSlotsPerPath) &&
             stage2_floats_per_token(r, g.s1d) <= static_cast<size_t>(kLdsFloats);
  // lanes per output row (4..16): the fewest that leave each lane at most
  // kRowWords of the row's words per path
  int kq_log2 = 2;
  while (kq_log2 < 4 && (nw + (1 << kq_log2) - 1) >> kq_log2 > kRowWords) ++kq_log2;
  g.kq_log2 = kq_log2;
  // rows per lane: enough to keep the stage-2 workgroups near 256
  const int rows_per_pass = kThreads >> kq_log2;
  const int groups = (d_out + rows_per_pass - 1) / rows_per_pass;
  int passes = (groups + 255) / 256;
  if (passes > max_passes(T)) passes = max_passes(T);
  if (passes < 1) passes = 1;
  g.rows2 = rows_per_pass * passes;
  g.n_s2 = (d_out + g.rows2 - 1) / g.rows2;
  // tokens per stage-2 chunk: LDS for the gathered slots and the tables, and one
  // gather round per chunk
  const int nsrc = g.direct ? g.s1d : 1;
  const size_t per_tok = stage2_floats_per_token(r, nsrc);
  int tch = per_tok > 0 ? static_cast<int>(kLdsFloats / per_tok) : tt;
  const int per_tok_slots = nsrc * r;  // per path
  const int tch_slots = per_tok_slots > 0 ? kThreads * kSlotsPerPath / per_tok_slots : tt;
  if (tch > tch_slots) tch = tch_slots;
  if (tch > tt) tch = tt;
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
  const uintptr_t xa = a.act_dt == kDtF32 ? 16 : 8, ga = a.sc_dt == kDtF32 ? 16 : 8;
  P.x_vec = (reinterpret_cast<uintptr_t>(a.x) % xa == 0) && (a.d_in % 4 == 0);
  P.g_vec = (reinterpret_cast<uintptr_t>(a.g[0]) % ga == 0) && (reinterpret_cast<uintptr_t>(a.g[1]) % ga == 0);
  P.T = a.T;
  P.d_in = a.d_in;
  P.d_out = a.d_out;
  P.r = a.r;
  P.nkt = g.nkt;
  P.cb = g.cb;
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
  switch (a.act_dt) {
    case kDtF32: return launch_act<kDtF32>(P, grid, smem, stream);
    case kDtF16: return launch_act<kDtF16>(P, grid, smem, stream);
    default: return launch_act<kDtBF16>(P, grid, smem, stream);
  }
}

}  // namespace lb
