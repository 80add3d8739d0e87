// Matrix-core decode kernel (up to 64 tokens): one launch computes both
// binary contractions of Proposition 1 (Eq. proposition1) for both paths
// (Sec. 3.3, Eq. final_weight_approx_res) with v_mfma_f32_16x16x32_bf16.
//
// Stage 1 (z_p = V_p^T (g_p (.) x), scaled by l_p):
//   D[k][t] = sum_j (s(V_p[j][k]) g_p[j]) x[t][j]
//   A operand (16 latents x 32 inputs): the packed sign bits of V_p XORed into
//     the sign bits of bf16 terms of g_p.  g_p is cut into terms whose sum is
//     exactly g_p (1 for bf16, 2 for f16, 3 for fp32 scales), so every A value
//     is an exact signed term of g_p.
//   B operand (32 inputs x 16 tokens): x, cut the same way into exact bf16
//     terms (1 for bf16, 2 for f16, 3 for fp32 activations).
//   Every product of two bf16 terms is exact in fp32 and the matrix cores
//   accumulate in fp32, so the contraction is an fp32 sum of the exact
//   products s * g * x.
// Stage 2 (y = sum_p h_p (.) U_p w_p, w_p = l_p (.) z_p):
//   D[i][t] = sum_k s(U_p[i][k]) w_p[t][k]
//   A operand: U_p's sign bits as bf16 +-1; B operand: w_p as a sum of bf16
//   terms (2, i.e. 16 significant bits, for 16-bit outputs; 3 for fp32).
//
// Fragment layout: for the 16x16x32 shape, lane l holds row l % 16 of A (and
// column l % 16 of B) at 8 reduction slots; register v of lane group
// gq = l / 16 holds the pair of reduction indices (4 gq + v, 4 gq + v + 16)
// of a 32-wide block, which puts bit (4 gq + v) of a packed word (LB layout v1)
// at the bf16 sign position of the low half and bit (4 gq + v + 16) at the
// high half with one shift and one mask.  The output lane holds rows
// 4 gq + e (e < 4) of column l % 16.
//
// Loads are buffer loads: a read past the end of a buffer returns zero, so
// operands of absent tokens, latents and blocks need no address clamping or
// masking (only the inputs past d_in inside a row of x are masked, in the one
// tail block).
//
// Launch structure (as in the look-up-table decode kernel): stage-1
// workgroups (lowest block ids; one path, one tile of 16 latents, one run of
// d_in; the 4 waves split the run and are summed in LDS in a fixed order)
// publish l (.) z as tagged 64-bit slots; stage-2 workgroups (16 rows of U
// per wave) prefetch their U words and h, gather the slots of both paths
// until every tag is this call's, and contract.  With many partials, the
// highest run of each tile first adds the others ("two-level").  Waits only
// target lower block ids and are bounded; the epoch / done-counter protocol
// is the same.
#include <atomic>
#include <type_traits>

#include "device_common.h"

namespace lb {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr int kMaxRuns = 32;                  // d_in runs per latent tile (partials per z value)
constexpr int kMaxUWords = kMmaMaxRank / 32;  // stage 2: full U words of one row and path in registers
constexpr int kGather = 8;                    // stage 2: slots a thread gathers per round
constexpr int kDirectMaxSlots = 8192;         // stage 2 reads every partial when there are at most this many

// 32-wide input blocks a stage-1 wave holds in registers per round
__host__ __device__ constexpr int kpw_of(int tt, int act) {
  return (tt == 1 ? 8 : (tt == 2 ? 6 : 4)) / (act == kDtF32 ? 2 : 1);
}

struct MmaParams {
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
  int T, d_in, d_out, r;
  int nmf;     // 16-latent tiles per path
  int s1d;     // d_in runs per tile
  int bpr;     // 32-wide input blocks per run
  int n_s1;    // stage-1 workgroups (2 * nmf * s1d)
  int n_s2;    // stage-2 workgroups
  uint32_t* ctr;  // counter of this linear's finished stage-2 workgroups (in the control block, or a
                  // list launch's line of its own)
  int n_members;  // linears of the launch sharing the control block (1: a single call)
  int direct;  // stage 2 reads every run's partial (else the two-level sums)
  int vec;     // x and g may be read as aligned 4-element vectors
  uint32_t x_bytes, g_bytes, v_bytes, u_bytes, h_bytes, l_bytes;
  uint32_t magic_r;  // ceil(2^32 / r) (0 for r = 1): e / r as one multiply-high
};

// ---------------------------------------------------------------------------
// stage 1
// ---------------------------------------------------------------------------
// One 32-wide block's loads (raw bits): the packed word of this lane's latent,
// and x, g at the 8 inputs of this lane's slots (runs h = 0, 1 of 4 inputs).
template <int TT>
struct S1Loads {
  uint32_t w;
  uint32_t g[2][4];
  uint32_t x[TT][2][4];
};

struct S1Ctx {
  rsrc_t vr, gr, xr;
  int ka;  // this lane's latent (A row)
  int gq, n16;
  int d_in, r;
};

// Loads of full block b (valid; else every load reads past the buffers: zeros).
template <int TT, int ACT, int SC, bool VEC>
__device__ __forceinline__ void s1_issue(const S1Ctx& C, int b, bool valid, S1Loads<TT>& L) {
  L.w = __builtin_amdgcn_raw_buffer_load_b32(C.vr, valid ? static_cast<uint32_t>(b * C.r + C.ka) * 4u : kOob, 0, 0);
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const uint32_t j0 = 32 * b + 4 * C.gq + 16 * h;
    bload4<SC, VEC>(C.gr, j0, valid, L.g[h]);
#pragma unroll
    for (int tt = 0; tt < TT; ++tt)
      bload4<ACT, VEC>(C.xr, static_cast<uint32_t>(16 * tt + C.n16) * C.d_in + j0, valid, L.x[tt][h]);
  }
}

// the tail block's packed word of latent ka (from the tail plane)
__device__ __forceinline__ uint32_t s1_tail_word(const S1Ctx& C, bool valid) {
  const int nbv = C.d_in >> 5, tailv = C.d_in & 31;
  const uint32_t plane = 4u * nbv * C.r;
  const uint32_t off = tailv <= 16 ? plane + 2u * C.ka : plane + 4u * C.ka;
  const uint32_t lo = static_cast<uint16_t>(__builtin_amdgcn_raw_buffer_load_b16(C.vr, valid ? off : kOob, 0, 0));
  const uint32_t hi =
      static_cast<uint16_t>(__builtin_amdgcn_raw_buffer_load_b16(C.vr, valid && tailv > 16 ? off + 2 : kOob, 0, 0));
  return lo | (hi << 16);
}

// MASK: the tail block; inputs j >= d_in of x are zeroed (g reads zero there)
template <int TT, int ACT, int SC, bool VEC, bool MASK>
__device__ __forceinline__ void s1_compute(const S1Ctx& C, int b, uint32_t word, const S1Loads<TT>& L,
                                           floatx4 (&acc)[TT]) {
  constexpr int NG = nterms<SC>(), NX = nterms<ACT>();
  u32x4 A[NG];  // signs on the g terms
  {
    uint32_t gt[NG][4];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      if constexpr (NG == 1) {
        gt[0][v] = raw16<VEC>(L.g[0], v) | (raw16<VEC>(L.g[1], v) << 16);
      } else {
        uint32_t lo[NG], hi[NG];
        split_exact<NG>(raw4_elem<SC, VEC>(L.g[0], v), lo);
        split_exact<NG>(raw4_elem<SC, VEC>(L.g[1], v), hi);
#pragma unroll
        for (int s = 0; s < NG; ++s) gt[s][v] = lo[s] | (hi[s] << 16);
      }
    }
#pragma unroll
    for (int s = 0; s < NG; ++s) A[s] = sign_terms(word, C.gq, gt[s]);
  }
#pragma unroll
  for (int tt = 0; tt < TT; ++tt) {
    u32x4 X[NX];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int j = 32 * b + 4 * C.gq + v;
      const bool ok0 = !MASK || j < C.d_in, ok1 = !MASK || j + 16 < C.d_in;
      if constexpr (NX == 1) {
        X[0][v] = (ok0 ? raw16<VEC>(L.x[tt][0], v) : 0u) | ((ok1 ? raw16<VEC>(L.x[tt][1], v) : 0u) << 16);
      } else {
        uint32_t lo[NX], hi[NX];
        split_exact<NX>(ok0 ? raw4_elem<ACT, VEC>(L.x[tt][0], v) : 0.0f, lo);
        split_exact<NX>(ok1 ? raw4_elem<ACT, VEC>(L.x[tt][1], v) : 0.0f, hi);
#pragma unroll
        for (int a = 0; a < NX; ++a) X[a][v] = lo[a] | (hi[a] << 16);
      }
    }
#pragma unroll
    for (int s = 0; s < NG; ++s)
#pragma unroll
      for (int a = 0; a < NX; ++a) acc[tt] = mfma(A[s], X[a], acc[tt]);
  }
}

template <int TT, int ACT, int SC, bool VEC>
__device__ __forceinline__ void mma_stage1(const MmaParams& P, int wg, float* smem) {
  constexpr int KPW = kpw_of(TT, ACT);
  const int per_path = P.nmf * P.s1d;
  const int p = wg / per_path;
  const int rem = wg - p * per_path;
  const int mf = rem / P.s1d;
  const int c = rem - mf * P.s1d;
  const int T = P.T, r = P.r;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;  // wave index in a scalar
  const int k0 = 16 * mf;
  const int nbt = nblocks32(P.d_in), nbv = P.d_in >> 5;
  const int b0 = c * P.bpr;
  const int b1 = min(nbt, b0 + P.bpr);
  const int bf = min(b1, nbv);  // end of this run's full blocks
  S1Ctx C;
  C.vr = make_rsrc(p ? P.V[1] : P.V[0], P.v_bytes);
  C.gr = make_rsrc(p ? P.g[1] : P.g[0], P.g_bytes);
  C.xr = make_rsrc(P.x, P.x_bytes);
  C.ka = k0 + (lane & 15);
  C.gq = lane >> 4;
  C.n16 = lane & 15;
  C.d_in = P.d_in;
  C.r = r;

  floatx4 acc[TT];
#pragma unroll
  for (int tt = 0; tt < TT; ++tt) acc[tt] = floatx4{0.f, 0.f, 0.f, 0.f};

  // the tail block (if this run holds it: it is then block b1 - 1 = nbv) goes
  // to wave 0; its loads are issued with the first round's
  const bool tail = b1 > nbv && wave == 0;
  S1Loads<TT> LT;
  {
    // x and g of the tail block, read as element loads past d_in give zero
    // for g; x is masked in s1_compute
    S1Ctx CT = C;
    s1_issue<TT, ACT, SC, false>(CT, nbv, tail, LT);
  }
  const uint32_t tword = s1_tail_word(C, tail);
  // latent scales of the output lane (latents k0 + 4gq + e), and the epoch
  const rsrc_t lr = make_rsrc(p ? P.l[1] : P.l[0], P.l_bytes);
  uint32_t lbits[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) lbits[e] = bload<SC>(lr, k0 + 4 * C.gq + e);
  uint32_t epoch = load_epoch<3>(P.ctrl);

  // full blocks, in rounds of KPW blocks per wave
  for (int rb = b0; rb < bf; rb += kWaves * KPW) {
    const int wb = rb + wave * KPW;
    S1Loads<TT> L[KPW];
#pragma unroll
    for (int u = 0; u < KPW; ++u) s1_issue<TT, ACT, SC, VEC>(C, wb + u, wb + u < bf, L[u]);
#pragma unroll
    for (int u = 0; u < KPW; ++u) s1_compute<TT, ACT, SC, VEC, false>(C, wb + u, L[u].w, L[u], acc);
  }
  if (tail) s1_compute<TT, ACT, SC, false, true>(C, nbv, tword, LT, acc);

  // fixed-order sum over the 4 waves through LDS
  floatx4* red = reinterpret_cast<floatx4*>(smem);  // [wave][tt][lane]
#pragma unroll
  for (int tt = 0; tt < TT; ++tt) red[(wave * TT + tt) * 64 + lane] = acc[tt];
  __syncthreads();
  if (wave < TT) {
    const int tt = wave;
    const floatx4 a0 = red[(0 * TT + tt) * 64 + lane], a1 = red[(1 * TT + tt) * 64 + lane];
    const floatx4 a2 = red[(2 * TT + tt) * 64 + lane], a3 = red[(3 * TT + tt) * 64 + lane];
    const int t = 16 * tt + C.n16;
    pin(epoch);
    const uint32_t tag = epoch + 1u;
    const bool reducer = !P.direct && c == P.s1d - 1;
    float sv[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) sv[e] = ((a0[e] + a1[e]) + (a2[e] + a3[e])) * bits_to_f32<SC>(lbits[e]);
    bool ok = true;
#pragma unroll 1
    for (int e = 0; e < 4; ++e) {
      const int k = k0 + 4 * C.gq + e;
      const float s = e == 0 ? sv[0] : (e == 1 ? sv[1] : (e == 2 ? sv[2] : sv[3]));
      if (t < T && k < r) {
        uint64_t* pt = P.partial + (static_cast<int64_t>(p) * T + t) * P.s1d * r + k;
        if (!reducer) {
          put_slot(pt + static_cast<int64_t>(c) * r, tag, s);
        } else {
          float others = 0.0f;
          const bool got = gather_sum<kMaxRuns>(pt, r, P.s1d - 1, tag, others);
          ok = ok && got;
          put_slot(P.wbuf + (static_cast<int64_t>(p) * T + t) * r + k, tag, got ? others + s : __builtin_nanf(""));
        }
      }
    }
    if (!ok) atomic_store_relaxed(P.ctrl + kCtrlError, 1u);
  }
}

// ---------------------------------------------------------------------------
// stage 2
// ---------------------------------------------------------------------------
template <int ACT, int SC, int RB>
__device__ __forceinline__ void mma_stage2(const MmaParams& P, int q, float* smem) {
  constexpr int NW = ACT == kDtF32 ? 3 : 2;  // bf16 terms of w
  const int T = P.T, r = P.r, d_out = P.d_out;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;  // wave index in a scalar
  const int n16 = lane & 15, gq = lane >> 4;
  const int nkb = nblocks32(r);
  const int nbu = r >> 5, tailu = r & 31;
  const int nsrc = P.direct ? P.s1d : 1;
  const int tch = min(16, T);  // tokens per chunk
  const int R32 = 32 * nkb;    // row stride of the summed w (zero past r)
  constexpr int RW = 64 * RB;  // rows of this workgroup: RB blocks of 64 (list launches take several)
  const int qrow0 = q * RW;

  // LDS: U words [2][nkb][RW rows] (block nbu holds the tail word), summed w
  // [2][tch][R32], and (when there are several partials per value) the
  // gathered partials [2][tch][nsrc][r]
  uint32_t* uwl = reinterpret_cast<uint32_t*>(smem);
  float* wsum = smem + 2 * nkb * RW;
  float* raw = wsum + 2 * tch * R32;

  // prefetch (cooperative, raw): the U words of this workgroup's rows, and
  // the row scales of this lane's output rows; then the epoch
  constexpr int kUPer = (kMaxUWords + 1) * RW / kThreads + 1;  // entries per thread and path
  uint32_t ulo[2][kUPer], uhi[2][kUPer];
#pragma unroll
  for (int pp = 0; pp < 2; ++pp) {
    const rsrc_t ur = make_rsrc(pp ? P.U[1] : P.U[0], P.u_bytes);
#pragma unroll
    for (int j = 0; j < kUPer; ++j) {
      const int e = tid + kThreads * j;  // (kb, row) = (e / RW, e % RW)
      const int kb = e / RW, row = qrow0 + (e % RW);
      const bool full = kb < nbu, tl = kb == nbu && tailu != 0;
      const uint32_t plane = 4u * nbu * d_out;
      const uint32_t toff = tailu <= 16 ? plane + 2u * row : plane + 4u * row;
      // full word as two halves (so both cases are the same two 16-bit loads)
      const uint32_t off = full ? static_cast<uint32_t>(kb * d_out + row) * 4u : (tl ? toff : kOob);
      ulo[pp][j] = static_cast<uint16_t>(__builtin_amdgcn_raw_buffer_load_b16(ur, off, 0, 0));
      uhi[pp][j] = static_cast<uint16_t>(
          __builtin_amdgcn_raw_buffer_load_b16(ur, full || (tl && tailu > 16) ? off + 2 : kOob, 0, 0));
    }
  }
  uint32_t hb[RB][2][4];
#pragma unroll
  for (int b = 0; b < RB; ++b)
#pragma unroll
    for (int pp = 0; pp < 2; ++pp) {
      const rsrc_t hr = make_rsrc(pp ? P.h[1] : P.h[0], P.h_bytes);
#pragma unroll
      for (int e = 0; e < 4; ++e) hb[b][pp][e] = bload<SC>(hr, qrow0 + 64 * b + wave * 16 + 4 * gq + e);
    }
  uint32_t epoch = load_epoch<4>(P.ctrl);
  pin(epoch);
  const uint32_t tag = epoch + 1u;
  // count this workgroup as one that has read the epoch (used at the end)
  uint32_t done_before = 0u;
  if (tid == 0) done_before = atomic_add_relaxed(P.ctr, 1u);
#pragma unroll
  for (int pp = 0; pp < 2; ++pp)
#pragma unroll
    for (int j = 0; j < kUPer; ++j) {
      const int e = tid + kThreads * j;
      if (e < nkb * RW) uwl[pp * nkb * RW + e] = ulo[pp][j] | (uhi[pp][j] << 16);
    }

  bool ok = true;
  for (int t0 = 0; t0 < T; t0 += 16) {
    const int tn = min(16, T - t0);
    // zero the latents past r of every summed row
    for (int e = tid; e < 2 * tch * (R32 - r); e += kThreads) {
      const int row = e / (R32 - r);
      wsum[row * R32 + r + (e - row * (R32 - r))] = 0.0f;
    }
    // gather both paths' slots of tokens t0..t0+tn-1 (contiguous per path):
    // rounds of loads, then re-reads of any slot whose tag is not this call's
    const int n1 = tn * nsrc * r;
#pragma unroll
    for (int pp = 0; pp < 2; ++pp) {
      const uint64_t* src = P.direct ? P.partial + (static_cast<int64_t>(pp) * T + t0) * nsrc * r
                                     : P.wbuf + (static_cast<int64_t>(pp) * T + t0) * r;
      for (int e0 = 0; e0 < n1; e0 += kThreads * kGather) {
        uint64_t sv[kGather];
#pragma unroll
        for (int j = 0; j < kGather; ++j) {
          const int e = e0 + tid + kThreads * j;
          sv[j] = get_slot(src + (e < n1 ? e : 0));
        }
        for (uint32_t it = 0;; ++it) {
          bool ready = true;
#pragma unroll
          for (int j = 0; j < kGather; ++j) ready = ready && (e0 + tid + kThreads * j >= n1 || slot_ready(sv[j], tag));
          if (ready) break;
          if (it >= kSpinLimit) {
            ok = false;
            break;
          }
          __builtin_amdgcn_s_sleep(1);
#pragma unroll
          for (int j = 0; j < kGather; ++j) {
            const int e = e0 + tid + kThreads * j;
            if (e < n1 && !slot_ready(sv[j], tag)) sv[j] = get_slot(src + e);
          }
        }
#pragma unroll
        for (int j = 0; j < kGather; ++j) {
          const int e = e0 + tid + kThreads * j;
          if (e < n1) {
            // a slot a timed-out wait never saw carrying this call's tag is NaN
            const float v = slot_ready(sv[j], tag) ? slot_value(sv[j]) : __builtin_nanf("");
            if (nsrc > 1) {
              raw[pp * tch * nsrc * r + e] = v;
            } else {
              const int tl = static_cast<int>(fast_div(e, P.magic_r));
              wsum[(pp * tch + tl) * R32 + (e - tl * r)] = v;
            }
          }
        }
      }
    }
    if (nsrc > 1) {
      // sum each value's partials in ascending run order
      __syncthreads();
      for (int e = tid; e < 2 * tn * r; e += kThreads) {
        const int pt = static_cast<int>(fast_div(e, P.magic_r));  // pp * tn + tl
        const int k = e - pt * r;
        const int pp = pt >= tn ? 1 : 0;
        const int tl = pt - pp * tn;
        const float* rs = raw + ((pp * tch + tl) * nsrc) * r + k;
        float s = 0.0f;
        for (int c = 0; c < nsrc; ++c) s += rs[c * r];
        wsum[(pp * tch + tl) * R32 + k] = s;
      }
    }
    __syncthreads();
    // contraction: A = the signs of U row qrow0 + wave * 16 + n16 (+-1), B = w
    // of token column n16 at latents 32 kb + 4 gq + v (+16), as NW bf16 terms
    floatx4 acc[RB][2];
#pragma unroll
    for (int b = 0; b < RB; ++b) acc[b][0] = acc[b][1] = floatx4{0.f, 0.f, 0.f, 0.f};
    const uint32_t ones[4] = {0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u};
#pragma unroll
    for (int pp = 0; pp < 2; ++pp) {
      const float* wrow = wsum + (pp * tch + (n16 < tch ? n16 : 0)) * R32 + 4 * gq;
      const uint32_t* ucol = uwl + pp * nkb * RW + wave * 16 + n16;
      for (int kb = 0; kb < nkb; ++kb) {
        const float4 w0 = *reinterpret_cast<const float4*>(wrow + 32 * kb);
        const float4 w1 = *reinterpret_cast<const float4*>(wrow + 32 * kb + 16);
        const float wl[4] = {w0.x, w0.y, w0.z, w0.w}, wh[4] = {w1.x, w1.y, w1.z, w1.w};
        uint32_t lo[4][NW], hi[4][NW];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          split_round<NW>(wl[v], lo[v]);
          split_round<NW>(wh[v], hi[v]);
        }
        u32x4 B[NW];
#pragma unroll
        for (int a = 0; a < NW; ++a)
#pragma unroll
          for (int v = 0; v < 4; ++v) B[a][v] = lo[v][a] | (hi[v][a] << 16);
        // the w terms of this block serve every row block
#pragma unroll
        for (int b = 0; b < RB; ++b) {
          const u32x4 A = sign_terms(ucol[kb * RW + 64 * b], gq, ones);
#pragma unroll
          for (int a = 0; a < NW; ++a) acc[b][pp] = mfma(A, B[a], acc[b][pp]);
        }
      }
    }
    // y[t][i] = h_0[i] acc_0 + h_1[i] acc_1 for rows i = qrow0 + 64 b + wave * 16 + 4 gq + e
    const int t = t0 + n16;
#pragma unroll
    for (int b = 0; b < RB; ++b)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int i = qrow0 + 64 * b + wave * 16 + 4 * gq + e;
        if (t < T && i < d_out)
          st<ACT>(P.y, static_cast<int64_t>(t) * d_out + i,
                  bits_to_f32<SC>(hb[b][0][e]) * acc[b][0][e] + bits_to_f32<SC>(hb[b][1][e]) * acc[b][1][e]);
      }
    __syncthreads();  // the next chunk reuses the LDS
  }
  if (!ok) atomic_store_relaxed(P.ctrl + kCtrlError, 1u);
  // The last stage-2 workgroup to count itself stores the tag as the next
  // epoch.  Every workgroup of this call has read the epoch by then: stage-2
  // workgroups counted themselves after reading it, and every stage-1
  // workgroup published values carrying the tag, which this workgroup has
  // gathered (directly, or through the two-level reducers).
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

template <int TT, int ACT, int SC, bool VEC>
__global__ void __launch_bounds__(kThreads, 1) decode_mma_kernel(MmaParams P) {
  extern __shared__ __attribute__((aligned(16))) float smem[];
  const int wg = blockIdx.x;
  if (wg < P.n_s1)
    mma_stage1<TT, ACT, SC, VEC>(P, wg, smem);
  else
    mma_stage2<ACT, SC, 1>(P, wg - P.n_s1, smem);
}

// A list of independent linears in one launch (the stage-1 workgroups of
// every linear, then the stage-2 workgroups, in list order, so every wait
// still targets lower block ids); its members share the token tiles TT and
// the load form VEC.
struct MmaBatch {
  int n;
  int s1_end[kDecodeMaxBatch];  // one past each linear's last stage-1 workgroup
  int s2_end[kDecodeMaxBatch];  // the same for stage 2, counted from the first stage-2 workgroup
  MmaParams p[kDecodeMaxBatch];
};

constexpr int kMmaListRows = 2;  // stage 2 of a list launch: blocks of 64 rows per workgroup

template <int TT, int ACT, int SC, bool VEC>
__global__ void __launch_bounds__(kThreads, 1) decode_mma_batch_kernel(MmaBatch B) {
  extern __shared__ __attribute__((aligned(16))) float smem[];
  const int wg = blockIdx.x;
  const int s1tot = B.s1_end[B.n - 1];
  if (wg < s1tot) {
    int i = 0;
    while (wg >= B.s1_end[i]) ++i;
    const MmaParams P = B.p[i];
    mma_stage1<TT, ACT, SC, VEC>(P, wg - (i ? B.s1_end[i - 1] : 0), smem);
  } else {
    const int w2 = wg - s1tot;
    int i = 0;
    while (w2 >= B.s2_end[i]) ++i;
    const MmaParams P = B.p[i];
    mma_stage2<ACT, SC, kMmaListRows>(P, w2 - (i ? B.s2_end[i - 1] : 0), smem);
  }
}

// one launch of the single-linear (MmaParams) or list (MmaBatch) kernel
template <int TT, int ACT, int SC, bool VEC, typename A>
hipError_t launch_one(const A& args, dim3 grid, size_t smem, hipStream_t stream) {
  constexpr bool kOne = std::is_same<A, MmaParams>::value;
  // more than the default dynamic LDS limit (the CU has 160 KB): raise the
  // kernel's limit once per size increase, so calls captured in a graph after
  // an eager call of the same shape make no attribute call
  static std::atomic<size_t> limit{65536};
  if (smem > limit.load()) {
    const void* fn = kOne ? reinterpret_cast<const void*>(&decode_mma_kernel<TT, ACT, SC, VEC>)
                          : reinterpret_cast<const void*>(&decode_mma_batch_kernel<TT, ACT, SC, VEC>);
    const hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(smem));
    if (e != hipSuccess) return e;
    limit.store(smem);
  }
  if constexpr (kOne)
    hipLaunchKernelGGL((decode_mma_kernel<TT, ACT, SC, VEC>), grid, dim3(kThreads), smem, stream, args);
  else
    hipLaunchKernelGGL((decode_mma_batch_kernel<TT, ACT, SC, VEC>), grid, dim3(kThreads), smem, stream, args);
  return hipGetLastError();
}

template <int ACT, int SC, bool VEC, typename A>
hipError_t launch_tt(const A& args, int T, dim3 grid, size_t smem, hipStream_t stream) {
  switch ((T + 15) / 16) {
    case 1: return launch_one<1, ACT, SC, VEC>(args, grid, smem, stream);
    case 2: return launch_one<2, ACT, SC, VEC>(args, grid, smem, stream);
    case 3: return launch_one<3, ACT, SC, VEC>(args, grid, smem, stream);
    case 4: return launch_one<4, ACT, SC, VEC>(args, grid, smem, stream);
    default: return hipErrorInvalidValue;  // T <= kMmaMaxTokens is checked by the caller
  }
}

template <int ACT, int SC, typename A>
hipError_t launch_vec(const A& args, int T, bool vec, dim3 grid, size_t smem, hipStream_t stream) {
  // element-wise x and g loads (unaligned or d_in % 4 != 0) are compiled for
  // the widest token count only; it serves every T (absent columns dropped)
  return vec ? launch_tt<ACT, SC, true>(args, T, grid, smem, stream)
             : launch_one<4, ACT, SC, false>(args, grid, smem, stream);
}

template <int ACT, typename A>
hipError_t launch_sc(const A& args, int T, bool vec, int sc_dt, dim3 grid, size_t smem, hipStream_t stream) {
  switch (sc_dt) {
    case kDtF32: return launch_vec<ACT, kDtF32>(args, T, vec, grid, smem, stream);
    case kDtF16: return launch_vec<ACT, kDtF16>(args, T, vec, grid, smem, stream);
    default: return launch_vec<ACT, kDtBF16>(args, T, vec, grid, smem, stream);
  }
}

template <typename A>
hipError_t launch_any(const A& args, int act_dt, int T, bool vec, int sc_dt, dim3 grid, size_t smem,
                      hipStream_t stream) {
  switch (act_dt) {
    case kDtF32: return launch_sc<kDtF32>(args, T, vec, sc_dt, grid, smem, stream);
    case kDtF16: return launch_sc<kDtF16>(args, T, vec, sc_dt, grid, smem, stream);
    default: return launch_sc<kDtBF16>(args, T, vec, sc_dt, grid, smem, stream);
  }
}

size_t align256(size_t b) { return (b + 255) / 256 * 256; }

int64_t packed_bytes(int64_t n_out, int64_t n_red) {
  const int64_t w = n_red & 31;
  return 4 * (n_red >> 5) * n_out + (w == 0 ? 0 : (w <= 16 ? 2 : 4)) * n_out;
}

}  // namespace

MmaGeom decode_mma_geometry(int T, int d_in, int d_out, int r, int act_dt) {
  MmaGeom g{};
  const int tt = T > 0 ? (T + 15) / 16 : 1;
  g.nmf = (r + 15) / 16;
  const int nbt = nblocks32(d_in);
  const int per_round = kWaves * kpw_of(tt, act_dt);
  // one round of loads per run when possible, at most kMaxRuns runs
  int s1d = (nbt + per_round - 1) / per_round;
  if (s1d > kMaxRuns) s1d = kMaxRuns;
  if (s1d < 1) s1d = 1;
  g.bpr = nbt > 0 ? (nbt + s1d - 1) / s1d : 1;
  g.s1d = nbt > 0 ? (nbt + g.bpr - 1) / g.bpr : 1;
  g.n_s1 = 2 * g.nmf * g.s1d;
  // stage 2 reads every partial when there are few, else the two-level sums
  g.direct = g.s1d == 1 || static_cast<int64_t>(2) * T * g.s1d * r <= kDirectMaxSlots;
  g.n_s2 = (d_out + kWaves * 16 - 1) / (kWaves * 16);
  const int nsrc = g.direct ? g.s1d : 1;
  const size_t tch = T < 16 ? T : 16;
  const size_t nkb = nblocks32(r);
  // stage 1 sums the waves' [tt][64 lanes] float4 accumulators; the
  // element-wise (unaligned) variant is compiled for 4 token fragments
  const size_t s1_lds = static_cast<size_t>(kWaves) * 4 * 64 * 16;
  const size_t s2_lds = 4 * (2 * nkb * 64 + 2 * tch * 32 * nkb + (nsrc > 1 ? 2 * tch * nsrc * r : 0));
  g.smem_bytes = s1_lds > s2_lds ? s1_lds : s2_lds;
  g.partial_off = kCtrlBytes;
  g.partial_slots = static_cast<size_t>(2) * g.s1d * T * r;
  g.wbuf_off = g.partial_off + align256(8 * g.partial_slots);
  g.wbuf_slots = g.direct ? 0 : static_cast<size_t>(2) * T * r;
  g.ws_bytes = g.wbuf_off + align256(8 * g.wbuf_slots);
  return g;
}

bool decode_mma_supports(int64_t T, int64_t d_in, int64_t d_out, int64_t r) {
  // buffer offsets are 32-bit: every operand, and every offset formed for
  // the (up to 16 * ceil(T / 16)) token rows read, stays below 2^31 bytes
  const int64_t lim = int64_t(1) << 31;
  const int64_t rows = 16 * ((T + 15) / 16);
  return T <= kMmaMaxTokens && r <= kMmaMaxRank && (rows + 1) * d_in * 4 < lim &&
         packed_bytes(d_out, r) < lim && packed_bytes(r, d_in) < lim && d_out * 4 < lim;
}

namespace {

// kernel parameters of one linear
void mma_params(const ForwardArgs& a, const MmaGeom& g, MmaParams& P) {
  P = MmaParams{};
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
  P.nmf = g.nmf;
  P.s1d = g.s1d;
  P.bpr = g.bpr;
  P.n_s1 = g.n_s1;
  P.n_s2 = g.n_s2;
  P.ctr = P.ctrl + kCtrlDone;
  P.n_members = 1;
  P.direct = g.direct;
  const int64_t ex = a.act_dt == kDtF32 ? 4 : 2, es = a.sc_dt == kDtF32 ? 4 : 2;
  const uintptr_t xa = 4 * ex, ga = 4 * es;
  P.vec = (reinterpret_cast<uintptr_t>(a.x) % xa == 0) && (a.d_in % 4 == 0) &&
          (reinterpret_cast<uintptr_t>(a.g[0]) % ga == 0) && (reinterpret_cast<uintptr_t>(a.g[1]) % ga == 0);
  P.x_bytes = static_cast<uint32_t>(static_cast<int64_t>(a.T) * a.d_in * ex);
  P.g_bytes = static_cast<uint32_t>(a.d_in * es);
  P.h_bytes = static_cast<uint32_t>(a.d_out * es);
  P.l_bytes = static_cast<uint32_t>(a.r * es);
  P.v_bytes = static_cast<uint32_t>(packed_bytes(a.r, a.d_in));
  P.u_bytes = static_cast<uint32_t>(packed_bytes(a.d_out, a.r));
  P.magic_r = a.r > 1 ? static_cast<uint32_t>(((uint64_t(1) << 32) + a.r - 1) / a.r) : 0u;
}

}  // namespace

hipError_t launch_decode_mma(const ForwardArgs& a, const MmaGeom& g, hipStream_t stream) {
  MmaParams P;
  mma_params(a, g, P);
  return launch_any(P, a.act_dt, a.T, P.vec != 0, a.sc_dt, dim3(g.n_s1 + g.n_s2), g.smem_bytes, stream);
}

hipError_t launch_decode_mma_batch(const ForwardArgs* a, int n, hipStream_t stream) {
  if (n <= 0 || n > kDecodeMaxBatch) return hipErrorInvalidValue;
  // a stage-1 wave's blocks per round depend on the token tiles and on the
  // load form, so members are launched in sub-lists of equal (tiles, form):
  // each linear then runs exactly the arithmetic of its own call
  MmaParams P[kDecodeMaxBatch];
  MmaGeom G[kDecodeMaxBatch];
  bool done[kDecodeMaxBatch] = {};
  for (int i = 0; i < n; ++i) {
    if (a[i].act_dt != a[0].act_dt || a[i].sc_dt != a[0].sc_dt) return hipErrorInvalidValue;
    G[i] = decode_mma_geometry(a[i].T, a[i].d_in, a[i].d_out, a[i].r, a[i].act_dt);
    mma_params(a[i], G[i], P[i]);
  }
  for (int i = 0; i < n; ++i) {
    if (done[i]) continue;
    const int tt = (a[i].T + 15) / 16;
    const bool vec = P[i].vec != 0;
    MmaBatch B{};
    int s1 = 0, s2 = 0, T = 0;
    size_t smem = 0;
    // LDS of a member in a list launch (U words of kMmaListRows x 64 rows)
    auto list_smem = [&](int j) {
      return G[j].smem_bytes + static_cast<size_t>(4) * 2 * nblocks32(a[j].r) * 64 * (kMmaListRows - 1);
    };
    constexpr size_t kMaxLds = 160 * 1024;
    for (int j = i; j < n; ++j) {
      if (done[j] || (a[j].T + 15) / 16 != tt || (P[j].vec != 0) != vec) continue;
      if (list_smem(j) > kMaxLds && B.n > 0) continue;  // a launch of its own later
      done[j] = true;
      if (list_smem(j) > kMaxLds) {  // j == i: alone, as a single call
        B.p[0] = P[j];
        B.n = 1;
        break;
      }
      B.p[B.n] = P[j];
      // kMmaListRows row blocks per stage-2 workgroup: that many fewer
      // workgroups, U words of that many rows in LDS
      B.p[B.n].n_s2 = (G[j].n_s2 + kMmaListRows - 1) / kMmaListRows;
      s1 += G[j].n_s1;
      s2 += B.p[B.n].n_s2;
      B.s1_end[B.n] = s1;
      B.s2_end[B.n] = s2;
      T = a[j].T > T ? a[j].T : T;
      smem = list_smem(j) > smem ? list_smem(j) : smem;
      ++B.n;
    }
    // members that share a control block end the call together: each counts
    // its stage-2 workgroups on a line of its own after the control block,
    // the last member to finish stores the epoch
    for (int k = 0; k < B.n; ++k) {
      int cnt = 0;
      for (int m = 0; m < B.n; ++m) cnt += B.p[m].ctrl == B.p[k].ctrl ? 1 : 0;
      if (cnt > 1) {
        B.p[k].ctr = reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(B.p[k].ctrl) + kCtrlBytes +
                                                 kListCtrStride * static_cast<size_t>(k));
        B.p[k].n_members = cnt;
      }
    }
    const hipError_t e = B.n == 1 ? launch_any(P[i], a[i].act_dt, a[i].T, vec, a[i].sc_dt,
                                               dim3(G[i].n_s1 + G[i].n_s2), G[i].smem_bytes, stream)
                                  : launch_any(B, a[0].act_dt, T, vec, a[0].sc_dt, dim3(s1 + s2), smem, stream);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace lb
