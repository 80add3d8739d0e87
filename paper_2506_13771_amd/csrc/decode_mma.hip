// Matrix-core decode kernel (up to 64 tokens): one launch computes both
// binary contractions of Proposition 1 (Eq. proposition1) for both paths
// (Sec. 3.3, Eq. final_weight_approx_res) with v_mfma_f32_16x16x32_bf16.
//
// Stage 1 (z_p = V_p^T (g_p (.) x), scaled by l_p):
//   D[k][t] = sum_j (s(V_p[j][k]) g_p[j]) x[t][j]
//   A operand (16 latents x 32 inputs): the packed sign bits of V_p XORed into
//     the sign bits of bf16 terms of g_p.  g_p is split into terms whose sum is
//     exactly g_p (1 for bf16, 2 for f16, 3 for fp32 scales), so every A value
//     is an exact signed term of g_p.
//   B operand (32 inputs x 16 tokens): x, also split into exact bf16 terms
//     (1 for bf16, 2 for f16, 3 for fp32 activations).
//   Every product of two bf16 terms is exact in fp32 and the matrix cores
//   accumulate in fp32, so the contraction equals the fp32 sum of the exact
//   products s * g * x.
// Stage 2 (y = sum_p h_p (.) U_p w_p, w_p = l_p (.) z_p):
//   D[i][t] = sum_k s(U_p[i][k]) w_p[t][k]
//   A operand: U_p's sign bits as bf16 +-1; B operand: w_p split into bf16
//   terms (2 for 16-bit outputs, 3 for fp32 outputs).
//
// Fragment layout: for the 16x16x32 shape, lane l holds row l % 16 of A (and
// column l % 16 of B) at 8 reduction slots; register v of lane group
// gq = l / 16 holds the pair of reduction indices (4 gq + v, 4 gq + v + 16)
// of a 32-wide block, which puts bit (4 gq + v) of a packed word (LB layout v1)
// at the bf16 sign position of the low half and bit (4 gq + v + 16) at the
// high half with one shift and one mask.  The output lane holds rows
// 4 gq + e (e < 4) of column l % 16.
//
// Launch structure (as in the look-up-table decode kernel): stage-1
// workgroups (lowest block ids; one path, one tile of 16 latents, one run of
// d_in; the 4 waves split the run and are summed in LDS in a fixed order)
// publish l (.) z as tagged 64-bit slots; stage-2 workgroups (rows of U)
// prefetch their U words and h, gather the slots until every tag is this
// call's, and contract.  With many runs, the highest run of each tile first
// adds the others ("two-level").  Waits only target lower block ids and are
// bounded; the epoch / done-counter protocol is the same.
#include <atomic>

#include "device_common.h"

namespace lb {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// floats rounded up to a multiple of 4 (16-byte alignment of what follows)
__host__ __device__ constexpr int align4(int n) { return (n + 3) & ~3; }

constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr int kMaxRuns = 32;         // d_in runs per latent tile (partials per z value)
constexpr int kMaxUWords = kMmaMaxRank / 32;  // stage 2: U words per row and path held in registers
constexpr int kSlotsPerRound = 8;    // stage 2: slots a thread gathers per round
constexpr int kDirectMax = 512;      // stage 2 reads every partial when s1d * r <= this

// exact bf16 terms per dtype
template <int DT>
__host__ __device__ constexpr int nterms() {
  return DT == kDtF32 ? 3 : (DT == kDtF16 ? 2 : 1);
}
// K-steps (32-wide input blocks) a stage-1 wave holds in registers per round
template <int TT, int ACT>
__host__ __device__ constexpr int kpw_max() {
  return (TT == 1 ? 8 : (TT == 2 ? 6 : 4)) / (ACT == kDtF32 ? 2 : 1);
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
  int direct;  // stage 2 reads every run's partial (else the two-level sums)
  int vec;     // x and g may be read as aligned 4-element vectors
};

// split v into N bf16 terms (round-to-nearest-even each); their sum is v for
// the term counts used here (nterms of v's storage dtype)
template <int N>
__device__ __forceinline__ void split_terms(float v, uint32_t (&o)[N]) {
  float rem = v;
#pragma unroll
  for (int s = 0; s < N; ++s) {
    const uint32_t b = f32_to_bf16_bits(rem);
    o[s] = b;
    rem = rem - bf16_bits_to_f32(b);
  }
}

__device__ __forceinline__ floatx4 mfma(u32x4 a, u32x4 b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0,
                                                 0, 0);
}

// raw bits of 4 consecutive elements starting at i (element e < nvalid, else p[0])
template <int DT, bool VEC>
__device__ __forceinline__ void ld4(const void* p, int64_t i, int nvalid, uint32_t (&o)[4]) {
  ld4_bits<DT, VEC>(p, nvalid > 0 ? i : 0, nvalid, o);
}

// ---------------------------------------------------------------------------
// stage 1
// ---------------------------------------------------------------------------
// One K-step's loads (raw bits): the packed word of this lane's latent (full
// blocks; the tail block's word is loaded once per round), and x, g at the 8
// inputs of this lane's slots (runs h = 0, 1 of 4 inputs).
template <int TT>
struct S1Loads {
  uint32_t w;
  uint32_t g[2][4];
  uint32_t x[TT][2][4];
};

template <int TT, int ACT, int SC, bool VEC>
__device__ __forceinline__ void s1_issue(const MmaParams& P, const uint32_t* Vw, const void* gp, int b, bool bvalid,
                                         int k, bool kvalid, int gq, int n16, S1Loads<TT>& L) {
  const int d_in = P.d_in, r = P.r;
  const int nbv = d_in >> 5, tailv = d_in & 31;
  const bool full = bvalid && b < nbv;
  L.w = full_words_or(Vw, nbv, P.ctrl)[full && kvalid ? static_cast<int64_t>(b) * r + k : 0];
  (void)tailv;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int j0 = 32 * b + 4 * gq + 16 * h;
    const int nv = bvalid ? min(4, max(0, d_in - j0)) : 0;
    ld4<SC, VEC>(gp, j0, nv, L.g[h]);
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
      const int t = min(16 * tt + n16, P.T - 1);  // columns past T are computed and dropped
      ld4<ACT, VEC>(P.x, static_cast<int64_t>(t) * d_in + j0, nv, L.x[tt][h]);
    }
  }
}

template <int TT, int ACT, int SC, bool VEC>
__device__ __forceinline__ void s1_compute(const MmaParams& P, int b, bool bvalid, int gq, const S1Loads<TT>& L,
                                           uint32_t tailword, floatx4 (&acc)[TT]) {
  constexpr int NG = nterms<SC>(), NX = nterms<ACT>();
  const int d_in = P.d_in;
  const int nbv = d_in >> 5;
  const uint32_t word = b < nbv ? L.w : tailword;
  const uint32_t ws = word >> (4 * gq);
  // g terms paired per register: low half input 4gq+v, high half 4gq+v+16
  uint32_t gt[NG][4];
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    uint32_t lo[NG], hi[NG];
    const int j = 32 * b + 4 * gq + v;
    const bool ok0 = bvalid && j < d_in, ok1 = bvalid && j + 16 < d_in;
    split_terms<NG>(ok0 ? raw4_elem<SC, VEC>(L.g[0], v) : 0.0f, lo);
    split_terms<NG>(ok1 ? raw4_elem<SC, VEC>(L.g[1], v) : 0.0f, hi);
#pragma unroll
    for (int s = 0; s < NG; ++s) gt[s][v] = lo[s] | (hi[s] << 16);
  }
  u32x4 A[NG];
#pragma unroll
  for (int s = 0; s < NG; ++s)
#pragma unroll
    for (int v = 0; v < 4; ++v) A[s][v] = ((ws << (15 - v)) & 0x80008000u) ^ gt[s][v];
#pragma unroll
  for (int tt = 0; tt < TT; ++tt) {
    u32x4 X[NX];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int j = 32 * b + 4 * gq + v;
      const bool ok0 = bvalid && j < d_in, ok1 = bvalid && j + 16 < d_in;
      if constexpr (NX == 1) {
        // bf16 activations: the raw bits are the term (zeroed beyond d_in)
        uint32_t a0, a1;
        if constexpr (VEC) {
          a0 = (L.x[tt][0][v >> 1] >> (16 * (v & 1))) & 0xffffu;
          a1 = (L.x[tt][1][v >> 1] >> (16 * (v & 1))) & 0xffffu;
        } else {
          a0 = L.x[tt][0][v];
          a1 = L.x[tt][1][v];
        }
        X[0][v] = (ok0 ? a0 : 0u) | ((ok1 ? a1 : 0u) << 16);
      } else {
        uint32_t lo[NX], hi[NX];
        split_terms<NX>(ok0 ? raw4_elem<ACT, VEC>(L.x[tt][0], v) : 0.0f, lo);
        split_terms<NX>(ok1 ? raw4_elem<ACT, VEC>(L.x[tt][1], v) : 0.0f, hi);
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
  constexpr int KPW = kpw_max<TT, ACT>();
  const int per_path = P.nmf * P.s1d;
  const int p = wg / per_path;
  const int rem = wg - p * per_path;
  const int mf = rem / P.s1d;
  const int c = rem - mf * P.s1d;
  const int T = P.T, r = P.r;
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int n16 = lane & 15, gq = lane >> 4;
  const int k0 = 16 * mf;
  const int nbt = nblocks32(P.d_in);
  const int b0 = c * P.bpr;
  const int b1 = min(nbt, b0 + P.bpr);
  const uint32_t* Vw = static_cast<const uint32_t*>(p ? P.V[1] : P.V[0]);
  const void* gp = p ? P.g[1] : P.g[0];
  const void* lp = p ? P.l[1] : P.l[0];

  // A-operand lane: latent k0 + n16 (its packed words); output lane: latents
  // k0 + 4gq + e of token column n16
  const int ka = k0 + n16;
  const bool ka_ok = ka < r;
  floatx4 acc[TT];
#pragma unroll
  for (int tt = 0; tt < TT; ++tt) acc[tt] = floatx4{0.f, 0.f, 0.f, 0.f};

  // latent scales of the output lane, and the epoch (both used at the end)
  uint32_t lbits[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) lbits[e] = ld_bits<SC>(lp, min(k0 + 4 * gq + e, r - 1));
  uint32_t epoch = load_epoch<3>(P.ctrl);

  // the run's blocks, split over the waves in rounds of KPW blocks per wave
  const int nbv = P.d_in >> 5, tailv = P.d_in & 31;
  for (int rb = b0; rb < b1; rb += kWaves * KPW) {
    const int wb = rb + wave * KPW;  // this wave's first block of the round
    S1Loads<TT> L[KPW];
#pragma unroll
    for (int u = 0; u < KPW; ++u) {
      const int b = wb + u;
      const bool bvalid = b < b1;
      s1_issue<TT, ACT, SC, VEC>(P, Vw, gp, bvalid ? b : b0, bvalid, ka, ka_ok, gq, n16, L[u]);
    }
    // the tail block's word (if the tail block is among this wave's blocks)
    uint32_t tlo, thi;
    ld_tail_bits(Vw, nbv, r, tailv, ka, ka_ok && nbv >= wb && nbv < wb + KPW && nbv < b1, tlo, thi);
    const uint32_t tailword = tail_word(tlo, thi, tailv);
#pragma unroll
    for (int u = 0; u < KPW; ++u) {
      const int b = wb + u;
      s1_compute<TT, ACT, SC, VEC>(P, b < b1 ? b : b0, b < b1, gq, L[u], tailword, acc);
    }
  }

  // fixed-order sum over the 4 waves through LDS
  floatx4* red = reinterpret_cast<floatx4*>(smem);  // [wave][tt][lane]
#pragma unroll
  for (int tt = 0; tt < TT; ++tt) red[(wave * TT + tt) * 64 + lane] = acc[tt];
  __syncthreads();
  if (wave < TT) {
    const int tt = wave;
    const floatx4 a0 = red[(0 * TT + tt) * 64 + lane], a1 = red[(1 * TT + tt) * 64 + lane];
    const floatx4 a2 = red[(2 * TT + tt) * 64 + lane], a3 = red[(3 * TT + tt) * 64 + lane];
    const int t = 16 * tt + n16;
    pin(epoch);
    const uint32_t tag = epoch + 1u;
    const bool reducer = !P.direct && c == P.s1d - 1;
    bool ok = true;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int k = k0 + 4 * gq + e;
      if (t < T && k < r) {
        const float s = ((a0[e] + a1[e]) + (a2[e] + a3[e])) * bits_to_f32<SC>(lbits[e]);
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
template <int TT, int ACT, int SC>
__device__ __forceinline__ void mma_stage2(const MmaParams& P, int q, float* smem) {
  constexpr int NW = ACT == kDtF32 ? 3 : 2;  // bf16 terms of w
  const int T = P.T, r = P.r, d_out = P.d_out;
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int n16 = lane & 15, gq = lane >> 4;
  const int nkb = nblocks32(r);
  const int nbu = r >> 5, tailu = r & 31;
  const int nsrc = P.direct ? P.s1d : 1;
  const int row0 = (q * kWaves + wave) * 16;  // this wave's 16 rows

  // prefetch, raw: the U words of this lane's A row (row0 + n16) and the row
  // scales of its output rows (row0 + 4 gq + e), both paths; then the epoch
  uint32_t uw[2][kMaxUWords];
  uint32_t ut_lo[2], ut_hi[2];
  uint32_t hb[2][4];
  const int ia = row0 + n16;
  const bool aok = ia < d_out;
#pragma unroll
  for (int pp = 0; pp < 2; ++pp) {
    const uint32_t* Uw = static_cast<const uint32_t*>(pp ? P.U[1] : P.U[0]);
    const void* hp = pp ? P.h[1] : P.h[0];
#pragma unroll
    for (int kb = 0; kb < kMaxUWords; ++kb) {
      const bool ok = aok && kb < nbu;
      uw[pp][kb] = full_words_or(Uw, nbu, P.ctrl)[ok ? static_cast<int64_t>(kb) * d_out + ia : 0];
    }
    ld_tail_bits(Uw, nbu, d_out, tailu, ia, aok, ut_lo[pp], ut_hi[pp]);
#pragma unroll
    for (int e = 0; e < 4; ++e) hb[pp][e] = ld_bits<SC>(hp, min(row0 + 4 * gq + e, d_out - 1));
  }
  uint32_t epoch = load_epoch<4>(P.ctrl);
  pin(epoch);  // waits for the epoch only (the prefetch loads were issued before it... or after)
  const uint32_t tag = epoch + 1u;
  // count this workgroup as one that has read the epoch (used at the end)
  uint32_t done_before = 0u;
  if (tid == 0) done_before = atomic_add_relaxed(P.ctrl + kCtrlDone, 1u);

  float* raw = smem;                                                        // [16][nsrc][r] slot values
  u32x4* frag = reinterpret_cast<u32x4*>(smem + align4(16 * nsrc * r));     // [nkb][NW][64 lanes]
  bool ok = true;
  for (int t0 = 0; t0 < T; t0 += 16) {
    const int tn = min(16, T - t0);
    floatx4 acc[2];
    acc[0] = acc[1] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int pp = 0; pp < 2; ++pp) {
      // gather this path's slots for tokens t0..t0+tn-1: contiguous
      // [tn][nsrc][r]; loads in rounds, re-reads of any slot whose tag is not
      // yet this call's
      const int n = tn * nsrc * r;
      const uint64_t* src = P.direct ? P.partial + (static_cast<int64_t>(pp) * T + t0) * nsrc * r
                                     : P.wbuf + (static_cast<int64_t>(pp) * T + t0) * r;
      for (int e0 = 0; e0 < n; e0 += kThreads * kSlotsPerRound) {
        uint64_t sv[kSlotsPerRound];
#pragma unroll
        for (int j = 0; j < kSlotsPerRound; ++j) {
          const int e = e0 + tid + kThreads * j;
          sv[j] = get_slot(src + (e < n ? e : 0));
        }
        for (uint32_t it = 0;; ++it) {
          bool ready = true;
#pragma unroll
          for (int j = 0; j < kSlotsPerRound; ++j)
            ready = ready && (e0 + tid + kThreads * j >= n || slot_ready(sv[j], tag));
          if (ready) break;
          if (it >= kSpinLimit) {
            ok = false;
            break;
          }
          __builtin_amdgcn_s_sleep(1);
#pragma unroll
          for (int j = 0; j < kSlotsPerRound; ++j) {
            const int e = e0 + tid + kThreads * j;
            if (e < n && !slot_ready(sv[j], tag)) sv[j] = get_slot(src + e);
          }
        }
#pragma unroll
        for (int j = 0; j < kSlotsPerRound; ++j) {
          const int e = e0 + tid + kThreads * j;
          if (e < n) raw[e] = slot_value(sv[j]);
        }
      }
      __syncthreads();
      // B fragments of w_p: item (kb, lane'); its 8 values are latents
      // 32 kb + 4 gq' + v (+16) of token t0 + n16', the sum of the runs'
      // partials in ascending order, split into NW bf16 terms
      for (int item = tid; item < nkb * 64; item += kThreads) {
        const int kb = item >> 6, il = item & 63;
        const int tl = il & 15, g4 = il >> 4;
        uint32_t lo[4][NW], hi[4][NW];
#pragma unroll
        for (int v = 0; v < 8; ++v) {
          const int k = 32 * kb + 4 * g4 + (v & 3) + 16 * (v >> 2);
          float sum = 0.0f;
          if (tl < tn && k < r)
            for (int c = 0; c < nsrc; ++c) sum += raw[(tl * nsrc + c) * r + k];
          if (v < 4)
            split_terms<NW>(sum, lo[v]);
          else
            split_terms<NW>(sum, hi[v - 4]);
        }
#pragma unroll
        for (int a = 0; a < NW; ++a) {
          u32x4 f;
#pragma unroll
          for (int v = 0; v < 4; ++v) f[v] = lo[v][a] | (hi[v][a] << 16);
          frag[(kb * NW + a) * 64 + il] = f;
        }
      }
      __syncthreads();
      // contraction with this lane's U row
      const uint32_t tailword = tail_word(ut_lo[pp], ut_hi[pp], tailu);
#pragma unroll
      for (int kb = 0; kb < kMaxUWords + 1; ++kb) {
        if (kb >= nkb) continue;
        const uint32_t word = kb < nbu ? uw[pp][kb < kMaxUWords ? kb : 0] : tailword;
        const uint32_t ws = word >> (4 * gq);
        u32x4 A;
#pragma unroll
        for (int v = 0; v < 4; ++v) A[v] = ((ws << (15 - v)) & 0x80008000u) | 0x3F803F80u;
#pragma unroll
        for (int a = 0; a < NW; ++a) acc[pp] = mfma(A, frag[(kb * NW + a) * 64 + lane], acc[pp]);
      }
      __syncthreads();
    }
    // y[t][i] = h_0[i] acc_0 + h_1[i] acc_1 for rows i = row0 + 4 gq + e
    const int t = t0 + n16;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int i = row0 + 4 * gq + e;
      if (t < T && i < d_out)
        st<ACT>(P.y, static_cast<int64_t>(t) * d_out + i,
                bits_to_f32<SC>(hb[0][e]) * acc[0][e] + bits_to_f32<SC>(hb[1][e]) * acc[1][e]);
    }
  }
  if (!ok) atomic_store_relaxed(P.ctrl + kCtrlError, 1u);
  // The last stage-2 workgroup to count itself stores the tag as the next
  // epoch.  Every workgroup of this call has read the epoch by then: stage-2
  // workgroups counted themselves after reading it, and every stage-1
  // workgroup published values carrying the tag, which this workgroup has
  // gathered (directly, or through the two-level reducers).
  if (tid == 0 && done_before == static_cast<uint32_t>(P.n_s2 - 1)) {
    atomic_store_relaxed(P.ctrl + kCtrlDone, 0u);
    atomic_store_relaxed(P.ctrl + kCtrlEpoch, tag);
  }
}

template <int TT, int ACT, int SC, bool VEC>
__global__ void __launch_bounds__(kThreads, 1) decode_mma_kernel(MmaParams P) {
  extern __shared__ __attribute__((aligned(16))) float smem[];
  const int wg = blockIdx.x;
  if (wg < P.n_s1)
    mma_stage1<TT, ACT, SC, VEC>(P, wg, smem);
  else
    mma_stage2<TT, ACT, SC>(P, wg - P.n_s1, smem);
}

template <int TT, int ACT, int SC, bool VEC>
hipError_t launch_one(const MmaParams& P, dim3 grid, size_t smem, hipStream_t stream) {
  // more than the default dynamic LDS limit (the CU has 160 KB): raise the
  // kernel's limit once per size increase, so calls captured in a graph after
  // an eager call of the same shape make no attribute call
  static std::atomic<size_t> limit{65536};
  if (smem > limit.load()) {
    const void* fn = reinterpret_cast<const void*>(&decode_mma_kernel<TT, ACT, SC, VEC>);
    const hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(smem));
    if (e != hipSuccess) return e;
    limit.store(smem);
  }
  hipLaunchKernelGGL((decode_mma_kernel<TT, ACT, SC, VEC>), grid, dim3(kThreads), smem, stream, P);
  return hipGetLastError();
}

template <int ACT, int SC, bool VEC>
hipError_t launch_tt(const MmaParams& P, dim3 grid, size_t smem, hipStream_t stream) {
  switch ((P.T + 15) / 16) {
    case 1: return launch_one<1, ACT, SC, VEC>(P, grid, smem, stream);
    case 2: return launch_one<2, ACT, SC, VEC>(P, grid, smem, stream);
    case 3: return launch_one<3, ACT, SC, VEC>(P, grid, smem, stream);
    case 4: return launch_one<4, ACT, SC, VEC>(P, grid, smem, stream);
    default: return hipErrorInvalidValue;  // T <= kMmaMaxTokens is checked by the caller
  }
}

template <int ACT, int SC>
hipError_t launch_vec(const MmaParams& P, dim3 grid, size_t smem, hipStream_t stream) {
  return P.vec ? launch_tt<ACT, SC, true>(P, grid, smem, stream) : launch_tt<ACT, SC, false>(P, grid, smem, stream);
}

template <int ACT>
hipError_t launch_sc(const MmaParams& P, int sc_dt, dim3 grid, size_t smem, hipStream_t stream) {
  switch (sc_dt) {
    case kDtF32: return launch_vec<ACT, kDtF32>(P, grid, smem, stream);
    case kDtF16: return launch_vec<ACT, kDtF16>(P, grid, smem, stream);
    default: return launch_vec<ACT, kDtBF16>(P, grid, smem, stream);
  }
}

size_t align256(size_t b) { return (b + 255) / 256 * 256; }

int kpw_for(int T, int act_dt) {
  const int tt = (T + 15) / 16;
  const int base = tt == 1 ? 8 : (tt == 2 ? 6 : 4);
  return act_dt == kDtF32 ? base / 2 : base;
}

}  // namespace

MmaGeom decode_mma_geometry(int T, int d_in, int d_out, int r, int act_dt) {
  MmaGeom g{};
  const int tt = T > 0 ? (T + 15) / 16 : 1;
  g.nmf = (r + 15) / 16;
  const int nbt = nblocks32(d_in);
  const int per_round = kWaves * kpw_for(T, act_dt);
  // one round of loads per run when possible, at most kMaxRuns runs
  int s1d = (nbt + per_round - 1) / per_round;
  if (s1d > kMaxRuns) s1d = kMaxRuns;
  if (s1d < 1) s1d = 1;
  g.bpr = nbt > 0 ? (nbt + s1d - 1) / s1d : 1;
  g.s1d = nbt > 0 ? (nbt + g.bpr - 1) / g.bpr : 1;
  g.n_s1 = 2 * g.nmf * g.s1d;
  // stage 2 reads every partial when there are few, else the two-level sums
  g.direct = g.s1d * r <= kDirectMax;
  g.n_s2 = (d_out + kWaves * 16 - 1) / (kWaves * 16);
  const int nw = act_dt == kDtF32 ? 3 : 2;
  const int nsrc = g.direct ? g.s1d : 1;
  const size_t s1_lds = static_cast<size_t>(kWaves) * tt * 64 * 16;
  const size_t s2_lds = 4 * static_cast<size_t>(align4(16 * nsrc * r)) + static_cast<size_t>(nblocks32(r)) * nw * 64 * 16;
  g.smem_bytes = s1_lds > s2_lds ? s1_lds : s2_lds;
  g.partial_off = kCtrlBytes;
  g.partial_slots = static_cast<size_t>(2) * g.s1d * T * r;
  g.wbuf_off = g.partial_off + align256(8 * g.partial_slots);
  g.wbuf_slots = g.direct ? 0 : static_cast<size_t>(2) * T * r;
  g.ws_bytes = g.wbuf_off + align256(8 * g.wbuf_slots);
  return g;
}

bool decode_mma_supports(int64_t T, int64_t r) { return T <= kMmaMaxTokens && r <= kMmaMaxRank; }

hipError_t launch_decode_mma(const ForwardArgs& a, const MmaGeom& g, hipStream_t stream) {
  MmaParams P{};
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
  P.T = a.T;
  P.d_in = a.d_in;
  P.d_out = a.d_out;
  P.r = a.r;
  P.nmf = g.nmf;
  P.s1d = g.s1d;
  P.bpr = g.bpr;
  P.n_s1 = g.n_s1;
  P.n_s2 = g.n_s2;
  P.direct = g.direct;
  const uintptr_t xa = a.act_dt == kDtF32 ? 16 : 8, ga = a.sc_dt == kDtF32 ? 16 : 8;
  P.vec = (reinterpret_cast<uintptr_t>(a.x) % xa == 0) && (a.d_in % 4 == 0) &&
          (reinterpret_cast<uintptr_t>(a.g[0]) % ga == 0) && (reinterpret_cast<uintptr_t>(a.g[1]) % ga == 0);
  const dim3 grid(g.n_s1 + g.n_s2);
  switch (a.act_dt) {
    case kDtF32: return launch_sc<kDtF32>(P, a.sc_dt, grid, g.smem_bytes, stream);
    case kDtF16: return launch_sc<kDtF16>(P, a.sc_dt, grid, g.smem_bytes, stream);
    default: return launch_sc<kDtBF16>(P, a.sc_dt, grid, g.smem_bytes, stream);
  }
}

}  // namespace lb
