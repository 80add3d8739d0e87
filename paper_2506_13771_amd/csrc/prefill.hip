// Prefill kernels (long token runs): the two binary contractions of
// Proposition 1 (Eq. proposition1) for both paths (Sec. 3.3, Eq.
// final_weight_approx_res) as matrix-core products on gfx950, in three
// launches.
//
//   P1:  z_p[t][k] = sum_j (s(V_p)[j][k] g_p[j]) x[t][j]           (M = latents, N = tokens, K = d_in)
//   P1b: w_p[t][k] = l_p[k] z_p[t][k], cut into bf16 terms
//   P2:  y[t][i]   = sum_p h_p[i] sum_k s(U_p)[i][k] w_p[t][k]    (M = outputs, N = tokens, K = r)
//
// Every product is exact: the A operand of P1 is the sign of V_p XORed into
// the sign bits of exact bf16 terms of g_p (1 term for bf16, 2 for f16, 3 for
// fp32 scales), its B operand the exact bf16 terms of x (1, 2 or 3 by the
// activation dtype); P2 multiplies exact +-1 signs by w cut into NW bf16 terms
// (2 for bf16/f16 outputs: 16 significant bits; 3 for fp32 outputs: all 24).
// The matrix cores accumulate in fp32.
//
// P1.  A workgroup of 8 waves owns 64 tokens, a range of d_in (split over
// `ks` workgroups, about 256 in all) and a tile of latents.  Waves 0-1 take
// path 0 and waves 2-3 path 1, each MS interleaved 16-latent subtiles of its
// path, so a wave holds MS x 4 accumulator tiles and no sum crosses paths;
// waves 4-7 repeat these roles on the odd 32-input steps (kSplit1 groups of 4
// waves take turns), and the groups are added once in LDS at the end, in a
// fixed order.  The steps stream through an LDS ring filled by global-to-LDS
// loads (x of the 64 tokens, written in B-fragment order, and each wave's V
// words), several rounds in flight; one barrier per round hands slots from
// their loads to their readers and back.  The g terms of the range are cut
// once into LDS.
// P1b.  Sums the ks partials in ascending order, scales by l and stores w as
// NW bf16 terms laid out as B fragments of P2.
// P2.  A workgroup of 8 waves owns 64 tokens and a group of 128-output
// units.  It loads the w fragments of its tokens into LDS once (when they
// fit; else per chunk) and then runs its units: the two halves of 4 waves
// take alternate units, a wave 64 outputs x 32 tokens.  The packed U words,
// row scales and tail words of a half's next unit are loaded into LDS while
// its current unit runs.  Both paths accumulate separately and
// y = h_0 acc_0 + h_1 acc_1 is rounded once.
//
// P1 fragment order.  A 32-input step of B (x) is read as 16 bytes per lane:
// lane group gq holds inputs 8 gq .. 8 gq + 7 of the step, register v the pair
// (8 gq + 2 v, 8 gq + 2 v + 1), which is the memory order of x.  The A operand
// takes the same order from a packed word: with t = word >> 8 gq,
// d = (t & 0xffff) | ((t << 15) & 0xffff0000) holds the bit of input 2 v of the
// group at bit 2 v and that of input 2 v + 1 at bit 2 v + 16, and one shift
// by 15 - 2 v moves the pair onto the two bf16 sign bits.  P2 uses the
// relabelled order of sign_terms (its B operand is produced by P1b in that
// order).
#include <atomic>

#include "device_common.h"
#include "lb_backward.h"

namespace lb {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = 4;
// P1
constexpr int kSplit1 = 2;      // groups of 4 waves taking turns over the 32-input steps
constexpr int kThreads1 = 256 * kSplit1;
constexpr int kTok1 = 64;       // tokens per workgroup (4 subtiles of 16)
constexpr int kTn1 = 4;
constexpr int kMaxMs = 6;       // 16-latent subtiles per wave
constexpr int kMinSteps = 12;   // fewest 32-input steps per split (when d_in allows)
constexpr int kMaxKbPer = 64;   // most 32-input steps per split (its g terms are held in LDS)
constexpr int kMinWg1 = 128;    // P1 workgroups wanted before latent tiles get thinner
constexpr int kPart = kTn1 * 64 * 4;  // partial floats per (token tile, path, subtile)
// P2
constexpr int kThreads2 = 512;  // 8 waves: two halves of 4 take alternate units
constexpr int kWaves2 = 8;
constexpr int kTok2 = 64;       // tokens per workgroup
constexpr int kUnit = 128;      // outputs per unit: 2 waves x 64
constexpr int kIm2 = 4;         // 16-output subtiles per wave
constexpr int kTn2 = 2;         // 16-token subtiles per wave
constexpr int kMaxKbc = 8;      // 32-latent blocks per chunk when w is not resident
constexpr size_t kLdsBudget = 160 * 1024;

typedef __attribute__((address_space(3))) void* lds_ptr;

struct PrefillParams {
  const void* x;
  void* y;
  const void* U[2];
  const void* V[2];
  const void* h[2];
  const void* g[2];
  const void* l[2];
  float* pbuf;      // P1: [ks][token tile][path][ns16p][4 token subtiles][64 lanes][4] partial sums
  uint32_t* wterm;  // [2][NW][nkb][T][4 lane groups] x 16 B: w terms as P2 B fragments
  void* lat;        // latent cache [T][2][r] (the latent-cache calls only)
  int T, d_in, d_out, r;
  int nkb, ns16;    // 32-latent blocks, 16-latent subtiles per path
  int n_tt, n_lt;   // P1 token tiles, latent tiles
  int ks, kb_per;   // P1 splits of d_in, 32-input steps per split
  int ns16p;        // P1 partial subtile slots per path
  int n_un, n_og, n_tt2;  // P2 units, unit groups, token tiles
  int res, kbc;     // P2: w resident / blocks per chunk
  int xdma;         // x rows are whole 16-byte chunks: global-to-LDS loads
  int vw;           // P1 V words in 16-byte loads (r % 4 == 0, V 16-byte aligned)
  int fast;         // P2 fast path (see prefill_p2)
  uint32_t v_bytes, u_bytes, g_bytes, h_bytes, l_bytes, wt_bytes;
  uint32_t wd_off;  // P2: byte offset of the U-word buffers in LDS
  int wdp;          // P2: U-word block slots per wave and buffer
};

// s_waitcnt: at most VM vector-memory operations outstanding, no LDS access
template <int VM>
__device__ __forceinline__ void wait_vm_lds() {
  static_assert(VM >= 0 && VM < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((VM & 15) | ((VM >> 4) << 14) | (7 << 4));
}

// ---------------------------------------------------------------------------
// P1
// ---------------------------------------------------------------------------
__host__ __device__ constexpr int p1_nx(int act) { return act == kDtF32 ? 2 : 1; }  // 16-byte chunks per lane
// V-word loads per wave and step: one 16-byte load (4 words a lane) when
// r % 4 == 0 and V is 16-byte aligned (VW), else dword loads of 64 words
__host__ __device__ constexpr int p1_nv(int ms, bool vw) { return vw ? 1 : (ms + 3) / 4; }
__host__ __device__ constexpr size_t p1_gt_bytes(int kb_per, int G) {
  return static_cast<size_t>(2) * kb_per * 4 * G * 16;
}
__host__ __device__ constexpr size_t p1_xslot(int nx) { return static_cast<size_t>(kTn1) * nx * 1024; }
__host__ __device__ constexpr size_t p1_vslot(int ms, bool vw) {
  return static_cast<size_t>(kWaves) * (vw ? 1024 : p1_nv(ms, false) * 256);
}
// 32-input steps staged in LDS, a whole number of rounds (fp32 x takes twice
// the room per step)
__host__ __device__ constexpr int p1_ring(int act) { return kSplit1 * (act == kDtF32 ? 4 : 6); }
__host__ __device__ constexpr size_t p1_lds(int kb_per, int G, int act, int ms, bool vw) {
  const size_t ring = p1_gt_bytes(kb_per, G) + p1_ring(act) * (p1_xslot(p1_nx(act)) + p1_vslot(ms, vw));
  const size_t red = static_cast<size_t>(kWaves) * ms * kTn1 * 64 * 16;
  return ring > red ? ring : red;
}

template <int MS, int ACT, int SC, bool VW>
__global__ void __launch_bounds__(kThreads1, 1) prefill_p1(PrefillParams P) {
  constexpr int G = nterms<SC>(), E = nterms<ACT>();
  constexpr int NX = p1_nx(ACT), NV = p1_nv(MS, VW), RING = p1_ring(ACT), RR = RING / kSplit1;
  constexpr int XSLOT = static_cast<int>(p1_xslot(NX)), VSLOT = static_cast<int>(p1_vslot(MS, VW));
  extern __shared__ __attribute__((aligned(16))) char lds[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (scalar)
  const int n16 = lane & 15, gq = lane >> 4;
  const int grp = wave >> 2, w4 = wave & 3;  // step group; the wave's role within its group
  const int pw = w4 >> 1, hw = w4 & 1;        // path and subtile half
  const int tiles = P.n_tt * P.n_lt;
  const int ksi = blockIdx.x / tiles;
  const int tile = blockIdx.x - ksi * tiles;
  const int lt = tile / P.n_tt;
  const int tt = tile - lt * P.n_tt;
  const int T = P.T, d_in = P.d_in, r = P.r;
  const int t0 = tt * kTok1;
  const int nbv = d_in >> 5, tailv = d_in & 31, nbt = nblocks32(d_in);
  const int kbs = ksi * P.kb_per, kbe = min(nbt, kbs + P.kb_per), ns = kbe - kbs;
  const int sb0 = lt * 2 * MS + hw;  // subtile of slot m: sb0 + 2 m

  u32x4* gt = reinterpret_cast<u32x4*>(lds);  // g terms [2][ns][4 lane groups][G]
  char* xs = lds + p1_gt_bytes(P.kb_per, G);  // x ring [RING][4 token subtiles][NX][64] x 16 B
  char* vs = xs + RING * XSLOT;               // V-word ring [RING][4 roles][VSLOT / 4]
  const int ex = ACT == kDtF32 ? 4 : 2;
  const int rows = min(kTok1, T - t0);
  // x of this tile's tokens (reads past the last token return zero)
  const rsrc_t xr = make_rsrc_uniform(static_cast<const char*>(P.x) + static_cast<int64_t>(t0) * d_in * ex,
                                      static_cast<uint32_t>(rows * d_in * ex));
  const rsrc_t vr = make_rsrc(pw ? P.V[1] : P.V[0], P.v_bytes);

  // loads of step n (split-local) into its ring slot, by the waves of its
  // group: the packed V words of this wave's subtiles (word of latent
  // 16 (sb0 + 2 m) + i at word 16 m + i of the wave's slice; zero past r, past
  // the range and for the tail step, whose words come through registers) and
  // token subtile w4 of x (zero past d_in and past the range)
  auto issue = [&](int n) {
    const int kb = kbs + n, sl = n % RING;
    const bool valid = n < ns;
    char* vd = vs + sl * VSLOT + w4 * (VSLOT / kWaves);
    if constexpr (VW) {
      // lane l: words of latents 16 (sb0 + 2 (l / 4)) + 4 (l % 4) .. + 3
      const int m = lane >> 2;
      const int k = 16 * (sb0 + 2 * m) + 4 * (lane & 3);
      const bool ok = valid && kb < nbv && m < MS && k < r;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(vr, (lds_ptr)vd, 16,
                                               ok ? static_cast<uint32_t>(kb * r + k) * 4u : kOob, 0, 0, 0);
    } else {
      // lane l of load d: the word of latent 16 (sb0 + 2 m) + l % 16, m = 4 d + l / 16
#pragma unroll
      for (int d = 0; d < NV; ++d) {
        const int m = 4 * d + gq;
        const int k = 16 * (sb0 + 2 * m) + n16;
        const bool ok = valid && kb < nbv && m < MS && k < r;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(vr, (lds_ptr)(vd + d * 256), 4,
                                                 ok ? static_cast<uint32_t>(kb * r + k) * 4u : kOob, 0, 0, 0);
      }
    }
    const int row = 16 * w4 + n16;
    char* xd = xs + sl * XSLOT + w4 * NX * 1024;
    if (P.xdma) {
#pragma unroll
      for (int c = 0; c < NX; ++c) {
        const int j = 32 * kb + 8 * gq + 4 * c;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            xr, (lds_ptr)(xd + c * 1024), 16,
            valid && j < d_in ? static_cast<uint32_t>(row * d_in + j) * static_cast<uint32_t>(ex) : kOob, 0, 0, 0);
      }
    } else {
      // element loads (rows not whole 16-byte chunks), written in the same order
#pragma unroll
      for (int c = 0; c < NX; ++c) {
        const int j = 32 * kb + 8 * gq + 4 * c;
        const uint32_t e0 = static_cast<uint32_t>(row * d_in + j);
        u32x4 dv;
        if constexpr (ACT == kDtF32) {
#pragma unroll
          for (int e = 0; e < 4; ++e) dv[e] = bload<ACT>(xr, e0 + e, valid && j + e < d_in);
        } else {
#pragma unroll
          for (int v = 0; v < 4; ++v)
            dv[v] = bload<ACT>(xr, e0 + 2 * v, valid && j + 2 * v < d_in) |
                    (bload<ACT>(xr, e0 + 2 * v + 1, valid && j + 2 * v + 1 < d_in) << 16);
        }
        *reinterpret_cast<u32x4*>(xd + c * 1024 + lane * 16) = dv;
      }
    }
  };

  // the first RR - 1 rounds (kSplit1 steps each, one per group) in flight
#pragma unroll
  for (int d = 0; d < RR - 1; ++d) issue(kSplit1 * d + grp);

  // packed V words of the tail step (tail plane: 16- or 32-bit entries)
  uint32_t tw[MS];
  const bool has_tail = tailv != 0 && kbe == nbt;
#pragma unroll
  for (int m = 0; m < MS; ++m) {
    const int k = 16 * (sb0 + 2 * m) + n16;
    const bool ok = has_tail && k < r;
    const uint32_t off = 4u * nbv * r + (tailv <= 16 ? 2u : 4u) * k;
    const uint32_t lo = __builtin_amdgcn_raw_buffer_load_b16(vr, ok ? off : kOob, 0, 0);
    const uint32_t hi = __builtin_amdgcn_raw_buffer_load_b16(vr, ok && tailv > 16 ? off + 2 : kOob, 0, 0);
    tw[m] = (lo & 0xffffu) | (hi << 16);
  }
  // g terms of both paths for this split's steps, in A-operand order:
  // gt[p][step][lane group][term], register v = terms of inputs 2 v, 2 v + 1
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    const rsrc_t gr = make_rsrc(p ? P.g[1] : P.g[0], P.g_bytes);
    for (int it = tid; it < ns * 4; it += kThreads1) {
      const int kbl = it >> 2, g4 = it & 3;
      const int j0 = 32 * (kbs + kbl) + 8 * g4;
      uint32_t tm[8][G];
#pragma unroll
      for (int e = 0; e < 8; ++e) split_exact<G>(bits_to_f32<SC>(bload<SC>(gr, j0 + e, j0 + e < d_in)), tm[e]);
#pragma unroll
      for (int s = 0; s < G; ++s) {
        u32x4 dv;
#pragma unroll
        for (int v = 0; v < 4; ++v) dv[v] = tm[2 * v][s] | (tm[2 * v + 1][s] << 16);
        gt[((p * ns + kbl) * 4 + g4) * G + s] = dv;
      }
    }
  }

  floatx4 acc[MS][kTn1];
#pragma unroll
  for (int m = 0; m < MS; ++m)
#pragma unroll
    for (int tn = 0; tn < kTn1; ++tn) acc[m][tn] = floatx4{0.f, 0.f, 0.f, 0.f};

  const u32x4* gtp = gt + pw * ns * 4 * G;
  const int nr = (ns + kSplit1 - 1) / kSplit1;  // rounds: step kSplit1 i + grp in round i
  for (int i = 0; i < nr; ++i) {
    // round i has landed (each wave waits for its own loads, the barrier for
    // everyone's) and every wave is done with the slots of round i - 1
    asm volatile("" ::: "memory");  // round i - 1's LDS reads stay above the barrier
    wait_vm_lds<(RR - 2) * (NX + NV)>();
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    const int n = kSplit1 * i + grp;
    if (n >= ns) {  // (a short last round: the later groups sit it out)
      issue(kSplit1 * (i + RR - 1) + grp);
      continue;
    }
    const int sl = n % RING;
    const bool tail = kbs + n == nbv;

    // B: x of the 4 token subtiles as E exact bf16 terms
    u32x4 B[kTn1][E];
    const char* xsl = xs + sl * XSLOT;
#pragma unroll
    for (int tn = 0; tn < kTn1; ++tn) {
      if constexpr (ACT == kDtBF16) {
        B[tn][0] = *reinterpret_cast<const u32x4*>(xsl + tn * 1024 + lane * 16);
      } else {
        uint32_t el[8];
        if constexpr (ACT == kDtF32) {
          const u32x4 a = *reinterpret_cast<const u32x4*>(xsl + (2 * tn) * 1024 + lane * 16);
          const u32x4 b = *reinterpret_cast<const u32x4*>(xsl + (2 * tn + 1) * 1024 + lane * 16);
#pragma unroll
          for (int e = 0; e < 4; ++e) el[e] = a[e], el[4 + e] = b[e];
        } else {
          const u32x4 a = *reinterpret_cast<const u32x4*>(xsl + tn * 1024 + lane * 16);
#pragma unroll
          for (int v = 0; v < 4; ++v) el[2 * v] = a[v] & 0xffffu, el[2 * v + 1] = a[v] >> 16;
        }
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          uint32_t lo[E], hi[E];
          split_exact<E>(bits_to_f32<ACT>(el[2 * v]), lo);
          split_exact<E>(bits_to_f32<ACT>(el[2 * v + 1]), hi);
#pragma unroll
          for (int e = 0; e < E; ++e) B[tn][e][v] = lo[e] | (hi[e] << 16);
        }
      }
    }
    // A: V signs on the g terms of this wave's path
    u32x4 gv[G];
#pragma unroll
    for (int s = 0; s < G; ++s) gv[s] = gtp[(n * 4 + gq) * G + s];
    const uint32_t* vw = reinterpret_cast<const uint32_t*>(vs + sl * VSLOT + w4 * (VSLOT / kWaves));
    uint32_t words[MS];
#pragma unroll
    for (int m = 0; m < MS; ++m) words[m] = tail ? tw[m] : vw[16 * m + n16];
    // the loads of round i + RR - 1 (into the slots of round i - 1, free since
    // the barrier), issued once this step's LDS reads are out
    issue(kSplit1 * (i + RR - 1) + grp);
    u32x4 A[MS][G];
#pragma unroll
    for (int m = 0; m < MS; ++m) {
      const uint32_t word = words[m];
      const uint32_t t = word >> (8 * gq);
      const uint32_t dd = (t & 0xffffu) | ((t << 15) & 0xffff0000u);
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const uint32_t sv = (dd << (15 - 2 * v)) & 0x80008000u;
#pragma unroll
        for (int s = 0; s < G; ++s) A[m][s][v] = sv ^ gv[s][v];
      }
    }
#pragma unroll
    for (int s = 0; s < G; ++s)
#pragma unroll
      for (int e = 0; e < E; ++e)
#pragma unroll
        for (int m = 0; m < MS; ++m)
#pragma unroll
          for (int tn = 0; tn < kTn1; ++tn) acc[m][tn] = mfma(A[m][s], B[tn][e], acc[m][tn]);
  }

  // the groups' sums, in a fixed order (((group 0 + group 1) + group 2) ...),
  // through LDS (the ring is dead after the first barrier), then this role's
  // partial sums: pbuf[ks][token tile][path][subtile][token subtile][lane][4]
  asm volatile("" ::: "memory");
  wait_vm_lds<0>();
  floatx4* red = reinterpret_cast<floatx4*>(lds) + w4 * MS * kTn1 * 64;
#pragma unroll
  for (int src = 1; src < kSplit1; ++src) {
    __syncthreads();
    if (grp == src) {
#pragma unroll
      for (int m = 0; m < MS; ++m)
#pragma unroll
        for (int tn = 0; tn < kTn1; ++tn) red[(m * kTn1 + tn) * 64 + lane] = acc[m][tn];
    }
    __syncthreads();
    if (grp == 0) {
#pragma unroll
      for (int m = 0; m < MS; ++m)
#pragma unroll
        for (int tn = 0; tn < kTn1; ++tn) acc[m][tn] += red[(m * kTn1 + tn) * 64 + lane];
    }
  }
  if (grp == 0) {
    float* part = P.pbuf + ((static_cast<int64_t>(ksi) * P.n_tt + tt) * 2 + pw) * P.ns16p * kPart;
#pragma unroll
    for (int m = 0; m < MS; ++m) {
      const int s = sb0 + 2 * m;
      if (s < P.ns16) {
#pragma unroll
        for (int tn = 0; tn < kTn1; ++tn)
          *reinterpret_cast<floatx4*>(part + (s * kTn1 + tn) * 256 + lane * 4) = acc[m][tn];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// P1b: w = l (.) (sum of the ks partials, ascending) as NW bf16 terms in P2's
// B-fragment layout wterm[p][term][kbl][t][lane group]; one thread per
// (pair, token tile, token subtile, P2 lane), so a wave reads 1 KB runs.  The
// latent-cache kernels share its thread mapping: prefill_latent_out stores w
// itself (the cache), prefill_latent_in cuts a stored w into the terms.
// ---------------------------------------------------------------------------
struct PairItem {
  int t, p, kbl, g4;  // token, path, 32-latent block, lane group
  int tt, tn, ln;     // P1 token tile, its 16-token subtile, P2 lane
};

// the item of this thread; false past the last pair or token
__device__ __forceinline__ bool pair_item(const PrefillParams& P, PairItem& it, int bid = -1) {
  const int item = (bid < 0 ? static_cast<int>(blockIdx.x) : bid) * kThreads + threadIdx.x;
  it.ln = item & 63;
  it.tn = (item >> 6) & 3;
  const int rest = item >> 8;
  it.tt = rest % P.n_tt;
  const int q = rest / P.n_tt;  // (path, 32-latent block)
  if (q >= 2 * P.nkb) return false;
  it.t = it.tt * kTok1 + 16 * it.tn + (it.ln & 15);
  if (it.t >= P.T) return false;
  it.g4 = it.ln >> 4;
  it.p = q >= P.nkb ? 1 : 0;
  it.kbl = q - it.p * P.nkb;
  return true;
}

// w0[v] = w of latent 32 kbl + 4 g4 + v and w1[v] of the same + 16 (0 past r):
// the ks partial sums added in ascending split order, times l (SCALE) or not
template <int SC, bool SCALE = true>
__device__ __forceinline__ void latent_w(const PrefillParams& P, const PairItem& it, float (&w0)[4], float (&w1)[4]) {
  // subtiles 2 kbl (latents 32 kbl + 4 g4 + v) and 2 kbl + 1 (the same + 16)
  const float* src =
      P.pbuf + ((static_cast<int64_t>(it.tt) * 2 + it.p) * P.ns16p + 2 * it.kbl) * kPart + it.tn * 256 + it.ln * 4;
  const int64_t kstride = static_cast<int64_t>(P.n_tt) * 2 * P.ns16p * kPart;
  floatx4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = s0;
#pragma unroll 8
  for (int k2 = 0; k2 < P.ks; ++k2) {
    const float* sp = src + k2 * kstride;
    s0 += *reinterpret_cast<const floatx4*>(sp);
    s1 += *reinterpret_cast<const floatx4*>(sp + kPart);
  }
  const int r = P.r;
  const rsrc_t lr = make_rsrc(it.p ? P.l[1] : P.l[0], P.l_bytes);
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int k = 32 * it.kbl + 4 * it.g4 + v;
    const float a = SCALE ? s0[v] * bits_to_f32<SC>(bload<SC>(lr, k, k < r)) : s0[v];
    const float b = SCALE ? s1[v] * bits_to_f32<SC>(bload<SC>(lr, k + 16, k + 16 < r)) : s1[v];
    w0[v] = k < r ? a : 0.0f;
    w1[v] = k + 16 < r ? b : 0.0f;
  }
}

// w0 / w1 (as from latent_w) cut into NW bf16 terms, stored as P2 B fragments
template <int NW>
__device__ __forceinline__ void store_wterm(const PrefillParams& P, const PairItem& it, const float (&w0)[4],
                                            const float (&w1)[4]) {
  uint32_t lo[NW][4], hi[NW][4];
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    uint32_t a[NW], b[NW];
    split_round<NW>(w0[v], a);
    split_round<NW>(w1[v], b);
#pragma unroll
    for (int e = 0; e < NW; ++e) lo[e][v] = a[e], hi[e][v] = b[e];
  }
#pragma unroll
  for (int e = 0; e < NW; ++e) {
    u32x4 d;
#pragma unroll
    for (int v = 0; v < 4; ++v) d[v] = lo[e][v] | (hi[e][v] << 16);
    reinterpret_cast<u32x4*>(P.wterm)[((static_cast<int64_t>(it.p * NW + e) * P.nkb + it.kbl) * P.T + it.t) * 4 +
                                      it.g4] = d;
  }
}

template <int ACT, int SC>
__global__ void __launch_bounds__(kThreads) prefill_p1b(PrefillParams P) {
  constexpr int NW = ACT == kDtF32 ? 3 : 2;
  PairItem it;
  if (!pair_item(P, it)) return;
  float w0[4], w1[4];
  latent_w<SC>(P, it, w0, w1);
  store_wterm<NW>(P, it, w0, w1);
}

// The latent cache [T][2][r] (dtype LD, rounded to nearest even when 16-bit):
// element (t, p, k) at (2 t + p) r + k.  SCALE: l (.) z (the cache); else z
// itself (the backward keeps it in fp32)
template <int SC, int LD, bool SCALE = true>
__global__ void __launch_bounds__(kThreads) prefill_latent_out(PrefillParams P) {
  PairItem it;
  if (!pair_item(P, it)) return;
  float w0[4], w1[4];
  latent_w<SC, SCALE>(P, it, w0, w1);
  const int r = P.r;
  const int64_t row = (static_cast<int64_t>(it.t) * 2 + it.p) * r;
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int k = 32 * it.kbl + 4 * it.g4 + v;
    if (k < r) st<LD>(P.lat, row + k, w0[v]);
    if (k + 16 < r) st<LD>(P.lat, row + k + 16, w1[v]);
  }
}

// w terms of P2 from a stored [T][2][r] array: the cache itself, or (SC >= 0)
// its product with l (the backward's dz = l (.) dw)
// fp32 stage-1 sums (no l) of two linears in one launch: the first nb0
// workgroups for Q0, the rest for Q1
template <int SC>
__global__ void __launch_bounds__(kThreads) prefill_sums2(PrefillParams Q0, PrefillParams Q1, int nb0) {
  const bool second = static_cast<int>(blockIdx.x) >= nb0;
  const PrefillParams& P = second ? Q1 : Q0;
  PairItem it;
  if (!pair_item(P, it, second ? static_cast<int>(blockIdx.x) - nb0 : static_cast<int>(blockIdx.x))) return;
  float w0[4], w1[4];
  latent_w<SC, false>(P, it, w0, w1);
  const int r = P.r;
  const int64_t row = (static_cast<int64_t>(it.t) * 2 + it.p) * r;
  float* z = static_cast<float*>(P.lat);
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int k = 32 * it.kbl + 4 * it.g4 + v;
    if (k < r) z[row + k] = w0[v];
    if (k + 16 < r) z[row + k + 16] = w1[v];
  }
}

template <int ACT, int LD, int SC = -1>
__global__ void __launch_bounds__(kThreads) prefill_latent_in(PrefillParams P) {
  constexpr int NW = ACT == kDtF32 ? 3 : 2;
  PairItem it;
  if (!pair_item(P, it)) return;
  const int r = P.r;
  const int64_t row = (static_cast<int64_t>(it.t) * 2 + it.p) * r;
  float w0[4], w1[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int k = 32 * it.kbl + 4 * it.g4 + v;
    w0[v] = ld_or0<LD>(P.lat, row + k, k < r);
    w1[v] = ld_or0<LD>(P.lat, row + k + 16, k + 16 < r);
  }
  if constexpr (SC >= 0) {
    const rsrc_t lr = make_rsrc(it.p ? P.l[1] : P.l[0], P.l_bytes);
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int k = 32 * it.kbl + 4 * it.g4 + v;
      w0[v] *= bits_to_f32<SC>(bload<SC>(lr, k, k < r));
      w1[v] *= bits_to_f32<SC>(bload<SC>(lr, k + 16, k + 16 < r));
    }
  }
  store_wterm<NW>(P, it, w0, w1);
}

// ---------------------------------------------------------------------------
// P2
// ---------------------------------------------------------------------------
// LDS of P2: w fragments [held pairs][4 token subtiles][NW][64 lanes] x 16 B,
// then per buffer and wave: U words [held pairs][64] x 4 B, row scales
// [2 paths][256 B] and 16-bit tail words [2 paths][256 B]
__host__ __device__ constexpr size_t p2_w_bytes(int pairs, int nw) {
  return static_cast<size_t>(pairs) * 4 * nw * 1024;
}
__host__ __device__ constexpr int p2_wave_bytes(int pairs) { return pairs * 256 + 1024; }
__host__ __device__ constexpr size_t p2_wd_bytes(int pairs, int bufs) {
  return static_cast<size_t>(bufs) * kWaves2 * p2_wave_bytes(pairs);
}

// two fp32 values rounded to nearest-even bf16 / f16, packed (the gfx950
// packed converts)
template <int DT>
__device__ __forceinline__ uint32_t pack2(float a, float b) {
  typedef float f2 __attribute__((ext_vector_type(2)));
  // f16: round the fp32 values themselves (see st<>)
  if constexpr (DT != kDtBF16) asm volatile("" : "+v"(a), "+v"(b));
  const f2 v = {a, b};
  if constexpr (DT == kDtBF16) {
    typedef __bf16 h2 __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, h2));
  } else {
    typedef _Float16 h2 __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, h2));
  }
}

// sign_terms for +-1.0 pairs with one bitfield insert per register: M (the
// two bf16 sign bits) and B (two bf16 1.0) are kept in registers by the
// caller, opaque to constant folding, so that (x & M) | (B & ~M) becomes
// v_bfi_b32 instead of an and and an or with literals
__device__ __forceinline__ u32x4 sign_ones(uint32_t word, int gq, uint32_t M, uint32_t B) {
  const uint32_t ws = word >> (4 * gq);
  u32x4 a;
#pragma unroll
  for (int v = 0; v < 4; ++v) a[v] = ((ws << (15 - v)) & M) | (B & ~M);
  return a;
}

// FAST: d_out % 4 == 0 and aligned U, h and y, so the U words of a unit come
// in 16-byte global-to-LDS loads (4 blocks of 64 outputs a load), its scales
// and 16-bit tail words in dword ones (all prefetched a unit ahead) and y in
// 4-output stores; otherwise words come in dword loads, scales and tail words
// per unit through registers and y element by element
template <int ACT, int SC, bool FAST>
__global__ void __launch_bounds__(kThreads2, 1) prefill_p2(PrefillParams P) {
  constexpr int NW = ACT == kDtF32 ? 3 : 2;
  constexpr int ES = SC == kDtF32 ? 4 : 2;
  extern __shared__ __attribute__((aligned(16))) char lds[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (scalar)
  const int n16 = lane & 15, gq = lane >> 4;
  const int hu = wave >> 2, w4 = wave & 3;  // unit parity; the wave's role within its half
  const int oh = w4 & 1, th = w4 >> 1;      // output half, token half of a unit
  const int tt = blockIdx.x % P.n_tt2;
  const int og = blockIdx.x / P.n_tt2;
  const int T = P.T, d_out = P.d_out, r = P.r, nkb = P.nkb;
  const int t0 = tt * kTok2;
  const int nbu = r >> 5, tailu = r & 31;
  const int nfull = nbu + (tailu > 16 ? 1 : 0);  // blocks with 32-bit words
  const bool t16 = tailu != 0 && tailu <= 16;     // block nbu has 16-bit words
  const bool res = P.res != 0;
  const int held = res ? 2 * nkb : P.kbc;  // w pairs in LDS at once
  const int wdp = P.wdp;                   // U-word block slots per wave and buffer
  const int ws1 = res ? wdp / 2 : 0;       // slot of path 1's first block (resident)
  const int wvb = p2_wave_bytes(wdp);
  const rsrc_t wr = make_rsrc(P.wterm, P.wt_bytes);
  const rsrc_t ur[2] = {make_rsrc(P.U[0], P.u_bytes), make_rsrc(P.U[1], P.u_bytes)};
  const rsrc_t hr[2] = {make_rsrc(P.h[0], P.h_bytes), make_rsrc(P.h[1], P.h_bytes)};
  char* wl = lds;
  char* wd = lds + P.wd_off;
  auto region = [&](int buf) { return wd + (buf * kWaves2 + wave) * wvb; };

  // w fragments of pairs (p, kb0 .. kb0 + nb - 1) into held slots from hs0
  auto load_w = [&](int p, int kb0, int nb, int hs0) {
    const int ng = nb * 4 * NW;
    for (int gi = wave; gi < ng; gi += kWaves2) {
      const int e = gi % NW;
      const int tn = (gi / NW) & 3;
      const int kbl = gi / (4 * NW);
      const int t = t0 + 16 * tn + n16;
      const uint32_t off =
          static_cast<uint32_t>(((static_cast<int64_t>(p * NW + e) * nkb + kb0 + kbl) * T + t) * 4 + gq) * 16u;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(wr, (lds_ptr)(wl + ((hs0 + kbl) * 4 * NW + (gi % (4 * NW))) * 1024),
                                               16, t < T ? off : kOob, 0, 0, 0);
    }
  };
  // U words (32-bit: full words and a tail block of more than 16 latents) of
  // blocks kb0 .. kb0 + nb - 1 of path p for this wave's 64 outputs of unit u
  auto load_words = [&](int u, int p, int kb0, int nb, int buf, int hs0) {
    char* dst = region(buf) + hs0 * 256;
    const int nf = min(nb, nfull - kb0);
    if constexpr (FAST) {
      // lane l: block kb0 + kbl0 + l / 16, outputs ob + 4 (l % 16) .. + 3
      const int o = u * kUnit + 64 * oh + 4 * (lane & 15);
      for (int kbl0 = 0; kbl0 < nf; kbl0 += 4) {
        const int kbl = kbl0 + (lane >> 4);
        const int kb = kb0 + kbl;
        const uint32_t off = kb < nbu ? static_cast<uint32_t>(kb * d_out + o) * 4u : 4u * nbu * d_out + 4u * o;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(ur[p], (lds_ptr)(dst + kbl0 * 256), 16,
                                                 kbl < nf && o < d_out ? off : kOob, 0, 0, 0);
      }
    } else {
      const int o = u * kUnit + 64 * oh + lane;
      const bool ok = o < d_out;
      for (int kbl = 0; kbl < nf; ++kbl) {
        const int kb = kb0 + kbl;
        const uint32_t off = kb < nbu ? static_cast<uint32_t>(kb * d_out + o) * 4u : 4u * nbu * d_out + 4u * o;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(ur[p], (lds_ptr)(dst + kbl * 256), 4, ok ? off : kOob, 0, 0, 0);
      }
    }
  };
  // FAST: row scales and 16-bit tail words of unit u as whole dwords (lane l:
  // scales of outputs 2 l, 2 l + 1 for 16-bit scales, l for fp32; tail words
  // of outputs 2 l, 2 l + 1)
  auto load_side = [&](int u, int buf) {
    const int ob = u * kUnit + 64 * oh;
    char* dst = region(buf) + wdp * 256;
    const int oe = ES == 2 ? ob + 2 * lane : ob + lane;
    const int ot = ob + 2 * lane;
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      __builtin_amdgcn_raw_ptr_buffer_load_lds(hr[p], (lds_ptr)(dst + p * 256), 4,
                                               oe < d_out ? static_cast<uint32_t>(oe) * ES : kOob, 0, 0, 0);
      if (t16)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(ur[p], (lds_ptr)(dst + 512 + p * 256), 4,
                                                 ot < d_out ? 4u * nbu * d_out + 2u * ot : kOob, 0, 0, 0);
    }
  };
  // not FAST: 16-bit tail words of this wave's outputs of unit u in registers
  auto load_tw = [&](int u, uint32_t (&tw)[2][kIm2]) {
    const int ob = u * kUnit + 64 * oh;
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
      for (int im = 0; im < kIm2; ++im) {
        const int i = ob + 16 * im + n16;
        tw[p][im] = __builtin_amdgcn_raw_buffer_load_b16(ur[p], t16 && i < d_out ? 4u * nbu * d_out + 2u * i : kOob,
                                                         0, 0);
      }
  };
  // row scales of outputs ob + 16 im + 4 gq + e as floats
  auto scales = [&](int u, int buf, float (&hf)[2][kIm2][4]) {
    const int ob = u * kUnit + 64 * oh;
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
      for (int im = 0; im < kIm2; ++im) {
        uint32_t raw[4];
        if constexpr (FAST) {
          const char* src = region(buf) + wdp * 256 + p * 256 + (16 * im + 4 * gq) * ES;
          if constexpr (ES == 4) {
            const u32x4 v = *reinterpret_cast<const u32x4*>(src);
            raw[0] = v[0], raw[1] = v[1], raw[2] = v[2], raw[3] = v[3];
          } else {
            const u32x2 v = *reinterpret_cast<const u32x2*>(src);
            raw[0] = v[0], raw[1] = v[1], raw[2] = raw[3] = 0u;
          }
#pragma unroll
          for (int e = 0; e < 4; ++e) hf[p][im][e] = raw4_elem<SC, true>(raw, e);
        } else {
          bload4<SC, false>(hr[p], ob + 16 * im + 4 * gq, true, raw);
#pragma unroll
          for (int e = 0; e < 4; ++e) hf[p][im][e] = raw4_elem<SC, false>(raw, e);
        }
      }
  };

  floatx4 acc[2][kIm2][kTn2];
  uint32_t sgn_m = 0x80008000u, one_b = 0x3F803F80u;
  asm volatile("" : "+v"(sgn_m), "+v"(one_b));
  // products of one held pair: w from held slot hs, the U words from LDS
  // (full) or the 16-bit tail words (W16)
  auto pair = [&](auto pc, auto w16, int hs, const uint32_t* words, int buf, const uint32_t (&tw)[kIm2]) {
    constexpr int p = decltype(pc)::value;
    constexpr bool W16 = decltype(w16)::value;
    u32x4 B[kTn2][NW];
#pragma unroll
    for (int tn = 0; tn < kTn2; ++tn)
#pragma unroll
      for (int e = 0; e < NW; ++e)
        B[tn][e] = *reinterpret_cast<const u32x4*>(wl + ((hs * 4 + 2 * th + tn) * NW + e) * 1024 + lane * 16);
#pragma unroll
    for (int im = 0; im < kIm2; ++im) {
      uint32_t word;
      if constexpr (!W16)
        word = words[16 * im + n16];
      else if constexpr (FAST)
        word = *reinterpret_cast<const uint16_t*>(region(buf) + wdp * 256 + 512 + p * 256 + (16 * im + n16) * 2);
      else
        word = tw[im] & 0xffffu;
      const u32x4 A = sign_ones(word, gq, sgn_m, one_b);
#pragma unroll
      for (int e = 0; e < NW; ++e)
#pragma unroll
        for (int tn = 0; tn < kTn2; ++tn) acc[p][im][tn] = mfma(A, B[tn][e], acc[p][im][tn]);
    }
  };
  using False = std::integral_constant<bool, false>;
  using True = std::integral_constant<bool, true>;
  // products of held pairs (p, kb0 .. kb0 + nb - 1): w at held slots from
  // hs0, U words at word slots from ds0
  auto run = [&](auto pc, int kb0, int nb, int hs0, int ds0, int buf, const uint32_t (&tw)[kIm2]) {
    const uint32_t* words = reinterpret_cast<const uint32_t*>(region(buf) + ds0 * 256);
    const int nf = max(0, min(nb, nfull - kb0));
    for (int kbl = 0; kbl < nf; ++kbl) pair(pc, False{}, hs0 + kbl, words + kbl * 64, buf, tw);
    if (t16 && nbu >= kb0 && nbu < kb0 + nb) pair(pc, True{}, hs0 + nbu - kb0, words, buf, tw);
  };
  // y[t][i] = h_0[i] acc_0 + h_1[i] acc_1, outputs i = ob + 16 im + 4 gq + e of
  // token t = t0 + 16 (2 th + tn) + n16
  const int ey = ACT == kDtF32 ? 4 : 2;
  const rsrc_t yr = make_rsrc_uniform(static_cast<char*>(P.y) + static_cast<int64_t>(t0) * d_out * ey,
                                      static_cast<uint32_t>(min(kTok2, T - t0) * d_out * ey));
  auto store = [&](int u, const float (&hf)[2][kIm2][4]) {
    const int ob = u * kUnit + 64 * oh;
#pragma unroll
    for (int im = 0; im < kIm2; ++im) {
      const int ib = ob + 16 * im + 4 * gq;
#pragma unroll
      for (int tn = 0; tn < kTn2; ++tn) {
        const int t = t0 + 16 * (2 * th + tn) + n16;
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = hf[0][im][e] * acc[0][im][tn][e] + hf[1][im][e] * acc[1][im][tn][e];
        const uint32_t base = static_cast<uint32_t>((t - t0) * d_out + ib);  // within the tile's rows
        if constexpr (FAST) {
          // whole groups of 4 outputs (d_out % 4 == 0); rows past T are past the buffer
          const bool ok = t < T && ib < d_out;
          if constexpr (ACT == kDtF32) {
            const u32x4 d = {__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]),
                             __float_as_uint(v[3])};
            __builtin_amdgcn_raw_buffer_store_b128(d, yr, ok ? base * 4u : kOob, 0, 0);
          } else {
            const u32x2 d = {pack2<ACT>(v[0], v[1]), pack2<ACT>(v[2], v[3])};
            __builtin_amdgcn_raw_buffer_store_b64(d, yr, ok ? base * 2u : kOob, 0, 0);
          }
        } else {
          if (t < T) {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (ib + e < d_out) st<ACT>(P.y, static_cast<int64_t>(t) * d_out + ib + e, v[e]);
          }
        }
      }
    }
  };
  auto zero_acc = [&]() {
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
      for (int im = 0; im < kIm2; ++im)
#pragma unroll
        for (int tn = 0; tn < kTn2; ++tn) acc[p][im][tn] = floatx4{0.f, 0.f, 0.f, 0.f};
  };
  using P0 = std::integral_constant<int, 0>;
  using P1 = std::integral_constant<int, 1>;

  uint32_t tw[2][kIm2] = {};
  float hf[2][kIm2][4];
  if (FAST && res) {
    // every w fragment of the tile, once; then the units, each with the next
    // unit's words, scales and tail words in flight (global-to-LDS loads only:
    // the one wait per unit sits before its stores, so no unit waits for its
    // own stores)
    load_w(0, 0, nkb, 0);
    load_w(1, 0, nkb, nkb);
    int u = og + hu * P.n_og;
    if (u < P.n_un) {
      load_words(u, 0, 0, nkb, 0, 0);
      load_words(u, 1, 0, nkb, 0, ws1);
      load_side(u, 0);
    }
    __builtin_amdgcn_s_waitcnt(0);  // global-to-LDS loads count as memory loads
    __syncthreads();
    for (int k = 0; u < P.n_un; ++k, u += 2 * P.n_og) {
      asm volatile("" ::: "memory");  // the previous unit's LDS reads stay above the next loads
      const int un = u + 2 * P.n_og;
      const int buf = k & 1;
      if (un < P.n_un) {
        load_words(un, 0, 0, nkb, buf ^ 1, 0);
        load_words(un, 1, 0, nkb, buf ^ 1, ws1);
        load_side(un, buf ^ 1);
      }
      zero_acc();
      run(P0{}, 0, nkb, 0, 0, buf, tw[0]);
      run(P1{}, 0, nkb, nkb, ws1, buf, tw[1]);
      // the next unit's loads (issued a unit ago) and the previous unit's
      // stores have landed: this wait is before the stores, not after them
      __builtin_amdgcn_s_waitcnt(0);
      scales(u, buf, hf);
      store(u, hf);
    }
  } else {
    // per pair of units (one per half), per chunk of held blocks of one
    // path, everything waited for (a half without a unit only keeps the
    // barriers)
    for (int u0 = og; u0 < P.n_un; u0 += 2 * P.n_og) {
      const int u = u0 + hu * P.n_og;
      const bool act = u < P.n_un;
      if (!FAST && act) load_tw(u, tw);
      zero_acc();
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        for (int kb0 = 0; kb0 < nkb; kb0 += held) {
          const int nb = min(held, nkb - kb0);
          __syncthreads();  // the previous chunk's readers are done
          load_w(p, kb0, nb, 0);
          if (act) {
            load_words(u, p, kb0, nb, 0, 0);
            if (FAST && p == 0 && kb0 == 0) load_side(u, 0);
          }
          __builtin_amdgcn_s_waitcnt(0);
          __syncthreads();
          if (act) {
            if (p == 0)
              run(P0{}, kb0, nb, 0, 0, 0, tw[0]);
            else
              run(P1{}, kb0, nb, 0, 0, 0, tw[1]);
          }
        }
      }
      if (act) {
        scales(u, 0, hf);
        store(u, hf);
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

template <int MS, int ACT, int SC, bool VW>
hipError_t launch_p1v(const PrefillParams& P, const PrefillGeom& g, hipStream_t stream) {
  static std::atomic<size_t> limit{65536};
  hipError_t e = raise_lds_limit(&prefill_p1<MS, ACT, SC, VW>, g.smem1, limit);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((prefill_p1<MS, ACT, SC, VW>), dim3(g.n_tt * g.n_lt * g.ks), dim3(kThreads1), g.smem1, stream,
                     P);
  return hipGetLastError();
}
template <int MS, int ACT, int SC>
hipError_t launch_p1(const PrefillParams& P, const PrefillGeom& g, hipStream_t stream) {
  return P.vw ? launch_p1v<MS, ACT, SC, true>(P, g, stream) : launch_p1v<MS, ACT, SC, false>(P, g, stream);
}

template <int ACT, int SC, bool FAST>
hipError_t launch_p2(const PrefillParams& P, const PrefillGeom& g, hipStream_t stream) {
  static std::atomic<size_t> limit{65536};
  hipError_t e = raise_lds_limit(&prefill_p2<ACT, SC, FAST>, g.smem2, limit);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((prefill_p2<ACT, SC, FAST>), dim3(g.n_og * g.n_tt2), dim3(kThreads2), g.smem2, stream, P);
  return hipGetLastError();
}

template <int ACT, int SC>
hipError_t launch_p1_ms(const PrefillParams& P, const PrefillGeom& g, hipStream_t stream) {
  switch (g.ms) {
    case 1: return launch_p1<1, ACT, SC>(P, g, stream);
    case 2: return launch_p1<2, ACT, SC>(P, g, stream);
    case 3: return launch_p1<3, ACT, SC>(P, g, stream);
    case 4: return launch_p1<4, ACT, SC>(P, g, stream);
    case 5: return launch_p1<5, ACT, SC>(P, g, stream);
    default: return launch_p1<kMaxMs, ACT, SC>(P, g, stream);
  }
}

// grid of the pair kernels (P1b and the latent-cache kernels)
dim3 pair_grid(const PrefillParams& P) {
  const int items = 2 * P.nkb * P.n_tt * 256;
  return dim3((items + kThreads - 1) / kThreads);
}

template <int ACT, int SC>
hipError_t launch_p2_any(const PrefillParams& P, const PrefillGeom& g, hipStream_t stream) {
  return P.fast ? launch_p2<ACT, SC, true>(P, g, stream) : launch_p2<ACT, SC, false>(P, g, stream);
}

template <int ACT, int SC>
hipError_t launch_all(const PrefillParams& P, const PrefillGeom& g, hipStream_t stream) {
  hipError_t e = launch_p1_ms<ACT, SC>(P, g, stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((prefill_p1b<ACT, SC>), pair_grid(P), dim3(kThreads), 0, stream, P);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return launch_p2_any<ACT, SC>(P, g, stream);
}

template <int ACT>
hipError_t launch_act(const PrefillParams& P, int sc_dt, const PrefillGeom& g, hipStream_t stream) {
  switch (sc_dt) {
    case kDtF32: return launch_all<ACT, kDtF32>(P, g, stream);
    case kDtF16: return launch_all<ACT, kDtF16>(P, g, stream);
    default: return launch_all<ACT, kDtBF16>(P, g, stream);
  }
}

// latent call: P1, then the cache store (lat_dt < 0: fp32 sums without l)
template <int ACT, int SC>
hipError_t launch_latent_typed(const PrefillParams& P, int lat_dt, const PrefillGeom& g, hipStream_t stream) {
  hipError_t e = launch_p1_ms<ACT, SC>(P, g, stream);
  if (e != hipSuccess) return e;
  switch (lat_dt) {
    case -1:
      hipLaunchKernelGGL((prefill_latent_out<SC, kDtF32, false>), pair_grid(P), dim3(kThreads), 0, stream, P);
      break;
    case kDtF32: hipLaunchKernelGGL((prefill_latent_out<SC, kDtF32>), pair_grid(P), dim3(kThreads), 0, stream, P); break;
    case kDtF16: hipLaunchKernelGGL((prefill_latent_out<SC, kDtF16>), pair_grid(P), dim3(kThreads), 0, stream, P); break;
    default: hipLaunchKernelGGL((prefill_latent_out<SC, kDtBF16>), pair_grid(P), dim3(kThreads), 0, stream, P); break;
  }
  return hipGetLastError();
}
template <int ACT>
hipError_t launch_latent_act(const PrefillParams& P, int sc_dt, int lat_dt, const PrefillGeom& g,
                             hipStream_t stream) {
  switch (sc_dt) {
    case kDtF32: return launch_latent_typed<ACT, kDtF32>(P, lat_dt, g, stream);
    case kDtF16: return launch_latent_typed<ACT, kDtF16>(P, lat_dt, g, stream);
    default: return launch_latent_typed<ACT, kDtBF16>(P, lat_dt, g, stream);
  }
}

// from-latent call: the cache cut into w terms, then P2 (lat_dt < 0: an fp32
// array times l)
template <int ACT, int SC>
hipError_t launch_from_latent_typed(const PrefillParams& P, int lat_dt, const PrefillGeom& g, hipStream_t stream) {
  switch (lat_dt) {
    case -1:
      hipLaunchKernelGGL((prefill_latent_in<ACT, kDtF32, SC>), pair_grid(P), dim3(kThreads), 0, stream, P);
      break;
    case kDtF32: hipLaunchKernelGGL((prefill_latent_in<ACT, kDtF32>), pair_grid(P), dim3(kThreads), 0, stream, P); break;
    case kDtF16: hipLaunchKernelGGL((prefill_latent_in<ACT, kDtF16>), pair_grid(P), dim3(kThreads), 0, stream, P); break;
    default: hipLaunchKernelGGL((prefill_latent_in<ACT, kDtBF16>), pair_grid(P), dim3(kThreads), 0, stream, P); break;
  }
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_p2_any<ACT, SC>(P, g, stream);
}
template <int ACT>
hipError_t launch_from_latent_act(const PrefillParams& P, int sc_dt, int lat_dt, const PrefillGeom& g,
                                  hipStream_t stream) {
  switch (sc_dt) {
    case kDtF32: return launch_from_latent_typed<ACT, kDtF32>(P, lat_dt, g, stream);
    case kDtF16: return launch_from_latent_typed<ACT, kDtF16>(P, lat_dt, g, stream);
    default: return launch_from_latent_typed<ACT, kDtBF16>(P, lat_dt, g, stream);
  }
}

size_t align256(size_t b) { return (b + 255) / 256 * 256; }

int64_t packed_bytes(int64_t n_out, int64_t n_red) {
  const int64_t w = n_red & 31;
  return 4 * (n_red >> 5) * n_out + (w == 0 ? 0 : (w <= 16 ? 2 : 4)) * n_out;
}

// U-word block slots per wave and buffer of P2
int p2_wdp(const PrefillGeom& g, bool fast) {
  const int nkb4 = fast ? (g.nkb + 3) / 4 * 4 : g.nkb;
  return g.res ? 2 * nkb4 : (fast ? (g.kbc + 3) / 4 * 4 : g.kbc);
}

// LDS sizes and the P2 plan for the activation / scale dtypes: P2 holds all w
// fragments of its token tile when they fit, else chunks of kMaxKbc blocks,
// and runs about 256 workgroups per CU-round (two per CU when the LDS allows)
void plan_lds(PrefillGeom& g, int act, int sc, bool vw, bool fast) {
  const int G = sc == kDtF32 ? 3 : (sc == kDtF16 ? 2 : 1);
  g.smem1 = p1_lds(g.kb_per, G, act, g.ms, vw);
  const int nw = act == kDtF32 ? 3 : 2;
  // U-word slots: 16-byte loads fill 4 blocks at a time, so each path's run
  // of slots is a multiple of 4 (FAST)
  const int nkb4 = fast ? (g.nkb + 3) / 4 * 4 : g.nkb;
  const size_t res_bytes = p2_w_bytes(2 * g.nkb, nw) + p2_wd_bytes(2 * nkb4, 2);
  g.res = res_bytes <= kLdsBudget ? 1 : 0;
  g.kbc = g.nkb < kMaxKbc ? g.nkb : kMaxKbc;
  g.smem2 = g.res ? res_bytes : p2_w_bytes(g.kbc, nw) + p2_wd_bytes(p2_wdp(g, fast), 1);
  int og = 256 / g.n_tt2;
  if (og < 1) og = 1;
  if (og > g.n_un) og = g.n_un;
  // the fewest groups that give the same number of units per group
  const int upg = (g.n_un + og - 1) / og;
  g.n_og = (g.n_un + upg - 1) / upg;
}

}  // namespace

PrefillGeom prefill_geometry(int T, int d_in, int d_out, int r) {
  PrefillGeom g{};
  const int tt = T > 0 ? T : 1;
  const int rr = r > 0 ? r : 1;
  g.nkb = nblocks32(rr);
  g.ns16 = (rr + 15) / 16;
  // P1: each wave takes ms interleaved subtiles of its path (2 waves a path);
  // about 256 workgroups, splits of d_in of at least kMinSteps steps (when
  // d_in has them) and at most kMaxKbPer.  With few token tiles, fewer
  // subtiles per wave (more latent tiles, x re-read per tile) rather than
  // more splits: the largest ms that still gives kMinWg1 workgroups.
  g.n_tt = (tt + kTok1 - 1) / kTok1;
  const int nbt = nblocks32(d_in > 0 ? d_in : 1);
  const int ks_min = (nbt + kMaxKbPer - 1) / kMaxKbPer;
  // the plan for at most `ms` subtiles per wave; returns its workgroup count
  auto plan = [&](int ms) {
    g.n_lt = (g.ns16 + 2 * ms - 1) / (2 * ms);
    g.ms = (g.ns16 + 2 * g.n_lt - 1) / (2 * g.n_lt);
    const int tiles = g.n_tt * g.n_lt;
    int ks = (256 + tiles - 1) / tiles;
    if (ks > nbt / kMinSteps) ks = nbt / kMinSteps;
    if (ks < ks_min) ks = ks_min;
    if (ks < 1) ks = 1;
    g.kb_per = (nbt + ks - 1) / ks;
    g.ks = (nbt + g.kb_per - 1) / g.kb_per;
    return tiles * g.ks;
  };
  int ms = kMaxMs;
  while (plan(ms) < kMinWg1 && ms > 1) --ms;
  g.ns16p = g.n_lt * 2 * g.ms;
  g.n_un = (d_out > 0 ? d_out + kUnit - 1 : kUnit) / kUnit;
  g.n_tt2 = (tt + kTok2 - 1) / kTok2;
  plan_lds(g, kDtF32, kDtF32, false, false);
  // workspace (nothing beyond the control block when there is nothing to compute)
  const bool work = T > 0 && d_in > 0 && r > 0;
  g.pbuf_off = kCtrlBytes;
  g.pbuf_floats = work ? static_cast<size_t>(g.ks) * g.n_tt * 2 * g.ns16p * kPart : 0;
  g.wterm_off = g.pbuf_off + align256(4 * g.pbuf_floats);
  g.wterm_bytes = work ? static_cast<size_t>(2) * 3 * g.nkb * T * 64 : 0;
  g.ws_bytes = g.wterm_off + align256(g.wterm_bytes);
  return g;
}

bool prefill_supports(int64_t T, int64_t d_in, int64_t d_out, int64_t r) {
  // 32-bit buffer offsets
  const int64_t lim = int64_t(1) << 31;
  const PrefillGeom g = prefill_geometry(static_cast<int>(T), static_cast<int>(d_in), static_cast<int>(d_out),
                                         static_cast<int>(r));
  return int64_t(kTok2) * d_out * 4 < lim && int64_t(kTok1) * d_in * 4 < lim && packed_bytes(d_out, r) < lim &&
         packed_bytes(r, d_in) < lim && static_cast<int64_t>(g.wterm_bytes) < lim;
}

namespace {

// The kernels' parameters for a.  The workspace holds the P1 partial sums at
// pbuf_off and the w terms at wterm_off of g.
PrefillParams prefill_params(const ForwardArgs& a, PrefillGeom& g) {
  const int64_t ex = a.act_dt == kDtF32 ? 4 : 2, es = a.sc_dt == kDtF32 ? 4 : 2;
  auto al = [](const void* q, int64_t n) { return reinterpret_cast<uintptr_t>(q) % n == 0; };
  // 16-byte V-word loads: whole 4-word groups per latent block row
  const bool vw = a.r % 4 == 0 && al(a.V[0], 16) && al(a.V[1], 16);
  // P2 fast path: whole 4-output groups, 16-byte aligned U words, aligned h and y
  const bool fast = a.d_out % 4 == 0 && al(a.U[0], 16) && al(a.U[1], 16) && al(a.h[0], 4 * es) &&
                    al(a.h[1], 4 * es) && al(a.y, 4 * ex);
  plan_lds(g, a.act_dt, a.sc_dt, vw, fast);
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
  P.ns16 = g.ns16;
  P.n_tt = g.n_tt;
  P.n_lt = g.n_lt;
  P.ks = g.ks;
  P.kb_per = g.kb_per;
  P.ns16p = g.ns16p;
  P.n_un = g.n_un;
  P.n_og = g.n_og;
  P.n_tt2 = g.n_tt2;
  P.res = g.res;
  P.kbc = g.kbc;
  // global-to-LDS x loads need 16-byte aligned rows of whole 16-byte chunks
  P.xdma = al(a.x, 16) && (a.d_in * ex) % 16 == 0;
  P.vw = vw;
  P.fast = fast;
  P.wdp = p2_wdp(g, fast);
  P.v_bytes = static_cast<uint32_t>(packed_bytes(a.r, a.d_in));
  P.u_bytes = static_cast<uint32_t>(packed_bytes(a.d_out, a.r));
  P.g_bytes = static_cast<uint32_t>(a.d_in * es);
  P.h_bytes = static_cast<uint32_t>(a.d_out * es);
  P.l_bytes = static_cast<uint32_t>(a.r * es);
  const int nw = a.act_dt == kDtF32 ? 3 : 2;
  P.wt_bytes = static_cast<uint32_t>(static_cast<int64_t>(2) * nw * g.nkb * a.T * 64);
  P.wd_off = static_cast<uint32_t>(p2_w_bytes(g.res ? 2 * g.nkb : g.kbc, nw));
  return P;
}

// d_in that gives the smallest stage-1 plan (the from-latent call has no stage 1)
constexpr int kNoStage1 = 32;

}  // namespace

hipError_t launch_prefill(const ForwardArgs& a, const PrefillGeom& g0, hipStream_t stream) {
  PrefillGeom g = g0;
  const PrefillParams P = prefill_params(a, g);
  switch (a.act_dt) {
    case kDtF32: return launch_act<kDtF32>(P, a.sc_dt, g, stream);
    case kDtF16: return launch_act<kDtF16>(P, a.sc_dt, g, stream);
    default: return launch_act<kDtBF16>(P, a.sc_dt, g, stream);
  }
}

// ---------------------------------------------------------------------------
// latent cache
// ---------------------------------------------------------------------------
bool latent_supports(int64_t T, int64_t d_in, int64_t r) { return prefill_supports(T, d_in, 0, r); }

bool from_latent_supports(int64_t T, int64_t d_out, int64_t r) {
  return prefill_supports(T, kNoStage1, d_out, r);
}

size_t latent_workspace_bytes(int T, int d_in, int r) {
  const PrefillGeom g = prefill_geometry(T, d_in, 0, r);
  return g.pbuf_off + align256(4 * g.pbuf_floats);
}

size_t from_latent_workspace_bytes(int T, int r) {
  const PrefillGeom g = prefill_geometry(T, kNoStage1, 0, r);
  return kCtrlBytes + align256(g.wterm_bytes);
}

hipError_t launch_latent(const ForwardArgs& a, int lat_dt, hipStream_t stream) {
  PrefillGeom g = prefill_geometry(a.T, a.d_in, 0, a.r);
  PrefillParams P = prefill_params(a, g);
  P.lat = a.y;
  switch (a.act_dt) {
    case kDtF32: return launch_latent_act<kDtF32>(P, a.sc_dt, lat_dt, g, stream);
    case kDtF16: return launch_latent_act<kDtF16>(P, a.sc_dt, lat_dt, g, stream);
    default: return launch_latent_act<kDtBF16>(P, a.sc_dt, lat_dt, g, stream);
  }
}

hipError_t launch_stage1_sums(const ForwardArgs& a, float* z, hipStream_t stream) {
  ForwardArgs b = a;
  b.y = z;
  return launch_latent(b, -1, stream);
}

hipError_t launch_stage1_sums2(const ForwardArgs& a0, float* z0, const ForwardArgs& a1, float* z1,
                               hipStream_t stream) {
  if (a0.act_dt != a1.act_dt || a0.sc_dt != a1.sc_dt || a0.T != a1.T || a0.r != a1.r) return hipErrorInvalidValue;
  PrefillGeom g0 = prefill_geometry(a0.T, a0.d_in, 0, a0.r), g1 = prefill_geometry(a1.T, a1.d_in, 0, a1.r);
  PrefillParams Q0 = prefill_params(a0, g0), Q1 = prefill_params(a1, g1);
  Q0.lat = z0;
  Q1.lat = z1;
  hipError_t e;
  auto p1 = [&](const PrefillParams& Q, const PrefillGeom& g) -> hipError_t {
    switch (a0.act_dt * 3 + a0.sc_dt) {
      case kDtF32 * 3 + kDtF32: return launch_p1_ms<kDtF32, kDtF32>(Q, g, stream);
      case kDtF32 * 3 + kDtF16: return launch_p1_ms<kDtF32, kDtF16>(Q, g, stream);
      case kDtF32 * 3 + kDtBF16: return launch_p1_ms<kDtF32, kDtBF16>(Q, g, stream);
      case kDtF16 * 3 + kDtF32: return launch_p1_ms<kDtF16, kDtF32>(Q, g, stream);
      case kDtF16 * 3 + kDtF16: return launch_p1_ms<kDtF16, kDtF16>(Q, g, stream);
      case kDtF16 * 3 + kDtBF16: return launch_p1_ms<kDtF16, kDtBF16>(Q, g, stream);
      case kDtBF16 * 3 + kDtF32: return launch_p1_ms<kDtBF16, kDtF32>(Q, g, stream);
      case kDtBF16 * 3 + kDtF16: return launch_p1_ms<kDtBF16, kDtF16>(Q, g, stream);
      default: return launch_p1_ms<kDtBF16, kDtBF16>(Q, g, stream);
    }
  };
  if ((e = p1(Q0, g0)) != hipSuccess) return e;
  if ((e = p1(Q1, g1)) != hipSuccess) return e;
  const int nb0 = static_cast<int>(pair_grid(Q0).x), nb1 = static_cast<int>(pair_grid(Q1).x);
  switch (a0.sc_dt) {
    case kDtF32: hipLaunchKernelGGL((prefill_sums2<kDtF32>), dim3(nb0 + nb1), dim3(kThreads), 0, stream, Q0, Q1, nb0); break;
    case kDtF16: hipLaunchKernelGGL((prefill_sums2<kDtF16>), dim3(nb0 + nb1), dim3(kThreads), 0, stream, Q0, Q1, nb0); break;
    default: hipLaunchKernelGGL((prefill_sums2<kDtBF16>), dim3(nb0 + nb1), dim3(kThreads), 0, stream, Q0, Q1, nb0); break;
  }
  return hipGetLastError();
}

hipError_t launch_stage2_scaled(const ForwardArgs& a, const float* w, hipStream_t stream) {
  return launch_from_latent(a, w, -1, stream);
}

hipError_t launch_from_latent(const ForwardArgs& a, const void* lat, int lat_dt, hipStream_t stream) {
  PrefillGeom g = prefill_geometry(a.T, kNoStage1, a.d_out, a.r);
  g.wterm_off = kCtrlBytes;  // no partial sums
  PrefillParams P = prefill_params(a, g);
  P.lat = const_cast<void*>(lat);
  switch (a.act_dt) {
    case kDtF32: return launch_from_latent_act<kDtF32>(P, a.sc_dt, lat_dt, g, stream);
    case kDtF16: return launch_from_latent_act<kDtF16>(P, a.sc_dt, lat_dt, g, stream);
    default: return launch_from_latent_act<kDtBF16>(P, a.sc_dt, lat_dt, g, stream);
  }
}

}  // namespace lb
