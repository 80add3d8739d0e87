// Backward of one LittleBit linear for quantization-aware training (Sec. 4
// "Training Details": QAT of the latent factors and scales, with SmoothSign,
// Appendix "SmoothSign versus Straight-Through Estimator": the sign in the
// forward, the derivative of tanh(kappa u), kappa = 100, in the backward).
//
// The chain rule through Proposition 1 (Eq. proposition1), per path p, with
// a = g (.) x, z = a V_s, w = l (.) z, u = w U_s^T and an upstream gradient dy:
//   dw   = (h (.) dy) U_s          binary contraction over outputs   (prefill stage 1 on dy,
//                                                                      U_s packed with role V)
//   dz   = l (.) dw
//   dx   = sum_p g_p (.) (dz_p V_s^T)  binary contraction over latents (prefill stage 2 from dz,
//                                                                      V_s packed with role U)
//   C_U  = dy^T w                  dense, over tokens:  dU = h (.) C_U (.) slope(U_lat),
//                                                       dh = rowsum(U_s (.) C_U)
//   C_V  = x^T dz                  dense, over tokens:  dV = g (.) C_V (.) slope(V_lat),
//                                                       dg = rowsum(V_s (.) C_V)
//   dl   = sum_t dw (.) z           (partial sums in the B-term pass of the V side, added by its epilogue)
// with slope(u) = kappa sech^2(kappa u).  z (of x) and dw (of dy) are kept in
// fp32 [T][2][r] in the workspace.
//
// The two token contractions run on the matrix cores (tgemm): a workgroup of
// 4 waves owns 128 rows (outputs or inputs; two 16-row blocks per wave, which
// share each B fragment) and up to 128 latents of one path
// and a run of 32-token steps; each step stages the tile of A (dy or x, cut
// into its exact bf16 terms) and of B (w or dz: fp32, cut into three exact
// bf16 terms once by a pre-pass, bterms, which writes them with the tokens of
// a step contiguous) in LDS with tokens contiguous, so that both operands read
// their 8 reduction slots as one 16-byte LDS load.  Every product is exact and the
// matrix cores accumulate in fp32; token splits are added in ascending order
// by the epilogue.
#include "device_common.h"
#include "lb_backward.h"

namespace lb {

namespace {

constexpr int kGThreads = 256;  // 4 waves
constexpr int kGRB = 2;         // 16-row blocks per wave
constexpr int kGM = 64 * kGRB;  // rows per workgroup
constexpr int kGTok = 32;       // tokens per step
constexpr int kGMaxNk = 8;      // 16-latent subtiles per workgroup
constexpr int kRow = 40;        // LDS row stride in bf16 (32 tokens + 8 pad)
constexpr int kGWantWg = 512;   // workgroups aimed at by the token splits
constexpr int kGMinSteps = 2;   // fewest steps per token split

struct GemmParams {
  const void* A;        // [T][M] act dtype
  const uint16_t* Bt;   // [steps][2][3][kpad][32]: bf16 terms of l (.) B, tokens contiguous
  float* part;          // [ks][2][M][r]
  int T, M, r, kpad;
  int n_mt, n_kt, ks, steps_per;
};

struct GemmGeom {
  int nk, n_mt, n_kt, ks, steps_per, kpad;
  size_t part_floats;
};

GemmGeom gemm_geom(int T, int M, int r) {
  GemmGeom g{};
  // empty sizes plan as size 1 (their calls launch nothing)
  if (M < 1) M = 1;
  if (r < 1) r = 1;
  const int ns16 = (r + 15) / 16;
  g.nk = ns16 < kGMaxNk ? ns16 : kGMaxNk;
  g.n_kt = (ns16 + g.nk - 1) / g.nk;
  g.n_mt = (M + kGM - 1) / kGM;
  const int steps = T > kGTok ? (T + kGTok - 1) / kGTok : 1;
  const int tiles = g.n_mt * g.n_kt * 2;
  int ks = (kGWantWg + tiles - 1) / tiles;
  const int ks_max = steps / kGMinSteps > 1 ? steps / kGMinSteps : 1;
  if (ks > ks_max) ks = ks_max;
  if (ks < 1) ks = 1;
  g.steps_per = (steps + ks - 1) / ks;
  g.ks = (steps + g.steps_per - 1) / g.steps_per;
  g.part_floats = static_cast<size_t>(g.ks) * 2 * r * M;
  g.kpad = g.n_kt * 16 * g.nk;
  return g;
}

// partial sums of dl: one per 8-token group
int dl_parts(int T) { return 4 * (T > kGTok ? (T + kGTok - 1) / kGTok : 1); }

// bytes of the B terms [steps][2][3][kpad][32] bf16
size_t bterm_bytes(int T, int r) {
  const GemmGeom g = gemm_geom(T, 1, r);
  const int steps = T > kGTok ? (T + kGTok - 1) / kGTok : 1;
  return static_cast<size_t>(steps) * 2 * 3 * g.kpad * kGTok * 2;
}

__device__ __forceinline__ float load_scale(const void* p, int i, int dt) { return load_as_f32(p, i, dt); }

// B terms: one thread per (step, path, latent, 8-token group) cuts
// l[k] B[t][p][k] (fp32 product) into its three exact bf16 terms and writes
// them with the 32 tokens of a step contiguous (zero past T and past r)
// With zz (the V side, B = dw): also the partial sums of dl over the thread's
// 8 tokens, dlp[step][oct][p r + k] = sum_s dw z
// Both sides in one launch: the first nb1 workgroups take job 0 (U side:
// B = z), the rest job 1 (V side: B = dw, with zz = z and the dl partials).
struct BtermJob {
  const float* B;
  uint16_t* Bt;
  const float* zz;
  float* dlp;
};
__global__ void __launch_bounds__(256) bterms(BtermJob j0, BtermJob j1, int nb1, const void* l0, const void* l1,
                                              int sc_dt, int T, int r, int kpad) {
  const bool second = static_cast<int>(blockIdx.x) >= nb1;
  const BtermJob& J = second ? j1 : j0;
  const float* B = J.B;
  uint16_t* Bt = J.Bt;
  const float* zz = J.zz;
  float* dlp = J.dlp;
  const int64_t item = static_cast<int64_t>(second ? blockIdx.x - nb1 : blockIdx.x) * 256 + threadIdx.x;
  const int oct = static_cast<int>(item & 3);
  int64_t rest = item >> 2;
  const int k = static_cast<int>(rest % kpad);
  rest /= kpad;
  const int p = static_cast<int>(rest & 1);
  const int64_t step = rest >> 1;
  const int steps = T > kGTok ? (T + kGTok - 1) / kGTok : 1;
  if (step >= steps) return;
  const bool kok = k < r;
  const float lv = kok ? load_scale(p ? l1 : l0, k, sc_dt) : 0.0f;
  uint32_t t3[8][3];
  float dls = 0.0f;
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    const int64_t t = step * kGTok + 8 * oct + s;
    const bool ok = kok && t < T;
    const int64_t i = ok ? (t * 2 + p) * r + k : 0;
    const float v = B[i];
    split_exact<3>(ok ? v * lv : 0.0f, t3[s]);
    if (zz) dls += ok ? v * zz[i] : 0.0f;
  }
  if (zz && kok) dlp[(step * 4 + oct) * 2 * r + p * r + k] = dls;
#pragma unroll
  for (int f = 0; f < 3; ++f) {
    u32x4 d;
#pragma unroll
    for (int v = 0; v < 4; ++v) d[v] = t3[2 * v][f] | (t3[2 * v + 1][f] << 16);
    *reinterpret_cast<u32x4*>(Bt + (((step * 2 + p) * 3 + f) * kpad + k) * kGTok + 8 * oct) = d;
  }
}

template <int ADT, int NK>
__global__ void __launch_bounds__(kGThreads) tgemm(GemmParams P) {
  constexpr int E = nterms<ADT>();
  constexpr int KT = 16 * NK;
  constexpr int NBI = (3 * KT * 4 + kGThreads - 1) / kGThreads;  // 16-byte B pieces per thread
  __shared__ __attribute__((aligned(16))) uint16_t As[E][kGM][kRow];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[3][KT][kRow];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int bid = blockIdx.x;
  const int mt = bid % P.n_mt;
  bid /= P.n_mt;
  const int kt = bid % P.n_kt;
  bid /= P.n_kt;
  const int p = bid & 1, sp = bid >> 1;
  const int m0 = mt * kGM, k0 = kt * KT;
  const int T = P.T, M = P.M, r = P.r;
  const int steps = (T + kGTok - 1) / kGTok;
  const int st0 = sp * P.steps_per;
  int nst = steps - st0;
  if (nst > P.steps_per) nst = P.steps_per;

  // A loader: rows am + 64 i, tokens 8 aq .. 8 aq + 7 of a step
  const int am = tid & 63, aq = tid >> 6;
  // B loader pieces: 16 bytes (8 tokens) of term f of latent k0 + bk
  uint32_t ra[kGRB][8];
  u32x4 rb[NBI];
  auto load = [&](int st) {
    const int tb = (st0 + st) * kGTok;
#pragma unroll
    for (int i = 0; i < kGRB; ++i) {
      const bool a_ok = m0 + am + 64 * i < M;
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const int t = tb + 8 * aq + s;
        const bool ok = a_ok && t < T;
        const uint32_t u = ld_bits<ADT>(P.A, ok ? static_cast<int64_t>(t) * M + m0 + am + 64 * i : 0);
        ra[i][s] = ok ? u : 0u;
      }
    }
    const uint16_t* bsrc = P.Bt + ((static_cast<int64_t>(st0 + st) * 2 + p) * 3 * P.kpad + k0) * kGTok;
#pragma unroll
    for (int i = 0; i < NBI; ++i) {
      const int idx = tid + kGThreads * i;  // (f, bk, oct) with oct fastest
      if (idx < 3 * KT * 4) {
        const int f = idx / (KT * 4), rem = idx - f * KT * 4;
        rb[i] = *reinterpret_cast<const u32x4*>(bsrc + (static_cast<int64_t>(f) * P.kpad + (rem >> 2)) * kGTok +
                                                8 * (rem & 3));
      }
    }
  };
  auto store = [&]() {
#pragma unroll
    for (int i = 0; i < kGRB; ++i) {
      uint32_t at[8][E];
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        if constexpr (ADT == kDtBF16)
          at[s][0] = ra[i][s];
        else
          split_exact<E>(bits_to_f32<ADT>(ra[i][s]), at[s]);
      }
#pragma unroll
      for (int e = 0; e < E; ++e) {
        u32x4 d;
#pragma unroll
        for (int v = 0; v < 4; ++v) d[v] = at[2 * v][e] | (at[2 * v + 1][e] << 16);
        *reinterpret_cast<u32x4*>(&As[e][am + 64 * i][8 * aq]) = d;
      }
    }
#pragma unroll
    for (int i = 0; i < NBI; ++i) {
      const int idx = tid + kGThreads * i;
      if (idx < 3 * KT * 4) {
        const int f = idx / (KT * 4), rem = idx - f * KT * 4;
        *reinterpret_cast<u32x4*>(&Bs[f][rem >> 2][8 * (rem & 3)]) = rb[i];
      }
    }
  };

  floatx4 acc[kGRB][NK];
#pragma unroll
  for (int i = 0; i < kGRB; ++i)
#pragma unroll
    for (int j = 0; j < NK; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  const int fr = lane & 15, fq = lane >> 4;
  if (nst > 0) {
    load(0);
    store();
    __syncthreads();
    for (int st = 0; st < nst; ++st) {
      if (st + 1 < nst) load(st + 1);
      u32x4 a[kGRB][E];
#pragma unroll
      for (int i = 0; i < kGRB; ++i)
#pragma unroll
        for (int e = 0; e < E; ++e)
          a[i][e] = *reinterpret_cast<const u32x4*>(&As[e][16 * (wave + 4 * i) + fr][8 * fq]);
#pragma unroll
      for (int f = 0; f < 3; ++f) {
#pragma unroll
        for (int j = 0; j < NK; ++j) {
          const u32x4 b = *reinterpret_cast<const u32x4*>(&Bs[f][16 * j + fr][8 * fq]);
#pragma unroll
          for (int i = 0; i < kGRB; ++i)
#pragma unroll
            for (int e = 0; e < E; ++e) acc[i][j] = mfma(a[i][e], b, acc[i][j]);
        }
      }
      __syncthreads();
      if (st + 1 < nst) {
        store();
        __syncthreads();
      }
    }
  }
  // partial sums [m][k]: rows 16 (wave + 4 i) + 4 fq + e of latent 16 j + fr
  float* out = P.part + (static_cast<int64_t>(sp) * 2 + p) * r * static_cast<int64_t>(M);
#pragma unroll
  for (int j = 0; j < NK; ++j) {
    const int k = k0 + 16 * j + fr;
    if (k >= r) continue;
#pragma unroll
    for (int i = 0; i < kGRB; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int m = m0 + 16 * (wave + 4 * i) + 4 * fq + e;
        if (m < M) out[static_cast<int64_t>(m) * r + k] = acc[i][j][e];
      }
  }
}

struct EpiParams {
  const float* part;  // [ks][2][M][r]
  const float* lat[2];
  const void* s[2];   // row scales (h or g)
  float* dlat[2];
  float* drow[2];
  int M, r, ks, sc_dt;
  float kappa;
  // with dlp: the workgroups past the rows' also add dl's partial sums
  const float* dlp;
  int n_dl;  // partials per column
  float* dl[2];
};

// d/du tanh(kappa u) = kappa sech^2(kappa u) = 4 kappa e / (1 + e)^2 with
// e = exp(-2 |kappa u|): no cancellation for large |u|
__device__ __forceinline__ float smooth_slope(float kappa, float u) {
  const float e = expf(-2.0f * fabsf(kappa * u));
  const float d = 1.0f + e;
  return 4.0f * kappa * e / (d * d);
}

// one wave per (path, row), lanes over latents: sums the token splits in
// ascending order, writes the latent-factor gradient, and the row-scale
// gradient through a fixed butterfly over the wave
// dl[p][k] = sum of the partials of column c = p r + k, by one wave: lanes
// over the partials in a fixed order, then a fixed butterfly
__device__ void dl_column(const float* part, int n, int r, int c, int lane, float* dl0, float* dl1) {
  float s = 0.0f;
  for (int i = lane; i < n; i += 64) s += part[static_cast<int64_t>(i) * 2 * r + c];
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o, 64);
  if (lane == 0) {
    if (c < r)
      dl0[c] = s;
    else
      dl1[c - r] = s;
  }
}

__global__ void __launch_bounds__(256) tgemm_epilogue(EpiParams P) {
  const int lane = threadIdx.x & 63;
  const int nrow_wg = (2 * P.M + 3) / 4;
  if (static_cast<int>(blockIdx.x) >= nrow_wg) {  // dl: one wave per column
    const int c = (blockIdx.x - nrow_wg) * 4 + (threadIdx.x >> 6);
    if (c < 2 * P.r) dl_column(P.dlp, P.n_dl, P.r, c, lane, P.dl[0], P.dl[1]);
    return;
  }
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= 2 * P.M) return;  // whole waves leave together
  const int p = row >= P.M ? 1 : 0;
  const int m = row - p * P.M;
  const int M = P.M, r = P.r;
  const float sc = load_scale(P.s[p], m, P.sc_dt);
  const float* lat = P.lat[p] + static_cast<int64_t>(m) * r;
  float* dlat = P.dlat[p] + static_cast<int64_t>(m) * r;
  const float* src = P.part + (static_cast<int64_t>(p) * M + m) * r;
  const int64_t sstride = static_cast<int64_t>(2) * M * r;
  float acc = 0.0f;
  for (int k = lane; k < r; k += 64) {
    float c = 0.0f;
    for (int s = 0; s < P.ks; ++s) c += src[s * sstride + k];
    const float u = lat[k];
    acc += u < 0.0f ? -c : c;
    dlat[k] = sc * c * smooth_slope(P.kappa, u);
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) acc += __shfl_xor(acc, o, 64);
  if (lane == 0) P.drow[p][m] = acc;
}

template <int ADT>
hipError_t launch_tgemm_nk(const GemmParams& P, int nk, hipStream_t stream) {
  const dim3 grid(P.n_mt * P.n_kt * 2 * P.ks), block(kGThreads);
  switch (nk) {
    case 1: hipLaunchKernelGGL((tgemm<ADT, 1>), grid, block, 0, stream, P); break;
    case 2: hipLaunchKernelGGL((tgemm<ADT, 2>), grid, block, 0, stream, P); break;
    case 3: hipLaunchKernelGGL((tgemm<ADT, 3>), grid, block, 0, stream, P); break;
    case 4: hipLaunchKernelGGL((tgemm<ADT, 4>), grid, block, 0, stream, P); break;
    case 5: hipLaunchKernelGGL((tgemm<ADT, 5>), grid, block, 0, stream, P); break;
    case 6: hipLaunchKernelGGL((tgemm<ADT, 6>), grid, block, 0, stream, P); break;
    case 7: hipLaunchKernelGGL((tgemm<ADT, 7>), grid, block, 0, stream, P); break;
    default: hipLaunchKernelGGL((tgemm<ADT, kGMaxNk>), grid, block, 0, stream, P); break;
  }
  return hipGetLastError();
}

// the B terms of both sides (z for U, dw for V) and dl's partial sums
hipError_t run_bterms(const BackwardArgs& b, const float* z, const float* dw, uint16_t* bt_u, uint16_t* bt_v,
                      float* dlp, hipStream_t stream) {
  const GemmGeom g = gemm_geom(b.T, 1, b.r);
  const int steps = b.T > kGTok ? (b.T + kGTok - 1) / kGTok : 1;
  const int64_t items = static_cast<int64_t>(steps) * 2 * g.kpad * 4;
  const int nb1 = static_cast<int>((items + 255) / 256);
  const BtermJob ju{z, bt_u, nullptr, nullptr}, jv{dw, bt_v, z, dlp};
  hipLaunchKernelGGL(bterms, dim3(2 * nb1), dim3(256), 0, stream, ju, jv, nb1, b.l[0], b.l[1], b.sc_dt, b.T, b.r,
                     g.kpad);
  return hipGetLastError();
}

// C = A^T Bt (the terms of l (.) B) over tokens, then the epilogue into dlat / drow
hipError_t run_token_gemm(const BackwardArgs& b, const void* A, int M, const uint16_t* Bt, float* part,
                          const float* const* lat, const void* const* s, float* const* dlat, float* const* drow,
                          float* dlp, bool with_dl, hipStream_t stream) {
  const GemmGeom g = gemm_geom(b.T, M, b.r);
  hipError_t e;
  GemmParams P{};
  P.A = A;
  P.Bt = Bt;
  P.part = part;
  P.T = b.T;
  P.M = M;
  P.r = b.r;
  P.kpad = g.kpad;
  P.n_mt = g.n_mt;
  P.n_kt = g.n_kt;
  P.ks = g.ks;
  P.steps_per = g.steps_per;
  switch (b.act_dt) {
    case kDtF32: e = launch_tgemm_nk<kDtF32>(P, g.nk, stream); break;
    case kDtF16: e = launch_tgemm_nk<kDtF16>(P, g.nk, stream); break;
    default: e = launch_tgemm_nk<kDtBF16>(P, g.nk, stream); break;
  }
  if (e != hipSuccess) return e;
  EpiParams Q{};
  Q.part = part;
  for (int p = 0; p < 2; ++p) {
    Q.lat[p] = lat[p];
    Q.s[p] = s[p];
    Q.dlat[p] = dlat[p];
    Q.drow[p] = drow[p];
  }
  Q.M = M;
  Q.r = b.r;
  Q.ks = g.ks;
  Q.sc_dt = b.sc_dt;
  Q.kappa = b.kappa;
  // the V side's epilogue also adds dl's partial sums (formed by its B-term
  // pass), in workgroups of their own after the rows'
  const int n_dl_wg = with_dl ? (2 * b.r + 3) / 4 : 0;
  if (with_dl) {
    Q.dlp = dlp;
    Q.n_dl = dl_parts(b.T);
    Q.dl[0] = b.dl[0];
    Q.dl[1] = b.dl[1];
  }
  hipLaunchKernelGGL(tgemm_epilogue, dim3((2 * M + 3) / 4 + n_dl_wg), dim3(256), 0, stream, Q);
  return hipGetLastError();
}

size_t align256(size_t n) { return (n + 255) / 256 * 256; }

struct BackwardLayout {
  size_t z_off, dw_off, stage_off, stage2_off, part_off, bt_off, bt2_off, dl_off, total;
};

BackwardLayout backward_layout(int T, int d_in, int d_out, int r) {
  BackwardLayout L{};
  const size_t lat = align256(static_cast<size_t>(T) * 2 * r * 4);
  // stage areas: x's stage 1 then dx's stage 2 in the first, dy's stage 1 in
  // the second (both stage-1 runs' partials are alive at once)
  size_t stage = latent_workspace_bytes(T, d_in, r);
  const size_t s2 = latent_workspace_bytes(T, d_out, r);
  const size_t s3 = from_latent_workspace_bytes(T, r);
  if (s3 > stage) stage = s3;
  const GemmGeom gu = gemm_geom(T, d_out, r), gv = gemm_geom(T, d_in, r);
  const size_t part = align256(4 * (gu.part_floats > gv.part_floats ? gu.part_floats : gv.part_floats));
  L.z_off = kCtrlBytes;
  L.dw_off = L.z_off + lat;
  L.stage_off = L.dw_off + lat;
  L.stage2_off = L.stage_off + align256(stage);
  L.part_off = L.stage2_off + align256(s2);
  L.bt_off = L.part_off + part;
  L.bt2_off = L.bt_off + align256(bterm_bytes(T, r));
  L.dl_off = L.bt2_off + align256(bterm_bytes(T, r));
  L.total = L.dl_off + align256(static_cast<size_t>(dl_parts(T)) * 2 * r * 4);
  return L;
}

}  // namespace

bool backward_supports(int64_t T, int64_t d_in, int64_t d_out, int64_t r) {
  const int64_t lim = int64_t(1) << 31;
  if (!latent_supports(T, d_in, r) || !latent_supports(T, d_out, r) || !from_latent_supports(T, d_in, r))
    return false;
  const int64_t m = d_in > d_out ? d_in : d_out;
  const int64_t steps = (T + kGTok - 1) / kGTok;
  // token-split partial sums, [T][2][r] arrays and the row offsets of the token tiles
  return steps * 2 * r * m < lim && 2 * T * r < lim && (T + kGTok) * m < lim;
}

size_t backward_workspace_bytes(int T, int d_in, int d_out, int r) { return backward_layout(T, d_in, d_out, r).total; }

hipError_t launch_backward(const BackwardArgs& b, hipStream_t stream) {
  const BackwardLayout L = backward_layout(b.T, b.d_in, b.d_out, b.r);
  char* ws = static_cast<char*>(b.ws);
  float* z = reinterpret_cast<float*>(ws + L.z_off);
  float* dw = reinterpret_cast<float*>(ws + L.dw_off);
  float* part = reinterpret_cast<float*>(ws + L.part_off);
  float* dlp = reinterpret_cast<float*>(ws + L.dl_off);
  uint16_t* bt = reinterpret_cast<uint16_t*>(ws + L.bt_off);
  uint16_t* bt2 = reinterpret_cast<uint16_t*>(ws + L.bt2_off);
  void* stage = ws + L.stage_off;
  const size_t stage_bytes = L.stage2_off - L.stage_off;
  hipError_t e;
  // z of x (stage 1 through V and g) and dw of dy (stage 1 through U, role V
  // packing, and h): two stage-1 launches, one launch for both split sums
  {
    ForwardArgs ax{}, ay{};
    ax.x = b.x;
    ax.act_dt = b.act_dt;
    ax.T = b.T;
    ax.d_in = b.d_in;
    ax.r = b.r;
    for (int p = 0; p < 2; ++p) ax.V[p] = b.V[p], ax.g[p] = b.g[p], ax.l[p] = b.l[p];
    ax.sc_dt = b.sc_dt;
    ax.ws = stage;
    ax.ws_bytes = stage_bytes;
    ay = ax;
    ay.x = b.dy;
    ay.d_in = b.d_out;
    for (int p = 0; p < 2; ++p) ay.V[p] = b.Ut[p], ay.g[p] = b.h[p];
    ay.ws = ws + L.stage2_off;
    ay.ws_bytes = L.part_off - L.stage2_off;
    if ((e = launch_stage1_sums2(ax, z, ay, dw, stream)) != hipSuccess) return e;
  }
  // dx from dz = l (.) dw: stage 2 through V (role U packing) and g
  if (b.dx) {
    ForwardArgs a{};
    a.act_dt = b.act_dt;
    a.T = b.T;
    a.d_out = b.d_in;
    a.r = b.r;
    for (int p = 0; p < 2; ++p) a.U[p] = b.Vt[p], a.h[p] = b.g[p], a.l[p] = b.l[p];
    a.sc_dt = b.sc_dt;
    a.y = b.dx;
    a.ws = stage;
    a.ws_bytes = stage_bytes;
    if ((e = launch_stage2_scaled(a, dw, stream)) != hipSuccess) return e;
  }
  // dU, dh from C_U = dy^T (l (.) z); dV, dg from C_V = x^T (l (.) dw)
  // B terms of both sides in one launch (the V side's pass also forms the
  // partial sums of dl = sum_t dw (.) z, which its epilogue adds)
  if ((e = run_bterms(b, z, dw, bt, bt2, dlp, stream)) != hipSuccess) return e;
  if ((e = run_token_gemm(b, b.dy, b.d_out, bt, part, b.U_lat, b.h, b.dU, b.dh, nullptr, false, stream)) !=
      hipSuccess)
    return e;
  return run_token_gemm(b, b.x, b.d_in, bt2, part, b.V_lat, b.g, b.dV, b.dg, dlp, true, stream);
}

}  // namespace lb
