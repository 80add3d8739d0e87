// Latent cache entries for a few tokens in one launch (paragraph "KV Cache
// Compression": the scaled stage-1 latent of Proposition 1 cached per token,
// here for the one to four tokens of a decoding step).
//
//   w[t][p][k] = l_p[k] * sum_j s(V_p[j][k]) (g_p[j] x[t][j])
//
// A workgroup owns 16 latents of one path.  The products a[t][j] = g_p[j]
// x[t][j] of a chunk of inputs are formed once in LDS (fp32; exact for bf16
// and f16 operands; zero past d_in up to the block end); then each thread
// takes one latent and every sixteenth 32-input block of the chunk, reads the
// block's packed word (LB layout v1, role V: the words of consecutive latents
// are consecutive) and adds the 32 products with their signs flipped by the
// word's bits (pad bits are 0: +1 times a zero product).  The 16 lanes of a
// latent group read the same LDS address.  The sixteen block groups are added
// in a fixed order at the end, scaled by l and stored (rounded to nearest
// even for a 16-bit cache).
#include "device_common.h"
#include "lb_latent.h"

namespace lb {

namespace {

constexpr int kLThreads = 256;
constexpr int kLLat = 16;                     // latents per workgroup
constexpr int kLGroups = kLThreads / kLLat;   // block groups
constexpr int kLStage = 8192;                 // fp32 products staged in LDS (all tokens)

struct SmallParams {
  const void* x;
  const void* V[2];
  const void* g[2];
  const void* l[2];
  void* lat;  // [T][2][r]
  int T, d_in, r, n_lt;
};

template <int ACT, int SC, int LD, int TT>
__global__ void __launch_bounds__(kLThreads) latent_small(SmallParams P) {
  constexpr int CH = kLStage / TT;  // inputs per chunk, a multiple of 32
  __shared__ __attribute__((aligned(16))) float a[TT][CH];
  __shared__ float red[kLGroups][TT][kLLat];
  const int tid = threadIdx.x;
  const int lt = blockIdx.x % P.n_lt, p = blockIdx.x / P.n_lt;
  const int kk = tid % kLLat, jg = tid / kLLat;
  const int k = lt * kLLat + kk;
  const bool kok = k < P.r;
  const int d_in = P.d_in, r = P.r;
  const PackedView Vv{static_cast<const uint32_t*>(P.V[p]), r, d_in >> 5, d_in & 31};
  const void* g = P.g[p];
  float acc[TT];
#pragma unroll
  for (int t = 0; t < TT; ++t) acc[t] = 0.0f;
  constexpr int NWB = CH / 32 / kLGroups;  // blocks of a chunk per thread
  for (int c0 = 0; c0 < d_in; c0 += CH) {
    const int cn = d_in - c0 < CH ? d_in - c0 : CH;
    const int cn32 = (cn + 31) & ~31;
    const int nbc = cn32 >> 5;
    // the chunk's sign words first, so that their loads overlap the products'
    uint32_t wv[NWB];
#pragma unroll
    for (int q = 0; q < NWB; ++q) {
      const int bl = jg + q * kLGroups;
      wv[q] = kok && bl < nbc ? load_word(Vv, (c0 >> 5) + bl, k) : 0u;
    }
    __syncthreads();  // the previous chunk's readers are done
#pragma unroll 8
    for (int j = tid; j < cn32; j += kLThreads) {
      const bool jok = j < cn;
      const float gj = ld_or0<SC>(g, c0 + j, jok);
#pragma unroll
      for (int t = 0; t < TT; ++t) {
        const bool ok = jok && t < P.T;
        a[t][j] = gj * ld_or0<ACT>(P.x, static_cast<int64_t>(t) * d_in + c0 + j, ok);
      }
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < NWB; ++q) {
      const int bl = jg + q * kLGroups;
      if (bl >= nbc) break;
      const uint32_t word = wv[q];
#pragma unroll
      for (int i4 = 0; i4 < 8; ++i4) {
#pragma unroll
        for (int t = 0; t < TT; ++t) {
          const float4 v = *reinterpret_cast<const float4*>(&a[t][32 * bl + 4 * i4]);
          const float vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const uint32_t sgn = (word << (31 - (4 * i4 + e))) & 0x80000000u;
            acc[t] += __uint_as_float(__float_as_uint(vv[e]) ^ sgn);
          }
        }
      }
    }
  }
#pragma unroll
  for (int t = 0; t < TT; ++t) red[jg][t][kk] = acc[t];
  __syncthreads();
  if (jg == 0 && kok) {
    const float lk = ld<SC>(P.l[p], k);
#pragma unroll
    for (int t = 0; t < TT; ++t) {
      if (t >= P.T) break;
      float s = 0.0f;
#pragma unroll
      for (int q = 0; q < kLGroups; ++q) s += red[q][t][kk];
      st<LD>(P.lat, (static_cast<int64_t>(t) * 2 + p) * r + k, s * lk);
    }
  }
}

template <int ACT, int SC, int LD>
hipError_t launch_tt(const SmallParams& P, hipStream_t stream) {
  const dim3 grid(2 * P.n_lt), block(kLThreads);
  switch (P.T) {
    case 1: hipLaunchKernelGGL((latent_small<ACT, SC, LD, 1>), grid, block, 0, stream, P); break;
    case 2: hipLaunchKernelGGL((latent_small<ACT, SC, LD, 2>), grid, block, 0, stream, P); break;
    default: hipLaunchKernelGGL((latent_small<ACT, SC, LD, 4>), grid, block, 0, stream, P); break;
  }
  return hipGetLastError();
}

template <int ACT, int SC>
hipError_t launch_ld(const SmallParams& P, int lat_dt, hipStream_t stream) {
  switch (lat_dt) {
    case kDtF32: return launch_tt<ACT, SC, kDtF32>(P, stream);
    case kDtF16: return launch_tt<ACT, SC, kDtF16>(P, stream);
    default: return launch_tt<ACT, SC, kDtBF16>(P, stream);
  }
}

template <int ACT>
hipError_t launch_sc(const SmallParams& P, int sc_dt, int lat_dt, hipStream_t stream) {
  switch (sc_dt) {
    case kDtF32: return launch_ld<ACT, kDtF32>(P, lat_dt, stream);
    case kDtF16: return launch_ld<ACT, kDtF16>(P, lat_dt, stream);
    default: return launch_ld<ACT, kDtBF16>(P, lat_dt, stream);
  }
}

}  // namespace

bool latent_small_supports(int64_t T, int64_t d_in, int64_t r) {
  return T >= 1 && T <= kLatentSmallMaxT && d_in >= 1 && r >= 1 && (r + kLLat - 1) / kLLat <= 65535;
}

hipError_t launch_latent_small(const ForwardArgs& a, int lat_dt, hipStream_t stream) {
  SmallParams P{};
  P.x = a.x;
  for (int p = 0; p < 2; ++p) {
    P.V[p] = a.V[p];
    P.g[p] = a.g[p];
    P.l[p] = a.l[p];
  }
  P.lat = a.y;
  P.T = a.T;
  P.d_in = a.d_in;
  P.r = a.r;
  P.n_lt = (a.r + kLLat - 1) / kLLat;
  switch (a.act_dt) {
    case kDtF32: return launch_sc<kDtF32>(P, a.sc_dt, lat_dt, stream);
    case kDtF16: return launch_sc<kDtF16>(P, a.sc_dt, lat_dt, stream);
    default: return launch_sc<kDtBF16>(P, a.sc_dt, lat_dt, stream);
  }
}

}  // namespace lb
