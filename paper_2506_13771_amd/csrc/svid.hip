// Dual-SVID conversion of a dense weight into the two LittleBit paths
// (Sec. 3.2 "Dual-SVID Initialization", Eqs. sign_init_concise,
// scale_init_rank1_concise, latent_scale_init_concise_0; the residual path from
// the primary path's error, Sec. 3.3 "Residual Compensation"), on the GPU in
// fp64.
//
// Per path, for a weight W [m x n] and rank r:
//   1. the top-r singular triplets of W by block subspace iteration: a block of
//      b = min(r + oversample, m, n) vectors, alternately multiplied by W and
//      W^T and orthonormalised each time, then a Rayleigh-Ritz step on the
//      final block (eigenvectors of Z^T Z with Z = W^T Q);
//   2. each singular pair signed so that the left vector's entry of largest
//      magnitude is positive (first such index on a tie), U' = U_r sqrt(S),
//      V' = V_r sqrt(S);
//   3. the best rank-1 approximations |U'| ~ h l_u^T and |V'| ~ g l_v^T, the
//      top singular value split evenly and signed so that the left factor sums
//      to >= 0; l = l_u (.) l_v;
//   4. for the primary path, W_res = W - diag(h) sign(U') diag(l) sign(V')^T diag(g),
//      the weight the residual path starts from.
// The contractions (W and W^T times a block, Gram matrices, basis changes, the
// effective weight) run on the fp64 matrix cores; the small symmetric
// eigenproblems (b x b and r x r) run as a parallel cyclic Jacobi method on one
// workgroup.  Every block, the final one included, is orthonormalised by
// Cholesky of its Gram matrix (CholQR, pivots below 1e-13 of the largest
// dropped), so a rank-deficient block gives zero columns, which the
// Rayleigh-Ritz step carries as zero eigenvalues.  Sums are in a fixed order
// (split-K partial sums added in slab order), so a call is deterministic.
#include <algorithm>
#include <cmath>

#include "lb_internal.h"

namespace lb {
namespace {

typedef double d4 __attribute__((ext_vector_type(4)));

constexpr int kDtF64 = 100;  // operand code of the internal fp64 arrays
constexpr int kGT = 64;      // GEMM output tile (rows and columns)
constexpr int kGK = 32;      // GEMM K per LDS stage
constexpr int kEigThreads = 1024;
constexpr int kCholThreads = 1024;  // CholQR: one workgroup (fewer threads were slower at b = 120)
constexpr int kMaxBlock = 1024;     // largest eigenproblem: one workgroup, one pair per thread
constexpr int kEigLdsMax = 128;     // b <= 128: the matrix stays in LDS during the sweeps
constexpr int kPackMax = 192;       // b <= 192: one triangle of it stays in LDS (b (b + 1) / 2 doubles)
constexpr int kEigMaxSweeps = 80;
constexpr int kApplyCols = 8;       // rotation replay: columns of the accumulated rotations per workgroup
constexpr int kApplyThreads = 256;
constexpr int kRotBatch = 16;       // rotation replay: steps whose coefficients are staged in LDS at once

__device__ __forceinline__ double load_op(const void* p, int64_t idx, int dt) {
  if (dt == kDtF64) return static_cast<const double*>(p)[idx];
  return static_cast<double>(load_as_f32(p, idx, dt));
}
// the same with the dtype fixed at compile time
template <int DT>
__device__ __forceinline__ double load_t(const void* p, int64_t idx) {
  if constexpr (DT == kDtF64)
    return static_cast<const double*>(p)[idx];
  else
    return static_cast<double>(load_as_f32(p, idx, DT));
}

enum { kEpiStore = 0, kEpiResid = 1 };

struct GemmArgs {
  const void* A;  // op(A)(i, k) = A[i * sai + k * sak]
  int a_dt, a_abs;
  int64_t sai, sak;
  const void* B;  // B(k, j) = B[k * sbk + j * sbj]
  int b_dt, b_abs;
  int64_t sbk, sbj;
  double* C;      // C[i * ldc + j]; with ksplit > 1 the partial slab z at C + z * pstride
  int64_t ldc, pstride;
  int M, N, K, kchunk, ksplit;
  int epi;        // kEpiResid: C = W(i, j) - h[i] g[j] acc
  const void* W;
  int w_dt;
  int64_t ldw;
  const double* h;
  const double* g;
};

__device__ __forceinline__ void gemm_store(const GemmArgs& g, int i, int j, double acc) {
  if (g.epi == kEpiResid) {
    const double w = load_op(g.W, static_cast<int64_t>(i) * g.ldw + j, g.w_dt);
    g.C[static_cast<int64_t>(i) * g.ldc + j] = w - g.h[i] * g.g[j] * acc;
  } else {
    g.C[static_cast<int64_t>(i) * g.ldc + j] = acc;
  }
}

// C = op(A) [M x K] * B [K x N] on the fp64 matrix cores (16x16x4 per
// instruction).  A 64 x 64 output tile per workgroup of four waves (32 x 32
// each), K staged through LDS 16 at a time; blockIdx.z takes K range
// [z * kchunk, (z + 1) * kchunk) and, when ksplit > 1, writes its own slab.
// AK: A's k stride is 1 (else its i stride is); BJ: B's j stride is 1 (else
// its k stride is) -- the tile loads walk the contiguous index.
// (ADT: A's dtype; B is always fp64)
template <bool AK, bool BJ, int ADT>
__global__ __launch_bounds__(256) void gemm64_kernel(GemmArgs g) {
  __shared__ double As[kGK][kGT + 1];
  __shared__ double Bs[kGK][kGT + 1];
  constexpr int kPer = kGT * kGK / 256;  // elements of each operand a thread stages
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int i0 = blockIdx.x * kGT, j0 = blockIdx.y * kGT;
  const int kz0 = blockIdx.z * g.kchunk;
  const int kz1 = min(g.K, kz0 + g.kchunk);
  const int wi = (wv >> 1) * 32, wj = (wv & 1) * 32;
  d4 acc[2][2];
  for (int a = 0; a < 2; ++a)
    for (int b = 0; b < 2; ++b) acc[a][b] = d4{0.0, 0.0, 0.0, 0.0};
  // the stage at k0 into registers: element e = tid + 256 u of each operand
  // tile, the source's contiguous index walking fastest; with 256 threads,
  // 64-wide tiles and 32-deep stages, element u of a thread sits at a fixed
  // offset plus u times a uniform stride (rows 8 u or k 4 u further)
  static_assert(kGT == 64 && kGK == 32, "the staging map assumes 64 x 32 tiles and 256 threads");
  const int a_i = AK ? (tid >> 5) : (tid & 63), a_k = AK ? (tid & 31) : (tid >> 6);
  const int a_di = AK ? 8 : 0, a_dk = AK ? 0 : 4;
  const int b_j = BJ ? (tid & 63) : (tid >> 5), b_k = BJ ? (tid >> 6) : (tid & 31);
  const int b_dj = BJ ? 0 : 8, b_dk = BJ ? 4 : 0;
  const int64_t a_step = static_cast<int64_t>(a_di) * g.sai + static_cast<int64_t>(a_dk) * g.sak;
  const int64_t b_step = static_cast<int64_t>(b_dk) * g.sbk + static_cast<int64_t>(b_dj) * g.sbj;
  double ra[kPer], rb[kPer];
  auto load_stage = [&](int k0) {
    const int64_t a0 = static_cast<int64_t>(i0 + a_i) * g.sai + static_cast<int64_t>(k0 + a_k) * g.sak;
    const int64_t b0 = static_cast<int64_t>(k0 + b_k) * g.sbk + static_cast<int64_t>(j0 + b_j) * g.sbj;
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      // out-of-range elements read element 0 and are replaced by 0
      const bool oka = i0 + a_i + a_di * u < g.M && k0 + a_k + a_dk * u < kz1;
      double va = load_t<ADT>(g.A, oka ? a0 + u * a_step : 0);
      if (g.a_abs) va = fabs(va);
      ra[u] = oka ? va : 0.0;
      const bool okb = j0 + b_j + b_dj * u < g.N && k0 + b_k + b_dk * u < kz1;
      double vb = load_t<kDtF64>(g.B, okb ? b0 + u * b_step : 0);
      if (g.b_abs) vb = fabs(vb);
      rb[u] = okb ? vb : 0.0;
    }
  };
  auto store_stage = [&]() {
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      As[a_k + a_dk * u][a_i + a_di * u] = ra[u];
      Bs[b_k + b_dk * u][b_j + b_dj * u] = rb[u];
    }
  };
  load_stage(kz0);
  for (int k0 = kz0; k0 < kz1; k0 += kGK) {
    store_stage();
    __syncthreads();
    // the next stage's loads are in flight while this stage's products run
    if (k0 + kGK < kz1) load_stage(k0 + kGK);
#pragma unroll
    for (int kk = 0; kk < kGK; kk += 4) {
      double av[2], bv[2];
#pragma unroll
      for (int a = 0; a < 2; ++a) av[a] = As[kk + (lane >> 4)][wi + a * 16 + (lane & 15)];
#pragma unroll
      for (int b = 0; b < 2; ++b) bv[b] = Bs[kk + (lane >> 4)][wj + b * 16 + (lane & 15)];
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) acc[a][b] = __builtin_amdgcn_mfma_f64_16x16x4f64(av[a], bv[b], acc[a][b], 0, 0, 0);
    }
    __syncthreads();
  }
  // D register v of lane l holds row (l / 16) + 4 v, column l % 16 of the 16 x 16 block
  for (int a = 0; a < 2; ++a)
    for (int b = 0; b < 2; ++b)
      for (int v = 0; v < 4; ++v) {
        const int i = i0 + wi + a * 16 + (lane >> 4) + 4 * v;
        const int j = j0 + wj + b * 16 + (lane & 15);
        if (i >= g.M || j >= g.N) continue;
        if (g.ksplit > 1)
          g.C[blockIdx.z * g.pstride + static_cast<int64_t>(i) * g.ldc + j] = acc[a][b][v];
        else
          gemm_store(g, i, j, acc[a][b][v]);
      }
}

// Sum of the split-K slabs P [z][M][N] in slab order, then the epilogue into
// g.C.
__global__ __launch_bounds__(256) void gemm_reduce_kernel(GemmArgs g, const double* P) {
  const int64_t total = static_cast<int64_t>(g.M) * g.N;
  for (int64_t e = blockIdx.x * 256ll + threadIdx.x; e < total; e += static_cast<int64_t>(gridDim.x) * 256) {
    double s = 0.0;
    for (int z = 0; z < g.ksplit; ++z) s += P[z * total + e];
    gemm_store(g, static_cast<int>(e / g.N), static_cast<int>(e % g.N), s);
  }
}

// Partner of index k in step s of the round-robin (circle) ordering of n2
// (even) indices: every pair meets once in n2 - 1 steps, each step's pairs are
// disjoint.
__device__ __forceinline__ void rr_pair(int n2, int s, int k, int& p, int& q) {
  const int m = n2 - 1;  // 0 <= s < m, 0 <= k < n2 / 2: one subtraction reduces modulo m
  if (k == 0) {
    p = m;
    q = s;
  } else {
    p = s + k;
    if (p >= m) p -= m;
    q = s - k + m;
    if (q >= m) q -= m;
  }
  if (p > q) {
    const int t = p;
    p = q;
    q = t;
  }
}

// Eigen-decomposition of a symmetric b x b matrix A (row-major, overwritten)
// by the cyclic Jacobi method with the round-robin ordering: each step rotates
// b/2 disjoint pairs at once (A <- J^T A J, the accumulated J in Et, one
// eigenvector per row), until a sweep rotates nothing (|a_pq| <= 1e-15
// sqrt(|a_pp a_qq|), or below 1e-17 of the largest starting diagonal entry)
// or kEigMaxSweeps sweeps.  Eigenvalues descending (index order on ties) to
// lam; eigenvectors to the columns of E [b x b].  One workgroup; the matrix
// lives in LDS when b <= kEigLdsMax.
template <bool kLds>
__global__ __launch_bounds__(kEigThreads) void jacobi_eig_kernel(double* A, double* Et, double* E, double* lam,
                                                                  int b) {
  extern __shared__ double eig_smem[];
  __shared__ int pp[kMaxBlock / 2], pq[kMaxBlock / 2], pa[kMaxBlock / 2];
  __shared__ double pc[kMaxBlock / 2], ps[kMaxBlock / 2];
  __shared__ int rot;
  __shared__ double floor_abs;
  const int tid = threadIdx.x;
  const int n2 = b + (b & 1), np = n2 / 2;
  double* M = kLds ? eig_smem : A;
  if (kLds)
    for (int e = tid; e < b * b; e += kEigThreads) M[e] = A[e];
  for (int e = tid; e < b * b; e += kEigThreads) Et[e] = (e / b == e % b) ? 1.0 : 0.0;
  if (tid == 0) {
    double mx = 0.0;
    for (int i = 0; i < b; ++i) mx = fmax(mx, fabs(A[static_cast<int64_t>(i) * b + i]));
    floor_abs = 1e-17 * mx;
  }
  __syncthreads();
  for (int sweep = 0; sweep < kEigMaxSweeps; ++sweep) {
    if (tid == 0) rot = 0;
    __syncthreads();
    for (int s = 0; s < n2 - 1; ++s) {
      if (tid < np) {
        int p, q;
        rr_pair(n2, s, tid, p, q);
        double c = 1.0, sn = 0.0;
        bool act = false;
        if (q < b) {
          const double app = M[p * b + p], aqq = M[q * b + q], apq = M[p * b + q];
          if (apq != 0.0 && fabs(apq) > 1e-15 * sqrt(fabs(app * aqq)) && fabs(apq) > floor_abs) {
            const double zeta = (aqq - app) / (2.0 * apq);
            const double t = (zeta >= 0.0 ? 1.0 : -1.0) / (fabs(zeta) + sqrt(1.0 + zeta * zeta));
            c = 1.0 / sqrt(1.0 + t * t);
            sn = c * t;
            act = true;
          }
        }
        pp[tid] = p;
        pq[tid] = q;
        pa[tid] = act ? 1 : 0;
        pc[tid] = c;
        ps[tid] = sn;
        if (act) atomicAdd(&rot, 1);
      }
      __syncthreads();
      // A <- J^T A J one 2 x 2 block (rows of pair kr, columns of pair kc) at a
      // time: the blocks are disjoint, so one phase does the whole step; the
      // rows of the inactive pairs' and the dummy index's blocks are identity.
      for (int e = tid; e < np * np; e += kEigThreads) {
        const int kr = e / np, kc = e - kr * np;
        if (!pa[kr] && !pa[kc]) continue;
        const int p = pp[kr], q = pq[kr], u = pp[kc], v = pq[kc];
        const bool qv = q < b, vv = v < b;
        const double cr = pc[kr], sr = ps[kr], cc = pc[kc], sc = ps[kc];
        const double a00 = M[p * b + u], a01 = vv ? M[p * b + v] : 0.0;
        const double a10 = qv ? M[q * b + u] : 0.0, a11 = (qv && vv) ? M[q * b + v] : 0.0;
        const double b00 = cr * a00 - sr * a10, b01 = cr * a01 - sr * a11;
        const double b10 = sr * a00 + cr * a10, b11 = sr * a01 + cr * a11;
        M[p * b + u] = cc * b00 - sc * b01;
        if (vv) M[p * b + v] = sc * b00 + cc * b01;
        if (qv) M[q * b + u] = cc * b10 - sc * b11;
        if (qv && vv) M[q * b + v] = sc * b10 + cc * b11;
      }
      // rows p, q of the accumulated rotations
      for (int e = tid; e < np * b; e += kEigThreads) {
        const int k = e / b, j = e - k * b;
        if (!pa[k]) continue;
        const int p = pp[k], q = pq[k];
        const double c = pc[k], sn = ps[k];
        const double ep = Et[static_cast<int64_t>(p) * b + j], eq = Et[static_cast<int64_t>(q) * b + j];
        Et[static_cast<int64_t>(p) * b + j] = c * ep - sn * eq;
        Et[static_cast<int64_t>(q) * b + j] = sn * ep + c * eq;
      }
      __syncthreads();
    }
    if (rot == 0) break;
    __syncthreads();
  }
  // rank of each eigenvalue (descending, index order on ties), then the outputs
  for (int i = tid; i < b; i += kEigThreads) {
    const double li = M[i * b + i];
    int rank = 0;
    for (int j = 0; j < b; ++j) {
      const double lj = M[j * b + j];
      rank += (lj > li || (lj == li && j < i)) ? 1 : 0;
    }
    lam[rank] = li;
    for (int row = 0; row < b; ++row) E[static_cast<int64_t>(row) * b + rank] = Et[static_cast<int64_t>(i) * b + row];
  }
}

// The same Jacobi iteration for b <= kEigLdsMax in two kernels, so that the
// accumulated rotations never need global memory inside the iteration:
// jacobi_log_kernel (one workgroup, the matrix in LDS) writes the eigenvalues
// (unsorted) to lraw, the number of sweeps to nsw and every step's rotations
// to rlog [sweep][step][pair] as (c, s) ((1, 0) for a pair not rotated);
// rot_apply_kernel then replays them on column slabs of the accumulated
// rotation matrix (its columns are independent under row rotations) and
// writes the outputs of jacobi_eig_kernel.
__global__ __launch_bounds__(kEigThreads) void jacobi_log_kernel(const double* A, double* lraw, int* nsw, double2* rlog,
                                                                 int b) {
  extern __shared__ double eig_smem[];
  __shared__ int pp[kEigLdsMax / 2], pq[kEigLdsMax / 2], pa[kEigLdsMax / 2];
  __shared__ double pc[kEigLdsMax / 2], ps[kEigLdsMax / 2];
  __shared__ int rot;
  __shared__ double floor_abs;
  const int tid = threadIdx.x;
  const int n2 = b + (b & 1), np = n2 / 2;
  double* M = eig_smem;
  for (int e = tid; e < b * b; e += kEigThreads) M[e] = A[e];
  if (tid == 0) {
    double mx = 0.0;
    for (int i = 0; i < b; ++i) mx = fmax(mx, fabs(A[static_cast<int64_t>(i) * b + i]));
    floor_abs = 1e-17 * mx;
  }
  __syncthreads();
  int sweeps = kEigMaxSweeps;
  for (int sweep = 0; sweep < kEigMaxSweeps; ++sweep) {
    if (tid == 0) rot = 0;
    __syncthreads();
    for (int s = 0; s < n2 - 1; ++s) {
      if (tid < np) {
        int p, q;
        rr_pair(n2, s, tid, p, q);
        double c = 1.0, sn = 0.0;
        bool act = false;
        if (q < b) {
          const double app = M[p * b + p], aqq = M[q * b + q], apq = M[p * b + q];
          if (apq != 0.0 && fabs(apq) > 1e-15 * sqrt(fabs(app * aqq)) && fabs(apq) > floor_abs) {
            const double zeta = (aqq - app) / (2.0 * apq);
            const double t = (zeta >= 0.0 ? 1.0 : -1.0) / (fabs(zeta) + sqrt(1.0 + zeta * zeta));
            c = 1.0 / sqrt(1.0 + t * t);
            sn = c * t;
            act = true;
          }
        }
        pp[tid] = p;
        pq[tid] = q;
        pa[tid] = act ? 1 : 0;
        pc[tid] = c;
        ps[tid] = sn;
        rlog[(static_cast<int64_t>(sweep) * (n2 - 1) + s) * np + tid] = make_double2(c, sn);
        if (act) atomicAdd(&rot, 1);
      }
      __syncthreads();
      // A <- J^T A J one 2 x 2 block at a time (rows of pair kr, columns of
      // pair kc): thread t takes row pair t / 16 and column pairs t % 16 + 16 j
      {
        const int kr = tid >> 4;
        if (kr < np) {
          const int p = pp[kr], q = pq[kr];
          const bool ar = pa[kr] != 0, qv = q < b;
          const double cr = pc[kr], sr = ps[kr];
          for (int kc = tid & 15; kc < np; kc += 16) {
            if (!ar && !pa[kc]) continue;
            const int u = pp[kc], v = pq[kc];
            const bool vv = v < b;
            const double cc = pc[kc], sc = ps[kc];
            const double a00 = M[p * b + u], a01 = vv ? M[p * b + v] : 0.0;
            const double a10 = qv ? M[q * b + u] : 0.0, a11 = (qv && vv) ? M[q * b + v] : 0.0;
            const double b00 = cr * a00 - sr * a10, b01 = cr * a01 - sr * a11;
            const double b10 = sr * a00 + cr * a10, b11 = sr * a01 + cr * a11;
            const double d00 = cc * b00 - sc * b01, d01 = sc * b00 + cc * b01;
            const double d10 = cc * b10 - sc * b11, d11 = sc * b10 + cc * b11;
            M[p * b + u] = d00;
            if (vv) M[p * b + v] = d01;
            if (qv) M[q * b + u] = d10;
            if (qv && vv) M[q * b + v] = d11;
          }
        }
      }
      __syncthreads();
    }
    if (rot == 0) {
      sweeps = sweep;  // a sweep that rotated nothing need not be replayed
      break;
    }
    __syncthreads();
  }
  for (int i = tid; i < b; i += kEigThreads) lraw[i] = M[i * b + i];
  if (tid == 0) *nsw = sweeps;
}

// jacobi_log_kernel for kEigLdsMax < b <= kPackMax: the symmetric matrix as
// its upper triangle in LDS (row i holds columns i .. b-1), each unordered
// 2 x 2 block {pair kr, pair kc} updated once; the thread group g (16
// threads) takes row pairs g and np - 1 - g, so every group has np + 1 blocks.
__device__ __forceinline__ int tri_up(int i, int j, int b) { return i * b - ((i * (i - 1)) >> 1) + (j - i); }
__device__ __forceinline__ int sym_at(int i, int j, int b) { return i <= j ? tri_up(i, j, b) : tri_up(j, i, b); }

__global__ __launch_bounds__(kEigThreads) void jacobi_log_packed_kernel(const double* A, double* lraw, int* nsw,
                                                                        double2* rlog, int b) {
  extern __shared__ double eig_smem[];
  __shared__ int pp[kPackMax / 2], pq[kPackMax / 2], pa[kPackMax / 2];
  __shared__ double pc[kPackMax / 2], ps[kPackMax / 2];
  __shared__ int rot;
  __shared__ double floor_abs;
  const int tid = threadIdx.x;
  const int n2 = b + (b & 1), np = n2 / 2;
  double* M = eig_smem;  // upper triangle, tri_up
  for (int i = tid >> 5; i < b; i += kEigThreads / 32)
    for (int j = i + (tid & 31); j < b; j += 32) M[tri_up(i, j, b)] = A[static_cast<int64_t>(i) * b + j];
  if (tid == 0) {
    double mx = 0.0;
    for (int i = 0; i < b; ++i) mx = fmax(mx, fabs(A[static_cast<int64_t>(i) * b + i]));
    floor_abs = 1e-17 * mx;
  }
  __syncthreads();
  const int grp = tid >> 4, gl = tid & 15;
  const int ngrp = (np + 1) / 2;
  int sweeps = kEigMaxSweeps;
  for (int sweep = 0; sweep < kEigMaxSweeps; ++sweep) {
    if (tid == 0) rot = 0;
    __syncthreads();
    for (int s = 0; s < n2 - 1; ++s) {
      if (tid < np) {
        int p, q;
        rr_pair(n2, s, tid, p, q);
        double c = 1.0, sn = 0.0;
        bool act = false;
        if (q < b) {
          const double app = M[tri_up(p, p, b)], aqq = M[tri_up(q, q, b)], apq = M[tri_up(p, q, b)];
          if (apq != 0.0 && fabs(apq) > 1e-15 * sqrt(fabs(app * aqq)) && fabs(apq) > floor_abs) {
            const double zeta = (aqq - app) / (2.0 * apq);
            const double t = (zeta >= 0.0 ? 1.0 : -1.0) / (fabs(zeta) + sqrt(1.0 + zeta * zeta));
            c = 1.0 / sqrt(1.0 + t * t);
            sn = c * t;
            act = true;
          }
        }
        pp[tid] = p;
        pq[tid] = q;
        pa[tid] = act ? 1 : 0;
        pc[tid] = c;
        ps[tid] = sn;
        rlog[(static_cast<int64_t>(sweep) * (n2 - 1) + s) * np + tid] = make_double2(c, sn);
        if (act) atomicAdd(&rot, 1);
      }
      __syncthreads();
      if (grp < ngrp) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int kr = h == 0 ? grp : np - 1 - grp;
          if (h == 1 && kr == grp) break;  // np odd: the middle row pair once
          const int p = pp[kr], q = pq[kr];
          const bool ar = pa[kr] != 0, qv = q < b;
          const double cr = pc[kr], sr = ps[kr];
          for (int kc = kr + gl; kc < np; kc += 16) {
            if (!ar && !pa[kc]) continue;
            const int u = pp[kc], v = pq[kc];
            const bool vv = v < b;
            const double cc = pc[kc], sc = ps[kc];
            const int i00 = sym_at(p, u, b), i01 = vv ? sym_at(p, v, b) : 0;
            const int i10 = qv ? sym_at(q, u, b) : 0, i11 = (qv && vv) ? sym_at(q, v, b) : 0;
            const double a00 = M[i00], a01 = vv ? M[i01] : 0.0;
            const double a10 = qv ? M[i10] : 0.0, a11 = (qv && vv) ? M[i11] : 0.0;
            const double b00 = cr * a00 - sr * a10, b01 = cr * a01 - sr * a11;
            const double b10 = sr * a00 + cr * a10, b11 = sr * a01 + cr * a11;
            const double d00 = cc * b00 - sc * b01, d01 = sc * b00 + cc * b01;
            const double d10 = cc * b10 - sc * b11, d11 = sc * b10 + cc * b11;
            M[i00] = d00;
            if (kc == kr) {
              // the diagonal block: (p, q) once, from the upper element
              if (qv) {
                M[i01] = d01;
                M[i11] = d11;
              }
            } else {
              if (vv) M[i01] = d01;
              if (qv) M[i10] = d10;
              if (qv && vv) M[i11] = d11;
            }
          }
        }
      }
      __syncthreads();
    }
    if (rot == 0) {
      sweeps = sweep;
      break;
    }
    __syncthreads();
  }
  for (int i = tid; i < b; i += kEigThreads) lraw[i] = M[tri_up(i, i, b)];
  if (tid == 0) *nsw = sweeps;
}

// Replay of jacobi_log_kernel's rotations on columns [kApplyCols * blockIdx.x,
// + kApplyCols) of the accumulated rotation matrix (identity at the start;
// row i is eigenvector i), then the outputs: eigenvalues descending (index
// order on ties) to lam, eigenvectors to the columns of E.
__global__ __launch_bounds__(kApplyThreads) void rot_apply_kernel(const double2* __restrict__ rlog,
                                                                  const int* __restrict__ nsw,
                                                                  const double* __restrict__ lraw, double* E,
                                                                  double* lam, int b) {
  extern __shared__ double ap_smem[];
  constexpr int C = kApplyCols;
  const int tid = threadIdx.x;
  const int n2 = b + (b & 1), np = n2 / 2, nst = n2 - 1;
  const int j0 = blockIdx.x * C;
  double* Ec = ap_smem;                                             // [b][C]
  double2* cs = reinterpret_cast<double2*>(ap_smem + b * C);        // [2][kRotBatch * np]
  const int per = kRotBatch * np;
  constexpr int kPer = (kRotBatch * (kPackMax / 2) + kApplyThreads - 1) / kApplyThreads;
  for (int e = tid; e < b * C; e += kApplyThreads) Ec[e] = (e / C == j0 + e % C) ? 1.0 : 0.0;
  const int total = *nsw * nst;
  const int nbatch = (total + kRotBatch - 1) / kRotBatch;
  // coefficients of batch bb: rlog entries [bb * per, (bb + 1) * per) (steps past the log: identity)
  auto fetch = [&](int bb, int e) {
    const int64_t g = static_cast<int64_t>(bb) * per + e;
    return bb * kRotBatch + e / np < total ? rlog[g] : make_double2(1.0, 0.0);
  };
  for (int e = tid; e < per; e += kApplyThreads) cs[e] = fetch(0, e);
  __syncthreads();
  for (int bb = 0; bb < nbatch; ++bb) {
    double2 nxt[kPer];
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int e = tid + kApplyThreads * u;
      nxt[u] = (e < per && bb + 1 < nbatch) ? fetch(bb + 1, e) : make_double2(1.0, 0.0);
    }
    const double2* cur = cs + (bb & 1) * per;
    for (int st = 0; st < kRotBatch; ++st) {
      const int gs = bb * kRotBatch + st;
      if (gs >= total) break;
      const int s = gs % nst;
      for (int e = tid; e < np * C; e += kApplyThreads) {
        const int k = e / C, jj = e - k * C;
        int p, q;
        rr_pair(n2, s, k, p, q);
        if (q < b) {
          const double2 r = cur[st * np + k];
          const double ep = Ec[p * C + jj], eq = Ec[q * C + jj];
          Ec[p * C + jj] = r.x * ep - r.y * eq;
          Ec[q * C + jj] = r.y * ep + r.x * eq;
        }
      }
      __syncthreads();
    }
    double2* other = cs + ((bb + 1) & 1) * per;
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int e = tid + kApplyThreads * u;
      if (e < per) other[e] = nxt[u];
    }
    __syncthreads();
  }
  for (int i = tid; i < b; i += kApplyThreads) {
    const double li = lraw[i];
    int rank = 0;
    for (int j = 0; j < b; ++j) {
      const double lj = lraw[j];
      rank += (lj > li || (lj == li && j < i)) ? 1 : 0;
    }
    if (blockIdx.x == 0) lam[rank] = li;
    for (int jj = 0; jj < C && j0 + jj < b; ++jj) E[static_cast<int64_t>(j0 + jj) * b + rank] = Ec[i * C + jj];
  }
}

// Orthonormalisation by Cholesky (CholQR): for the Gram matrix G = Y^T Y
// [b x b], G = L L^T (lower, in place in G's lower triangle), then T = L^-T
// (upper) into T, so that Q = Y T has orthonormal columns.  A pivot <= 1e-13
// of the largest diagonal entry is dropped (that column of L and of L^-1 is
// zero), so a rank-deficient block gives zero columns instead of a breakdown.
// X = L^-1 (lower triangular) is computed by right-looking forward
// substitution; its diagonal is 1 / L_kk.  One workgroup.  When b <=
// kEigLdsMax everything stays in LDS: L in the lower triangle of one b x b
// array and the strict lower part of X, flipped, in its upper triangle
// (X[i][c] at [b-1-i][b-1-c], c < i, so that a row of X is contiguous); column
// k of L is copied to a vector while it is scaled.  Else G and the scratch X
// [b x b] are used in global memory.
// factor_only (LDS variant): stop after the factorisation and write L to T
// with 1 / L_kk on its diagonal (for chol_solve_kernel).
template <bool kLds>
__global__ __launch_bounds__(kCholThreads) void chol_orth_kernel(double* G, double* X, double* T, int b,
                                                                 int factor_only) {
  extern __shared__ double chol_smem[];
  __shared__ double invs[kMaxBlock];
  __shared__ double colk[kMaxBlock];
  __shared__ double thr;
  const int tid = threadIdx.x;
  double* L = kLds ? chol_smem : G;
  if (kLds)
    for (int e = tid; e < b * b; e += kCholThreads) L[e] = G[e];
  else
    for (int e = tid; e < b * b; e += kCholThreads) X[e] = (e / b == e % b) ? 1.0 : 0.0;
  if (tid == 0) {
    double mx = 0.0;
    for (int i = 0; i < b; ++i) mx = fmax(mx, G[static_cast<int64_t>(i) * b + i]);
    thr = 1e-13 * mx;
  }
  __syncthreads();
  for (int k = 0; k < b; ++k) {
    const double d = L[k * b + k];
    const double inv = d > thr ? 1.0 / sqrt(d) : 0.0;
    if (tid == 0) invs[k] = inv;
    for (int i = k + 1 + tid; i < b; i += kCholThreads) {
      const double v = L[i * b + k] * inv;
      L[i * b + k] = v;
      colk[i] = v;
    }
    __syncthreads();
    // trailing update of the lower triangle: rows k + 1 + tid / 32 + 32 n,
    // columns k + 1 + tid % 32 + 32 n' <= row
    for (int i = k + 1 + (tid >> 5); i < b; i += kCholThreads / 32) {
      const double lik = colk[i];
      for (int j = k + 1 + (tid & 31); j <= i; j += 32) L[i * b + j] -= lik * colk[j];
    }
    __syncthreads();
  }
  if constexpr (kLds) {
    if (factor_only) {
      for (int e = tid; e < b * b; e += kCholThreads) {
        const int i = e / b, j = e - i * b;
        T[e] = j < i ? L[e] : (j == i ? invs[i] : 0.0);
      }
      return;
    }
    const int b1 = b - 1;
    // X's strict lower part (in the upper triangle) starts at 0
    for (int e = tid; e < b * b; e += kCholThreads)
      if (e % b > e / b) L[e] = 0.0;
    for (int i = tid; i < b; i += kCholThreads) colk[i] = 0.0;
    __syncthreads();
    // row k of X: X[k][c] = invs[k] * (updated right-hand side), c <= k (the
    // diagonal is invs[k] itself); the rows below subtract L_ik times it
    for (int k = 0; k < b; ++k) {
      const double inv = invs[k];
      double* xk = L + (b1 - k) * b + b1;  // X[k][c] at xk[-c]
      for (int c = tid; c < k; c += kCholThreads) xk[-c] *= inv;
      for (int i = k + 1 + tid; i < b; i += kCholThreads) colk[i] = L[i * b + k];
      __syncthreads();
      for (int i = k + 1 + (tid >> 5); i < b; i += kCholThreads / 32) {
        const double lik = colk[i];
        double* xi = L + (b1 - i) * b + b1;
        for (int c = tid & 31; c <= k; c += 32) xi[-c] -= lik * (c < k ? xk[-c] : inv);
      }
      __syncthreads();
    }
    for (int e = tid; e < b * b; e += kCholThreads) {
      const int j = e / b, k = e % b;  // T[j][k] = X[k][j]
      T[e] = j < k ? L[(b1 - k) * b + (b1 - j)] : (j == k ? invs[k] : 0.0);
    }
  } else {
    for (int k = 0; k < b; ++k) {
      const double inv = invs[k];
      for (int c = tid; c <= k; c += kCholThreads) X[static_cast<int64_t>(k) * b + c] *= inv;
      __syncthreads();
      const int w = b - k - 1;
      for (int e = tid; e < w * (k + 1); e += kCholThreads) {
        const int i = k + 1 + e / (k + 1), c = e % (k + 1);
        X[static_cast<int64_t>(i) * b + c] -= L[i * b + k] * X[static_cast<int64_t>(k) * b + c];
      }
      __syncthreads();
    }
    for (int e = tid; e < b * b; e += kCholThreads) {
      const int j = e / b, k = e % b;
      T[e] = X[static_cast<int64_t>(k) * b + j];
    }
  }
}

// Top eigenpair of the r x r Gram matrix A = F^T F of a nonnegative F (the
// rank-1 factors need nothing else) by power iteration from the all-ones
// vector, whose projection on the (nonnegative) Perron vector is positive:
// v <- A v / ||A v|| until ||A v - lambda v|| <= 1e-13 lambda (lambda = v^T A
// v) or kPowMaxIter steps.  The vector to column 0 of E, lambda to lam[0]
// (0 with v = e_1 for a zero matrix).  One workgroup; A in LDS when r <=
// kEigLdsMax, else read from global memory.
constexpr int kPowMaxIter = 20000;

__global__ __launch_bounds__(kEigThreads) void top_eig_kernel(const double* A, double* E, double* lam, int r) {
  extern __shared__ double pw_smem[];
  __shared__ double v[kMaxBlock], w[kMaxBlock];
  __shared__ double red[kEigThreads / 64][2];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const bool in_lds = r <= kEigLdsMax;
  const double* M = in_lds ? pw_smem : A;
  if (in_lds)
    for (int e = tid; e < r * r; e += kEigThreads) pw_smem[e] = A[e];
  const double v0 = 1.0 / sqrt(static_cast<double>(r));
  for (int i = tid; i < r; i += kEigThreads) v[i] = v0;
  __syncthreads();
  // two block sums (each wave's lanes by shuffles, then the waves in order)
  auto sum2 = [&](double a, double b, double& sa, double& sb) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      a += __shfl_xor(a, o);
      b += __shfl_xor(b, o);
    }
    if (lane == 0) {
      red[wv][0] = a;
      red[wv][1] = b;
    }
    __syncthreads();
    sa = 0.0;
    sb = 0.0;
    for (int k = 0; k < kEigThreads / 64; ++k) {
      sa += red[k][0];
      sb += red[k][1];
    }
    __syncthreads();
  };
  double lambda = 0.0;
  for (int it = 0; it < kPowMaxIter; ++it) {
    // w = A v: 8 threads per row, rows tid / 8 + 128 n
    for (int i0 = 0; i0 < r; i0 += kEigThreads / 8) {
      const int i = i0 + (tid >> 3);
      double s = 0.0;
      if (i < r)
        for (int j = tid & 7; j < r; j += 8) s += M[static_cast<int64_t>(i) * r + j] * v[j];
      s += __shfl_xor(s, 4);
      s += __shfl_xor(s, 2);
      s += __shfl_xor(s, 1);
      if (i < r && (tid & 7) == 0) w[i] = s;
    }
    __syncthreads();
    double pa = 0.0, pb = 0.0;
    for (int i = tid; i < r; i += kEigThreads) {
      pa += v[i] * w[i];
      pb += w[i] * w[i];
    }
    double vw, ww;
    sum2(pa, pb, vw, ww);
    lambda = vw;
    // residual ||w - lambda v||^2 and the new v
    double pr = 0.0;
    for (int i = tid; i < r; i += kEigThreads) {
      const double d = w[i] - lambda * v[i];
      pr += d * d;
    }
    double rr, unused;
    sum2(pr, 0.0, rr, unused);
    if (ww <= 0.0) {
      // a zero matrix: lambda 0, v = e_1
      lambda = 0.0;
      for (int i = tid; i < r; i += kEigThreads) v[i] = i == 0 ? 1.0 : 0.0;
      __syncthreads();
      break;
    }
    const bool conv = sqrt(rr) <= 1e-13 * fabs(lambda);
    const double inv = 1.0 / sqrt(ww);
    if (!conv)
      for (int i = tid; i < r; i += kEigThreads) v[i] = w[i] * inv;
    __syncthreads();
    if (conv) break;
  }
  for (int i = tid; i < r; i += kEigThreads) E[static_cast<int64_t>(i) * r] = v[i];
  if (tid == 0) lam[0] = lambda;
}

// Q = Y L^-T for CholQR with b <= kPackMax, row by row: q L^T = y, so
// q_k = (y_k - sum_{c<k} q_c L_kc) / L_kk.  64 rows per workgroup, 16 lanes
// per row (one DPP row): lane t holds y_c and q_c for c = t + 16 j in
// registers (the steps are unrolled, so the slot j is a constant), its part
// of each sum is added over the row by DPP, and the lane that holds y_k
// computes q_k; no LDS traffic or barrier per step.  L (lower, 1 / L_kk on
// the diagonal, as chol_orth_kernel's factor_only output) as its packed lower
// triangle in LDS.
constexpr int kSolveRows = 64;

// a double moved across lanes by a DPP control (both 32-bit halves)
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
  const uint64_t u = __double_as_longlong(v);
  const int lo = __builtin_amdgcn_update_dpp(0, static_cast<int>(u & 0xffffffffu), CTRL, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp(0, static_cast<int>(u >> 32), CTRL, 0xF, 0xF, false);
  return __longlong_as_double((static_cast<uint64_t>(static_cast<uint32_t>(hi)) << 32) | static_cast<uint32_t>(lo));
}
// the sum over the 16 lanes of a DPP row, in every lane (quad swaps, then the
// half-row and row mirrors)
__device__ __forceinline__ double row16_sum(double v) {
  v += dpp_f64<0xB1>(v);   // quad_perm [1, 0, 3, 2]
  v += dpp_f64<0x4E>(v);   // quad_perm [2, 3, 0, 1]
  v += dpp_f64<0x141>(v);  // row_half_mirror
  v += dpp_f64<0x140>(v);  // row_mirror
  return v;
}

template <int kSolveSlots>  // b <= 16 kSolveSlots
__global__ __launch_bounds__(kCholThreads) void chol_solve_kernel(const double* Y, const double* Lf, double* Q,
                                                                  int rows, int b) {
  extern __shared__ double sv_smem[];
  double* Lp = sv_smem;  // tri_lo
  const int tid = threadIdx.x;
  for (int i = tid >> 5; i < b; i += kCholThreads / 32)
    for (int j = tid & 31; j <= i; j += 32) Lp[((i * (i + 1)) >> 1) + j] = Lf[static_cast<int64_t>(i) * b + j];
  const int t = tid & 15;
  const int row = blockIdx.x * kSolveRows + (tid >> 4);
  const bool ok = row < rows;
  double q[kSolveSlots];
#pragma unroll
  for (int j = 0; j < kSolveSlots; ++j) {
    const int c = t + 16 * j;
    q[j] = ok && c < b ? Y[static_cast<int64_t>(row) * b + c] : 0.0;  // y, replaced by q step by step
  }
  __syncthreads();
#pragma unroll
  for (int kb = 0; kb < kSolveSlots; ++kb) {
#pragma unroll
    for (int t0 = 0; t0 < 16; ++t0) {
      const int k = 16 * kb + t0;
      if (k >= b) break;
      const double* lk = Lp + ((k * (k + 1)) >> 1);
      double s = 0.0;
#pragma unroll
      for (int j = 0; j <= kb; ++j) {
        const int c = t + 16 * j;
        if (c < k) s += q[j] * lk[c];
      }
      s = row16_sum(s);
      if (t == t0) q[kb] = (q[kb] - s) * lk[k];
    }
  }
#pragma unroll
  for (int j = 0; j < kSolveSlots; ++j) {
    const int c = t + 16 * j;
    if (ok && c < b) Q[static_cast<int64_t>(row) * b + c] = q[j];
  }
}

// CholQR for kEigLdsMax < b <= kPackMax (factor_only: stop after the
// factorisation, as chol_orth_kernel): L as its lower triangle in LDS (row
// i holds columns 0 .. i), factorised as in chol_orth_kernel; then L^-1 in
// place, from the last column to the first: column j of L^-1 below the
// diagonal is -(1 / L_jj) times the already inverted trailing block applied to
// column j of L (each row's sum on 32 lanes); the diagonal is 1 / L_jj (0 for
// a dropped pivot, whose row and column of L^-1 are then 0).  T = L^-T.
__device__ __forceinline__ int tri_lo(int i, int j) { return ((i * (i + 1)) >> 1) + j; }

__global__ __launch_bounds__(kCholThreads) void chol_orth_packed_kernel(const double* G, double* T, int b,
                                                                        int factor_only) {
  extern __shared__ double chol_smem[];
  __shared__ double invs[kPackMax];
  __shared__ double colk[kPackMax];
  __shared__ double thr;
  const int tid = threadIdx.x;
  const int lane32 = tid & 31;
  double* L = chol_smem;  // tri_lo
  for (int i = tid >> 5; i < b; i += kCholThreads / 32)
    for (int j = lane32; j <= i; j += 32) L[tri_lo(i, j)] = G[static_cast<int64_t>(i) * b + j];
  if (tid == 0) {
    double mx = 0.0;
    for (int i = 0; i < b; ++i) mx = fmax(mx, G[static_cast<int64_t>(i) * b + i]);
    thr = 1e-13 * mx;
  }
  __syncthreads();
  for (int k = 0; k < b; ++k) {
    const double d = L[tri_lo(k, k)];
    const double inv = d > thr ? 1.0 / sqrt(d) : 0.0;
    if (tid == 0) invs[k] = inv;
    for (int i = k + 1 + tid; i < b; i += kCholThreads) {
      const double v = L[tri_lo(i, k)] * inv;
      L[tri_lo(i, k)] = v;
      colk[i] = v;
    }
    __syncthreads();
    for (int i = k + 1 + (tid >> 5); i < b; i += kCholThreads / 32) {
      const double lik = colk[i];
      double* row = L + tri_lo(i, 0);
      for (int j = k + 1 + lane32; j <= i; j += 32) row[j] -= lik * colk[j];
    }
    __syncthreads();
  }
  for (int i = tid; i < b; i += kCholThreads) L[tri_lo(i, i)] = invs[i];
  __syncthreads();
  if (factor_only) {
    // L with 1 / L_kk on its diagonal, for chol_solve_kernel
    for (int e = tid; e < b * b; e += kCholThreads) {
      const int i = e / b, j = e - i * b;
      T[e] = j <= i ? L[tri_lo(i, j)] : 0.0;
    }
    return;
  }
  for (int j = b - 1; j >= 0; --j) {
    for (int i = j + 1 + tid; i < b; i += kCholThreads) colk[i] = L[tri_lo(i, j)];
    __syncthreads();
    for (int i = j + 1 + (tid >> 5); i < b; i += kCholThreads / 32) {
      const double* row = L + tri_lo(i, 0);
      double acc = 0.0;
      for (int c = j + 1 + lane32; c <= i; c += 32) acc += row[c] * colk[c];
#pragma unroll
      for (int o = 16; o >= 1; o >>= 1) acc += __shfl_xor(acc, o);
      if (lane32 == 0) L[tri_lo(i, j)] = -invs[j] * acc;
    }
    __syncthreads();
  }
  for (int e = tid; e < b * b; e += kCholThreads) {
    const int jj = e / b, k = e - jj * b;  // T[jj][k] = X[k][jj]
    T[e] = jj <= k ? L[tri_lo(k, jj)] : 0.0;
  }
}

// Uniform values in [-1, 1) from the SplitMix64 generator (Steele, Lea and
// Flood, 2014) at counter seed + idx: the subspace iteration's starting block.
__global__ void rand_fill_kernel(double* Z, int64_t n, uint64_t seed) {
  for (int64_t i = blockIdx.x * 256ll + threadIdx.x; i < n; i += static_cast<int64_t>(gridDim.x) * 256) {
    uint64_t z = seed + static_cast<uint64_t>(i + 1) * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    z ^= z >> 31;
    Z[i] = static_cast<double>(z >> 11) * 0x1.0p-52 - 1.0;
  }
}

// Fixed-order sum of v[0 .. n) over one workgroup of 256 threads (strided
// partial sums, then a tree); every thread gets the result.
__device__ double block_sum(double v, double* red) {
  const int tid = threadIdx.x;
  red[tid] = v;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (tid < w) red[tid] += red[tid + w];
    __syncthreads();
  }
  const double s = red[0];
  __syncthreads();
  return s;
}

// One workgroup per singular pair k: sigma_k = sqrt(max(lambda_k, 0)); the
// left vector (column k of U) signed so that its entry of largest magnitude is
// positive (first index on a tie), the right vector = Vraw[:, k] / sigma_k
// (zero if sigma_k == 0) with the same sign; U' = U sqrt(sigma), V' = V
// sqrt(sigma), fp64 to Ul, Vl and fp32 to the caller's arrays.
__global__ __launch_bounds__(256) void sign_scale_kernel(const double* U, const double* Vraw, const double* lam, int m,
                                                         int n, int r, double* Ul, double* Vl, float* Uo, float* Vo,
                                                         float* sig) {
  __shared__ double bv[256];
  __shared__ int bi[256];
  const int k = blockIdx.x, tid = threadIdx.x;
  double best = -1.0;
  int besti = 0;
  for (int i = tid; i < m; i += 256) {
    const double v = fabs(U[static_cast<int64_t>(i) * r + k]);
    if (v > best) {
      best = v;
      besti = i;
    }
  }
  bv[tid] = best;
  bi[tid] = besti;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (tid < w) {
      const double o = bv[tid + w];
      const int oi = bi[tid + w];
      if (o > bv[tid] || (o == bv[tid] && oi < bi[tid])) {
        bv[tid] = o;
        bi[tid] = oi;
      }
    }
    __syncthreads();
  }
  const double s = sqrt(fmax(lam[k], 0.0));
  const double f = U[static_cast<int64_t>(bi[0]) * r + k] < 0.0 ? -1.0 : 1.0;
  const double rs = sqrt(s);
  if (tid == 0 && sig) sig[k] = static_cast<float>(s);
  for (int i = tid; i < m; i += 256) {
    const int64_t e = static_cast<int64_t>(i) * r + k;
    const double v = f * U[e] * rs;
    Ul[e] = v;
    Uo[e] = static_cast<float>(v);
  }
  for (int j = tid; j < n; j += 256) {
    const int64_t e = static_cast<int64_t>(j) * r + k;
    const double v = s > 0.0 ? f * (Vraw[e] / s) * rs : 0.0;
    Vl[e] = v;
    Vo[e] = static_cast<float>(v);
  }
}

// Rank-1 factors of a nonnegative M [d x r] from the top eigenpair (lambda_1,
// e_1) of M^T M and u = M e_1: sigma_1 = sqrt(lambda_1), left factor
// f u / sqrt(sigma_1), right factor f sqrt(sigma_1) e_1, f = +-1 so that the
// left factor sums to >= 0 (zero factors when lambda_1 <= 0).  One workgroup.
__global__ __launch_bounds__(256) void rank1_finish_kernel(const double* u, const double* lam, const double* E, int d,
                                                           int r, double* left, float* left_o, double* right) {
  __shared__ double red[256];
  const int tid = threadIdx.x;
  double part = 0.0;
  for (int i = tid; i < d; i += 256) part += u[i];
  const double sum = block_sum(part, red);
  const double f = sum >= 0.0 ? 1.0 : -1.0;
  const double l1 = lam[0];
  const double q = l1 > 0.0 ? sqrt(sqrt(l1)) : 0.0;
  for (int i = tid; i < d; i += 256) {
    const double v = q > 0.0 ? f * u[i] / q : 0.0;
    left[i] = v;
    left_o[i] = static_cast<float>(v);
  }
  for (int k = tid; k < r; k += 256) right[k] = f * q * E[static_cast<int64_t>(k) * r];
}

// l = l_u (.) l_v; the operands of the effective weight, Us[i][k] =
// sign(U'[i][k]) l[k] and Vs[j][k] = sign(V'[j][k]) (sign: -1 iff < 0).
__global__ void latent_and_signs_kernel(const double* lu, const double* lv, const double* Ul, const double* Vl, int m,
                                        int n, int r, double* l, float* l_o, double* Us, double* Vs) {
  const int64_t nu = static_cast<int64_t>(m) * r, nv = static_cast<int64_t>(n) * r;
  for (int64_t e = blockIdx.x * 256ll + threadIdx.x; e < nu + nv + r; e += static_cast<int64_t>(gridDim.x) * 256) {
    if (e < nu) {
      const int k = static_cast<int>(e % r);
      Us[e] = (Ul[e] < 0.0 ? -1.0 : 1.0) * (lu[k] * lv[k]);
    } else if (e < nu + nv) {
      const int64_t f = e - nu;
      Vs[f] = Vl[f] < 0.0 ? -1.0 : 1.0;
    } else {
      const int k = static_cast<int>(e - nu - nv);
      l[k] = lu[k] * lv[k];
      l_o[k] = static_cast<float>(l[k]);
    }
  }
}

__global__ void f64_to_f32_kernel(const double* s, float* d, int64_t n) {
  for (int64_t i = blockIdx.x * 256ll + threadIdx.x; i < n; i += static_cast<int64_t>(gridDim.x) * 256)
    d[i] = static_cast<float>(s[i]);
}

int grid_for(int64_t n) { return static_cast<int>(std::min<int64_t>(4096, std::max<int64_t>(1, (n + 255) / 256))); }

size_t a256(size_t b) { return (b + 255) / 256 * 256; }

struct SvidLayout {
  int m, n, r, b;
  size_t wres, y, q, z, z2, part, gram, e, et, lam, lraw, nsw, rlog, ud, vd, ul, vl, us, vs, u, h, g, lu, lv, l, total;
  size_t part_elems;
};

SvidLayout svid_layout(int m, int n, int r, int over) {
  SvidLayout L{};
  L.m = m;
  L.n = n;
  L.r = r;
  L.b = std::min<int64_t>(static_cast<int64_t>(r) + over, std::min(m, n));
  const size_t b = L.b, mx = std::max(m, n);
  L.part_elems = std::max<size_t>(64 * b * b, 8 * mx * b);
  size_t off = 0;
  auto take = [&](size_t elems) {
    const size_t o = off;
    off += a256(elems * sizeof(double));
    return o;
  };
  L.wres = take(static_cast<size_t>(m) * n);
  L.y = take(static_cast<size_t>(m) * b);
  L.q = take(static_cast<size_t>(m) * b);
  L.z = take(static_cast<size_t>(n) * b);
  L.z2 = take(static_cast<size_t>(n) * b);
  L.part = take(L.part_elems);
  L.gram = take(b * b);
  L.e = take(b * b);
  L.et = take(b * b);
  L.lam = take(b);
  L.lraw = take(b);
  L.nsw = take(1);
  {
    // rotation log of the largest eigenproblem solved in LDS (b or r)
    size_t bl = 0;
    if (b <= static_cast<size_t>(kPackMax)) bl = b;
    if (static_cast<size_t>(r) <= static_cast<size_t>(kPackMax) && static_cast<size_t>(r) > bl) bl = r;
    const size_t n2 = bl + (bl & 1);
    L.rlog = take(bl > 0 ? 2 * static_cast<size_t>(kEigMaxSweeps) * (n2 - 1) * (n2 / 2) : 0);
  }
  L.ud = take(static_cast<size_t>(m) * r);
  L.vd = take(static_cast<size_t>(n) * r);
  L.ul = take(static_cast<size_t>(m) * r);
  L.vl = take(static_cast<size_t>(n) * r);
  L.us = take(static_cast<size_t>(m) * r);
  L.vs = take(static_cast<size_t>(n) * r);
  L.u = take(mx);
  L.h = take(m);
  L.g = take(n);
  L.lu = take(r);
  L.lv = take(r);
  L.l = take(r);
  L.total = off;
  return L;
}

struct Svid {
  const SvidLayout& L;
  char* ws;
  hipStream_t st;
  double* at(size_t off) const { return reinterpret_cast<double*>(ws + off); }

  template <int ADT>
  void launch_gemm(const GemmArgs& run, dim3 grid) const {
    const bool ak = run.sak == 1, bj = run.sbj == 1;
    if (ak && bj)
      hipLaunchKernelGGL((gemm64_kernel<true, true, ADT>), grid, dim3(256), 0, st, run);
    else if (ak)
      hipLaunchKernelGGL((gemm64_kernel<true, false, ADT>), grid, dim3(256), 0, st, run);
    else if (bj)
      hipLaunchKernelGGL((gemm64_kernel<false, true, ADT>), grid, dim3(256), 0, st, run);
    else
      hipLaunchKernelGGL((gemm64_kernel<false, false, ADT>), grid, dim3(256), 0, st, run);
  }

  // C [M x N] = op(A) [M x K] * B [K x N]; K split so that the launch has
  // about 512 workgroups, when the partial slabs fit and each split keeps at
  // least 256 of K.
  hipError_t gemm(GemmArgs g) const {
    if (g.M <= 0 || g.N <= 0) return hipSuccess;
    const int tiles = ((g.M + kGT - 1) / kGT) * ((g.N + kGT - 1) / kGT);
    const size_t slab = static_cast<size_t>(g.M) * g.N;
    int split = std::max(1, 512 / tiles);
    split = std::min(split, std::max(1, g.K / 256));
    split = static_cast<int>(std::min<size_t>(split, std::max<size_t>(1, L.part_elems / slab)));
    const int kchunk = std::max(kGK, ((g.K + split - 1) / split + kGK - 1) / kGK * kGK);
    split = std::max(1, (g.K + kchunk - 1) / kchunk);
    g.kchunk = kchunk;
    g.ksplit = split;
    GemmArgs run = g;
    if (split > 1) {
      run.C = at(L.part);
      run.ldc = g.N;
      run.pstride = static_cast<int64_t>(slab);
    }
    const dim3 grid((g.M + kGT - 1) / kGT, (g.N + kGT - 1) / kGT, split);
    if (g.b_dt != kDtF64) return hipErrorInvalidValue;  // every B operand is an fp64 array of this file
    switch (g.a_dt) {
      case kDtF64: launch_gemm<kDtF64>(run, grid); break;
      case kDtF32: launch_gemm<kDtF32>(run, grid); break;
      case kDtF16: launch_gemm<kDtF16>(run, grid); break;
      default: launch_gemm<kDtBF16>(run, grid); break;
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || split == 1) return e;
    hipLaunchKernelGGL(gemm_reduce_kernel, dim3(grid_for(static_cast<int64_t>(slab))), dim3(256), 0, st, g,
                       static_cast<const double*>(at(L.part)));
    return hipGetLastError();
  }

  hipError_t eig(double* A, double* E, double* lam, int b) const {
    if (b <= kPackMax) {
      // full matrix in LDS up to kEigLdsMax, its upper triangle above
      const bool full = b <= kEigLdsMax;
      const int smem = static_cast<int>(sizeof(double) * (full ? b * b : b * (b + 1) / 2));
      const void* fn = full ? reinterpret_cast<const void*>(&jacobi_log_kernel)
                            : reinterpret_cast<const void*>(&jacobi_log_packed_kernel);
      if (smem > 65536) {
        const hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, smem);
        if (e != hipSuccess) return e;
      }
      double2* rl = reinterpret_cast<double2*>(at(L.rlog));
      int* ns = reinterpret_cast<int*>(at(L.nsw));
      if (full)
        hipLaunchKernelGGL(jacobi_log_kernel, dim3(1), dim3(kEigThreads), smem, st, static_cast<const double*>(A),
                           at(L.lraw), ns, rl, b);
      else
        hipLaunchKernelGGL(jacobi_log_packed_kernel, dim3(1), dim3(kEigThreads), smem, st,
                           static_cast<const double*>(A), at(L.lraw), ns, rl, b);
      if (const hipError_t e = hipGetLastError(); e != hipSuccess) return e;
      const int np = (b + (b & 1)) / 2;
      const size_t smem2 = sizeof(double) * b * kApplyCols + sizeof(double2) * 2 * kRotBatch * np;
      hipLaunchKernelGGL(rot_apply_kernel, dim3((b + kApplyCols - 1) / kApplyCols), dim3(kApplyThreads), smem2, st,
                         static_cast<const double2*>(rl), static_cast<const int*>(ns),
                         static_cast<const double*>(at(L.lraw)), E, lam, b);
    } else {
      hipLaunchKernelGGL((jacobi_eig_kernel<false>), dim3(1), dim3(kEigThreads), 0, st, A, at(L.et), E, lam, b);
    }
    return hipGetLastError();
  }

  // C = op(A) * B with A, B given by element strides (see GemmArgs)
  hipError_t mm(const void* A, int adt, int64_t sai, int64_t sak, bool aabs, const void* B, int bdt, int64_t sbk,
                int64_t sbj, bool babs, double* C, int64_t ldc, int M, int N, int K) const {
    GemmArgs g{};
    g.A = A;
    g.a_dt = adt;
    g.a_abs = aabs;
    g.sai = sai;
    g.sak = sak;
    g.B = B;
    g.b_dt = bdt;
    g.b_abs = babs;
    g.sbk = sbk;
    g.sbj = sbj;
    g.C = C;
    g.ldc = ldc;
    g.M = M;
    g.N = N;
    g.K = K;
    g.epi = kEpiStore;
    return gemm(g);
  }

  // Y [rows x b] -> a basis of its range in Qo [rows x b] by CholQR: G =
  // Y^T Y = L L^T, Qo = Y L^-T (dropped pivots give zero columns); the
  // columns are orthonormal up to about cond(Y)^2 times the rounding unit,
  // which is all the iteration needs
  // Qo = Y L^-T from the factor chol_orth_*_kernel left in L.e (b <= kPackMax)
  hipError_t solve(const double* Y, double* Qo, int rows, int b) const {
    const int smem = static_cast<int>(sizeof(double) * b * (b + 1) / 2);
    const void* fn = b <= 128 ? reinterpret_cast<const void*>(&chol_solve_kernel<8>)
                              : reinterpret_cast<const void*>(&chol_solve_kernel<12>);
    if (smem > 65536) {
      const hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, smem);
      if (e != hipSuccess) return e;
    }
    const dim3 grid((rows + kSolveRows - 1) / kSolveRows);
    if (b <= 128)
      hipLaunchKernelGGL(chol_solve_kernel<8>, grid, dim3(kCholThreads), smem, st, Y,
                         static_cast<const double*>(at(L.e)), Qo, rows, b);
    else
      hipLaunchKernelGGL(chol_solve_kernel<12>, grid, dim3(kCholThreads), smem, st, Y,
                         static_cast<const double*>(at(L.e)), Qo, rows, b);
    return hipGetLastError();
  }

  hipError_t orth_chol(const double* Y, double* Qo, int rows) const {
    const int b = L.b;
    hipError_t e;
    if ((e = mm(Y, kDtF64, 1, b, false, Y, kDtF64, b, 1, false, at(L.gram), b, b, b, rows)) != hipSuccess) return e;
    if (b <= kEigLdsMax) {
      const int smem = static_cast<int>(sizeof(double) * b * b);
      if (smem > 65536) {
        e = hipFuncSetAttribute(reinterpret_cast<const void*>(&chol_orth_kernel<true>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, smem);
        if (e != hipSuccess) return e;
      }
      hipLaunchKernelGGL((chol_orth_kernel<true>), dim3(1), dim3(kCholThreads), smem, st, at(L.gram), at(L.et),
                         at(L.e), b, 1);
      if ((e = hipGetLastError()) != hipSuccess) return e;
      return solve(Y, Qo, rows, b);
    } else if (b <= kPackMax) {
      const int smem = static_cast<int>(sizeof(double) * b * (b + 1) / 2);
      if (smem > 65536) {
        e = hipFuncSetAttribute(reinterpret_cast<const void*>(&chol_orth_packed_kernel),
                                hipFuncAttributeMaxDynamicSharedMemorySize, smem);
        if (e != hipSuccess) return e;
      }
      hipLaunchKernelGGL(chol_orth_packed_kernel, dim3(1), dim3(kCholThreads), smem, st,
                         static_cast<const double*>(at(L.gram)), at(L.e), b, 1);
      if ((e = hipGetLastError()) != hipSuccess) return e;
      return solve(Y, Qo, rows, b);
    } else {
      hipLaunchKernelGGL((chol_orth_kernel<false>), dim3(1), dim3(kCholThreads), 0, st, at(L.gram), at(L.et),
                         at(L.e), b, 0);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return mm(Y, kDtF64, b, 1, false, at(L.e), kDtF64, b, 1, false, Qo, b, rows, b, b);
  }

  // Rank-1 factors of |F| for F [d x r] (fp64): left to left/left_o, right to right
  hipError_t rank1(const double* F, int d, double* left, float* left_o, double* right) const {
    const int r = L.r;
    hipError_t e;
    if ((e = mm(F, kDtF64, 1, r, true, F, kDtF64, r, 1, true, at(L.gram), r, r, r, d)) != hipSuccess) return e;
    // the top eigenpair of |F|^T |F| (column 0 of E, lam[0])
    {
      const int smem = r <= kEigLdsMax ? static_cast<int>(sizeof(double) * r * r) : 0;
      if (smem > 65536) {
        e = hipFuncSetAttribute(reinterpret_cast<const void*>(&top_eig_kernel),
                                hipFuncAttributeMaxDynamicSharedMemorySize, smem);
        if (e != hipSuccess) return e;
      }
      hipLaunchKernelGGL(top_eig_kernel, dim3(1), dim3(kEigThreads), smem, st, static_cast<const double*>(at(L.gram)),
                         at(L.e), at(L.lam), r);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    // u = |F| e_1 (the first column of E)
    if ((e = mm(F, kDtF64, r, 1, true, at(L.e), kDtF64, r, 1, false, at(L.u), 1, d, 1, r)) != hipSuccess) return e;
    hipLaunchKernelGGL(rank1_finish_kernel, dim3(1), dim3(256), 0, st, static_cast<const double*>(at(L.u)),
                       static_cast<const double*>(at(L.lam)), static_cast<const double*>(at(L.e)), d, r, left, left_o,
                       right);
    return hipGetLastError();
  }

  // One path from W (dtype wdt, [m x n] row-major) into the caller's outputs.
  hipError_t path(const void* W, int wdt, const lb_svid_out& o, int iters, uint64_t seed) const {
    const int m = L.m, n = L.n, r = L.r, b = L.b;
    double *Y = at(L.y), *Q = at(L.q), *Z = at(L.z), *Z2 = at(L.z2);
    hipError_t e;
    hipLaunchKernelGGL(rand_fill_kernel, dim3(grid_for(static_cast<int64_t>(n) * b)), dim3(256), 0, st, Z,
                       static_cast<int64_t>(n) * b, seed);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // Y = W Z; per round Q = orth_chol(Y), Z = orth_chol(W^T Q), Y = W Z;
    // then Q = orth_chol(Y)
    if ((e = mm(W, wdt, n, 1, false, Z, kDtF64, b, 1, false, Y, b, m, b, n)) != hipSuccess) return e;
    for (int it = 0; it < iters; ++it) {
      if ((e = orth_chol(Y, Q, m)) != hipSuccess) return e;
      if ((e = mm(W, wdt, 1, n, false, Q, kDtF64, b, 1, false, Z2, b, n, b, m)) != hipSuccess) return e;
      if ((e = orth_chol(Z2, Z, n)) != hipSuccess) return e;
      if ((e = mm(W, wdt, n, 1, false, Z, kDtF64, b, 1, false, Y, b, m, b, n)) != hipSuccess) return e;
    }
    if ((e = orth_chol(Y, Q, m)) != hipSuccess) return e;
    // Rayleigh-Ritz: Z = W^T Q, Z^T Z = E diag(lambda) E^T, U = Q E_r, V = Z E_r / sigma
    if ((e = mm(W, wdt, 1, n, false, Q, kDtF64, b, 1, false, Z, b, n, b, m)) != hipSuccess) return e;
    if ((e = mm(Z, kDtF64, 1, b, false, Z, kDtF64, b, 1, false, at(L.gram), b, b, b, n)) != hipSuccess) return e;
    if ((e = eig(at(L.gram), at(L.e), at(L.lam), b)) != hipSuccess) return e;
    if ((e = mm(Q, kDtF64, b, 1, false, at(L.e), kDtF64, b, 1, false, at(L.ud), r, m, r, b)) != hipSuccess) return e;
    if ((e = mm(Z, kDtF64, b, 1, false, at(L.e), kDtF64, b, 1, false, at(L.vd), r, n, r, b)) != hipSuccess) return e;
    hipLaunchKernelGGL(sign_scale_kernel, dim3(r), dim3(256), 0, st, static_cast<const double*>(at(L.ud)),
                       static_cast<const double*>(at(L.vd)), static_cast<const double*>(at(L.lam)), m, n, r,
                       at(L.ul), at(L.vl), o.U_latent, o.V_latent, o.sigma);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = rank1(at(L.ul), m, at(L.h), o.h, at(L.lu))) != hipSuccess) return e;
    if ((e = rank1(at(L.vl), n, at(L.g), o.g, at(L.lv))) != hipSuccess) return e;
    const int64_t nl = static_cast<int64_t>(m + n) * r + r;
    hipLaunchKernelGGL(latent_and_signs_kernel, dim3(grid_for(nl)), dim3(256), 0, st,
                       static_cast<const double*>(at(L.lu)), static_cast<const double*>(at(L.lv)),
                       static_cast<const double*>(at(L.ul)), static_cast<const double*>(at(L.vl)), m, n, r, at(L.l),
                       o.l, at(L.us), at(L.vs));
    return hipGetLastError();
  }

  // W_res = W - diag(h) sign(U') diag(l) sign(V')^T diag(g) of the path just run
  hipError_t residual(const void* W, int wdt) const {
    const int m = L.m, n = L.n, r = L.r;
    GemmArgs g{};
    g.A = at(L.us);
    g.a_dt = kDtF64;
    g.sai = r;
    g.sak = 1;
    g.B = at(L.vs);
    g.b_dt = kDtF64;
    g.sbk = 1;
    g.sbj = r;
    g.C = at(L.wres);
    g.ldc = n;
    g.M = m;
    g.N = n;
    g.K = r;
    g.epi = kEpiResid;
    g.W = W;
    g.w_dt = wdt;
    g.ldw = n;
    g.h = at(L.h);
    g.g = at(L.g);
    return gemm(g);
  }
};

}  // namespace

bool svid_supports(int64_t d_out, int64_t d_in, int64_t r, int64_t over) {
  if (d_out <= 0 || d_in <= 0 || r <= 0 || over < 0) return false;
  if (r > std::min(d_out, d_in)) return false;
  return std::min<int64_t>(r + over, std::min(d_out, d_in)) <= kMaxBlock;
}

size_t svid_workspace_bytes(int d_out, int d_in, int r, int over) {
  return svid_layout(d_out, d_in, r, over).total;
}

hipError_t launch_dual_svid(const void* W, int wdt, int d_out, int d_in, int r, int over, int iters, uint64_t seed,
                            const lb_svid_out* out, float* W_res, void* ws, hipStream_t stream) {
  const SvidLayout L = svid_layout(d_out, d_in, r, over);
  const Svid S{L, static_cast<char*>(ws), stream};
  hipError_t e;
  if ((e = S.path(W, wdt, out[0], iters, seed)) != hipSuccess) return e;
  if ((e = S.residual(W, wdt)) != hipSuccess) return e;
  if (W_res) {
    const int64_t nw = static_cast<int64_t>(d_out) * d_in;
    hipLaunchKernelGGL(f64_to_f32_kernel, dim3(grid_for(nw)), dim3(256), 0, stream,
                       static_cast<const double*>(S.at(L.wres)), W_res, nw);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return S.path(S.at(L.wres), kDtF64, out[1], iters, seed + 0x632BE59BD9B4E019ull);
}

}  // namespace lb
