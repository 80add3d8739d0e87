// Host-side driver for the sanitizer build (AddressSanitizer and
// UndefinedBehaviorSanitizer on the host code only): exercises the C ABI's
// validation paths and pure helpers, which enqueue nothing, and the oracle's C
// functions on small inputs.  Exits non-zero on the first unexpected result.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "../../include/littlebit.h"

extern "C" {
int64_t lbo_packed_bytes(int64_t rows, int64_t r, int role);
int64_t lbo_pack(const double* src, int64_t rows, int64_t r, int role, uint8_t* dst);
void lbo_unpack(const uint8_t* buf, int64_t rows, int64_t r, int role, int8_t* out);
void lbo_forward_factored(const double* x, int64_t T, int64_t d_in, int64_t d_out, int64_t r,
                          const int8_t* const* U, const int8_t* const* V, const double* const* h,
                          const double* const* g, const double* const* l, int npaths, double* y);
void lbo_forward_factored_par(const double* x, int64_t T, int64_t d_in, int64_t d_out, int64_t r,
                              const int8_t* const* U, const int8_t* const* V, const double* const* h,
                              const double* const* g, const double* const* l, int npaths, int nthreads,
                              double* y);
void lbo_dense_weight(int64_t d_in, int64_t d_out, int64_t r, const int8_t* const* U, const int8_t* const* V,
                      const double* const* h, const double* const* g, const double* const* l, int npaths,
                      double* W);
void lbo_latent(const double* x, int64_t T, int64_t d_in, int64_t r, const int8_t* const* V,
                const double* const* g, const double* const* l, int npaths, double* w);
void lbo_from_latent(const double* w, int64_t T, int64_t d_out, int64_t r, const int8_t* const* U,
                     const double* const* h, int npaths, double* y);
}

static int failures = 0;
#define EXPECT(c)                                                   \
  do {                                                              \
    if (!(c)) {                                                     \
      std::fprintf(stderr, "%s:%d: failed: %s\n", __FILE__, __LINE__, #c); \
      ++failures;                                                   \
    }                                                               \
  } while (0)

// Host addresses standing in for device pointers: validation never reads them.
static char fake_buf[1 << 12] __attribute__((aligned(256)));

static lb_path fake_path() {
  return lb_path{fake_buf, fake_buf, fake_buf, fake_buf, fake_buf};
}

static void abi_checks() {
  EXPECT(lb_abi_version() == LB_ABI_VERSION);
  for (int s = 0; s <= 8; ++s) EXPECT(lb_status_str(static_cast<lb_status>(s)) != nullptr);
  // pure helpers over a sweep of sizes (overflow and rounding paths)
  for (int64_t d : {int64_t(0), int64_t(1), int64_t(31), int64_t(32), int64_t(33), int64_t(4096), int64_t(28672), (int64_t(1) << 31) - 1, int64_t(1) << 40}) {
    for (int64_t r : {int64_t(0), int64_t(1), int64_t(16), int64_t(17), int64_t(80), int64_t(1024)}) {
      (void)lb_packed_bytes(LB_ROLE_U, d, r);
      (void)lb_packed_bytes(LB_ROLE_V, d, r);
      (void)lb_forward_workspace_bytes(4, d, d, r);
      (void)lb_forward_workspace_bytes(2048, d, d, r);
      (void)lb_latent_workspace_bytes(64, d, r);
      (void)lb_from_latent_workspace_bytes(64, r);
      (void)lb_backward_workspace_bytes(512, d, d, r);
      (void)lb_bits_per_weight(d, d, r, 2);
    }
    for (double b : {0.0, 0.1, 0.55, 1.0, 16.0, -1.0, double(NAN), double(INFINITY)}) (void)lb_rank_for_bpw(d, d, b, 16);
  }
  EXPECT(lb_rank_for_bpw(4096, 4096, 0.1, 16) == 80);
  // forward validation: every failing path returns before anything is enqueued
  lb_path paths[2] = {fake_path(), fake_path()};
  EXPECT(lb_linear_forward(fake_buf, static_cast<lb_dtype>(9), 4, 64, 64, 16, paths, LB_F16, fake_buf, fake_buf,
                           1 << 30, nullptr) == LB_ERR_DTYPE);
  EXPECT(lb_linear_forward(fake_buf, LB_BF16, -1, 64, 64, 16, paths, LB_F16, fake_buf, fake_buf, 1 << 30,
                           nullptr) == LB_ERR_SHAPE);
  EXPECT(lb_linear_forward(fake_buf, LB_BF16, 4, 64, 64, 16, nullptr, LB_F16, fake_buf, fake_buf, 1 << 30,
                           nullptr) == LB_ERR_NULL);
  EXPECT(lb_linear_forward(fake_buf + 1, LB_BF16, 4, 64, 64, 16, paths, LB_F16, fake_buf, fake_buf, 1 << 30,
                           nullptr) == LB_ERR_ALIGN);
  EXPECT(lb_linear_forward(fake_buf, LB_BF16, 4, 64, 64, 16, paths, LB_F16, fake_buf, fake_buf, 16, nullptr) ==
         LB_ERR_WORKSPACE);
  EXPECT(lb_linear_forward(fake_buf, LB_BF16, 0, 64, 64, 16, paths, LB_F16, fake_buf, fake_buf, 0, nullptr) ==
         LB_OK);
  EXPECT(lb_linear_forward_kernel(fake_buf, LB_BF16, 8, 64, 64, 16, paths, LB_F16, fake_buf, fake_buf, 1 << 30,
                                  LB_KERNEL_DECODE, nullptr) == LB_ERR_SHAPE);
  EXPECT(lb_workspace_status(nullptr, 256, reinterpret_cast<int32_t*>(fake_buf), nullptr) == LB_ERR_NULL);
  EXPECT(lb_workspace_status(fake_buf, 8, reinterpret_cast<int32_t*>(fake_buf), nullptr) == LB_ERR_WORKSPACE);
  // list validation over a long list (the overlap check is quadratic in n)
  std::vector<lb_linear_desc> descs(600);
  for (size_t i = 0; i < descs.size(); ++i) {
    lb_linear_desc& d = descs[i];
    d.x = fake_buf;
    d.act_dtype = LB_BF16;
    d.T = 1;
    d.d_in = 64;
    d.d_out = 64;
    d.r = 16;
    d.paths[0] = d.paths[1] = fake_path();
    d.scale_dtype = LB_F16;
    d.y = fake_buf + 128;  // every y overlaps every other: rejected
  }
  EXPECT(lb_forward_many_workspace_bytes(descs.data(), static_cast<int64_t>(descs.size())) > 0);
  EXPECT(lb_linear_forward_many(descs.data(), static_cast<int64_t>(descs.size()), fake_buf, size_t(1) << 40,
                                nullptr) == LB_ERR_ARG);
  descs[3].T = -1;
  EXPECT(lb_linear_forward_many(descs.data(), static_cast<int64_t>(descs.size()), fake_buf, size_t(1) << 40,
                                nullptr) == LB_ERR_SHAPE);
  EXPECT(lb_linear_forward_many(nullptr, 3, fake_buf, 256, nullptr) == LB_ERR_NULL);
  EXPECT(lb_linear_forward_many(descs.data(), -1, fake_buf, 256, nullptr) == LB_ERR_ARG);
  // pack, latent, backward and dense-reference validation
  EXPECT(lb_pack_signs(fake_buf, LB_F32, 64, 16, static_cast<lb_role>(5), fake_buf + 64, nullptr, nullptr) ==
         LB_ERR_ARG);
  EXPECT(lb_pack_signs(fake_buf, LB_F32, 64, 16, LB_ROLE_U, fake_buf + 64, nullptr, nullptr) == LB_ERR_ARG);
  EXPECT(lb_linear_latent(fake_buf, LB_BF16, 4, 64, 16, paths, LB_F16, fake_buf, static_cast<lb_dtype>(4), fake_buf,
                          1 << 20, nullptr) == LB_ERR_DTYPE);
  EXPECT(lb_linear_from_latent(fake_buf, LB_BF16, 4, 64, 16, nullptr, LB_F16, fake_buf, LB_BF16, fake_buf, 1 << 20,
                               nullptr) == LB_ERR_NULL);
  EXPECT(lb_linear_backward(fake_buf, fake_buf, LB_BF16, 4, 64, 64, 16, paths, LB_F16, nullptr, 100.0f, nullptr,
                            fake_buf, 1 << 20, nullptr) == LB_ERR_NULL);
  EXPECT(lb_linear_backward(fake_buf, fake_buf, LB_BF16, 4, 64, 64, 16, paths, LB_F16, nullptr, -1.0f, nullptr,
                            fake_buf, 1 << 20, nullptr) == LB_ERR_ARG);
  EXPECT(lb_dense_reference_weight(paths, LB_F16, 64, 70000, 16, reinterpret_cast<float*>(fake_buf), nullptr) ==
         LB_ERR_SHAPE);
}

static void oracle_checks() {
  const int64_t T = 3, d_in = 45, d_out = 37, r = 19;
  std::vector<double> x(T * d_in), lat_u(d_out * r), lat_v(d_in * r);
  std::vector<double> h[2], g[2], l[2];
  uint64_t s = 88172645463325252ull;
  auto rnd = [&]() {
    s ^= s << 13, s ^= s >> 7, s ^= s << 17;
    return static_cast<double>(s % 2000001) / 1e6 - 1.0;
  };
  for (auto& v : x) v = rnd();
  std::vector<int8_t> U[2], V[2];
  for (int p = 0; p < 2; ++p) {
    for (auto& v : lat_u) v = rnd();
    for (auto& v : lat_v) v = rnd();
    std::vector<uint8_t> bu(lbo_packed_bytes(d_out, r, 0)), bv(lbo_packed_bytes(d_in, r, 1));
    EXPECT(lbo_pack(lat_u.data(), d_out, r, 0, bu.data()) == 0);
    EXPECT(lbo_pack(lat_v.data(), d_in, r, 1, bv.data()) == 0);
    U[p].resize(d_out * r);
    V[p].resize(d_in * r);
    lbo_unpack(bu.data(), d_out, r, 0, U[p].data());
    lbo_unpack(bv.data(), d_in, r, 1, V[p].data());
    for (int64_t i = 0; i < d_out * r; ++i) EXPECT(U[p][i] == (lat_u[i] < 0 ? -1 : 1));
    h[p].resize(d_out), g[p].resize(d_in), l[p].resize(r);
    for (auto& v : h[p]) v = rnd();
    for (auto& v : g[p]) v = rnd();
    for (auto& v : l[p]) v = rnd();
  }
  const int8_t* Up[2] = {U[0].data(), U[1].data()};
  const int8_t* Vp[2] = {V[0].data(), V[1].data()};
  const double* hp[2] = {h[0].data(), h[1].data()};
  const double* gp[2] = {g[0].data(), g[1].data()};
  const double* lp[2] = {l[0].data(), l[1].data()};
  std::vector<double> y1(T * d_out), y2(T * d_out), y3(T * d_out), W(d_out * d_in), w(2 * T * r);
  lbo_forward_factored(x.data(), T, d_in, d_out, r, Up, Vp, hp, gp, lp, 2, y1.data());
  lbo_forward_factored_par(x.data(), T, d_in, d_out, r, Up, Vp, hp, gp, lp, 2, 3, y2.data());
  EXPECT(std::memcmp(y1.data(), y2.data(), sizeof(double) * y1.size()) == 0);
  lbo_latent(x.data(), T, d_in, r, Vp, gp, lp, 2, w.data());
  lbo_from_latent(w.data(), T, d_out, r, Up, hp, 2, y3.data());
  EXPECT(std::memcmp(y1.data(), y3.data(), sizeof(double) * y1.size()) == 0);
  lbo_dense_weight(d_in, d_out, r, Up, Vp, hp, gp, lp, 2, W.data());
  for (int64_t t = 0; t < T; ++t)
    for (int64_t i = 0; i < d_out; ++i) {
      double acc = 0.0;
      for (int64_t j = 0; j < d_in; ++j) acc += W[i * d_in + j] * x[t * d_in + j];
      EXPECT(std::fabs(acc - y1[t * d_out + i]) <= 1e-12 * (1.0 + std::fabs(acc)));
    }
}

int main() {
  abi_checks();
  oracle_checks();
  if (failures) {
    std::fprintf(stderr, "%d check(s) failed\n", failures);
    return 1;
  }
  std::printf("sanitized host checks passed\n");
  return 0;
}
