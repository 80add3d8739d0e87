// C ABI of the LittleBit library: host-side validation, dispatch and launch.
// Every argument is checked before anything touches HIP, so every error path
// is testable without a GPU; nothing here allocates device memory.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <vector>

#include "lb_backward.h"
#include "lb_latent.h"

namespace {

constexpr int64_t kMaxElems = (int64_t(1) << 31) - 1;

// The value of an enum argument as an int, read without an enum-typed load: C
// callers may pass any int, and a value outside an enum's range must reach
// the range checks below, not be read as the enum first.
template <typename E>
int enum_value(const E& e) {
  static_assert(sizeof(E) == sizeof(int), "enums of the ABI are int-sized");
  int v;
  std::memcpy(&v, &e, sizeof v);
  return v;
}

bool dtype_ok(const lb_dtype& d) {
  const int v = enum_value(d);
  return v == LB_F32 || v == LB_F16 || v == LB_BF16;
}
bool role_ok(const lb_role& r) {
  const int v = enum_value(r);
  return v == LB_ROLE_U || v == LB_ROLE_V;
}
bool kernel_ok(const lb_kernel& k) {
  const int v = enum_value(k);
  return v == LB_KERNEL_AUTO || v == LB_KERNEL_DECODE || v == LB_KERNEL_PREFILL || v == LB_KERNEL_DECODE_MFMA;
}
size_t dtype_size(lb_dtype d) { return d == LB_F32 ? 4 : 2; }
bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

size_t packed_bytes(int64_t n_out, int64_t n_red) {
  const int64_t nb = n_red / 32, w = n_red - 32 * nb;
  const int64_t tail = w == 0 ? 0 : (w <= 16 ? 2 : 4);
  return static_cast<size_t>(4 * nb * n_out + tail * n_out);
}

bool fits(int64_t a, int64_t b) { return a == 0 || b <= kMaxElems / a; }

lb_status check_sizes(int64_t T, int64_t d_in, int64_t d_out, int64_t r) {
  if (T < 0 || d_in < 0 || d_out < 0 || r < 0) return LB_ERR_SHAPE;
  if (!fits(T, d_in) || !fits(T, d_out) || !fits(d_in, r) || !fits(d_out, r) || !fits(2 * T, r))
    return LB_ERR_SHAPE;
  return LB_OK;
}

// with_l / with_u: l / U are read (l by every call but the from-latent one,
// U by every call but the backward)
lb_status check_paths(const lb_path* paths, lb_dtype sc, int64_t d_in, int64_t d_out, int64_t r,
                      bool with_l = true, bool with_u = true) {
  if (!paths) return LB_ERR_NULL;
  const size_t es = dtype_size(sc);
  for (int p = 0; p < 2; ++p) {
    const lb_path& P = paths[p];
    if ((with_u && r > 0 && d_out > 0 && !P.U) || (r > 0 && d_in > 0 && !P.V) || (d_out > 0 && !P.h) ||
        (d_in > 0 && !P.g) || (with_l && r > 0 && !P.l))
      return LB_ERR_NULL;
    if (!aligned(P.U, 4) || !aligned(P.V, 4) || !aligned(P.h, es) || !aligned(P.g, es) || !aligned(P.l, es))
      return LB_ERR_ALIGN;
  }
  return LB_OK;
}

lb::ForwardArgs make_args(const void* x, lb_dtype act, int64_t T, int64_t d_in, int64_t d_out, int64_t r,
                          const lb_path* paths, lb_dtype sc, void* y, void* ws, size_t ws_bytes) {
  lb::ForwardArgs a{};
  a.x = x;
  a.act_dt = act;
  a.T = static_cast<int>(T);
  a.d_in = static_cast<int>(d_in);
  a.d_out = static_cast<int>(d_out);
  a.r = static_cast<int>(r);
  for (int p = 0; p < 2; ++p) {
    a.U[p] = paths[p].U;
    a.V[p] = paths[p].V;
    a.h[p] = paths[p].h;
    a.g[p] = paths[p].g;
    a.l[p] = paths[p].l;
  }
  a.sc_dt = sc;
  a.y = y;
  a.ws = ws;
  a.ws_bytes = ws_bytes;
  return a;
}

constexpr int64_t kAutoLutTokens = 2;  // AUTO sends T <= this to the look-up-table decode kernel

// AUTO between the matrix-core decode kernel and the prefill kernels: the
// decode kernel's single launch wins while T r d_out is small; the prefill
// kernels' cost barely grows with T up to one 64-token tile.  Thresholds from
// timings of both kernels on the Llama2-7B and -70B linear shapes (0.1 and
// 0.55 bits per weight, T = 4 .. 64).
bool prefer_prefill(int64_t T, int64_t d_out, int64_t r) {
  const int64_t rd = r * d_out;
  return T >= 32 || (T >= 16 && rd >= 3000000) || rd >= 8000000;
}

// The kernel AUTO runs for a linear with work (T, d_in, d_out, r >= 1), or
// LB_KERNEL_AUTO itself when no kernel takes the sizes.
lb_kernel auto_kernel(int64_t T, int64_t d_in, int64_t d_out, int64_t r) {
  if (T <= kAutoLutTokens && lb::decode_supports(T, d_in, d_out, r)) return LB_KERNEL_DECODE;
  const bool pf = lb::prefill_supports(T, d_in, d_out, r);
  if (lb::decode_mma_supports(T, d_in, d_out, r) && !(prefer_prefill(T, d_out, r) && pf))
    return LB_KERNEL_DECODE_MFMA;
  return pf ? LB_KERNEL_PREFILL : LB_KERNEL_AUTO;
}

}  // namespace

extern "C" {

int lb_abi_version(void) { return LB_ABI_VERSION; }

const char* lb_status_str(lb_status s) {
  switch (enum_value(s)) {
    case LB_OK: return "LB_OK";
    case LB_ERR_NULL: return "LB_ERR_NULL";
    case LB_ERR_SHAPE: return "LB_ERR_SHAPE";
    case LB_ERR_DTYPE: return "LB_ERR_DTYPE";
    case LB_ERR_ALIGN: return "LB_ERR_ALIGN";
    case LB_ERR_WORKSPACE: return "LB_ERR_WORKSPACE";
    case LB_ERR_HIP: return "LB_ERR_HIP";
    case LB_ERR_ARG: return "LB_ERR_ARG";
  }
  return "LB_ERR_UNKNOWN";
}

size_t lb_packed_bytes(lb_role role, int64_t rows, int64_t r) {
  if (rows < 0 || r < 0 || !role_ok(role)) return 0;
  return role == LB_ROLE_U ? packed_bytes(rows, r) : packed_bytes(r, rows);
}

double lb_bits_per_weight(int64_t d_in, int64_t d_out, int64_t r, int npaths) {
  if (d_in <= 0 || d_out <= 0 || r < 0 || (npaths != 1 && npaths != 2)) return -1.0;
  // per path: 1 bit per element of U_sign [d_out x r] and V_sign [d_in x r],
  // 16 bits per element of h [d_out], g [d_in], l [r]
  const double per_path = double(d_out) * r + double(d_in) * r + 16.0 * (double(d_out) + double(d_in) + r);
  return npaths * per_path / (double(d_in) * double(d_out));
}

int64_t lb_rank_for_bpw(int64_t d_in, int64_t d_out, double bpw, int64_t mult) {
  if (d_in <= 0 || d_out <= 0 || mult < 1 || !(bpw >= 0.0) || !std::isfinite(bpw)) return -1;
  const double budget = bpw * double(d_in) * double(d_out);
  // total bits 2 r (d_in + d_out) + 32 (d_in + d_out) + 32 r is increasing in r
  const double s = double(d_in) + double(d_out);
  const double r_real = (budget - 32.0 * s) / (2.0 * s + 32.0);
  if (r_real < mult) return 0;
  int64_t r = static_cast<int64_t>(std::floor(r_real / mult)) * mult;
  auto bits = [&](int64_t rr) { return 2.0 * rr * s + 32.0 * s + 32.0 * rr; };
  while (r > 0 && bits(r) > budget) r -= mult;
  while (bits(r + mult) <= budget) r += mult;
  return r;
}

lb_status lb_pack_signs(const void* src, lb_dtype src_dtype, int64_t rows, int64_t r, lb_role role, void* dst,
                        int32_t* nan_count, hipStream_t stream) {
  if (!role_ok(role)) return LB_ERR_ARG;
  if (!dtype_ok(src_dtype)) return LB_ERR_DTYPE;
  if (rows < 0 || r < 0 || !fits(rows, r)) return LB_ERR_SHAPE;
  if (rows == 0 || r == 0) return LB_OK;
  if (!src || !dst) return LB_ERR_NULL;
  if (!aligned(src, dtype_size(src_dtype)) || !aligned(dst, 4) || !aligned(nan_count, 4)) return LB_ERR_ALIGN;
  const size_t nbytes = lb_packed_bytes(role, rows, r);
  const char* s = static_cast<const char*>(src);
  const char* d = static_cast<const char*>(dst);
  const size_t sbytes = static_cast<size_t>(rows * r) * dtype_size(src_dtype);
  if (d < s + sbytes && s < d + nbytes) return LB_ERR_ARG;  // overlapping buffers
  const hipError_t e = lb::launch_pack(src, src_dtype, static_cast<int>(rows), static_cast<int>(r), role, dst,
                                       nan_count, stream);
  return e == hipSuccess ? LB_OK : LB_ERR_HIP;
}

int64_t lb_decode_max_tokens(void) { return lb::kDecodeMaxTokens; }

size_t lb_forward_workspace_bytes(int64_t T, int64_t d_in, int64_t d_out, int64_t r) {
  if (check_sizes(T, d_in, d_out, r) != LB_OK) return 0;
  size_t need = lb::kCtrlBytes;
  const int iT = static_cast<int>(T), ii = static_cast<int>(d_in), io = static_cast<int>(d_out),
            ir = static_cast<int>(r);
  if (lb::decode_supports(T, d_in, d_out, r)) {
    const lb::DecodeGeom g = lb::decode_geometry(iT, ii, io, ir);
    if (g.ws_bytes > need) need = g.ws_bytes;
  }
  if (lb::decode_mma_supports(T, d_in, d_out, r)) {
    // the geometry depends on the activation dtype: cover all of them
    for (int dt : {lb::kDtF32, lb::kDtF16, lb::kDtBF16}) {
      const lb::MmaGeom g = lb::decode_mma_geometry(iT, ii, io, ir, dt);
      if (g.ws_bytes > need) need = g.ws_bytes;
    }
  }
  const lb::PrefillGeom pg = lb::prefill_geometry(iT, ii, io, ir);
  if (pg.ws_bytes > need) need = pg.ws_bytes;
  return need;
}

lb_status lb_workspace_init(void* workspace, size_t bytes, hipStream_t stream) {
  if (bytes == 0) return LB_OK;
  if (!workspace) return LB_ERR_NULL;
  if (!aligned(workspace, 256) || bytes % 4 != 0) return LB_ERR_ALIGN;
  return lb::launch_fill_zero(workspace, bytes, stream) == hipSuccess ? LB_OK : LB_ERR_HIP;
}

lb_status lb_workspace_status(void* workspace, size_t workspace_bytes, int32_t* status, hipStream_t stream) {
  if (!workspace || !status) return LB_ERR_NULL;
  if (!aligned(workspace, 256) || !aligned(status, 4)) return LB_ERR_ALIGN;
  if (workspace_bytes < lb::kCtrlBytes) return LB_ERR_WORKSPACE;
  const hipError_t e = lb::launch_take_status(static_cast<uint32_t*>(workspace), status, stream);
  return e == hipSuccess ? LB_OK : LB_ERR_HIP;
}

lb_status lb_linear_forward_kernel(const void* x, lb_dtype act_dtype, int64_t T, int64_t d_in, int64_t d_out,
                                   int64_t r, const lb_path* paths, lb_dtype scale_dtype, void* y, void* workspace,
                                   size_t workspace_bytes, lb_kernel kernel, hipStream_t stream) {
  if (!kernel_ok(kernel)) return LB_ERR_ARG;
  if (!dtype_ok(act_dtype) || !dtype_ok(scale_dtype)) return LB_ERR_DTYPE;
  lb_status st = check_sizes(T, d_in, d_out, r);
  if (st != LB_OK) return st;
  if (kernel == LB_KERNEL_DECODE && !lb::decode_supports(T, d_in, d_out, r)) return LB_ERR_SHAPE;
  if (kernel == LB_KERNEL_DECODE_MFMA && !lb::decode_mma_supports(T, d_in, d_out, r)) return LB_ERR_SHAPE;
  if (kernel == LB_KERNEL_PREFILL && !lb::prefill_supports(T, d_in, d_out, r)) return LB_ERR_SHAPE;
  if (T == 0 || d_out == 0) return LB_OK;
  if (!y || (d_in > 0 && !x)) return LB_ERR_NULL;
  if (!aligned(x, dtype_size(act_dtype)) || !aligned(y, dtype_size(act_dtype))) return LB_ERR_ALIGN;
  st = check_paths(paths, scale_dtype, d_in, d_out, r);
  if (st != LB_OK) return st;
  const size_t need = lb_forward_workspace_bytes(T, d_in, d_out, r);
  if (!workspace) return LB_ERR_NULL;
  if (!aligned(workspace, 256)) return LB_ERR_ALIGN;
  if (workspace_bytes < need) return LB_ERR_WORKSPACE;
  lb::ForwardArgs a = make_args(x, act_dtype, T, d_in, d_out, r, paths, scale_dtype, y, workspace, workspace_bytes);
  hipError_t e;
  if (d_in == 0 || r == 0) {
    // empty reduction: y = 0 (Proposition 1 with an empty sum)
    e = lb::launch_zero_elems(y, T * d_out, act_dtype, stream);
    return e == hipSuccess ? LB_OK : LB_ERR_HIP;
  }
  if (kernel == LB_KERNEL_AUTO) {
    // the look-up-table kernel is the fastest for one or two tokens; from
    // three on the matrix-core decode kernel, then the prefill kernels
    kernel = auto_kernel(T, d_in, d_out, r);
    if (kernel == LB_KERNEL_AUTO) return LB_ERR_SHAPE;
  }
  if (kernel == LB_KERNEL_DECODE)
    e = lb::launch_decode(a, lb::decode_geometry(a.T, a.d_in, a.d_out, a.r), stream);
  else if (kernel == LB_KERNEL_DECODE_MFMA)
    e = lb::launch_decode_mma(a, lb::decode_mma_geometry(a.T, a.d_in, a.d_out, a.r, a.act_dt), stream);
  else
    e = lb::launch_prefill(a, lb::prefill_geometry(a.T, a.d_in, a.d_out, a.r), stream);
  return e == hipSuccess ? LB_OK : LB_ERR_HIP;
}

lb_status lb_linear_forward(const void* x, lb_dtype act_dtype, int64_t T, int64_t d_in, int64_t d_out, int64_t r,
                            const lb_path* paths, lb_dtype scale_dtype, void* y, void* workspace,
                            size_t workspace_bytes, hipStream_t stream) {
  if (!dtype_ok(act_dtype) || !dtype_ok(scale_dtype)) return LB_ERR_DTYPE;  // before passing them on
  return lb_linear_forward_kernel(x, act_dtype, T, d_in, d_out, r, paths, scale_dtype, y, workspace,
                                  workspace_bytes, LB_KERNEL_AUTO, stream);
}

}  // extern "C"

namespace {

// Workspace of lb_linear_forward_noalloc: a file-scope device array, one copy
// per GPU, held until the process ends.  Host code never uses the array's
// name as an address: each device's copy is resolved once with
// hipGetSymbolAddress (that device current) and that pointer is what the
// kernels get.
constexpr size_t kNoAllocScratchBytes = size_t(32) << 20;
__device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
struct ScratchSlot {
  std::mutex mu;
  bool ready = false;
  void* ptr = nullptr;
};
ScratchSlot g_scratch[kMaxDevices];

// The current device's scratch, resolved and zero-filled (by a fill kernel on
// `stream`, before the call that needs it) on its first use.  The first use
// on a device must not be captured in a graph (LB_ERR_ARG): its zero fill
// must run before every later call, captured or not.
lb_status scratch_for_current_device(hipStream_t stream, void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return LB_ERR_HIP;
  ScratchSlot& s = g_scratch[dev];
  std::lock_guard<std::mutex> lock(s.mu);
  if (!s.ready) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(stream, &cs) != hipSuccess) return LB_ERR_HIP;
    if (cs != hipStreamCaptureStatusNone) return LB_ERR_ARG;
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) return LB_ERR_HIP;
    if (lb::launch_fill_zero(ptr, kNoAllocScratchBytes, stream) != hipSuccess) return LB_ERR_HIP;
    s.ptr = ptr;
    s.ready = true;
  }
  *out = s.ptr;
  return LB_OK;
}

}  // namespace

extern "C" {

size_t lb_noalloc_scratch_bytes(void) { return kNoAllocScratchBytes; }

lb_status lb_linear_forward_noalloc(const void* x, lb_dtype act_dtype, int64_t T, int64_t d_in, int64_t d_out,
                                    int64_t r, const lb_path* paths, lb_dtype scale_dtype, void* y,
                                    hipStream_t stream) {
  if (!dtype_ok(act_dtype) || !dtype_ok(scale_dtype)) return LB_ERR_DTYPE;
  const lb_status st = check_sizes(T, d_in, d_out, r);
  if (st != LB_OK) return st;
  if (lb_forward_workspace_bytes(T, d_in, d_out, r) > kNoAllocScratchBytes) return LB_ERR_WORKSPACE;
  if (T == 0 || d_out == 0) return LB_OK;
  if (!y || (d_in > 0 && !x)) return LB_ERR_NULL;
  if (!aligned(x, dtype_size(act_dtype)) || !aligned(y, dtype_size(act_dtype))) return LB_ERR_ALIGN;
  const lb_status sp = check_paths(paths, scale_dtype, d_in, d_out, r);
  if (sp != LB_OK) return sp;
  void* ws = nullptr;
  const lb_status ss = scratch_for_current_device(stream, &ws);
  if (ss != LB_OK) return ss;
  return lb_linear_forward_kernel(x, act_dtype, T, d_in, d_out, r, paths, scale_dtype, y, ws, kNoAllocScratchBytes,
                                  LB_KERNEL_AUTO, stream);
}

namespace {

size_t align256(size_t b) { return (b + 255) / 256 * 256; }

// the checks of lb_linear_forward_kernel before its workspace checks
lb_status check_forward(const lb_linear_desc& d) {
  if (!dtype_ok(d.act_dtype) || !dtype_ok(d.scale_dtype)) return LB_ERR_DTYPE;
  const lb_status st = check_sizes(d.T, d.d_in, d.d_out, d.r);
  if (st != LB_OK) return st;
  if (d.T == 0 || d.d_out == 0) return LB_OK;
  if (!d.y || (d.d_in > 0 && !d.x)) return LB_ERR_NULL;
  if (!aligned(d.x, dtype_size(d.act_dtype)) || !aligned(d.y, dtype_size(d.act_dtype))) return LB_ERR_ALIGN;
  return check_paths(d.paths, d.scale_dtype, d.d_in, d.d_out, d.r);
}

bool has_work(const lb_linear_desc& d) { return d.T > 0 && d.d_out > 0 && d.d_in > 0 && d.r > 0; }

// a linear with work that no kernel of the automatic choice takes
bool auto_unsupported(const lb_linear_desc& d) {
  return has_work(d) && auto_kernel(d.T, d.d_in, d.d_out, d.r) == LB_KERNEL_AUTO;
}

// the list launch a linear joins: the look-up-table or the matrix-core decode
// kernel (what AUTO runs for it), or none (a call of its own)
lb_kernel list_kernel(const lb_linear_desc& d) {
  if (!has_work(d)) return LB_KERNEL_AUTO;
  const lb_kernel k = auto_kernel(d.T, d.d_in, d.d_out, d.r);
  return k == LB_KERNEL_DECODE || k == LB_KERNEL_DECODE_MFMA ? k : LB_KERNEL_AUTO;
}

size_t slice_bytes(const lb_linear_desc& d) {
  return align256(lb_forward_workspace_bytes(d.T, d.d_in, d.d_out, d.r));
}

bool overlap(const void* a, size_t na, const void* b, size_t nb) {
  if (na == 0 || nb == 0) return false;
  const uintptr_t pa = reinterpret_cast<uintptr_t>(a), pb = reinterpret_cast<uintptr_t>(b);
  return pa < pb + nb && pb < pa + na;
}

}  // namespace

size_t lb_forward_many_workspace_bytes(const lb_linear_desc* descs, int64_t n) {
  if (n <= 0 || !descs) return 0;
  size_t need = lb::kListHdrBytes;
  for (int64_t i = 0; i < n; ++i) {
    if (check_sizes(descs[i].T, descs[i].d_in, descs[i].d_out, descs[i].r) != LB_OK) return 0;
    need += slice_bytes(descs[i]);
  }
  return need;
}

lb_status lb_linear_forward_many(const lb_linear_desc* descs, int64_t n, void* workspace, size_t workspace_bytes,
                                 hipStream_t stream) {
  if (n < 0) return LB_ERR_ARG;
  if (n == 0) return LB_OK;
  if (!descs) return LB_ERR_NULL;
  for (int64_t i = 0; i < n; ++i) {
    const lb_status st = check_forward(descs[i]);
    if (st != LB_OK) return st;
    if (auto_unsupported(descs[i])) return LB_ERR_SHAPE;
  }
  // the linears run concurrently: no output may overlap another linear's
  // input or output
  for (int64_t i = 0; i < n; ++i) {
    const lb_linear_desc& a = descs[i];
    const size_t ny = static_cast<size_t>(a.T * a.d_out) * dtype_size(a.act_dtype);
    for (int64_t j = 0; j < n; ++j) {
      if (j == i) continue;
      const lb_linear_desc& b = descs[j];
      const size_t es = dtype_size(b.act_dtype);
      if (overlap(a.y, ny, b.y, static_cast<size_t>(b.T * b.d_out) * es) ||
          overlap(a.y, ny, b.x, static_cast<size_t>(b.T * b.d_in) * es))
        return LB_ERR_ARG;
    }
  }
  const size_t need = lb_forward_many_workspace_bytes(descs, n);
  if (!workspace) return LB_ERR_NULL;
  if (!aligned(workspace, 256)) return LB_ERR_ALIGN;
  if (workspace_bytes < need) return LB_ERR_WORKSPACE;

  // runs of linears that one decode kernel takes, of one dtype pair, go out
  // as list launches of up to kDecodeMaxBatch; every other linear as its own
  // call
  lb::ForwardArgs batch[lb::kDecodeMaxBatch];
  int nb = 0;
  lb_kernel bk = LB_KERNEL_AUTO;
  auto flush = [&]() -> lb_status {
    if (nb == 0) return LB_OK;
    const lb::ForwardArgs& a0 = batch[0];
    hipError_t e;
    if (bk == LB_KERNEL_DECODE)
      e = nb == 1 ? lb::launch_decode(a0, lb::decode_geometry(a0.T, a0.d_in, a0.d_out, a0.r), stream)
                  : lb::launch_decode_batch(batch, nb, stream);
    else
      e = nb == 1 ? lb::launch_decode_mma(a0, lb::decode_mma_geometry(a0.T, a0.d_in, a0.d_out, a0.r, a0.act_dt),
                                          stream)
                  : lb::launch_decode_mma_batch(batch, nb, stream);
    nb = 0;
    return e == hipSuccess ? LB_OK : LB_ERR_HIP;
  };
  char* ws = static_cast<char*>(workspace);
  size_t off = lb::kListHdrBytes;
  for (int64_t i = 0; i < n; ++i) {
    const lb_linear_desc& d = descs[i];
    const size_t sb = slice_bytes(d);
    const lb_kernel k = list_kernel(d);
    if (k != LB_KERNEL_AUTO) {
      if (nb > 0 && (nb == lb::kDecodeMaxBatch || k != bk || static_cast<int>(d.act_dtype) != batch[0].act_dt ||
                     static_cast<int>(d.scale_dtype) != batch[0].sc_dt)) {
        const lb_status st = flush();
        if (st != LB_OK) return st;
      }
      bk = k;
      batch[nb] = make_args(d.x, d.act_dtype, d.T, d.d_in, d.d_out, d.r, d.paths, d.scale_dtype, d.y, ws + off, sb);
      // one control block for the whole list: the start of its workspace
      batch[nb++].ctrl = workspace;
    } else {
      const lb_status st = lb_linear_forward_kernel(d.x, d.act_dtype, d.T, d.d_in, d.d_out, d.r, d.paths,
                                                    d.scale_dtype, d.y, ws + off, sb, LB_KERNEL_AUTO, stream);
      if (st != LB_OK) return st;
    }
    off += sb;
  }
  return flush();
}

namespace {

// FNV-1a over the fields of the descriptors (not their bytes: padding is not
// part of a descriptor's value)
struct Fnv {
  uint64_t h = 1469598103934665603ull;
  void add(uint64_t v) {
    for (int i = 0; i < 8; ++i) {
      h ^= (v >> (8 * i)) & 0xffu;
      h *= 1099511628211ull;
    }
  }
  void add(const void* p) { add(static_cast<uint64_t>(reinterpret_cast<uintptr_t>(p))); }
};

uint64_t list_fingerprint(const lb_linear_desc* descs, int64_t n) {
  Fnv f;
  f.add(static_cast<uint64_t>(n));
  for (int64_t i = 0; i < n; ++i) {
    const lb_linear_desc& d = descs[i];
    f.add(d.x);
    f.add(d.y);
    f.add(static_cast<uint64_t>(enum_value(d.act_dtype)));
    f.add(static_cast<uint64_t>(enum_value(d.scale_dtype)));
    f.add(static_cast<uint64_t>(d.T));
    f.add(static_cast<uint64_t>(d.d_in));
    f.add(static_cast<uint64_t>(d.d_out));
    f.add(static_cast<uint64_t>(d.r));
    for (int p = 0; p < 2; ++p) {
      f.add(d.paths[p].U);
      f.add(d.paths[p].V);
      f.add(d.paths[p].h);
      f.add(d.paths[p].g);
      f.add(d.paths[p].l);
    }
  }
  return f.h;
}

// Outputs of a list overlap nothing the list reads or writes, in O(n log n):
// the y ranges sorted by start must be disjoint, and no x range may meet one.
bool list_outputs_disjoint(const lb_linear_desc* descs, int64_t n) {
  struct Range {
    uintptr_t lo, hi;
    int64_t who;
  };
  std::vector<Range> ys, xs;
  for (int64_t i = 0; i < n; ++i) {
    const lb_linear_desc& d = descs[i];
    const size_t es = dtype_size(d.act_dtype);
    const size_t ny = static_cast<size_t>(d.T * d.d_out) * es, nx = static_cast<size_t>(d.T * d.d_in) * es;
    if (ny > 0) ys.push_back({reinterpret_cast<uintptr_t>(d.y), reinterpret_cast<uintptr_t>(d.y) + ny, i});
    if (nx > 0) xs.push_back({reinterpret_cast<uintptr_t>(d.x), reinterpret_cast<uintptr_t>(d.x) + nx, i});
  }
  std::sort(ys.begin(), ys.end(), [](const Range& a, const Range& b) { return a.lo < b.lo; });
  for (size_t k = 1; k < ys.size(); ++k)
    if (ys[k].lo < ys[k - 1].hi) return false;
  for (const Range& x : xs) {
    // the first y starting at or after x.lo, and the one before it
    // (a linear's y may overlap its own x: its output is written after its
    // input has been read; the ys are disjoint, so the walk below stops at
    // the first other y inside x)
    auto it = std::lower_bound(ys.begin(), ys.end(), x.lo, [](const Range& a, uintptr_t v) { return a.lo < v; });
    if (it != ys.begin() && (it - 1)->hi > x.lo && (it - 1)->who != x.who) return false;
    for (; it != ys.end() && it->lo < x.hi; ++it)
      if (it->who != x.who) return false;
  }
  return true;
}

// the validation lb_list_* share; on success fills args (one per descriptor)
lb_status list_check(const lb_linear_desc* descs, int64_t n, std::vector<lb::ForwardArgs>& args) {
  if (n < 0 || n > 65535) return LB_ERR_ARG;
  if (n > 0 && !descs) return LB_ERR_NULL;
  int act = -1, sc = -1;
  args.clear();
  for (int64_t i = 0; i < n; ++i) {
    const lb_linear_desc& d = descs[i];
    const lb_status st = check_forward(d);
    if (st != LB_OK) return st;
    lb::ForwardArgs a = make_args(d.x, d.act_dtype, d.T, d.d_in, d.d_out, d.r, d.paths, d.scale_dtype, d.y, nullptr, 0);
    if (d.T > 0 && d.d_out > 0 && d.d_in > 0 && d.r > 0) {
      if (!lb::stream_supports(a)) return LB_ERR_SHAPE;
      if (act < 0) act = a.act_dt, sc = a.sc_dt;
      if (a.act_dt != act || a.sc_dt != sc) return LB_ERR_DTYPE;
    }
    args.push_back(a);
  }
  if (!lb::stream_list_supports(args.data(), static_cast<int>(n))) return LB_ERR_SHAPE;
  if (!list_outputs_disjoint(descs, n)) return LB_ERR_ARG;
  return LB_OK;
}

}  // namespace

size_t lb_list_workspace_bytes(const lb_linear_desc* descs, int64_t n) {
  std::vector<lb::ForwardArgs> args;
  if (list_check(descs, n, args) != LB_OK) return 0;
  return lb::stream_workspace_bytes(args.data(), static_cast<int>(n));
}

lb_status lb_list_init(const lb_linear_desc* descs, int64_t n, void* workspace, size_t workspace_bytes,
                       hipStream_t stream) {
  std::vector<lb::ForwardArgs> args;
  lb_status st = list_check(descs, n, args);
  if (st != LB_OK) return st;
  const size_t need = lb::stream_workspace_bytes(args.data(), static_cast<int>(n));
  if (!workspace) return LB_ERR_NULL;
  if (!aligned(workspace, 256)) return LB_ERR_ALIGN;
  if (workspace_bytes < need) return LB_ERR_WORKSPACE;
  const hipError_t e =
      lb::stream_init(args.data(), static_cast<int>(n), list_fingerprint(descs, n), workspace, stream);
  return e == hipSuccess ? LB_OK : LB_ERR_HIP;
}

lb_status lb_list_forward(const lb_linear_desc* descs, int64_t n, void* workspace, size_t workspace_bytes,
                          hipStream_t stream) {
  std::vector<lb::ForwardArgs> args;
  lb_status st = list_check(descs, n, args);
  if (st != LB_OK) return st;
  const size_t need = lb::stream_workspace_bytes(args.data(), static_cast<int>(n));
  if (!workspace) return LB_ERR_NULL;
  if (!aligned(workspace, 256)) return LB_ERR_ALIGN;
  if (workspace_bytes < need) return LB_ERR_WORKSPACE;
  hipError_t e = hipSuccess;
  // linears with an empty reduction: y = 0
  for (int64_t i = 0; i < n && e == hipSuccess; ++i) {
    const lb_linear_desc& d = descs[i];
    if (d.T > 0 && d.d_out > 0 && (d.d_in == 0 || d.r == 0))
      e = lb::launch_zero_elems(d.y, d.T * d.d_out, d.act_dtype, stream);
  }
  if (e == hipSuccess)
    e = lb::stream_forward(args.data(), static_cast<int>(n), list_fingerprint(descs, n), workspace, stream);
  return e == hipSuccess ? LB_OK : LB_ERR_HIP;
}

size_t lb_latent_workspace_bytes(int64_t T, int64_t d_in, int64_t r) {
  if (check_sizes(T, d_in, 0, r) != LB_OK || !lb::latent_supports(T, d_in, r)) return 0;
  return lb::latent_workspace_bytes(static_cast<int>(T), static_cast<int>(d_in), static_cast<int>(r));
}

lb_status lb_linear_latent(const void* x, lb_dtype act_dtype, int64_t T, int64_t d_in, int64_t r,
                           const lb_path* paths, lb_dtype scale_dtype, void* w, lb_dtype latent_dtype,
                           void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (!dtype_ok(act_dtype) || !dtype_ok(scale_dtype) || !dtype_ok(latent_dtype)) return LB_ERR_DTYPE;
  lb_status st = check_sizes(T, d_in, 0, r);
  if (st != LB_OK) return st;
  if (!lb::latent_supports(T, d_in, r)) return LB_ERR_SHAPE;
  if (T == 0 || r == 0) return LB_OK;
  if (!w || (d_in > 0 && !x)) return LB_ERR_NULL;
  if (!aligned(x, dtype_size(act_dtype)) || !aligned(w, dtype_size(latent_dtype))) return LB_ERR_ALIGN;
  if (!paths) return LB_ERR_NULL;
  // only V, g and l are read
  lb_path used[2];
  for (int p = 0; p < 2; ++p) used[p] = lb_path{nullptr, paths[p].V, nullptr, paths[p].g, paths[p].l};
  st = check_paths(used, scale_dtype, d_in, 0, r);
  if (st != LB_OK) return st;
  const size_t nw = static_cast<size_t>(2 * T * r) * dtype_size(latent_dtype);
  if (overlap(w, nw, x, static_cast<size_t>(T * d_in) * dtype_size(act_dtype))) return LB_ERR_ARG;
  const size_t need = lb_latent_workspace_bytes(T, d_in, r);
  if (!workspace) return LB_ERR_NULL;
  if (!aligned(workspace, 256)) return LB_ERR_ALIGN;
  if (workspace_bytes < need) return LB_ERR_WORKSPACE;
  hipError_t e;
  if (d_in == 0) {
    // empty reduction: every latent is zero
    e = lb::launch_zero_elems(w, 2 * T * r, latent_dtype, stream);
  } else {
    lb::ForwardArgs a = make_args(x, act_dtype, T, d_in, 0, r, used, scale_dtype, w, workspace, workspace_bytes);
    // a decoding step's few tokens: one launch; otherwise the prefill stage 1
    e = lb::latent_small_supports(T, d_in, r) ? lb::launch_latent_small(a, latent_dtype, stream)
                                              : lb::launch_latent(a, latent_dtype, stream);
  }
  return e == hipSuccess ? LB_OK : LB_ERR_HIP;
}

size_t lb_from_latent_workspace_bytes(int64_t T, int64_t r) {
  if (check_sizes(T, 0, 0, r) != LB_OK || !lb::from_latent_supports(T, 0, r)) return 0;
  return lb::from_latent_workspace_bytes(static_cast<int>(T), static_cast<int>(r));
}

lb_status lb_linear_from_latent(const void* w, lb_dtype latent_dtype, int64_t T, int64_t d_out, int64_t r,
                                const lb_path* paths, lb_dtype scale_dtype, void* y, lb_dtype out_dtype,
                                void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (!dtype_ok(latent_dtype) || !dtype_ok(scale_dtype) || !dtype_ok(out_dtype)) return LB_ERR_DTYPE;
  lb_status st = check_sizes(T, 0, d_out, r);
  if (st != LB_OK) return st;
  if (!lb::from_latent_supports(T, d_out, r)) return LB_ERR_SHAPE;
  if (T == 0 || d_out == 0) return LB_OK;
  if (!y || (r > 0 && !w)) return LB_ERR_NULL;
  if (!aligned(w, dtype_size(latent_dtype)) || !aligned(y, dtype_size(out_dtype))) return LB_ERR_ALIGN;
  if (!paths) return LB_ERR_NULL;
  // only U and h are read
  lb_path used[2];
  for (int p = 0; p < 2; ++p) used[p] = lb_path{paths[p].U, nullptr, paths[p].h, nullptr, nullptr};
  st = check_paths(used, scale_dtype, 0, d_out, r, false);
  if (st != LB_OK) return st;
  const size_t ny = static_cast<size_t>(T * d_out) * dtype_size(out_dtype);
  if (overlap(y, ny, w, static_cast<size_t>(2 * T * r) * dtype_size(latent_dtype))) return LB_ERR_ARG;
  const size_t need = lb_from_latent_workspace_bytes(T, r);
  if (!workspace) return LB_ERR_NULL;
  if (!aligned(workspace, 256)) return LB_ERR_ALIGN;
  if (workspace_bytes < need) return LB_ERR_WORKSPACE;
  hipError_t e;
  if (r == 0) {
    e = lb::launch_zero_elems(y, T * d_out, out_dtype, stream);
  } else {
    lb::ForwardArgs a = make_args(nullptr, out_dtype, T, 0, d_out, r, used, scale_dtype, y, workspace, workspace_bytes);
    e = lb::launch_from_latent(a, w, latent_dtype, stream);
  }
  return e == hipSuccess ? LB_OK : LB_ERR_HIP;
}

size_t lb_backward_workspace_bytes(int64_t T, int64_t d_in, int64_t d_out, int64_t r) {
  if (check_sizes(T, d_in, d_out, r) != LB_OK || !lb::backward_supports(T, d_in, d_out, r)) return 0;
  return lb::backward_workspace_bytes(static_cast<int>(T), static_cast<int>(d_in), static_cast<int>(d_out),
                                      static_cast<int>(r));
}

lb_status lb_linear_backward(const void* x, const void* dy, lb_dtype act_dtype, int64_t T, int64_t d_in,
                             int64_t d_out, int64_t r, const lb_path* paths, lb_dtype scale_dtype,
                             const lb_path_train* train, float kappa, void* dx, void* workspace,
                             size_t workspace_bytes, hipStream_t stream) {
  if (!dtype_ok(act_dtype) || !dtype_ok(scale_dtype)) return LB_ERR_DTYPE;
  lb_status st = check_sizes(T, d_in, d_out, r);
  if (st != LB_OK) return st;
  if (!lb::backward_supports(T, d_in, d_out, r)) return LB_ERR_SHAPE;
  if (!(kappa > 0.0f) || !std::isfinite(kappa)) return LB_ERR_ARG;
  if (!paths || !train) return LB_ERR_NULL;
  const size_t ea = dtype_size(act_dtype);
  if ((T * d_in > 0 && !x) || (T * d_out > 0 && !dy)) return LB_ERR_NULL;
  if (!aligned(x, ea) || !aligned(dy, ea) || !aligned(dx, ea)) return LB_ERR_ALIGN;
  // forward parameters read: V, h, g, l
  lb_path used[2];
  for (int p = 0; p < 2; ++p) used[p] = lb_path{nullptr, paths[p].V, paths[p].h, paths[p].g, paths[p].l};
  st = check_paths(used, scale_dtype, d_in, d_out, r, true, false);
  if (st != LB_OK) return st;
  for (int p = 0; p < 2; ++p) {
    const lb_path_train& q = train[p];
    if ((d_out * r > 0 && (!q.U_latent || !q.Ut || !q.dU)) || (d_in * r > 0 && (!q.V_latent || !q.Vt || !q.dV)) ||
        (d_out > 0 && !q.dh) || (d_in > 0 && !q.dg) || (r > 0 && !q.dl))
      return LB_ERR_NULL;
    if (!aligned(q.U_latent, 4) || !aligned(q.V_latent, 4) || !aligned(q.Ut, 4) || !aligned(q.Vt, 4) ||
        !aligned(q.dU, 4) || !aligned(q.dV, 4) || !aligned(q.dh, 4) || !aligned(q.dg, 4) || !aligned(q.dl, 4))
      return LB_ERR_ALIGN;
  }
  const size_t ndx = static_cast<size_t>(T * d_in) * ea;
  if (dx && (overlap(dx, ndx, x, ndx) || overlap(dx, ndx, dy, static_cast<size_t>(T * d_out) * ea)))
    return LB_ERR_ARG;
  const size_t need = lb_backward_workspace_bytes(T, d_in, d_out, r);
  if (!workspace) return LB_ERR_NULL;
  if (!aligned(workspace, 256)) return LB_ERR_ALIGN;
  if (workspace_bytes < need) return LB_ERR_WORKSPACE;
  hipError_t e = hipSuccess;
  if (T == 0 || d_in == 0 || d_out == 0 || r == 0) {
    // an empty sum somewhere in every gradient: the non-empty ones are zero
    for (int p = 0; p < 2 && e == hipSuccess; ++p) {
      const lb_path_train& q = train[p];
      if ((e = lb::launch_zero_elems(q.dU, d_out * r, LB_F32, stream)) != hipSuccess) break;
      if ((e = lb::launch_zero_elems(q.dV, d_in * r, LB_F32, stream)) != hipSuccess) break;
      if ((e = lb::launch_zero_elems(q.dh, d_out, LB_F32, stream)) != hipSuccess) break;
      if ((e = lb::launch_zero_elems(q.dg, d_in, LB_F32, stream)) != hipSuccess) break;
      e = lb::launch_zero_elems(q.dl, r, LB_F32, stream);
    }
    if (e == hipSuccess && dx) e = lb::launch_zero_elems(dx, T * d_in, act_dtype, stream);
    return e == hipSuccess ? LB_OK : LB_ERR_HIP;
  }
  lb::BackwardArgs b{};
  b.x = x;
  b.dy = dy;
  b.act_dt = act_dtype;
  b.sc_dt = scale_dtype;
  b.T = static_cast<int>(T);
  b.d_in = static_cast<int>(d_in);
  b.d_out = static_cast<int>(d_out);
  b.r = static_cast<int>(r);
  for (int p = 0; p < 2; ++p) {
    b.V[p] = paths[p].V;
    b.h[p] = paths[p].h;
    b.g[p] = paths[p].g;
    b.l[p] = paths[p].l;
    b.Ut[p] = train[p].Ut;
    b.Vt[p] = train[p].Vt;
    b.U_lat[p] = train[p].U_latent;
    b.V_lat[p] = train[p].V_latent;
    b.dU[p] = train[p].dU;
    b.dV[p] = train[p].dV;
    b.dh[p] = train[p].dh;
    b.dg[p] = train[p].dg;
    b.dl[p] = train[p].dl;
  }
  b.dx = dx;
  b.kappa = kappa;
  b.ws = workspace;
  b.ws_bytes = workspace_bytes;
  e = lb::launch_backward(b, stream);
  return e == hipSuccess ? LB_OK : LB_ERR_HIP;
}

size_t lb_dual_svid_workspace_bytes(int64_t d_out, int64_t d_in, int64_t r, int64_t oversample) {
  if (!fits(d_out, d_in) || check_sizes(1, d_in, d_out, r) != LB_OK) return 0;
  if (!lb::svid_supports(d_out, d_in, r, oversample)) return 0;
  return lb::svid_workspace_bytes(static_cast<int>(d_out), static_cast<int>(d_in), static_cast<int>(r),
                                  static_cast<int>(std::min<int64_t>(oversample, 1 << 20)));
}

lb_status lb_dual_svid(const void* W, lb_dtype w_dtype, int64_t d_out, int64_t d_in, int64_t r, int64_t oversample,
                       int32_t iters, uint64_t seed, const lb_svid_out* out, float* W_res, void* workspace,
                       size_t workspace_bytes, hipStream_t stream) {
  if (!dtype_ok(w_dtype)) return LB_ERR_DTYPE;
  if (d_out <= 0 || d_in <= 0 || r <= 0 || oversample < 0 || !fits(d_out, d_in) ||
      check_sizes(1, d_in, d_out, r) != LB_OK || !lb::svid_supports(d_out, d_in, r, oversample))
    return LB_ERR_SHAPE;
  if (iters < 0 || iters > 1000) return LB_ERR_ARG;
  if (!W || !out || !workspace) return LB_ERR_NULL;
  for (int p = 0; p < 2; ++p) {
    const lb_svid_out& o = out[p];
    if (!o.U_latent || !o.V_latent || !o.h || !o.g || !o.l) return LB_ERR_NULL;
    if (!aligned(o.U_latent, 4) || !aligned(o.V_latent, 4) || !aligned(o.h, 4) || !aligned(o.g, 4) ||
        !aligned(o.l, 4) || !aligned(o.sigma, 4))
      return LB_ERR_ALIGN;
  }
  if (!aligned(W, dtype_size(w_dtype)) || !aligned(W_res, 4) || !aligned(workspace, 256)) return LB_ERR_ALIGN;
  if (workspace_bytes < lb_dual_svid_workspace_bytes(d_out, d_in, r, oversample)) return LB_ERR_WORKSPACE;
  const int over = static_cast<int>(std::min<int64_t>(oversample, 1 << 20));
  return lb::launch_dual_svid(W, w_dtype, static_cast<int>(d_out), static_cast<int>(d_in), static_cast<int>(r), over,
                              iters, seed, out, W_res, workspace, stream) == hipSuccess
             ? LB_OK
             : LB_ERR_HIP;
}

lb_status lb_dense_reference_weight(const lb_path* paths, lb_dtype scale_dtype, int64_t d_in, int64_t d_out,
                                    int64_t r, float* W, hipStream_t stream) {
  if (!dtype_ok(scale_dtype)) return LB_ERR_DTYPE;
  if (d_in < 0 || d_out < 0 || r < 0 || !fits(d_in, d_out) || !fits(d_in, r) || !fits(d_out, r))
    return LB_ERR_SHAPE;
  if (d_out > 65535 || r > 16384) return LB_ERR_SHAPE;
  if (d_in == 0 || d_out == 0) return LB_OK;
  if (!W) return LB_ERR_NULL;
  if (!aligned(W, 4)) return LB_ERR_ALIGN;
  lb_status st = check_paths(paths, scale_dtype, d_in, d_out, r);
  if (st != LB_OK) return st;
  lb::ForwardArgs a = make_args(nullptr, LB_F32, 0, d_in, d_out, r, paths, scale_dtype, nullptr, nullptr, 0);
  return lb::launch_dense_ref(a, W, stream) == hipSuccess ? LB_OK : LB_ERR_HIP;
}

}  // extern "C"
