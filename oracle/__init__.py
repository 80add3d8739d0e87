"""LittleBit reference oracle -- TEST INFRASTRUCTURE ONLY.

Python access to the fp64 CPU oracle in ``lb_oracle.c`` (plain C, built with
gcc).  Only the test suite, the smoke check and the benchmark's CPU-baseline
leg may import this package.  The GPU product path (the C-ABI library and its
Python binding) never imports it, and it never imports them: the two share no
code.

Stored-dtype decoding lives here too, written independently of the product:
bf16 is the upper half of an IEEE binary32, fp16 is IEEE binary16; both are
widened to fp64 exactly.

Functions and the passages of arXiv 2506.13771 they follow:
  pack / unpack            sign binarisation, Sec. 3.1 Eq. (uv_sign), in the
                           packed sign layout "LB layout v1";
  forward_factored (O1)    Proposition 1, Eq. (proposition1), summed over the
                           primary and residual paths, Sec. 3.3
                           Eq. (final_weight_approx_res);
  forward_sampled          O1 restricted to chosen output elements;
  dense_weight (O2)        Eqs. (w_primary_hat), (res_approx_structure),
                           (final_weight_approx_res);
  dense_forward (O2)       Y = X W_hat^T, the left side of Proposition 1;
  latent / from_latent     the rank-r latent cache and the output from it,
  (O5)                     Sec. "Analysis", paragraph "KV Cache Compression";
  backward (O6)            the chain rule through Proposition 1 with the
                           SmoothSign surrogate for the sign's derivative,
                           Sec. 4 "Training Details" and Appendix "SmoothSign
                           versus Straight-Through Estimator";
  svd / rank1 /            Dual-SVID initialisation, Sec. 3.2 "Dual-SVID
  svid_path / dual_svid    Initialization" (Eqs. sign_init_concise,
  (O7)                     scale_init_rank1_concise, latent_scale_init_concise_0),
                           and the residual path from the primary path's
                           error, Sec. 3.3 "Residual Compensation";
  bpw / rank_real /
  rank_for_bpw             Appendix "Average Bits Per Weight Calculation",
                           Eqs. (b_calculation) and (r_calculation).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "lb_oracle.c")
_LIB = os.path.join(_HERE, "liblb_oracle.so")

F32, F16, BF16 = "f32", "f16", "bf16"


def build(force: bool = False) -> str:
    """Compile lb_oracle.c into liblb_oracle.so with gcc (fp64, -O2, no fast-math)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.run(["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-fno-fast-math",
                        "-ffp-contract=off", "-fopenmp", _SRC, "-o", tmp, "-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        lib = ctypes.CDLL(build())
        i64, f64, i32 = ctypes.c_int64, ctypes.c_double, ctypes.c_int
        vp = ctypes.c_void_p
        lib.lbo_packed_bytes.restype = i64
        lib.lbo_packed_bytes.argtypes = [i64, i64, i32]
        lib.lbo_pack.restype = i64
        lib.lbo_pack.argtypes = [vp, i64, i64, i32, vp]
        lib.lbo_unpack.restype = None
        lib.lbo_unpack.argtypes = [vp, i64, i64, i32, vp]
        lib.lbo_pad_bits_clear.restype = i32
        lib.lbo_pad_bits_clear.argtypes = [vp, i64, i64, i32]
        lib.lbo_forward_factored.restype = None
        lib.lbo_forward_factored.argtypes = [vp, i64, i64, i64, i64, vp, vp, vp, vp, vp, i32, vp]
        lib.lbo_forward_factored_par.restype = None
        lib.lbo_forward_factored_par.argtypes = [vp, i64, i64, i64, i64, vp, vp, vp, vp, vp, i32, i32, vp]
        lib.lbo_svd.restype = None
        lib.lbo_svd.argtypes = [vp, i64, i64, vp, vp, vp]
        lib.lbo_rank1.restype = None
        lib.lbo_rank1.argtypes = [vp, i64, i64, vp, vp]
        lib.lbo_svid_path.restype = None
        lib.lbo_svid_path.argtypes = [vp, i64, i64, i64, vp, vp, vp, vp, vp]
        lib.lbo_path_weight.restype = None
        lib.lbo_path_weight.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, vp]
        lib.lbo_dual_svid.restype = None
        lib.lbo_dual_svid.argtypes = [vp, i64, i64, i64, vp, vp, vp, vp, vp, vp]
        lib.lbo_max_threads.restype = i32
        lib.lbo_max_threads.argtypes = []
        lib.lbo_forward_sampled.restype = None
        lib.lbo_forward_sampled.argtypes = [vp, i64, i64, i64, i64, vp, vp, vp, vp, vp, i32, vp, vp, i64, vp]
        lib.lbo_latent.restype = None
        lib.lbo_latent.argtypes = [vp, i64, i64, i64, vp, vp, vp, i32, vp]
        lib.lbo_from_latent.restype = None
        lib.lbo_from_latent.argtypes = [vp, i64, i64, i64, vp, vp, i32, vp]
        lib.lbo_backward.restype = None
        lib.lbo_backward.argtypes = [vp, vp, i64, i64, i64, i64, vp, vp, vp, vp, vp, i32, f64, vp, vp, vp, vp,
                                     vp, vp]
        lib.lbo_dense_weight.restype = None
        lib.lbo_dense_weight.argtypes = [i64, i64, i64, vp, vp, vp, vp, vp, i32, vp]
        lib.lbo_dense_forward.restype = None
        lib.lbo_dense_forward.argtypes = [vp, i64, i64, i64, vp, vp]
        lib.lbo_bpw.restype = f64
        lib.lbo_bpw.argtypes = [i64, i64, i64, i32]
        lib.lbo_total_bits.restype = f64
        lib.lbo_total_bits.argtypes = [i64, i64, i64, i32]
        lib.lbo_rank_real.restype = f64
        lib.lbo_rank_real.argtypes = [i64, i64, f64]
        lib.lbo_rank_for_bpw.restype = i64
        lib.lbo_rank_for_bpw.argtypes = [i64, i64, f64, i64, i32]
        _lib = lib
    return _lib


# ----------------------------------------------------------------------------
# stored dtypes -> fp64 (exact)
# ----------------------------------------------------------------------------
def to_f64(raw: np.ndarray, dtype: str) -> np.ndarray:
    """Widen stored values to fp64 exactly.  bf16/fp16 are given as uint16 bit patterns."""
    raw = np.ascontiguousarray(raw)
    if dtype == F32:
        return raw.astype(np.float32, copy=False).astype(np.float64)
    if dtype == F16:
        return raw.view(np.uint16).view(np.float16).astype(np.float64)
    if dtype == BF16:
        return (raw.view(np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    raise ValueError(dtype)


def _p(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data)


def _ptr_array(arrs):
    arr = (ctypes.c_void_p * len(arrs))(*[a.ctypes.data for a in arrs])
    return arr


# ----------------------------------------------------------------------------
# packing (LB layout v1)
# ----------------------------------------------------------------------------
ROLE_U, ROLE_V = 0, 1


def packed_bytes(rows: int, r: int, role: int) -> int:
    return int(_load().lbo_packed_bytes(rows, r, role))


def pack(src: np.ndarray, role: int):
    """Signs of a natural-orientation matrix src[rows][r] -> (bytes as uint8 array, nan count)."""
    src = np.ascontiguousarray(src, dtype=np.float64)
    rows, r = src.shape
    out = np.zeros(packed_bytes(rows, r, role), dtype=np.uint8)
    nans = _load().lbo_pack(_p(src), rows, r, role, _p(out))
    return out, int(nans)


def unpack(buf: np.ndarray, rows: int, r: int, role: int) -> np.ndarray:
    """Packed bytes -> int8 matrix [rows][r] with values -1/+1."""
    buf = np.ascontiguousarray(buf).view(np.uint8)
    assert buf.size == packed_bytes(rows, r, role)
    out = np.empty((rows, r), dtype=np.int8)
    _load().lbo_unpack(_p(buf), rows, r, role, _p(out))
    return out


def pad_bits_clear(buf: np.ndarray, rows: int, r: int, role: int) -> bool:
    buf = np.ascontiguousarray(buf).view(np.uint8)
    return bool(_load().lbo_pad_bits_clear(_p(buf), rows, r, role))


# ----------------------------------------------------------------------------
# forward
# ----------------------------------------------------------------------------
def _paths(U, V, h, g, l):
    U = [np.ascontiguousarray(u, dtype=np.int8) for u in U]
    V = [np.ascontiguousarray(v, dtype=np.int8) for v in V]
    h = [np.ascontiguousarray(a, dtype=np.float64) for a in h]
    g = [np.ascontiguousarray(a, dtype=np.float64) for a in g]
    l = [np.ascontiguousarray(a, dtype=np.float64) for a in l]
    n = len(U)
    assert n in (1, 2) and all(len(a) == n for a in (V, h, g, l))
    return U, V, h, g, l, n


def forward_factored(x, U, V, h, g, l) -> np.ndarray:
    """O1.  x [T,d_in] fp64; U[p] int8 [d_out,r]; V[p] int8 [d_in,r]; h,g,l fp64 per path."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    U, V, h, g, l, n = _paths(U, V, h, g, l)
    T, d_in = x.shape
    d_out, r = U[0].shape
    y = np.empty((T, d_out), dtype=np.float64)
    keep = (U, V, h, g, l)
    _load().lbo_forward_factored(_p(x), T, d_in, d_out, r, _ptr_array(U), _ptr_array(V),
                                 _ptr_array(h), _ptr_array(g), _ptr_array(l), n, _p(y))
    del keep
    return y


def forward_factored_par(x, U, V, h, g, l, nthreads: int = 0) -> np.ndarray:
    """O1 on several host threads (OpenMP); bit-identical to forward_factored."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    U, V, h, g, l, n = _paths(U, V, h, g, l)
    T, d_in = x.shape
    d_out, r = U[0].shape
    y = np.empty((T, d_out), dtype=np.float64)
    keep = (U, V, h, g, l)
    _load().lbo_forward_factored_par(_p(x), T, d_in, d_out, r, _ptr_array(U), _ptr_array(V),
                                     _ptr_array(h), _ptr_array(g), _ptr_array(l), n, int(nthreads), _p(y))
    del keep
    return y


def max_threads() -> int:
    """Threads an OpenMP region of the oracle library uses by default."""
    return int(_load().lbo_max_threads())


def latent(x, V, g, l) -> np.ndarray:
    """O5.  The cached latent w [npaths, T, r] of x [T, d_in] (fp64)."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    V = [np.ascontiguousarray(v, dtype=np.int8) for v in V]
    g = [np.ascontiguousarray(a, dtype=np.float64) for a in g]
    l = [np.ascontiguousarray(a, dtype=np.float64) for a in l]
    n = len(V)
    T, d_in = x.shape
    r = V[0].shape[1]
    w = np.empty((n, T, r), dtype=np.float64)
    _load().lbo_latent(_p(x), T, d_in, r, _ptr_array(V), _ptr_array(g), _ptr_array(l), n, _p(w))
    return w


def from_latent(w, U, h) -> np.ndarray:
    """O5.  y [T, d_out] from a cached latent w [npaths, T, r] (fp64)."""
    w = np.ascontiguousarray(w, dtype=np.float64)
    U = [np.ascontiguousarray(u, dtype=np.int8) for u in U]
    h = [np.ascontiguousarray(a, dtype=np.float64) for a in h]
    n, T, r = w.shape
    d_out = U[0].shape[0]
    y = np.empty((T, d_out), dtype=np.float64)
    _load().lbo_from_latent(_p(w), T, d_out, r, _ptr_array(U), _ptr_array(h), n, _p(y))
    return y


SMOOTHSIGN_K = 100.0  # the tanh slope of SmoothSign (Sec. 4 "Training Details")


def backward(x, dy, U_lat, V_lat, h, g, l, kappa: float = SMOOTHSIGN_K) -> dict:
    """O6.  Gradients of a loss with upstream gradient dy [T, d_out] for x [T, d_in] through both
    paths, the signs taken of the real latent factors U_lat [d_out, r] and V_lat [d_in, r], the
    sign's derivative replaced by that of tanh(kappa u).  Returns dx and per-path lists dU, dV,
    dh, dg, dl (fp64)."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    dy = np.ascontiguousarray(dy, dtype=np.float64)
    U_lat = [np.ascontiguousarray(a, dtype=np.float64) for a in U_lat]
    V_lat = [np.ascontiguousarray(a, dtype=np.float64) for a in V_lat]
    h = [np.ascontiguousarray(a, dtype=np.float64) for a in h]
    g = [np.ascontiguousarray(a, dtype=np.float64) for a in g]
    l = [np.ascontiguousarray(a, dtype=np.float64) for a in l]
    n = len(U_lat)
    T, d_in = x.shape
    d_out, r = U_lat[0].shape
    dx = np.empty((T, d_in))
    dU = [np.empty((d_out, r)) for _ in range(n)]
    dV = [np.empty((d_in, r)) for _ in range(n)]
    dh = [np.empty(d_out) for _ in range(n)]
    dg = [np.empty(d_in) for _ in range(n)]
    dl = [np.empty(r) for _ in range(n)]
    _load().lbo_backward(_p(x), _p(dy), T, d_in, d_out, r, _ptr_array(U_lat), _ptr_array(V_lat), _ptr_array(h),
                         _ptr_array(g), _ptr_array(l), n, float(kappa), _p(dx), _ptr_array(dU), _ptr_array(dV),
                         _ptr_array(dh), _ptr_array(dg), _ptr_array(dl))
    return {"dx": dx, "dU": dU, "dV": dV, "dh": dh, "dg": dg, "dl": dl}


def forward_sampled(x, U, V, h, g, l, ts, is_) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float64)
    U, V, h, g, l, n = _paths(U, V, h, g, l)
    T, d_in = x.shape
    d_out, r = U[0].shape
    ts = np.ascontiguousarray(ts, dtype=np.int64)
    is_ = np.ascontiguousarray(is_, dtype=np.int64)
    assert ts.shape == is_.shape and (ts.size == 0 or (ts.min() >= 0 and ts.max() < T
                                                       and is_.min() >= 0 and is_.max() < d_out))
    out = np.empty(ts.size, dtype=np.float64)
    _load().lbo_forward_sampled(_p(x), T, d_in, d_out, r, _ptr_array(U), _ptr_array(V),
                                _ptr_array(h), _ptr_array(g), _ptr_array(l), n,
                                _p(ts), _p(is_), ts.size, _p(out))
    return out


def dense_weight(U, V, h, g, l) -> np.ndarray:
    U, V, h, g, l, n = _paths(U, V, h, g, l)
    d_out, r = U[0].shape
    d_in = V[0].shape[0]
    W = np.empty((d_out, d_in), dtype=np.float64)
    _load().lbo_dense_weight(d_in, d_out, r, _ptr_array(U), _ptr_array(V),
                             _ptr_array(h), _ptr_array(g), _ptr_array(l), n, _p(W))
    return W


def dense_forward(x, W) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float64)
    W = np.ascontiguousarray(W, dtype=np.float64)
    T, d_in = x.shape
    d_out = W.shape[0]
    assert W.shape[1] == d_in
    y = np.empty((T, d_out), dtype=np.float64)
    _load().lbo_dense_forward(_p(x), T, d_in, d_out, _p(W), _p(y))
    return y


# ----------------------------------------------------------------------------
# bits per weight / rank
# ----------------------------------------------------------------------------
def total_bits(d_in: int, d_out: int, r: int, npaths: int = 2) -> float:
    return float(_load().lbo_total_bits(d_in, d_out, r, npaths))


def bpw(d_in: int, d_out: int, r: int, npaths: int = 2) -> float:
    return float(_load().lbo_bpw(d_in, d_out, r, npaths))


def rank_real(d_in: int, d_out: int, b: float) -> float:
    return float(_load().lbo_rank_real(d_in, d_out, b))


def rank_for_bpw(d_in: int, d_out: int, b: float, mult: int = 16, mode: int = 1) -> int:
    """mode 0: nearest integer (paper's examples); mode 1: largest multiple of mult within budget."""
    return int(_load().lbo_rank_for_bpw(d_in, d_out, b, mult, mode))


# ----------------------------------------------------------------------------
# O7: Dual-SVID initialisation
# ----------------------------------------------------------------------------
def svd(A):
    """Thin SVD by one-sided Jacobi: A [m, n] = U diag(s) V^T, U [m, k], V [n, k], k = min(m, n),
    s descending, each left vector's entry of largest magnitude positive."""
    A = np.ascontiguousarray(A, dtype=np.float64)
    m, n = A.shape
    k = min(m, n)
    U = np.zeros((m, k))
    V = np.zeros((n, k))
    s = np.zeros(k)
    _load().lbo_svd(_p(A), m, n, _p(U), _p(s), _p(V))
    return U, s, V


def rank1(M):
    """Best rank-1 approximation M ~ a b^T of a nonnegative matrix M [d, r], the top singular value
    split evenly between a and b."""
    M = np.ascontiguousarray(M, dtype=np.float64)
    d, r = M.shape
    a = np.zeros(d)
    b = np.zeros(r)
    _load().lbo_rank1(_p(M), d, r, _p(a), _p(b))
    return a, b


def svid_path(W, r):
    """One path of Dual-SVID: (U_latent [d_out, r], V_latent [d_in, r], h0, g0, l0)."""
    W = np.ascontiguousarray(W, dtype=np.float64)
    d_out, d_in = W.shape
    if not 1 <= r <= min(d_out, d_in):
        raise ValueError("rank out of range")
    Ul = np.zeros((d_out, r))
    Vl = np.zeros((d_in, r))
    h, g, l = np.zeros(d_out), np.zeros(d_in), np.zeros(r)
    _load().lbo_svid_path(_p(W), d_out, d_in, r, _p(Ul), _p(Vl), _p(h), _p(g), _p(l))
    return Ul, Vl, h, g, l


def path_weight(Ul, Vl, h, g, l):
    """diag(h) sign(U_latent) diag(l) sign(V_latent)^T diag(g) of one path."""
    Ul = np.ascontiguousarray(Ul, dtype=np.float64)
    Vl = np.ascontiguousarray(Vl, dtype=np.float64)
    h, g, l = (np.ascontiguousarray(a, dtype=np.float64) for a in (h, g, l))
    d_out, r = Ul.shape
    d_in = Vl.shape[0]
    W = np.zeros((d_out, d_in))
    _load().lbo_path_weight(_p(Ul), _p(Vl), _p(h), _p(g), _p(l), d_out, d_in, r, _p(W))
    return W


def dual_svid(W, r) -> dict:
    """Dual-SVID of both paths: the primary from W, the residual from W - W_hat_pri,0.  Returns
    {"U": [2 x U_latent], "V": [...], "h": [...], "g": [...], "l": [...], "Wres": W - W_hat_pri,0}."""
    W = np.ascontiguousarray(W, dtype=np.float64)
    d_out, d_in = W.shape
    if not 1 <= r <= min(d_out, d_in):
        raise ValueError("rank out of range")
    U = [np.zeros((d_out, r)) for _ in range(2)]
    V = [np.zeros((d_in, r)) for _ in range(2)]
    h = [np.zeros(d_out) for _ in range(2)]
    g = [np.zeros(d_in) for _ in range(2)]
    l = [np.zeros(r) for _ in range(2)]
    Wres = np.zeros((d_out, d_in))
    _load().lbo_dual_svid(_p(W), d_out, d_in, r, _ptr_array(U), _ptr_array(V), _ptr_array(h), _ptr_array(g),
                          _ptr_array(l), _p(Wres))
    return {"U": U, "V": V, "h": h, "g": g, "l": l, "Wres": Wres}
