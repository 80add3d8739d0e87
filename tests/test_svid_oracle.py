"""Pins of the Dual-SVID oracle (O7): Sec. 3.2 "Dual-SVID Initialization" (Eqs.
sign_init_concise, scale_init_rank1_concise, latent_scale_init_concise_0) and the
residual path's initialisation from the primary path's error (Sec. 3.3 "Residual
Compensation").  Pinned against numpy's LAPACK SVD (another implementation), the
Eckart-Young error of a truncation, an exact-recovery family whose magnitude
matrices are rank-1 by construction, equivariances of the effective weight
(scaling, transposition, permutations) and composition; planted mistakes in a
copy of the oracle must fail a pin."""
import ctypes
import os
import subprocess

import numpy as np
import pytest

import oracle as O


def _rel(a, b):
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300)


# ---------------------------------------------------------------------------
# the SVD
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("m,n", [(30, 20), (20, 30), (16, 16), (1, 7), (7, 1), (64, 48), (33, 65)])
def test_svd_against_lapack(m, n):
    rs = np.random.default_rng(m * 100 + n)
    A = rs.standard_normal((m, n))
    U, s, V = O.svd(A)
    ref = np.linalg.svd(A, compute_uv=False)
    assert np.abs(s - ref).max() <= 1e-12 * ref.max()
    assert _rel(U @ np.diag(s) @ V.T, A) < 1e-13
    k = min(m, n)
    assert np.abs(U.T @ U - np.eye(k)).max() < 1e-12
    assert np.abs(V.T @ V - np.eye(k)).max() < 1e-12
    assert np.all(np.diff(s) <= 0)
    # sign convention: each left vector's entry of largest magnitude is positive
    for c in range(k):
        assert U[np.argmax(np.abs(U[:, c])), c] > 0


def test_svd_rank_deficient_and_eckart_young():
    rs = np.random.default_rng(5)
    A = rs.standard_normal((40, 6)) @ rs.standard_normal((6, 30))  # rank 6
    U, s, V = O.svd(A)
    ref = np.linalg.svd(A, compute_uv=False)
    assert np.abs(s - ref).max() <= 1e-11 * ref.max()
    assert s[6:].max() < 1e-10 * s[0]
    # truncations: the Frobenius error is the root of the discarded sigma^2 (Eckart-Young)
    B = rs.standard_normal((50, 35))
    U, s, V = O.svd(B)
    for r in (1, 5, 20, 35):
        Br = U[:, :r] @ np.diag(s[:r]) @ V[:, :r].T
        assert abs(np.linalg.norm(B - Br) - np.sqrt(np.sum(s[r:] ** 2))) < 1e-11 * np.linalg.norm(B)


def test_rank1_of_nonnegative_matrices():
    rs = np.random.default_rng(7)
    a0, b0 = rs.random(23) + 0.1, rs.random(9) + 0.1
    a, b = O.rank1(np.outer(a0, b0))
    assert _rel(np.outer(a, b), np.outer(a0, b0)) < 1e-13
    assert np.all(a > 0) and np.all(b > 0)
    assert abs(np.linalg.norm(a) - np.linalg.norm(b)) < 1e-12 * np.linalg.norm(a)  # even split
    M = np.abs(rs.standard_normal((31, 12)))
    a, b = O.rank1(M)
    s = np.linalg.svd(M, compute_uv=False)
    assert abs(np.linalg.norm(M - np.outer(a, b)) - np.sqrt(np.sum(s[1:] ** 2))) < 1e-11 * np.linalg.norm(M)
    assert np.all(a >= 0) and np.all(b >= 0)


# ---------------------------------------------------------------------------
# Dual-SVID: exact recovery
# ---------------------------------------------------------------------------
def _hadamard(n):
    H = np.array([[1.0]])
    while H.shape[0] < n:
        H = np.block([[H, H], [H, -H]])
    return H


def exact_family(d_out, d_in, r, seed):
    """W = diag(h) S_U diag(l) S_V^T diag(g) whose Dual-SVID is exact: S_U, S_V are the first r
    columns of Sylvester-Hadamard matrices, h and g are constant on blocks of r consecutive
    indices (so the columns of diag(h) S_U stay orthogonal: the low bits of the row index, which
    the first r Walsh columns depend on, see equal weights), l is positive with distinct values.
    The SVD factors are then diag(h) S_U, diag(g) S_V up to column scales: |U'| and |V'| are rank-1."""
    rs = np.random.default_rng(seed)
    SU, SV = _hadamard(d_out)[:, :r], _hadamard(d_in)[:, :r]
    h = np.repeat(rs.random(d_out // r) + 0.5, r)
    g = np.repeat(rs.random(d_in // r) + 0.5, r)
    l = np.sort(rs.random(r) + 0.2)[::-1] * np.linspace(1.0, 0.5, r)
    W = np.diag(h) @ SU @ np.diag(l) @ SV.T @ np.diag(g)
    return W, SU, SV, h, g, l


@pytest.mark.parametrize("d_out,d_in,r", [(64, 32, 4), (32, 128, 8), (64, 64, 16), (16, 16, 1)])
def test_exact_recovery(d_out, d_in, r):
    W, SU, SV, h, g, l = exact_family(d_out, d_in, r, d_out + d_in + r)
    Ul, Vl, h0, g0, l0 = O.svid_path(W, r)
    What = O.path_weight(Ul, Vl, h0, g0, l0)
    assert _rel(What, W) < 1e-11
    # the signs are those of the construction, up to one sign per latent (both factors together)
    su, sv = np.sign(Ul), np.sign(Vl)
    flip = np.sign(np.sum(su * SU, axis=0))
    assert np.array_equal(su, SU * flip) and np.array_equal(sv, SV * flip)
    # h0, g0 proportional to h, g
    assert _rel(h0 / np.linalg.norm(h0), h / np.linalg.norm(h)) < 1e-12
    assert _rel(g0 / np.linalg.norm(g0), g / np.linalg.norm(g)) < 1e-12
    # the residual of the primary path is (numerically) zero
    d = O.dual_svid(W, r)
    assert np.linalg.norm(d["Wres"]) < 1e-11 * np.linalg.norm(W)


# ---------------------------------------------------------------------------
# Dual-SVID: equivariances and composition on generic weights
# ---------------------------------------------------------------------------
def low_rank_plus_noise(d_out, d_in, k, noise, seed):
    rs = np.random.default_rng(seed)
    A = rs.standard_normal((d_out, k)) * np.linspace(3.0, 1.0, k)
    B = rs.standard_normal((d_in, k))
    return A @ B.T / np.sqrt(k) + noise * rs.standard_normal((d_out, d_in))


def _what(W, r):
    return O.path_weight(*O.svid_path(W, r))


@pytest.mark.parametrize("d_out,d_in,r", [(48, 40, 6), (30, 50, 8), (64, 64, 12)])
def test_equivariances(d_out, d_in, r):
    W = low_rank_plus_noise(d_out, d_in, 2 * r, 0.05, d_out * d_in + r)
    base = _what(W, r)
    assert _rel(_what(3.7 * W, r), 3.7 * base) < 1e-10               # positive scaling
    assert _rel(_what(W.T.copy(), r), base.T) < 1e-10                # transposition swaps U and V
    rs = np.random.default_rng(1)
    P, Q = rs.permutation(d_out), rs.permutation(d_in)
    assert _rel(_what(W[P][:, Q].copy(), r), base[P][:, Q]) < 1e-10  # row and column permutations


def test_residual_path_composition():
    W = low_rank_plus_noise(56, 44, 16, 0.1, 3)
    r = 6
    d = O.dual_svid(W, r)
    prim = O.svid_path(W, r)
    for a, b in zip(prim, (d["U"][0], d["V"][0], d["h"][0], d["g"][0], d["l"][0])):
        assert np.array_equal(a, b)
    Wpri = O.path_weight(*prim)
    assert np.array_equal(d["Wres"], W - Wpri)
    res = O.svid_path(W - Wpri, r)
    for a, b in zip(res, (d["U"][1], d["V"][1], d["h"][1], d["g"][1], d["l"][1])):
        assert np.array_equal(a, b)
    # both approximations reduce the error (synthetic low-rank-plus-noise weight)
    Wres_hat = O.path_weight(*res)
    assert np.linalg.norm(W - Wpri) < np.linalg.norm(W)
    assert np.linalg.norm(W - Wpri - Wres_hat) < np.linalg.norm(W - Wpri)
    # the latent factors are the scaled SVD factors: U' V'^T is the truncated SVD
    U, s, V = np.linalg.svd(W)
    assert _rel(prim[0] @ prim[1].T, U[:, :r] @ np.diag(s[:r]) @ V[:r]) < 1e-11


# ---------------------------------------------------------------------------
# planted mistakes in a copy of the oracle fail a pin
# ---------------------------------------------------------------------------
SVID_MUTANTS = [
    ("svid: U' without sqrt(sigma)", "Ulat[i * r + c] = Us[i * k + c] * sqrt(sv[c]);", "Ulat[i * r + c] = Us[i * k + c];"),
    ("svid: latent scale drops l_v", "l[c] = lu[c] * lv[c];", "l[c] = lu[c];"),
    ("svid: V' from the left vectors", "Vlat[j * r + c] = Vs[j * k + c] * sqrt(sv[c]);",
     "Vlat[j * r + c] = Vs[(j % k) * k + (c + 1) % k] * sqrt(sv[c]);"),
    ("svid: residual adds the approximation", "Wres[e] = W[e] - Wres[e];", "Wres[e] = W[e] + Wres[e];"),
    ("svid: rank-1 takes the second triplet", "a[i] = k > 0 ? f * sg * Us[i * k] : 0.0;",
     "a[i] = k > 1 ? f * sg * Us[i * k + 1] : 0.0;"),
    ("svd: wrong rotation sign", "G[i * cols + q] = sn * gp + cs * gq;", "G[i * cols + q] = -sn * gp + cs * gq;"),
    ("svd: ascending order", "nrm[ord[i]] > nrm[ord[i - 1]]", "nrm[ord[i]] < nrm[ord[i - 1]]"),
]


def _svid_pins_fail(lib_path):
    lib = ctypes.CDLL(lib_path)
    vp, i64 = ctypes.c_void_p, ctypes.c_int64
    lib.lbo_svid_path.argtypes = [vp, i64, i64, i64, vp, vp, vp, vp, vp]
    lib.lbo_svid_path.restype = None
    lib.lbo_dual_svid.argtypes = [vp, i64, i64, i64, vp, vp, vp, vp, vp, vp]
    lib.lbo_dual_svid.restype = None
    lib.lbo_svd.argtypes = [vp, i64, i64, vp, vp, vp]
    lib.lbo_svd.restype = None

    def svid(W, r):
        W = np.ascontiguousarray(W)
        d_out, d_in = W.shape
        out = [np.zeros((d_out, r)), np.zeros((d_in, r)), np.zeros(d_out), np.zeros(d_in), np.zeros(r)]
        lib.lbo_svid_path(W.ctypes.data, d_out, d_in, r, *[a.ctypes.data for a in out])
        return out

    ok = True
    W, *_ = exact_family(64, 32, 4, 11)
    ok &= _rel(O.path_weight(*svid(W, 4)), W) < 1e-11
    A = np.random.default_rng(2).standard_normal((20, 12))
    U, s, V = np.zeros((20, 12)), np.zeros(12), np.zeros((12, 12))
    lib.lbo_svd(A.ctypes.data, 20, 12, U.ctypes.data, s.ctypes.data, V.ctypes.data)
    ok &= np.abs(s - np.linalg.svd(A, compute_uv=False)).max() < 1e-10 and _rel(U @ np.diag(s) @ V.T, A) < 1e-12
    Wg = low_rank_plus_noise(40, 36, 10, 0.1, 4)
    r = 5
    outs = [[np.zeros((40, r)) for _ in range(2)], [np.zeros((36, r)) for _ in range(2)],
            [np.zeros(40) for _ in range(2)], [np.zeros(36) for _ in range(2)], [np.zeros(r) for _ in range(2)]]
    pp = lambda A: (ctypes.c_void_p * 2)(*[a.ctypes.data for a in A])
    Wres = np.zeros((40, 36))
    lib.lbo_dual_svid(Wg.ctypes.data, 40, 36, r, *[pp(a) for a in outs], Wres.ctypes.data)
    prim = [outs[i][0] for i in range(5)]
    ok &= np.allclose(Wres, Wg - O.path_weight(*prim), rtol=0, atol=1e-12)
    return not ok


@pytest.mark.parametrize("desc,orig,repl", SVID_MUTANTS, ids=[m[0] for m in SVID_MUTANTS])
def test_svid_pins_catch_planted_mistakes(tmp_path, desc, orig, repl):
    src = open(os.path.join(os.path.dirname(O.__file__), "lb_oracle.c")).read()
    assert orig in src, desc
    cpath = tmp_path / "mut.c"
    cpath.write_text(src.replace(orig, repl, 1))
    lpath = str(tmp_path / "libmut.so")
    subprocess.run(["gcc", "-O1", "-fPIC", "-shared", str(cpath), "-o", lpath, "-lm"], check=True)
    assert _svid_pins_fail(lpath), desc
