"""Pins of the fp64 oracle against what the paper and the mathematics fix.

None of these tests re-types the oracle's own formula: they check values the
paper prints (worked BPW examples, the op-count example), hand-worked examples,
closed forms (all-ones signs, rank 1), invariants of the factorisation, and
brute force on tiny inputs.  A dropped term, a wrong sign, a transposed factor
or a swapped index in the oracle fails at least one of them (see
test_pins_catch_planted_mistakes, which plants such mistakes in a copy of the
oracle on the CPU).
"""
import itertools
import json
import os
import subprocess
import ctypes

import numpy as np
import pytest

import oracle as O


def _rand_layer(rs, T, d_in, d_out, r, npaths=2, neg_scales=True):
    U = [np.where(rs.standard_normal((d_out, r)) < 0, -1, 1).astype(np.int8) for _ in range(npaths)]
    V = [np.where(rs.standard_normal((d_in, r)) < 0, -1, 1).astype(np.int8) for _ in range(npaths)]
    sc = (lambda n: rs.standard_normal(n)) if neg_scales else (lambda n: np.abs(rs.standard_normal(n)))
    h = [sc(d_out) for _ in range(npaths)]
    g = [sc(d_in) for _ in range(npaths)]
    l = [sc(r) for _ in range(npaths)]
    x = rs.standard_normal((T, d_in))
    return x, U, V, h, g, l


# ---------------------------------------------------------------------------
# values printed in the paper
# ---------------------------------------------------------------------------
def test_bpw_worked_examples(golden_dir):
    """Appendix 'Average Bits Per Weight Calculation', Examples 1 and 2."""
    fx = json.load(open(os.path.join(golden_dir, "bpw_examples.json")))
    for ex in fx["examples"]:
        d_in, d_out = ex["d_in"], ex["d_out"]
        if ex.get("erratum_params"):
            # printed count differs from the product; the conclusions hold under both
            assert d_in * d_out != ex["printed_params"]
            r_printed = (ex["target_b"] * ex["printed_params"] - 32 * ex["printed_sum"]) / (2 * ex["printed_sum"] + 32)
            assert abs(r_printed - ex["printed_rank"]) <= ex["rank_abs_tol"]
        else:
            assert d_in * d_out == ex["printed_params"]
        assert d_in + d_out == ex["printed_sum"]
        r_real = O.rank_real(d_in, d_out, ex["target_b"])
        assert abs(r_real - ex["printed_rank"]) <= ex["rank_abs_tol"], (ex["name"], r_real)
        assert O.rank_for_bpw(d_in, d_out, ex["target_b"], 1, 0) == ex["chosen_rank"]
        b = O.bpw(d_in, d_out, ex["chosen_rank"])
        assert abs(b - ex["printed_b"]) <= ex["b_abs_tol"], (ex["name"], b)
        # the achieved b is below the target for these two examples
        assert b < ex["target_b"]


def test_op_count_example(golden_dir):
    """Appendix 'Inference Efficiency Analysis', Theoretical Cost Analysis: r = 431 at 0.3 BPW."""
    oc = json.load(open(os.path.join(golden_dir, "bpw_examples.json")))["op_count"]
    d_in, d_out = oc["d_in"], oc["d_out"]
    assert O.rank_for_bpw(d_in, d_out, oc["target_b"], 1, 0) == oc["printed_rank"]
    assert abs(2 * d_in * d_out / 1e6 - oc["printed_dense_mflops"]) <= oc["mflops_abs_tol"]
    assert abs(2 * (d_in + d_out) * oc["printed_rank"] / 1e6 - oc["printed_lb_mflops"]) <= oc["mflops_abs_tol"]


def test_bpw_single_path_halves():
    """Without the residual path the factor 2 is dropped (note under Eq. b_calculation)."""
    for d_in, d_out, r in [(4096, 4096, 80), (11008, 4096, 133), (7, 5, 3)]:
        assert O.total_bits(d_in, d_out, r, 2) == 2 * O.total_bits(d_in, d_out, r, 1)
        # per path: 1 bit per sign element, 16 bits per scale element
        assert O.total_bits(d_in, d_out, r, 1) == d_out * r + d_in * r + 16 * (d_out + d_in + r)


def test_rank_rule_benchmark_shapes():
    """Largest multiple of 16 within the b*d_in*d_out budget (the benchmark configurations'
    rounding; 4096x4096 at 0.1 BPW -> r = 80 is stated with the configuration)."""
    table = {(4096, 4096, 0.1): 80, (4096, 4096, 0.55): 544, (4096, 11008, 0.1): 128,
             (11008, 4096, 0.1): 128, (4096, 11008, 0.55): 800, (11008, 4096, 0.55): 800,
             (5120, 5120, 0.1): 96, (5120, 13824, 0.1): 160, (13824, 5120, 0.1): 160,
             (8192, 8192, 0.1): 176, (8192, 1024, 0.1): 16, (8192, 28672, 0.1): 288,
             (28672, 8192, 0.1): 288}
    for (d_in, d_out, b), r in table.items():
        got = O.rank_for_bpw(d_in, d_out, b, 16, 1)
        assert got == r, (d_in, d_out, b, got)
        assert O.total_bits(d_in, d_out, r) <= b * d_in * d_out
        assert O.total_bits(d_in, d_out, r + 16) > b * d_in * d_out


def test_rank_real_inverts_bpw():
    """Eq. (r_calculation) is the inverse of Eq. (b_calculation)."""
    for d_in, d_out, r in [(4096, 4096, 80), (8192, 28672, 288), (100, 37, 5)]:
        assert O.rank_real(d_in, d_out, O.bpw(d_in, d_out, r)) == pytest.approx(r, rel=1e-12)


# ---------------------------------------------------------------------------
# hand-worked forward
# ---------------------------------------------------------------------------
def _load_tiny(golden_dir):
    fx = json.load(open(os.path.join(golden_dir, "tiny_forward.json")))
    P = fx["paths"]
    U = [np.array(p["U"], dtype=np.int8) for p in P]
    V = [np.array(p["V"], dtype=np.int8) for p in P]
    h = [np.array(p["h"], dtype=np.float64) for p in P]
    g = [np.array(p["g"], dtype=np.float64) for p in P]
    l = [np.array(p["l"], dtype=np.float64) for p in P]
    x = np.array(fx["x"], dtype=np.float64)
    return fx, x, U, V, h, g, l


def test_tiny_forward_hand_worked(golden_dir):
    fx, x, U, V, h, g, l = _load_tiny(golden_dir)
    y = O.forward_factored(x, U, V, h, g, l)
    assert np.array_equal(y, np.array(fx["y"], dtype=np.float64))
    y0 = O.forward_factored(x, U[:1], V[:1], h[:1], g[:1], l[:1])
    assert np.array_equal(y0, np.array(fx["y_path0"], dtype=np.float64))
    y1 = O.forward_factored(x, U[1:], V[1:], h[1:], g[1:], l[1:])
    assert np.array_equal(y1, np.array(fx["y_path1"], dtype=np.float64))
    W0 = O.dense_weight(U[:1], V[:1], h[:1], g[:1], l[:1])
    assert np.array_equal(W0[0], np.array(fx["W_path0_row0"], dtype=np.float64))
    W = O.dense_weight(U, V, h, g, l)
    assert W.shape == (fx["d_out"], fx["d_in"])
    assert np.array_equal(O.dense_forward(x, W), np.array(fx["y"], dtype=np.float64))


# ---------------------------------------------------------------------------
# Proposition 1: factored == dense, brute force on tiny inputs
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("d_in,d_out,r,T", [
    (1, 1, 1, 1), (2, 3, 1, 3), (3, 2, 2, 1), (31, 33, 16, 3), (32, 64, 17, 1),
    (33, 31, 32, 3), (64, 32, 16, 2), (64, 64, 32, 1), (17, 5, 7, 4)])
def test_factored_equals_dense(d_in, d_out, r, T):
    rs = np.random.default_rng(1000 + d_in * 7 + d_out * 13 + r + T)
    x, U, V, h, g, l = _rand_layer(rs, T, d_in, d_out, r)
    y1 = O.forward_factored(x, U, V, h, g, l)
    W = O.dense_weight(U, V, h, g, l)
    y2 = O.dense_forward(x, W)
    scale = np.abs(y2).max() + 1e-300
    assert np.abs(y1 - y2).max() / scale < 1e-12


@pytest.mark.parametrize("d_in,d_out,r,T", [(1, 1, 1, 1), (33, 31, 32, 3), (100, 77, 19, 5), (64, 300, 40, 2)])
@pytest.mark.parametrize("nthreads", [1, 3, 8])
def test_parallel_forward_is_bit_identical(d_in, d_out, r, T, nthreads):
    """The OpenMP form of O1 computes every output with the same operations in the same
    order as the serial one, so it must agree bit for bit, at any thread count; and it
    meets the brute-force dense route like the serial one."""
    rs = np.random.default_rng(7000 + d_in + d_out + r + T)
    x, U, V, h, g, l = _rand_layer(rs, T, d_in, d_out, r)
    y1 = O.forward_factored(x, U, V, h, g, l)
    yp = O.forward_factored_par(x, U, V, h, g, l, nthreads)
    assert np.array_equal(y1, yp)
    y2 = O.dense_forward(x, O.dense_weight(U, V, h, g, l))
    assert np.abs(yp - y2).max() / (np.abs(y2).max() + 1e-300) < 1e-12


def test_brute_force_python_loops():
    """Independent brute force: enumerate every W_hat entry with Python loops, from the
    definition diag(h) U diag(l) V^T diag(g), for both paths."""
    rs = np.random.default_rng(7)
    T, d_in, d_out, r = 2, 5, 4, 3
    x, U, V, h, g, l = _rand_layer(rs, T, d_in, d_out, r)
    y_ref = np.zeros((T, d_out))
    for t in range(T):
        for i in range(d_out):
            acc = 0.0
            for j in range(d_in):
                wij = 0.0
                for p in range(2):
                    for k in range(r):
                        wij += h[p][i] * float(U[p][i, k]) * l[p][k] * float(V[p][j, k]) * g[p][j]
                acc += x[t, j] * wij
            y_ref[t, i] = acc
    y = O.forward_factored(x, U, V, h, g, l)
    assert np.allclose(y, y_ref, rtol=1e-12, atol=1e-12 * np.abs(y_ref).max())


# ---------------------------------------------------------------------------
# closed forms
# ---------------------------------------------------------------------------
def test_all_ones_closed_form():
    """All signs +1: y[t,i] = sum_p h_p[i] * (sum_k l_p[k]) * (sum_j g_p[j] x[t,j])."""
    rs = np.random.default_rng(11)
    T, d_in, d_out, r = 3, 40, 24, 16
    x, U, V, h, g, l = _rand_layer(rs, T, d_in, d_out, r)
    U = [np.ones_like(u) for u in U]
    V = [np.ones_like(v) for v in V]
    y = O.forward_factored(x, U, V, h, g, l)
    ref = sum(np.outer(x @ g[p], h[p]) * l[p].sum() for p in range(2))
    assert np.allclose(y, ref, rtol=1e-12, atol=1e-12 * np.abs(ref).max())


def test_all_minus_ones_closed_form():
    """All signs -1: the two sign flips cancel, same closed form as all +1."""
    rs = np.random.default_rng(12)
    T, d_in, d_out, r = 2, 9, 6, 4
    x, U, V, h, g, l = _rand_layer(rs, T, d_in, d_out, r)
    U = [-np.ones_like(u) for u in U]
    V = [-np.ones_like(v) for v in V]
    y = O.forward_factored(x, U, V, h, g, l)
    ref = sum(np.outer(x @ g[p], h[p]) * l[p].sum() for p in range(2))
    assert np.allclose(y, ref, rtol=1e-12, atol=1e-12 * np.abs(ref).max())


def test_rank_one_closed_form():
    """r = 1: y = sum_p h_p * u_p * l_p * (v_p . (g_p * x))."""
    rs = np.random.default_rng(13)
    T, d_in, d_out = 4, 12, 7
    x, U, V, h, g, l = _rand_layer(rs, T, d_in, d_out, 1)
    y = O.forward_factored(x, U, V, h, g, l)
    ref = np.zeros((T, d_out))
    for p in range(2):
        s = (x * g[p][None, :]) @ V[p][:, 0].astype(np.float64)       # [T]
        ref += np.outer(s * l[p][0], h[p] * U[p][:, 0])
    assert np.allclose(y, ref, rtol=1e-12, atol=1e-12 * np.abs(ref).max())


def test_identity_like_layer():
    """d_in = d_out = r = 1, one path: y = h * u * l * v * g * x exactly."""
    for u, v in itertools.product([-1, 1], repeat=2):
        y = O.forward_factored(np.array([[3.0]]), [np.array([[u]], np.int8)], [np.array([[v]], np.int8)],
                               [np.array([2.0])], [np.array([5.0])], [np.array([0.25])])
        assert y[0, 0] == 2.0 * u * 0.25 * v * 5.0 * 3.0


# ---------------------------------------------------------------------------
# the latent cache (O5): composition with the rest of the forward, closed
# forms, the latent-scale sign invariant, brute force
# ---------------------------------------------------------------------------
def test_latent_composes_to_the_forward():
    rs = np.random.default_rng(31)
    for T, d_in, d_out, r in [(3, 33, 17, 5), (1, 64, 40, 16), (4, 7, 9, 1)]:
        x, U, V, h, g, l = _rand_layer(rs, T, d_in, d_out, r)
        w = O.latent(x, V, g, l)
        assert w.shape == (2, T, r)
        assert np.array_equal(O.from_latent(w, U, h), O.forward_factored(x, U, V, h, g, l))
        W = O.dense_weight(U, V, h, g, l)
        assert np.allclose(O.from_latent(w, U, h), O.dense_forward(x, W), rtol=1e-12, atol=1e-12)


def test_latent_closed_forms():
    """All V signs +1: w_p[t,k] = l_p[k] sum_j g_p[j] x[t,j]; all U signs +1:
    y[t,i] = sum_p h_p[i] sum_k w_p[t,k]."""
    rs = np.random.default_rng(32)
    T, d_in, d_out, r = 3, 40, 24, 16
    x, U, V, h, g, l = _rand_layer(rs, T, d_in, d_out, r)
    w = O.latent(x, [np.ones_like(v) for v in V], g, l)
    ref = np.stack([np.outer(x @ g[p], l[p]) for p in range(2)])
    assert np.allclose(w, ref, rtol=1e-12, atol=1e-12 * np.abs(ref).max())
    wr = rs.standard_normal((2, T, r))
    y = O.from_latent(wr, [np.ones_like(u) for u in U], h)
    ref = sum(np.outer(wr[p].sum(axis=1), h[p]) for p in range(2))
    assert np.allclose(y, ref, rtol=1e-12, atol=1e-12 * np.abs(ref).max())


def test_latent_sign_invariant():
    """Negating column k of V_p together with l_p[k] leaves the latent unchanged."""
    rs = np.random.default_rng(33)
    x, U, V, h, g, l = _rand_layer(rs, 2, 48, 40, 20)
    w = O.latent(x, V, g, l)
    for p, k in [(0, 0), (1, 7)]:
        V2, l2 = [a.copy() for a in V], [a.copy() for a in l]
        V2[p][:, k] *= -1
        l2[p][k] *= -1
        assert np.array_equal(O.latent(x, V2, g, l2), w)


def test_latent_brute_force_python_loops():
    rs = np.random.default_rng(34)
    T, d_in, d_out, r = 2, 5, 4, 3
    x, U, V, h, g, l = _rand_layer(rs, T, d_in, d_out, r)
    w = O.latent(x, V, g, l)
    for p in range(2):
        for t in range(T):
            for k in range(r):
                s = 0.0
                for j in range(d_in):
                    s += float(V[p][j, k]) * float(x[t, j]) * float(g[p][j])
                assert abs(w[p, t, k] - s * l[p][k]) <= 1e-12 * (1 + abs(s))
    y = O.from_latent(w, U, h)
    for t in range(T):
        for i in range(d_out):
            s = 0.0
            for p in range(2):
                s += h[p][i] * sum(float(U[p][i, k]) * w[p, t, k] for k in range(r))
            assert abs(y[t, i] - s) <= 1e-12 * (1 + abs(s))


# ---------------------------------------------------------------------------
# invariants (bitwise in fp64 where the arithmetic is exact)
# ---------------------------------------------------------------------------
@pytest.fixture
def layer():
    rs = np.random.default_rng(21)
    return _rand_layer(rs, 3, 48, 40, 20)


def _copy(ls):
    return [a.copy() for a in ls]


def test_invariant_latent_column_flip(layer):
    x, U, V, h, g, l = layer
    y = O.forward_factored(x, U, V, h, g, l)
    for p, k in [(0, 0), (1, 7), (0, 19)]:
        U2, l2 = _copy(U), _copy(l)
        U2[p][:, k] *= -1
        l2[p][k] *= -1
        assert np.array_equal(O.forward_factored(x, U2, V, h, g, l2), y)
        V2, l3 = _copy(V), _copy(l)
        V2[p][:, k] *= -1
        l3[p][k] *= -1
        assert np.array_equal(O.forward_factored(x, U, V2, h, g, l3), y)
        # flipping only one of them is not invariant
        assert not np.allclose(O.forward_factored(x, U2, V, h, g, l), y)


def test_invariant_row_flips(layer):
    x, U, V, h, g, l = layer
    y = O.forward_factored(x, U, V, h, g, l)
    U2, h2 = _copy(U), _copy(h)
    U2[1][5, :] *= -1
    h2[1][5] *= -1
    assert np.array_equal(O.forward_factored(x, U2, V, h2, g, l), y)
    V2, g2 = _copy(V), _copy(g)
    V2[0][11, :] *= -1
    g2[0][11] *= -1
    assert np.array_equal(O.forward_factored(x, U, V2, h, g2, l), y)
    # flipping only the row of U negates exactly that output column's path-1 part
    U3 = _copy(U)
    U3[1][5, :] *= -1
    y3 = O.forward_factored(x, U3, V, h, g, l)
    mask = np.ones(y.shape[1], bool)
    mask[5] = False
    assert np.array_equal(y3[:, mask], y[:, mask])


def test_invariant_latent_permutation(layer):
    x, U, V, h, g, l = layer
    y = O.forward_factored(x, U, V, h, g, l)
    perm = np.random.default_rng(3).permutation(U[0].shape[1])
    y2 = O.forward_factored(x, [u[:, perm] for u in U], [v[:, perm] for v in V], h, g, [a[perm] for a in l])
    assert np.allclose(y2, y, rtol=1e-12, atol=1e-12 * np.abs(y).max())


def test_invariant_path_swap_and_single_path(layer):
    x, U, V, h, g, l = layer
    y = O.forward_factored(x, U, V, h, g, l)
    ys = O.forward_factored(x, U[::-1], V[::-1], h[::-1], g[::-1], l[::-1])
    assert np.array_equal(ys, y)
    h0 = [h[0], np.zeros_like(h[1])]
    y_single = O.forward_factored(x, U[:1], V[:1], h[:1], g[:1], l[:1])
    assert np.array_equal(O.forward_factored(x, U, V, h0, g, l), y_single)
    # additivity over paths
    y_res = O.forward_factored(x, U[1:], V[1:], h[1:], g[1:], l[1:])
    assert np.allclose(y_single + y_res, y, rtol=1e-13, atol=1e-13 * np.abs(y).max())


def test_invariant_linearity(layer):
    x, U, V, h, g, l = layer
    y = O.forward_factored(x, U, V, h, g, l)
    assert np.array_equal(O.forward_factored(4.0 * x, U, V, h, g, l), 4.0 * y)
    x2 = np.random.default_rng(5).standard_normal(x.shape)
    y2 = O.forward_factored(x2, U, V, h, g, l)
    y12 = O.forward_factored(x + x2, U, V, h, g, l)
    assert np.allclose(y12, y + y2, rtol=1e-12, atol=1e-12 * np.abs(y12).max())
    # tokens are independent rows
    assert np.array_equal(O.forward_factored(x[1:2], U, V, h, g, l), y[1:2])


def test_sampled_matches_full(layer):
    x, U, V, h, g, l = layer
    y = O.forward_factored(x, U, V, h, g, l)
    ts = np.array([0, 2, 1, 2])
    is_ = np.array([0, 39, 17, 3])
    assert np.allclose(O.forward_sampled(x, U, V, h, g, l, ts, is_), y[ts, is_], rtol=1e-13, atol=0)


# ---------------------------------------------------------------------------
# packing (LB layout v1)
# ---------------------------------------------------------------------------
def test_pack_hand_worked(golden_dir):
    fx = json.load(open(os.path.join(golden_dir, "pack_examples.json")))
    for c in fx["cases"]:
        role = O.ROLE_U if c["role"] == "U" else O.ROLE_V
        src = np.ones((c["rows"], c["r"]))
        for a, b in c["negatives"]:
            src[a, b] = -1.0
        for a, b in c["negative_zero"]:
            src[a, b] = -0.0
        buf, nans = O.pack(src, role)
        assert nans == 0
        assert buf.tobytes().hex() == c["hex"] + c["hex_tail"], c["name"]
        S = O.unpack(buf, c["rows"], c["r"], role)
        assert np.array_equal(S, np.where(src < 0, -1, 1))


@pytest.mark.parametrize("rows,r,role", [
    (64, 16, 0), (64, 80, 0), (128, 176, 0), (96, 32, 0), (40, 50, 0), (33, 7, 0),
    (4096 // 64, 80, 1), (96, 16, 1), (48, 3, 1), (50, 33, 1), (32, 1, 1)])
def test_pack_roundtrip_and_counts(rows, r, role):
    rs = np.random.default_rng(rows * 31 + r * 7 + role)
    src = rs.standard_normal((rows, r))
    buf, nans = O.pack(src, role)
    assert nans == 0
    assert buf.size == O.packed_bytes(rows, r, role)
    assert np.array_equal(O.unpack(buf, rows, r, role), np.where(src < 0, -1, 1))
    popcount = int(np.unpackbits(buf).sum())
    assert popcount == int((src < 0).sum())
    assert O.pad_bits_clear(buf, rows, r, role)
    pos, _ = O.pack(np.abs(src), role)
    assert not pos.any()
    neg, _ = O.pack(-np.abs(src) - 1.0, role)
    assert int(np.unpackbits(neg).sum()) == rows * r
    assert O.pad_bits_clear(neg, rows, r, role)


def test_packed_sizes_no_overhead():
    # zero padding for the benchmark shapes; the tail plane keeps r % 32 == 16 at 1 bit per sign
    assert O.packed_bytes(4096, 80, O.ROLE_V) == 40960
    assert O.packed_bytes(4096, 80, O.ROLE_U) == 32768 + 8192
    assert O.packed_bytes(1024, 16, O.ROLE_U) == 2048
    for rows, r in [(4096, 80), (11008, 128), (28672, 288), (1024, 16), (8192, 176)]:
        for role in (0, 1):
            assert O.packed_bytes(rows, r, role) * 8 == rows * r


def test_pack_nan_counted():
    src = np.ones((32, 2))
    src[3, 1] = np.nan
    buf, nans = O.pack(src, O.ROLE_V)
    assert nans == 1


# ---------------------------------------------------------------------------
# dtype widening
# ---------------------------------------------------------------------------
def test_to_f64_exact():
    # bf16 0x3F80 = 1.0, 0xC000 = -2.0, 0x0001 = smallest subnormal 2^-133
    b = np.array([0x3F80, 0xC000, 0x0001, 0x7F7F], dtype=np.uint16)
    v = O.to_f64(b, O.BF16)
    assert v[0] == 1.0 and v[1] == -2.0 and v[2] == 2.0 ** -133
    assert v[3] == (2 - 2 ** -7) * 2.0 ** 127
    # fp16 0x3C00 = 1.0, 0x0001 = 2^-24 (subnormal), 0x7BFF = 65504
    f = np.array([0x3C00, 0x0001, 0x7BFF, 0x8400], dtype=np.uint16)
    v = O.to_f64(f, O.F16)
    assert list(v) == [1.0, 2.0 ** -24, 65504.0, -(2.0 ** -14)]


# ---------------------------------------------------------------------------
# the backward (O6): the dense route of the same loss, finite differences,
# linearity, the SmoothSign factor
# ---------------------------------------------------------------------------
def _rand_train_layer(rs, T, d_in, d_out, r, lat_scale=0.02):
    """Real latent factors (of the order of 1 / kappa, so the surrogate factor varies), scales of
    both signs, x and an upstream gradient dy."""
    U_lat = [lat_scale * rs.standard_normal((d_out, r)) for _ in range(2)]
    V_lat = [lat_scale * rs.standard_normal((d_in, r)) for _ in range(2)]
    h = [rs.standard_normal(d_out) for _ in range(2)]
    g = [rs.standard_normal(d_in) for _ in range(2)]
    l = [rs.standard_normal(r) for _ in range(2)]
    x = rs.standard_normal((T, d_in))
    dy = rs.standard_normal((T, d_out))
    return x, dy, U_lat, V_lat, h, g, l


def _signs(a):
    return np.where(a < 0, -1, 1).astype(np.int8)


def _tanh_slope_fd(u, kappa, eps=1e-7):
    """d/du tanh(kappa u) by central differences of numpy's tanh."""
    return (np.tanh(kappa * (u + eps)) - np.tanh(kappa * (u - eps))) / (2 * eps)


def _dense_route(x, dy, U_lat, V_lat, h, g, l, kappa):
    """Gradients of L = sum(dy * (x W_hat^T)) from the dense weight: with G = dy^T x, L = sum(G * W_hat)
    and W_hat = sum_p diag(h_p) U_p diag(l_p) V_p^T diag(g_p), so every gradient is a contraction of G
    with the other factors (numpy matrix products), then the SmoothSign slope from finite differences."""
    U = [_signs(a) for a in U_lat]
    V = [_signs(a) for a in V_lat]
    G = dy.T @ x
    out = {"dx": dy @ O.dense_weight(U, V, h, g, l), "dU": [], "dV": [], "dh": [], "dg": [], "dl": []}
    for p in range(2):
        Us, Vs = U[p].astype(np.float64), V[p].astype(np.float64)
        core = (Us * l[p]) @ Vs.T  # U diag(l) V^T
        out["dh"].append((G * core * g[p][None, :]).sum(axis=1))
        out["dg"].append((G * core * h[p][:, None]).sum(axis=0))
        out["dl"].append(np.einsum("ij,ik,jk->k", G, h[p][:, None] * Us, g[p][:, None] * Vs))
        dUs = h[p][:, None] * ((G * g[p][None, :]) @ Vs) * l[p][None, :]
        dVs = g[p][:, None] * ((G.T * h[p][None, :]) @ Us) * l[p][None, :]
        out["dU"].append(dUs * _tanh_slope_fd(U_lat[p], kappa))
        out["dV"].append(dVs * _tanh_slope_fd(V_lat[p], kappa))
    return out


def _close(a, b, rtol):
    return np.allclose(a, b, rtol=rtol, atol=rtol * max(1.0, np.abs(b).max()))


@pytest.mark.parametrize("T,d_in,d_out,r", [(3, 9, 7, 5), (1, 33, 17, 16), (4, 5, 40, 1), (2, 64, 32, 33)])
def test_backward_matches_the_dense_route(T, d_in, d_out, r):
    rs = np.random.default_rng(T * 1000 + d_in + r)
    args = _rand_train_layer(rs, T, d_in, d_out, r)
    got = O.backward(*args)
    ref = _dense_route(*args, kappa=O.SMOOTHSIGN_K)
    assert _close(got["dx"], ref["dx"], 1e-11)
    for key in ("dh", "dg", "dl"):
        for p in range(2):
            assert _close(got[key][p], ref[key][p], 1e-11), (key, p)
    for key in ("dU", "dV"):
        for p in range(2):
            assert _close(got[key][p], ref[key][p], 1e-6), (key, p)  # finite-difference slope


def test_backward_finite_differences():
    """L is linear in each of x, h_p, g_p, l_p, so a central difference along any direction is the
    directional derivative up to rounding."""
    rs = np.random.default_rng(41)
    x, dy, U_lat, V_lat, h, g, l = _rand_train_layer(rs, 3, 12, 10, 6)
    U, V = [_signs(a) for a in U_lat], [_signs(a) for a in V_lat]
    got = O.backward(x, dy, U_lat, V_lat, h, g, l)

    def loss(x_, h_, g_, l_):
        return float((dy * O.forward_factored(x_, U, V, h_, g_, l_)).sum())

    eps = 1e-3
    d = rs.standard_normal(x.shape)
    fd = (loss(x + eps * d, h, g, l) - loss(x - eps * d, h, g, l)) / (2 * eps)
    assert abs(fd - (got["dx"] * d).sum()) <= 1e-9 * (1 + abs(fd))
    for p in range(2):
        for name, vecs, key in (("h", h, "dh"), ("g", g, "dg"), ("l", l, "dl")):
            dv = rs.standard_normal(vecs[p].shape)
            plus = [v.copy() for v in vecs]
            minus = [v.copy() for v in vecs]
            plus[p] += eps * dv
            minus[p] -= eps * dv
            argsp = {"h": h, "g": g, "l": l}
            argsm = dict(argsp)
            argsp[name], argsm[name] = plus, minus
            fd = (loss(x, argsp["h"], argsp["g"], argsp["l"]) - loss(x, argsm["h"], argsm["g"], argsm["l"])) / (2 * eps)
            assert abs(fd - (got[key][p] * dv).sum()) <= 1e-9 * (1 + abs(fd)), (name, p)


def test_backward_linear_in_dy_and_zero_for_zero_dy():
    rs = np.random.default_rng(42)
    x, dy, U_lat, V_lat, h, g, l = _rand_train_layer(rs, 2, 16, 12, 8)
    dy2 = rs.standard_normal(dy.shape)
    a = O.backward(x, dy, U_lat, V_lat, h, g, l)
    b = O.backward(x, dy2, U_lat, V_lat, h, g, l)
    c = O.backward(x, dy + dy2, U_lat, V_lat, h, g, l)
    assert _close(c["dx"], a["dx"] + b["dx"], 1e-12)
    for key in ("dU", "dV", "dh", "dg", "dl"):
        for p in range(2):
            assert _close(c[key][p], a[key][p] + b[key][p], 1e-12), key
    z = O.backward(x, np.zeros_like(dy), U_lat, V_lat, h, g, l)
    assert not z["dx"].any() and not any(z[k][p].any() for k in ("dU", "dV", "dh", "dg", "dl") for p in range(2))


def test_backward_smoothsign_factor():
    """At u = 0 the surrogate slope is kappa; far from 0 it vanishes; the sign itself follows the
    forward's convention (u = 0 counts as +1, so flipping the sign of a zero latent changes nothing)."""
    rs = np.random.default_rng(43)
    x, dy, U_lat, V_lat, h, g, l = _rand_train_layer(rs, 2, 10, 8, 4)
    for A in U_lat + V_lat:
        A[0, :] = 0.0
        A[1, :] = 1.0  # kappa u = 100: slope below 1e-80
    for kappa in (100.0, 7.0):
        got = O.backward(x, dy, U_lat, V_lat, h, g, l, kappa=kappa)
        ref = _dense_route(x, dy, U_lat, V_lat, h, g, l, kappa=1.0)  # slope(0) = 1 for kappa = 1 ...
        for p in range(2):
            # ... so at u = 0 the dense-route value is the sign gradient itself
            assert _close(got["dU"][p][0], kappa * ref["dU"][p][0], 1e-6)
            assert _close(got["dV"][p][0], kappa * ref["dV"][p][0], 1e-6)
        if kappa == 100.0:
            assert all(np.abs(got[k][p][1]).max() < 1e-60 for k in ("dU", "dV") for p in range(2))
    U2 = [a.copy() for a in U_lat]
    U2[0][0, :] = -0.0
    a = O.backward(x, dy, U_lat, V_lat, h, g, l)
    b = O.backward(x, dy, U2, V_lat, h, g, l)
    assert np.array_equal(a["dx"], b["dx"])


# ---------------------------------------------------------------------------
# the pins catch planted mistakes (mutations are applied to a copy of the oracle
# source on the CPU; the real oracle is never modified)
# ---------------------------------------------------------------------------
MUTANTS = [
    # (description, original snippet, replacement)
    ("transposed V index", "V[p][j * r + k] * a[j]", "V[p][(j % r) * r + (k % r)] * a[j]"),
    ("dropped latent scale", "z[k] = s * l[p][k];", "z[k] = s;"),
    ("dropped row scale", "y[t * d_out + i] += s * h[p][i];", "y[t * d_out + i] += s;"),
    ("wrong column scale", "a[j] = x[t * d_in + j] * g[p][j];", "a[j] = x[t * d_in + j];"),
    ("residual path ignored", "for (int p = 0; p < npaths; p++) {\n    for (int64_t t = 0; t < T; t++) {",
     "for (int p = 0; p < 1; p++) {\n    for (int64_t t = 0; t < T; t++) {"),
    ("sign flipped", "s += (double)U[p][i * r + k] * z[k];", "s -= (double)U[p][i * r + k] * z[k];"),
    ("latent: dropped latent scale", "w[(p * T + t) * r + k] = s * l[p][k];", "w[(p * T + t) * r + k] = s;"),
    ("latent: transposed V index", "s += (double)V[p][j * r + k] * a[j];\n        w[",
     "s += (double)V[p][(j % r) * r + (k % r)] * a[j];\n        w["),
    ("from latent: wrong path", "U[p][i * r + k] * w[(p * T + t) * r + k];", "U[p][i * r + k] * w[(0 * T + t) * r + k];"),
    ("from latent: dropped row scale", "        y[t * d_out + i] += s * h[p][i];\n      }\n    }\n  }\n}",
     "        y[t * d_out + i] += s;\n      }\n    }\n  }\n}"),
    ("backward: dropped row scale", "du[i] = dyt[i] * h[p][i];", "du[i] = dyt[i];"),
    ("backward: dropped latent scale in dz", "dz[k] = s * l[p][k];", "dz[k] = s;"),
    ("backward: dl from w", "dl[p][k] += s * z[k];", "dl[p][k] += s * w[k];"),
    ("backward: dg from a", "dg[p][j] += s * xt[j];", "dg[p][j] += s * a[j];"),
    ("backward: surrogate sign", "dU[p][i] *= kappa * (1.0 - th * th);", "dU[p][i] *= kappa * (1.0 + th * th);"),
    ("backward: transposed dV", "dV[p][j * r + k] += a[j] * dz[k];", "dV[p][j * r + k] += a[j] * dz[(k + 1) % r];"),
    ("backward: dx misses g", "dx[t * d_in + j] += s * g[p][j];", "dx[t * d_in + j] += s;"),
]


def _checks_fail_for(lib_path):
    """Run a subset of the pins against a mutated library; returns True if some pin fails."""
    lib = ctypes.CDLL(lib_path)
    vp, i64 = ctypes.c_void_p, ctypes.c_int64
    lib.lbo_forward_factored.argtypes = [vp, i64, i64, i64, i64, vp, vp, vp, vp, vp, ctypes.c_int, vp]
    lib.lbo_forward_factored.restype = None
    lib.lbo_latent.argtypes = [vp, i64, i64, i64, vp, vp, vp, ctypes.c_int, vp]
    lib.lbo_latent.restype = None
    lib.lbo_from_latent.argtypes = [vp, i64, i64, i64, vp, vp, ctypes.c_int, vp]
    lib.lbo_from_latent.restype = None

    def fwd(x, U, V, h, g, l):
        x = np.ascontiguousarray(x, np.float64)
        T, d_in = x.shape
        d_out, r = U[0].shape
        arrs = [[np.ascontiguousarray(a, dt) for a in A] for A, dt in
                ((U, np.int8), (V, np.int8), (h, np.float64), (g, np.float64), (l, np.float64))]
        ptrs = [(ctypes.c_void_p * len(A))(*[a.ctypes.data for a in A]) for A in arrs]
        y = np.empty((T, d_out))
        lib.lbo_forward_factored(x.ctypes.data, T, d_in, d_out, r, *ptrs, len(U), y.ctypes.data)
        return y

    rs = np.random.default_rng(99)
    x, U, V, h, g, l = _rand_layer(rs, 2, 9, 7, 5)
    ok_dense = np.allclose(fwd(x, U, V, h, g, l), O.dense_forward(x, O.dense_weight(U, V, h, g, l)),
                           rtol=1e-12, atol=1e-12)
    fx, xt, Ut, Vt, ht, gt, lt = _load_tiny(os.path.join(os.path.dirname(__file__), "golden"))
    ok_tiny = np.array_equal(fwd(xt, Ut, Vt, ht, gt, lt), np.array(fx["y"], dtype=np.float64))
    # the latent pair composes to the dense result
    arrs = [[np.ascontiguousarray(a, dt) for a in A] for A, dt in
            ((U, np.int8), (V, np.int8), (h, np.float64), (g, np.float64), (l, np.float64))]
    pU, pV, ph, pg, pl = [(ctypes.c_void_p * len(A))(*[a.ctypes.data for a in A]) for A in arrs]
    T, d_in = x.shape
    d_out, r = U[0].shape
    xc = np.ascontiguousarray(x, np.float64)
    w = np.empty((2, T, r))
    lib.lbo_latent(xc.ctypes.data, T, d_in, r, pV, pg, pl, 2, w.ctypes.data)
    y2 = np.empty((T, d_out))
    lib.lbo_from_latent(w.ctypes.data, T, d_out, r, pU, ph, 2, y2.ctypes.data)
    ok_latent = np.allclose(y2, O.dense_forward(x, O.dense_weight(U, V, h, g, l)), rtol=1e-12, atol=1e-12)
    # the backward against the dense route
    lib.lbo_backward.argtypes = [vp, vp, i64, i64, i64, i64, vp, vp, vp, vp, vp, ctypes.c_int, ctypes.c_double,
                                 vp, vp, vp, vp, vp, vp]
    lib.lbo_backward.restype = None
    args = _rand_train_layer(np.random.default_rng(98), 3, 9, 7, 5)
    xb, dyb, Ul, Vl, hb, gb, lb_ = [a if isinstance(a, list) else np.ascontiguousarray(a) for a in args]
    T, d_in = xb.shape
    d_out, r = Ul[0].shape
    outs = {"dU": [np.empty((d_out, r)) for _ in range(2)], "dV": [np.empty((d_in, r)) for _ in range(2)],
            "dh": [np.empty(d_out) for _ in range(2)], "dg": [np.empty(d_in) for _ in range(2)],
            "dl": [np.empty(r) for _ in range(2)]}
    dxb = np.empty((T, d_in))
    pp = lambda A: (ctypes.c_void_p * len(A))(*[np.ascontiguousarray(a).ctypes.data for a in A])
    lib.lbo_backward(xb.ctypes.data, dyb.ctypes.data, T, d_in, d_out, r, pp(Ul), pp(Vl), pp(hb), pp(gb), pp(lb_),
                     2, O.SMOOTHSIGN_K, dxb.ctypes.data, pp(outs["dU"]), pp(outs["dV"]), pp(outs["dh"]),
                     pp(outs["dg"]), pp(outs["dl"]))
    ref = _dense_route(*args, kappa=O.SMOOTHSIGN_K)
    ok_bwd = _close(dxb, ref["dx"], 1e-11) and all(
        _close(outs[k][p], ref[k][p], 1e-6) for k in outs for p in range(2))
    return not (ok_dense and ok_tiny and ok_latent and ok_bwd)


@pytest.mark.parametrize("desc,orig,repl", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_mistakes(tmp_path, desc, orig, repl):
    src = open(os.path.join(os.path.dirname(O.__file__), "lb_oracle.c")).read()
    assert orig in src, desc
    mutated = src.replace(orig, repl, 1)
    cpath = tmp_path / "mut.c"
    cpath.write_text(mutated)
    lpath = str(tmp_path / "libmut.so")
    subprocess.run(["gcc", "-O1", "-fPIC", "-shared", str(cpath), "-o", lpath, "-lm"], check=True)
    assert _checks_fail_for(lpath), desc
