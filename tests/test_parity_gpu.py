"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle on the
same seeded inputs.

Bars: packing is bit-exact; fp32 activations must reach relative L2 <= 1e-5;
bf16 / f16 activations (fp32 accumulation) must reach max relative error
<= 1e-2 per token row (max_i |y - y*| / max_i |y*|).  Sizes span several
tiles and ragged tails; the benchmark shapes run at full size and every token
of every output is compared with the oracle.
"""
import numpy as np
import pytest

import oracle as O
from paper_2506_13771_amd import synth
import lbtest_utils as U
from conftest import gpu_available

pytestmark = pytest.mark.gpu

if gpu_available():
    import torch
    import paper_2506_13771_amd as lb

KERNELS = {"decode": 1, "prefill": 2, "auto": 0, "mma": 3}
MMA_MAX_T, MMA_MAX_R = 64, 832


def _run(li, kernel="auto", pack_on_gpu=True):
    x, paths, _ = U.to_device(li, pack_on_gpu)
    y = lb.lb_linear_forward(x, paths, li.r, kernel=KERNELS[kernel])
    torch.cuda.synchronize()
    return U.torch_to_raw(y, li.act_dtype)


def _check(li, y_raw, tokens=None, label=""):
    ref = U.oracle_forward(li, tokens)
    y = O.to_f64(y_raw, li.act_dtype)
    if tokens is not None:
        y = y[tokens]
    assert np.all(np.isfinite(y)), label
    if li.act_dtype == "f32":
        err = U.rel_l2(y, ref)
        assert err <= U.TOL_F32_REL_L2, (label, err)
    else:
        err = U.row_inf_rel(y, ref)
        assert err <= U.TOL_BF16_ROW_INF, (label, err, U.rel_l2(y, ref))
    return err


# ---------------------------------------------------------------------------
# packing: bit-exact against the oracle packer
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("rows,r", [(512, 32), (4096, 80), (11008, 128), (4096, 544), (1024, 16), (33, 7),
                                    (40, 50), (100, 17), (1, 1), (64, 31)])
@pytest.mark.parametrize("dt", ["f32", "bf16", "f16"])
def test_pack_bit_exact(rows, r, dt):
    rs = np.random.default_rng(rows * 13 + r)
    src64 = rs.standard_normal((rows, r))
    src64[0, 0] = -0.0
    raw = synth.quantize(src64, dt)
    src_t = U.raw_to_torch(raw, dt)
    src_exact = O.to_f64(raw, dt)
    for role in (lb.LB_ROLE_U, lb.LB_ROLE_V):
        got = lb.lb_pack_signs(src_t, role)
        torch.cuda.synchronize()
        ref, _ = O.pack(src_exact, role)
        assert got.cpu().numpy().tobytes() == ref.tobytes(), (rows, r, dt, role)


def test_pack_nan_count():
    src = torch.randn(64, 48, device="cuda")
    src[3, 5] = float("nan")
    src[10, 40] = float("nan")
    cnt = torch.zeros(1, dtype=torch.int32, device="cuda")
    got = lb.lb_pack_signs(src, lb.LB_ROLE_V, nan_count=cnt)
    torch.cuda.synchronize()
    assert int(cnt.item()) == 2
    ref, nans = O.pack(src.cpu().double().numpy(), O.ROLE_V)
    assert nans == 2 and got.cpu().numpy().tobytes() == ref.tobytes()


# ---------------------------------------------------------------------------
# forward: configuration 0 (512x512, r=32, T=4, fp32) on every kernel, and vs dense
# ---------------------------------------------------------------------------
def cfg0():
    return synth.make_linear(512, 512, 32, 4, act_dtype="f32", scale_dtype="f32", cfg=0, l_over_sqrt_r=True)


@pytest.mark.parametrize("kernel", ["decode", "prefill", "mma", "auto"])
def test_cfg0_fp32(kernel):
    li = cfg0()
    y = _run(li, kernel)
    _check(li, y, label=f"cfg0 {kernel}")
    # also against the brute-force dense reconstruction (Proposition 1 identity)
    Us, Vs, _, _ = U.oracle_signs(li)
    h, g, l = U.oracle_scales(li)
    Wd = O.dense_weight(Us, Vs, h, g, l)
    ref = O.dense_forward(O.to_f64(li.x, "f32"), Wd)
    assert U.rel_l2(O.to_f64(y, "f32"), ref) <= U.TOL_F32_REL_L2


def test_dense_reference_weight_cfg0():
    li = cfg0()
    x, paths, _ = U.to_device(li)
    W = lb.lb_dense_reference_weight(paths, li.d_in, li.d_out, li.r)
    torch.cuda.synchronize()
    Us, Vs, _, _ = U.oracle_signs(li)
    h, g, l = U.oracle_scales(li)
    ref = O.dense_weight(Us, Vs, h, g, l)
    err = np.abs(W.cpu().double().numpy() - ref).max() / np.abs(ref).max()
    assert err <= 1e-6, err


# ---------------------------------------------------------------------------
# configuration 1: Llama2-7B q_proj 4096x4096 at 0.1 BPW (r=80), T=1, bf16
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("kernel", ["auto", "prefill", "mma"])
def test_cfg1_q_proj(kernel):
    li = synth.make_linear(4096, 4096, 80, 1, cfg=1)
    _check(li, _run(li, kernel), label=f"cfg1 {kernel}")


# ---------------------------------------------------------------------------
# configuration 2: all 7 linears of a Llama2-7B block at 0.1 / 0.55 BPW, T in {1, 16, 64}
# ---------------------------------------------------------------------------
RANKS_7B = {0.1: {4096: 80, 11008: 128}, 0.55: {4096: 544, 11008: 800}}


def _rank_7b(bpw, d_in, d_out):
    return RANKS_7B[bpw][max(d_in, d_out)]


@pytest.mark.parametrize("bpw", [0.1, 0.55])
@pytest.mark.parametrize("T", [1, 16, 64])
def test_cfg2_llama2_7b_block(bpw, T):
    for li_idx, (name, d_in, d_out) in enumerate(synth.LLAMA2_7B):
        r = _rank_7b(bpw, d_in, d_out)
        assert lb.lb_rank_for_bpw(d_in, d_out, bpw, 16) == r
        li = synth.make_linear(d_in, d_out, r, T, cfg=2, linear=li_idx + (100 if bpw > 0.5 else 0))
        _check(li, _run(li), label=f"cfg2 {name} bpw={bpw} T={T}")


@pytest.mark.parametrize("T", [1, 2, 4])
def test_cfg2_both_kernels_agree_with_oracle(T):
    li = synth.make_linear(11008, 4096, 128, T, cfg=2, linear=50)
    for k in ("decode", "prefill", "mma"):
        _check(li, _run(li, k), label=f"down T={T} {k}")


@pytest.mark.parametrize("d_in,d_out,r", [(4096, 4096, 544), (11008, 4096, 800), (4096, 11008, 800),
                                          (8192, 28672, 288), (28672, 8192, 288), (8192, 1024, 16)])
@pytest.mark.parametrize("T", [1, 3])
def test_decode_large_rank_and_long_inputs(d_in, d_out, r, T):
    """Decode geometry extremes: two-level reduction (many d_in runs), 16 lanes per
    output row, several rows per lane."""
    li = synth.make_linear(d_in, d_out, r, T, cfg=11, linear=d_in + r, direct_words=True)
    _check(li, _run(li, "decode"), label=f"decode {d_in}x{d_out} r={r} T={T}")


@pytest.mark.parametrize("d_in,d_out,r", [(4096, 4096, 544), (11008, 4096, 800), (4096, 11008, 800),
                                          (8192, 28672, 288), (28672, 8192, 288), (8192, 1024, 16),
                                          (4000, 3000, 832)])
@pytest.mark.parametrize("T", [5, 16, 33, 64])
def test_mma_large_rank_and_long_inputs(d_in, d_out, r, T):
    """Matrix-core decode geometry extremes: many d_in runs (two-level sums), the
    largest rank it takes, 1 to 4 token fragments."""
    li = synth.make_linear(d_in, d_out, r, T, cfg=12, linear=d_in + r + T, direct_words=True)
    _check(li, _run(li, "mma"), label=f"mma {d_in}x{d_out} r={r} T={T}")


# ---------------------------------------------------------------------------
# configuration 3: Llama2-13B block shapes at 0.1 BPW, prefill T=2048
# ---------------------------------------------------------------------------
RANKS_13B = {(5120, 5120): 96, (5120, 13824): 160, (13824, 5120): 160}


@pytest.mark.parametrize("which", range(7))
def test_cfg3_llama2_13b_prefill(which):
    name, d_in, d_out = synth.LLAMA2_13B[which]
    r = RANKS_13B[(d_in, d_out)]
    li = synth.make_linear(d_in, d_out, r, 2048, cfg=3, linear=which)
    # every token: all 32 token tiles of 64 and every 16-token subtile of the MFMA path
    _check(li, _run(li), label=f"cfg3 {name}")


# ---------------------------------------------------------------------------
# configuration 4: Llama2-70B linear shapes at 0.1 BPW, T in {1, 8, 64}
# (packed words drawn directly, read by the oracle through its own unpacker)
# ---------------------------------------------------------------------------
RANKS_70B = {(8192, 8192): 176, (8192, 1024): 16, (8192, 28672): 288, (28672, 8192): 288}


@pytest.mark.parametrize("T", [1, 8, 64])
def test_cfg4_llama2_70b_shapes(T):
    for which, (name, d_in, d_out) in enumerate(synth.LLAMA2_70B):
        if name in ("k", "up", "o"):
            continue  # same shapes as v, gate and q
        r = RANKS_70B[(d_in, d_out)]
        li = synth.make_linear(d_in, d_out, r, T, cfg=4, linear=which, direct_words=True)
        _check(li, _run(li), label=f"cfg4 {name} T={T}")


# ---------------------------------------------------------------------------
# ragged shapes, dtypes, edge cases
# ---------------------------------------------------------------------------
RAGGED = [(100, 77, 19, 3), (33, 200, 50, 5), (257, 130, 16, 1), (31, 64, 1, 2), (70, 45, 33, 9),
          (1000, 999, 96, 16), (96, 4100, 48, 70), (1, 1, 1, 1), (5, 3, 2, 130)]


@pytest.mark.parametrize("d_in,d_out,r,T", RAGGED)
@pytest.mark.parametrize("kernel", ["decode", "prefill", "mma"])
@pytest.mark.parametrize("act,sc", [("bf16", "f16"), ("f32", "f32"), ("f16", "bf16"), ("f16", "f32"),
                                    ("bf16", "bf16")])
def test_ragged(d_in, d_out, r, T, kernel, act, sc):
    if kernel == "decode" and T > lb.lb_decode_max_tokens():
        pytest.skip("decode kernel covers small T only")
    if kernel == "mma" and (T > MMA_MAX_T or r > MMA_MAX_R):
        pytest.skip("matrix-core decode kernel covers T <= 64, r <= 832")
    li = synth.make_linear(d_in, d_out, r, T, act_dtype=act, scale_dtype=sc, cfg=9,
                           linear=d_in * 7 + d_out * 3 + r + T)
    # scales of both signs: nothing in the kernels may assume positive scales
    rs = np.random.default_rng(d_in + d_out)
    for p in range(2):
        li.h[p] = synth.quantize(rs.standard_normal(d_out), sc)
        li.g[p] = synth.quantize(rs.standard_normal(d_in), sc)
        li.l[p] = synth.quantize(rs.standard_normal(r), sc)
    _check(li, _run(li, kernel), label=f"ragged {d_in}x{d_out} r={r} T={T} {kernel} {act}/{sc}")


@pytest.mark.parametrize("T,d_in,d_out,r", [(0, 64, 64, 16), (4, 0, 64, 16), (4, 64, 64, 0), (4, 64, 0, 16)])
@pytest.mark.parametrize("kernel", ["decode", "prefill", "mma", "auto"])
def test_degenerate_sizes(T, d_in, d_out, r, kernel):
    li = synth.make_linear(max(d_in, 1), max(d_out, 1), max(r, 1), max(T, 1), cfg=8)
    x = torch.randn(T, d_in, device="cuda").to(torch.bfloat16)
    paths = []
    for p in range(2):
        paths.append(lb.LittleBitPath(
            U=torch.zeros(max(lb.lb_packed_bytes(lb.LB_ROLE_U, d_out, r), 4), dtype=torch.uint8, device="cuda"),
            V=torch.zeros(max(lb.lb_packed_bytes(lb.LB_ROLE_V, d_in, r), 4), dtype=torch.uint8, device="cuda"),
            h=torch.ones(d_out, dtype=torch.float16, device="cuda"),
            g=torch.ones(d_in, dtype=torch.float16, device="cuda"),
            l=torch.ones(r, dtype=torch.float16, device="cuda")))
    y = torch.full((T, d_out), 7.0, dtype=torch.bfloat16, device="cuda")
    lb.lb_linear_forward(x, paths, r, y=y, kernel=KERNELS[kernel])
    torch.cuda.synchronize()
    assert torch.all(y == 0).item() or y.numel() == 0
    del li


def test_single_path_via_zero_residual_h():
    li = synth.make_linear(256, 192, 32, 3, cfg=7)
    li.h[1] = synth.quantize(np.zeros(192), "f16")
    y = _run(li)
    Us, Vs, _, _ = U.oracle_signs(li)
    h, g, l = U.oracle_scales(li)
    ref = O.forward_factored(O.to_f64(li.x, "bf16"), Us[:1], Vs[:1], h[:1], g[:1], l[:1])
    assert U.row_inf_rel(O.to_f64(y, "bf16"), ref) <= U.TOL_BF16_ROW_INF


def test_fp16_subnormal_scales_exact():
    """fp16 scales include subnormals; they must be widened exactly (fp32 activations)."""
    li = synth.make_linear(128, 128, 16, 2, act_dtype="f32", scale_dtype="f16", cfg=6)
    for p in range(2):
        g = li.g[p].copy()
        g[::7] = 0x0001 + (np.arange(g[::7].size) % 0x3FF).astype(np.uint16)  # subnormal fp16 patterns
        li.g[p] = g
    for k in ("decode", "prefill"):
        _check(li, _run(li, k), label=f"subnormal {k}")


# ---------------------------------------------------------------------------
# determinism and workspace reuse (counters must reset themselves)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("T,kernel", [(1, "decode"), (1, "mma"), (16, "mma"), (64, "mma")])
def test_decode_bitwise_deterministic(T, kernel):
    li = synth.make_linear(4096, 4096, 80, T, cfg=1)
    x, paths, _ = U.to_device(li)
    ws = lb.alloc_workspace(T, 4096, 4096, 80)
    ys = []
    for _ in range(20):
        ys.append(lb.lb_linear_forward(x, paths, 80, workspace=ws, kernel=KERNELS[kernel]).clone())
    torch.cuda.synchronize()
    for y in ys[1:]:
        assert torch.equal(y.view(torch.int16), ys[0].view(torch.int16))


def test_workspace_reuse_across_shapes():
    shapes = [(1, 4096, 4096, 80), (16, 4096, 11008, 128), (3, 512, 512, 32), (100, 1000, 300, 48),
              (1, 4096, 4096, 80), (8, 11008, 4096, 800), (2, 700, 900, 17), (64, 2048, 2048, 64)]
    max_ws = max(lb.lb_forward_workspace_bytes(*s) for s in shapes)
    ws = torch.zeros(max_ws, dtype=torch.uint8, device="cuda")
    for rep in range(2):
        for i, (T, d_in, d_out, r) in enumerate(shapes):
            li = synth.make_linear(d_in, d_out, r, T, cfg=5, linear=i)
            x, paths, _ = U.to_device(li)
            y = lb.lb_linear_forward(x, paths, r, workspace=ws)
            torch.cuda.synchronize()
            tokens = None if T <= 16 else np.arange(0, T, 9)
            _check(li, U.torch_to_raw(y, "bf16"), tokens=tokens, label=f"reuse {i} rep {rep}")
    # the control block is back to its idle state (word 0 holds the decode call
    # tag; every counter and the error word are zero)
    ctrl_bytes = lb.lb_forward_workspace_bytes(0, 0, 0, 0)
    ctrl = ws[:ctrl_bytes].view(torch.int32)
    assert int(ctrl[0].item()) > 0
    assert int(ctrl[1:].abs().sum().item()) == 0


def test_back_to_back_launches_stress():
    """Many back-to-back decode launches with changing inputs on one workspace; every
    result checked against a GPU-side dense reference built by the checking kernel."""
    d_in, d_out, r, T = 1024, 1024, 48, 2
    li = synth.make_linear(d_in, d_out, r, T, cfg=4, linear=77)
    x0, paths, _ = U.to_device(li)
    W = lb.lb_dense_reference_weight(paths, d_in, d_out, r)
    ws = lb.alloc_workspace(T, d_in, d_out, r)
    g = torch.Generator(device="cuda").manual_seed(5)
    outs, xs = [], []
    for i in range(300):
        x = torch.randn(T, d_in, device="cuda", generator=g).to(torch.bfloat16)
        xs.append(x)
        outs.append(lb.lb_linear_forward(x, paths, r, workspace=ws))
    torch.cuda.synchronize()
    for x, y in zip(xs, outs):
        ref = x.float() @ W.t()
        err = ((y.float() - ref).abs().max(dim=1).values / ref.abs().max(dim=1).values).max().item()
        assert err <= U.TOL_BF16_ROW_INF, err


@pytest.mark.parametrize("T,kernel", [(1, "decode"), (4, "decode"), (16, "mma"), (100, "prefill")])
def test_graph_replays_match_eager(T, kernel):
    """Launches captured in a HIP graph: every replay (with eager work and syncs in
    between) must reproduce the eager result."""
    li = synth.make_linear(2048, 1536, 64, T, cfg=10, linear=T)
    x, paths, _ = U.to_device(li)
    ws = lb.alloc_workspace(T, 2048, 1536, 64)
    y_eager = lb.lb_linear_forward(x, paths, 64, workspace=ws, kernel=KERNELS[kernel]).clone()
    torch.cuda.synchronize()
    y_graph = torch.empty_like(y_eager)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        lb.lb_linear_forward(x, paths, 64, y=y_graph, workspace=ws, kernel=KERNELS[kernel])
    for rep in range(5):
        y_graph.zero_()
        g.replay()
        torch.cuda.synchronize()
        # eager work on the same workspace between replays
        y_mid = lb.lb_linear_forward(x, paths, 64, workspace=ws, kernel=KERNELS[kernel])
        torch.cuda.synchronize()
        if kernel in ("decode", "mma"):
            assert torch.equal(y_graph.view(torch.int16), y_eager.view(torch.int16)), rep
            assert torch.equal(y_mid.view(torch.int16), y_eager.view(torch.int16)), rep
        else:
            _check(li, U.torch_to_raw(y_graph, "bf16"), label=f"graph replay {rep}")
            _check(li, U.torch_to_raw(y_mid, "bf16"), label=f"eager between replays {rep}")
