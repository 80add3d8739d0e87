"""GPU parity of the latent-cache calls (lb_linear_latent, lb_linear_from_latent)
against the oracle's latent and from-latent functions, and their composition
against the prefill forward.

Bars: an fp32 cache must reach relative L2 <= 1e-5 against the oracle latent
(every product exact, fp32 sums); a 16-bit cache must be the round-to-nearest-
even of the fp32 one, bit for bit.  From a cache, the output bars are those of
the forward (fp32: relative L2 <= 1e-5; bf16 / f16: max relative error
<= 1e-2 per token row).  latent then from-latent on an fp32 cache must give
exactly what the prefill forward gives.
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

PREFILL = 2

# (T, d_in, d_out, r, act dtype, scale dtype): several tiles, ragged tails,
# splits of d_in, a benchmark width
SHAPES = [
    (130, 512, 384, 48, "bf16", "f16"),
    (64, 1000, 300, 17, "f32", "f32"),
    (5, 96, 64, 31, "bf16", "bf16"),
    (33, 333, 65, 16, "f16", "f16"),
    (1, 700, 900, 40, "bf16", "f16"),      # T <= 4: the one-launch latent kernel
    (3, 9000, 500, 33, "f32", "f16"),      # ... several LDS chunks, a ragged tail block
    (4, 4096, 4096, 80, "bf16", "f16"),
    (2, 4096, 4096, 544, "f16", "bf16"),
    (200, 4096, 4096, 80, "bf16", "f16"),
    (77, 2048, 1024, 160, "f32", "f16"),
]
SMALL_T = 4  # lb_linear_latent's one-launch kernel takes T <= 4


def _setup(shape, cfg):
    T, d_in, d_out, r, act, sc = shape
    li = synth.make_linear(d_in, d_out, r, T, act_dtype=act, scale_dtype=sc, cfg=cfg)
    x, paths, _ = U.to_device(li)
    return li, x, paths


def _oracle_latent(li, tokens=None):
    """[T, 2, r] (token-major, as the cache stores it) from the oracle (fp64)."""
    _, V, _, _ = U.oracle_signs(li)
    _, g, l = U.oracle_scales(li)
    x = O.to_f64(li.x, li.act_dtype)
    if tokens is not None:
        x = x[tokens]
    return np.ascontiguousarray(O.latent(x, V, g, l).transpose(1, 0, 2))


def _tokens(T):
    return None if T <= 256 else np.unique(np.r_[np.arange(0, T, 37), T - 1])


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_latent_matches_oracle(shape):
    li, x, paths = _setup(shape, cfg=31)
    r = li.r
    w32 = lb.lb_linear_latent(x, paths, r, latent_dtype=torch.float32)
    wb = lb.lb_linear_latent(x, paths, r, latent_dtype=torch.bfloat16)
    wh = lb.lb_linear_latent(x, paths, r, latent_dtype=torch.float16)
    torch.cuda.synchronize()
    assert w32.shape == (li.T, 2, r)
    got = w32.cpu().numpy()
    tokens = _tokens(li.T)
    ref = _oracle_latent(li, tokens)
    got_s = got if tokens is None else got[tokens]
    err = U.rel_l2(got_s.astype(np.float64), ref)
    assert err <= U.TOL_F32_REL_L2, (shape, err)
    # the 16-bit caches are the fp32 latents rounded once
    assert np.array_equal(U.torch_to_raw(wb, "bf16"), synth.quantize(got, "bf16")), shape
    assert np.array_equal(wh.cpu().numpy(), got.astype(np.float16)), shape


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("cache", ["f32", "bf16"])
def test_from_latent_matches_oracle(shape, cache):
    li, _, paths = _setup(shape, cfg=32)
    tokens = _tokens(li.T)
    w64 = _oracle_latent(li)
    # the cache holds the oracle's latents, rounded to the cache dtype on the host
    raw = synth.quantize(w64, cache)
    w_dev = U.raw_to_torch(raw, cache)
    Us, _, _, _ = U.oracle_signs(li)
    h, _, _ = U.oracle_scales(li)
    w_exact = O.to_f64(raw, cache)
    if tokens is not None:
        w_exact = w_exact[tokens]
    ref = O.from_latent(np.ascontiguousarray(w_exact.transpose(1, 0, 2)), Us, h)
    for out in ("f32", "bf16", "f16"):
        y = lb.lb_linear_from_latent(w_dev, paths, out_dtype=U.torch_dtype(out))
        torch.cuda.synchronize()
        yy = O.to_f64(U.torch_to_raw(y, out), out)
        if tokens is not None:
            yy = yy[tokens]
        assert np.all(np.isfinite(yy))
        if out == "f32":
            err = U.rel_l2(yy, ref)
            assert err <= U.TOL_F32_REL_L2, (shape, cache, out, err)
        else:
            err = U.row_inf_rel(yy, ref)
            assert err <= U.TOL_BF16_ROW_INF, (shape, cache, out, err)


@pytest.mark.parametrize("shape", [s for s in SHAPES if s[0] > SMALL_T], ids=lambda s: "x".join(map(str, s)))
def test_latent_then_from_latent_is_the_prefill_forward(shape):
    li, x, paths = _setup(shape, cfg=33)
    w = lb.lb_linear_latent(x, paths, li.r, latent_dtype=torch.float32)
    y = lb.lb_linear_from_latent(w, paths, out_dtype=x.dtype)
    ref = lb.lb_linear_forward(x, paths, li.r, kernel=PREFILL)
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16 if y.element_size() == 2 else torch.int32),
                       ref.view(torch.int16 if ref.element_size() == 2 else torch.int32)), shape


@pytest.mark.parametrize("shape", [s for s in SHAPES if s[0] <= SMALL_T], ids=lambda s: "x".join(map(str, s)))
def test_small_t_latent_then_from_latent_meets_the_forward_bar(shape):
    # the one-launch latent adds in a different order than the prefill stage 1: the composition
    # is checked against the oracle forward instead of bit for bit
    li, x, paths = _setup(shape, cfg=37)
    w = lb.lb_linear_latent(x, paths, li.r, latent_dtype=torch.float32)
    y = lb.lb_linear_from_latent(w, paths, out_dtype=x.dtype)
    torch.cuda.synchronize()
    ref = U.oracle_forward(li)
    got = O.to_f64(U.torch_to_raw(y, li.act_dtype), li.act_dtype)
    if li.act_dtype == "f32":
        assert U.rel_l2(got, ref) <= U.TOL_F32_REL_L2
    else:
        assert U.row_inf_rel(got, ref) <= U.TOL_BF16_ROW_INF


def test_cache_filled_in_steps():
    # a prompt of 150 tokens, then single tokens appended, in one cache buffer;
    # the output over the whole cache meets the forward's bar
    T0, steps, d_in, d_out, r = 150, 6, 1024, 768, 64
    T = T0 + steps
    li = synth.make_linear(d_in, d_out, r, T, act_dtype="bf16", scale_dtype="f16", cfg=34)
    x, paths, _ = U.to_device(li)
    cache = torch.full((T + 10, 2, r), float("nan"), dtype=torch.bfloat16, device="cuda")
    lb.lb_linear_latent(x[:T0], paths, r, w=cache[:T0])
    for s in range(steps):
        t = T0 + s
        lb.lb_linear_latent(x[t:t + 1], paths, r, w=cache[t:t + 1])
    y = lb.lb_linear_from_latent(cache[:T], paths, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    assert torch.isnan(cache[T:].float()).all()  # nothing written past the tokens
    # latents against the oracle (bf16 cache: within one rounding of the fp64 value)
    ref_w = _oracle_latent(li)
    got_w = O.to_f64(U.torch_to_raw(cache[:T], "bf16"), "bf16")
    scale = np.abs(ref_w).max(axis=2, keepdims=True)
    assert np.all(np.abs(got_w - ref_w) <= 2.0 ** -8 * np.abs(ref_w) + 1e-5 * scale)
    # outputs against the oracle forward of x (the bf16 cache is part of the error budget)
    ref_y = U.oracle_forward(li)
    err = U.row_inf_rel(O.to_f64(U.torch_to_raw(y, "bf16"), "bf16"), ref_y)
    assert err <= U.TOL_BF16_ROW_INF, err


def test_latent_edge_cases():
    # d_in == 0: the latents are zero; r == 0: the outputs are zero; T == 0: nothing
    li, x, paths = _setup((9, 64, 48, 16, "bf16", "f16"), cfg=35)
    w = lb.lb_linear_latent(x[:, :0].contiguous(), paths, 16, latent_dtype=torch.float32)
    torch.cuda.synchronize()
    assert w.shape == (9, 2, 16) and bool((w == 0).all())
    y = torch.full((9, 48), 7.0, dtype=torch.bfloat16, device="cuda")
    lb.lb_linear_from_latent(torch.empty((9, 2, 0), dtype=torch.float32, device="cuda"), paths, y=y)
    torch.cuda.synchronize()
    assert bool((y == 0).all())
    w0 = lb.lb_linear_latent(x[:0], paths, 16)
    y0 = lb.lb_linear_from_latent(torch.empty((0, 2, 16), device="cuda"), paths, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    assert w0.shape == (0, 2, 16) and y0.shape == (0, 48)


def test_latent_calls_in_a_graph():
    li, x, paths = _setup((100, 512, 640, 48, "bf16", "f16"), cfg=36)
    ws1 = torch.empty(lb.lb_latent_workspace_bytes(100, 512, 48), dtype=torch.uint8, device="cuda")
    ws2 = torch.empty(lb.lb_from_latent_workspace_bytes(100, 48), dtype=torch.uint8, device="cuda")
    w = lb.lb_linear_latent(x, paths, 48, workspace=ws1)
    y_eager = lb.lb_linear_from_latent(w, paths, out_dtype=torch.bfloat16, workspace=ws2).clone()
    w_g = torch.empty_like(w)
    y_g = torch.empty_like(y_eager)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        lb.lb_linear_latent(x, paths, 48, w=w_g, workspace=ws1)
        lb.lb_linear_from_latent(w_g, paths, y=y_g, workspace=ws2)
    for _ in range(3):
        w_g.zero_()
        y_g.zero_()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(w_g, w) and torch.equal(y_g.view(torch.int16), y_eager.view(torch.int16))
        lb.lb_linear_forward(x, paths, 48)  # eager work between replays
        torch.cuda.synchronize()


@pytest.mark.parametrize("T", [2, 64])
def test_latent_cache_at_the_70b_gate_width(T):
    # 8192 -> 28672 at 0.1 BPW (r = 288 per path): the widest linear of the 70B sweep
    shape = (T, 8192, 28672, 288, "bf16", "f16")
    li, x, paths = _setup(shape, cfg=38)
    w = lb.lb_linear_latent(x, paths, li.r, latent_dtype=torch.bfloat16)
    y = lb.lb_linear_from_latent(w, paths, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    ref_w = _oracle_latent(li)
    got_w = O.to_f64(U.torch_to_raw(w, "bf16"), "bf16")
    scale = np.abs(ref_w).max(axis=2, keepdims=True)
    assert np.all(np.abs(got_w - ref_w) <= 2.0 ** -8 * np.abs(ref_w) + 1e-5 * scale)
    # the output from the bf16 cache, on a sample of tokens, against the oracle forward
    tokens = np.arange(0, T, max(1, T // 8))
    ref_y = U.oracle_forward(li, tokens)
    got_y = O.to_f64(U.torch_to_raw(y, "bf16"), "bf16")[tokens]
    assert U.row_inf_rel(got_y, ref_y) <= U.TOL_BF16_ROW_INF
