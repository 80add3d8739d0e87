"""GPU parity of the streaming list forward (lb_list_init / lb_list_forward).

Lists of linears of at most two tokens run on the look-up-table kernels: every
linear must give bit for bit what the single-launch look-up-table decode kernel
gives for it (lb_linear_forward_kernel(..., LB_KERNEL_DECODE)) and meet the oracle
bar.  Lists with a linear of more than two tokens run on the matrix-core kernels:
every token of every linear meets the oracle bar of the forward (fp32: relative L2
<= 1e-5; bf16 / f16: max relative error <= 1e-2 per token row), and repeated calls
give the same bits.  Lists mix ragged shapes (tails of d_in, r and d_out, ranks that
are not a multiple of 64 or 16, token counts that are not a multiple of 16), runs
of one and of several blocks, empty linears; the plan check, graph replays and the
Llama2-70B layer shapes are covered for both kinds."""
import numpy as np
import pytest

from paper_2506_13771_amd import synth
import lbtest_utils as U
from conftest import gpu_available

pytestmark = pytest.mark.gpu

if gpu_available():
    import torch
    import paper_2506_13771_amd as lb

from test_parity_gpu import _check


def _linears(specs, cfg, act="bf16", sc="f16", direct=False):
    out = []
    for i, (T, d_in, d_out, r) in enumerate(specs):
        li = synth.make_linear(d_in, d_out, r, T, act_dtype=act, scale_dtype=sc, cfg=cfg, linear=i,
                               direct_words=direct)
        x, paths, _ = U.to_device(li)
        out.append((li, x, paths))
    return out


def _decode_single(lins):
    out = []
    for li, x, paths in lins:
        out.append(lb.lb_linear_forward(x, paths, li.r, kernel=lb.LB_KERNEL_DECODE))
    torch.cuda.synchronize()
    return out


def _same_bits(a, b):
    if a.numel() == 0:
        return b.numel() == 0
    v = torch.int16 if a.element_size() == 2 else torch.int32
    return torch.equal(a.view(v), b.view(v))


def _run_list(lins):
    L = lb.LittleBitList([(x, paths, li.r, None) for li, x, paths in lins])
    ys = L.forward()
    torch.cuda.synchronize()
    return L, ys


RAGGED = [(1, 100, 77, 19), (2, 33, 200, 50), (1, 257, 130, 16), (2, 31, 64, 1), (1, 70, 45, 33),
          (2, 1000, 999, 96), (1, 96, 4100, 48), (1, 1, 1, 1), (2, 4000, 300, 200), (1, 5000, 700, 80),
          (1, 2048, 640, 130), (2, 700, 64, 64), (1, 6500, 2000, 288), (2, 3000, 1500, 176)]


@pytest.mark.parametrize("act,sc", [("bf16", "f16"), ("f32", "f32"), ("f16", "bf16"), ("bf16", "bf16")])
def test_list_ragged_bit_identical_to_decode(act, sc):
    lins = _linears(RAGGED, cfg=40, act=act, sc=sc)
    # scales of both signs: nothing may assume positive scales
    for j, (li, x, paths) in enumerate(lins):
        rs = np.random.default_rng(j)
        for p in range(2):
            li.h[p] = synth.quantize(rs.standard_normal(li.d_out), sc)
            li.g[p] = synth.quantize(rs.standard_normal(li.d_in), sc)
            li.l[p] = synth.quantize(rs.standard_normal(li.r), sc)
            paths[p].h.copy_(U.raw_to_torch(li.h[p], sc))
            paths[p].g.copy_(U.raw_to_torch(li.g[p], sc))
            paths[p].l.copy_(U.raw_to_torch(li.l[p], sc))
    ref = _decode_single(lins)
    L, ys = _run_list(lins)
    for i, ((li, _, _), y, r) in enumerate(zip(lins, ys, ref)):
        assert _same_bits(y, r), (i, RAGGED[i], act, sc)
        _check(li, U.torch_to_raw(y, act), label=f"list {RAGGED[i]} {act}/{sc}")
    assert lb.lb_workspace_status(L.workspace) == 0


def test_list_llama2_70b_layer_shapes():
    """One Llama2-70B layer at 0.1 bits per weight (q, k, v, o, gate, up, down), one token."""
    ranks = {(8192, 8192): 176, (8192, 1024): 16, (8192, 28672): 288, (28672, 8192): 288}
    specs = [(1, d_in, d_out, ranks[(d_in, d_out)]) for _, d_in, d_out in synth.LLAMA2_70B]
    lins = _linears(specs, cfg=4, direct=True)
    ref = _decode_single(lins)
    L, ys = _run_list(lins)
    for i, ((li, _, _), y, r) in enumerate(zip(lins, ys, ref)):
        assert _same_bits(y, r), (i, specs[i])
        _check(li, U.torch_to_raw(y, "bf16"), label=f"70b list {specs[i]}")
    # repeated forwards give the same bits
    for _ in range(3):
        again = L.forward()
        torch.cuda.synchronize()
        for y, r in zip(again, ref):
            assert _same_bits(y, r)


def test_list_empty_members():
    specs = [(1, 512, 384, 32), (1, 64, 64, 16), (2, 300, 200, 40)]
    lins = _linears(specs, cfg=41)
    items = [(x, paths, li.r, None) for li, x, paths in lins]
    # an empty reduction (d_in = 0 and r = 0) gives y = 0; T = 0 and d_out = 0 are skipped
    dev = "cuda"
    zx = torch.empty((3, 0), dtype=torch.bfloat16, device=dev)
    zpaths = [lb.LittleBitPath(U=torch.zeros(64, dtype=torch.uint8, device=dev), V=None,
                               h=torch.ones(16, dtype=torch.float16, device=dev), g=None,
                               l=torch.ones(4, dtype=torch.float16, device=dev)) for _ in range(2)]
    y_empty = torch.full((3, 16), 7.0, dtype=torch.bfloat16, device=dev)
    items.insert(1, (zx, zpaths, 4, y_empty))
    t0x = torch.empty((0, 64), dtype=torch.bfloat16, device=dev)
    items.append((t0x, lins[1][2], 16, None))
    L = lb.LittleBitList(items)
    ys = L.forward()
    torch.cuda.synchronize()
    ref = _decode_single(lins)
    assert _same_bits(ys[0], ref[0]) and _same_bits(ys[2], ref[1]) and _same_bits(ys[3], ref[2])
    assert torch.count_nonzero(y_empty.float()) == 0
    assert ys[4].numel() == 0


def test_list_plan_mismatch_computes_nothing():
    lins = _linears([(1, 512, 384, 32), (1, 640, 256, 48)], cfg=42)
    L, ys = _run_list(lins)
    before = [y.clone() for y in ys]
    # a descriptor array whose output pointer differs from the plan's
    other = torch.full_like(ys[0], 3.0)
    arr, _ = lb.make_descs([(x, paths, li.r, other if i == 0 else ys[i]) for i, (li, x, paths) in enumerate(lins)])
    st = lb.load_library().lb_list_forward(arr, 2, L.workspace.data_ptr(), L.workspace.numel(),
                                           torch.cuda.current_stream().cuda_stream)
    assert st == lb.LB_OK
    torch.cuda.synchronize()
    assert torch.all(other == 3.0)
    assert all(torch.equal(a, b) for a, b in zip(before, ys))
    assert lb.lb_workspace_status(L.workspace) == 2
    assert lb.lb_workspace_status(L.workspace) == 0
    # the matching descriptors still work
    again = L.forward()
    torch.cuda.synchronize()
    assert all(_same_bits(a, b) for a, b in zip(again, before))


def test_list_graph_replays_match_eager():
    specs = [(1, 2048, 1536, 64), (1, 1024, 4096, 80), (2, 512, 512, 32), (1, 8192, 1024, 16), (2, 3000, 700, 130)]
    lins = _linears(specs, cfg=43)
    L, ys = _run_list(lins)
    y_eager = [y.clone() for y in ys]
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        L.forward()
    for rep in range(4):
        for y in ys:
            y.zero_()
        graph.replay()
        torch.cuda.synchronize()
        for i in range(len(lins)):
            assert _same_bits(ys[i], y_eager[i]), (rep, i)
        # eager work on the same workspace between replays
        L.forward()
        torch.cuda.synchronize()
        for i in range(len(lins)):
            assert _same_bits(ys[i], y_eager[i]), (rep, i)


# ---------------------------------------------------------------------------
# lists with linears of more than two tokens: the matrix-core kernels (every
# linear of such a list, whatever its own token count); parity with the oracle
# at the forward's bar, every token compared
# ---------------------------------------------------------------------------
RAGGED_MMA = [(3, 100, 77, 19), (8, 36, 200, 50), (16, 256, 130, 16), (17, 32, 64, 1), (64, 1000, 999, 96),
              (33, 96, 4100, 48), (1, 4, 1, 1), (8, 4000, 300, 200), (5, 5000, 700, 80), (64, 2048, 640, 130),
              (2, 700, 64, 64), (48, 6500, 2000, 288), (8, 3000, 1500, 176), (64, 4096, 4096, 1024)]


@pytest.mark.parametrize("act,sc", [("bf16", "f16"), ("f32", "f32"), ("f16", "bf16"), ("bf16", "bf16")])
def test_mma_list_ragged_matches_oracle(act, sc):
    lins = _linears(RAGGED_MMA, cfg=44, act=act, sc=sc)
    for j, (li, x, paths) in enumerate(lins):
        rs = np.random.default_rng(100 + j)
        for p in range(2):
            li.h[p] = synth.quantize(rs.standard_normal(li.d_out), sc)
            li.g[p] = synth.quantize(rs.standard_normal(li.d_in), sc)
            li.l[p] = synth.quantize(rs.standard_normal(li.r), sc)
            paths[p].h.copy_(U.raw_to_torch(li.h[p], sc))
            paths[p].g.copy_(U.raw_to_torch(li.g[p], sc))
            paths[p].l.copy_(U.raw_to_torch(li.l[p], sc))
    L, ys = _run_list(lins)
    for i, ((li, _, _), y) in enumerate(zip(lins, ys)):
        _check(li, U.torch_to_raw(y, act), label=f"mma list {RAGGED_MMA[i]} {act}/{sc}")
    assert lb.lb_workspace_status(L.workspace) == 0
    # repeated forwards give the same bits (fixed summation order)
    again = L.forward()
    torch.cuda.synchronize()
    assert all(_same_bits(a, b) for a, b in zip(again, ys))


@pytest.mark.parametrize("T", [8, 64])
def test_mma_list_llama2_70b_layer_shapes(T):
    """One Llama2-70B layer at 0.1 bits per weight (q, k, v, o, gate, up, down), T tokens."""
    ranks = {(8192, 8192): 176, (8192, 1024): 16, (8192, 28672): 288, (28672, 8192): 288}
    specs = [(T, d_in, d_out, ranks[(d_in, d_out)]) for _, d_in, d_out in synth.LLAMA2_70B]
    lins = _linears(specs, cfg=5, direct=True)
    L, ys = _run_list(lins)
    for i, ((li, _, _), y) in enumerate(zip(lins, ys)):
        _check(li, U.torch_to_raw(y, "bf16"), label=f"70b mma list {specs[i]}")
    assert lb.lb_workspace_status(L.workspace) == 0


def test_mma_list_plan_mismatch_and_graph_replays():
    specs = [(8, 2048, 1536, 64), (64, 1024, 4096, 80), (3, 512, 512, 32)]
    lins = _linears(specs, cfg=45)
    L, ys = _run_list(lins)
    y_eager = [y.clone() for y in ys]
    other = torch.full_like(ys[0], 3.0)
    arr, _ = lb.make_descs([(x, paths, li.r, other if i == 0 else ys[i]) for i, (li, x, paths) in enumerate(lins)])
    st = lb.load_library().lb_list_forward(arr, len(specs), L.workspace.data_ptr(), L.workspace.numel(),
                                           torch.cuda.current_stream().cuda_stream)
    assert st == lb.LB_OK
    torch.cuda.synchronize()
    assert torch.all(other == 3.0)
    assert lb.lb_workspace_status(L.workspace) == 2
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        L.forward()
    for rep in range(3):
        for y in ys:
            y.zero_()
        graph.replay()
        torch.cuda.synchronize()
        for i in range(len(lins)):
            assert _same_bits(ys[i], y_eager[i]), (rep, i)
        L.forward()
        torch.cuda.synchronize()
        for i in range(len(lins)):
            assert _same_bits(ys[i], y_eager[i]), (rep, i)
    assert lb.lb_workspace_status(L.workspace) == 0
