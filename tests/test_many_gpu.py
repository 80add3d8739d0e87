"""GPU parity of the list forward (lb_linear_forward_many): every linear of a
list must give exactly what lb_linear_forward gives for it alone (same kernel,
same arithmetic), and that result must meet the oracle bar.  Lists mix shapes,
token counts (look-up-table decode linears batched into list launches, the
rest as single calls), dtypes (which split the list launches), empty linears,
more linears than one list launch takes, repeated calls on one workspace and
graph replays."""
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


def _linears(specs, cfg):
    out = []
    for i, (T, d_in, d_out, r, act, sc) in enumerate(specs):
        li = synth.make_linear(d_in, d_out, r, T, act_dtype=act, scale_dtype=sc, cfg=cfg, linear=i)
        x, paths, _ = U.to_device(li)
        out.append((li, x, paths))
    return out


def _many(lins, ws=None, ys=None):
    items = [(x, paths, li.r, None if ys is None else ys[i]) for i, (li, x, paths) in enumerate(lins)]
    if ws is None:
        arr, _ = lb.make_descs(items)
        need = lb.lb_forward_many_workspace_bytes(arr, len(items))
        ws = lb.lb_workspace_init(torch.empty(max(need, 256), dtype=torch.uint8, device="cuda"))
    out = lb.lb_linear_forward_many(items, workspace=ws)
    torch.cuda.synchronize()
    return out, ws


def _singles(lins):
    out = []
    for li, x, paths in lins:
        out.append(lb.lb_linear_forward(x, paths, li.r))
    torch.cuda.synchronize()
    return out


def _same_bits(a, b):
    if a.numel() == 0:
        return b.numel() == 0
    return torch.equal(a.view(torch.int16 if a.element_size() == 2 else torch.int32),
                       b.view(torch.int16 if b.element_size() == 2 else torch.int32))


MIXED = [
    (1, 4096, 4096, 80, "bf16", "f16"),
    (1, 512, 512, 32, "bf16", "f16"),
    (2, 1000, 300, 48, "bf16", "f16"),
    (1, 700, 900, 17, "bf16", "f16"),
    (2, 4096, 11008, 128, "bf16", "f16"),
    (1, 333, 65, 16, "f32", "f32"),     # another dtype pair: a list launch of its own
    (2, 96, 64, 31, "f32", "f32"),
    (1, 64, 64, 16, "bf16", "f16"),
    (3, 512, 512, 32, "bf16", "f16"),   # T = 3: a single call (matrix-core decode)
    (100, 256, 384, 48, "bf16", "f16"),  # a single call (prefill)
    (0, 64, 64, 16, "bf16", "f16"),     # empty
    (1, 96, 0, 16, "bf16", "f16"),      # empty
]


def test_many_matches_single_calls_and_the_oracle():
    lins = _linears(MIXED, cfg=21)
    ys, _ = _many(lins)
    ref = _singles(lins)
    for i, ((li, _, _), y, r) in enumerate(zip(lins, ys, ref)):
        assert _same_bits(y, r), (i, MIXED[i])
        if li.T > 0 and li.d_out > 0:
            tokens = None if li.T <= 16 else np.arange(0, li.T, 7)
            _check(li, U.torch_to_raw(y, li.act_dtype), tokens=tokens, label=f"many {i}")


def test_many_more_than_one_list_launch():
    specs = [(1 + (i % 2), 128 + 32 * (i % 5), 64 + 16 * (i % 7), 16 * (1 + i % 4), "bf16", "f16")
             for i in range(37)]
    lins = _linears(specs, cfg=22)
    ys, _ = _many(lins)
    ref = _singles(lins)
    for i, (y, r) in enumerate(zip(ys, ref)):
        assert _same_bits(y, r), (i, specs[i])
    for i in (0, 16, 17, 36):
        _check(lins[i][0], U.torch_to_raw(ys[i], "bf16"), label=f"long list {i}")


def test_many_matrix_core_decode_lists():
    # T = 3 .. 64 linears that the matrix-core decode kernel takes, in runs
    # broken by a look-up-table linear, a prefill-sized one and a dtype change
    specs = [(8, 1024, 1024, 80, "bf16", "f16"), (16, 512, 768, 48, "bf16", "f16"),
             (3, 700, 900, 17, "bf16", "f16"), (64, 256, 512, 32, "bf16", "f16"),
             (1, 512, 512, 32, "bf16", "f16"), (8, 2048, 1024, 64, "bf16", "f16"),
             (40, 512, 4096, 128, "bf16", "f16"), (5, 96, 64, 31, "f32", "f32"),
             (8, 64, 160, 16, "f32", "f32")] + [(4 + i, 256 + 64 * i, 128 + 32 * i, 16 + 16 * (i % 3), "bf16", "f16")
                                                for i in range(18)]
    lins = _linears(specs, cfg=25)
    ys, _ = _many(lins)
    ref = _singles(lins)
    for i, ((li, _, _), y, r) in enumerate(zip(lins, ys, ref)):
        assert _same_bits(y, r), (i, specs[i])
    for i in (0, 3, 7, 26):
        _check(lins[i][0], U.torch_to_raw(ys[i], specs[i][4]), label=f"mma list {i}")


def test_many_repeated_calls_on_one_workspace():
    specs = [(1, 4096, 4096, 80, "bf16", "f16"), (2, 1024, 2048, 48, "bf16", "f16"),
             (1, 2048, 512, 64, "bf16", "f16"), (8, 1024, 1024, 80, "bf16", "f16"),
             (16, 2048, 512, 64, "bf16", "f16")]
    lins = _linears(specs, cfg=23)
    ws = None
    g = torch.Generator(device="cuda").manual_seed(23)
    for rep in range(4):
        if rep:
            for _, x, _ in lins:
                x.copy_(torch.randn(x.shape, generator=g, device="cuda").to(x.dtype))
        ys, ws = _many(lins, ws=ws)
        ref = _singles(lins)
        for i, (y, r) in enumerate(zip(ys, ref)):
            assert _same_bits(y, r), (rep, i)


def test_many_graph_replays_match_eager():
    specs = [(1, 2048, 1536, 64, "bf16", "f16"), (1, 1024, 4096, 80, "bf16", "f16"),
             (2, 512, 512, 32, "bf16", "f16"), (16, 512, 768, 48, "bf16", "f16"),
             (8, 1024, 1024, 80, "bf16", "f16")]
    lins = _linears(specs, cfg=24)
    y_eager, ws = _many(lins)
    y_eager = [y.clone() for y in y_eager]
    y_graph = [torch.empty_like(y) for y in y_eager]
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        lb.lb_linear_forward_many([(x, paths, li.r, y_graph[i]) for i, (li, x, paths) in enumerate(lins)],
                                  workspace=ws)
    for rep in range(4):
        for y in y_graph:
            y.zero_()
        graph.replay()
        torch.cuda.synchronize()
        y_mid, _ = _many(lins, ws=ws)  # eager work on the same workspace between replays
        for i in range(len(lins)):
            assert _same_bits(y_graph[i], y_eager[i]), (rep, i)
            assert _same_bits(y_mid[i], y_eager[i]), (rep, i)


def test_many_one_token_lists_of_every_row_block_count():
    # one-token list launches give each stage-2 workgroup 4, 2 or 1 blocks of 64 rows by the U
    # words a lane holds (ranks up to 256, up to 512, above); ragged row counts leave the last
    # workgroup's blocks partly or wholly past d_out
    for specs in ([(1, 640, 900, 200, "bf16", "f16"), (1, 512, 70, 64, "bf16", "f16"), (1, 300, 1000, 96, "bf16", "f16")],
                  [(1, 1024, 700, 300, "bf16", "f16"), (1, 512, 65, 200, "bf16", "f16"), (1, 2048, 2112, 288, "bf16", "f16")],
                  [(1, 1024, 777, 600, "bf16", "f16"), (1, 640, 130, 40, "bf16", "f16")]):
        lins = _linears(specs, cfg=26)
        ys, _ = _many(lins)
        ref = _singles(lins)
        for i, ((li, _, _), y, r) in enumerate(zip(lins, ys, ref)):
            assert _same_bits(y, r), (i, specs[i])
            _check(li, U.torch_to_raw(y, "bf16"), label=f"row blocks {specs[i]}")


def test_many_large_lists_launch_stage_one_apart():
    # lists with more than 1024 stage-1 workgroups go out as a stage-1 launch and a stage-2 launch;
    # the second list has an unaligned member (element-wise loads, four-token tables whose LDS
    # exceeds the default limit) and mixed token counts
    for specs in ([(1, 8192, 2048, 176, "bf16", "f16")] * 5 + [(1, 4096, 3000, 288, "bf16", "f16"),
                                                                (1, 7000, 1100, 100, "bf16", "f16")],
                  [(2, 8192, 1024, 176, "bf16", "f16")] * 4 + [(2, 8190, 700, 160, "bf16", "f16"),
                                                               (1, 6000, 900, 300, "bf16", "f16")]):
        lins = _linears(specs, cfg=27)
        ys, ws = _many(lins)
        ref = _singles(lins)
        for i, ((li, _, _), y, r) in enumerate(zip(lins, ys, ref)):
            assert _same_bits(y, r), (i, specs[i])
            _check(li, U.torch_to_raw(y, "bf16"), label=f"split list {specs[i]}")
        again, _ = _many(lins, ws=ws)  # the same workspace again: the call protocol's next epoch
        for i in range(len(lins)):
            assert _same_bits(again[i], ys[i]), i


def test_many_layouts_change_on_one_workspace():
    """One workspace serves lists of different layouts in turn ([A], then [B, A], then [A]
    again, several times): linear A's intermediate values move between calls while the control
    block stays at the start of the workspace, so every result must still be bit-identical to
    A's (and B's) single call, and the workspace's error word must stay clear."""
    lins = _linears([(1, 8192, 2048, 176, "bf16", "f16"), (1, 512, 512, 32, "bf16", "f16"),
                     (8, 1024, 1024, 80, "bf16", "f16")], cfg=28)
    ref = _singles(lins)
    layouts = ([0], [1, 0], [2, 1, 0], [0], [0, 2])
    need = 0
    for idx in layouts:
        arr, _ = lb.make_descs([(lins[i][1], lins[i][2], lins[i][0].r, None) for i in idx])
        need = max(need, lb.lb_forward_many_workspace_bytes(arr, len(idx)))
    ws = lb.lb_workspace_init(torch.empty(need, dtype=torch.uint8, device="cuda"))
    for rep in range(3):
        for idx in layouts:
            ys, _ = _many([lins[i] for i in idx], ws=ws)
            for i, y in zip(idx, ys):
                assert _same_bits(y, ref[i]), (rep, idx, i)
    assert lb.lb_workspace_status(ws) == 0


def test_workspace_status_after_calls():
    """The error word of a workspace reads 0 after calls of every decode kernel and a list on
    it (no bounded wait expired), and reading it clears it."""
    lins = _linears([(1, 4096, 4096, 80, "bf16", "f16"), (3, 1024, 2048, 48, "bf16", "f16"),
                     (2, 8192, 1024, 16, "bf16", "f16")], cfg=29)
    need = max(lb.lb_forward_workspace_bytes(li.T, li.d_in, li.d_out, li.r) for li, _, _ in lins)
    ws = lb.lb_workspace_init(torch.empty(need, dtype=torch.uint8, device="cuda"))
    for li, x, paths in lins:
        for k in (lb.LB_KERNEL_AUTO, lb.LB_KERNEL_DECODE, lb.LB_KERNEL_DECODE_MFMA):
            lb.lb_linear_forward(x, paths, li.r, workspace=ws, kernel=k)
    torch.cuda.synchronize()
    assert lb.lb_workspace_status(ws) == 0
    _, ws2 = _many(lins)
    assert lb.lb_workspace_status(ws2) == 0
    assert lb.lb_workspace_status(ws2) == 0
