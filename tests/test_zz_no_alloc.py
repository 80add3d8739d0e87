"""The no-allocation forward (lb_linear_forward_noalloc), for callers that cannot
allocate: called through the C ABI on two calls in a row, the second with a
smaller input, its outputs must equal lb_linear_forward's (same kernels, same
arithmetic: bit for bit) and meet the oracle bar; sizes beyond the scratch are
rejected.  Runs alone in a fresh process or after the other tests."""
import ctypes

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


def _noalloc_raw(lib, li, x, paths, y):
    arr, sc = lb._paths_struct(paths)
    return lib.lb_linear_forward_noalloc(ctypes.c_void_p(x.data_ptr()), lb._dtype_code(x), li.T, li.d_in, li.d_out,
                                         li.r, arr, sc, ctypes.c_void_p(y.data_ptr()),
                                         ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))


def _same_bits(a, b):
    v = torch.int16 if a.element_size() == 2 else torch.int32
    return torch.equal(a.view(v), b.view(v))


@pytest.mark.parametrize("first,second", [
    ((64, 2048, 1024, 96, "bf16", "f16"), (1, 512, 384, 32, "bf16", "f16")),
    ((1, 4096, 4096, 80, "bf16", "f16"), (1, 1000, 999, 96, "f32", "f32")),
    ((300, 1024, 768, 64, "bf16", "f16"), (3, 700, 900, 17, "f16", "bf16")),
])
def test_noalloc_matches_workspace_call_twice(first, second):
    lib = lb.load_library()
    assert lib.lb_noalloc_scratch_bytes() == 32 << 20
    for k, (T, d_in, d_out, r, act, sc) in enumerate((first, second)):
        li = synth.make_linear(d_in, d_out, r, T, act_dtype=act, scale_dtype=sc, cfg=60, linear=k)
        x, paths, _ = U.to_device(li)
        y = torch.full((T, d_out), float("nan"), dtype=x.dtype, device="cuda")
        assert _noalloc_raw(lib, li, x, paths, y) == lb.LB_OK, (k, first, second)
        ref = lb.lb_linear_forward(x, paths, r)
        torch.cuda.synchronize()
        assert _same_bits(y, ref), (k, first, second)
        _check(li, U.torch_to_raw(y, act), label=f"noalloc {k}")
    # repeated calls on the shared scratch keep giving the same result
    y2 = torch.empty_like(y)
    assert _noalloc_raw(lib, li, x, paths, y2) == lb.LB_OK
    torch.cuda.synchronize()
    assert _same_bits(y2, ref)


def test_noalloc_rejects_sizes_beyond_the_scratch():
    lib = lb.load_library()
    li = synth.make_linear(64, 64, 16, 1, cfg=61)
    x, paths, _ = U.to_device(li)
    arr, sc = lb._paths_struct(paths)
    y = torch.empty((1, 64), dtype=x.dtype, device="cuda")
    # a workspace need far above 32 MiB (a long prefill of a wide layer)
    st = lib.lb_linear_forward_noalloc(ctypes.c_void_p(x.data_ptr()), lb._dtype_code(x), 65536, 16384, 16384, 256,
                                       arr, sc, ctypes.c_void_p(y.data_ptr()), None)
    assert st == lb.LB_ERR_WORKSPACE
