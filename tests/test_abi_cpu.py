"""CPU tests of the C-ABI boundary: the library loads, exports every function
include/littlebit.h declares, its pure host helpers agree with the oracle's,
and every validation error is returned before anything is enqueued (so none
of these calls needs a GPU)."""
import ctypes
import os
import re

import pytest

import oracle as O
import paper_2506_13771_amd as lb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "littlebit.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(lb.LIB_PATH):
        from paper_2506_13771_amd import _build
        _build.build()
    return lb.load_library()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lb_[a-z_0-9]+)\s*\(", text)))


def test_header_declares_the_boundary():
    fns = declared_functions()
    for name in ["lb_pack_signs", "lb_linear_forward", "lb_dense_reference_weight", "lb_packed_bytes",
                 "lb_rank_for_bpw", "lb_forward_workspace_bytes"]:
        assert name in fns


def test_exports_every_declared_symbol(lib):
    raw = ctypes.CDLL(lb.LIB_PATH)
    missing = [f for f in declared_functions() if not hasattr(raw, f)]
    assert not missing, missing


def test_abi_version_and_status_strings(lib):
    assert lib.lb_abi_version() == lb.ABI_VERSION
    for code, name in [(0, "LB_OK"), (1, "LB_ERR_NULL"), (2, "LB_ERR_SHAPE"), (3, "LB_ERR_DTYPE"),
                       (4, "LB_ERR_ALIGN"), (5, "LB_ERR_WORKSPACE"), (6, "LB_ERR_HIP"), (7, "LB_ERR_ARG")]:
        assert lb.lb_status_str(code) == name


@pytest.mark.parametrize("rows,r", [(4096, 80), (11008, 128), (28672, 288), (1024, 16), (40, 50), (33, 7),
                                    (1, 1), (0, 5), (7, 0), (5, 17)])
def test_packed_bytes_matches_oracle(lib, rows, r):
    assert lb.lb_packed_bytes(lb.LB_ROLE_U, rows, r) == O.packed_bytes(rows, r, O.ROLE_U)
    assert lb.lb_packed_bytes(lb.LB_ROLE_V, rows, r) == O.packed_bytes(rows, r, O.ROLE_V)


def test_packed_bytes_invalid(lib):
    assert lb.lb_packed_bytes(5, 10, 10) == 0
    assert lb.lb_packed_bytes(lb.LB_ROLE_U, -1, 10) == 0


@pytest.mark.parametrize("d_in,d_out,b", [(4096, 4096, 0.1), (4096, 4096, 0.55), (4096, 11008, 0.1),
                                          (11008, 4096, 0.55), (5120, 13824, 0.1), (8192, 1024, 0.1),
                                          (28672, 8192, 0.1), (100, 37, 0.9), (64, 64, 0.01)])
def test_rank_and_bpw_match_oracle(lib, d_in, d_out, b):
    assert lb.lb_rank_for_bpw(d_in, d_out, b, 16) == O.rank_for_bpw(d_in, d_out, b, 16, 1)
    assert lb.lb_rank_for_bpw(d_in, d_out, b, 1) == O.rank_for_bpw(d_in, d_out, b, 1, 1)
    for r in (0, 16, 80, 288):
        assert lb.lb_bits_per_weight(d_in, d_out, r, 2) == pytest.approx(O.bpw(d_in, d_out, r, 2), rel=1e-15)
        assert lb.lb_bits_per_weight(d_in, d_out, r, 1) == pytest.approx(O.bpw(d_in, d_out, r, 1), rel=1e-15)


def test_rank_invalid(lib):
    assert lb.lb_rank_for_bpw(0, 10, 0.1, 16) == -1
    assert lb.lb_rank_for_bpw(10, 10, 0.1, 0) == -1
    assert lb.lb_rank_for_bpw(10, 10, float("nan"), 16) == -1
    assert lb.lb_bits_per_weight(10, 10, 3, 3) == -1.0


def test_workspace_sizes(lib):
    for T, d_in, d_out, r in [(1, 4096, 4096, 80), (64, 11008, 4096, 800), (2048, 5120, 13824, 160),
                              (4, 512, 512, 32), (3, 33, 17, 5), (0, 10, 10, 2)]:
        n = lb.lb_forward_workspace_bytes(T, d_in, d_out, r)
        assert n > 0 and n % 256 == 0
        # at least the prefill stage-1 result buffer fits
        assert n >= 2 * T * r * 4
    assert lb.lb_forward_workspace_bytes(-1, 4, 4, 4) == 0
    assert lb.lb_decode_max_tokens() >= 1


# ---------------------------------------------------------------------------
# validation errors (no GPU needed: validation precedes every HIP call)
# ---------------------------------------------------------------------------
FAKE = 0x10000  # a 256-byte aligned address that is never dereferenced


def _paths(U=FAKE, V=FAKE, h=FAKE, g=FAKE, l=FAKE):
    arr = (lb.lb_path * 2)()
    for i in range(2):
        arr[i] = lb.lb_path(U, V, h, g, l)
    return arr


def _fwd(lib, x=FAKE, act=lb.LB_BF16, T=4, d_in=64, d_out=64, r=16, paths=None, sc=lb.LB_F16, y=FAKE,
         ws=FAKE, ws_bytes=None, kernel=lb.LB_KERNEL_AUTO):
    if paths is None:
        paths = _paths()
    if ws_bytes is None:
        ws_bytes = lb.lb_forward_workspace_bytes(max(T, 0), max(d_in, 0), max(d_out, 0), max(r, 0)) - 1
    return lib.lb_linear_forward_kernel(x, act, T, d_in, d_out, r, paths, sc, y, ws, ws_bytes, kernel, None)


def test_forward_validation_errors(lib):
    # the baseline call fails only on the (deliberately) too-small workspace
    assert _fwd(lib) == lb.LB_ERR_WORKSPACE
    assert _fwd(lib, act=7) == lb.LB_ERR_DTYPE
    assert _fwd(lib, sc=-1) == lb.LB_ERR_DTYPE
    assert _fwd(lib, T=-1) == lb.LB_ERR_SHAPE
    assert _fwd(lib, d_in=-3) == lb.LB_ERR_SHAPE
    assert _fwd(lib, r=-1) == lb.LB_ERR_SHAPE
    assert _fwd(lib, T=1 << 20, d_in=1 << 12) == lb.LB_ERR_SHAPE  # T*d_in >= 2^31
    assert _fwd(lib, kernel=9) == lb.LB_ERR_ARG
    assert _fwd(lib, kernel=lb.LB_KERNEL_DECODE, T=lb.lb_decode_max_tokens() + 1) == lb.LB_ERR_SHAPE
    assert _fwd(lib, kernel=lb.LB_KERNEL_DECODE_MFMA, T=65) == lb.LB_ERR_SHAPE
    assert _fwd(lib, kernel=lb.LB_KERNEL_DECODE_MFMA, r=848) == lb.LB_ERR_SHAPE
    assert _fwd(lib, x=0) == lb.LB_ERR_NULL
    assert _fwd(lib, y=0) == lb.LB_ERR_NULL
    assert _fwd(lib, x=FAKE + 1) == lb.LB_ERR_ALIGN
    assert _fwd(lib, act=lb.LB_F32, y=FAKE + 2) == lb.LB_ERR_ALIGN
    assert _fwd(lib, paths=None or _paths(U=0)) == lb.LB_ERR_NULL
    assert _fwd(lib, paths=_paths(l=0)) == lb.LB_ERR_NULL
    assert _fwd(lib, paths=_paths(V=FAKE + 2)) == lb.LB_ERR_ALIGN
    assert _fwd(lib, paths=_paths(h=FAKE + 1)) == lb.LB_ERR_ALIGN
    assert _fwd(lib, sc=lb.LB_F32, paths=_paths(g=FAKE + 2)) == lb.LB_ERR_ALIGN
    assert _fwd(lib, ws=0) == lb.LB_ERR_NULL
    assert _fwd(lib, ws=FAKE + 64, ws_bytes=1 << 30) == lb.LB_ERR_ALIGN
    assert lib.lb_linear_forward_kernel(FAKE, lb.LB_BF16, 4, 64, 64, 16, None, lb.LB_F16, FAKE, FAKE, 1 << 30,
                                        0, None) == lb.LB_ERR_NULL
    # empty problems succeed without touching the GPU
    assert _fwd(lib, T=0) == lb.LB_OK
    assert _fwd(lib, d_out=0) == lb.LB_OK
    # lb_linear_forward (AUTO) goes through the same checks
    assert lib.lb_linear_forward(FAKE, 9, 4, 64, 64, 16, _paths(), lb.LB_F16, FAKE, FAKE, 1 << 30, None) == \
        lb.LB_ERR_DTYPE


def test_noalloc_validation_errors(lib):
    # every check runs before the scratch is touched, so none of these calls reaches the GPU
    assert lib.lb_noalloc_scratch_bytes() == 32 << 20

    def na(x=FAKE, act=lb.LB_BF16, T=4, d_in=64, d_out=64, r=16, paths=None, sc=lb.LB_F16, y=FAKE):
        return lib.lb_linear_forward_noalloc(x, act, T, d_in, d_out, r, _paths() if paths is None else paths, sc,
                                             y, None)

    assert na(act=9) == lb.LB_ERR_DTYPE
    assert na(sc=-1) == lb.LB_ERR_DTYPE
    assert na(T=-1) == lb.LB_ERR_SHAPE
    assert na(r=-1) == lb.LB_ERR_SHAPE
    # a workspace need beyond the 32 MiB scratch: a long prefill of a wide layer
    assert lb.lb_forward_workspace_bytes(4096, 8192, 8192, 256) > 32 << 20
    assert na(T=4096, d_in=8192, d_out=8192, r=256) == lb.LB_ERR_WORKSPACE
    assert na(x=0) == lb.LB_ERR_NULL
    assert na(y=0) == lb.LB_ERR_NULL
    assert na(x=FAKE + 1) == lb.LB_ERR_ALIGN
    assert na(paths=_paths(U=0)) == lb.LB_ERR_NULL
    assert na(paths=_paths(h=FAKE + 1)) == lb.LB_ERR_ALIGN
    assert na(T=0) == lb.LB_OK
    assert na(d_out=0) == lb.LB_OK


def test_dual_svid_workspace_and_validation(lib):
    ws = lb.lb_dual_svid_workspace_bytes
    # the residual weight (8 d_out d_in bytes) dominates at layer sizes; the rest are the blocks,
    # the split-K slabs and the eigensolver's rotation log (9 MB for a block of 120)
    assert ws(4096, 4096, 80, 40) >= 8 * 4096 * 4096
    assert ws(4096, 4096, 80, 40) < 8 * 4096 * 4096 + (80 << 20)
    assert ws(64, 32, 8, 4) > 0 and ws(64, 32, 32, 0) > 0
    for bad in ((0, 32, 8, 4), (64, 0, 8, 4), (64, 32, 0, 4), (64, 32, 33, 0), (64, 32, 8, -1),
                (4096, 4096, 1000, 100), (1 << 20, 1 << 12, 8, 0)):
        assert ws(*bad) == 0, bad
    out = (lb.lb_svid_out * 2)()
    for p in range(2):
        out[p] = lb.lb_svid_out(FAKE, FAKE, FAKE, FAKE, FAKE, 0)

    def call(W=FAKE, dt=lb.LB_F32, d_out=64, d_in=32, r=8, over=4, iters=5, o=out, wres=0, w=FAKE,
             wb=1 << 30):
        return lib.lb_dual_svid(W, dt, d_out, d_in, r, over, iters, 0, o, wres, w, wb, None)

    assert call(dt=9) == lb.LB_ERR_DTYPE
    assert call(r=0) == lb.LB_ERR_SHAPE
    assert call(r=33) == lb.LB_ERR_SHAPE
    assert call(over=-1) == lb.LB_ERR_SHAPE
    assert call(d_out=4096, d_in=4096, r=1000, over=100) == lb.LB_ERR_SHAPE
    assert call(iters=-1) == lb.LB_ERR_ARG
    assert call(iters=1001) == lb.LB_ERR_ARG
    assert call(W=0) == lb.LB_ERR_NULL
    assert call(o=None) == lb.LB_ERR_NULL
    assert call(w=0) == lb.LB_ERR_NULL
    bad = (lb.lb_svid_out * 2)()
    bad[0] = lb.lb_svid_out(FAKE, FAKE, FAKE, FAKE, 0, 0)
    bad[1] = out[1]
    assert call(o=bad) == lb.LB_ERR_NULL
    bad[0] = lb.lb_svid_out(FAKE, FAKE, FAKE + 2, FAKE, FAKE, 0)
    assert call(o=bad) == lb.LB_ERR_ALIGN
    assert call(W=FAKE + 2) == lb.LB_ERR_ALIGN
    assert call(W=FAKE + 2, dt=lb.LB_BF16, wb=1024) == lb.LB_ERR_WORKSPACE  # 2-byte aligned is enough for bf16
    assert call(wres=FAKE + 1) == lb.LB_ERR_ALIGN
    assert call(w=FAKE + 64) == lb.LB_ERR_ALIGN
    assert call(wb=1024) == lb.LB_ERR_WORKSPACE


def test_pack_validation_errors(lib):
    assert lib.lb_pack_signs(FAKE, lb.LB_F32, 64, 16, 5, FAKE * 2, None, None) == lb.LB_ERR_ARG
    assert lib.lb_pack_signs(FAKE, 3, 64, 16, lb.LB_ROLE_U, FAKE * 2, None, None) == lb.LB_ERR_DTYPE
    assert lib.lb_pack_signs(FAKE, lb.LB_F32, -1, 16, lb.LB_ROLE_U, FAKE * 2, None, None) == lb.LB_ERR_SHAPE
    assert lib.lb_pack_signs(0, lb.LB_F32, 64, 16, lb.LB_ROLE_U, FAKE * 2, None, None) == lb.LB_ERR_NULL
    assert lib.lb_pack_signs(FAKE, lb.LB_F32, 64, 16, lb.LB_ROLE_U, 0, None, None) == lb.LB_ERR_NULL
    assert lib.lb_pack_signs(FAKE + 2, lb.LB_F32, 64, 16, lb.LB_ROLE_U, FAKE * 2, None, None) == lb.LB_ERR_ALIGN
    assert lib.lb_pack_signs(FAKE, lb.LB_F32, 64, 16, lb.LB_ROLE_U, FAKE * 2 + 2, None, None) == lb.LB_ERR_ALIGN
    assert lib.lb_pack_signs(FAKE, lb.LB_BF16, 64, 16, lb.LB_ROLE_U, FAKE * 2, FAKE + 1, None) == lb.LB_ERR_ALIGN
    # overlapping src/dst
    assert lib.lb_pack_signs(FAKE, lb.LB_F32, 64, 16, lb.LB_ROLE_U, FAKE + 64, None, None) == lb.LB_ERR_ARG
    # empty matrices are a no-op
    assert lib.lb_pack_signs(0, lb.LB_F32, 0, 16, lb.LB_ROLE_U, 0, None, None) == lb.LB_OK


def test_dense_ref_validation_errors(lib):
    assert lib.lb_dense_reference_weight(_paths(), 5, 64, 64, 16, FAKE, None) == lb.LB_ERR_DTYPE
    assert lib.lb_dense_reference_weight(_paths(), lb.LB_F16, -1, 64, 16, FAKE, None) == lb.LB_ERR_SHAPE
    assert lib.lb_dense_reference_weight(_paths(), lb.LB_F16, 64, 64, 16, 0, None) == lb.LB_ERR_NULL
    assert lib.lb_dense_reference_weight(_paths(), lb.LB_F16, 64, 64, 16, FAKE + 2, None) == lb.LB_ERR_ALIGN
    assert lib.lb_dense_reference_weight(None, lb.LB_F16, 64, 64, 16, FAKE, None) == lb.LB_ERR_NULL
    assert lib.lb_dense_reference_weight(_paths(), lb.LB_F16, 0, 64, 16, FAKE, None) == lb.LB_OK


def test_workspace_init_validation(lib):
    assert lib.lb_workspace_init(0, 256, None) == lb.LB_ERR_NULL
    assert lib.lb_workspace_init(FAKE + 4, 256, None) == lb.LB_ERR_ALIGN
    assert lib.lb_workspace_init(FAKE, 6, None) == lb.LB_ERR_ALIGN
    assert lib.lb_workspace_init(0, 0, None) == lb.LB_OK


def test_workspace_status_validation(lib):
    assert lib.lb_workspace_status(0, 256, FAKE, None) == lb.LB_ERR_NULL
    assert lib.lb_workspace_status(FAKE, 256, 0, None) == lb.LB_ERR_NULL
    assert lib.lb_workspace_status(FAKE + 4, 256, FAKE, None) == lb.LB_ERR_ALIGN
    assert lib.lb_workspace_status(FAKE, 256, FAKE + 2, None) == lb.LB_ERR_ALIGN
    assert lib.lb_workspace_status(FAKE, 255, FAKE, None) == lb.LB_ERR_WORKSPACE


def test_binding_refuses_cpu_tensors(lib):
    import torch
    x = torch.zeros(2, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        lb.lb_pack_signs(x, lb.LB_ROLE_U)


# ---------------------------------------------------------------------------
# list forward (lb_linear_forward_many): validation and workspace sizing
# ---------------------------------------------------------------------------
def _desc(x=FAKE, act=lb.LB_BF16, T=1, d_in=64, d_out=64, r=16, paths=None, sc=lb.LB_F16, y=FAKE):
    d = lb.lb_linear_desc()
    d.x, d.act_dtype, d.T, d.d_in, d.d_out, d.r, d.scale_dtype, d.y = x, act, T, d_in, d_out, r, sc, y
    p = paths if paths is not None else _paths()
    d.paths[0], d.paths[1] = p[0], p[1]
    return d


def _descs(*ds):
    arr = (lb.lb_linear_desc * len(ds))()
    for i, d in enumerate(ds):
        arr[i] = d
    return arr


def test_many_workspace_bytes_is_the_sum_of_rounded_slices(lib):
    shapes = [(1, 4096, 4096, 80), (2, 512, 1000, 17), (16, 64, 64, 16), (0, 5, 5, 5), (300, 100, 77, 48)]
    arr = _descs(*[_desc(T=T, d_in=a, d_out=b, r=r) for T, a, b, r in shapes])
    # the list header (control block + 16 counter lines of 256 bytes) and the rounded slices
    want = 256 + 16 * 256 + sum((lb.lb_forward_workspace_bytes(*s) + 255) // 256 * 256 for s in shapes)
    assert lb.lb_forward_many_workspace_bytes(arr, len(shapes)) == want
    assert lb.lb_forward_many_workspace_bytes(arr, 0) == 0
    assert lb.lb_forward_many_workspace_bytes(None, 3) == 0
    assert lb.lb_forward_many_workspace_bytes(_descs(_desc(T=-1)), 1) == 0


def test_many_validation_errors(lib):
    y2 = FAKE + (1 << 20)
    ok2 = [_desc(), _desc(y=y2, x=FAKE + (2 << 20))]
    need = lb.lb_forward_many_workspace_bytes(_descs(*ok2), 2)

    def call(ds, ws=FAKE * 64, ws_bytes=None, n=None):
        arr = _descs(*ds)
        return lib.lb_linear_forward_many(arr, len(ds) if n is None else n, ws,
                                          need - 1 if ws_bytes is None else ws_bytes, None)

    # the baseline list fails only on the (deliberately) too-small workspace
    assert call(ok2) == lb.LB_ERR_WORKSPACE
    assert call(ok2, n=-1) == lb.LB_ERR_ARG
    assert lib.lb_linear_forward_many(None, 0, 0, 0, None) == lb.LB_OK
    assert lib.lb_linear_forward_many(None, 2, FAKE, 1 << 30, None) == lb.LB_ERR_NULL
    # every descriptor is validated before anything is enqueued
    assert call([ok2[0], _desc(act=9, y=y2)]) == lb.LB_ERR_DTYPE
    assert call([ok2[0], _desc(T=-1, y=y2)]) == lb.LB_ERR_SHAPE
    assert call([ok2[0], _desc(x=0, y=y2)]) == lb.LB_ERR_NULL
    assert call([ok2[0], _desc(y=y2 + 2, act=lb.LB_F32)]) == lb.LB_ERR_ALIGN
    assert call([ok2[0], _desc(y=y2, paths=_paths(h=0))]) == lb.LB_ERR_NULL
    # outputs overlapping another linear's output or input
    assert call([_desc(), _desc(y=FAKE + 64)]) == lb.LB_ERR_ARG
    assert call([_desc(y=y2), _desc(x=y2 + 32, y=FAKE + (3 << 20))]) == lb.LB_ERR_ARG
    # workspace
    assert call(ok2, ws=0, ws_bytes=1 << 30) == lb.LB_ERR_NULL
    assert call(ok2, ws=FAKE * 64 + 128, ws_bytes=1 << 30) == lb.LB_ERR_ALIGN
    # empty linears need no work and no GPU
    assert call([_desc(T=0), _desc(d_out=0, y=y2)], ws_bytes=1 << 20) == lb.LB_OK


# ---------------------------------------------------------------------------
# latent cache calls (validation only; the GPU parity tests run them)
# ---------------------------------------------------------------------------
FAR = FAKE * 16  # a second aligned address, far from FAKE


def _lat(lib, x=FAKE, act=lb.LB_BF16, T=4, d_in=64, r=16, paths=None, sc=lb.LB_F16, w=FAR, ld=lb.LB_F32,
         ws=FAKE * 64, ws_bytes=None):
    if paths is None:
        paths = _paths(U=0, h=0)  # U and h are not read
    if ws_bytes is None:
        ws_bytes = lb.lb_latent_workspace_bytes(max(T, 0), max(d_in, 0), max(r, 0)) - 1
    return lib.lb_linear_latent(x, act, T, d_in, r, paths, sc, w, ld, ws, ws_bytes, None)


def _from(lib, w=FAKE, ld=lb.LB_F32, T=4, d_out=64, r=16, paths=None, sc=lb.LB_F16, y=FAR, out=lb.LB_BF16,
          ws=FAKE * 64, ws_bytes=None):
    if paths is None:
        paths = _paths(V=0, g=0, l=0)  # V, g and l are not read
    if ws_bytes is None:
        ws_bytes = lb.lb_from_latent_workspace_bytes(max(T, 0), max(r, 0)) - 1
    return lib.lb_linear_from_latent(w, ld, T, d_out, r, paths, sc, y, out, ws, ws_bytes, None)


def test_latent_workspace_sizes(lib):
    for T, d_in, r in [(1, 4096, 80), (2048, 5120, 96), (64, 11008, 800), (3, 33, 5)]:
        n = lb.lb_latent_workspace_bytes(T, d_in, r)
        # at least one fp32 partial per latent, token and path
        assert n % 256 == 0 and n >= 2 * T * r * 4
        m = lb.lb_from_latent_workspace_bytes(T, r)
        # the w terms: up to three bf16 terms per latent, token and path (32-latent blocks)
        assert m % 256 == 0 and m >= 2 * 3 * 2 * T * 32 * ((r + 31) // 32)
    assert lb.lb_latent_workspace_bytes(-1, 4, 4) == 0
    assert lb.lb_from_latent_workspace_bytes(4, -1) == 0


def test_latent_validation_errors(lib):
    assert _lat(lib) == lb.LB_ERR_WORKSPACE
    assert _lat(lib, act=5) == lb.LB_ERR_DTYPE
    assert _lat(lib, sc=5) == lb.LB_ERR_DTYPE
    assert _lat(lib, ld=3) == lb.LB_ERR_DTYPE
    assert _lat(lib, T=-1) == lb.LB_ERR_SHAPE
    assert _lat(lib, r=-2) == lb.LB_ERR_SHAPE
    assert _lat(lib, T=1 << 20, d_in=1 << 12) == lb.LB_ERR_SHAPE
    assert _lat(lib, x=0) == lb.LB_ERR_NULL
    assert _lat(lib, w=0) == lb.LB_ERR_NULL
    assert _lat(lib, x=FAKE + 1) == lb.LB_ERR_ALIGN
    assert _lat(lib, w=FAR + 2) == lb.LB_ERR_ALIGN
    assert _lat(lib, w=FAR + 2, ld=lb.LB_BF16) == lb.LB_ERR_WORKSPACE
    assert _lat(lib, paths=_paths(U=0, h=0, V=0)) == lb.LB_ERR_NULL
    assert _lat(lib, paths=_paths(U=0, h=0, l=0)) == lb.LB_ERR_NULL
    assert _lat(lib, paths=_paths(U=0, h=0, g=FAKE + 1)) == lb.LB_ERR_ALIGN
    # U and h are not read, so not checked either
    assert _lat(lib, paths=_paths(U=FAKE + 1, h=FAKE + 1)) == lb.LB_ERR_WORKSPACE
    assert lib.lb_linear_latent(FAKE, lb.LB_BF16, 4, 64, 16, None, lb.LB_F16, FAR, lb.LB_F32, FAKE * 64, 1 << 30,
                                None) == lb.LB_ERR_NULL
    assert _lat(lib, w=FAKE + 256) == lb.LB_ERR_ARG  # w overlaps x
    assert _lat(lib, ws=0) == lb.LB_ERR_NULL
    assert _lat(lib, ws=FAKE * 64 + 16, ws_bytes=1 << 30) == lb.LB_ERR_ALIGN
    assert _lat(lib, T=0) == lb.LB_OK
    assert _lat(lib, r=0) == lb.LB_OK


def test_from_latent_validation_errors(lib):
    assert _from(lib) == lb.LB_ERR_WORKSPACE
    assert _from(lib, ld=9) == lb.LB_ERR_DTYPE
    assert _from(lib, out=9) == lb.LB_ERR_DTYPE
    assert _from(lib, sc=9) == lb.LB_ERR_DTYPE
    assert _from(lib, d_out=-1) == lb.LB_ERR_SHAPE
    assert _from(lib, T=1 << 20, d_out=1 << 12) == lb.LB_ERR_SHAPE
    assert _from(lib, w=0) == lb.LB_ERR_NULL
    assert _from(lib, y=0) == lb.LB_ERR_NULL
    assert _from(lib, w=FAKE + 2) == lb.LB_ERR_ALIGN
    assert _from(lib, y=FAR + 1) == lb.LB_ERR_ALIGN
    assert _from(lib, paths=_paths(V=0, g=0, l=0, U=0)) == lb.LB_ERR_NULL
    assert _from(lib, paths=_paths(V=0, g=0, l=0, h=0)) == lb.LB_ERR_NULL
    assert _from(lib, paths=_paths(V=0, g=0, l=0, U=FAKE + 2)) == lb.LB_ERR_ALIGN
    # V, g and l are not read, so not checked either
    assert _from(lib, paths=_paths(V=FAKE + 1, g=FAKE + 1, l=FAKE + 1)) == lb.LB_ERR_WORKSPACE
    assert _from(lib, y=FAKE + 128) == lb.LB_ERR_ARG  # y overlaps w
    assert _from(lib, ws=0) == lb.LB_ERR_NULL
    assert _from(lib, T=0) == lb.LB_OK
    assert _from(lib, d_out=0) == lb.LB_OK


# ---------------------------------------------------------------------------
# backward (validation only)
# ---------------------------------------------------------------------------
def _train(**kw):
    arr = (lb.lb_path_train * 2)()
    base = dict(U_latent=FAKE, V_latent=FAKE, Ut=FAKE, Vt=FAKE, dU=FAR, dV=FAR, dh=FAR, dg=FAR, dl=FAR)
    base.update(kw)
    for i in range(2):
        arr[i] = lb.lb_path_train(*[base[f] for f in ("U_latent", "V_latent", "Ut", "Vt", "dU", "dV", "dh", "dg",
                                                      "dl")])
    return arr


def _bwd(lib, x=FAKE, dy=FAKE * 2, act=lb.LB_BF16, T=4, d_in=64, d_out=48, r=16, paths=None, sc=lb.LB_F16,
         train=None, kappa=100.0, dx=FAR * 4, ws=FAKE * 64, ws_bytes=None):
    if paths is None:
        paths = _paths(U=0)  # U is not read
    if train is None:
        train = _train()
    if ws_bytes is None:
        ws_bytes = lb.lb_backward_workspace_bytes(max(T, 0), max(d_in, 0), max(d_out, 0), max(r, 0)) - 1
    return lib.lb_linear_backward(x, dy, act, T, d_in, d_out, r, paths, sc, train, kappa, dx, ws, ws_bytes, None)


def test_backward_workspace_sizes(lib):
    for T, d_in, d_out, r in [(2048, 4096, 4096, 80), (64, 11008, 4096, 128), (3, 33, 17, 5), (1, 64, 64, 300)]:
        n = lb.lb_backward_workspace_bytes(T, d_in, d_out, r)
        # z and dw of both paths in fp32, plus the stage and split buffers
        assert n % 256 == 0 and n >= 2 * (2 * T * r * 4)
    assert lb.lb_backward_workspace_bytes(-1, 4, 4, 4) == 0
    # empty sizes plan without dividing by zero (regression) and still reserve the control block
    for T, d_in, d_out, r in [(0, 64, 48, 16), (8, 0, 48, 16), (8, 64, 0, 16), (8, 64, 48, 0), (0, 0, 0, 0)]:
        assert lb.lb_backward_workspace_bytes(T, d_in, d_out, r) >= 256


def test_backward_validation_errors(lib):
    assert _bwd(lib) == lb.LB_ERR_WORKSPACE
    assert _bwd(lib, act=3) == lb.LB_ERR_DTYPE
    assert _bwd(lib, sc=3) == lb.LB_ERR_DTYPE
    assert _bwd(lib, T=-1) == lb.LB_ERR_SHAPE
    assert _bwd(lib, T=1 << 20, d_in=1 << 12) == lb.LB_ERR_SHAPE
    assert _bwd(lib, kappa=0.0) == lb.LB_ERR_ARG
    assert _bwd(lib, kappa=float("inf")) == lb.LB_ERR_ARG
    assert _bwd(lib, kappa=float("nan")) == lb.LB_ERR_ARG
    assert _bwd(lib, x=0) == lb.LB_ERR_NULL
    assert _bwd(lib, dy=0) == lb.LB_ERR_NULL
    assert _bwd(lib, x=FAKE + 1) == lb.LB_ERR_ALIGN
    assert _bwd(lib, dx=FAR * 4 + 1) == lb.LB_ERR_ALIGN
    assert _bwd(lib, paths=_paths(U=0, V=0)) == lb.LB_ERR_NULL
    assert _bwd(lib, paths=_paths(U=0, h=FAKE + 1)) == lb.LB_ERR_ALIGN
    assert lib.lb_linear_backward(FAKE, FAKE * 2, lb.LB_BF16, 4, 64, 48, 16, None, lb.LB_F16, _train(), 100.0,
                                  FAR * 4, FAKE * 64, 1 << 30, None) == lb.LB_ERR_NULL
    assert lib.lb_linear_backward(FAKE, FAKE * 2, lb.LB_BF16, 4, 64, 48, 16, _paths(U=0), lb.LB_F16, None, 100.0,
                                  FAR * 4, FAKE * 64, 1 << 30, None) == lb.LB_ERR_NULL
    for f in ("U_latent", "V_latent", "Ut", "Vt", "dU", "dV", "dh", "dg", "dl"):
        assert _bwd(lib, train=_train(**{f: 0})) == lb.LB_ERR_NULL, f
        assert _bwd(lib, train=_train(**{f: FAR + 2})) == lb.LB_ERR_ALIGN, f
    assert _bwd(lib, dx=FAKE + 64) == lb.LB_ERR_ARG  # dx overlaps x
    assert _bwd(lib, dx=FAKE * 2 + 64) == lb.LB_ERR_ARG  # dx overlaps dy
    assert _bwd(lib, ws=0) == lb.LB_ERR_NULL
    assert _bwd(lib, ws=FAKE * 64 + 8, ws_bytes=1 << 30) == lb.LB_ERR_ALIGN
    # dx may be NULL (not computed); U of the paths is never read
    assert _bwd(lib, dx=0) == lb.LB_ERR_WORKSPACE
    assert _bwd(lib, paths=_paths(U=FAKE + 1)) == lb.LB_ERR_WORKSPACE


def _list_descs(n, T=1, d_in=64, d_out=64, r=16, act=lb.LB_BF16, sc=lb.LB_F16, ystep=4096):
    arr = (lb.lb_linear_desc * n)()
    for i in range(n):
        arr[i] = lb.lb_linear_desc(FAKE, act, T, d_in, d_out, r, _paths(), sc, FAKE * 4 + i * ystep)
    return arr


def test_list_validation(lib):
    arr = _list_descs(3)
    need = lib.lb_list_workspace_bytes(arr, 3)
    assert need > 0
    # lists with more than two tokens run on the matrix cores (up to 64 tokens, d_in a multiple of 4)
    assert lib.lb_list_workspace_bytes(_list_descs(2, T=3), 2) > 0
    assert lib.lb_list_workspace_bytes(_list_descs(2, T=64, ystep=1 << 16), 2) > 0
    mix = _list_descs(2)
    mix[1].T = 8
    assert lib.lb_list_workspace_bytes(mix, 2) > 0
    # out of scope: 65 tokens, d_in not a multiple of 4 with more than two tokens, a rank above 1024,
    # mixed dtypes
    assert lib.lb_list_workspace_bytes(_list_descs(2, T=65), 2) == 0
    assert lib.lb_list_workspace_bytes(_list_descs(2, T=8, d_in=30), 2) == 0
    assert lib.lb_list_workspace_bytes(_list_descs(2, T=2, d_in=30), 2) > 0
    assert lib.lb_list_workspace_bytes(_list_descs(2, r=1040), 2) == 0
    assert lib.lb_list_init(_list_descs(2, T=65), 2, FAKE, 1 << 30, None) == lb.LB_ERR_SHAPE
    mixed = _list_descs(2)
    mixed[1].act_dtype = lb.LB_F32
    assert lib.lb_list_init(mixed, 2, FAKE, 1 << 30, None) == lb.LB_ERR_DTYPE
    assert lib.lb_list_forward(mixed, 2, FAKE, 1 << 30, None) == lb.LB_ERR_DTYPE
    # overlapping outputs, and an output over another linear's input
    assert lib.lb_list_init(_list_descs(2, ystep=2), 2, FAKE, 1 << 30, None) == lb.LB_ERR_ARG
    over = _list_descs(2)
    over[1].x = over[0].y
    assert lib.lb_list_forward(over, 2, FAKE, 1 << 30, None) == lb.LB_ERR_ARG
    # a linear's output may overlap its own input
    own = _list_descs(1)
    own[0].y = own[0].x
    assert lib.lb_list_workspace_bytes(own, 1) > 0
    # workspace checks
    assert lib.lb_list_init(arr, 3, 0, need, None) == lb.LB_ERR_NULL
    assert lib.lb_list_init(arr, 3, FAKE + 16, need, None) == lb.LB_ERR_ALIGN
    assert lib.lb_list_init(arr, 3, FAKE, need - 1, None) == lb.LB_ERR_WORKSPACE
    assert lib.lb_list_forward(arr, 3, FAKE, need - 1, None) == lb.LB_ERR_WORKSPACE
    assert lib.lb_list_forward(None, 3, FAKE, need, None) == lb.LB_ERR_NULL
    assert lib.lb_list_forward(arr, -1, FAKE, need, None) == lb.LB_ERR_ARG
    assert lib.lb_list_forward(arr, 70000, FAKE, need, None) == lb.LB_ERR_ARG
    # the workspace grows with the list
    assert lib.lb_list_workspace_bytes(_list_descs(600), 600) > need
