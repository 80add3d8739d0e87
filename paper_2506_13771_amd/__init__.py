"""LittleBit linear layer on MI355X (gfx950): Python binding of liblittlebit.so.

This module only marshals arguments into the C ABI declared in
include/littlebit.h: every step of the computation runs in the library's HIP
kernels.  PyTorch provides device memory and the current stream.  If the
library is not built, or a tensor is not on a GPU, calls raise instead of
falling back to anything else.

The names follow the C ABI:
  lb_pack_signs, lb_linear_forward, lb_dense_reference_weight,
  lb_packed_bytes, lb_bits_per_weight, lb_rank_for_bpw,
  lb_forward_workspace_bytes, lb_workspace_init, lb_workspace_status, lb_decode_max_tokens,
  lb_linear_forward_many, lb_forward_many_workspace_bytes,
  lb_list_workspace_bytes, lb_list_init, lb_list_forward (class LittleBitList),
  lb_linear_latent, lb_latent_workspace_bytes,
  lb_linear_from_latent, lb_from_latent_workspace_bytes,
  lb_linear_backward, lb_backward_workspace_bytes.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional, Sequence

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblittlebit.so")

LB_OK, LB_ERR_NULL, LB_ERR_SHAPE, LB_ERR_DTYPE, LB_ERR_ALIGN, LB_ERR_WORKSPACE, LB_ERR_HIP, LB_ERR_ARG = range(8)
LB_F32, LB_F16, LB_BF16 = 0, 1, 2
LB_ROLE_U, LB_ROLE_V = 0, 1
LB_KERNEL_AUTO, LB_KERNEL_DECODE, LB_KERNEL_PREFILL, LB_KERNEL_DECODE_MFMA = 0, 1, 2, 3
ABI_VERSION = 7


class LittleBitError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {lb_status_str(status)} ({status})")
        self.status = status


class lb_path(ctypes.Structure):
    _fields_ = [("U", ctypes.c_void_p), ("V", ctypes.c_void_p), ("h", ctypes.c_void_p),
                ("g", ctypes.c_void_p), ("l", ctypes.c_void_p)]


class lb_linear_desc(ctypes.Structure):
    _fields_ = [("x", ctypes.c_void_p), ("act_dtype", ctypes.c_int), ("T", ctypes.c_int64),
                ("d_in", ctypes.c_int64), ("d_out", ctypes.c_int64), ("r", ctypes.c_int64),
                ("paths", lb_path * 2), ("scale_dtype", ctypes.c_int), ("y", ctypes.c_void_p)]


class lb_path_train(ctypes.Structure):
    _fields_ = [("U_latent", ctypes.c_void_p), ("V_latent", ctypes.c_void_p), ("Ut", ctypes.c_void_p),
                ("Vt", ctypes.c_void_p), ("dU", ctypes.c_void_p), ("dV", ctypes.c_void_p), ("dh", ctypes.c_void_p),
                ("dg", ctypes.c_void_p), ("dl", ctypes.c_void_p)]


class lb_svid_out(ctypes.Structure):
    _fields_ = [("U_latent", ctypes.c_void_p), ("V_latent", ctypes.c_void_p), ("h", ctypes.c_void_p),
                ("g", ctypes.c_void_p), ("l", ctypes.c_void_p), ("sigma", ctypes.c_void_p)]


_lib = None


def load_library(path: str = LIB_PATH):
    """Load liblittlebit.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"LittleBit HIP library not built: {path} is missing "
                           "(run __graft_entry__.build() or python paper_2506_13771_amd/_build.py)")
    lib = ctypes.CDLL(path)
    i64, sz, vp, i32 = ctypes.c_int64, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int
    lib.lb_abi_version.restype = i32
    lib.lb_abi_version.argtypes = []
    lib.lb_status_str.restype = ctypes.c_char_p
    lib.lb_status_str.argtypes = [i32]
    lib.lb_packed_bytes.restype = sz
    lib.lb_packed_bytes.argtypes = [i32, i64, i64]
    lib.lb_bits_per_weight.restype = ctypes.c_double
    lib.lb_bits_per_weight.argtypes = [i64, i64, i64, i32]
    lib.lb_rank_for_bpw.restype = i64
    lib.lb_rank_for_bpw.argtypes = [i64, i64, ctypes.c_double, i64]
    lib.lb_pack_signs.restype = i32
    lib.lb_pack_signs.argtypes = [vp, i32, i64, i64, i32, vp, vp, vp]
    lib.lb_forward_workspace_bytes.restype = sz
    lib.lb_forward_workspace_bytes.argtypes = [i64, i64, i64, i64]
    lib.lb_workspace_init.restype = i32
    lib.lb_workspace_init.argtypes = [vp, sz, vp]
    lib.lb_workspace_status.restype = i32
    lib.lb_workspace_status.argtypes = [vp, sz, vp, vp]
    lib.lb_decode_max_tokens.restype = i64
    lib.lb_decode_max_tokens.argtypes = []
    lib.lb_linear_forward.restype = i32
    lib.lb_linear_forward.argtypes = [vp, i32, i64, i64, i64, i64, ctypes.POINTER(lb_path), i32, vp, vp, sz, vp]
    lib.lb_linear_forward_kernel.restype = i32
    lib.lb_linear_forward_kernel.argtypes = [vp, i32, i64, i64, i64, i64, ctypes.POINTER(lb_path), i32, vp, vp,
                                             sz, i32, vp]
    lib.lb_noalloc_scratch_bytes.restype = sz
    lib.lb_noalloc_scratch_bytes.argtypes = []
    lib.lb_linear_forward_noalloc.restype = i32
    lib.lb_linear_forward_noalloc.argtypes = [vp, i32, i64, i64, i64, i64, ctypes.POINTER(lb_path), i32, vp, vp]
    lib.lb_forward_many_workspace_bytes.restype = sz
    lib.lb_forward_many_workspace_bytes.argtypes = [ctypes.POINTER(lb_linear_desc), i64]
    lib.lb_linear_forward_many.restype = i32
    lib.lb_linear_forward_many.argtypes = [ctypes.POINTER(lb_linear_desc), i64, vp, sz, vp]
    lib.lb_list_workspace_bytes.restype = sz
    lib.lb_list_workspace_bytes.argtypes = [ctypes.POINTER(lb_linear_desc), i64]
    lib.lb_list_init.restype = i32
    lib.lb_list_init.argtypes = [ctypes.POINTER(lb_linear_desc), i64, vp, sz, vp]
    lib.lb_list_forward.restype = i32
    lib.lb_list_forward.argtypes = [ctypes.POINTER(lb_linear_desc), i64, vp, sz, vp]
    lib.lb_latent_workspace_bytes.restype = sz
    lib.lb_latent_workspace_bytes.argtypes = [i64, i64, i64]
    lib.lb_linear_latent.restype = i32
    lib.lb_linear_latent.argtypes = [vp, i32, i64, i64, i64, ctypes.POINTER(lb_path), i32, vp, i32, vp, sz, vp]
    lib.lb_from_latent_workspace_bytes.restype = sz
    lib.lb_from_latent_workspace_bytes.argtypes = [i64, i64]
    lib.lb_linear_from_latent.restype = i32
    lib.lb_linear_from_latent.argtypes = [vp, i32, i64, i64, i64, ctypes.POINTER(lb_path), i32, vp, i32, vp, sz,
                                          vp]
    lib.lb_backward_workspace_bytes.restype = sz
    lib.lb_backward_workspace_bytes.argtypes = [i64, i64, i64, i64]
    lib.lb_linear_backward.restype = i32
    lib.lb_linear_backward.argtypes = [vp, vp, i32, i64, i64, i64, i64, ctypes.POINTER(lb_path), i32,
                                       ctypes.POINTER(lb_path_train), ctypes.c_float, vp, vp, sz, vp]
    lib.lb_dense_reference_weight.restype = i32
    lib.lb_dense_reference_weight.argtypes = [ctypes.POINTER(lb_path), i32, i64, i64, i64, vp, vp]
    lib.lb_dual_svid_workspace_bytes.restype = sz
    lib.lb_dual_svid_workspace_bytes.argtypes = [i64, i64, i64, i64]
    lib.lb_dual_svid.restype = i32
    lib.lb_dual_svid.argtypes = [vp, i32, i64, i64, i64, i64, i32, ctypes.c_uint64, ctypes.POINTER(lb_svid_out), vp,
                                 vp, sz, vp]
    if lib.lb_abi_version() != ABI_VERSION:
        raise RuntimeError("liblittlebit.so ABI version mismatch")
    _lib = lib
    return lib


# ----------------------------------------------------------------------------
# pure host helpers
# ----------------------------------------------------------------------------
def lb_status_str(status: int) -> str:
    return load_library().lb_status_str(status).decode()


def lb_packed_bytes(role: int, rows: int, r: int) -> int:
    return int(load_library().lb_packed_bytes(role, rows, r))


def lb_bits_per_weight(d_in: int, d_out: int, r: int, npaths: int = 2) -> float:
    return float(load_library().lb_bits_per_weight(d_in, d_out, r, npaths))


def lb_rank_for_bpw(d_in: int, d_out: int, bpw: float, mult: int = 16) -> int:
    return int(load_library().lb_rank_for_bpw(d_in, d_out, bpw, mult))


def lb_forward_workspace_bytes(T: int, d_in: int, d_out: int, r: int) -> int:
    return int(load_library().lb_forward_workspace_bytes(T, d_in, d_out, r))


def lb_decode_max_tokens() -> int:
    return int(load_library().lb_decode_max_tokens())


# ----------------------------------------------------------------------------
# tensor marshalling
# ----------------------------------------------------------------------------
def _torch():
    import torch
    return torch


def _dtype_code(t) -> int:
    torch = _torch()
    m = {torch.float32: LB_F32, torch.float16: LB_F16, torch.bfloat16: LB_BF16}
    if t.dtype not in m:
        raise TypeError(f"unsupported dtype {t.dtype}")
    return m[t.dtype]


def _torch_dtype(code: int):
    torch = _torch()
    return {LB_F32: torch.float32, LB_F16: torch.float16, LB_BF16: torch.bfloat16}[code]


def _dev_ptr(t, name: str) -> int:
    if t is None:
        return 0
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _stream(stream) -> int:
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _check(status: int, what: str):
    if status != LB_OK:
        raise LittleBitError(status, what)


@dataclass
class LittleBitPath:
    """One path's packed signs (uint8 device tensors in LB layout v1) and scales."""
    U: object
    V: object
    h: object
    g: object
    l: object


def _paths_struct(paths: Sequence[LittleBitPath]):
    if len(paths) != 2:
        raise ValueError("exactly two paths (primary, residual) are required")
    arr = (lb_path * 2)()
    for i, p in enumerate(paths):
        arr[i] = lb_path(_dev_ptr(p.U, "U"), _dev_ptr(p.V, "V"), _dev_ptr(p.h, "h"),
                         _dev_ptr(p.g, "g"), _dev_ptr(p.l, "l"))
    sc = {_dtype_code(t) for p in paths for t in (p.h, p.g, p.l) if t is not None}
    if len(sc) != 1:
        raise TypeError("all scales must share one dtype")
    return arr, sc.pop()


def lb_pack_signs(src, role: int, dst=None, nan_count=None, stream=None):
    """Pack the signs of src [rows, r] (latent U or V) into dst (uint8, LB layout v1)."""
    torch = _torch()
    lib = load_library()
    rows, r = src.shape
    n = lb_packed_bytes(role, rows, r)
    if dst is None:
        dst = torch.empty(n, dtype=torch.uint8, device=src.device)
    if dst.numel() * dst.element_size() < n:
        raise ValueError("dst too small")
    st = lib.lb_pack_signs(_dev_ptr(src, "src"), _dtype_code(src), rows, r, role, _dev_ptr(dst, "dst"),
                           _dev_ptr(nan_count, "nan_count"), _stream(stream))
    _check(st, "lb_pack_signs")
    return dst


def lb_workspace_init(ws, stream=None):
    st = load_library().lb_workspace_init(_dev_ptr(ws, "workspace"), ws.numel() * ws.element_size(), _stream(stream))
    _check(st, "lb_workspace_init")
    return ws


def lb_workspace_status(ws, stream=None) -> int:
    """Read and clear the workspace's error word (0: no bounded wait expired since the last clear);
    synchronises the stream to return the value."""
    torch = _torch()
    out = torch.full((1,), -1, dtype=torch.int32, device=ws.device)
    st = load_library().lb_workspace_status(_dev_ptr(ws, "workspace"), ws.numel() * ws.element_size(),
                                            _dev_ptr(out, "status"), _stream(stream))
    _check(st, "lb_workspace_status")
    return int(out.item())


def alloc_workspace(T: int, d_in: int, d_out: int, r: int, device="cuda"):
    """A zero-filled workspace tensor of lb_forward_workspace_bytes(T, d_in, d_out, r) bytes."""
    torch = _torch()
    n = lb_forward_workspace_bytes(T, d_in, d_out, r)
    ws = torch.empty(max(n, 256), dtype=torch.uint8, device=device)
    return lb_workspace_init(ws)


def lb_linear_forward(x, paths: Sequence[LittleBitPath], r: int, y=None, workspace=None,
                      kernel: int = LB_KERNEL_AUTO, stream=None):
    """y [T, d_out] = LittleBit forward of x [T, d_in] with both paths; returns y."""
    torch = _torch()
    lib = load_library()
    T, d_in = x.shape
    d_out = paths[0].h.shape[0]
    arr, sc = _paths_struct(paths)
    if y is None:
        y = torch.empty((T, d_out), dtype=x.dtype, device=x.device)
    if workspace is None:
        workspace = alloc_workspace(T, d_in, d_out, r, device=x.device)
    st = lib.lb_linear_forward_kernel(_dev_ptr(x, "x"), _dtype_code(x), T, d_in, d_out, r, arr, sc,
                                      _dev_ptr(y, "y"), _dev_ptr(workspace, "workspace"),
                                      workspace.numel() * workspace.element_size(), kernel, _stream(stream))
    _check(st, "lb_linear_forward")
    return y


def lb_linear_forward_noalloc(x, paths: Sequence[LittleBitPath], r: int, y=None, stream=None):
    """lb_linear_forward with the library's static per-GPU scratch as workspace (no workspace argument,
    nothing allocated by the call); y is allocated here when None."""
    torch = _torch()
    lib = load_library()
    T, d_in = x.shape
    d_out = paths[0].h.shape[0]
    arr, sc = _paths_struct(paths)
    if y is None:
        y = torch.empty((T, d_out), dtype=x.dtype, device=x.device)
    st = lib.lb_linear_forward_noalloc(_dev_ptr(x, "x"), _dtype_code(x), T, d_in, d_out, r, arr, sc,
                                       _dev_ptr(y, "y"), _stream(stream))
    _check(st, "lb_linear_forward_noalloc")
    return y


def make_descs(items):
    """A ctypes array of lb_linear_desc for items (x, paths, r, y) (y allocated when None); returns
    (array, list of y).  The tensors must outlive every call that uses the array."""
    torch = _torch()
    arr = (lb_linear_desc * max(len(items), 1))()
    ys = []
    for i, (x, paths, r, y) in enumerate(items):
        T, d_in = x.shape
        d_out = paths[0].h.shape[0]
        parr, sc = _paths_struct(paths)
        if y is None:
            y = torch.empty((T, d_out), dtype=x.dtype, device=x.device)
        arr[i] = lb_linear_desc(_dev_ptr(x, "x"), _dtype_code(x), T, d_in, d_out, r, parr, sc, _dev_ptr(y, "y"))
        ys.append(y)
    return arr, ys


def lb_forward_many_workspace_bytes(descs, n: int) -> int:
    return int(load_library().lb_forward_many_workspace_bytes(descs, n))


def lb_linear_forward_many(items, workspace=None, stream=None):
    """The LittleBit forward of every (x, paths, r, y) of items (independent linears) in as few launches as
    the library can; returns the list of y."""
    torch = _torch()
    lib = load_library()
    arr, ys = make_descs(items)
    n = len(items)
    if workspace is None:
        need = lb_forward_many_workspace_bytes(arr, n)
        workspace = lb_workspace_init(torch.empty(max(need, 256), dtype=torch.uint8, device=ys[0].device if ys else "cuda"))
    st = lib.lb_linear_forward_many(arr, n, _dev_ptr(workspace, "workspace"),
                                    workspace.numel() * workspace.element_size(), _stream(stream))
    _check(st, "lb_linear_forward_many")
    return ys


def lb_list_workspace_bytes(descs, n: int) -> int:
    return int(load_library().lb_list_workspace_bytes(descs, n))


class LittleBitList:
    """A fixed list of decode-sized linears (items (x, paths, r, y), y allocated when None) run by the
    streaming list forward: the plan is written once into the list's workspace (lb_list_init) and every
    forward() is three launches (lb_list_forward).  The tensors must outlive the object and keep their
    storage (the plan holds their addresses)."""

    def __init__(self, items, stream=None):
        torch = _torch()
        self.items = items
        self.descs, self.ys = make_descs(items)
        self.n = len(items)
        lib = load_library()
        need = lb_list_workspace_bytes(self.descs, self.n)
        if need == 0:
            raise LittleBitError(LB_ERR_SHAPE, "lb_list_workspace_bytes (list out of scope or invalid)")
        dev = self.ys[0].device if self.ys else "cuda"
        self.workspace = torch.empty(need, dtype=torch.uint8, device=dev)
        st = lib.lb_list_init(self.descs, self.n, _dev_ptr(self.workspace, "workspace"), need, _stream(stream))
        _check(st, "lb_list_init")

    def forward(self, stream=None):
        st = load_library().lb_list_forward(self.descs, self.n, _dev_ptr(self.workspace, "workspace"),
                                            self.workspace.numel(), _stream(stream))
        _check(st, "lb_list_forward")
        return self.ys


def lb_latent_workspace_bytes(T: int, d_in: int, r: int) -> int:
    return int(load_library().lb_latent_workspace_bytes(T, d_in, r))


def lb_from_latent_workspace_bytes(T: int, r: int) -> int:
    return int(load_library().lb_from_latent_workspace_bytes(T, r))


def _scratch(n: int, device):
    torch = _torch()
    return torch.empty(max(n, 256), dtype=torch.uint8, device=device)


def lb_linear_latent(x, paths: Sequence[LittleBitPath], r: int, w=None, latent_dtype=None, workspace=None,
                     stream=None):
    """The latent cache entries w [T, 2, r] of x [T, d_in] (only V, g, l of the paths are read; latent_dtype
    defaults to float32); returns w."""
    torch = _torch()
    lib = load_library()
    T, d_in = x.shape
    arr, sc = _paths_struct(paths)
    if w is None:
        w = torch.empty((T, 2, r), dtype=latent_dtype or torch.float32, device=x.device)
    if workspace is None:
        workspace = _scratch(lb_latent_workspace_bytes(T, d_in, r), x.device)
    st = lib.lb_linear_latent(_dev_ptr(x, "x"), _dtype_code(x), T, d_in, r, arr, sc, _dev_ptr(w, "w"),
                              _dtype_code(w), _dev_ptr(workspace, "workspace"),
                              workspace.numel() * workspace.element_size(), _stream(stream))
    _check(st, "lb_linear_latent")
    return w


def lb_linear_from_latent(w, paths: Sequence[LittleBitPath], y=None, out_dtype=None, workspace=None, stream=None):
    """y [T, d_out] of the layer from cached latents w [T, 2, r] (only U, h of the paths are read; out_dtype
    defaults to w's dtype); returns y."""
    torch = _torch()
    lib = load_library()
    T, two, r = w.shape
    if two != 2:
        raise ValueError("w must be [T, 2, r]")
    d_out = paths[0].h.shape[0]
    arr, sc = _paths_struct(paths)
    if y is None:
        y = torch.empty((T, d_out), dtype=out_dtype or w.dtype, device=w.device)
    if workspace is None:
        workspace = _scratch(lb_from_latent_workspace_bytes(T, r), w.device)
    st = lib.lb_linear_from_latent(_dev_ptr(w, "w"), _dtype_code(w), T, d_out, r, arr, sc, _dev_ptr(y, "y"),
                                   _dtype_code(y), _dev_ptr(workspace, "workspace"),
                                   workspace.numel() * workspace.element_size(), _stream(stream))
    _check(st, "lb_linear_from_latent")
    return y


def lb_backward_workspace_bytes(T: int, d_in: int, d_out: int, r: int) -> int:
    return int(load_library().lb_backward_workspace_bytes(T, d_in, d_out, r))


@dataclass
class LittleBitPathTrain:
    """One path's fp32 latent factors, their signs packed in the backward's orientation (Ut: U packed
    with LB_ROLE_V, Vt: V packed with LB_ROLE_U) and, after lb_linear_backward, the gradients."""
    U_latent: object
    V_latent: object
    Ut: object = None
    Vt: object = None
    dU: object = None
    dV: object = None
    dh: object = None
    dg: object = None
    dl: object = None


def lb_linear_backward(x, dy, paths: Sequence[LittleBitPath], train: Sequence[LittleBitPathTrain],
                       kappa: float = 100.0, dx=None, need_dx: bool = True, workspace=None, stream=None):
    """Gradients of one layer for x [T, d_in] and dy [T, d_out]: fills (allocating when None) Ut, Vt (packed
    from the latents), dU, dV, dh, dg, dl of each train entry; returns dx (None when need_dx is False)."""
    torch = _torch()
    lib = load_library()
    T, d_in = x.shape
    d_out = dy.shape[1]
    r = train[0].U_latent.shape[1]
    arr, sc = _paths_struct(paths)
    tarr = (lb_path_train * 2)()
    dev = x.device
    for i, q in enumerate(train):
        if q.Ut is None:
            q.Ut = lb_pack_signs(q.U_latent, LB_ROLE_V, stream=stream)
        if q.Vt is None:
            q.Vt = lb_pack_signs(q.V_latent, LB_ROLE_U, stream=stream)
        for name, shape in (("dU", (d_out, r)), ("dV", (d_in, r)), ("dh", (d_out,)), ("dg", (d_in,)), ("dl", (r,))):
            if getattr(q, name) is None:
                setattr(q, name, torch.empty(shape, dtype=torch.float32, device=dev))
        tarr[i] = lb_path_train(*[_dev_ptr(getattr(q, f), f) for f in ("U_latent", "V_latent", "Ut", "Vt", "dU",
                                                                         "dV", "dh", "dg", "dl")])
    if need_dx and dx is None:
        dx = torch.empty((T, d_in), dtype=x.dtype, device=dev)
    if workspace is None:
        workspace = _scratch(lb_backward_workspace_bytes(T, d_in, d_out, r), dev)
    st = lib.lb_linear_backward(_dev_ptr(x, "x"), _dev_ptr(dy, "dy"), _dtype_code(x), T, d_in, d_out, r, arr, sc,
                                tarr, float(kappa), _dev_ptr(dx, "dx") if need_dx else 0,
                                _dev_ptr(workspace, "workspace"), workspace.numel() * workspace.element_size(),
                                _stream(stream))
    _check(st, "lb_linear_backward")
    return dx if need_dx else None


def lb_dense_reference_weight(paths: Sequence[LittleBitPath], d_in: int, d_out: int, r: int, W=None, stream=None):
    """Dense fp32 W_hat [d_out, d_in] from the packed buffers (checking path)."""
    torch = _torch()
    lib = load_library()
    arr, sc = _paths_struct(paths)
    if W is None:
        W = torch.empty((d_out, d_in), dtype=torch.float32, device=paths[0].h.device)
    st = lib.lb_dense_reference_weight(arr, sc, d_in, d_out, r, _dev_ptr(W, "W"), _stream(stream))
    _check(st, "lb_dense_reference_weight")
    return W


def lb_dual_svid_workspace_bytes(d_out: int, d_in: int, r: int, oversample: int) -> int:
    return int(load_library().lb_dual_svid_workspace_bytes(d_out, d_in, r, oversample))


def svid_defaults(r: int, d_out: int, d_in: int):
    """(oversample, iters) used when lb_dual_svid is not given them: a block of about 1.5 r vectors
    (at least r + 16) and 12 rounds of subspace iteration."""
    return max(16, r // 2), 12


def lb_dual_svid(W, r: int, oversample=None, iters=None, seed: int = 0, residual: bool = False, workspace=None,
                 stream=None) -> dict:
    """Dual-SVID of a dense weight W [d_out, d_in] (device, f32 / f16 / bf16) at rank r.  Returns
    {"U": [U'_0, U'_1], "V": [...], "h": [...], "g": [...], "l": [...], "sigma": [...]} (fp32 device
    tensors; U' [d_out, r], V' [d_in, r]) and, with residual=True, "W_res" = W - W_hat_pri,0 (fp32)."""
    torch = _torch()
    lib = load_library()
    d_out, d_in = W.shape
    ov, it = svid_defaults(r, d_out, d_in)
    oversample = ov if oversample is None else oversample
    iters = it if iters is None else iters
    dev = W.device
    f32 = dict(dtype=torch.float32, device=dev)
    out = {"U": [torch.empty((d_out, r), **f32) for _ in range(2)],
           "V": [torch.empty((d_in, r), **f32) for _ in range(2)],
           "h": [torch.empty(d_out, **f32) for _ in range(2)], "g": [torch.empty(d_in, **f32) for _ in range(2)],
           "l": [torch.empty(r, **f32) for _ in range(2)], "sigma": [torch.empty(r, **f32) for _ in range(2)]}
    arr = (lb_svid_out * 2)()
    for p in range(2):
        arr[p] = lb_svid_out(*(_dev_ptr(out[k][p], k) for k in ("U", "V", "h", "g", "l", "sigma")))
    W_res = torch.empty((d_out, d_in), **f32) if residual else None
    need = lb_dual_svid_workspace_bytes(d_out, d_in, r, oversample)
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
    st = lib.lb_dual_svid(_dev_ptr(W, "W"), _dtype_code(W), d_out, d_in, r, oversample, iters,
                          ctypes.c_uint64(seed), arr, _dev_ptr(W_res, "W_res"), _dev_ptr(workspace, "workspace"),
                          workspace.numel() * workspace.element_size(), _stream(stream))
    _check(st, "lb_dual_svid")
    if residual:
        out["W_res"] = W_res
    return out


def littlebit_from_dense(W, r: int, scale_dtype=None, **kw):
    """A LittleBit linear initialised from the dense W [d_out, d_in] by Dual-SVID: the two paths with
    packed signs (LB layout v1) and scales in scale_dtype (default fp16), ready for lb_linear_forward."""
    torch = _torch()
    sd = torch.float16 if scale_dtype is None else scale_dtype
    s = lb_dual_svid(W, r, **kw)
    paths = []
    for p in range(2):
        paths.append(LittleBitPath(U=lb_pack_signs(s["U"][p], LB_ROLE_U), V=lb_pack_signs(s["V"][p], LB_ROLE_V),
                                   h=s["h"][p].to(sd), g=s["g"][p].to(sd), l=s["l"][p].to(sd)))
    return paths


__all__ = [
    "LB_OK", "LB_ERR_NULL", "LB_ERR_SHAPE", "LB_ERR_DTYPE", "LB_ERR_ALIGN", "LB_ERR_WORKSPACE", "LB_ERR_HIP",
    "LB_ERR_ARG", "LB_F32", "LB_F16", "LB_BF16", "LB_ROLE_U", "LB_ROLE_V", "LB_KERNEL_AUTO", "LB_KERNEL_DECODE",
    "LB_KERNEL_PREFILL", "LB_KERNEL_DECODE_MFMA", "LittleBitError", "LittleBitPath", "lb_path", "load_library", "lb_status_str",
    "lb_packed_bytes", "lb_bits_per_weight", "lb_rank_for_bpw", "lb_forward_workspace_bytes",
    "lb_decode_max_tokens", "lb_pack_signs", "lb_workspace_init", "lb_workspace_status", "alloc_workspace", "lb_linear_forward",
    "lb_dense_reference_weight", "lb_linear_forward_noalloc", "lb_linear_desc", "make_descs", "lb_forward_many_workspace_bytes",
    "lb_linear_forward_many", "lb_list_workspace_bytes", "LittleBitList", "lb_latent_workspace_bytes", "lb_from_latent_workspace_bytes", "lb_linear_latent",
    "lb_linear_from_latent", "lb_path_train", "LittleBitPathTrain", "lb_backward_workspace_bytes",
    "lb_linear_backward", "lb_svid_out", "lb_dual_svid_workspace_bytes", "svid_defaults", "lb_dual_svid",
    "littlebit_from_dense",
]
