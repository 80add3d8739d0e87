"""Shared helpers for the parity tests: move seeded inputs to the GPU and to the
oracle, and compare results.  The oracle side widens the stored bytes itself
and packs/unpacks signs with its own packer; nothing here does the method's
arithmetic."""
from __future__ import annotations

import numpy as np

import oracle as O
from paper_2506_13771_amd import synth

DT_TORCH = {}


def torch_dtype(code: str):
    import torch
    return {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}[code]


def raw_to_torch(raw: np.ndarray, code: str, device="cuda"):
    import torch
    if code == "f32":
        t = torch.from_numpy(np.ascontiguousarray(raw, dtype=np.float32))
    else:
        t = torch.from_numpy(np.ascontiguousarray(raw).view(np.int16)).view(torch_dtype(code))
    return t.to(device)


def torch_to_raw(t, code: str) -> np.ndarray:
    import torch
    t = t.detach().cpu().contiguous()
    if code == "f32":
        return t.numpy()
    return t.view(torch.int16).numpy().view(np.uint16)


def oracle_signs(li: synth.LinearInputs):
    """(U, V) int8 sign matrices per path, derived by the ORACLE's own packer/unpacker."""
    U, V, Ub, Vb = [], [], [], []
    for p in range(len(li.h)):
        if li.U_latent is not None:
            ub, _ = O.pack(li.U_latent[p].astype(np.float64), O.ROLE_U)
            vb, _ = O.pack(li.V_latent[p].astype(np.float64), O.ROLE_V)
        else:
            ub, vb = li.U_words[p], li.V_words[p]
        Ub.append(ub)
        Vb.append(vb)
        U.append(O.unpack(ub, li.d_out, li.r, O.ROLE_U))
        V.append(O.unpack(vb, li.d_in, li.r, O.ROLE_V))
    return U, V, Ub, Vb


def oracle_scales(li: synth.LinearInputs):
    h = [O.to_f64(a, li.scale_dtype) for a in li.h]
    g = [O.to_f64(a, li.scale_dtype) for a in li.g]
    l = [O.to_f64(a, li.scale_dtype) for a in li.l]
    return h, g, l


def oracle_forward(li: synth.LinearInputs, tokens=None):
    """O1 on the layer's inputs (every token, or the given ones).  Runs the OpenMP form of
    O1, which performs the same operations per output in the same order as the serial one
    (bit-identical, pinned in test_oracle.py), on the host's cores."""
    U, V, _, _ = oracle_signs(li)
    h, g, l = oracle_scales(li)
    x = O.to_f64(li.x, li.act_dtype)
    if tokens is not None:
        x = x[tokens]
    return O.forward_factored_par(x, U, V, h, g, l, host_threads())


def host_threads() -> int:
    import os
    n = len(os.sched_getaffinity(0))
    env = os.environ.get("OMP_NUM_THREADS", "")
    if env.isdigit() and int(env) > 0:
        n = min(n, int(env))
    return max(1, min(n, 16))


def to_device(li: synth.LinearInputs, pack_on_gpu: bool = True):
    """Device tensors for the product path.  Signs are packed by lb_pack_signs on the GPU
    from the fp32 latents (or uploaded as drawn words)."""
    import torch
    import paper_2506_13771_amd as lb
    paths = []
    packed = []
    for p in range(2):
        if li.U_latent is not None and pack_on_gpu:
            Ut = torch.from_numpy(li.U_latent[p]).cuda()
            Vt = torch.from_numpy(li.V_latent[p]).cuda()
            ub = lb.lb_pack_signs(Ut, lb.LB_ROLE_U)
            vb = lb.lb_pack_signs(Vt, lb.LB_ROLE_V)
        else:
            ub = torch.from_numpy(np.ascontiguousarray(li.U_words[p])).cuda()
            vb = torch.from_numpy(np.ascontiguousarray(li.V_words[p])).cuda()
        packed.append((ub, vb))
        paths.append(lb.LittleBitPath(U=ub, V=vb, h=raw_to_torch(li.h[p], li.scale_dtype),
                                      g=raw_to_torch(li.g[p], li.scale_dtype),
                                      l=raw_to_torch(li.l[p], li.scale_dtype)))
    x = raw_to_torch(li.x, li.act_dtype)
    return x, paths, packed


def row_inf_rel(y: np.ndarray, ref: np.ndarray) -> float:
    """max over token rows of max_i |y - ref| / max_i |ref| (the bf16 tolerance metric)."""
    if y.size == 0:
        return 0.0
    num = np.abs(y - ref).max(axis=1)
    den = np.abs(ref).max(axis=1)
    den = np.where(den == 0, 1.0, den)
    return float((num / den).max())


def rel_l2(y: np.ndarray, ref: np.ndarray) -> float:
    n = np.linalg.norm(ref)
    return float(np.linalg.norm(y - ref) / (n if n > 0 else 1.0))


# tolerances (stated by the benchmark configurations): fp32 activations -> relative L2 1e-5;
# bf16 activations with fp32 accumulation -> max relative error 1e-2, read per token row.
TOL_F32_REL_L2 = 1e-5
TOL_BF16_ROW_INF = 1e-2
