"""Seeded synthetic inputs for LittleBit linear layers.

This module only draws random numbers and stores them in the layer's input
dtypes; it holds none of the method's arithmetic.  The GPU path and the fp64
oracle both consume exactly the bytes produced here, so both see identical
inputs.

Recipe (the paper's own kernel benchmark uses layer shapes only, no trained
weights; trained LittleBit checkpoints are not available, so these stand in):
  * signs:  latent factors U_p [d_out x r], V_p [d_in x r] drawn N(0,1) in
            fp32 (their signs are Bernoulli(1/2)); for very large sweeps the
            packed words are drawn directly as uniform random 32-bit words,
            which is Bernoulli(1/2) per bit under any bit layout;
  * scales: h_p, g_p, l_p drawn |N(0,1)| (l_p optionally divided by sqrt(r))
            in fp64, rounded once (round-to-nearest-even) to fp16 or fp32;
  * x:      N(0,1) in fp64, rounded to fp32 (RNE) and, for bf16, from there to
            bf16 (RNE).
Every tensor has its own PCG64 stream keyed by (BASE_SEED, config id, linear
id, tensor id), so any tensor can be regenerated alone.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

BASE_SEED = 2506137710

F32, F16, BF16 = "f32", "f16", "bf16"

# tensor ids inside one linear
_T_X, _T_U, _T_V, _T_H, _T_G, _T_L = 0, 1, 2, 3, 4, 5


def rng(cfg: int, linear: int, tensor: int, path: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64([BASE_SEED, cfg, linear, tensor, path]))


def quantize(v: np.ndarray, dtype: str) -> np.ndarray:
    """fp64 values -> stored representation: float32 array, or uint16 bit patterns for f16/bf16."""
    v = np.asarray(v, dtype=np.float64)
    if dtype == F32:
        return v.astype(np.float32)
    if dtype == F16:
        return v.astype(np.float16).view(np.uint16)
    if dtype == BF16:
        u = v.astype(np.float32).view(np.uint32).astype(np.uint64)
        nan = np.isnan(v)
        u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
        out = u.astype(np.uint16)
        out[nan] = 0x7FC0
        return out
    raise ValueError(dtype)


def elem_bytes(dtype: str) -> int:
    return 4 if dtype == F32 else 2


@dataclass
class LinearInputs:
    d_in: int
    d_out: int
    r: int
    T: int
    act_dtype: str
    scale_dtype: str
    x: np.ndarray                      # raw [T, d_in]
    h: List[np.ndarray]                # raw [d_out] per path
    g: List[np.ndarray]                # raw [d_in] per path
    l: List[np.ndarray]                # raw [r] per path
    U_latent: Optional[List[np.ndarray]] = None   # float32 [d_out, r] per path
    V_latent: Optional[List[np.ndarray]] = None   # float32 [d_in, r] per path
    U_words: Optional[List[np.ndarray]] = None    # uint8 packed bytes per path (direct draw)
    V_words: Optional[List[np.ndarray]] = None
    meta: dict = field(default_factory=dict)


def make_x(T: int, d_in: int, act_dtype: str, cfg: int, linear: int) -> np.ndarray:
    v = rng(cfg, linear, _T_X).standard_normal((T, d_in))
    return quantize(v.astype(np.float32).astype(np.float64), act_dtype)


def make_linear(d_in: int, d_out: int, r: int, T: int, act_dtype: str = BF16, scale_dtype: str = F16,
                cfg: int = 0, linear: int = 0, l_over_sqrt_r: bool = False,
                direct_words: bool = False, npaths: int = 2) -> LinearInputs:
    """Draw one linear layer's inputs.  With direct_words, packed sign buffers are drawn as
    uniform random bytes of the sizes given by the layout (requires shapes with no pad bits:
    d_in % 32 == 0 and r % 32 in {0, 16})."""
    x = make_x(T, d_in, act_dtype, cfg, linear)
    h, g, l = [], [], []
    U_lat, V_lat, U_w, V_w = [], [], [], []
    for p in range(npaths):
        h.append(quantize(np.abs(rng(cfg, linear, _T_H, p).standard_normal(d_out)), scale_dtype))
        g.append(quantize(np.abs(rng(cfg, linear, _T_G, p).standard_normal(d_in)), scale_dtype))
        lv = np.abs(rng(cfg, linear, _T_L, p).standard_normal(r))
        if l_over_sqrt_r:
            lv = lv / np.sqrt(r)
        l.append(quantize(lv, scale_dtype))
        if direct_words:
            if d_in % 32 != 0 or (r % 32) not in (0, 16):
                raise ValueError("direct word draw needs d_in % 32 == 0 and r % 32 in {0, 16}")
            nbu = (r // 32) * 4 * d_out + (2 * d_out if r % 32 == 16 else 0)
            nbv = (d_in // 32) * 4 * r
            U_w.append(rng(cfg, linear, _T_U, p).integers(0, 256, nbu, dtype=np.uint8))
            V_w.append(rng(cfg, linear, _T_V, p).integers(0, 256, nbv, dtype=np.uint8))
        else:
            U_lat.append(rng(cfg, linear, _T_U, p).standard_normal((d_out, r), dtype=np.float32))
            V_lat.append(rng(cfg, linear, _T_V, p).standard_normal((d_in, r), dtype=np.float32))
    return LinearInputs(d_in, d_out, r, T, act_dtype, scale_dtype, x, h, g, l,
                        U_latent=None if direct_words else U_lat,
                        V_latent=None if direct_words else V_lat,
                        U_words=U_w if direct_words else None,
                        V_words=V_w if direct_words else None)


_T_W = 6


def dense_weight(d_out: int, d_in: int, k: int, noise: float, cfg: int, linear: int = 0) -> np.ndarray:
    """A dense weight for the Dual-SVID conversion, fp32 [d_out, d_in]: a rank-k part whose column
    scales fall linearly from 3 to 1 (A [d_out, k], B [d_in, k] standard normal, A diag(s) B^T /
    sqrt(k)) plus i.i.d. N(0, noise^2) entries -- a decaying spectrum above a noise floor, as in the
    pretrained weights the conversion is applied to."""
    rs = rng(cfg, linear, _T_W)
    A = rs.standard_normal((d_out, k)) * np.linspace(3.0, 1.0, k) if k > 0 else np.zeros((d_out, 0))
    B = rs.standard_normal((d_in, k))
    W = A @ B.T / np.sqrt(max(k, 1)) + noise * rs.standard_normal((d_out, d_in))
    return W.astype(np.float32)


# ----------------------------------------------------------------------------
# The benchmark configurations (shapes of Llama-2 7B / 13B / 70B linears).
# ----------------------------------------------------------------------------
LLAMA2_7B = [("q", 4096, 4096), ("k", 4096, 4096), ("v", 4096, 4096), ("o", 4096, 4096),
             ("gate", 4096, 11008), ("up", 4096, 11008), ("down", 11008, 4096)]
LLAMA2_13B = [("q", 5120, 5120), ("k", 5120, 5120), ("v", 5120, 5120), ("o", 5120, 5120),
              ("gate", 5120, 13824), ("up", 5120, 13824), ("down", 13824, 5120)]
LLAMA2_70B = [("q", 8192, 8192), ("k", 8192, 1024), ("v", 8192, 1024), ("o", 8192, 8192),
              ("gate", 8192, 28672), ("up", 8192, 28672), ("down", 28672, 8192)]
