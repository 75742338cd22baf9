"""Seeded synthetic workloads for the Z-order top-k attention forward.

This module only draws random inputs.  It holds none of the method's
arithmetic (no quantisation, no Morton codes, no selection, no attention), so
both the CPU oracle's callers and the GPU path's callers may use it.

Shapes follow the paper's workloads: head counts and value widths from the
experiment details (Appendix C: 8 heads of d_V = 512/8 for LRA, 12 heads of
768/12 for WikiText-103, d_K = 3), the default k = 32 from the k ablation
(Section 4.5), and the longest length N = 65536 of the efficiency table
(Table 3).  None of the paper's datasets is available, so these draws stand in
for them.

Every tensor is laid out ``[B, H, N, d]`` row-major.  Draws are made in
float32 from ``numpy.random.default_rng([seed, stream])`` with stream 0 for q,
1 for k, 2 for v, 3 for mixture centres and 4 for mixture labels.  For bf16
workloads the float32 draws are rounded to bfloat16 (round to nearest, ties to
even, on the bit pattern) and returned as ``uint16`` bit patterns; float32
workloads return ``float32`` arrays.
"""

from __future__ import annotations

import dataclasses
from typing import Dict, Optional, Tuple

import numpy as np

EPS_DEFAULT = 0.5  # gamma^2 = sigmoid(0): the initial value of the learnable scale


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic workload shape."""

    name: str
    B: int
    H: int
    N: int
    dk: int
    dv: int
    topk: int
    dtype: str  # "f32" or "bf16"
    bits: int  # quantisation bits per axis
    causal: Tuple[bool, ...]  # variants to run
    keys: str = "normal"  # "normal" or "mixture16"
    seed: int = 0

    @property
    def segments(self) -> int:
        return self.B * self.H

    @property
    def code_bits(self) -> int:
        return self.dk * self.bits


CONFIGS: Dict[int, Workload] = {
    1: Workload("tiny-single-head", 1, 1, 1024, 3, 64, 32, "f32", 10, (True,), "normal", 1001),
    2: Workload("associative-recall-batch", 32, 4, 2048, 3, 64, 32, "bf16", 10, (True,), "normal", 1002),
    3: Workload("long-range-classification", 16, 8, 4096, 3, 64, 64, "bf16", 10, (False, True), "mixture16", 1003),
    4: Workload("language-model-layer", 8, 12, 8192, 3, 64, 64, "bf16", 10, (True,), "normal", 1004),
    5: Workload("long-context-stress", 1, 16, 65536, 3, 128, 128, "bf16", 6, (True,), "normal", 1005),
}


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even); return uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    if not np.all(np.isfinite(x)):
        raise ValueError("only finite values are rounded")
    # Finite patterns stay below 0xFF800000, so the sum cannot wrap.
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def _draw_normal(seed: int, stream: int, shape) -> np.ndarray:
    return np.random.default_rng([seed, stream]).standard_normal(shape, dtype=np.float32)


def _draw_mixture_keys(seed: int, B: int, H: int, N: int, dk: int, n_comp: int = 16,
                       sigma: float = 0.1) -> np.ndarray:
    """Keys from a per-segment Gaussian mixture: centres ~ N(0, I), labels uniform."""
    centres = np.random.default_rng([seed, 3]).standard_normal((B, H, n_comp, dk), dtype=np.float32)
    labels = np.random.default_rng([seed, 4]).integers(0, n_comp, size=(B, H, N))
    noise = _draw_normal(seed, 1, (B, H, N, dk))
    bi = np.arange(B)[:, None, None]
    hi = np.arange(H)[None, :, None]
    return (centres[bi, hi, labels] + np.float32(sigma) * noise).astype(np.float32)


def generate(w: Workload, seed: Optional[int] = None, *, with_v: bool = True) -> Dict[str, np.ndarray]:
    """Draw q, k, v for workload ``w``.

    Returns a dict with ``q`` [B,H,N,dk], ``k`` [B,H,N,dk] and (if ``with_v``)
    ``v`` [B,H,N,dv] as float32 arrays (dtype "f32") or uint16 bfloat16 bit
    patterns (dtype "bf16").
    """
    seed = w.seed if seed is None else seed
    q = _draw_normal(seed, 0, (w.B, w.H, w.N, w.dk))
    if w.keys == "normal":
        k = _draw_normal(seed, 1, (w.B, w.H, w.N, w.dk))
    elif w.keys == "mixture16":
        k = _draw_mixture_keys(seed, w.B, w.H, w.N, w.dk)
    else:
        raise ValueError(f"unknown key distribution {w.keys!r}")
    out = {"q": q, "k": k}
    if with_v:
        out["v"] = _draw_normal(seed, 2, (w.B, w.H, w.N, w.dv))
    if w.dtype == "bf16":
        out = {name: f32_to_bf16_bits(a) for name, a in out.items()}
    elif w.dtype != "f32":
        raise ValueError(f"unknown dtype {w.dtype!r}")
    return out


def custom(name: str = "custom", *, B=1, H=1, N=64, dk=3, dv=64, topk=8, dtype="f32", bits=10,
           causal=(True,), keys="normal", seed=7) -> Workload:
    """A workload of arbitrary shape, for edge-case tests."""
    return Workload(name, B, H, N, dk, dv, topk, dtype, bits, tuple(causal), keys, seed)


def random_codes(seed: int, shape, code_bits: int) -> np.ndarray:
    """Uniform random codes below 2**code_bits (uint32), for sort and select tests."""
    return np.random.default_rng([seed, 5]).integers(0, 1 << code_bits, size=shape,
                                                    dtype=np.uint64).astype(np.uint32)


def generate_dout(w: Workload, seed: Optional[int] = None) -> np.ndarray:
    """Upstream gradient dL/do for the backward tests, [B,H,N,dv]: N(0,1) in
    stream 6, float32 or bfloat16 bit patterns like v."""
    seed = w.seed if seed is None else seed
    d = _draw_normal(seed, 6, (w.B, w.H, w.N, w.dv))
    return f32_to_bf16_bits(d) if w.dtype == "bf16" else d
