"""Helpers shared by the GPU parity tests: host <-> device marshalling and
cached oracle results for the named workloads."""

from __future__ import annotations

import functools
import sys

import numpy as np
import torch

import oracle
import workloads

TOL = {"f32": 1e-4, "bf16": 2e-2}  # max-abs output error against the float64 oracle


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def device() -> torch.device:
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need a ROCm device")
    return torch.device("cuda:0")


def to_dev(a: np.ndarray, dtype: str) -> torch.Tensor:
    """float32 array, or bfloat16 bit patterns (uint16), to a device tensor."""
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(device())
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device())


def u32_to_dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint32)).to(device())


def i32_to_dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(device())


def host(t: torch.Tensor) -> np.ndarray:
    if t.dtype == torch.bfloat16:
        return t.float().cpu().numpy()
    return t.cpu().numpy()


@functools.lru_cache(maxsize=2)
def inputs(cfg: int):
    """Raw inputs of a named workload plus their float32 values shaped [S, N, d]."""
    w = workloads.CONFIGS[cfg]
    x = workloads.generate(w)
    S = w.segments
    f = {n: oracle.as_f32(a, w.dtype).reshape(S, w.N, a.shape[-1]) for n, a in x.items()}
    return w, x, f


@functools.lru_cache(maxsize=2)
def oracle_codes(cfg: int):
    """Oracle encode and sort of a named workload (cheap at every size)."""
    w, _, f = inputs(cfg)
    qc, kc, lo, hi = oracle.morton_encode(f["q"], f["k"], w.bits)
    sc, perm = oracle.sort_keys(kc)
    return dict(q_codes=qc, k_codes=kc, lo=lo, hi=hi, sorted_codes=sc, perm=perm)


@functools.lru_cache(maxsize=4)
def oracle_select(cfg: int, causal: bool):
    w, _, _ = inputs(cfg)
    oc = oracle_codes(cfg)
    return oracle.select_topk(oc["q_codes"], oc["k_codes"], w.topk, causal)


def sample_rows(N: int, n: int, seed: int) -> np.ndarray:
    """Query positions for sampled checks: the first rows, rows around every
    power of two (where the causal prefix lists switch level), the last rows
    and random ones."""
    edge = {0, 1, 2, 3, N - 1, N - 2}
    t = 1
    while t < N:
        edge.update({t - 1, t, t + 1})
        t <<= 1
    rng = np.random.default_rng(seed)
    rand = set(rng.integers(0, N, size=n).tolist())
    return np.array(sorted(r for r in edge | rand if 0 <= r < N), dtype=np.int64)
