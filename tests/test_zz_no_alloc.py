"""The allocation-free encode (zeta_morton_encode_static) through the C ABI
against the workspace call (zeta_morton_encode): identical codes and range on
two calls in a row, the second smaller (the per-GPU scratch keeps the first
call's partials, which the second must not read), both dtypes, and with a
caller range (no scratch used)."""

import numpy as np
import pytest
import torch

import oracle
import paper_2501_14577_amd as zeta
import workloads
from gpu_util import device, host, log, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    device()
    zeta.load_library()


CALLS = [  # (B, H, N, d_k, bits, dtype): the second of each pair is smaller
    ((1, 16, 65536, 3, 6, "bf16"), (2, 3, 1000, 3, 6, "bf16")),
    ((4, 8, 4097, 3, 10, "f32"), (1, 1, 37, 3, 10, "f32")),
    ((2, 5, 3000, 5, 6, "bf16"), (1, 2, 513, 2, 16, "bf16")),
]


@pytest.mark.parametrize("pair", CALLS, ids=[f"{a[2]}-then-{b[2]}" for a, b in CALLS])
def test_static_encode_matches_workspace_encode(pair):
    for n, (B, H, N, dk, bits, dtype) in enumerate(pair):
        log(f"static encode call {n}: B={B} H={H} N={N} d_k={dk} bits={bits} {dtype}")
        w = workloads.custom(B=B, H=H, N=N, dk=dk, dtype=dtype, bits=bits, seed=N + dk)
        x = workloads.generate(w, with_v=False)
        q, k = to_dev(x["q"], dtype), to_dev(x["k"], dtype)
        S = w.segments
        r1 = torch.empty((S, 2, dk), dtype=torch.float32, device=device())
        r2 = torch.empty_like(r1)
        qa, ka = zeta.zeta_morton_encode(q, k, bits, range_out=r1)
        qb, kb = zeta.zeta_morton_encode_static(q, k, bits, range_out=r2)
        torch.cuda.synchronize()
        assert torch.equal(qa, qb) and torch.equal(ka, kb)
        assert torch.equal(r1, r2)
        # Codes as the oracle gives them (the workspace call is pinned to it elsewhere).
        f = {m: oracle.as_f32(x[m], dtype).reshape(S, N, dk) for m in ("q", "k")}
        eq, ek, _, _ = oracle.morton_encode(f["q"], f["k"], bits)
        assert np.array_equal(host(qb).reshape(S, N), eq) and np.array_equal(host(kb).reshape(S, N), ek)


def test_static_encode_caller_range():
    """With a caller range the call needs no scratch; codes equal the workspace call's."""
    w = workloads.custom(B=1, H=3, N=777, dk=3, dtype="bf16", bits=10, seed=5)
    x = workloads.generate(w, with_v=False)
    q, k = to_dev(x["q"], "bf16"), to_dev(x["k"], "bf16")
    lohi = torch.tensor([[[-1.5] * 3, [1.25] * 3]] * 3, dtype=torch.float32, device=device())
    qa, ka = zeta.zeta_morton_encode(q, k, 10, range_lohi=lohi)
    qb, kb = zeta.zeta_morton_encode_static(q, k, 10, range_lohi=lohi)
    torch.cuda.synchronize()
    assert torch.equal(qa, qb) and torch.equal(ka, kb)
