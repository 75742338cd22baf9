"""GPU parity of the attention gradients (zeta_topk_attn_bwd) against the
float64 oracle (Appendix E.2), for windows chosen by the oracle's selection.

Gradients are float32 on the GPU for both input dtypes, computed from the
exact input values, so one tolerance serves both: max-abs error at most
1e-4 * (1 + max |oracle|) per tensor, and relative 1e-4 for the eps gradient.
"""

import numpy as np
import pytest
import torch

import oracle
import paper_2501_14577_amd as zeta
import workloads
from gpu_util import device, host, i32_to_dev, inputs, log, oracle_select, to_dev

pytestmark = pytest.mark.gpu

# (config, causal, segments compared)
BWD = [(1, True, 1), (2, True, 4), (3, False, 3), (3, True, 3), (4, True, 2)]


@pytest.fixture(scope="module", autouse=True)
def _lib():
    device()
    zeta.load_library()


def _close(got, ref, name):
    tol = 1e-4 * (1.0 + float(np.abs(ref).max()))
    err = float(np.abs(got - ref).max())
    assert err <= tol, (name, err, tol)


def _run(q, k, v, dout, idx, eps, dtype, q_order=None):
    """Upload [S,N,*] arrays as [1,S,N,*] tensors and run the backward."""
    up = (lambda a: to_dev(a[None], dtype))
    out = zeta.zeta_topk_attn_bwd(up(q), up(k), up(v), i32_to_dev(idx[None]), up(dout), eps,
                                  q_order=None if q_order is None else i32_to_dev(q_order))
    torch.cuda.synchronize()
    return [host(t) for t in out]


@pytest.mark.parametrize("cfg,causal,nseg", BWD)
def test_bwd_config(cfg, causal, nseg):
    w, x, f = inputs(cfg)
    log(f"bwd config {cfg} causal={causal} segments={nseg}")
    S = w.segments
    dout_raw = workloads.generate_dout(w).reshape(S, w.N, w.dv)
    raw = {n: a.reshape(S, w.N, -1) for n, a in x.items()}
    idx = oracle_select(cfg, causal)[:nseg]
    dq, dk, dv, deps = _run(raw["q"][:nseg], raw["k"][:nseg], raw["v"][:nseg], dout_raw[:nseg], idx, 0.5, w.dtype)
    dout = oracle.as_f32(dout_raw[:nseg], w.dtype)
    rq, rk, rv, reps = oracle.attend_bwd(f["q"][:nseg], f["k"][:nseg], f["v"][:nseg], idx, 0.5, dout)
    _close(dq.reshape(rq.shape), rq, "dq")
    _close(dk.reshape(rk.shape), rk, "dk")
    _close(dv.reshape(rv.shape), rv, "dv")
    assert abs(float(deps[0]) - reps) <= 1e-4 * (1.0 + abs(reps)), (float(deps[0]), reps)


EDGE = [
    dict(N=1, topk=8, dk=3, dv=64, dtype="f32"),
    dict(N=37, topk=7, dk=3, dv=32, dtype="bf16"),
    dict(N=300, topk=33, dk=2, dv=256, dtype="f32"),
    dict(N=500, topk=64, dk=4, dv=128, dtype="bf16"),
    dict(N=700, topk=1024, dk=3, dv=256, dtype="bf16"),
    dict(N=129, topk=1, dk=3, dv=64, dtype="f32"),
]


@pytest.mark.parametrize("shape", EDGE, ids=[f"N{e['N']}-k{e['topk']}-dk{e['dk']}-dv{e['dv']}-{e['dtype']}" for e in EDGE])
def test_bwd_edges(shape):
    """Small and ragged shapes, every d_v, both dtypes, with empty and partly
    padded windows (the selection's -1 slots, plus rows emptied here)."""
    w = workloads.custom(B=1, H=2, seed=shape["N"] * 7 + shape["topk"], bits=8, **shape)
    log(f"bwd edge {shape}")
    x = workloads.generate(w)
    S = w.segments
    raw = {n: a.reshape(S, w.N, -1) for n, a in x.items()}
    f = {n: oracle.as_f32(a, w.dtype) for n, a in raw.items()}
    qc, kc, _, _ = oracle.morton_encode(f["q"], f["k"], 8 if shape["dk"] <= 4 else 4)
    idx = oracle.select_topk(qc, kc, w.topk, True)
    idx[:, ::5] = -1  # rows without candidates
    dout_raw = workloads.generate_dout(w).reshape(S, w.N, w.dv)
    dq, dk, dv, deps = _run(raw["q"], raw["k"], raw["v"], dout_raw, idx, 0.3, w.dtype)
    rq, rk, rv, reps = oracle.attend_bwd(f["q"], f["k"], f["v"], idx, 0.3, oracle.as_f32(dout_raw, w.dtype))
    _close(dq.reshape(rq.shape), rq, "dq")
    _close(dk.reshape(rk.shape), rk, "dk")
    _close(dv.reshape(rv.shape), rv, "dv")
    assert abs(float(deps[0]) - reps) <= 1e-4 * (1.0 + abs(reps)), (float(deps[0]), reps)
    assert np.all(dq.reshape(rq.shape)[:, ::5] == 0.0)


def test_bwd_long_context():
    """Workload 5 at full size: (1) rows sampled across positions keep their
    windows, every other row is emptied, and all gradients match the oracle;
    (2) with every window, the gradients obey the invariants of the
    definition: shifting every q and k together changes nothing, so
    sum dq + sum dk = 0, and each row's weights sum to 1, so sum dv = sum dout."""
    cfg = 5
    w, x, f = inputs(cfg)
    log("bwd long context")
    S = w.segments
    raw = {n: a.reshape(S, w.N, -1) for n, a in x.items()}
    dout_raw = workloads.generate_dout(w).reshape(S, w.N, w.dv)
    q, k, v, dout = (to_dev(a[None], w.dtype) for a in (raw["q"], raw["k"], raw["v"], dout_raw))
    res = zeta.forward(q.reshape(1, S, w.N, -1), k.reshape(1, S, w.N, -1), v.reshape(1, S, w.N, -1), w.topk, 0.5,
                       True, w.bits, return_intermediates=True)
    idx = res["idx"]
    dq, dk, dv, deps = zeta.zeta_topk_attn_bwd(q, k, v, idx, dout, 0.5, q_order=res["q_order"])
    torch.cuda.synchronize()
    dq, dk, dv = (host(t).reshape(S, w.N, -1).astype(np.float64) for t in (dq, dk, dv))
    dsum = dq.sum(axis=1) + dk.sum(axis=1)
    scale = np.abs(dq).sum(axis=1) + np.abs(dk).sum(axis=1)
    assert np.all(np.abs(dsum) <= 1e-4 * (1.0 + scale)), (dsum, scale)
    dsv = oracle.as_f32(dout_raw, w.dtype).astype(np.float64).sum(axis=1)
    assert np.allclose(dv.sum(axis=1), dsv, rtol=1e-4, atol=1e-2), np.abs(dv.sum(axis=1) - dsv).max()
    assert np.isfinite(float(host(deps)[0]))

    # Sampled rows only, against the oracle (segment 3).
    s = 3
    idx_h = host(idx).reshape(S, w.N, w.topk)[s:s + 1].copy()
    rows = np.unique(np.concatenate([np.arange(4), [127, 128, 255, 256, 4095, 4096, 32767, 32768],
                                     np.random.default_rng(5).integers(0, w.N, 40), [w.N - 1]]))
    keep = np.zeros(w.N, dtype=bool)
    keep[rows] = True
    idx_h[0, ~keep] = -1
    dq1, dk1, dv1, deps1 = _run(raw["q"][s:s + 1], raw["k"][s:s + 1], raw["v"][s:s + 1], dout_raw[s:s + 1], idx_h, 0.5,
                                w.dtype)
    rq, rk, rv, reps = oracle.attend_bwd(f["q"][s:s + 1], f["k"][s:s + 1], f["v"][s:s + 1], idx_h, 0.5,
                                         oracle.as_f32(dout_raw[s:s + 1], w.dtype))
    _close(dq1.reshape(rq.shape), rq, "dq")
    _close(dk1.reshape(rk.shape), rk, "dk")
    _close(dv1.reshape(rv.shape), rv, "dv")
    assert abs(float(deps1[0]) - reps) <= 1e-4 * (1.0 + abs(reps))


def test_bwd_processing_order_and_repeat():
    """Every gradient is bit-identical across runs and processing orders: a
    query's sums are its own, a key's sums run over its queries in sorted
    (query, slot) order, and deps is reduced in a fixed order."""
    cfg = 2
    w, x, _ = inputs(cfg)
    log("bwd processing order")
    S = 8
    raw = {n: a.reshape(w.segments, w.N, -1)[:S] for n, a in x.items()}
    dout_raw = workloads.generate_dout(w).reshape(w.segments, w.N, w.dv)[:S]
    idx = oracle_select(cfg, True)[:S]
    rng = np.random.default_rng(3)
    runs = [_run(raw["q"], raw["k"], raw["v"], dout_raw, idx, 0.5, w.dtype),
            _run(raw["q"], raw["k"], raw["v"], dout_raw, idx, 0.5, w.dtype,
                 q_order=np.stack([rng.permutation(w.N) for _ in range(S)]).astype(np.int32))]
    a, b = runs
    for t in range(4):
        assert np.array_equal(a[t], b[t]), t
