"""GPU parity of the history-mean candidate (Section 3.4, last paragraph)
against the float64 oracle: the means themselves (zeta_history_mean), the
attention with the candidate added (both forward paths) and the gradients
carried back through the means.

Tolerances: the float32 means within 1e-4 * (1 + max |oracle|) (running
float32 sums of up to 65536 terms); outputs within the forward's bounds
(1e-4 float32, 2e-2 bfloat16); gradients as for the plain backward,
1e-4 * (1 + max |oracle|) per tensor and relative 1e-4 for eps.
"""

import numpy as np
import pytest
import torch

import oracle
import paper_2501_14577_amd as zeta
import workloads
from gpu_util import TOL, device, host, i32_to_dev, inputs, log, oracle_select, sample_rows, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    device()
    zeta.load_library()


def _close(got, ref, name):
    tol = 1e-4 * (1.0 + float(np.abs(ref).max()))
    err = float(np.abs(got - ref).max())
    assert err <= tol, (name, err, tol)


def _dev4(a, dtype):
    """[S, N, d] host array -> [1, S, N, d] device tensor."""
    return to_dev(a[None], dtype)


# (config, causal, segments compared)
MEANS = [(1, True, 1), (1, False, 1), (2, True, 8), (3, False, 8), (4, True, 4), (5, True, 2)]


@pytest.mark.parametrize("cfg,causal,nseg", MEANS)
def test_history_mean_config(cfg, causal, nseg):
    w, x, f = inputs(cfg)
    log(f"history mean config {cfg} causal={causal}")
    S = w.segments
    raw = {n: a.reshape(S, w.N, -1)[:nseg] for n, a in x.items()}
    mk, mv = zeta.zeta_history_mean(_dev4(raw["k"], w.dtype), _dev4(raw["v"], w.dtype), causal)
    torch.cuda.synchronize()
    rk, rv = oracle.history_mean(f["k"][:nseg], f["v"][:nseg], causal)
    _close(host(mk).reshape(rk.shape), rk, "mean_k")
    _close(host(mv).reshape(rv.shape), rv, "mean_v")


SHAPES = [
    dict(N=1, dk=3, dv=64, dtype="f32"),
    dict(N=63, dk=3, dv=32, dtype="bf16"),
    dict(N=65, dk=2, dv=256, dtype="f32"),
    dict(N=1000, dk=5, dv=128, dtype="bf16"),
    dict(N=4097, dk=8, dv=256, dtype="bf16"),
    dict(N=129, dk=4, dv=32, dtype="f32"),
]


@pytest.mark.parametrize("shape", SHAPES, ids=[f"N{e['N']}-dk{e['dk']}-dv{e['dv']}-{e['dtype']}" for e in SHAPES])
@pytest.mark.parametrize("causal", [True, False])
def test_history_mean_shapes(shape, causal):
    """Ragged chunk tails, one-row segments, every d_v, d_k from 2 to 8."""
    w = workloads.custom(B=2, H=2, seed=shape["N"] * 3 + shape["dk"], topk=4, bits=4, **shape)
    log(f"history mean shape {shape} causal={causal}")
    x = workloads.generate(w)
    S = w.segments
    raw = {n: a.reshape(S, w.N, -1) for n, a in x.items()}
    mk, mv = zeta.zeta_history_mean(_dev4(raw["k"], w.dtype), _dev4(raw["v"], w.dtype), causal)
    torch.cuda.synchronize()
    rk, rv = oracle.history_mean(oracle.as_f32(raw["k"], w.dtype), oracle.as_f32(raw["v"], w.dtype), causal)
    _close(host(mk).reshape(rk.shape), rk, "mean_k")
    _close(host(mv).reshape(rv.shape), rv, "mean_v")


FORWARD = [(c, causal) for c in (1, 2, 3, 4) for causal in workloads.CONFIGS[c].causal]


@pytest.mark.parametrize("cfg,causal", FORWARD)
def test_history_forward_config(cfg, causal):
    """Both forward paths with the candidate: the windows are the oracle's,
    outputs match the oracle's attention with its own means, and float32
    one-pass outputs are the two calls' bits."""
    w, x, f = inputs(cfg)
    log(f"history forward config {cfg} causal={causal}")
    q, k, v = (to_dev(x[n], w.dtype) for n in ("q", "k", "v"))
    two = zeta.forward(q, k, v, w.topk, 0.5, causal, w.bits, history=True, return_intermediates=True)
    one = zeta.forward(q, k, v, w.topk, 0.5, causal, w.bits, fused=True, history=True, return_intermediates=True)
    torch.cuda.synchronize()
    S = w.segments
    idx = host(two["idx"]).reshape(S, w.N, w.topk)
    assert np.array_equal(idx, oracle_select(cfg, causal))
    assert torch.equal(two["idx"], one["idx"])
    if w.dtype == "f32":
        assert torch.equal(two["out"].view(torch.int32), one["out"].view(torch.int32))
    out2 = host(two["out"]).reshape(S, w.N, w.dv)
    out1 = host(one["out"]).reshape(S, w.N, w.dv)
    for s in range(0, S, max(1, S // 6)):
        mk, mv = oracle.history_mean(f["k"][s:s + 1], f["v"][s:s + 1], causal)
        ref = oracle.attend(f["q"][s:s + 1], f["k"][s:s + 1], f["v"][s:s + 1], idx[s:s + 1], 0.5,
                            mean_k=mk, mean_v=mv)[0]
        assert np.abs(out2[s] - ref).max() <= TOL[w.dtype], ("two calls", s)
        assert np.abs(out1[s] - ref).max() <= TOL[w.dtype], ("one pass", s)


def test_history_forward_long_context():
    """Workload 5 at full size, one-pass path: sampled rows of every segment
    against the oracle's attention with its own means."""
    cfg = 5
    w, x, f = inputs(cfg)
    log("history forward long context")
    q, k, v = (to_dev(x[n], w.dtype) for n in ("q", "k", "v"))
    one = zeta.forward(q, k, v, w.topk, 0.5, True, w.bits, fused=True, history=True, return_intermediates=True)
    torch.cuda.synchronize()
    S = w.segments
    idx = host(one["idx"]).reshape(S, w.N, w.topk)
    out = host(one["out"]).reshape(S, w.N, w.dv)
    rows = sample_rows(w.N, 24, 91)
    for s in range(0, S, 3):
        mk, mv = oracle.history_mean(f["k"][s:s + 1], f["v"][s:s + 1], True)
        ref = oracle.attend(f["q"][s:s + 1], f["k"][s:s + 1], f["v"][s:s + 1], idx[s:s + 1, rows], 0.5, rows=rows,
                            mean_k=mk, mean_v=mv)[0]
        assert np.abs(out[s, rows] - ref).max() <= TOL[w.dtype], s


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_history_empty_window_attends_the_mean(dtype):
    """A row with no valid index attends to its history mean alone."""
    w = workloads.custom(B=1, H=1, N=300, topk=8, dk=3, dv=64, dtype=dtype, bits=8, seed=5)
    x = workloads.generate(w)
    log(f"history empty window {dtype}")
    q, k, v = (to_dev(x[n], dtype) for n in ("q", "k", "v"))
    idx = np.full((1, 1, w.N, w.topk), -1, dtype=np.int32)
    idx[0, 0, ::2, 0] = np.arange(0, w.N, 2)  # every other row keeps its own key
    mk, mv = zeta.zeta_history_mean(k, v, True)
    out = zeta.zeta_topk_attn_fwd(q, k, v, i32_to_dev(idx), 0.5, mean_k=mk, mean_v=mv)
    torch.cuda.synchronize()
    got = host(out)[0, 0, 1::2]
    want = host(mv)[0, 0, 1::2]
    assert np.abs(got - want).max() <= (1e-6 if dtype == "f32" else 1e-2 * (1 + np.abs(want).max()))


@pytest.mark.parametrize("cfg,causal", [(2, True), (3, False)])
def test_history_one_pass_processing_order(cfg, causal):
    """With the candidate, a query's one-pass bits still depend only on its
    own window and means: every processing order gives the same output."""
    from gpu_util import oracle_codes, u32_to_dev
    w, x, _ = inputs(cfg)
    log(f"history processing order config {cfg}")
    oc = oracle_codes(cfg)
    q, k, v = (to_dev(x[n], w.dtype) for n in ("q", "k", "v"))
    mk, mv = zeta.zeta_history_mean(k, v, causal)
    qc, sc, perm = u32_to_dev(oc["q_codes"]), u32_to_dev(oc["sorted_codes"]), i32_to_dev(oc["perm"])
    S = w.segments
    z = np.argsort(oc["q_codes"], axis=1, kind="stable").astype(np.int32)
    rng = np.random.default_rng(12)
    orders = [None, zeta.zeta_query_order(i32_to_dev(z), w.N, S, w.topk, causal),
              i32_to_dev(np.stack([rng.permutation(w.N) for _ in range(S)]))]
    outs = [zeta.zeta_select_attend_fwd(q, k, v, qc, sc, perm, w.topk, causal, 0.5, q_order=o, mean_k=mk,
                                        mean_v=mv) for o in orders]
    torch.cuda.synchronize()
    for o in outs[1:]:
        assert torch.equal(outs[0].view(torch.int16), o.view(torch.int16))


def _bwd(raw, dout_raw, idx, eps, dtype, causal, q_order=None):
    q, k, v = (_dev4(raw[n], dtype) for n in ("q", "k", "v"))
    dout = _dev4(dout_raw, dtype)
    mk, mv = zeta.zeta_history_mean(k, v, causal)
    out = zeta.zeta_topk_attn_bwd(q, k, v, i32_to_dev(idx[None]), dout, eps, mean_k=mk, mean_v=mv, causal=causal,
                                  q_order=None if q_order is None else i32_to_dev(q_order))
    torch.cuda.synchronize()
    return [host(t) for t in out]


def _bwd_check(got, f, dout, idx, eps, causal):
    rq, rk, rv, reps = oracle.attend_bwd(f["q"], f["k"], f["v"], idx, eps, dout, history=True, causal=causal)
    dq, dk, dv, deps = got
    _close(dq.reshape(rq.shape), rq, "dq")
    _close(dk.reshape(rk.shape), rk, "dk")
    _close(dv.reshape(rv.shape), rv, "dv")
    assert abs(float(deps[0]) - reps) <= 1e-4 * (1.0 + abs(reps)), (float(deps[0]), reps)


BWD = [(1, True, 1), (2, True, 4), (3, False, 3), (4, True, 2)]


@pytest.mark.parametrize("cfg,causal,nseg", BWD)
def test_history_bwd_config(cfg, causal, nseg):
    w, x, f = inputs(cfg)
    log(f"history bwd config {cfg} causal={causal}")
    S = w.segments
    raw = {n: a.reshape(S, w.N, -1)[:nseg] for n, a in x.items()}
    dout_raw = workloads.generate_dout(w).reshape(S, w.N, w.dv)[:nseg]
    idx = oracle_select(cfg, causal)[:nseg]
    got = _bwd(raw, dout_raw, idx, 0.5, w.dtype, causal)
    ff = {n: a[:nseg] for n, a in f.items()}
    _bwd_check(got, ff, oracle.as_f32(dout_raw, w.dtype), idx, 0.5, causal)


BWD_EDGE = [
    dict(N=1, topk=8, dk=3, dv=64, dtype="f32"),
    dict(N=37, topk=7, dk=3, dv=32, dtype="bf16"),
    dict(N=300, topk=33, dk=2, dv=256, dtype="f32"),
    dict(N=500, topk=64, dk=4, dv=128, dtype="bf16"),
    dict(N=129, topk=1, dk=3, dv=64, dtype="f32"),
]


@pytest.mark.parametrize("shape", BWD_EDGE,
                         ids=[f"N{e['N']}-k{e['topk']}-dk{e['dk']}-dv{e['dv']}-{e['dtype']}" for e in BWD_EDGE])
@pytest.mark.parametrize("causal", [True, False])
def test_history_bwd_edges(shape, causal):
    """Ragged shapes with rows whose window is empty (they attend to their
    history mean alone)."""
    w = workloads.custom(B=1, H=2, seed=shape["N"] * 5 + shape["topk"], bits=8, **shape)
    log(f"history bwd edge {shape} causal={causal}")
    x = workloads.generate(w)
    S = w.segments
    raw = {n: a.reshape(S, w.N, -1) for n, a in x.items()}
    f = {n: oracle.as_f32(a, w.dtype) for n, a in raw.items()}
    qc, kc, _, _ = oracle.morton_encode(f["q"], f["k"], 8 if shape["dk"] <= 4 else 4)
    idx = oracle.select_topk(qc, kc, w.topk, causal)
    idx[:, ::5] = -1
    dout_raw = workloads.generate_dout(w).reshape(S, w.N, w.dv)
    got = _bwd(raw, dout_raw, idx, 0.3, w.dtype, causal)
    _bwd_check(got, f, oracle.as_f32(dout_raw, w.dtype), idx, 0.3, causal)


def test_history_bwd_long_context_segment():
    """Workload 5, one segment at full length (N = 65536): sampled rows keep
    their windows and every row has its history mean; all gradients match the
    oracle, including the reverse sums over 65536 rows."""
    cfg = 5
    w, x, f = inputs(cfg)
    log("history bwd long context")
    S = w.segments
    s = 5
    raw = {n: a.reshape(S, w.N, -1)[s:s + 1] for n, a in x.items()}
    dout_raw = workloads.generate_dout(w).reshape(S, w.N, w.dv)[s:s + 1]
    q, k, v = (_dev4(raw[n], w.dtype) for n in ("q", "k", "v"))
    res = zeta.forward(q, k, v, w.topk, 0.5, True, w.bits, return_intermediates=True)
    torch.cuda.synchronize()
    idx = host(res["idx"]).reshape(1, w.N, w.topk).copy()
    keep = np.zeros(w.N, dtype=bool)
    keep[sample_rows(w.N, 40, 17)] = True
    idx[0, ~keep] = -1
    got = _bwd(raw, dout_raw, idx, 0.5, w.dtype, True)
    ff = {n: a[s:s + 1] for n, a in f.items()}
    _bwd_check(got, ff, oracle.as_f32(dout_raw, w.dtype), idx, 0.5, True)


def test_history_bwd_processing_order_and_repeat():
    """Bit-identical gradients across runs and processing orders with the
    candidate: the reverse sums run in a fixed order too."""
    cfg = 2
    w, x, _ = inputs(cfg)
    log("history bwd processing order")
    S = 8
    raw = {n: a.reshape(w.segments, w.N, -1)[:S] for n, a in x.items()}
    dout_raw = workloads.generate_dout(w).reshape(w.segments, w.N, w.dv)[:S]
    idx = oracle_select(cfg, True)[:S]
    rng = np.random.default_rng(4)
    a = _bwd(raw, dout_raw, idx, 0.5, w.dtype, True)
    b = _bwd(raw, dout_raw, idx, 0.5, w.dtype, True,
             q_order=np.stack([rng.permutation(w.N) for _ in range(S)]).astype(np.int32))
    for t in range(4):
        assert np.array_equal(a[t], b[t]), t


@pytest.mark.parametrize("dv", [32, 128, 256])
@pytest.mark.parametrize("causal", [True, False])
def test_history_tile_widths(dv, causal):
    """The bfloat16 one-pass call with the candidate at every other value
    width of the matrix-core tiles (the configurations use d_v = 64), on a
    ragged length: the oracle's attention with its own means, and the same
    bits in position order as in level order."""
    w = workloads.custom(B=1, H=2, N=650, dv=dv, topk=24, dtype="bf16", bits=8, seed=dv + 3)
    log(f"history tiles dv={dv} causal={causal}")
    x = workloads.generate(w)
    S = w.segments
    f = {n: oracle.as_f32(a, w.dtype).reshape(S, w.N, -1) for n, a in x.items()}
    q, k, v = (to_dev(x[n], w.dtype) for n in ("q", "k", "v"))
    res = zeta.forward(q, k, v, w.topk, 0.5, causal, w.bits, fused=True, history=True, return_intermediates=True)
    pos = zeta.zeta_select_attend_fwd(q, k, v, res["q_codes"], res["sorted_codes"], res["perm"], w.topk, causal, 0.5,
                                      mean_k=res["mean_k"], mean_v=res["mean_v"])
    torch.cuda.synchronize()
    assert torch.equal(res["out"].view(torch.int16), pos.view(torch.int16))
    idx = host(res["idx"]).reshape(S, w.N, w.topk)
    qc, kc, _, _ = oracle.morton_encode(f["q"], f["k"], w.bits)
    assert np.array_equal(idx, oracle.select_topk(qc, kc, w.topk, causal))
    mk, mv = oracle.history_mean(f["k"], f["v"], causal)
    ref = oracle.attend(f["q"], f["k"], f["v"], idx, 0.5, mean_k=mk, mean_v=mv)
    out = host(res["out"]).reshape(S, w.N, w.dv)
    assert np.abs(out - ref).max() <= TOL[w.dtype], (causal, dv)
