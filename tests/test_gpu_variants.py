"""GPU parity of the variants against the float64 oracle: the paper's chunked
causal rule (Section 3.2.2; Algorithm 1, Step 4; pool = positions below
floor(i / M) * M) and the score variants it compares with the Cauchy score
(Section 4.3; Appendix G.2; equation 3).

Indices are compared bit for bit; outputs within the forward's bounds
(max-abs 1e-4 float32, 2e-2 bfloat16).  float32 one-pass outputs are the
two-call outputs' bits.
"""

import numpy as np
import pytest
import torch

import oracle
import paper_2501_14577_amd as zeta
import workloads
from gpu_util import (TOL, device, host, i32_to_dev, inputs, log, oracle_codes, sample_rows, to_dev,
                      u32_to_dev)

pytestmark = pytest.mark.gpu

MODES = ["dot", "neg_euclid", "inv_euclid", "norm_dot"]


@pytest.fixture(scope="module", autouse=True)
def _lib():
    device()
    zeta.load_library()


# The paper sets the number of chunks to 4, 8, 16 or 32 (Appendix C).
CHUNKED = [(1, 4), (2, 16), (3, 8), (4, 32)]


@pytest.mark.parametrize("cfg,nchunks", CHUNKED)
def test_chunked_select_config(cfg, nchunks):
    """The chunked rule's windows on the named workloads, both select paths."""
    w, x, f = inputs(cfg)
    M = w.N // nchunks
    log(f"chunked select config {cfg} M={M}")
    oc = oracle_codes(cfg)
    want = oracle.select_topk(oc["q_codes"], oc["k_codes"], w.topk, True, chunk=M)
    qc, sc, perm = u32_to_dev(oc["q_codes"]), u32_to_dev(oc["sorted_codes"]), i32_to_dev(oc["perm"])
    got = host(zeta.zeta_select_topk(qc, sc, perm, w.topk, True, chunk=M))
    assert np.array_equal(got.reshape(want.shape), want)
    q, k, v = (to_dev(x[n], w.dtype) for n in ("q", "k", "v"))
    idx1 = torch.empty((w.B, w.H, w.N, w.topk), dtype=torch.int32, device=device())
    out = zeta.zeta_select_attend_fwd(q, k, v, qc, sc, perm, w.topk, True, 0.5, chunk=M,
                                      idx_out=idx1)
    torch.cuda.synchronize()
    assert np.array_equal(host(idx1).reshape(want.shape), want)
    out = host(out).reshape(w.segments, w.N, w.dv)
    assert np.all(out[:, :M] == 0.0)  # the first chunk attends to nothing
    for s in range(0, w.segments, max(1, w.segments // 6)):
        ref = oracle.attend(f["q"][s:s + 1], f["k"][s:s + 1], f["v"][s:s + 1], want[s:s + 1, M:], 0.5,
                            rows=np.arange(M, w.N))[0]
        assert np.abs(out[s, M:] - ref).max() <= TOL[w.dtype], s


CHUNK_EDGE = [
    dict(N=1, topk=8, chunk=1, dtype="f32"),
    dict(N=37, topk=7, chunk=1, dtype="bf16"),
    dict(N=300, topk=16, chunk=7, dtype="bf16"),
    dict(N=1000, topk=100, chunk=999, dtype="f32"),
    dict(N=700, topk=1024, chunk=64, dtype="bf16"),
    dict(N=513, topk=64, chunk=2000, dtype="bf16"),
    dict(N=4097, topk=33, chunk=300, dtype="f32"),
    # The window search's 16-bit positions at their largest N, then 32-bit.
    dict(N=65536, topk=16, chunk=4096, dtype="bf16"),
    dict(N=70001, topk=16, chunk=5000, dtype="bf16"),
]


@pytest.mark.parametrize("shape", CHUNK_EDGE, ids=[f"N{e['N']}-k{e['topk']}-M{e['chunk']}-{e['dtype']}"
                                                   for e in CHUNK_EDGE])
@pytest.mark.parametrize("fused", [False, True])
def test_chunked_forward_edges(shape, fused):
    """Chunk sizes of 1, of N - 1 and beyond N, chunks not dividing N, and
    windows longer than the pool: the whole forward against the oracle."""
    M = shape["chunk"]
    w = workloads.custom(B=2, H=1, seed=shape["N"] + M, N=shape["N"], topk=shape["topk"], dtype=shape["dtype"],
                         dv=64, bits=8)
    log(f"chunked forward edge {shape} fused={fused}")
    x = workloads.generate(w)
    S = w.segments
    f = {n: oracle.as_f32(a, w.dtype).reshape(S, w.N, -1) for n, a in x.items()}
    ref = oracle.forward(f["q"], f["k"], f["v"], w.topk, 0.5, True, w.bits, chunk=M)
    res = zeta.forward(to_dev(x["q"], w.dtype), to_dev(x["k"], w.dtype), to_dev(x["v"], w.dtype), w.topk, 0.5, True,
                       w.bits, fused=fused, chunk=M, return_intermediates=True)
    torch.cuda.synchronize()
    assert np.array_equal(host(res["idx"]).reshape(S, w.N, w.topk), ref["idx"])
    out = host(res["out"]).reshape(S, w.N, w.dv)
    empty = np.all(ref["idx"] < 0, axis=-1)
    assert np.all(out[empty] == 0.0)
    assert np.abs(out[~empty] - ref["out"][~empty]).max(initial=0.0) <= TOL[w.dtype]


def test_chunked_long_context_sampled():
    """Workload 5 with 32 chunks (M = 2048), one-pass path: the windows and
    outputs of sampled rows of every segment."""
    cfg = 5
    w, x, f = inputs(cfg)
    M = w.N // 32
    log(f"chunked long context M={M}")
    oc = oracle_codes(cfg)
    q, k, v = (to_dev(x[n], w.dtype) for n in ("q", "k", "v"))
    res = zeta.forward(q, k, v, w.topk, 0.5, True, w.bits, fused=True, chunk=M, return_intermediates=True)
    torch.cuda.synchronize()
    S = w.segments
    idx = host(res["idx"]).reshape(S, w.N, w.topk)
    out = host(res["out"]).reshape(S, w.N, w.dv)
    rows = np.unique(np.concatenate([sample_rows(w.N, 16, 8), [M - 1, M, M + 1, 2 * M - 1, 2 * M]]))
    rows = rows[rows >= M]
    for s in range(0, S, 3):
        sel = np.stack([oracle.select_one(int(oc["q_codes"][s, i]), oc["k_codes"][s], int(i), w.topk, True, chunk=M)
                        for i in rows])
        assert np.array_equal(idx[s, rows], sel), s
        ref = oracle.attend(f["q"][s:s + 1], f["k"][s:s + 1], f["v"][s:s + 1], sel[None], 0.5, rows=rows)[0]
        assert np.abs(out[s, rows] - ref).max() <= TOL[w.dtype], s
    assert np.all(idx[:, :M] == -1) and np.all(out[:, :M] == 0.0)


def test_chunked_processing_order():
    """The chunked windows do not depend on the processing order."""
    cfg = 3
    w, x, _ = inputs(cfg)
    M = w.N // 16
    log("chunked processing order")
    oc = oracle_codes(cfg)
    qc, sc, perm = u32_to_dev(oc["q_codes"]), u32_to_dev(oc["sorted_codes"]), i32_to_dev(oc["perm"])
    S = w.segments
    z = np.argsort(oc["q_codes"], axis=1, kind="stable").astype(np.int32)
    rng = np.random.default_rng(21)
    orders = [None, zeta.zeta_query_order(i32_to_dev(z), w.N, S, w.topk, True),
              zeta.zeta_query_order(i32_to_dev(z), w.N, S, w.topk, True, chunk=M),
              i32_to_dev(np.stack([rng.permutation(w.N) for _ in range(S)]))]
    q, k, v = (to_dev(x[n], w.dtype) for n in ("q", "k", "v"))
    idxs = [zeta.zeta_select_topk(qc, sc, perm, w.topk, True, chunk=M, q_order=o) for o in orders]
    outs = [zeta.zeta_select_attend_fwd(q, k, v, qc, sc, perm, w.topk, True, 0.5, chunk=M, q_order=o) for o in orders]
    torch.cuda.synchronize()
    for a in idxs[1:]:
        assert torch.equal(idxs[0], a)
    for a in outs[1:]:
        assert torch.equal(outs[0].view(torch.int16), a.view(torch.int16))


# ----------------------------------------------------------------------------
# Score variants
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("cfg,causal", [(1, True), (2, True), (3, False), (4, True)])
def test_score_modes_config(mode, cfg, causal):
    """Both forward paths with each variant: the two calls and the one-pass
    call agree (bit for bit in float32) and match the oracle."""
    w, x, f = inputs(cfg)
    log(f"score {mode} config {cfg} causal={causal}")
    q, k, v = (to_dev(x[n], w.dtype) for n in ("q", "k", "v"))
    two = zeta.forward(q, k, v, w.topk, 0.5, causal, w.bits, score=mode, return_intermediates=True)
    one = zeta.forward(q, k, v, w.topk, 0.5, causal, w.bits, fused=True, score=mode, return_intermediates=True)
    torch.cuda.synchronize()
    assert torch.equal(two["idx"], one["idx"])
    S = w.segments
    if w.dtype == "f32":
        assert torch.equal(two["out"].view(torch.int32), one["out"].view(torch.int32))
    idx = host(two["idx"]).reshape(S, w.N, w.topk)
    out1 = host(one["out"]).reshape(S, w.N, w.dv)
    out2 = host(two["out"]).reshape(S, w.N, w.dv)
    for s in range(0, S, max(1, S // 4)):
        ref = oracle.attend(f["q"][s:s + 1], f["k"][s:s + 1], f["v"][s:s + 1], idx[s:s + 1], 0.5, mode=mode)[0]
        assert np.abs(out2[s] - ref).max() <= TOL[w.dtype], ("two calls", s)
        assert np.abs(out1[s] - ref).max() <= TOL[w.dtype], ("one pass", s)


SCORE_EDGE = [
    dict(N=5, topk=8, dk=3, dv=32, dtype="f32"),
    dict(N=300, topk=33, dk=2, dv=256, dtype="bf16"),
    dict(N=600, topk=1024, dk=4, dv=128, dtype="f32"),
    dict(N=1000, topk=100, dk=5, dv=64, dtype="bf16"),
]


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("shape", SCORE_EDGE, ids=[f"N{e['N']}-k{e['topk']}-dk{e['dk']}-dv{e['dv']}-{e['dtype']}"
                                                   for e in SCORE_EDGE])
def test_score_modes_edges(mode, shape):
    """Every d_v, d_k from 2 to 5, windows longer than the pool, with the
    history-mean candidate and with rows emptied (they attend to it alone)."""
    w = workloads.custom(B=1, H=2, seed=shape["N"] * 11 + shape["dk"], bits=6, **shape)
    log(f"score {mode} edge {shape}")
    x = workloads.generate(w)
    S = w.segments
    f = {n: oracle.as_f32(a, w.dtype).reshape(S, w.N, -1) for n, a in x.items()}
    qc, kc, _, _ = oracle.morton_encode(f["q"], f["k"], 6 if shape["dk"] <= 5 else 4)
    idx = oracle.select_topk(qc, kc, w.topk, True)
    idx[:, ::7] = -1
    q, k, v = (to_dev(x[n], w.dtype) for n in ("q", "k", "v"))
    mk, mv = zeta.zeta_history_mean(k, v, True)
    out = zeta.zeta_topk_attn_fwd(q, k, v, i32_to_dev(idx.reshape(w.B, w.H, w.N, w.topk)), 0.3, score=mode,
                                  mean_k=mk, mean_v=mv)
    plain = zeta.zeta_topk_attn_fwd(q, k, v, i32_to_dev(idx.reshape(w.B, w.H, w.N, w.topk)), 0.3, score=mode)
    torch.cuda.synchronize()
    rk, rv = oracle.history_mean(f["k"], f["v"], True)
    ref = oracle.attend(f["q"], f["k"], f["v"], idx, 0.3, mean_k=rk, mean_v=rv, mode=mode)
    assert np.abs(host(out).reshape(ref.shape) - ref).max() <= TOL[w.dtype]
    keep = ~np.all(idx < 0, axis=-1)
    ref0 = oracle.attend(f["q"], f["k"], f["v"], np.where(keep[..., None], idx, 0), 0.3, mode=mode)
    got0 = host(plain).reshape(ref0.shape)
    assert np.abs(got0[keep] - ref0[keep]).max() <= TOL[w.dtype]
    assert np.all(got0[~keep] == 0.0)


def test_score_modes_long_context():
    """Workload 5, one-pass path with each variant (per-query kernels):
    sampled rows of a few segments."""
    cfg = 5
    w, x, f = inputs(cfg)
    q, k, v = (to_dev(x[n], w.dtype) for n in ("q", "k", "v"))
    rows = sample_rows(w.N, 12, 31)
    for mode in MODES:
        log(f"score {mode} long context")
        res = zeta.forward(q, k, v, w.topk, 0.5, True, w.bits, fused=True, score=mode, return_intermediates=True)
        torch.cuda.synchronize()
        idx = host(res["idx"]).reshape(w.segments, w.N, w.topk)
        out = host(res["out"]).reshape(w.segments, w.N, w.dv)
        for s in (0, 9):
            ref = oracle.attend(f["q"][s:s + 1], f["k"][s:s + 1], f["v"][s:s + 1], idx[s:s + 1, rows], 0.5, rows=rows,
                                mode=mode)[0]
            assert np.abs(out[s, rows] - ref).max() <= TOL[w.dtype], (mode, s)


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("history", [False, True])
def test_score_modes_tiles(mode, history):
    """The bfloat16 one-pass call with d_k = 3 runs every variant on the
    matrix-core tiles (online softmax per query for the softmax variants):
    it matches the oracle, with and without the history-mean candidate, and a
    query's bits do not depend on the processing order (its running maximum
    meets its own chunks in list order whatever tile it is in)."""
    cfg = 2
    w, x, f = inputs(cfg)
    log(f"score {mode} tiles history={history}")
    S = 4
    raw = {n: a.reshape(w.segments, w.N, -1)[:S] for n, a in x.items()}
    fs = {n: a[:S] for n, a in f.items()}
    q, k, v = (to_dev(raw[n][None], w.dtype) for n in ("q", "k", "v"))
    res = zeta.forward(q, k, v, w.topk, 0.5, True, w.bits, fused=True, score=mode, history=history,
                       return_intermediates=True)
    pos = zeta.zeta_select_attend_fwd(q, k, v, res["q_codes"], res["sorted_codes"], res["perm"], w.topk, True, 0.5,
                                      score=mode, mean_k=res["mean_k"], mean_v=res["mean_v"])
    torch.cuda.synchronize()
    assert torch.equal(res["out"].view(torch.int16), pos.view(torch.int16))
    idx = host(res["idx"]).reshape(S, w.N, w.topk)
    out = host(res["out"]).reshape(S, w.N, w.dv)
    mk = mv = None
    if history:
        mk, mv = oracle.history_mean(fs["k"], fs["v"], True)
    ref = oracle.attend(fs["q"], fs["k"], fs["v"], idx, 0.5, mean_k=mk, mean_v=mv, mode=mode)
    assert np.abs(out - ref).max() <= TOL[w.dtype]


@pytest.mark.parametrize("dv", [32, 256])
@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("mode", MODES)
def test_score_modes_tiles_widths(mode, causal, dv):
    """Every variant's tile kernel at the narrowest and widest value rows
    (one product block pair per lane at d_v = 32, sixteen at 256), both
    modes, on a ragged length: the oracle's outputs, and the same bits in
    position order as in level order."""
    w = workloads.custom(B=1, H=2, N=700, dv=dv, topk=40, dtype="bf16", bits=8, seed=dv + len(mode))
    log(f"score {mode} tiles dv={dv} causal={causal}")
    x = workloads.generate(w)
    S = w.segments
    f = {n: oracle.as_f32(a, w.dtype).reshape(S, w.N, -1) for n, a in x.items()}
    q, k, v = (to_dev(x[n], w.dtype) for n in ("q", "k", "v"))
    res = zeta.forward(q, k, v, w.topk, 0.5, causal, w.bits, fused=True, score=mode, return_intermediates=True)
    pos = zeta.zeta_select_attend_fwd(q, k, v, res["q_codes"], res["sorted_codes"], res["perm"], w.topk, causal, 0.5,
                                      score=mode)
    torch.cuda.synchronize()
    assert torch.equal(res["out"].view(torch.int16), pos.view(torch.int16))
    idx = host(res["idx"]).reshape(S, w.N, w.topk)
    qc, kc, _, _ = oracle.morton_encode(f["q"], f["k"], w.bits)
    assert np.array_equal(idx, oracle.select_topk(qc, kc, w.topk, causal))
    ref = oracle.attend(f["q"], f["k"], f["v"], idx, 0.5, mode=mode)
    out = host(res["out"]).reshape(S, w.N, w.dv)
    assert np.abs(out - ref).max() <= TOL[w.dtype], (mode, causal, dv)


@pytest.mark.parametrize("mode", MODES)
def test_score_modes_tiles_chunked(mode):
    """Score variants on the tiles under the chunked causal rule (the first
    chunk's queries have empty pools and give zero rows), with and without
    the history-mean candidate: the oracle's outputs, and the same bits in
    position order as in level order."""
    w = workloads.custom(B=1, H=2, N=1000, dv=64, topk=32, dtype="bf16", bits=8, seed=41 + len(mode))
    M = 125
    x = workloads.generate(w)
    S = w.segments
    f = {n: oracle.as_f32(a, w.dtype).reshape(S, w.N, -1) for n, a in x.items()}
    q, k, v = (to_dev(x[n], w.dtype) for n in ("q", "k", "v"))
    qc, kc, _, _ = oracle.morton_encode(f["q"], f["k"], w.bits)
    want = oracle.select_topk(qc, kc, w.topk, True, chunk=M)
    for history in (False, True):
        log(f"score {mode} tiles chunk={M} history={history}")
        res = zeta.forward(q, k, v, w.topk, 0.5, True, w.bits, fused=True, score=mode, chunk=M, history=history,
                           return_intermediates=True)
        pos = zeta.zeta_select_attend_fwd(q, k, v, res["q_codes"], res["sorted_codes"], res["perm"], w.topk, True,
                                          0.5, score=mode, chunk=M, mean_k=res["mean_k"], mean_v=res["mean_v"])
        torch.cuda.synchronize()
        assert torch.equal(res["out"].view(torch.int16), pos.view(torch.int16))
        idx = host(res["idx"]).reshape(S, w.N, w.topk)
        assert np.array_equal(idx, want)
        mk = mv = None
        if history:
            mk, mv = oracle.history_mean(f["k"], f["v"], True)
        ref = oracle.attend(f["q"], f["k"], f["v"], idx, 0.5, mean_k=mk, mean_v=mv, mode=mode)
        out = host(res["out"]).reshape(S, w.N, w.dv)
        assert np.abs(out - ref).max() <= TOL[w.dtype], (mode, history)
