"""GPU parity: every C ABI call against the CPU oracle on the same seeded inputs.

Codes, permutations and selected indices must be bit-exact; outputs must be
within max-abs 1e-4 (float32) or 2e-2 (bfloat16) of the float64 oracle.
Calls go through the Python binding, i.e. straight into libzeta.so.
"""

import numpy as np
import pytest
import torch

import oracle
import paper_2501_14577_amd as zeta
import workloads
from gpu_util import (TOL, device, host, i32_to_dev, inputs, log, oracle_codes, oracle_select, sample_rows,
                      to_dev, u32_to_dev)

pytestmark = pytest.mark.gpu

CONFIGS = sorted(workloads.CONFIGS)


@pytest.fixture(scope="module", autouse=True)
def _lib():
    device()
    zeta.load_library()


# ----------------------------------------------------------------------------
# Encode
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("cfg", CONFIGS)
def test_encode_config(cfg):
    w, x, f = inputs(cfg)
    log(f"encode config {cfg} {w.name}")
    oc = oracle_codes(cfg)
    q, k = to_dev(x["q"], w.dtype), to_dev(x["k"], w.dtype)
    rng_out = torch.empty((w.segments, 2, w.dk), dtype=torch.float32, device=device())
    qc, kc = zeta.zeta_morton_encode(q, k, w.bits, range_out=rng_out)
    torch.cuda.synchronize()
    S = w.segments
    assert np.array_equal(host(qc).reshape(S, w.N), oc["q_codes"])
    assert np.array_equal(host(kc).reshape(S, w.N), oc["k_codes"])
    r = host(rng_out)
    assert np.array_equal(r[:, 0], oc["lo"]) and np.array_equal(r[:, 1], oc["hi"])


def _edge_values(lo, hi, bits):
    """Values at, and 1-2 ulps either side of, every grid edge of [lo, hi]."""
    top = (1 << bits) - 1
    edges = lo + (hi - lo) * np.arange(top + 1, dtype=np.float64) / top
    vals = [edges.astype(np.float32)]
    for step in (1, 2):
        up, dn = vals[0].copy(), vals[0].copy()
        for _ in range(step):
            up = np.nextafter(up, np.float32(np.inf))
            dn = np.nextafter(dn, np.float32(-np.inf))
        vals += [up, dn]
    return np.concatenate(vals).astype(np.float32)


@pytest.mark.parametrize("pad8", [False, True])
@pytest.mark.parametrize("bits,lo,hi", [(10, -1.7, 2.3), (6, -3.1, 0.9), (10, 0.1, 0.30000001), (2, -1.0, 1.0)])
def test_encode_bucket_edges(bits, lo, hi, pad8):
    """pad8: a length that is a multiple of 8 (the vector form of the d_k = 3
    kernels), else a ragged one (the row-per-thread form)."""
    log(f"encode edges bits={bits} lo={lo} hi={hi} pad8={pad8}")
    vals = _edge_values(lo, hi, bits)
    vals = np.concatenate([vals, np.float32([lo - 1, hi + 1])])  # outside the range: clamps
    if pad8 != (len(vals) % 8 == 0):
        extra = (-len(vals)) % 8 if pad8 else 1
        vals = np.concatenate([vals, np.linspace(lo, hi, extra + 2, dtype=np.float32)[1:extra + 1]])
    n = len(vals)
    rng = np.random.default_rng(bits)
    q = np.stack([vals, rng.permutation(vals), rng.permutation(vals)], axis=-1)[None].astype(np.float32)
    k = np.stack([rng.permutation(vals), vals, rng.permutation(vals)], axis=-1)[None].astype(np.float32)
    lohi = np.array([[[lo] * 3, [hi] * 3]], dtype=np.float32)
    eq, ek, _, _ = oracle.morton_encode(q, k, bits, (lohi[:, 0], lohi[:, 1]))
    qc, kc = zeta.zeta_morton_encode(to_dev(q.reshape(1, 1, n, 3), "f32"), to_dev(k.reshape(1, 1, n, 3), "f32"),
                                     bits, range_lohi=torch.from_numpy(lohi).to(device()))
    torch.cuda.synchronize()
    assert np.array_equal(host(qc).reshape(1, n), eq)
    assert np.array_equal(host(kc).reshape(1, n), ek)


@pytest.mark.parametrize("dk,bits,dtype", [(1, 20, "f32"), (2, 16, "bf16"), (3, 10, "f32"), (3, 7, "bf16"),
                                           (4, 8, "f32"), (5, 6, "bf16"), (8, 4, "f32")])
@pytest.mark.parametrize("N", [5001, 5008])
def test_encode_shapes(dk, bits, dtype, N):
    log(f"encode dk={dk} bits={bits} {dtype} N={N}")
    w = workloads.custom(B=2, H=3, N=N, dk=dk, dtype=dtype, bits=bits, seed=dk * 100 + bits)
    x = workloads.generate(w, with_v=False)
    S = w.segments
    qf = oracle.as_f32(x["q"], dtype).reshape(S, w.N, dk)
    kf = oracle.as_f32(x["k"], dtype).reshape(S, w.N, dk)
    eq, ek, _, _ = oracle.morton_encode(qf, kf, bits)
    qc, kc = zeta.zeta_morton_encode(to_dev(x["q"], dtype), to_dev(x["k"], dtype), bits)
    torch.cuda.synchronize()
    assert np.array_equal(host(qc).reshape(S, w.N), eq)
    assert np.array_equal(host(kc).reshape(S, w.N), ek)


def test_encode_constant_inputs():
    """hi == lo on every axis: every code is 0."""
    q = np.full((1, 2, 77, 3), 0.25, dtype=np.float32)
    qc, kc = zeta.zeta_morton_encode(to_dev(q, "f32"), to_dev(q.copy(), "f32"), 10)
    torch.cuda.synchronize()
    assert not host(qc).any() and not host(kc).any()


# ----------------------------------------------------------------------------
# Sort
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("cfg", CONFIGS)
def test_sort_config(cfg):
    w, _, _ = inputs(cfg)
    log(f"sort config {cfg} {w.name}")
    oc = oracle_codes(cfg)
    sc, perm = zeta.zeta_sort_keys(u32_to_dev(oc["k_codes"]), w.code_bits)
    torch.cuda.synchronize()
    assert np.array_equal(host(perm), oc["perm"])
    assert np.array_equal(host(sc), oc["sorted_codes"])


@pytest.mark.parametrize("S,N,code_bits", [(1, 1, 30), (3, 63, 2), (2, 4095, 7), (2, 4096, 18), (2, 4097, 1),
                                            (3, 10000, 32), (1, 70001, 18), (5, 12289, 9), (1, 8192, 16),
                                            (1, 131072, 18), (2, 135169, 12), (1, 300001, 27)])
def test_sort_shapes(S, N, code_bits):
    """Ragged tails, one to three passes, and segments of up to 32 tiles of
    4096 keys (the scatter sums the earlier tiles' counts itself) or more
    (a scan kernel does)."""
    log(f"sort S={S} N={N} bits={code_bits}")
    kc = workloads.random_codes(S * 1000 + N + code_bits, (S, N), code_bits)
    esc, eperm = oracle.sort_keys(kc)
    sc, perm = zeta.zeta_sort_keys(u32_to_dev(kc), code_bits)
    torch.cuda.synchronize()
    assert np.array_equal(host(perm), eperm)
    assert np.array_equal(host(sc), esc)


@pytest.mark.parametrize("S,N,code_bits,high_values", [(2, 20000, 18, 4), (1, 9000, 18, 1), (3, 4097, 16, 2)])
def test_sort_clustered(S, N, code_bits, high_values):
    """Codes whose high digit takes only a few values (one value: every key
    shares it): heavily repeated digits in every tile of both passes, and
    long runs of equal high digit with the low digit deciding the order."""
    log(f"sort clustered S={S} N={N} bits={code_bits} high values={high_values}")
    low = (code_bits + 1) // 2
    rng = np.random.default_rng([S, N, code_bits, high_values])
    hi = rng.integers(0, high_values, size=(S, N), dtype=np.uint64) << np.uint64(low)
    lo = rng.integers(0, 1 << low, size=(S, N), dtype=np.uint64)
    kc = (hi | lo).astype(np.uint32)
    esc, eperm = oracle.sort_keys(kc)
    sc, perm = zeta.zeta_sort_keys(u32_to_dev(kc), code_bits)
    torch.cuda.synchronize()
    assert np.array_equal(host(perm), eperm)
    assert np.array_equal(host(sc), esc)


# ----------------------------------------------------------------------------
# Select
# ----------------------------------------------------------------------------

def _gpu_select(oc, topk, causal):
    return host(zeta.zeta_select_topk(u32_to_dev(oc["q_codes"]), u32_to_dev(oc["sorted_codes"]),
                                      i32_to_dev(oc["perm"]), topk, causal))


SELECT_FULL = [(c, causal) for c in (1, 2, 3, 4) for causal in workloads.CONFIGS[c].causal]


@pytest.mark.parametrize("cfg,causal", SELECT_FULL)
def test_select_config(cfg, causal):
    w, _, _ = inputs(cfg)
    log(f"select config {cfg} causal={causal}")
    got = _gpu_select(oracle_codes(cfg), w.topk, causal)
    expect = oracle_select(cfg, causal)
    assert np.array_equal(got, expect)


def _check_rows_valid(idx, kc, causal):
    """Properties of every row at any size: count, causality, -1 tail, and
    strictly increasing (code, position) order (hence distinct)."""
    S, N, k = idx.shape
    valid = idx >= 0
    cnt = valid.sum(-1)
    pool = (np.arange(N) + 1) if causal else np.full(N, N)
    assert np.array_equal(cnt, np.broadcast_to(np.minimum(k, pool), (S, N)))
    assert np.array_equal(valid, np.arange(k)[None, None, :] < cnt[..., None])
    if causal:
        assert np.all(np.where(valid, idx, 0) <= np.arange(N)[None, :, None])
    assert np.all(idx < N)
    codes = np.take_along_axis(kc.astype(np.int64), np.where(valid, idx, 0).reshape(S, -1), axis=1)
    key = codes.reshape(S, N, k) * (1 << 32) + idx
    both = valid[..., 1:]
    assert np.all(np.diff(key, axis=-1)[both] > 0)


def test_select_long_context_sampled():
    cfg = 5
    w, _, _ = inputs(cfg)
    oc = oracle_codes(cfg)
    log("select config 5: all rows by property, sampled rows exactly")
    got = _gpu_select(oc, w.topk, True)
    _check_rows_valid(got, oc["k_codes"], True)
    rows = sample_rows(w.N, 24, 5)
    for s in range(w.segments):
        for i in rows:
            expect = oracle.select_one(int(oc["q_codes"][s, i]), oc["k_codes"][s], int(i), w.topk, True)
            assert np.array_equal(got[s, i], expect), (s, i)


@pytest.mark.parametrize("N,topk,code_bits", [(1, 1, 6), (1, 8, 30), (2, 1, 2), (5, 3, 2), (100, 7, 3),
                                              (129, 64, 4), (300, 2, 30), (1000, 33, 3), (4097, 64, 6),
                                              (5000, 1024, 9), (3000, 1000, 2), (20000, 16, 12), (9000, 5, 1),
                                              (65536, 16, 12), (70001, 40, 6)])
@pytest.mark.parametrize("causal", [True, False])
def test_select_shapes(N, topk, code_bits, causal):
    """Every row against the oracle (sampled rows past 4 M index slots).  The
    window search tests positions as 16-bit values up to N = 65536 (the
    largest position and pool limit 65535 included) and as 32-bit values
    beyond."""
    log(f"select N={N} k={topk} bits={code_bits} causal={causal}")
    S = 2
    kc = workloads.random_codes(N * 7 + topk, (S, N), code_bits)
    qc = workloads.random_codes(N * 7 + topk + 1, (S, N), code_bits)
    sc, perm = oracle.sort_keys(kc)
    got = _gpu_select(dict(q_codes=qc, sorted_codes=sc, perm=perm), topk, causal)
    if N * topk <= 4_000_000:
        assert np.array_equal(got, oracle.select_topk(qc, kc, topk, causal))
    else:
        _check_rows_valid(got, kc, causal)
        for s in range(S):
            for i in sample_rows(N, 16, N):
                assert np.array_equal(got[s, i], oracle.select_one(int(qc[s, i]), kc[s], int(i), topk, causal))


# ----------------------------------------------------------------------------
# Attend
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("cfg,causal", SELECT_FULL)
def test_attend_config(cfg, causal):
    w, x, f = inputs(cfg)
    log(f"attend config {cfg} causal={causal}")
    idx = oracle_select(cfg, causal)
    out = zeta.zeta_topk_attn_fwd(to_dev(x["q"], w.dtype), to_dev(x["k"], w.dtype), to_dev(x["v"], w.dtype),
                                  i32_to_dev(idx.reshape(w.B, w.H, w.N, w.topk)), workloads.EPS_DEFAULT)
    got = host(out).reshape(w.segments, w.N, w.dv)
    segs = range(w.segments) if w.segments * w.N <= 300_000 else range(0, w.segments, 8)
    for s in segs:
        ref = oracle.attend(f["q"][s:s + 1], f["k"][s:s + 1], f["v"][s:s + 1], idx[s:s + 1], workloads.EPS_DEFAULT)
        err = np.abs(got[s] - ref[0]).max()
        assert err <= TOL[w.dtype], (s, err)


@pytest.mark.parametrize("dv", [32, 64, 128, 256])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("dk", [3, 1, 8])
def test_attend_shapes(dv, dtype, dk):
    log(f"attend dv={dv} {dtype} dk={dk}")
    w = workloads.custom(B=1, H=2, N=700, dk=dk, dv=dv, topk=45, dtype=dtype, seed=dv + dk)
    x = workloads.generate(w)
    S = w.segments
    f = {n: oracle.as_f32(a, dtype).reshape(S, w.N, -1) for n, a in x.items()}
    kc = workloads.random_codes(dv, (S, w.N), 8)
    idx = oracle.select_topk(workloads.random_codes(dv + 1, (S, w.N), 8), kc, w.topk, True)
    out = zeta.zeta_topk_attn_fwd(to_dev(x["q"], dtype), to_dev(x["k"], dtype), to_dev(x["v"], dtype),
                                  i32_to_dev(idx.reshape(1, 2, w.N, w.topk)), 0.37)
    ref = oracle.attend(f["q"], f["k"], f["v"], idx, 0.37)
    err = np.abs(host(out).reshape(S, w.N, dv) - ref).max()
    assert err <= TOL[dtype], err


def test_attend_empty_row_is_zero():
    """A row with no valid candidate is written as zeros (library contract)."""
    q = np.random.default_rng(0).standard_normal((1, 1, 4, 3)).astype(np.float32)
    v = np.random.default_rng(1).standard_normal((1, 1, 4, 64)).astype(np.float32)
    idx = np.array([[[[0, -1], [-1, -1], [1, 0], [3, -1]]]], dtype=np.int32)
    out = host(zeta.zeta_topk_attn_fwd(to_dev(q, "f32"), to_dev(q, "f32"), to_dev(v, "f32"), i32_to_dev(idx), 0.5))
    assert np.all(out[0, 0, 1] == 0)
    assert np.allclose(out[0, 0, 0], v[0, 0, 0], atol=1e-6)
    assert np.allclose(out[0, 0, 3], v[0, 0, 3], atol=1e-6)


# ----------------------------------------------------------------------------
# Whole forward
# ----------------------------------------------------------------------------

FORWARD = [(c, causal) for c in CONFIGS for causal in workloads.CONFIGS[c].causal]


@pytest.mark.parametrize("cfg,causal", FORWARD)
def test_forward_config(cfg, causal):
    """The four calls chained on one stream, every intermediate checked."""
    w, x, f = inputs(cfg)
    log(f"forward config {cfg} {w.name} causal={causal}")
    oc = oracle_codes(cfg)
    res = zeta.forward(to_dev(x["q"], w.dtype), to_dev(x["k"], w.dtype), to_dev(x["v"], w.dtype), w.topk,
                       workloads.EPS_DEFAULT, causal, w.bits, return_intermediates=True)
    torch.cuda.synchronize()
    S = w.segments
    assert np.array_equal(host(res["q_codes"]).reshape(S, w.N), oc["q_codes"])
    assert np.array_equal(host(res["k_codes"]).reshape(S, w.N), oc["k_codes"])
    assert np.array_equal(host(res["perm"]).reshape(S, w.N), oc["perm"])
    idx = host(res["idx"]).reshape(S, w.N, w.topk)
    out = host(res["out"]).reshape(S, w.N, w.dv)
    if cfg != 5:
        assert np.array_equal(idx, oracle_select(cfg, causal))
        segs = range(S) if S * w.N <= 300_000 else range(0, S, 12)
        for s in segs:
            ref = oracle.attend(f["q"][s:s + 1], f["k"][s:s + 1], f["v"][s:s + 1], idx[s:s + 1],
                                workloads.EPS_DEFAULT)
            assert np.abs(out[s] - ref[0]).max() <= TOL[w.dtype], s
    else:
        rows = sample_rows(w.N, 16, 55)
        for s in range(S):
            sel = np.stack([oracle.select_one(int(oc["q_codes"][s, i]), oc["k_codes"][s], int(i), w.topk, True)
                            for i in rows])
            assert np.array_equal(idx[s, rows], sel), s
            ref = oracle.attend(f["q"][s:s + 1], f["k"][s:s + 1], f["v"][s:s + 1], sel[None],
                                workloads.EPS_DEFAULT, rows=rows)
            assert np.abs(out[s, rows] - ref[0]).max() <= TOL[w.dtype], s


EDGE = [
    dict(N=1, topk=8, dk=3, dv=64, dtype="f32", bits=10),
    dict(N=5, topk=8, dk=3, dv=64, dtype="bf16", bits=10),
    dict(N=37, topk=7, dk=3, dv=32, dtype="f32", bits=2),
    dict(N=4097, topk=1, dk=3, dv=128, dtype="bf16", bits=6),
    dict(N=1500, topk=33, dk=2, dv=256, dtype="f32", bits=16),
    dict(N=2049, topk=64, dk=4, dv=64, dtype="bf16", bits=8),
    dict(N=600, topk=1024, dk=3, dv=128, dtype="f32", bits=10),
    dict(N=300, topk=16, dk=3, dv=32, dtype="bf16", bits=10),
    dict(N=1000, topk=100, dk=5, dv=256, dtype="bf16", bits=5),
    dict(N=700, topk=1024, dk=3, dv=128, dtype="bf16", bits=10),
    dict(N=900, topk=48, dk=3, dv=256, dtype="bf16", bits=7),
    # The window search's 16-bit positions at their largest N, then 32-bit.
    dict(N=65536, topk=16, dk=3, dv=32, dtype="bf16", bits=6),
    dict(N=70001, topk=16, dk=3, dv=32, dtype="bf16", bits=6),
]


@pytest.mark.parametrize("shape", EDGE, ids=[f"N{e['N']}-k{e['topk']}-dk{e['dk']}" for e in EDGE])
@pytest.mark.parametrize("causal", [True, False])
def test_forward_edges(shape, causal):
    w = workloads.custom(B=2, H=1, seed=shape["N"] + shape["topk"], **shape)
    log(f"forward edge {shape} causal={causal}")
    x = workloads.generate(w)
    S = w.segments
    f = {n: oracle.as_f32(a, w.dtype).reshape(S, w.N, -1) for n, a in x.items()}
    ref = oracle.forward(f["q"], f["k"], f["v"], w.topk, 0.5, causal, w.bits)
    res = zeta.forward(to_dev(x["q"], w.dtype), to_dev(x["k"], w.dtype), to_dev(x["v"], w.dtype), w.topk, 0.5,
                       causal, w.bits, return_intermediates=True)
    torch.cuda.synchronize()
    assert np.array_equal(host(res["k_codes"]).reshape(S, w.N), ref["k_codes"])
    assert np.array_equal(host(res["idx"]).reshape(S, w.N, w.topk), ref["idx"])
    assert np.abs(host(res["out"]).reshape(S, w.N, w.dv) - ref["out"]).max() <= TOL[w.dtype]


def test_forward_deterministic_and_complete():
    """Two runs into buffers poisoned with different sentinels agree bit for
    bit: every output element is written and nothing depends on timing."""
    cfg = 2
    w, x, _ = inputs(cfg)
    log("determinism config 2")
    q, k, v = (to_dev(x[n], w.dtype) for n in ("q", "k", "v"))
    runs = []
    for fill in (0x7F, 0x00):
        b = zeta.alloc_buffers(w.B, w.H, w.N, w.dv, w.topk, torch.bfloat16, device())
        for t in b.values():
            t.view(torch.uint8).fill_(fill)
        zeta.forward(q, k, v, w.topk, workloads.EPS_DEFAULT, True, w.bits, buffers=b)
        torch.cuda.synchronize()
        runs.append({n: t.view(torch.uint8).cpu().numpy() for n, t in b.items()})
    for n in runs[0]:
        assert np.array_equal(runs[0][n], runs[1][n]), n


# ----------------------------------------------------------------------------
# Processing order
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("causal", [True, False])
def test_processing_order_changes_nothing(causal):
    """select gives bit-identical results in position order, in the queries'
    Z-order and in a random order; entries outside 0..N-1 are skipped.  The
    bfloat16 attend call shares each 16 queries' rows when given an order:
    its outputs agree with the per-query ones to float32 rounding (one
    bfloat16 unit in the last place)."""
    cfg = 2
    w, x, _ = inputs(cfg)
    log(f"processing order config {cfg} causal={causal}")
    oc = oracle_codes(cfg)
    q, k, v = (to_dev(x[n], w.dtype) for n in ("q", "k", "v"))
    qc, sc, perm = u32_to_dev(oc["q_codes"]), u32_to_dev(oc["sorted_codes"]), i32_to_dev(oc["perm"])
    S = w.segments
    zorder = i32_to_dev(np.argsort(oc["q_codes"], axis=1, kind="stable"))
    rng = np.random.default_rng(9)
    shuffled = i32_to_dev(np.stack([rng.permutation(w.N) for _ in range(S)]))
    idx0 = zeta.zeta_select_topk(qc, sc, perm, w.topk, causal)
    out0 = zeta.zeta_topk_attn_fwd(q, k, v, idx0.reshape(w.B, w.H, w.N, w.topk), 0.5)
    for order in (zorder, shuffled):
        idx1 = zeta.zeta_select_topk(qc, sc, perm, w.topk, causal, q_order=order)
        out1 = zeta.zeta_topk_attn_fwd(q, k, v, idx0.reshape(w.B, w.H, w.N, w.topk), 0.5, q_order=order)
        torch.cuda.synchronize()
        torch.cuda.synchronize()
        assert torch.equal(idx0, idx1)
        a, b = host(out0).astype(np.float64), host(out1).astype(np.float64)
        assert np.all(np.abs(a - b) <= 2.0 ** -7 * np.maximum(np.abs(a), np.abs(b)) + 1e-5)
    # A partial order: rows whose slot holds an out-of-range entry stay untouched.
    part = np.argsort(oc["q_codes"], axis=1, kind="stable").astype(np.int32)
    part[:, ::3] = -1
    idx2 = torch.full_like(idx0, -7)
    zeta.zeta_select_topk(qc, sc, perm, w.topk, causal, q_order=i32_to_dev(part), idx=idx2)
    torch.cuda.synchronize()
    got, ref = host(idx2), host(idx0)
    done = np.zeros((S, w.N), dtype=bool)
    seg_ix, slot_ix = np.nonzero(part >= 0)
    done[seg_ix, part[seg_ix, slot_ix]] = True
    assert np.array_equal(got[done], ref[done])
    assert np.all(got[~done] == -7)


def test_forward_zorder_matches_position_order():
    cfg = 4
    w, x, _ = inputs(cfg)
    log("forward z-order vs position order, config 4")
    q, k, v = (to_dev(x[n], w.dtype) for n in ("q", "k", "v"))
    a = zeta.forward(q, k, v, w.topk, 0.5, True, w.bits, zorder=True, return_intermediates=True)
    b = zeta.forward(q, k, v, w.topk, 0.5, True, w.bits, zorder=False, return_intermediates=True)
    torch.cuda.synchronize()
    assert torch.equal(a["idx"], b["idx"])
    # The four calls: with the Z-order the attend call runs on shared tiles
    # (float32 rounding apart, one bfloat16 unit in the last place).
    oa, ob = host(a["out"]).astype(np.float64), host(b["out"]).astype(np.float64)
    assert np.all(np.abs(oa - ob) <= 2.0 ** -7 * np.maximum(np.abs(oa), np.abs(ob)) + 1e-5)
    c = zeta.forward(q, k, v, w.topk, 0.5, True, w.bits, zorder=True, fused=True)
    d = zeta.forward(q, k, v, w.topk, 0.5, True, w.bits, zorder=False, fused=True)
    torch.cuda.synchronize()
    assert torch.equal(c.view(torch.int16), d.view(torch.int16))


# ----------------------------------------------------------------------------
# Query order by list level
# ----------------------------------------------------------------------------

def _expected_level_order(z, N, topk, causal, chunk=0):
    """Regroup a per-segment order by the level of the list each query's
    pool is searched in: the largest pool position is i, or
    floor(i / chunk) * chunk - 1 under the chunked rule (an empty pool counts
    as the first level)."""
    t0 = max(0, (topk - 1).bit_length())
    t_hi = (N - 1).bit_length() - 1
    if not causal or t0 > t_hi:
        return z

    def level(i):
        lim = (i // chunk) * chunk - 1 if chunk else i
        return t0 if lim < 0 else min(max(t0, lim.bit_length()), t_hi + 1)

    lvl = np.array([level(i) for i in range(N)])
    return np.stack([zs[np.argsort(lvl[zs], kind="stable")] for zs in z])


@pytest.mark.parametrize("N,topk,causal,chunk", [(65536, 128, True, 0), (5000, 64, True, 0), (300, 1024, True, 0),
                                                 (777, 8, False, 0), (1, 1, True, 0), (4097, 1, True, 0),
                                                 (65536, 128, True, 2048), (5000, 64, True, 313), (300, 16, True, 1)])
def test_query_order(N, topk, causal, chunk):
    log(f"query order N={N} k={topk} causal={causal} chunk={chunk}")
    S = 3
    rng = np.random.default_rng(N + topk)
    z = np.stack([rng.permutation(N) for _ in range(S)]).astype(np.int32)
    got = host(zeta.zeta_query_order(i32_to_dev(z), N, S, topk, causal, chunk=chunk))
    assert np.array_equal(got, _expected_level_order(z, N, topk, causal, chunk))
    pos = host(zeta.zeta_query_order(None, N, S, topk, causal, chunk=chunk, device=device()))
    want = _expected_level_order(np.tile(np.arange(N, dtype=np.int32), (S, 1)), N, topk, causal, chunk)
    assert np.array_equal(pos, want)



# ----------------------------------------------------------------------------
# Select and attend in one pass
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("cfg,causal", FORWARD)
def test_select_attend_matches_two_calls(cfg, causal):
    """The one-pass call selects the two calls' windows.  float32 outputs are
    the two calls' bits; bfloat16 outputs (matrix-core products) are checked
    against the oracle's attention over those windows and against the two
    calls' output."""
    w, x, f = inputs(cfg)
    log(f"select+attend config {cfg} causal={causal}")
    q, k, v = (to_dev(x[n], w.dtype) for n in ("q", "k", "v"))
    two = zeta.forward(q, k, v, w.topk, 0.5, causal, w.bits, return_intermediates=True)
    one = zeta.forward(q, k, v, w.topk, 0.5, causal, w.bits, fused=True, return_intermediates=True)
    torch.cuda.synchronize()
    assert torch.equal(two["idx"], one["idx"])
    S = w.segments
    if w.dtype == "f32":
        assert torch.equal(two["out"].view(torch.int32), one["out"].view(torch.int32))
    else:
        out1, out2 = host(one["out"]).reshape(S, w.N, w.dv), host(two["out"]).reshape(S, w.N, w.dv)
        assert np.abs(out1 - out2).max() <= TOL[w.dtype]
        idx = host(one["idx"]).reshape(S, w.N, w.topk)
        rows = sample_rows(w.N, 64, 77) if w.N > 4096 else None
        for s in range(0, S, max(1, S // 8)):
            ref = oracle.attend(f["q"][s:s + 1], f["k"][s:s + 1], f["v"][s:s + 1],
                                (idx[s:s + 1, rows] if rows is not None else idx[s:s + 1]), 0.5, rows=rows)
            got = out1[s, rows] if rows is not None else out1[s]
            assert np.abs(got - ref[0]).max() <= TOL[w.dtype], s
    if cfg == 1:
        ref = oracle.forward(f["q"], f["k"], f["v"], w.topk, 0.5, causal, w.bits)
        assert np.array_equal(host(one["idx"]).reshape(w.segments, w.N, w.topk), ref["idx"])
        assert np.abs(host(one["out"]).reshape(w.segments, w.N, w.dv) - ref["out"]).max() <= TOL[w.dtype]


@pytest.mark.parametrize("cfg,causal", [(2, True), (3, False), (4, True)])
def test_select_attend_processing_order_changes_nothing(cfg, causal):
    """A query's one-pass result depends only on its own window: position
    order, Z-order, the level-regrouped Z-order and a random order give the
    same output bits."""
    w, x, _ = inputs(cfg)
    log(f"select+attend processing order config {cfg} causal={causal}")
    oc = oracle_codes(cfg)
    q, k, v = (to_dev(x[n], w.dtype) for n in ("q", "k", "v"))
    qc, sc, perm = u32_to_dev(oc["q_codes"]), u32_to_dev(oc["sorted_codes"]), i32_to_dev(oc["perm"])
    S = w.segments
    z = np.argsort(oc["q_codes"], axis=1, kind="stable").astype(np.int32)
    rng = np.random.default_rng(11)
    orders = [None, i32_to_dev(z), zeta.zeta_query_order(i32_to_dev(z), w.N, S, w.topk, causal),
              i32_to_dev(np.stack([rng.permutation(w.N) for _ in range(S)]))]
    outs = [zeta.zeta_select_attend_fwd(q, k, v, qc, sc, perm, w.topk, causal, 0.5, q_order=o) for o in orders]
    torch.cuda.synchronize()
    for o in outs[1:]:
        assert torch.equal(outs[0].view(torch.int16), o.view(torch.int16))


@pytest.mark.parametrize("shape", EDGE, ids=[f"N{e['N']}-k{e['topk']}-dk{e['dk']}" for e in EDGE])
@pytest.mark.parametrize("causal", [True, False])
def test_select_attend_edges(shape, causal):
    w = workloads.custom(B=2, H=1, seed=shape["N"] + shape["topk"], **shape)
    log(f"select+attend edge {shape} causal={causal}")
    x = workloads.generate(w)
    S = w.segments
    f = {n: oracle.as_f32(a, w.dtype).reshape(S, w.N, -1) for n, a in x.items()}
    ref = oracle.forward(f["q"], f["k"], f["v"], w.topk, 0.5, causal, w.bits)
    res = zeta.forward(to_dev(x["q"], w.dtype), to_dev(x["k"], w.dtype), to_dev(x["v"], w.dtype), w.topk, 0.5,
                       causal, w.bits, fused=True, return_intermediates=True)
    torch.cuda.synchronize()
    assert np.array_equal(host(res["idx"]).reshape(S, w.N, w.topk), ref["idx"])
    assert np.abs(host(res["out"]).reshape(S, w.N, w.dv) - ref["out"]).max() <= TOL[w.dtype]
    # Without the index output the result is the same.
    out2 = zeta.forward(to_dev(x["q"], w.dtype), to_dev(x["k"], w.dtype), to_dev(x["v"], w.dtype), w.topk, 0.5,
                        causal, w.bits, fused=True)
    torch.cuda.synchronize()
    assert np.array_equal(host(out2).reshape(S, w.N, w.dv), host(res["out"]).reshape(S, w.N, w.dv))
