"""Pins that tie the CPU oracle to what the paper and mathematics fix.

Each ``check_*`` function takes the oracle module (so a test can hand it a
deliberately broken copy) and raises AssertionError when the oracle departs
from a value or property that does not depend on the oracle itself:
hand-worked values (``tests/golden/``), closed forms, invariants, special
cases and brute force on tiny inputs.
"""

from __future__ import annotations

import itertools
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rows(name):
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                yield line.split()


# ----------------------------------------------------------------------------
# Input conversion: bfloat16 inputs read as the float32 values of their bits
# ----------------------------------------------------------------------------

def check_bf16_input(orc):
    """Fixed bfloat16 bit patterns give their hand-worked values
    (``tests/golden/bf16_values.txt``: normals, subnormals, the largest
    finite value, signed zeros, infinities), through ``bf16_bits_to_f32``
    and through ``as_f32(..., "bf16")`` on a multi-dimensional array; and
    float32 values exact in bfloat16 survive the round trip through the
    workload generator's rounding."""
    import workloads

    rows = list(_rows("bf16_values.txt"))
    bits = np.array([int(b, 16) for b, _ in rows], dtype=np.uint16)
    want = np.array([float(v) if "inf" in v else float.fromhex(v) for _, v in rows], dtype=np.float64)
    for got in (orc.bf16_bits_to_f32(bits), orc.as_f32(bits.reshape(2, -1), "bf16").reshape(-1)):
        assert got.dtype == np.float32
        assert np.array_equal(got.astype(np.float64), want), (got, want)
        assert np.array_equal(np.signbit(got), np.signbit(want))
    # Every finite bfloat16 value, rebuilt from its fields, round-trips.
    rng = np.random.default_rng(5)
    sign = rng.integers(0, 2, 4000)
    expo = rng.integers(1, 255, 4000)
    frac = rng.integers(0, 128, 4000)
    vals = np.where(sign == 1, -1.0, 1.0) * np.ldexp(1.0 + frac / 128.0, expo - 127)
    vals = vals.astype(np.float32)
    b = workloads.f32_to_bf16_bits(vals)
    assert np.array_equal(b.astype(np.int64), (sign << 15) | (expo << 7) | frac)
    assert np.array_equal(orc.as_f32(b, "bf16"), vals)


# ----------------------------------------------------------------------------
# Encode: equation Z and the discretisation (Section 3.1)
# ----------------------------------------------------------------------------

def check_morton_golden(orc):
    """Hand-worked Z-values of equation Z."""
    for bits, c0, c1, c2, code in _rows("morton_codes.txt"):
        bits = int(bits)
        got = int(orc.interleave(np.array([[int(c0), int(c1), int(c2)]], dtype=np.uint32), bits)[0])
        assert got == int(code, 16), (bits, c0, c1, c2, hex(got), code)


def check_morton_bijection(orc):
    """At b bits and d axes the full grid maps one-to-one onto [0, 2^(d b))."""
    for d, bits in ((3, 2), (2, 3), (1, 5), (4, 2)):
        grid = np.array(list(itertools.product(range(1 << bits), repeat=d)), dtype=np.uint32)
        z = orc.interleave(grid, bits).astype(np.int64)
        assert sorted(z.tolist()) == list(range(1 << (d * bits))), (d, bits)


def check_morton_axis_order(orc):
    """Incrementing the top bit of axis 0 outweighs every bit of the later axes,
    and raising any one coordinate raises Z (monotone per axis)."""
    rng = np.random.default_rng(11)
    bits = 4
    pts = rng.integers(0, 1 << bits, size=(500, 3)).astype(np.uint32)
    z = orc.interleave(pts, bits).astype(np.int64)
    for a in range(3):
        up = pts.copy()
        ok = up[:, a] < (1 << bits) - 1
        up[ok, a] += 1
        z2 = orc.interleave(up, bits).astype(np.int64)
        assert np.all(z2[ok] > z[ok]), a
    hi0 = np.array([[1 << (bits - 1), 0, 0]], dtype=np.uint32)
    rest = np.array([[(1 << (bits - 1)) - 1, (1 << bits) - 1, (1 << bits) - 1]], dtype=np.uint32)
    assert int(orc.interleave(hi0, bits)[0]) > int(orc.interleave(rest, bits)[0])


def check_quantise_golden(orc):
    """Hand-worked grid coordinates of the discretisation formula."""
    for bits, lo, hi, x, code in _rows("quantise.txt"):
        got = int(orc.quantise(np.float32(x), np.float32(lo), np.float32(hi), int(bits)))
        assert got == int(code), (bits, lo, hi, x, got, code)


def check_quantise_buckets(orc):
    """On an exactly representable grid (lo=0, hi=2^b-1) every integer value
    maps to itself and the float just below it to the cell below."""
    for bits in (2, 6, 10):
        top = (1 << bits) - 1
        xs = np.arange(top + 1, dtype=np.float32)
        got = orc.quantise(xs, np.float32(0), np.float32(top), bits)
        assert np.array_equal(got, xs.astype(np.uint32)), bits
        below = np.nextafter(xs[1:], np.float32(-np.inf))
        got = orc.quantise(below, np.float32(0), np.float32(top), bits)
        assert np.array_equal(got, np.arange(top, dtype=np.uint32)), bits


def check_encode_joint_range(orc):
    """Codes share one grid per segment: the smallest value of each axis over
    q and k gets grid coordinate 0 and the largest 2^b - 1; a point holding the
    per-axis minimum (maximum) of both sets gets code 0 (all ones)."""
    rng = np.random.default_rng(5)
    S, N, d, bits = 3, 40, 3, 10
    q = rng.standard_normal((S, N, d)).astype(np.float32)
    k = rng.standard_normal((S, N, d)).astype(np.float32) * 3 + 1
    both = np.concatenate([q, k], axis=1)
    lo, hi = both.min(axis=1), both.max(axis=1)
    q[:, 0, :] = lo
    k[:, 1, :] = hi
    qc, kc, lo2, hi2 = orc.morton_encode(q, k, bits)
    assert np.array_equal(lo2, lo) and np.array_equal(hi2, hi)
    assert np.all(qc[:, 0] == 0)
    assert np.all(kc[:, 1] == (1 << (d * bits)) - 1)
    assert qc.dtype == np.uint32 and kc.dtype == np.uint32
    # Caller range: values outside clamp to the grid's edges.
    lo_c = np.zeros((S, d), np.float32)
    hi_c = np.ones((S, d), np.float32)
    qc, kc, _, _ = orc.morton_encode(np.full((S, 1, d), -5, np.float32),
                                     np.full((S, 1, d), 5, np.float32), bits, (lo_c, hi_c))
    assert np.all(qc == 0) and np.all(kc == (1 << (d * bits)) - 1)


# ----------------------------------------------------------------------------
# Sort (Section 3.2.2; Algorithm 1, Step 2)
# ----------------------------------------------------------------------------

def check_sort_invariants(orc):
    """Sorted ascending, ties by ascending position, a permutation, and equal
    to Python's own sort on the (code, position) pairs."""
    rng = np.random.default_rng(3)
    for n, code_bits in ((1, 4), (50, 2), (300, 6), (1000, 18)):
        kc = rng.integers(0, 1 << code_bits, size=(2, n)).astype(np.uint32)
        sc, perm = orc.sort_keys(kc)
        for s in range(2):
            assert sorted(perm[s].tolist()) == list(range(n))
            assert np.array_equal(sc[s], kc[s][perm[s]])
            expect = sorted(range(n), key=lambda j: (int(kc[s, j]), j))
            assert perm[s].tolist() == expect


# ----------------------------------------------------------------------------
# Select (Section 3.2.2; Algorithm 1, Steps 3-5)
# ----------------------------------------------------------------------------

def _brute_window(kc, qc_i, i, k, causal):
    """The window rule written out with plain Python on one query."""
    pool = list(range(i + 1)) if causal else list(range(len(kc)))
    ordered = sorted(pool, key=lambda j: (int(kc[j]), j))
    p = sum(1 for j in pool if int(kc[j]) < int(qc_i))
    m = min(k, len(pool))
    start = p - k // 2
    start = max(start, 0)
    start = min(start, len(pool) - m)
    return ordered[start:start + m] + [-1] * (k - m)


def check_select_golden(orc):
    """The six-token hand-worked example, both modes."""
    rows = {r[0]: r[1:] for r in _rows("select_example.txt")}
    k = int(rows["k"][0])
    kc = np.array([[int(x) for x in rows["k_codes"]]], dtype=np.uint32)
    qc = np.array([[int(x) for x in rows["q_codes"]]], dtype=np.uint32)
    for mode, causal in (("causal", True), ("noncausal", False)):
        expect = [[int(x) for x in grp.split()] for grp in " ".join(rows[mode]).split("|")]
        got = orc.select_topk(qc, kc, k, causal)[0].tolist()
        assert got == expect, (mode, got, expect)
        for i in range(kc.shape[1]):
            assert orc.select_one(int(qc[0, i]), kc[0], i, k, causal).tolist() == expect[i], (mode, i)


def check_select_brute(orc):
    """Brute force on tiny inputs with heavy code ties (2 and 3 code bits)."""
    rng = np.random.default_rng(17)
    for n, code_bits, k in ((1, 2, 1), (5, 2, 3), (17, 2, 4), (33, 3, 7), (64, 2, 8), (40, 3, 64), (48, 6, 16)):
        kc = rng.integers(0, 1 << code_bits, size=(2, n)).astype(np.uint32)
        qc = rng.integers(0, 1 << code_bits, size=(2, n)).astype(np.uint32)
        for causal in (True, False):
            got = orc.select_topk(qc, kc, k, causal)
            for s in range(2):
                for i in range(n):
                    expect = _brute_window(kc[s], qc[s, i], i, k, causal)
                    assert got[s, i].tolist() == expect, (n, code_bits, k, causal, s, i)
                    one = orc.select_one(int(qc[s, i]), kc[s], i, k, causal)
                    assert one.tolist() == expect, (n, k, causal, s, i)


def check_select_invariants(orc):
    """Count, distinctness, causality, and the window being a contiguous run of
    the pool's (code, position) order that brackets the insertion point."""
    rng = np.random.default_rng(23)
    n, k = 200, 16
    for code_bits in (3, 12):
        kc = rng.integers(0, 1 << code_bits, size=(1, n)).astype(np.uint32)
        qc = rng.integers(0, 1 << code_bits, size=(1, n)).astype(np.uint32)
        for causal in (True, False):
            idx = orc.select_topk(qc, kc, k, causal)[0]
            for i in range(n):
                row = idx[i]
                L = i + 1 if causal else n
                sel = [j for j in row.tolist() if j >= 0]
                assert len(sel) == min(k, L)
                assert np.all(row[len(sel):] == -1)
                assert len(set(sel)) == len(sel)
                if causal:
                    assert max(sel) <= i
                ordered = sorted(range(L), key=lambda j: (int(kc[0, j]), j))
                start = ordered.index(sel[0])
                assert ordered[start:start + len(sel)] == sel
                p = sum(1 for j in range(L) if kc[0, j] < qc[0, i])
                # With k >= 2 the keys on both sides of the insertion point are in.
                if p >= 1:
                    assert ordered[p - 1] in sel, (i, p)
                if p < L:
                    assert ordered[p] in sel, (i, p)


def check_select_full_pool(orc):
    """With k at least the pool size the window is the whole pool."""
    rng = np.random.default_rng(29)
    n = 37
    kc = rng.integers(0, 64, size=(1, n)).astype(np.uint32)
    qc = rng.integers(0, 64, size=(1, n)).astype(np.uint32)
    for causal in (True, False):
        idx = orc.select_topk(qc, kc, n + 3, causal)[0]
        for i in range(n):
            L = i + 1 if causal else n
            sel = [j for j in idx[i].tolist() if j >= 0]
            assert sorted(sel) == list(range(L))


# ----------------------------------------------------------------------------
# Attend (Section 3.3, equation cauchy; Section 3.4; Appendix E.1)
# ----------------------------------------------------------------------------

def check_attend_hand(orc):
    """Two keys at squared distances 1 and 3 from q, eps = 1: scores 1/2 and
    1/4, weights 2/3 and 1/3."""
    q = np.zeros((1, 1, 3))
    k = np.array([[[1.0, 0, 0], [1.0, 1.0, 1.0]]])
    v = np.array([[[3.0, -6.0], [0.0, 9.0]]])
    qq = np.concatenate([q, np.zeros((1, 1, 3))], axis=1)
    idx = np.array([[[0, 1], [0, 1]]], dtype=np.int32)
    out = orc.attend(qq, k, v, idx, 1.0)
    assert np.allclose(out[0, 0], [2.0, -1.0], atol=1e-12), out[0, 0]
    # A padded slot contributes nothing.
    idx = np.array([[[0, -1], [1, -1]]], dtype=np.int32)
    out = orc.attend(qq, k, v, idx, 1.0)
    assert np.allclose(out[0], [[3.0, -6.0], [0.0, 9.0]], atol=1e-12)


def _dense_cauchy(q, k, v, eps, causal):
    """Dense Cauchy attention as one masked N x N matrix (float64)."""
    d2 = ((q[:, None, :] - k[None, :, :]) ** 2).sum(-1)
    s = 1.0 / (d2 + eps)
    if causal:
        s = np.tril(s)
    return (s @ v) / s.sum(axis=1, keepdims=True)


def check_attend_dense_limit(orc):
    """With k >= N the method is dense (causal) Cauchy attention."""
    rng = np.random.default_rng(31)
    for n, causal in ((64, True), (96, False), (80, True)):
        q = rng.standard_normal((2, n, 3)).astype(np.float32)
        k = rng.standard_normal((2, n, 3)).astype(np.float32)
        v = rng.standard_normal((2, n, 16)).astype(np.float32)
        res = orc.forward(q, k, v, n + 5, 0.5, causal, 10)
        for s in range(2):
            ref = _dense_cauchy(q[s].astype(np.float64), k[s].astype(np.float64),
                                v[s].astype(np.float64), 0.5, causal)
            assert np.allclose(res["out"][s], ref, rtol=1e-12, atol=1e-12), (n, causal)


def check_attend_special_cases(orc):
    """Causal o_0 = v_0; huge eps gives the plain mean over the window; a
    row without candidates is zero;
    identical keys give uniform weights; outputs stay inside the window's
    per-component range."""
    rng = np.random.default_rng(37)
    n, k, dv = 120, 16, 8
    q = rng.standard_normal((1, n, 3)).astype(np.float32)
    kk = rng.standard_normal((1, n, 3)).astype(np.float32)
    v = rng.standard_normal((1, n, dv)).astype(np.float32)
    res = orc.forward(q, kk, v, k, 0.5, True, 10)
    assert np.allclose(res["out"][0, 0], v[0, 0], atol=1e-15)
    idx = res["idx"][0]
    for i in range(n):
        sel = idx[i][idx[i] >= 0]
        rows64 = v[0][sel].astype(np.float64)
        lo, hi = rows64.min(axis=0), rows64.max(axis=0)
        assert np.all(res["out"][0, i] >= lo - 1e-12) and np.all(res["out"][0, i] <= hi + 1e-12)
    out_big = orc.attend(q, kk, v, res["idx"], 1e12)[0]
    for i in range(n):
        sel = idx[i][idx[i] >= 0]
        assert np.allclose(out_big[i], v[0][sel].astype(np.float64).mean(axis=0), atol=1e-9)
    same = np.repeat(kk[:, :1, :], n, axis=1)
    out_same = orc.attend(q, same, v, res["idx"], 0.5)[0]
    for i in range(n):
        sel = idx[i][idx[i] >= 0]
        assert np.allclose(out_same[i], v[0][sel].astype(np.float64).mean(axis=0), atol=1e-12)
    # A row without candidates (the chunked rule's first chunk) is zero.
    empty = res["idx"].copy()
    empty[0, 5] = -1
    assert np.all(orc.attend(q, kk, v, empty, 0.5)[0, 5] == 0.0)


def _frac(t):
    a, b = t.split("/")
    return float(a) / float(b)


def check_attend_bwd_golden(orc):
    """The hand-worked two-candidate example in golden/attend_bwd_example.txt."""
    rows = {}
    for line in open(os.path.join(GOLDEN, "attend_bwd_example.txt")):
        if line.strip() and not line.startswith("#"):
            key, *vals = line.split()
            rows[key] = vals
    q = np.array([[[float(x) for x in rows["q"]]]])
    k = np.array([[[float(x) for x in rows["k0"]], [float(x) for x in rows["k1"]]]])
    v = np.array([[[float(x)] for x in rows["v"]]])
    qq = np.concatenate([q, np.zeros((1, 1, 3))], axis=1)  # a second query row, unused (empty window)
    idx = np.array([[[0, 1], [-1, -1]]], dtype=np.int32)
    dout = np.array([[[float(rows["dout"][0])], [0.0]]])
    dq, dk, dv, deps = orc.attend_bwd(qq, k, v, idx, float(rows["eps"][0]), dout)
    assert np.allclose(dq[0, 0], [_frac(x) for x in rows["dq"]], atol=1e-12), dq[0, 0]
    assert np.allclose(dk[0, 0], [_frac(x) for x in rows["dk0"]], atol=1e-12), dk[0, 0]
    assert np.allclose(dk[0, 1], [_frac(x) for x in rows["dk1"]], atol=1e-12), dk[0, 1]
    assert np.allclose(dv[0, :, 0], [_frac(x) for x in rows["dv"]], atol=1e-12), dv[0]
    assert abs(deps - _frac(rows["deps"][0])) < 1e-12, deps
    assert np.all(dq[0, 1] == 0.0)


def _bwd_problem(seed, S=2, N=9, dk=3, dv=4, topk=4, causal=True):
    rng = np.random.default_rng(seed)
    q = rng.normal(size=(S, N, dk))
    k = rng.normal(size=(S, N, dk))
    v = rng.normal(size=(S, N, dv))
    dout = rng.normal(size=(S, N, dv))
    kc = rng.integers(0, 64, size=(S, N)).astype(np.uint32)
    qc = rng.integers(0, 64, size=(S, N)).astype(np.uint32)
    # Windows from a brute-force selection over the codes (any valid index sets would do).
    idx = np.full((S, N, topk), -1, dtype=np.int32)
    for s in range(S):
        for i in range(N):
            pool = sorted((int(kc[s, j]), j) for j in range(i + 1 if causal else N))
            p = sum(1 for c, _ in pool if c < int(qc[s, i]))
            m = min(topk, len(pool))
            st = min(max(p - topk // 2, 0), len(pool) - m)
            idx[s, i, :m] = [j for _, j in pool[st:st + m]]
    return q, k, v, dout, idx


def check_attend_bwd_finite_diff(orc):
    """Every gradient equals the central difference of L = sum dout . o, with
    o from orc.attend (Appendix E.1), in float64."""
    eps = 0.7
    q, k, v, dout, idx = _bwd_problem(71)
    dq, dk, dv, deps = orc.attend_bwd(q, k, v, idx, eps, dout)

    def loss(qx, kx, vx, e):
        return float(np.sum(dout * orc.attend(qx, kx, vx, idx, e)))

    h = 1e-6
    for name, arr, grad in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        for flat in range(arr.size):
            pos = np.unravel_index(flat, arr.shape)
            a1, a2 = arr.copy(), arr.copy()
            a1[pos] += h
            a2[pos] -= h
            args1 = {"q": q, "k": k, "v": v}
            args2 = dict(args1)
            args1[name], args2[name] = a1, a2
            fd = (loss(args1["q"], args1["k"], args1["v"], eps) - loss(args2["q"], args2["k"], args2["v"], eps)) / (2 * h)
            assert abs(fd - grad[pos]) <= 1e-6 * (1.0 + abs(fd)), (name, pos, fd, grad[pos])
    fd = (loss(q, k, v, eps + h) - loss(q, k, v, eps - h)) / (2 * h)
    assert abs(fd - deps) <= 1e-6 * (1.0 + abs(fd)), (fd, deps)


def check_attend_bwd_invariants(orc):
    """Shifting every q and k by one vector leaves each D unchanged, so
    sum dq + sum dk = 0; the weights of a row sum to 1, so sum dv = sum of
    dout over rows with candidates; a one-candidate row has o = v_j, so its q
    gradient is 0."""
    q, k, v, dout, idx = _bwd_problem(72, S=1, N=12, topk=5, causal=False)
    idx[0, 3, 1:] = -1  # a one-candidate row
    dq, dk, dv, deps = orc.attend_bwd(q, k, v, idx, 0.4, dout)
    assert np.allclose(dq.sum(axis=(0, 1)) + dk.sum(axis=(0, 1)), 0.0, atol=1e-10)
    assert np.allclose(dv.sum(axis=(0, 1)), dout.sum(axis=(0, 1)), atol=1e-10)
    assert np.allclose(dq[0, 3], 0.0, atol=1e-14)


# ----------------------------------------------------------------------------
# The paper's chunked causal rule (Section 3.2.2; Algorithm 1, Step 4)
# ----------------------------------------------------------------------------

def check_select_chunk_golden(orc):
    """The hand-worked example in golden/select_chunk_example.txt."""
    rows = {}
    want = {}
    for line in open(os.path.join(GOLDEN, "select_chunk_example.txt")):
        if line.strip() and not line.startswith("#"):
            key, *vals = line.split()
            if key == "row":
                want[int(vals[0])] = [int(x) for x in vals[1:]]
            else:
                rows[key] = [int(x) for x in vals]
    chunk, k = rows["chunk"][0], rows["k"][0]
    kc = np.array([rows["k_codes"]], dtype=np.uint32)
    qc = np.array([rows["q_codes"]], dtype=np.uint32)
    idx = orc.select_topk(qc, kc, k, True, chunk=chunk)
    for i, w in want.items():
        assert list(idx[0, i]) == w, (i, list(idx[0, i]), w)
        assert list(orc.select_one(int(qc[0, i]), kc[0], i, k, True, chunk=chunk)) == w, i


def check_select_chunk_brute(orc):
    """Brute force on tiny inputs: query i's pool is every key whose chunk
    index j // M is below the query's own i // M; the window is the rank
    window of the definition over that pool, in (code, position) order."""
    rng = np.random.default_rng(61)
    for n, M, k, bits in ((13, 3, 4, 2), (20, 4, 5, 3), (9, 1, 3, 2), (16, 16, 4, 2), (11, 20, 2, 2), (30, 7, 8, 2)):
        kc = rng.integers(0, 1 << bits, size=(1, n)).astype(np.uint32)
        qc = rng.integers(0, 1 << bits, size=(1, n)).astype(np.uint32)
        idx = orc.select_topk(qc, kc, k, True, chunk=M)
        for i in range(n):
            pool = sorted((int(kc[0, j]), j) for j in range(n) if j // M < i // M)
            p = sum(1 for c, _ in pool if c < int(qc[0, i]))
            m = min(k, len(pool))
            st = min(max(p - k // 2, 0), len(pool) - m)
            want = [j for _, j in pool[st:st + m]] + [-1] * (k - m)
            assert list(idx[0, i]) == want, (n, M, k, i, list(idx[0, i]), want)


def check_select_chunk_invariants(orc):
    """Queries of the first chunk see nothing; the queries of one chunk share
    one pool (so a common query code gives a common window); M = 1 is the
    exact prefix without the diagonal."""
    rng = np.random.default_rng(62)
    n, k = 64, 6
    kc = rng.integers(0, 16, size=(2, n)).astype(np.uint32)
    qc = rng.integers(0, 16, size=(2, n)).astype(np.uint32)
    for M in (5, 8, 64, 100):
        idx = orc.select_topk(qc, kc, k, True, chunk=M)
        assert np.all(idx[:, :min(M, n)] == -1), M
        same = np.broadcast_to(qc[:, :1], qc.shape).copy()
        idx_same = orc.select_topk(same, kc, k, True, chunk=M)
        for i in range(n):
            first = (i // M) * M
            assert np.array_equal(idx_same[:, i], idx_same[:, first]), (M, i)
            assert np.all(idx[:, i][idx[:, i] >= 0] < first), (M, i)
    one = orc.select_topk(qc, kc, k, True, chunk=1)
    for s in range(2):
        for i in range(1, n):
            pool = sorted((int(kc[s, j]), j) for j in range(i))
            p = sum(1 for c, _ in pool if c < int(qc[s, i]))
            m = min(k, len(pool))
            st = min(max(p - k // 2, 0), len(pool) - m)
            assert list(one[s, i, :m]) == [j for _, j in pool[st:st + m]], (s, i)


# ----------------------------------------------------------------------------
# Score variants (Section 4.3; Appendix G.2; equation 3)
# ----------------------------------------------------------------------------

def check_attend_modes_hand(orc):
    """Two candidates, q = (1,0,0), k_0 = (1,0,0), k_1 = (0,1,0), v = (1, 0),
    d = 3, eps = 1: each variant's output is the weight of k_0, in closed form."""
    import math
    q = np.array([[[1.0, 0.0, 0.0]]])
    k = np.array([[[1.0, 0.0, 0.0], [0.0, 1.0, 0.0]]])
    v = np.array([[[1.0], [0.0]]])
    idx = np.array([[[0, 1]]], dtype=np.int32)
    r3 = math.sqrt(3.0)
    want = {
        "dot": 1.0 / (1.0 + math.exp(-1.0 / r3)),  # logits 1/sqrt(3) and 0
        "norm_dot": 1.0 / (1.0 + math.exp(-1.0 / r3)),  # unit vectors: as dot
        "neg_euclid": 1.0 / (1.0 + math.exp(-2.0 / r3)),  # distances 0 and 2
        "inv_euclid": 1.0 / (1.0 + 1.0 / (math.sqrt(2.0) + 1.0)),  # 1/(0+1) and 1/(sqrt(2)+1)
        "cauchy": 1.0 / (1.0 + 1.0 / 3.0),  # 1/(0+1) and 1/(2+1)
    }
    for mode, w in want.items():
        got = float(orc.attend(q, k, v, idx, 1.0, mode=mode)[0, 0, 0])
        assert abs(got - w) < 1e-14, (mode, got, w)


def check_attend_modes_dense_limit(orc):
    """Softmax variants with every key in the window (k >= N, causal) equal
    masked softmax attention over the full score matrix (scipy's softmax of
    q K^T / sqrt(d), -D / sqrt(d) or the cosine matrix / sqrt(d))."""
    from scipy.special import softmax
    rng = np.random.default_rng(66)
    n, d, dv = 40, 3, 5
    q = rng.normal(size=(1, n, d))
    k = rng.normal(size=(1, n, d))
    v = rng.normal(size=(1, n, dv))
    qc, kc, _, _ = orc.morton_encode(q.astype(np.float32), k.astype(np.float32), 6)
    idx = orc.select_topk(qc, kc, n, True)
    mask = np.tril(np.ones((n, n), dtype=bool))
    qu = q[0] / np.linalg.norm(q[0], axis=1, keepdims=True)
    ku = k[0] / np.linalg.norm(k[0], axis=1, keepdims=True)
    d2 = ((q[0][:, None, :] - k[0][None, :, :]) ** 2).sum(-1)
    logits = {"dot": q[0] @ k[0].T / np.sqrt(d), "neg_euclid": -d2 / np.sqrt(d), "norm_dot": qu @ ku.T / np.sqrt(d)}
    for mode, z in logits.items():
        want = softmax(np.where(mask, z, -np.inf), axis=1) @ v[0]
        got = orc.attend(q, k, v, idx, 0.5, mode=mode)[0]
        assert np.allclose(got, want, atol=1e-12), mode


def check_attend_modes_invariants(orc):
    """neg_euclid on keys of one norm equals dot with the query doubled
    (-|q - k|^2 = 2 q.k - |q|^2 - |k|^2, the last two constant per row);
    norm_dot ignores the lengths of q and k; inv_euclid with a huge eps is
    the window mean; no variant depends on the history mean's place."""
    rng = np.random.default_rng(67)
    n, d, dv, kk = 30, 3, 4, 6
    q = rng.normal(size=(1, n, d))
    k = rng.normal(size=(1, n, d))
    k_sphere = 1.7 * k / np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.normal(size=(1, n, dv))
    qc, kc, _, _ = orc.morton_encode(q.astype(np.float32), k.astype(np.float32), 6)
    idx = orc.select_topk(qc, kc, kk, True)
    a = orc.attend(q, k_sphere, v, idx, 0.5, mode="neg_euclid")
    b = orc.attend(2.0 * q, k_sphere, v, idx, 0.5, mode="dot")
    assert np.allclose(a, b, atol=1e-12)
    scale_q = rng.uniform(0.2, 5.0, size=(1, n, 1))
    scale_k = rng.uniform(0.2, 5.0, size=(1, n, 1))
    a = orc.attend(q, k, v, idx, 0.5, mode="norm_dot")
    b = orc.attend(q * scale_q, k * scale_k, v, idx, 0.5, mode="norm_dot")
    assert np.allclose(a, b, atol=1e-12)
    big = orc.attend(q, k, v, idx, 1e13, mode="inv_euclid")[0]
    for i in range(n):
        sel = idx[0, i][idx[0, i] >= 0]
        assert np.allclose(big[i], v[0][sel].mean(axis=0), atol=1e-9), i
    # The history-mean candidate is one more key/value pair in every variant.
    mk, mv = orc.history_mean(k, v, True)
    k2 = np.concatenate([k, mk], axis=1)
    v2 = np.concatenate([v, mv], axis=1)
    idx2 = np.concatenate([idx, n + np.arange(n, dtype=np.int32)[None, :, None]], axis=2)
    q2 = np.concatenate([q, np.ones_like(q)], axis=1)
    idx2 = np.concatenate([idx2, np.zeros((1, n, kk + 1), dtype=np.int32)], axis=1)
    for mode in orc.SCORE_MODES:
        want = orc.attend(q2, k2, v2, idx2, 0.5, mode=mode)[:, :n]
        got = orc.attend(q, k, v, idx, 0.5, mean_k=mk, mean_v=mv, mode=mode)
        assert np.allclose(got, want, atol=1e-12), mode


# ----------------------------------------------------------------------------
# Locality preservation (Section 4.4)
# ----------------------------------------------------------------------------

def check_locality_golden(orc):
    """The hand-worked example in golden/locality_example.txt: windows,
    exact nearest keys (in order), shared counts and the mean share."""
    rows = {"window": {}, "nearest": {}}
    vals = {}
    for line in open(os.path.join(GOLDEN, "locality_example.txt")):
        if line.strip() and not line.startswith("#"):
            key, *rest = line.split()
            if key in rows:
                rows[key][int(rest[0])] = [int(x) for x in rest[1:]]
            else:
                vals[key] = rest
    bits, kn = int(vals["bits"][0]), int(vals["kn"][0])
    k = np.array(vals["keys"], dtype=np.float32).reshape(1, -1, 1)
    q = np.array(vals["queries"], dtype=np.float32).reshape(1, -1, 1)
    qc, kc, _, _ = orc.morton_encode(q, k, bits)
    win = orc.select_topk(qc, kc, kn, False)
    nn = orc.exact_knn(q, k, kn, False)
    for i, w in rows["window"].items():
        assert sorted(win[0, i]) == sorted(w), (i, win[0, i], w)
    for i, w in rows["nearest"].items():
        assert list(nn[0, i]) == w, (i, nn[0, i], w)
    assert list(orc.index_overlap(win, nn)[0]) == [int(x) for x in vals["shared"]]
    assert abs(orc.locality_overlap(q, k, bits, kn) - _frac(vals["overlap"][0])) < 1e-15


def check_knn_brute(orc):
    """Integer coordinates (float32 distances exact, many ties): the nearest
    keys of every query by exact integer arithmetic, ties by position, in
    both modes, for kn below and beyond the pool."""
    rng = np.random.default_rng(91)
    for d, n, kn in ((1, 12, 3), (2, 20, 5), (3, 17, 30), (5, 9, 4)):
        q = rng.integers(-3, 4, size=(2, n, d)).astype(np.float32)
        k = rng.integers(-3, 4, size=(2, n, d)).astype(np.float32)
        for causal in (False, True):
            got = orc.exact_knn(q, k, kn, causal)
            for s in range(2):
                for i in range(n):
                    pool = range(i + 1) if causal else range(n)
                    dist = {j: sum((int(q[s, i, a]) - int(k[s, j, a])) ** 2 for a in range(d)) for j in pool}
                    want = sorted(pool, key=lambda j: (dist[j], j))[:kn]
                    want = want + [-1] * (kn - len(want))
                    assert list(got[s, i]) == want, (d, n, kn, causal, s, i)


def check_knn_kdtree(orc):
    """Random float coordinates against scipy's k-d tree (float64), on the
    queries whose kn-th and next distances are well apart."""
    from scipy.spatial import cKDTree
    rng = np.random.default_rng(92)
    n, kn = 300, 16
    for d in (1, 3, 6):
        q = rng.normal(size=(1, n, d)).astype(np.float32)
        k = rng.normal(size=(1, n, d)).astype(np.float32)
        got = orc.exact_knn(q, k, kn, False)
        dist, ind = cKDTree(k[0].astype(np.float64)).query(q[0].astype(np.float64), k=kn + 1)
        checked = 0
        for i in range(n):
            if dist[i, kn] - dist[i, kn - 1] > 1e-4 * (1.0 + dist[i, kn]):
                assert set(got[0, i]) == set(ind[i, :kn]), (d, i)
                checked += 1
        assert checked > n // 2


def check_overlap_hand(orc):
    """Shared entries of two index rows, -1 ignored."""
    a = np.array([[1, 2, 3, -1], [5, -1, -1, -1], [-1, -1, -1, -1]], dtype=np.int32)
    b = np.array([[3, 4, 1], [6, 7, -1], [-1, -1, -1]], dtype=np.int32)
    assert list(orc.index_overlap(a, b)) == [2, 0, 0]


# ----------------------------------------------------------------------------
# History-mean candidate (Section 3.4, last paragraph)
# ----------------------------------------------------------------------------

def _history_example():
    rows = {}
    for line in open(os.path.join(GOLDEN, "history_mean_example.txt")):
        if line.strip() and not line.startswith("#"):
            key, *vals = line.split()
            rows[key] = vals
    q = np.array([[[float(x) for x in rows["q"]]] * 2])
    k = np.array([[[float(x) for x in rows["k0"]], [float(x) for x in rows["k1"]]]])
    v = np.array([[[float(x)] for x in rows["v"]]])
    idx = np.array([[[0, -1], [1, -1]]], dtype=np.int32)
    return rows, q, k, v, idx, float(rows["eps"][0])


def check_history_mean_golden(orc):
    """The hand-worked example in golden/history_mean_example.txt: the means,
    the outputs in both modes and every gradient of the causal case."""
    rows, q, k, v, idx, eps = _history_example()
    fr = lambda key: np.array([_frac(x) for x in rows[key]])  # noqa: E731
    mk, mv = orc.history_mean(k, v, True)
    assert np.allclose(mk[0, 0], fr("mean_k_causal0"), atol=1e-15) and np.allclose(mk[0, 1], fr("mean_k_causal1"), atol=1e-15)
    assert np.allclose(mv[0, :, 0], fr("mean_v_causal"), atol=1e-15)
    out = orc.attend(q, k, v, idx, eps, mean_k=mk, mean_v=mv)
    assert np.allclose(out[0, :, 0], fr("out_causal"), atol=1e-14), out
    fk, fv = orc.history_mean(k, v, False)
    assert np.allclose(fk[0], fr("mean_k_full")[None, :], atol=1e-15) and np.allclose(fv[0, :, 0], fr("mean_v_full")[0])
    out = orc.attend(q, k, v, idx, eps, mean_k=fk, mean_v=fv)
    assert np.allclose(out[0, :, 0], fr("out_full"), atol=1e-14), out
    dq, dk, dv, deps = orc.attend_bwd(q, k, v, idx, eps, np.ones((1, 2, 1)), history=True, causal=True)
    assert np.allclose(dq[0, 0], fr("dq0"), atol=1e-14) and np.allclose(dq[0, 1], fr("dq1"), atol=1e-14), dq
    assert np.allclose(dk[0, 0], fr("dk0"), atol=1e-14) and np.allclose(dk[0, 1], fr("dk1"), atol=1e-14), dk
    assert np.allclose(dv[0, :, 0], fr("dv"), atol=1e-14), dv
    assert abs(deps - _frac(rows["deps"][0])) < 1e-14, deps


def check_history_mean_brute(orc):
    """Each row's means summed term by term (math.fsum) over its history:
    rows 0..i when causal, all rows otherwise."""
    import math
    rng = np.random.default_rng(81)
    k = rng.normal(size=(2, 13, 3))
    v = rng.normal(size=(2, 13, 5))
    for causal in (True, False):
        mk, mv = orc.history_mean(k, v, causal)
        for seg in range(2):
            for i in range(13):
                hist = range(i + 1) if causal else range(13)
                for arr, mean in ((k, mk), (v, mv)):
                    for c in range(arr.shape[-1]):
                        want = math.fsum(arr[seg, j, c] for j in hist) / len(hist)
                        assert abs(mean[seg, i, c] - want) < 1e-14, (causal, seg, i, c)


def check_history_attend_augmented(orc):
    """The history-mean candidate is one more key/value pair: attending with
    it equals attending, without it, over keys and values extended by the
    mean rows, with row i's window extended by the index of its own mean row."""
    q, k, v, dout, idx = _bwd_problem(83, S=2, N=11, topk=4, causal=True)
    for causal in (True, False):
        mk, mv = orc.history_mean(k, v, causal)
        N = k.shape[1]
        k2 = np.concatenate([k, mk], axis=1)
        v2 = np.concatenate([v, mv], axis=1)
        extra = np.broadcast_to(N + np.arange(N, dtype=np.int32)[None, :, None], (2, N, 1))
        idx2 = np.concatenate([idx, extra], axis=2)
        q2 = np.concatenate([q, np.zeros_like(q)], axis=1)
        idx2 = np.concatenate([idx2, np.full((2, N, idx2.shape[2]), -1, dtype=np.int32)], axis=1)
        idx2[:, N:, 0] = 0  # the padding rows need a candidate; their output is not compared
        want = orc.attend(q2, k2, v2, idx2, 0.6)[:, :N]
        got = orc.attend(q, k, v, idx, 0.6, mean_k=mk, mean_v=mv)
        assert np.allclose(got, want, atol=1e-13), causal


def check_history_bwd_finite_diff(orc):
    """With the history-mean candidate, every gradient equals the central
    difference of L = sum dout . o, where o comes from orc.attend with the means
    of orc.history_mean recomputed from the perturbed k and v (so the
    difference also carries the means' dependence on every history row)."""
    eps = 0.45
    for causal in (True, False):
        q, k, v, dout, idx = _bwd_problem(84, S=1, N=8, topk=3, causal=causal)
        idx[0, 2, :] = -1  # a row that attends to its history mean alone
        dq, dk, dv, deps = orc.attend_bwd(q, k, v, idx, eps, dout, history=True, causal=causal)

        def loss(qx, kx, vx, e):
            mk, mv = orc.history_mean(kx, vx, causal)
            return float(np.sum(dout * orc.attend(qx, kx, vx, idx, e, mean_k=mk, mean_v=mv)))

        h = 1e-6
        for name, arr, grad in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
            for flat in range(arr.size):
                pos = np.unravel_index(flat, arr.shape)
                a1, a2 = arr.copy(), arr.copy()
                a1[pos] += h
                a2[pos] -= h
                args1 = {"q": q, "k": k, "v": v}
                args2 = dict(args1)
                args1[name], args2[name] = a1, a2
                fd = (loss(args1["q"], args1["k"], args1["v"], eps) - loss(args2["q"], args2["k"], args2["v"], eps)) / (2 * h)
                assert abs(fd - grad[pos]) <= 1e-6 * (1.0 + abs(fd)), (causal, name, pos, fd, grad[pos])
        fd = (loss(q, k, v, eps + h) - loss(q, k, v, eps - h)) / (2 * h)
        assert abs(fd - deps) <= 1e-6 * (1.0 + abs(fd)), (causal, fd, deps)


def check_history_bwd_invariants(orc):
    """With the history-mean candidate every row has a candidate and its
    weights (the mean's spread over the history) still sum to 1, so
    sum dv = sum dout over all rows; a common shift of q and k shifts the
    means too, so sum dq + sum dk = 0."""
    for causal in (True, False):
        q, k, v, dout, idx = _bwd_problem(85, S=2, N=10, topk=4, causal=causal)
        idx[1, 4, :] = -1
        dq, dk, dv, deps = orc.attend_bwd(q, k, v, idx, 0.3, dout, history=True, causal=causal)
        assert np.allclose(dv.sum(axis=(0, 1)), dout.sum(axis=(0, 1)), atol=1e-10), causal
        assert np.allclose(dq.sum(axis=(0, 1)) + dk.sum(axis=(0, 1)), 0.0, atol=1e-10), causal


ALL_PINS = [
    check_bf16_input,
    check_morton_golden,
    check_morton_bijection,
    check_morton_axis_order,
    check_quantise_golden,
    check_quantise_buckets,
    check_encode_joint_range,
    check_sort_invariants,
    check_select_golden,
    check_select_brute,
    check_select_invariants,
    check_select_full_pool,
    check_attend_hand,
    check_attend_dense_limit,
    check_attend_special_cases,
    check_attend_bwd_golden,
    check_attend_bwd_finite_diff,
    check_attend_bwd_invariants,
    check_attend_modes_hand,
    check_attend_modes_dense_limit,
    check_attend_modes_invariants,
    check_select_chunk_golden,
    check_select_chunk_brute,
    check_select_chunk_invariants,
    check_locality_golden,
    check_knn_brute,
    check_knn_kdtree,
    check_overlap_hand,
    check_history_mean_golden,
    check_history_mean_brute,
    check_history_attend_augmented,
    check_history_bwd_finite_diff,
    check_history_bwd_invariants,
]
