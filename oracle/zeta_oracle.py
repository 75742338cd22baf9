"""CPU oracle for the ZETA Z-order top-k attention forward pass and its gradients.

TEST INFRASTRUCTURE.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or run this module.  The
product path (the HIP library and its Python binding) never touches it, and
this module imports nothing from the product package.

It is a plain, slow, obviously correct NumPy restatement of what the paper
defines, one function per step, each citing the passage it follows:

1. ``joint_range`` / ``quantise``: normalise each coordinate to an integer grid
   of ``2**bits`` cells (Section 3.1, Z-order curves: normalisation and
   discretisation to an integer grid, the formula floor((x - min)(2^b - 1) /
   (max - min))).
2. ``interleave``: the Z-order value of the integer coordinates (Section 3.1,
   equation Z: bits interleaved most significant group first, axis 1 first in
   each group).
3. ``sort_keys``: keys sorted ascending by Z-value (Section 3.2.2; Algorithm 1,
   Step 2), ties by position.
4. ``select_topk`` / ``select_one``: per query, insertion point by binary search
   among the keys it may see, then a window of k keys centred there
   (Section 3.2.2, last two paragraphs; Algorithm 1, Steps 3-5).
5. ``attend``: Adaptive Cauchy-softmax over the selected keys and the weighted
   sum of their values (Section 3.3, equation cauchy; Section 3.4;
   Appendix E.1, steps 1-4).
6. ``attend_bwd``: the gradients of that attention with respect to q, k, v
   and eps for fixed windows (Appendix E.2, summary of gradient
   computations).
7. ``history_mean``: the mean key and mean value of each query's history,
   which ``attend`` and ``attend_bwd`` can append to every window as one more
   candidate (Section 3.4, last paragraph: the history mean appended to the
   top-k tokens with a cumulative sum, as smoothing).
8. Variants: ``pool_end`` with a chunk size gives the paper's chunked causal
   rule (Section 3.2.2; Algorithm 1, Step 4), and ``attend``'s ``mode`` the
   score variants it compares with the Cauchy score (Section 4.3; Appendix
   G.2; the dot-product softmax of equation 3).
9. The locality experiment (Section 4.4): ``exact_knn`` (the exact Euclidean
   nearest keys of each query), ``index_overlap`` and ``locality_overlap``
   (how many of them the Z-order window holds).

Readings where the paper is silent or ambiguous (each is also listed in the
design notes):

* Quantisation is evaluated in float32, left to right, one IEEE rounding per
  operation: den = hi - lo; t = x - lo; u = t * (2^b - 1); w = u / den;
  code = clamp(floor(w), 0, 2^b - 1); code = 0 when den is not positive.
* The range is per (batch, head, axis), joint over queries and keys, so both
  share one grid (Section 3.2.2 maps keys and queries into the same 1-D space).
  A caller-supplied range replaces it; values outside it clamp.
* Equation Z puts coordinate 1 (axis 0 here) at the most significant bit of
  each group of d bits; coordinates are read most significant bit first.
* Sort ties are broken by ascending position (a stable sort).
* The causal pool of query i is the exact prefix {0..i} (the chunk rule of
  Section 3.2.2 in the limit of chunk size 1, diagonal included); the
  non-causal pool is every key.
* The insertion point p counts the pool keys with a code strictly below the
  query's (torch.searchsorted's default left side).
* The window holds min(k, |pool|) keys: floor(k/2) before p and the rest at or
  after p, shifted inward at the pool's ends; it is emitted in (code,
  position) order, padded with -1 to length k.
* Distances use the unquantised q and k values; eps = gamma^2 > 0 is a scalar.
* The history-mean candidate (optional) is the pair (mean of k_0..k_i, mean of
  v_0..v_i) for causal query i, and the mean over all N rows when not causal.
  It is scored like any other candidate and joins the normaliser; a row with
  an empty window then attends to it alone.  Gradients flow through the means
  back to every key and value of the history.

Arithmetic: quantisation in float32 as above; attention in float64.
"""

from __future__ import annotations

import bisect
from typing import Optional, Tuple

import numpy as np


# ----------------------------------------------------------------------------
# Input conversion
# ----------------------------------------------------------------------------

def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact float32 value of each bfloat16 bit pattern (the top half of a float32)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def as_f32(x: np.ndarray, dtype: str) -> np.ndarray:
    """Float32 values of an input array given as float32 or as bfloat16 bits."""
    if dtype == "bf16":
        return bf16_bits_to_f32(x)
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32)
    raise ValueError(dtype)


# ----------------------------------------------------------------------------
# Step 1: normalise and discretise (Section 3.1, Z-order curves)
# ----------------------------------------------------------------------------

def joint_range(q: np.ndarray, k: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Per-segment, per-axis min and max over the queries and keys together.

    q, k: float32 [S, N, d].  Returns (lo, hi), each float32 [S, d].
    """
    both = np.concatenate([q, k], axis=1)
    return both.min(axis=1).astype(np.float32), both.max(axis=1).astype(np.float32)


def quantise(x: np.ndarray, lo: np.ndarray, hi: np.ndarray, bits: int) -> np.ndarray:
    """Integer grid coordinate of each value: floor((x - lo)(2^b - 1) / (hi - lo)).

    x: float32 [..., d]; lo, hi: float32 broadcastable to x.  Evaluated in
    float32 with one rounding per operation, clamped to [0, 2^b - 1]; a
    non-positive range gives 0.  Returns uint32 of x's shape.
    """
    x = np.asarray(x, dtype=np.float32)
    lo = np.asarray(lo, dtype=np.float32)
    hi = np.asarray(hi, dtype=np.float32)
    top = np.float32((1 << bits) - 1)
    with np.errstate(divide="ignore", invalid="ignore", over="ignore"):
        den = (hi - lo).astype(np.float32)
        t = (x - lo).astype(np.float32)
        u = (t * top).astype(np.float32)
        w = (u / den).astype(np.float32)
        w = np.where(den > np.float32(0), w, np.float32(0))
    c = np.clip(np.floor(w), np.float32(0), top)
    return c.astype(np.uint32)


# ----------------------------------------------------------------------------
# Step 2: bit interleave (Section 3.1, equation Z)
# ----------------------------------------------------------------------------

def interleave(coords: np.ndarray, bits: int) -> np.ndarray:
    """Z-order value of integer coordinates.

    coords: uint [..., d], each below 2**bits.  The value is the bit string
    b_{1,1} b_{2,1} .. b_{d,1} b_{1,2} .. b_{d,n}, where b_{a,1} is the most
    significant bit of coordinate a.  Bit s (counted from the least
    significant end) of coordinate a therefore lands at position
    d*s + (d - 1 - a) of the result.  Returns uint64 of shape coords.shape[:-1].
    """
    coords = np.asarray(coords).astype(np.uint64)
    d = coords.shape[-1]
    z = np.zeros(coords.shape[:-1], dtype=np.uint64)
    for a in range(d):
        for s in range(bits):
            bit = (coords[..., a] >> np.uint64(s)) & np.uint64(1)
            z |= bit << np.uint64(d * s + (d - 1 - a))
    return z


def morton_encode(q: np.ndarray, k: np.ndarray, bits: int,
                  range_lohi: Optional[Tuple[np.ndarray, np.ndarray]] = None):
    """Z-order codes of queries and keys on one shared grid per segment.

    q, k: float32 [S, N, d].  range_lohi: optional (lo, hi), each [S, d],
    replacing the joint min/max.  Returns (q_codes, k_codes, lo, hi) with
    codes as uint32 [S, N].
    """
    if range_lohi is None:
        lo, hi = joint_range(q, k)
    else:
        lo, hi = (np.asarray(a, dtype=np.float32) for a in range_lohi)
    qc = interleave(quantise(q, lo[:, None, :], hi[:, None, :], bits), bits)
    kc = interleave(quantise(k, lo[:, None, :], hi[:, None, :], bits), bits)
    return qc.astype(np.uint32), kc.astype(np.uint32), lo, hi


# ----------------------------------------------------------------------------
# Step 3: sort keys by Z-value (Section 3.2.2; Algorithm 1, Step 2)
# ----------------------------------------------------------------------------

def sort_keys(k_codes: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Ascending sort of each segment's key codes, ties by position.

    k_codes: uint32 [S, N].  Returns (sorted_codes uint32 [S, N], perm int32
    [S, N]) with sorted_codes[s] == k_codes[s][perm[s]].
    """
    perm = np.argsort(k_codes, axis=-1, kind="stable").astype(np.int32)
    return np.take_along_axis(k_codes, perm, axis=-1), perm


# ----------------------------------------------------------------------------
# Step 4: candidate window per query (Section 3.2.2; Algorithm 1, Steps 3-5)
# ----------------------------------------------------------------------------

def _window(p: int, pool_size: int, k: int) -> Tuple[int, int]:
    """Start and length of the k-window centred at insertion point p in a pool."""
    m = min(k, pool_size)
    s = min(max(p - k // 2, 0), pool_size - m)
    return s, m


def pool_end(i: int, n: int, causal: bool, chunk: int = 0) -> int:
    """One past the largest key position query i may see.

    Exact causal prefix (chunk 0): i + 1, the diagonal included.  The paper's
    chunked rule with chunk size M = chunk (Section 3.2.2; Algorithm 1, Step
    4): the first floor(i / M) chunks of positions, i.e. positions below
    floor(i / M) * M, so queries of the first chunk see no key.  Without
    causality: n.
    """
    if not causal:
        return n
    if chunk > 0:
        return (i // chunk) * chunk
    return i + 1


def select_one(q_code: int, k_codes: np.ndarray, i: int, k: int, causal: bool, chunk: int = 0) -> np.ndarray:
    """Window of one query, straight from the definition (no incremental state).

    k_codes: uint32 [N] of one segment; i: the query's position.  Returns
    int32 [k]: key positions in (code, position) order, padded with -1.
    """
    n = len(k_codes)
    pool = np.arange(pool_end(i, n, causal, chunk), dtype=np.int64)
    pc = k_codes[pool].astype(np.int64)
    order = pool[np.lexsort((pool, pc))]  # by code, then by position
    p = int(np.count_nonzero(pc < int(q_code)))
    s, m = _window(p, len(pool), k)
    out = np.full(k, -1, dtype=np.int32)
    out[:m] = order[s:s + m]
    return out


def select_topk(q_codes: np.ndarray, k_codes: np.ndarray, k: int, causal: bool, chunk: int = 0) -> np.ndarray:
    """Windows of every query of every segment.

    q_codes, k_codes: uint32 [S, N].  Returns int32 [S, N, k].  The causal
    case keeps the pool as a sorted Python list of (code, position) keys,
    adding keys up to ``pool_end`` before answering each query (the pool only
    grows with i); the non-causal case sorts all keys once.  Both give
    exactly what ``select_one`` gives.  ``chunk`` > 0 selects the paper's
    chunked causal rule (see ``pool_end``).
    """
    S, n = k_codes.shape
    idx = np.full((S, n, k), -1, dtype=np.int32)
    for seg in range(S):
        kc = k_codes[seg].astype(np.int64)
        qc = q_codes[seg].astype(np.int64)
        if causal:
            pool = []  # sorted keys code * 2^32 + position, i.e. (code, position) order
            for i in range(n):
                end = pool_end(i, n, True, chunk)
                while len(pool) < end:
                    j = len(pool)
                    bisect.insort(pool, (int(kc[j]) << 32) | j)
                p = bisect.bisect_left(pool, int(qc[i]) << 32)
                s, m = _window(p, end, k)
                idx[seg, i, :m] = [e & 0xFFFFFFFF for e in pool[s:s + m]]
        else:
            order = np.argsort(kc, kind="stable")
            sorted_codes = kc[order]
            ps = np.searchsorted(sorted_codes, qc, side="left")
            for i in range(n):
                s, m = _window(int(ps[i]), n, k)
                idx[seg, i, :m] = order[s:s + m]
    return idx


# ----------------------------------------------------------------------------
# Step 5: Adaptive Cauchy-softmax attention over the window
# (Section 3.3, equation cauchy; Section 3.4; Appendix E.1)
# ----------------------------------------------------------------------------

def history_mean(k: np.ndarray, v: np.ndarray, causal: bool) -> Tuple[np.ndarray, np.ndarray]:
    """Mean key and mean value of each query's history (Section 3.4, last
    paragraph: a cumulative sum gives the history's mean vector, appended to
    the top-k candidates).

    Causal: row i holds (k_0 + ... + k_i) / (i + 1) and likewise for v.  Not
    causal: every row holds the mean over all N rows.  k: [S, N, dk], v:
    [S, N, dv]; float64 results of the same shapes.
    """
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    N = k.shape[1]
    if causal:
        count = np.arange(1, N + 1, dtype=np.float64)[None, :, None]
        return np.cumsum(k, axis=1) / count, np.cumsum(v, axis=1) / count
    mk = np.broadcast_to(k.mean(axis=1, keepdims=True), k.shape).copy()
    mv = np.broadcast_to(v.mean(axis=1, keepdims=True), v.shape).copy()
    return mk, mv


SCORE_MODES = ("cauchy", "dot", "neg_euclid", "inv_euclid", "norm_dot")


def _variant_weights(mode: str, qr: np.ndarray, kr: np.ndarray, dist: np.ndarray, valid: np.ndarray, eps: float,
                     mk: Optional[np.ndarray]):
    """Unnormalised weights of the score variants compared in Section 4.3 and
    Appendix G.2, over one block of windows (qr [b, d], kr [b, c, d], dist
    [b, c] = ||q - k||^2), and of the history-mean candidate (mk [b, d]) or
    None.

      dot         softmax of q.k / sqrt(d)                    (equation 3)
      neg_euclid  softmax of -||q - k||^2 / sqrt(d)
      norm_dot    softmax of (q/|q|).(k/|k|) / sqrt(d)         (a zero vector stays zero)
      inv_euclid  1 / (||q - k|| + eps)

    Softmax weights are exponentials shifted by the row's largest logit
    (the mean candidate's included), which leaves the normalised result
    unchanged.
    """
    d = qr.shape[-1]

    def unit(x):
        n = np.linalg.norm(x, axis=-1, keepdims=True)
        return x / np.where(n > 0, n, 1.0)

    def terms(keys, dd):
        if mode == "inv_euclid":
            return 1.0 / (np.sqrt(dd) + eps)
        if mode == "dot":
            return np.einsum("bd,bcd->bc", qr, keys) / np.sqrt(d)
        if mode == "neg_euclid":
            return -dd / np.sqrt(d)
        if mode == "norm_dot":
            return np.einsum("bd,bcd->bc", unit(qr), unit(keys)) / np.sqrt(d)
        raise ValueError(f"unknown score mode {mode!r}")

    t = terms(kr, dist)
    tm = None
    if mk is not None:
        dm = qr - mk
        tm = terms(mk[:, None, :], np.sum(dm * dm, axis=-1)[:, None])[:, 0]
    if mode == "inv_euclid":
        return np.where(valid, t, 0.0), tm
    zmax = np.max(np.where(valid, t, -np.inf), axis=1)
    if tm is not None:
        zmax = np.maximum(zmax, tm)
    zmax = np.where(np.isfinite(zmax), zmax, 0.0)
    w = np.where(valid, np.exp(t - zmax[:, None]), 0.0)
    return w, (None if tm is None else np.exp(tm - zmax))


def attend(q: np.ndarray, k: np.ndarray, v: np.ndarray, idx: np.ndarray, eps: float,
           rows: Optional[np.ndarray] = None, block: int = 512,
           mean_k: Optional[np.ndarray] = None, mean_v: Optional[np.ndarray] = None,
           mode: str = "cauchy") -> np.ndarray:
    """o_i = sum_j S_ij v_j / sum_j S_ij with S_ij = 1 / (||q_i - k_j||^2 + eps).

    q, k: [S, N, dk]; v: [S, N, dv] (float values of any float dtype); idx:
    int32 [S, N, k] with -1 for empty slots (or [S, R, k] when ``rows`` gives
    the R query positions it belongs to).  Computed in float64.  Returns
    float64 [S, N, dv] (or [S, R, dv]).

    With ``mean_k`` and ``mean_v`` ([S, N, dk] and [S, N, dv], from
    ``history_mean``), row i's window gains one more candidate, the pair
    (mean_k[i], mean_v[i]), scored and normalised like the others.

    ``mode`` picks the score: "cauchy" (equation cauchy, the method's own) or
    one of the variants of ``_variant_weights``; the selection is the same.
    A row with no candidate at all (an empty pool under the chunked rule) is
    zero.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    with_mean = mean_k is not None
    S = q.shape[0]
    if rows is None:
        rows = np.arange(q.shape[1])
    out = np.zeros((S, len(rows), v.shape[-1]), dtype=np.float64)
    for seg in range(S):
        for r0 in range(0, len(rows), block):
            rr = rows[r0:r0 + block]
            ii = idx[seg, r0:r0 + len(rr)]
            valid = ii >= 0
            jj = np.where(valid, ii, 0)
            diff = q[seg, rr][:, None, :] - k[seg][jj]  # [b, k, dk]
            dist = np.sum(diff * diff, axis=-1)  # D_ij
            mk = np.asarray(mean_k[seg, rr], dtype=np.float64) if with_mean else None
            if mode == "cauchy":
                score = np.where(valid, 1.0 / (dist + eps), 0.0)  # S_ij
                if with_mean:
                    dm = q[seg, rr] - mk
                    sm = 1.0 / (np.sum(dm * dm, axis=-1) + eps)
            else:
                score, sm = _variant_weights(mode, q[seg, rr], k[seg][jj], dist, valid, eps, mk)
            z = score.sum(axis=1)  # Z_i
            num = np.einsum("bk,bkd->bd", score, v[seg][jj])
            if with_mean:  # the history-mean candidate
                z = z + sm
                num = num + sm[:, None] * np.asarray(mean_v[seg, rr], dtype=np.float64)
            zs = np.where(z > 0, z, 1.0)  # a row without candidates is zero
            out[seg, r0:r0 + len(rr)] = num / zs[:, None]
    return out


def attend_bwd(q: np.ndarray, k: np.ndarray, v: np.ndarray, idx: np.ndarray, eps: float, dout: np.ndarray,
               block: int = 512, history: bool = False, causal: bool = True):
    """Gradients of L = sum_i dout_i . o_i through the attention of ``attend``
    (Appendix E.2, summary of gradient computations), for fixed windows idx.

    With delta_ij = D_ij + eps, S_ij = 1 / delta_ij, Z_i = sum_j S_ij,
    A_ij = S_ij / Z_i and o_i = sum_j A_ij v_j:
      dL/dv_j   =  sum over queries i whose window holds j of A_ij dout_i
      dL/dq_i   = -2 sum_j [dout_i . (v_j - o_i)] / Z_i (q_i - k_j) / delta_ij^2
      dL/dk_j   =  2 sum over i of [dout_i . (v_j - o_i)] / Z_i (q_i - k_j) / delta_ij^2
      dL/deps   = -sum_i sum_j [dout_i . (v_j - o_i)] / Z_i / delta_ij^2
    o_i is recomputed here (it equals the forward output exactly in float64).
    The selection itself has no gradient.

    q, k: [S, N, dk]; v, dout: [S, N, dv]; idx: int32 [S, N, k] with -1 for
    empty slots.  Computed in float64.  Returns (dq [S, N, dk], dk [S, N, dk],
    dv [S, N, dv], deps float).

    With ``history`` the windows also hold the history-mean candidate of
    ``history_mean(k, v, causal)``.  Its terms are those of any candidate, with
    (mean_k[i], mean_v[i]) in place of (k_j, v_j); the gradients that reach
    mean_k[i] and mean_v[i] then pass to every row of query i's history, each
    divided by the history's length: row j receives the sum over the queries
    i >= j (causal) or over all queries (not causal).
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    dout = np.asarray(dout, dtype=np.float64)
    S, N = q.shape[0], q.shape[1]
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    deps = 0.0
    if history:
        mean_k, mean_v = history_mean(k, v, causal)
        dmk = np.zeros_like(k)  # gradient reaching mean_k[i]
        dmv = np.zeros_like(v)  # gradient reaching mean_v[i]
    for seg in range(S):
        for r0 in range(0, N, block):
            rr = np.arange(r0, min(N, r0 + block))
            ii = idx[seg, rr]
            valid = ii >= 0
            jj = np.where(valid, ii, 0)
            diff = q[seg, rr][:, None, :] - k[seg][jj]  # q_i - k_j, [b, k, dk]
            delta = np.sum(diff * diff, axis=-1) + eps  # delta_ij
            score = np.where(valid, 1.0 / delta, 0.0)  # S_ij
            z = score.sum(axis=1)  # Z_i
            if history:
                dm = q[seg, rr] - mean_k[seg, rr]  # q_i - mean_k[i]
                delta_m = np.sum(dm * dm, axis=-1) + eps
                z = z + 1.0 / delta_m
            has = z > 0
            zs = np.where(has, z, 1.0)
            a = score / zs[:, None]  # A_ij
            vj = v[seg][jj]  # [b, k, dv]
            o = np.einsum("bk,bkd->bd", a, vj)  # o_i
            if history:
                a_m = 1.0 / delta_m / zs
                o = o + a_m[:, None] * mean_v[seg, rr]
            du = dout[seg, rr]  # [b, dv]
            g = np.einsum("bd,bkd->bk", du, vj) - np.einsum("bd,bd->b", du, o)[:, None]  # dout_i . (v_j - o_i)
            w = np.where(valid, g / zs[:, None] / (delta * delta), 0.0)
            dq[seg, rr] = -2.0 * np.einsum("bk,bkd->bd", w, diff)
            sel = valid.ravel()
            np.add.at(dk[seg], jj.ravel()[sel], (2.0 * w[:, :, None] * diff).reshape(-1, diff.shape[-1])[sel])
            np.add.at(dv[seg], jj.ravel()[sel], (a[:, :, None] * du[:, None, :]).reshape(-1, du.shape[-1])[sel])
            deps -= float(w.sum())
            if history:
                g_m = np.einsum("bd,bd->b", du, mean_v[seg, rr] - o)
                w_m = g_m / zs / (delta_m * delta_m)
                dq[seg, rr] -= 2.0 * w_m[:, None] * dm
                dmk[seg, rr] = 2.0 * w_m[:, None] * dm
                dmv[seg, rr] = a_m[:, None] * du
                deps -= float(w_m.sum())
    if history:
        # Row j of the history receives d(mean)/d(row j) = 1 / (history length).
        if causal:
            count = np.arange(1, N + 1, dtype=np.float64)[None, :, None]
            dk += np.cumsum((dmk / count)[:, ::-1], axis=1)[:, ::-1]
            dv += np.cumsum((dmv / count)[:, ::-1], axis=1)[:, ::-1]
        else:
            dk += dmk.sum(axis=1, keepdims=True) / N
            dv += dmv.sum(axis=1, keepdims=True) / N
    return dq, dk, dv, deps


# ----------------------------------------------------------------------------
# The whole forward
# ----------------------------------------------------------------------------

def forward(q: np.ndarray, k: np.ndarray, v: np.ndarray, topk: int, eps: float, causal: bool,
            bits: int, range_lohi=None, history: bool = False, chunk: int = 0, mode: str = "cauchy") -> dict:
    """All five steps for float32 inputs shaped [S, N, d]; returns every
    intermediate.  ``history`` appends the history-mean candidate; ``chunk``
    and ``mode`` pick the chunked causal rule and a score variant."""
    qc, kc, lo, hi = morton_encode(q, k, bits, range_lohi)
    sorted_codes, perm = sort_keys(kc)
    idx = select_topk(qc, kc, topk, causal, chunk=chunk)
    mk, mv = history_mean(k, v, causal) if history else (None, None)
    out = attend(q, k, v, idx, eps, mean_k=mk, mean_v=mv, mode=mode)
    return dict(q_codes=qc, k_codes=kc, lo=lo, hi=hi, sorted_codes=sorted_codes, perm=perm,
                idx=idx, mean_k=mk, mean_v=mv, out=out)


# ----------------------------------------------------------------------------
# Locality preservation (Section 4.4)
# ----------------------------------------------------------------------------

def exact_knn(q: np.ndarray, k: np.ndarray, kn: int, causal: bool, rows: Optional[np.ndarray] = None) -> np.ndarray:
    """The kn keys nearest to each query in Euclidean distance, among the
    query's pool ({0..i} when causal, all keys otherwise), ordered by
    (distance, position) and padded with -1.

    The squared distance is computed in float32 as the GPU computes it (one
    rounding per subtraction, product and sum, axes in order, no fused
    multiply-add), so that both take the same decision where distances tie
    or nearly tie.  q, k: float32 [S, N, d].  Returns int32 [S, N, kn] (or
    [S, R, kn] for the R query positions ``rows``).
    """
    q = np.asarray(q, dtype=np.float32)
    k = np.asarray(k, dtype=np.float32)
    S, N, d = q.shape
    if rows is None:
        rows = np.arange(N)
    out = np.full((S, len(rows), kn), -1, dtype=np.int32)
    for seg in range(S):
        for r, i in enumerate(rows):
            end = i + 1 if causal else N
            d2 = np.zeros(end, dtype=np.float32)
            for a in range(d):
                diff = (q[seg, i, a] - k[seg, :end, a]).astype(np.float32)
                d2 = (d2 + (diff * diff).astype(np.float32)).astype(np.float32)
            order = np.lexsort((np.arange(end), d2))  # by distance, then position
            m = min(kn, end)
            out[seg, r, :m] = order[:m]
    return out


def index_overlap(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Per row, the number of indices (not -1) that rows a and b share.
    a: int32 [..., ka], b: int32 [..., kb] with distinct valid entries per
    row.  Returns int32 [...]."""
    a2 = a.reshape(-1, a.shape[-1])
    b2 = b.reshape(-1, b.shape[-1])
    out = np.zeros(a2.shape[0], dtype=np.int32)
    for r in range(a2.shape[0]):
        out[r] = len(set(int(x) for x in a2[r] if x >= 0) & set(int(x) for x in b2[r] if x >= 0))
    return out.reshape(a.shape[:-1])


def locality_overlap(q: np.ndarray, k: np.ndarray, bits: int, kn: int = 64, causal: bool = False) -> float:
    """The locality measure of Section 4.4: the mean, over queries, of the
    fraction of the kn exact nearest keys (``exact_knn``) that the Z-order
    window of the same size (``select_topk`` on ``morton_encode``'s codes)
    also holds.  q, k: float32 [S, N, d]."""
    qc, kc, _, _ = morton_encode(q, k, bits)
    win = select_topk(qc, kc, kn, causal)
    nn = exact_knn(q, k, kn, causal)
    return float(index_overlap(win, nn).sum()) / float(np.count_nonzero(nn >= 0))

