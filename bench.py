"""Benchmark of the Z-order top-k attention forward on one MI355X.

One step is the whole forward (encode, sort of the query and key codes, the
processing order, then select and attend in one pass: C ABI calls on one
stream) over one batch of the long-context workload (B=1, H=16,
N=65536, d_k=3, d_v=128, k=128, bf16, 6 bits per axis, causal), with inputs,
outputs and workspace resident in HBM before timing starts.

Prints one JSON line: query-tokens/s (B*N per second) of the whole step (K
steps between two synchronisations; per-step HIP events give the median, and
a cold-cache run writes a 512 MiB buffer before every step), the time of each
stage, the dominant call's roofline (the resource its counters show binding,
with the HBM traffic and the algorithmic byte rates beside it), the same step
through the separate select and attend calls, a timed device copy (the
measured HBM peak), and the CPU oracle timed on the whole workload on the
host's cores before the GPU is touched.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import workloads  # noqa: E402

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, vendor figure
# Vector-instruction issue of the whole chip: 256 compute units x 4 SIMDs, one
# wave64 VALU instruction per SIMD every 4 cycles (16 lanes wide), 2.4 GHz.
SIMDS = 256 * 4
CLOCK_GHZ = 2.4
VALU_PEAK_GINSTS = SIMDS * CLOCK_GHZ / 4.0  # 614.4 G wave64 VALU instructions/s
MFMA_BF16_PEAK_TFLOPS = 2500.0  # dense bf16 matrix-core peak
MAX_CPU_WORKERS = 16  # the host CPU share of one GPU
KERNEL_SRCS = [os.path.join(ROOT, "paper_2501_14577_amd", "csrc", n)
               for n in ("fused.hip", "tile.hip", "tile_device.h", "select.hip", "select_device.h", "attend_device.h",
                         "device_common.h", "layout.h")]
COUNTERS_FILE = os.path.join(ROOT, "profiles", "select_attend_long_context_counters.txt")


def elem_size(dtype: str) -> int:
    return 2 if dtype == "bf16" else 4


def candidates(w: workloads.Workload, causal: bool) -> int:
    """Exact number of selected (query, key) pairs over the whole batch."""
    N, k = w.N, w.topk
    if not causal:
        return w.segments * N * min(k, N)
    i = np.arange(N, dtype=np.int64)
    return int(w.segments * np.minimum(k, i + 1).sum())


def attend_bytes(w: workloads.Workload, causal: bool) -> int:
    """Algorithmic bytes of one attend launch: per query its q row, its k
    indices and its output row, per selected pair one key row and one value
    row; no reuse across queries is assumed."""
    s, d = elem_size(w.dtype), w.dk
    rows = w.segments * w.N
    return rows * (d * s + 4 * w.topk + w.dv * s) + candidates(w, causal) * (d * s + w.dv * s)


def sort_passes(code_bits: int) -> int:
    """Radix passes of the library's sort: digits of at most 9 bits."""
    return (code_bits + 8) // 9


def step_bytes(w: workloads.Workload, causal: bool) -> int:
    """Algorithmic bytes of the whole step: attend plus, per query row,
    encode 4*d*s + 8, sort 16 per radix pass and select 4 + 8k.  (The sort of
    the query codes, a scheduling aid, is not counted.)"""
    s, d = elem_size(w.dtype), w.dk
    rows = w.segments * w.N
    return attend_bytes(w, causal) + rows * ((4 * d * s + 8) + 16 * sort_passes(w.code_bits) + (4 + 8 * w.topk))


def compulsory_bytes(w: workloads.Workload) -> int:
    """Bytes any implementation must move: q, k and v read once, out written once."""
    s = elem_size(w.dtype)
    return w.segments * w.N * (2 * w.dk * s + 2 * w.dv * s)


def bwd_bytes(w: workloads.Workload, causal: bool) -> int:
    """Algorithmic bytes of one attention-gradient launch: per query row its
    q row, dout row, k indices, dq row and eps partial; per selected pair one
    key row and one value row read, and a read-modify-write of the float32
    dk and dv rows; no reuse across queries is assumed."""
    s, d = elem_size(w.dtype), w.dk
    rows = w.segments * w.N
    return rows * (d * s + w.dv * s + 4 * w.topk + 4 * d + 4) + candidates(w, causal) * (
        d * s + w.dv * s + 8 * d + 8 * w.dv)


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for path in KERNEL_SRCS:
        h.update(open(path, "rb").read())
    return h.hexdigest()


def read_counters():
    """Per-call counter totals of the one-pass select-and-attend call (its
    kernels summed) from the committed rocprofv3 summary; None when absent or
    taken on different kernel sources."""
    if not os.path.exists(COUNTERS_FILE):
        return None
    kv = {}
    for line in open(COUNTERS_FILE):
        if ":" in line and not line.startswith("#"):
            key, val = line.split(":", 1)
            kv[key.strip()] = val.strip()
    if kv.get("kernel_source_sha256") != kernel_source_hash():
        return None
    try:
        return {k: float(v) for k, v in kv.items() if k != "kernel_source_sha256"}
    except ValueError:
        return None


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_segment(job):
    """The whole oracle forward of one segment, single-threaded; returns its
    wall time."""
    import threadpoolctl

    import oracle

    q, k, v, topk, eps, causal, bits = job
    with threadpoolctl.threadpool_limits(1):
        t0 = time.perf_counter()
        oracle.forward(q, k, v, topk, eps, causal, bits)
        return time.perf_counter() - t0


def cpu_baseline(w: workloads.Workload, causal: bool, x: dict, segments: int):
    """The oracle, untuned, over ``segments`` segments of the workload (all of
    them by default), one segment per task on a pool of single-threaded
    worker processes, one per host core (at most the 16 of one GPU's share).
    Run before the GPU is initialised.  Scaled to query-tokens/s as the rows
    done over H per second (one query token carries H rows)."""
    import multiprocessing as mp

    import oracle

    S = w.segments
    segments = max(1, min(segments, S))
    f = {n: oracle.as_f32(a, w.dtype).reshape(S, w.N, a.shape[-1]) for n, a in x.items()}
    jobs = [(f["q"][s:s + 1], f["k"][s:s + 1], f["v"][s:s + 1], w.topk, workloads.EPS_DEFAULT, causal, w.bits)
            for s in range(segments)]
    cores = min(len(os.sched_getaffinity(0)), MAX_CPU_WORKERS, segments)
    t0 = time.perf_counter()
    with mp.get_context("fork").Pool(cores) as pool:
        per_seg = pool.map(_oracle_segment, jobs, chunksize=1)
    wall = time.perf_counter() - t0
    rows = segments * w.N
    one_core = w.N / w.H / float(np.mean(per_seg))
    return {
        "value": rows / w.H / wall,
        "unit": "query-tokens/s",
        "cores": cores,
        "kind": "oracle",
        "sample": (f"{segments} of {S} segments ({rows} query rows), whole oracle forward "
                   f"({'causal' if causal else 'non-causal'}), {cores} single-threaded worker processes, "
                   f"{wall:.1f} s wall; scaled as rows/H per second"),
        "cpu_model": cpu_model(),
        "host_cpus": len(os.sched_getaffinity(0)),
        "single_core_value": one_core,
        "single_core_segment_s": float(np.mean(per_seg)),
    }


def locality_experiment(zeta, torch, dev) -> dict:
    """Section 4.4's locality measure on synthetic N(0,1) queries and keys:
    the mean share of each query's 64 exact nearest keys that its Z-order
    window of 64 holds, for N in {512, 1024, 2048} and d_k = 1..8 (16
    segments each, not causal, bits = min(24, 32 // d_k)), with queries drawn
    apart from the keys and, second reading, with the keys as their own
    queries; plus the GPU time of the exact search and of the window
    selection at N = 2048, d_k = 3."""

    def measure(q, k, bits):
        shared, nn = zeta.locality_counts(q, k, bits, 64)
        return round(float(shared.sum().item()) / float((nn >= 0).sum().item()), 4)

    table, table_self = {}, {}
    for n in (512, 1024, 2048):
        for d in range(1, 9):
            w = workloads.custom(B=1, H=16, N=n, dk=d, dtype="f32", topk=64, bits=min(24, 32 // d), seed=n * 10 + d)
            x = workloads.generate(w)
            q, k = (torch.from_numpy(x[m]).to(dev) for m in ("q", "k"))
            table[f"N={n} d_k={d}"] = measure(q, k, w.bits)
            table_self[f"N={n} d_k={d}"] = measure(k, k, w.bits)
    w = workloads.custom(B=1, H=16, N=2048, dk=3, dtype="f32", topk=64, bits=10, seed=20483)
    x = workloads.generate(w)
    q, k = (torch.from_numpy(x[m]).to(dev) for m in ("q", "k"))
    ws = zeta.workspace_for(1, 16, 2048, 3, 10, 64, False, dev)
    qc, kc = zeta.zeta_morton_encode(q, k, 10, workspace=ws)
    sc, perm = zeta.zeta_sort_keys(kc, 30, workspace=ws)
    nn = zeta.zeta_exact_knn(q, k, 64, False)
    win = zeta.zeta_select_topk(qc, sc, perm, 64, False, workspace=ws)
    times = {}
    for name, fn in (("exact_knn_ms", lambda: zeta.zeta_exact_knn(q, k, 64, False, knn_idx=nn)),
                     ("select_ms", lambda: zeta.zeta_select_topk(qc, sc, perm, 64, False, idx=win, workspace=ws))):
        fn()
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        start.record()
        for _ in range(10):
            fn()
        stop.record()
        torch.cuda.synchronize()
        times[name] = start.elapsed_time(stop) / 10
    return {"measure": "mean share of the 64 exact nearest keys held by the Z-order window of 64",
            "overlap": table, "overlap_keys_as_queries": table_self, "timing_N2048_dk3_16_segments": times}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=5, help="workload number (parity cases 1-4, bench 5)")
    ap.add_argument("--noncausal", action="store_true")
    ap.add_argument("--cpu-segments", type=int, default=1 << 30,
                    help="segments in the oracle baseline (default all; 0 skips the CPU baseline)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run a plain 1 GiB device copy first (for counter calibration)")
    ap.add_argument("--parts", default="forward,backward,history,variants,locality",
                    help="comma list of the parts to time: forward (the metric), backward (attention gradients), "
                         "history (the history-mean candidate, forward and gradients), variants (the chunked "
                         "causal rule and the score variants), locality (the locality experiment); fields of "
                         "parts not timed are null, so that each part's profile holds only its own kernels")
    args = ap.parse_args()
    parts = set(args.parts.split(","))
    if not parts <= {"forward", "backward", "history", "variants", "locality"}:
        print(f"unknown part in --parts {args.parts}", file=sys.stderr)
        return 2

    if args.gpus != 1:
        print("bench.py runs on one GPU only: every (batch, head) segment is independent, "
              "so more GPUs would each run this same single-GPU step on their share.", file=sys.stderr)
        return 2

    w = workloads.CONFIGS[args.config]
    causal = not args.noncausal and True in w.causal
    x = workloads.generate(w)
    # The CPU baseline runs before anything touches the GPU (its worker
    # processes are forked from this one).
    cpu = cpu_baseline(w, causal, x, args.cpu_segments) if args.cpu_segments > 0 else None

    import torch

    import paper_2501_14577_amd as zeta

    if not torch.cuda.is_available():
        print("bench.py needs a ROCm GPU", file=sys.stderr)
        return 2
    zeta.load_library()
    dev = torch.device("cuda:0")

    def to_dev(a):
        if w.dtype == "bf16":
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(a).to(dev)

    q, k, v = to_dev(x["q"]), to_dev(x["k"]), to_dev(x["v"])
    tdtype = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    bufs = zeta.alloc_buffers(w.B, w.H, w.N, w.dv, w.topk, tdtype, dev)
    ws = zeta.workspace_for(w.B, w.H, w.N, w.dk, w.bits, w.topk, causal, dev)
    eps = workloads.EPS_DEFAULT
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)  # written between cold-cache steps

    if args.copy_calibration:
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    codes, sorted2, perm2 = bufs["codes"], bufs["sorted_codes2"], bufs["perm2"]

    def mark(ev, i):
        # record event i of a step's list (None entries are skipped)
        if ev is not None and i < len(ev) and ev[i] is not None:
            ev[i].record()

    def step_fused(ev=None):
        # encode -> joint sort -> processing order -> select and attend in one
        # pass; ev (optional): events at the start and after each stage
        mark(ev, 0)
        qc, kc = zeta.zeta_morton_encode(q, k, w.bits, q_codes=codes[0], k_codes=codes[1], workspace=ws)
        mark(ev, 1)
        zeta.zeta_sort_keys(codes, w.code_bits, sorted_codes=sorted2, perm=perm2, workspace=ws)
        mark(ev, 2)
        order = zeta.zeta_query_order(perm2[0], w.N, w.segments, w.topk, causal, order_out=bufs["order"],
                                      workspace=ws)
        mark(ev, 3)
        zeta.zeta_select_attend_fwd(q, k, v, qc, sorted2[1], perm2[1], w.topk, causal, eps, q_order=order,
                                    out=bufs["out"], workspace=ws)
        mark(ev, 4)

    def step(ev=None):
        # encode -> joint sort of query and key codes -> the query Z-order
        # regrouped by list level (processing order) -> select -> attend
        mark(ev, 0)
        qc, kc = zeta.zeta_morton_encode(q, k, w.bits, q_codes=codes[0], k_codes=codes[1], workspace=ws)
        zeta.zeta_sort_keys(codes, w.code_bits, sorted_codes=sorted2, perm=perm2, workspace=ws)
        order = zeta.zeta_query_order(perm2[0], w.N, w.segments, w.topk, causal, order_out=bufs["order"],
                                      workspace=ws)
        mark(ev, 1)
        idx = zeta.zeta_select_topk(qc, sorted2[1], perm2[1], w.topk, causal, q_order=order, idx=bufs["idx"],
                                    workspace=ws)
        mark(ev, 2)
        zeta.zeta_topk_attn_fwd(q, k, v, idx, eps, q_order=order, out=bufs["out"])
        mark(ev, 3)

    def new_events(n):
        return [[torch.cuda.Event(enable_timing=True) for _ in range(n)] for _ in range(args.steps)]

    def timed(fn, n_ev=2, cold=False):
        """W warm-up calls, then K timed calls between two synchronisations.
        Returns (total time / K, per-step event intervals [K, n_ev - 1], wall
        seconds).  cold: a 512 MiB buffer is written before every step,
        outside its events (the total then includes the writes)."""
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        evs = new_events(n_ev)
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        wall0 = time.perf_counter()
        start.record()
        for i in range(args.steps):
            if cold:
                flush.fill_(i & 0xFF)
            fn(evs[i])
        stop.record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - wall0
        iv = np.array([[e[j].elapsed_time(e[j + 1]) for j in range(n_ev - 1)] for e in evs])
        return start.elapsed_time(stop) / args.steps, iv, wall

    def whole(fn, n_ev):
        # a step's first to last event
        def g(ev=None):
            fn(None if ev is None else [ev[0]] + [None] * (n_ev - 2) + [ev[1]])
        return g

    rec = mark

    fwd = None
    if "forward" in parts:
        four_ms, four_iv, _ = timed(step, 4)
        ms_per_step, step_iv, wall = timed(whole(step_fused, 5), 2)
        _, stage_iv, _ = timed(step_fused, 5)
        _, cold_iv, _ = timed(whole(step_fused, 5), 2, cold=True)
        st = np.median(stage_iv, axis=0)
        fwd = dict(ms_per_step=ms_per_step, median_ms=float(np.median(step_iv[:, 0])), wall=wall,
                   cold_median_ms=float(np.median(cold_iv[:, 0])),
                   stages=dict(encode_ms=float(st[0]), sort_ms=float(st[1]), query_order_ms=float(st[2]),
                               select_attend_ms=float(st[3])),
                   four_ms=four_ms, four_median_ms=float(np.median(four_iv.sum(axis=1))),
                   select_ms=float(np.median(four_iv[:, 1])), attend_ms=float(np.median(four_iv[:, 2])))
        # The measured HBM peak: a plain 1 GiB device-to-device copy.
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev).fill_(3)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        c0.record()
        for _ in range(10):
            dst.copy_(src)
        c1.record()
        torch.cuda.synchronize()
        fwd["copy_GBs"] = 2.0 * (1 << 30) * 10 / (c0.elapsed_time(c1) * 1e-3) / 1e9
        del src, dst

    def per_s(amount, ms):  # amount per second, None when the part was not timed
        return None if ms is None else amount / (ms * 1e-3)

    def gbs(nbytes, ms):
        r = per_s(nbytes, ms)
        return None if r is None else r / 1e9

    def frac(nbytes, ms):
        r = gbs(nbytes, ms)
        return None if r is None else r / HBM_PEAK_GBS

    # Attention gradients (zeta_topk_attn_bwd) for the windows of the
    # four-call step, timed on their own; not part of the forward metric.
    dout = to_dev(workloads.generate_dout(w))
    f32 = dict(dtype=torch.float32, device=dev)
    gq = torch.empty((w.B, w.H, w.N, w.dk), **f32)
    gk = torch.empty_like(gq)
    gv = torch.empty((w.B, w.H, w.N, w.dv), **f32)
    geps = torch.empty(1, **f32)
    step()
    torch.cuda.synchronize()

    def call(fn):
        # one library call between two events
        def g(ev=None):
            rec(ev, 0)
            fn()
            rec(ev, 1)
        return g

    b_bytes = bwd_bytes(w, causal)
    bwd_ms = one_bwd_ms = None
    if "backward" in parts:
        bws = zeta.bwd_workspace_for(w.B, w.H, w.N, w.dk, w.dv, w.topk, "history" in parts, dev)
        bwd_ms = timed(call(lambda: zeta.zeta_topk_attn_bwd(q, k, v, bufs["idx"], dout, eps, q_order=bufs["order"],
                                                            dq=gq, dk=gk, dv=gv, deps=geps, workspace=bws)))[0]
        # The one-pass call's gradients (zeta_select_attend_bwd): the same
        # windows, from the lists, without an index tensor.
        tws = zeta.select_attend_bwd_workspace_for(w.B, w.H, w.N, w.dv, w.topk, causal, dev)
        one_bwd_ms = timed(call(lambda: zeta.zeta_select_attend_bwd(
            q, k, v, codes[0], sorted2[1], perm2[1], w.topk, causal, eps, dout, q_order=bufs["order"], dq=gq, dk=gk,
            dv=gv, deps=geps, workspace=tws)))[0]
        del tws

    # The history-mean candidate: the means (zeta_history_mean) timed alone,
    # the one-pass step with the candidate, and the gradients with it.
    mk = torch.empty((w.B, w.H, w.N, w.dk), **f32)
    mv = torch.empty((w.B, w.H, w.N, w.dv), **f32)

    def step_hist(ev=None):
        qc, kc = zeta.zeta_morton_encode(q, k, w.bits, q_codes=codes[0], k_codes=codes[1], workspace=ws)
        zeta.zeta_sort_keys(codes, w.code_bits, sorted_codes=sorted2, perm=perm2, workspace=ws)
        order = zeta.zeta_query_order(perm2[0], w.N, w.segments, w.topk, causal, order_out=bufs["order"],
                                      workspace=ws)
        zeta.zeta_history_mean(k, v, causal, mean_k=mk, mean_v=mv, workspace=ws)
        rec(ev, 0)
        zeta.zeta_select_attend_fwd(q, k, v, qc, sorted2[1], perm2[1], w.topk, causal, eps, q_order=order,
                                    mean_k=mk, mean_v=mv, out=bufs["out"], workspace=ws)
        rec(ev, 1)

    h_bytes = w.segments * w.N * (w.dk + w.dv) * (elem_size(w.dtype) + 4)  # read k, v once; write the means
    hist_ms = hist_step_ms = hist_fused_ms = hist_bwd_ms = hist_one_bwd_ms = None
    if "history" in parts:
        hist_ms = float(np.median(timed(call(lambda: zeta.zeta_history_mean(k, v, causal, mean_k=mk, mean_v=mv,
                                                                            workspace=ws)))[1]))
        hist_step_ms, iv, _ = timed(step_hist)
        hist_fused_ms = float(np.median(iv))
        hist_bwd_ms = timed(call(lambda: zeta.zeta_topk_attn_bwd(
            q, k, v, bufs["idx"], dout, eps, q_order=bufs["order"], mean_k=mk, mean_v=mv, causal=causal, dq=gq,
            dk=gk, dv=gv, deps=geps, workspace=bws)))[0] if "backward" in parts else None
        hws = zeta.select_attend_bwd_workspace_for(w.B, w.H, w.N, w.dv, w.topk, causal, dev, True)
        hist_one_bwd_ms = timed(call(lambda: zeta.zeta_select_attend_bwd(
            q, k, v, codes[0], sorted2[1], perm2[1], w.topk, causal, eps, dout, q_order=bufs["order"], mean_k=mk,
            mean_v=mv, dq=gq, dk=gk, dv=gv, deps=geps, workspace=hws)))[0]
        del hws

    # Variants: the paper's chunked causal rule with 32 chunks (the one-pass
    # step), and each score variant's one-pass call (matrix-core tiles).
    variants = None
    tokens = w.B * w.N
    f_bytes = attend_bytes(w, causal) + w.segments * w.N * 4  # plus each query's code, read instead of an index row
    if "variants" in parts:
        chunk = w.N // 32

        def step_chunked(ev=None):
            qc, kc = zeta.zeta_morton_encode(q, k, w.bits, q_codes=codes[0], k_codes=codes[1], workspace=ws)
            zeta.zeta_sort_keys(codes, w.code_bits, sorted_codes=sorted2, perm=perm2, workspace=ws)
            order = zeta.zeta_query_order(perm2[0], w.N, w.segments, w.topk, causal, chunk=chunk,
                                          order_out=bufs["order"], workspace=ws)
            rec(ev, 0)
            zeta.zeta_select_attend_fwd(q, k, v, qc, sorted2[1], perm2[1], w.topk, causal, eps, chunk=chunk,
                                        q_order=order, out=bufs["out"], workspace=ws)
            rec(ev, 1)

        chunk_step_ms, iv, _ = timed(step_chunked)
        step_fused()
        modes = {}
        for mode in ("dot", "neg_euclid", "inv_euclid", "norm_dot"):
            modes[mode] = float(np.median(timed(call(lambda mode=mode: zeta.zeta_select_attend_fwd(
                q, k, v, codes[0], sorted2[1], perm2[1], w.topk, causal, eps, score=mode, q_order=bufs["order"],
                out=bufs["out"], workspace=ws)))[1]))
        variants = {"chunk": chunk, "chunked_step_ms": chunk_step_ms,
                    "chunked_value": tokens / (chunk_step_ms * 1e-3),
                    "chunked_select_attend_ms": float(np.median(iv)), "score_select_attend_ms": modes,
                    "score_select_attend_GBs": {m: gbs(f_bytes, t) for m, t in modes.items()}}

    locality = locality_experiment(zeta, torch, dev) if "locality" in parts else None

    s_bytes = step_bytes(w, causal)
    c_bytes = compulsory_bytes(w)
    ctr = read_counters()
    call_ms = fwd["stages"]["select_attend_ms"] if fwd else None
    roofline = None
    if fwd is not None:
        valu = ctr.get("valu_insts_per_call") if ctr else None
        mfma = ctr.get("mfma_insts_per_call") if ctr else None
        traffic = ctr.get("hbm_bytes_per_call") if ctr else None
        achieved = None if valu is None else valu / (call_ms * 1e-3) / 1e9
        roofline = {
            # The call's kernels are bound by vector-instruction issue (their
            # counters): achieved = counted wave64 VALU instructions per call
            # over the call's time, peak = the chip's issue rate.
            "bound": "alu",
            "kernel": "zeta_select_attend_fwd (prefix lists, window bounds, 16-query matrix-core tiles)",
            "achieved": achieved,
            "peak": VALU_PEAK_GINSTS,
            "unit": "G wave64 VALU instructions/s",
            "frac": None if achieved is None else achieved / VALU_PEAK_GINSTS,
            "traffic": traffic,
            "kernel_ms": call_ms,
            "valu_insts_per_call": valu,
            "hbm_traffic_GBs": gbs(traffic, call_ms) if traffic else None,
            "hbm_traffic_frac": frac(traffic, call_ms) if traffic else None,
            "mfma_bf16_TFLOPs": None if mfma is None else mfma * 16384 / (call_ms * 1e-3) / 1e12,
            "mfma_bf16_frac": None if mfma is None else mfma * 16384 / (call_ms * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS,
            "lds_bank_conflict_cycles_per_call": ctr.get("lds_bank_conflict_cycles_per_call") if ctr else None,
            # Byte rates against the HBM peak: q, k, v read and out written
            # once (the compulsory bytes), and the no-reuse gather model (each
            # selected pair's key and value rows counted once per query).
            "compulsory_bytes": c_bytes,
            "compulsory_GBs": gbs(c_bytes, call_ms),
            "compulsory_frac": frac(c_bytes, call_ms),
            "no_reuse_model_bytes": f_bytes,
            "no_reuse_model_GBs": gbs(f_bytes, call_ms),
        }

    line = {
        "metric": "query-tokens/sec for Z-order top-k attn fwd; % of HBM roofline",
        "value": per_s(tokens, fwd["ms_per_step"]) if fwd else None,
        "unit": "query-tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": fwd["ms_per_step"] if fwd else None,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {
            "workload": f"{w.name}: B={w.B} H={w.H} N={w.N} d_k={w.dk} d_v={w.dv} k={w.topk} {w.dtype} "
                        f"{w.bits} bits/axis {'causal' if causal else 'non-causal'}",
            "global_batch": w.B,
            "seq_len": w.N,
            "parallelism": "none (1 GPU)",
        },
        "roofline": roofline,
        "step": None if fwd is None else {
            "median_ms": fwd["median_ms"],
            "cold_median_ms": fwd["cold_median_ms"],
            "cold_value": per_s(tokens, fwd["cold_median_ms"]),
            "stages_median_ms": fwd["stages"],
            "sort_and_order_share": (fwd["stages"]["sort_ms"] + fwd["stages"]["query_order_ms"]) / fwd["median_ms"],
            "algorithmic_bytes": s_bytes,
            "no_reuse_model_frac": frac(s_bytes, fwd["ms_per_step"]),
            "compulsory_frac": frac(c_bytes, fwd["ms_per_step"]),
            "copy_1GiB_GBs": fwd["copy_GBs"],
        },
        "four_call_path": None if fwd is None else {
            "ms_per_step": fwd["four_ms"],
            "value": per_s(tokens, fwd["four_ms"]),
            "select_ms": fwd["select_ms"],
            "attend_ms": fwd["attend_ms"],
            "attend_no_reuse_model_GBs": gbs(attend_bytes(w, causal), fwd["attend_ms"]),
        },
        "backward": {
            "ms": bwd_ms,
            "no_reuse_model_bytes": b_bytes,
            "no_reuse_model_GBs": gbs(b_bytes, bwd_ms),
            "one_pass_ms": one_bwd_ms,
            "one_pass_no_reuse_model_GBs": gbs(b_bytes, one_bwd_ms),
            "forward_backward_ms": (fwd["ms_per_step"] + one_bwd_ms) if (fwd and one_bwd_ms) else None,
        },
        "history_mean": {
            "step_ms": hist_step_ms,
            "value": per_s(tokens, hist_step_ms),
            "select_attend_ms": hist_fused_ms,
            "means_ms": hist_ms,
            "means_algorithmic_bytes": h_bytes,
            "means_GBs": gbs(h_bytes, hist_ms),
            "means_frac": frac(h_bytes, hist_ms),
            "backward_ms": hist_bwd_ms,
            "one_pass_backward_ms": hist_one_bwd_ms,
        },
        "locality": locality,
        "variants": variants,
        "query_rows_per_s": per_s(w.segments * w.N, fwd["ms_per_step"]) if fwd else None,
        "timed_wall_s": fwd["wall"] if fwd else None,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
