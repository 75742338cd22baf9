"""Benchmark of the Z-order top-k attention forward on one MI355X.

One step is the whole forward (encode, sort of the query and key codes, the
processing order, then select and attend in one pass: C ABI calls on one
stream) over one batch of the long-context workload (B=1, H=16,
N=65536, d_k=3, d_v=128, k=128, bf16, 6 bits per axis, causal), with inputs,
outputs and workspace resident in HBM before timing starts.

Prints one JSON line: query-tokens/s (B*N per second) of the whole step, the
dominant kernel's achieved algorithmic bandwidth against the HBM peak (timed
with HIP events on the stream it runs on), the same step through the separate
select and attend calls, and the CPU oracle timed on a bounded sample of the
same workload on the host's cores.
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
KERNEL_SRCS = [os.path.join(ROOT, "paper_2501_14577_amd", "csrc", n)
               for n in ("fused.hip", "tile.hip", "tile_device.h", "select.hip", "select_device.h", "attend_device.h",
                         "device_common.h", "layout.h")]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "select_attend_long_context_traffic.txt")


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


def step_bytes(w: workloads.Workload, causal: bool) -> int:
    """Algorithmic bytes of the whole step: attend plus, per query row,
    encode 4*d*s + 8, sort 16 per radix pass and select 4 + 8k.  (The sort of
    the query codes, a scheduling aid, is not counted.)"""
    s, d = elem_size(w.dtype), w.dk
    passes = (w.code_bits + 7) // 8
    rows = w.segments * w.N
    return attend_bytes(w, causal) + rows * ((4 * d * s + 8) + 16 * passes + (4 + 8 * w.topk))


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


def read_traffic():
    """HBM bytes per launch of the one-pass select-and-attend kernel, from the
    committed rocprofv3 counter summary; None when absent or taken on
    different kernel sources."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    kv = {}
    for line in open(TRAFFIC_FILE):
        if ":" in line and not line.startswith("#"):
            key, val = line.split(":", 1)
            kv[key.strip()] = val.strip()
    if kv.get("kernel_source_sha256") != kernel_source_hash():
        return None
    try:
        return int(float(kv["hbm_bytes_per_launch"]))
    except (KeyError, ValueError):
        return None


def cpu_baseline(w: workloads.Workload, causal: bool, x: dict, heads: int):
    """The oracle, untuned, on the first ``heads`` (batch 0) segments: the
    whole forward of each, one after another, in one process.  Scaled to
    query-tokens/s as rows / H per second (one query token carries H rows)."""
    import oracle

    S = w.segments
    heads = max(1, min(heads, S))
    f = {n: oracle.as_f32(a, w.dtype).reshape(S, w.N, a.shape[-1])[:heads] for n, a in x.items()}
    t0 = time.perf_counter()
    oracle.forward(f["q"], f["k"], f["v"], w.topk, workloads.EPS_DEFAULT, causal, w.bits)
    dt = time.perf_counter() - t0
    rows = heads * w.N
    return {
        "value": rows / w.H / dt,
        "unit": "query-tokens/s",
        "cores": 1,
        "kind": "oracle",
        "sample": (f"{heads} of {S} segments ({rows} query rows), whole oracle forward "
                   f"({'causal' if causal else 'non-causal'}), one process, {dt:.1f} s; "
                   f"scaled as rows/H per second"),
    }


def locality_experiment(zeta, torch, dev) -> dict:
    """Section 4.4's locality measure on synthetic N(0,1) queries and keys:
    the mean share of each query's 64 exact nearest keys that its Z-order
    window of 64 holds, for N in {512, 1024, 2048} and d_k = 1..8 (16
    segments each, not causal, bits = min(24, 32 // d_k)), with queries drawn
    apart from the keys and, second reading, with the keys as their own
    queries; plus the GPU time of the exact search and of the window
    selection at N = 2048, d_k = 3."""
    table, table_self = {}, {}
    for n in (512, 1024, 2048):
        for d in range(1, 9):
            w = workloads.custom(B=1, H=16, N=n, dk=d, dtype="f32", topk=64, bits=min(24, 32 // d), seed=n * 10 + d)
            x = workloads.generate(w)
            q, k = (torch.from_numpy(x[m]).to(dev) for m in ("q", "k"))
            table[f"N={n} d_k={d}"] = round(zeta.locality_overlap(q, k, w.bits, 64), 4)
            table_self[f"N={n} d_k={d}"] = round(zeta.locality_overlap(k, k, w.bits, 64), 4)
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
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=5, help="workload number (parity cases 1-4, bench 5)")
    ap.add_argument("--noncausal", action="store_true")
    ap.add_argument("--cpu-heads", type=int, default=8,
                    help="segments in the oracle sample (0 skips the CPU baseline)")
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

    import torch

    import paper_2501_14577_amd as zeta

    if not torch.cuda.is_available():
        print("bench.py needs a ROCm GPU", file=sys.stderr)
        return 2
    zeta.load_library()
    dev = torch.device("cuda:0")
    w = workloads.CONFIGS[args.config]
    causal = not args.noncausal and True in w.causal
    x = workloads.generate(w)

    def to_dev(a):
        if w.dtype == "bf16":
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(a).to(dev)

    q, k, v = to_dev(x["q"]), to_dev(x["k"]), to_dev(x["v"])
    tdtype = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    bufs = zeta.alloc_buffers(w.B, w.H, w.N, w.dv, w.topk, tdtype, dev)
    ws = zeta.workspace_for(w.B, w.H, w.N, w.dk, w.bits, w.topk, causal, dev)
    eps = workloads.EPS_DEFAULT

    if args.copy_calibration:
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    codes, sorted2, perm2 = bufs["codes"], bufs["sorted_codes2"], bufs["perm2"]

    def step_fused(ev=None):
        # encode -> joint sort -> processing order -> select and attend in one pass
        qc, kc = zeta.zeta_morton_encode(q, k, w.bits, q_codes=codes[0], k_codes=codes[1], workspace=ws)
        zeta.zeta_sort_keys(codes, w.code_bits, sorted_codes=sorted2, perm=perm2, workspace=ws)
        order = zeta.zeta_query_order(perm2[0], w.N, w.segments, w.topk, causal, order_out=bufs["order"],
                                      workspace=ws)
        if ev is not None:
            ev[0].record()
        zeta.zeta_select_attend_fwd(q, k, v, qc, sorted2[1], perm2[1], w.topk, causal, eps, q_order=order,
                                    out=bufs["out"], workspace=ws)
        if ev is not None:
            ev[1].record()

    def step(ev=None):
        # encode -> joint sort of query and key codes -> the query Z-order
        # regrouped by list level (processing order) -> select -> attend
        qc, kc = zeta.zeta_morton_encode(q, k, w.bits, q_codes=codes[0], k_codes=codes[1], workspace=ws)
        zeta.zeta_sort_keys(codes, w.code_bits, sorted_codes=sorted2, perm=perm2, workspace=ws)
        order = zeta.zeta_query_order(perm2[0], w.N, w.segments, w.topk, causal, order_out=bufs["order"],
                                      workspace=ws)
        idx = zeta.zeta_select_topk(qc, sorted2[1], perm2[1], w.topk, causal, q_order=order, idx=bufs["idx"],
                                    workspace=ws)
        if ev is not None:
            ev[0].record()
        zeta.zeta_topk_attn_fwd(q, k, v, idx, eps, q_order=order, out=bufs["out"])
        if ev is not None:
            ev[1].record()

    def timed(fn):
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(args.steps)]
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        wall0 = time.perf_counter()
        start.record()
        for i in range(args.steps):
            fn(evs[i])
        stop.record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - wall0
        return (start.elapsed_time(stop) / args.steps, float(np.mean([a.elapsed_time(b) for a, b in evs])), wall)

    if "forward" in parts:
        four_ms, attend_ms, _ = timed(step)
        ms_per_step, fused_ms, wall = timed(step_fused)
    else:
        four_ms = attend_ms = ms_per_step = fused_ms = wall = None

    # Attention gradients (zeta_topk_attn_bwd) for the windows of the
    # four-call step, timed on their own; not part of the forward metric.
    dout = to_dev(workloads.generate_dout(w))
    f32 = dict(dtype=torch.float32, device=dev)
    gq = torch.empty((w.B, w.H, w.N, w.dk), **f32)
    gk = torch.empty_like(gq)
    gv = torch.empty((w.B, w.H, w.N, w.dv), **f32)
    geps = torch.empty(1, **f32)
    bws = zeta.bwd_workspace_for(w.B, w.H, w.N, w.dk, w.dv, w.topk, "history" in parts, dev)
    step()
    torch.cuda.synchronize()

    def bwd(ev=None):
        if ev is not None:
            ev[0].record()
        zeta.zeta_topk_attn_bwd(q, k, v, bufs["idx"], dout, eps, q_order=bufs["order"], dq=gq, dk=gk, dv=gv,
                                deps=geps, workspace=bws)
        if ev is not None:
            ev[1].record()

    b_bytes = bwd_bytes(w, causal)
    bwd_ms = timed(bwd)[0] if "backward" in parts else None

    # The one-pass call's gradients (zeta_select_attend_bwd): the same
    # windows, from the lists, without an index tensor.
    tws = zeta.select_attend_bwd_workspace_for(w.B, w.H, w.N, w.dv, w.topk, causal, dev)

    def bwd_one_pass(ev=None):
        if ev is not None:
            ev[0].record()
        zeta.zeta_select_attend_bwd(q, k, v, codes[0], sorted2[1], perm2[1], w.topk, causal, eps, dout,
                                    q_order=bufs["order"], dq=gq, dk=gk, dv=gv, deps=geps, workspace=tws)
        if ev is not None:
            ev[1].record()

    one_bwd_ms = timed(bwd_one_pass)[0] if "backward" in parts else None

    # The history-mean candidate: the means (zeta_history_mean) timed alone,
    # the one-pass step with the candidate, and the gradients with it.
    mk = torch.empty((w.B, w.H, w.N, w.dk), **f32)
    mv = torch.empty((w.B, w.H, w.N, w.dv), **f32)

    def hist_means(ev=None):
        if ev is not None:
            ev[0].record()
        zeta.zeta_history_mean(k, v, causal, mean_k=mk, mean_v=mv, workspace=ws)
        if ev is not None:
            ev[1].record()

    def step_hist(ev=None):
        qc, kc = zeta.zeta_morton_encode(q, k, w.bits, q_codes=codes[0], k_codes=codes[1], workspace=ws)
        zeta.zeta_sort_keys(codes, w.code_bits, sorted_codes=sorted2, perm=perm2, workspace=ws)
        order = zeta.zeta_query_order(perm2[0], w.N, w.segments, w.topk, causal, order_out=bufs["order"],
                                      workspace=ws)
        zeta.zeta_history_mean(k, v, causal, mean_k=mk, mean_v=mv, workspace=ws)
        if ev is not None:
            ev[0].record()
        zeta.zeta_select_attend_fwd(q, k, v, qc, sorted2[1], perm2[1], w.topk, causal, eps, q_order=order,
                                    mean_k=mk, mean_v=mv, out=bufs["out"], workspace=ws)
        if ev is not None:
            ev[1].record()

    def bwd_hist(ev=None):
        if ev is not None:
            ev[0].record()
        zeta.zeta_topk_attn_bwd(q, k, v, bufs["idx"], dout, eps, q_order=bufs["order"], mean_k=mk, mean_v=mv,
                                causal=causal, dq=gq, dk=gk, dv=gv, deps=geps, workspace=bws)
        if ev is not None:
            ev[1].record()

    hws = (zeta.select_attend_bwd_workspace_for(w.B, w.H, w.N, w.dv, w.topk, causal, dev, True)
           if "history" in parts else None)

    def bwd_hist_one_pass(ev=None):
        if ev is not None:
            ev[0].record()
        zeta.zeta_select_attend_bwd(q, k, v, codes[0], sorted2[1], perm2[1], w.topk, causal, eps, dout,
                                    q_order=bufs["order"], mean_k=mk, mean_v=mv, dq=gq, dk=gk, dv=gv, deps=geps,
                                    workspace=hws)
        if ev is not None:
            ev[1].record()

    # Variants: the paper's chunked causal rule with 32 chunks (the one-pass
    # step), and each score variant's one-pass call (per-query kernels).
    variants = None
    if "variants" in parts:
        chunk = w.N // 32

        def step_chunked(ev=None):
            qc, kc = zeta.zeta_morton_encode(q, k, w.bits, q_codes=codes[0], k_codes=codes[1], workspace=ws)
            zeta.zeta_sort_keys(codes, w.code_bits, sorted_codes=sorted2, perm=perm2, workspace=ws)
            order = zeta.zeta_query_order(perm2[0], w.N, w.segments, w.topk, causal, chunk=chunk, order_out=bufs["order"],
                                          workspace=ws)
            if ev is not None:
                ev[0].record()
            zeta.zeta_select_attend_fwd(q, k, v, qc, sorted2[1], perm2[1], w.topk, causal, eps, chunk=chunk,
                                        q_order=order, out=bufs["out"], workspace=ws)
            if ev is not None:
                ev[1].record()

        chunk_step_ms, chunk_call_ms, _ = timed(step_chunked)
        step_fused()
        modes = {}
        for mode in ("dot", "neg_euclid", "inv_euclid", "norm_dot"):
            def call(ev=None, mode=mode):
                if ev is not None:
                    ev[0].record()
                zeta.zeta_select_attend_fwd(q, k, v, codes[0], sorted2[1], perm2[1], w.topk, causal, eps, score=mode,
                                            q_order=bufs["order"], out=bufs["out"], workspace=ws)
                if ev is not None:
                    ev[1].record()
            modes[mode] = timed(call)[1]
        variants = {"chunk": chunk, "chunked_step_ms": chunk_step_ms,
                    "chunked_value": w.B * w.N / (chunk_step_ms * 1e-3),
                    "chunked_select_attend_ms": chunk_call_ms, "score_select_attend_ms": modes}

    locality = locality_experiment(zeta, torch, dev) if "locality" in parts else None

    h_bytes = w.segments * w.N * (w.dk + w.dv) * (elem_size(w.dtype) + 4)  # read k, v once; write the means
    if "history" in parts:
        hist_ms = timed(hist_means)[1]
        hist_step_ms, hist_fused_ms, _ = timed(step_hist)
        hist_bwd_ms = timed(bwd_hist)[0]
        hist_one_bwd_ms = timed(bwd_hist_one_pass)[0]
    else:
        hist_ms = hist_step_ms = hist_fused_ms = hist_bwd_ms = hist_one_bwd_ms = None
    tokens = w.B * w.N
    a_bytes = attend_bytes(w, causal)
    f_bytes = a_bytes + w.segments * w.N * 4  # plus each query's code, read instead of an index row
    s_bytes = step_bytes(w, causal)
    traffic = read_traffic()

    def per_s(amount, ms):  # amount per second, None when the part was not timed
        return None if ms is None else amount / (ms * 1e-3)

    def gbs(nbytes, ms):
        r = per_s(nbytes, ms)
        return None if r is None else r / 1e9

    def frac(nbytes, ms):
        r = gbs(nbytes, ms)
        return None if r is None else r / HBM_PEAK_GBS

    achieved = gbs(f_bytes, fused_ms)

    cpu = None
    if args.cpu_heads > 0:
        cpu = cpu_baseline(w, causal, x, args.cpu_heads)

    line = {
        "metric": "query-tokens/sec for Z-order top-k attn fwd; % of HBM roofline",
        "value": per_s(tokens, ms_per_step),
        "unit": "query-tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
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
        "roofline": {
            "bound": "hbm",
            "kernel": "select_attend (one pass, 16-query matrix-core tiles)",
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": frac(f_bytes, fused_ms),
            "traffic": traffic,
            "algorithmic_bytes_per_launch": f_bytes,
            "kernel_ms": fused_ms,
            # Bytes that actually crossed HBM (calibrated counters) per second.
            "traffic_GBs": gbs(traffic, fused_ms) if traffic else None,
        },
        "four_call_path": {
            "ms_per_step": four_ms,
            "value": per_s(tokens, four_ms),
            "attend_ms": attend_ms,
            "attend_achieved_GBs": gbs(a_bytes, attend_ms),
        },
        "backward": {
            "ms": bwd_ms,
            "algorithmic_bytes": b_bytes,
            "achieved_GBs": gbs(b_bytes, bwd_ms),
            "frac": frac(b_bytes, bwd_ms),
            "one_pass_ms": one_bwd_ms,
            "one_pass_achieved_GBs": gbs(b_bytes, one_bwd_ms),
            "one_pass_frac": frac(b_bytes, one_bwd_ms),
            "forward_backward_ms": (ms_per_step + one_bwd_ms) if (ms_per_step and one_bwd_ms) else None,
        },
        "history_mean": {
            "step_ms": hist_step_ms,
            "value": per_s(tokens, hist_step_ms),
            "select_attend_ms": hist_fused_ms,
            "means_ms": hist_ms,
            "means_algorithmic_bytes": h_bytes,
            "means_achieved_GBs": gbs(h_bytes, hist_ms),
            "means_frac": frac(h_bytes, hist_ms),
            "backward_ms": hist_bwd_ms,
            "one_pass_backward_ms": hist_one_bwd_ms,
        },
        "locality": locality,
        "variants": None if variants is None else dict(
            variants, score_select_attend_GBs={m: gbs(f_bytes, t) for m, t in variants["score_select_attend_ms"].items()}),
        "step_hbm_frac": frac(s_bytes, ms_per_step),
        "step_algorithmic_bytes": s_bytes,
        "query_rows_per_s": per_s(w.segments * w.N, ms_per_step),
        "timed_wall_s": wall,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
