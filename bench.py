#!/usr/bin/env python3
"""Throughput of the batched tree-CRF hot path on one MI355X.

One step = one pass of the whole path over the batch: inside forward (log Z)
+ reverse pass (span marginals) in one fused call, then CKY decode (1-best
trees).  Inputs are resident in HBM before timing starts.  Prints one JSON
line.

  python bench.py [--steps K] [--warmup W] [--workload mixed] [--no-cpu-baseline]

Roofline: the dominant kernel is the fused inside+reverse kernel; it is bound
by plain vector-ALU work (log-sum-exp over split points), not HBM and not
MFMA.  Its algorithmic work per sentence of n words, with T(n) = (n+1)n(n-1)/6
split points and P(n) = n(n+1)/2 spans:
  forward  per split 1 exp + 4 VALU, per span 1 log + 2 VALU
  reverse  per split 1 exp + 4 VALU, per span 2 VALU
counting a transcendental as 4 issue slots (quarter rate), i.e. 16 slots per
split and 8 per span.  Peak = 256 CUs x 64 lanes x 2.4 GHz = 39.32 T lane
slots/s.  CKY: 3 slots per split (add, compare, select) and 1 per span.
"""
import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_SLOTS = 256 * 64 * 2.4e9   # VALU lane-slots per second
HBM_PEAK = 8.0e12               # bytes per second
METRIC = "sentences/sec for inside fwd+bwd and CKY decode; % of binding roofline"


def work_model(lengths, labels=1):
    n = lengths.astype(np.int64)
    T = (n + 1) * n * (n - 1) // 6
    P = n * (n + 1) // 2
    slots_inside = 16 * T.sum() + 8 * P.sum()
    if labels > 1:   # label log-sum-exp and per-label marginals: (exp + 3) + (exp + 2) per label
        slots_inside += P.sum() * labels * (4 + 3 + 4 + 2)
    slots_cky = 3 * T.sum() + P.sum()
    bytes_inside = 4 * P.sum() * labels * 2 + 4 * len(n)      # scores in, marginals out, logZ
    bytes_cky = 4 * P.sum() + 8 * (2 * n - 1).sum() + 4 * len(n)
    return dict(T=int(T.sum()), P=int(P.sum()), slots_inside=int(slots_inside),
                slots_cky=int(slots_cky), bytes_inside=int(bytes_inside), bytes_cky=int(bytes_cky))


def cpu_baseline(batch, threads, budget_s=12.0):
    """The float64 oracle (marginals + CKY) on the host, repeated over the
    workload until about budget_s seconds have been spent."""
    from oracle import oracle as orc

    out = np.empty((batch.B, batch.n1, batch.n1), np.float64)
    orc.marginals(batch.scores[:8], batch.lengths[:8], threads=1)   # load / build
    done, t0 = 0, time.perf_counter()
    while True:
        orc.marginals(batch.scores, batch.lengths, threads=threads, out=out)
        orc.cky(batch.scores, batch.lengths, threads=threads)
        done += batch.B
        el = time.perf_counter() - t0
        if el >= budget_s:
            break
    return {"value": round(done / el, 1), "unit": "sentences/s", "cores": threads,
            "kind": "oracle",
            "sample": f"whole {batch.name} batch ({batch.B} sentences) x {done // batch.B} passes "
                      f"of float64 marginals (reverse-mode) + CKY, {el:.1f} s, {threads} threads"}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="mixed")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-threads", type=int, default=min(16, os.cpu_count() or 1))
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU only (asked for --gpus {args.gpus}); "
              "sentences are independent and would be sharded by sentence, see DESIGN.md",
              file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2008_03736_amd import binding as B
    from paper_2008_03736_amd import workloads as W

    lib = B.load()
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    batch = W.make(args.workload, seed=args.seed)
    labels = batch.num_labels
    scores = torch.from_numpy(batch.scores).to(dev)
    plan = B.Plan(batch.lengths, n1=batch.n1, num_labels=labels, device=dev)
    logZ = torch.empty(batch.B, dtype=torch.float32, device=dev)
    marg = torch.zeros_like(scores)
    R = 2 * (batch.n1 - 1) - 1
    spans = torch.empty((batch.B, R, 2), dtype=torch.int32, device=dev)
    best = torch.empty(batch.B, dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream(dev)
    sp = ctypes.c_void_p(stream.cuda_stream)
    h = plan._handle
    P = ctypes.c_void_p
    a_scores, a_logz, a_marg = P(scores.data_ptr()), P(logZ.data_ptr()), P(marg.data_ptr())
    a_spans, a_best = P(spans.data_ptr()), P(best.data_ptr())
    decode = labels == 1

    def fwd_bwd():
        rc = lib.crf_inside_fwd_bwd(h, a_scores, None, a_logz, a_marg, sp)
        if rc:
            raise B.CrfError(rc, "crf_inside_fwd_bwd")

    def cky():
        rc = lib.crf_cky_decode(h, a_scores, a_spans, a_best, sp)
        if rc:
            raise B.CrfError(rc, "crf_cky_decode")

    def step():
        fwd_bwd()
        if decode:
            cky()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms_per_step = e0.elapsed_time(e1) / args.steps

    # Per-kernel durations, one event pair per launch on the launch stream.
    def per_launch_ms(fn, reps):
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(reps)]
        for a, b in evs:
            a.record(stream)
            fn()
            b.record(stream)
        torch.cuda.synchronize()
        return float(np.mean([a.elapsed_time(b) for a, b in evs]))

    reps = max(10, args.steps)
    t_inside = per_launch_ms(fwd_bwd, reps)
    t_cky = per_launch_ms(cky, reps) if decode else None

    wm = work_model(batch.lengths, labels)
    ach = wm["slots_inside"] / (t_inside * 1e-3)
    roof = {"bound": "alu", "kernel": "inside_kernel<rev=1> (fused inside + reverse)",
            "achieved": round(ach / 1e12, 3), "peak": round(PEAK_SLOTS / 1e12, 3),
            "unit": "T VALU lane-slots/s", "frac": round(ach / PEAK_SLOTS, 4),
            "traffic": None, "avg_ms": round(t_inside, 4),
            "algorithmic_slots": wm["slots_inside"], "algorithmic_bytes": wm["bytes_inside"],
            "hbm_frac": round(wm["bytes_inside"] / (t_inside * 1e-3) / HBM_PEAK, 4)}
    extra = {}
    if decode:
        ach_c = wm["slots_cky"] / (t_cky * 1e-3)
        extra["decode"] = {"bound": "alu", "kernel": "cky_kernel (float64 chart)",
                           "avg_ms": round(t_cky, 4), "achieved": round(ach_c / 1e12, 3),
                           "peak": round(PEAK_SLOTS / 1e12, 3), "frac": round(ach_c / PEAK_SLOTS, 4),
                           "sentences_per_s": round(batch.B / (t_cky * 1e-3), 1)}
    extra["fwd_bwd_sentences_per_s"] = round(batch.B / (t_inside * 1e-3), 1)

    cb = None if args.no_cpu_baseline else cpu_baseline(batch, args.cpu_threads)
    info = plan.info
    n = batch.lengths
    line = {
        "metric": METRIC,
        "value": round(batch.B / (ms_per_step * 1e-3), 1),
        "unit": "sentences/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32 (CKY chart f64)",
        "data": "synthetic",
        "config": {"workload": batch.name, "sentences": batch.B, "max_len": int(n.max()),
                   "mean_len": round(float(n.mean()), 2), "labels": labels, "seed": args.seed,
                   "passes": "fwd+bwd+decode" if decode else "fwd+bwd",
                   "lds_sentences": info["lds_count"], "spill_sentences": info["spill_count"]},
        "roofline": roof,
        "cpu_baseline": cb,
        **extra,
    }
    plan.close()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
