#!/usr/bin/env python3
"""Throughput of the batched tree-CRF hot path on one MI355X.

One step = one pass of the whole path over the batch: inside (log Z), span
marginals (the derivative of log Z, as inside x outside) and CKY decode
(1-best trees), in one fused launch.  Inputs are resident in HBM before timing starts.  Prints one JSON
line.

  python bench.py [--steps K] [--warmup W] [--workload mixed] [--no-cpu-baseline]

Roofline: the hot path is one launch (parse_kernel: inside + marginal and CKY
workgroups side by side).  It is bound by plain vector-ALU work and by the
dependency chain of width steps, not by HBM and not by MFMA.  Algorithmic work
per sentence of n words, with T(n) = (n+1)n(n-1)/6 split points and
P(n) = n(n+1)/2 spans, in VALU issue slots (a transcendental v_exp/v_log/v_rcp
costs 2 slots, as measured on gfx950), counting the marginals as a reverse-mode
pass (the cheaper formulation; the kernel's outside pass does more):
  inside   per split: add, max, sub, exp, add          = 6
           per span:  log, 2 adds                      = 4
  reverse  per split: sub, exp, mul, 2 adds            = 6
           per span:  add, rcp                         = 2
  CKY      per split: add, compare, select             = 3
           per span:  add                              = 1
Peak = 256 CUs x 64 lanes x 2.4 GHz = 39.32 T lane-slots/s.
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
# HBM bytes per launch of the timed kernel from rocprofv3 FETCH_SIZE / WRITE_SIZE,
# scaled by the same counters on a plain copy of known size, keyed by workload
# and by the kernel source they were taken on (reported only while it matches).
MEASURED_TRAFFIC = {"mixed": (76.01e6, "dd5a193d65ff39e9")}
METRIC = "sentences/sec for inside fwd+bwd and CKY decode; % of binding roofline"


def work_model(lengths, labels=1):
    n = lengths.astype(np.int64)
    T = (n + 1) * n * (n - 1) // 6
    P = n * (n + 1) // 2
    slots_inside = 12 * T.sum() + 6 * P.sum()
    if labels > 1:   # label log-sum-exp and per-label marginals: (exp + 3) + (exp + 2) per label
        slots_inside += P.sum() * labels * (2 + 3 + 2 + 2)
    slots_cky = 3 * T.sum() + P.sum()
    bytes_inside = 4 * P.sum() * labels * 2 + 4 * len(n)      # scores in, marginals out, logZ
    bytes_cky = 4 * P.sum() + 8 * (2 * n - 1).sum() + 4 * len(n)
    return dict(T=int(T.sum()), P=int(P.sum()), slots_inside=int(slots_inside),
                slots_cky=int(slots_cky), bytes_inside=int(bytes_inside), bytes_cky=int(bytes_cky))


def measured_traffic(workload):
    import hashlib

    if workload not in MEASURED_TRAFFIC:
        return None
    nbytes, digest = MEASURED_TRAFFIC[workload]
    src = os.path.join(ROOT, "paper_2008_03736_amd", "csrc", "crf_kernels.hip")
    with open(src, "rb") as f:
        now = hashlib.sha256(f.read()).hexdigest()[:16]
    return nbytes if now == digest else None


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
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="after timing, run a plain device copy of this many MiB a few times "
                         "(a known-size kernel to scale HBM counters by)")
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

    def parse():
        rc = lib.crf_inside_fwd_bwd_cky(h, a_scores, None, a_logz, a_marg, a_spans, a_best, sp)
        if rc:
            raise B.CrfError(rc, "crf_inside_fwd_bwd_cky")

    step = parse if decode else fwd_bwd

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

    # Per-launch durations, one event pair per launch on the launch stream.
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
    t_step = per_launch_ms(step, reps)
    t_inside = per_launch_ms(fwd_bwd, reps)
    t_cky = per_launch_ms(cky, reps) if decode else None

    # The longest sentence alone: the dependency chain no batch can beat.
    longest = int(np.argmax(batch.lengths))
    one = W.subset(batch, [longest])
    s1 = torch.from_numpy(one.scores).to(dev)
    plan1 = B.Plan(one.lengths, n1=one.n1, num_labels=labels, device=dev)
    if decode:
        t_one = per_launch_ms(lambda: plan1.parse(s1), reps)
    else:
        t_one = per_launch_ms(lambda: plan1.inside_fwd_bwd(s1), reps)
    plan1.close()

    wm = work_model(batch.lengths, labels)
    slots = wm["slots_inside"] + (wm["slots_cky"] if decode else 0)
    hbm = wm["bytes_inside"] + (wm["bytes_cky"] if decode else 0)
    ach = slots / (t_step * 1e-3)
    roof = {"bound": "alu",
            "kernel": "parse_kernel (inside + marginals + CKY, one launch)" if decode else "inside_kernel (inside + marginals)",
            "achieved": round(ach / 1e12, 4), "peak": round(PEAK_SLOTS / 1e12, 3),
            "unit": "T VALU lane-slots/s", "frac": round(ach / PEAK_SLOTS, 5),
            "traffic": measured_traffic(batch.name) if decode else None, "avg_ms": round(t_step, 4),
            "algorithmic_slots": int(slots), "algorithmic_bytes": int(hbm),
            "hbm_frac": round(hbm / (t_step * 1e-3) / HBM_PEAK, 5),
            "latency_floor_ms": round(t_one, 4),
            "latency_floor": f"the longest sentence (n={int(one.lengths[0])}) alone"}
    extra = {"fwd_bwd_ms": round(t_inside, 4),
             "fwd_bwd_sentences_per_s": round(batch.B / (t_inside * 1e-3), 1)}
    if decode:
        extra["decode_ms"] = round(t_cky, 4)
        extra["decode_sentences_per_s"] = round(batch.B / (t_cky * 1e-3), 1)

    if args.copy_mib > 0:
        src = torch.empty(args.copy_mib << 18, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

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
