#!/usr/bin/env python3
"""Throughput of the batched tree-CRF hot path on one MI355X.

One step = one pass of the whole path over the batch: inside (log Z), span
marginals (the derivative of log Z, as inside x outside) and CKY decode
(1-best trees), in one fused launch.  Inputs are resident in HBM before
timing starts.  Prints one JSON line.

  python bench.py [--steps K] [--warmup W] [--workload mixed] [--no-cpu-baseline]

Roofline: the hot path is one launch (parse_kernel: inside + marginal and CKY
workgroups side by side).  It is bound by plain vector-ALU work and by the
dependency chain of width steps, not by HBM and not by MFMA.  Algorithmic work
per sentence of n words, with T(n) = (n+1)n(n-1)/6 split points and
P(n) = n(n+1)/2 spans, in VALU issue slots, counting the marginals as a
reverse-mode pass (the cheaper formulation; the kernel's outside pass does
more).  Per split: inside 1 exp + 4 VALU, reverse 1 exp + 4 VALU, CKY 3 VALU;
per span: inside 1 log + 2, reverse 2, CKY 1.  Labelled scores add, per span
and label, 1 exp + 3 (label log-sum-exp) and 1 exp + 2 (per-label marginal).
A transcendental is priced two ways:
  frac                     4 slots (the scope document's op model, quarter rate)
  frac_measured_trans_rate 2 slots (v_exp_f32 / v_log_f32 measured at half the
                           fp32 add rate on gfx950 and not co-issued; see
                           --ceilings and profiles/ceilings_gfx950.txt)
Peak = 256 CUs x 64 lanes x 2.4 GHz = 39.32 T lane-slots/s.

  python bench.py --ceilings   measures the ceilings the model rests on
                               (fp32 add / FMA, fp64 add, exp2, log2, exp2 with
                               independent adds, LDS reads, barrier round trip)
                               with the microbenchmark kernels of
                               libcrfceilings.so and prints one JSON line.
"""
import argparse
import ctypes
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_SLOTS = 256 * 64 * 2.4e9   # VALU lane-slots per second
HBM_PEAK = 8.0e12               # bytes per second
# HBM bytes per launch of the timed kernel from rocprofv3 FETCH_SIZE /
# WRITE_SIZE, each scaled by the same counter on a plain copy of known size,
# keyed by workload and by the sources they were taken on (source_sha16:
# kernels, shared constants, plan): reported only while those are unchanged
# (else null).  `profile` names the committed
# summary that holds the counters and the scaling.
MEASURED_TRAFFIC = {
    "mixed": {"bytes": 73.94e6, "source_sha16": "344d6a0b90f8641c",
              "profile": "profiles/parse_kernel_mixed5000.txt"},
    "longer": {"bytes": 32.44e6, "source_sha16": "344d6a0b90f8641c",
               "profile": "profiles/parse_kernel_longer2000.txt"},
    "labeled": {"bytes": 118.57e6, "source_sha16": "344d6a0b90f8641c",
                "profile": "profiles/inside_kernel_labeled1000.txt"},
    "stress": {"bytes": 4706.67e6, "source_sha16": "344d6a0b90f8641c",
               "profile": "profiles/spill_kernels_stress64.txt"},
}
METRIC = "sentences/sec for inside fwd+bwd and CKY decode; % of binding roofline"


def work_model(lengths, labels=1, trans_slots=4):
    """Algorithmic VALU issue slots and HBM bytes of one pass (see the module
    docstring), with a transcendental priced at trans_slots."""
    n = lengths.astype(np.int64)
    T = int(((n + 1) * n * (n - 1) // 6).sum())
    P = int((n * (n + 1) // 2).sum())
    e = trans_slots
    slots_inside = (e + 4) * T + (e + 2) * P + (e + 4) * T + 2 * P
    if labels > 1:
        slots_inside += P * labels * ((e + 3) + (e + 2))
    slots_cky = 3 * T + P
    bytes_inside = 4 * P * labels * 2 + 4 * len(n)      # scores in, marginals out, logZ
    bytes_cky = 4 * P + 8 * int((2 * n - 1).sum()) + 4 * len(n)
    return dict(T=T, P=P, slots_inside=int(slots_inside), slots_cky=int(slots_cky),
                bytes_inside=int(bytes_inside), bytes_cky=int(bytes_cky))


def strip_comments(src):
    """C++ source without its comments and with runs of whitespace collapsed
    (string and character literals kept as they are)."""
    out, i, n = [], 0, len(src)
    while i < n:
        c = src[i]
        if c in "\"'":
            j = i + 1
            while j < n and src[j] != c:
                j += 2 if src[j] == "\\" else 1
            out.append(src[i:j + 1])
            i = j + 1
        elif src.startswith("//", i):
            j = src.find("\n", i)
            i = n if j < 0 else j
        elif src.startswith("/*", i):
            j = src.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def source_sha16():
    """Hash of the code (comments and layout aside) that decides what the CRF
    kernels do: the kernels, the shared constants and records, and the plan
    that lays out the launches."""
    import hashlib

    h = hashlib.sha256()
    for name in ("crf_kernels.hip", "crf_internal.h", "crf_plan.cpp"):
        with open(os.path.join(ROOT, "paper_2008_03736_amd", "csrc", name), encoding="utf-8") as f:
            h.update(strip_comments(f.read()).encode())
    return h.hexdigest()[:16]


def measured_traffic(workload):
    m = MEASURED_TRAFFIC.get(workload)
    if m is None or m["source_sha16"] != source_sha16():
        return None, None
    return m["bytes"], m["profile"]


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def oracle_rate(batch, threads, budget_s):
    """Sentences/s of the float64 oracle (marginals by the reverse-mode
    adjoint, then CKY) over whole passes of the batch, or over a prefix of it
    when one pass would take much longer than the budget."""
    from oracle import oracle as orc

    out = np.empty((batch.B, batch.n1, batch.n1), np.float64)
    orc.marginals(batch.scores[:8], batch.lengths[:8], threads=1)   # load / build
    # size the sample from a first timed chunk
    k = min(batch.B, 64)
    t0 = time.perf_counter()
    orc.marginals(batch.scores[:k], batch.lengths[:k], threads=threads, out=out[:k])
    orc.cky(batch.scores[:k], batch.lengths[:k], threads=threads)
    per = (time.perf_counter() - t0) / k
    m = int(min(batch.B, max(k, budget_s / max(per, 1e-9))))
    done, t0 = 0, time.perf_counter()
    while True:
        orc.marginals(batch.scores[:m], batch.lengths[:m], threads=threads, out=out[:m])
        orc.cky(batch.scores[:m], batch.lengths[:m], threads=threads)
        done += m
        el = time.perf_counter() - t0
        if el >= budget_s:
            break
    passes = done / batch.B
    what = (f"{done // m} passes over the whole {batch.name} batch ({batch.B} sentences)" if m == batch.B
            else f"{done // m} passes over its first {m} of {batch.B} sentences")
    return done / el, f"{what}: float64 marginals (reverse-mode) + CKY, {el:.1f} s, {threads} thread(s)", passes


def cpu_baseline(batch, threads, budget_s=10.0):
    """The oracle as it stands, timed on the host cores: all-core (threads)
    and single-threaded."""
    v_all, s_all, _ = oracle_rate(batch, threads, budget_s)
    v_one, s_one, _ = oracle_rate(batch, 1, budget_s)
    return {"value": round(v_all, 1), "unit": "sentences/s", "cores": threads, "kind": "oracle",
            "sample": s_all, "cpu_model": cpu_model(), "nproc": os.cpu_count(),
            "single_thread": {"value": round(v_one, 1), "cores": 1, "sample": s_one}}


def stats_ms(samples):
    a = np.asarray(samples, np.float64)
    return {"mean": round(float(a.mean()), 5), "median": round(float(np.median(a)), 5),
            "p10": round(float(np.percentile(a, 10)), 5), "p90": round(float(np.percentile(a, 90)), 5),
            "n": int(a.size)}


BF16_PEAK = 2.5e15   # dense bf16 MFMA FLOP/s


def bench_biaffine(torch, B, batch, dev, reps, d=500):
    """The biaffine span scorer (Eq. biaffine) that produces this batch's
    scores from boundary representations of the paper's size, d = 500: median
    launch time and MFMA roofline.  Algorithmic FLOPs per sentence of n words:
    the n left rows' [r^l;1]^T W (2 n (d+1) d) and the valid cells' inner
    products (2 d n(n+1)/2).  Inputs: seeded N(0,1) representations, W of sd
    2/d (scores of sd ~2, as the batch's), bf16."""
    g = torch.Generator(device=dev)
    g.manual_seed(0)
    shape = (batch.B, batch.n1, d)
    rl = torch.randn(shape, generator=g, device=dev).to(torch.bfloat16).view(torch.int16)
    rr = torch.randn(shape, generator=g, device=dev).to(torch.bfloat16).view(torch.int16)
    ldw = (d + 1 + 3) // 4 * 4
    w = (torch.randn((1, d, ldw), generator=g, device=dev) * (2.0 / d)).to(torch.bfloat16).view(torch.int16)
    scores = torch.empty((batch.B, batch.n1, batch.n1), dtype=torch.float32, device=dev)
    with B.Plan(batch.lengths, n1=batch.n1, device=dev) as plan:
        fn = lambda: plan.biaffine_scores(rl, rr, w, scores=scores)
        fn()
        torch.cuda.synchronize()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        for a, b in evs:
            a.record()
            fn()
            b.record()
        torch.cuda.synchronize()
        t = stats_ms([a.elapsed_time(b) for a, b in evs])
    n = batch.lengths.astype(np.int64)
    flops = int((2 * n * (d + 1) * d + d * n * (n + 1)).sum())
    ach = flops / (t["mean"] * 1e-3)
    return {"entry": "crf_biaffine_scores", "d": d, "launch_ms": t,
            "sentences_per_s": round(batch.B / (t["median"] * 1e-3), 1),
            "roofline": {"bound": "mfma", "achieved": round(ach / 1e12, 2), "peak": BF16_PEAK / 1e12,
                         "unit": "TFLOP/s", "frac": round(ach / BF16_PEAK, 4), "algorithmic_flops": flops}}


def run_ceilings():
    """Microbenchmarked ceilings of gfx950 (lane-operations per second)."""
    import torch

    from paper_2008_03736_amd import ceilings as C

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    res = C.measure_all(torch, dev)
    line = {"metric": "gfx950 ceilings", "peak_lane_slots_per_s": PEAK_SLOTS, "ceilings": res}
    print(json.dumps(line), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--launches", type=int, default=100,
                    help="per-launch event-timed launches for median/p10/p90 (at least 100)")
    ap.add_argument("--workload", default="mixed")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-threads", type=int, default=min(16, os.cpu_count() or 1))
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="after timing, run a plain device copy of this many MiB a few times "
                         "(a known-size kernel to scale HBM counters by)")
    ap.add_argument("--ceilings", action="store_true", help="measure the ALU / LDS ceilings and exit")
    ap.add_argument("--profile", choices=["parse", "fwd_bwd", "cky", "mbr", "loss", "lcky", "label_spans", "biaffine"],
                    help="launch only this entry point (warmup + steps launches, then exit): the program "
                         "that rocprofv3 summaries under profiles/ are taken on")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: runs on one GPU only (asked for --gpus {args.gpus}); sentences are "
              "independent, so more GPUs would each take a share of the batch by sentence",
              file=sys.stderr)
        sys.exit(2)
    if args.ceilings:
        run_ceilings()
        return

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

    def mbr():
        rc = lib.crf_mbr_decode(h, a_scores, a_logz, a_marg, a_spans, a_best, sp)
        if rc:
            raise B.CrfError(rc, "crf_mbr_decode")

    # gold trees for the loss: right-branching (any tree will do for timing)
    gold_np = np.full((batch.B, R, 2), -1, np.int32)
    for bi, nn in enumerate(batch.lengths):
        nn = int(nn)
        rows = [(i, nn) for i in range(nn - 1)]
        g2 = np.empty((2 * nn - 1, 2), np.int32)
        g2[0:2 * nn - 2:2] = rows
        g2[1:2 * nn - 2:2] = [(i, i + 1) for i in range(nn - 1)]
        g2[2 * nn - 2] = (nn - 1, nn)
        gold_np[bi, :2 * nn - 1] = g2
    gold = torch.from_numpy(gold_np).to(dev)
    labels_out = torch.empty((batch.B, R), dtype=torch.int32, device=dev)
    a_gold, a_labels = P(gold.data_ptr()), P(labels_out.data_ptr())

    def loss():
        rc = lib.crf_gold_loss(h, a_scores, a_gold, None, a_logz, a_marg, sp)
        if rc:
            raise B.CrfError(rc, "crf_gold_loss")

    def lcky():
        rc = lib.crf_cky_decode_labeled(h, a_scores, a_spans, a_labels, a_best, sp)
        if rc:
            raise B.CrfError(rc, "crf_cky_decode_labeled")

    def label_spans():
        rc = lib.crf_label_spans(h, a_scores, labels, a_spans, a_labels, sp)
        if rc:
            raise B.CrfError(rc, "crf_label_spans")

    step = parse if decode else fwd_bwd
    passes = {"parse": parse, "fwd_bwd": fwd_bwd, "cky": cky, "mbr": mbr, "loss": loss, "lcky": lcky,
              "label_spans": label_spans}
    if args.profile == "biaffine":
        bench_biaffine(torch, B, batch, dev, args.warmup + args.steps)
        print(json.dumps({"profile": "biaffine", "workload": batch.name}), flush=True)
        return
    if args.profile is not None:
        if args.profile == "label_spans":
            lcky()                       # spans to label
        fn = passes[args.profile]
        for _ in range(args.warmup + args.steps):
            fn()
        torch.cuda.synchronize()
        print(json.dumps({"profile": args.profile, "workload": batch.name, "launches": args.warmup + args.steps,
                          "warmup": args.warmup}), flush=True)
        if args.copy_mib > 0:
            src = torch.empty(args.copy_mib << 18, dtype=torch.float32, device=dev).fill_(1.0)
            dst = torch.empty_like(src)
            for _ in range(3):
                dst.copy_(src)
            torch.cuda.synchronize()
        plan.close()
        return

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

    # Labelled scores (877 MB padded, 38.6 MB valid) would otherwise be served
    # from the 256 MB Infinity Cache between launches: the timed launches
    # rotate over 8 copies of them (309 MB of valid cells), so that each one
    # reads a copy the cache no longer holds, and each event pair brackets the
    # launch alone.  (A 512 MiB fill between launches instead left the cache
    # full of dirty lines, whose write-back the next launch paid for.)
    copies = None if decode else [scores] + [scores.clone() for _ in range(7)]

    # Per-launch durations, one event pair per launch on the launch stream.
    def per_launch(fn, reps):
        nonlocal a_scores
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(reps)]
        for r, (a, b) in enumerate(evs):
            if copies is not None:
                a_scores = P(copies[r % len(copies)].data_ptr())
            a.record(stream)
            fn()
            b.record(stream)
        torch.cuda.synchronize()
        a_scores = P(scores.data_ptr())
        return stats_ms([a.elapsed_time(b) for a, b in evs])

    reps = max(100, args.launches)
    t_step = per_launch(step, reps)
    t_inside = per_launch(fwd_bwd, reps) if decode else t_step
    t_cky = per_launch(cky, reps) if decode else None
    # the other entry points on the same batch (median launch, microseconds)
    others = ["mbr", "loss"] if decode else ["lcky"]
    t_other = {k: per_launch(passes[k], reps) for k in others}

    # The longest sentence alone: the dependency chain no batch can beat.
    longest = int(np.argmax(batch.lengths))
    one = W.subset(batch, [longest])
    s1 = torch.from_numpy(one.scores).to(dev)
    plan1 = B.Plan(one.lengths, n1=one.n1, num_labels=labels, device=dev)
    if decode:
        t_one = per_launch(lambda: plan1.parse(s1), reps)
    else:
        t_one = per_launch(lambda: plan1.inside_fwd_bwd(s1), reps)
    plan1.close()

    def slots_of(trans):
        wm = work_model(batch.lengths, labels, trans)
        return wm, wm["slots_inside"] + (wm["slots_cky"] if decode else 0)

    wm, slots = slots_of(4)
    _, slots2 = slots_of(2)
    hbm = wm["bytes_inside"] + (wm["bytes_cky"] if decode else 0)
    avg_s = t_step["mean"] * 1e-3
    ach = slots / avg_s
    traffic, traffic_src = measured_traffic(batch.name)
    roof = {"bound": "alu",
            "kernel": "parse_kernel (inside + marginals + CKY, one launch)" if decode
            else "inside_kernel (inside + marginals)",
            "achieved": round(ach / 1e12, 4), "peak": round(PEAK_SLOTS / 1e12, 3),
            "unit": "T VALU lane-slots/s", "frac": round(ach / PEAK_SLOTS, 5),
            "frac_measured_trans_rate": round(slots2 / avg_s / PEAK_SLOTS, 5),
            "traffic": traffic, "traffic_profile": traffic_src,
            "avg_ms": t_step["mean"], "launch_ms": t_step,
            "algorithmic_slots": int(slots), "algorithmic_slots_trans2": int(slots2),
            "algorithmic_bytes": int(hbm),
            "hbm_frac": round(hbm / avg_s / HBM_PEAK, 5),
            "latency_floor_ms": t_one["median"],
            "latency_floor": f"the longest sentence (n={int(one.lengths[0])}) alone"}
    if copies is not None:
        roof["mall"] = "defeated: timed launches rotate over 8 copies of the scores"
    extra = {"fwd_bwd_ms": t_inside,
             "fwd_bwd_sentences_per_s": round(batch.B / (t_inside["median"] * 1e-3), 1)}
    if decode:
        extra["decode_ms"] = t_cky
        extra["decode_sentences_per_s"] = round(batch.B / (t_cky["median"] * 1e-3), 1)
    names = {"mbr": "mbr_decode", "loss": "gold_loss", "lcky": "labeled_decode"}
    for k, t in t_other.items():
        extra[names[k] + "_ms"] = t
        extra[names[k] + "_sentences_per_s"] = round(batch.B / (t["median"] * 1e-3), 1)

    extra["biaffine_scorer"] = bench_biaffine(torch, B, batch, dev, reps) if decode else None

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
