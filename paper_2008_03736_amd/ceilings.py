"""ctypes binding of ``libcrfceilings.so`` (``include/crf_ceilings.h``): the
gfx950 ceilings behind the CRF kernels' roofline, measured with event-timed
microbenchmark launches (measurement only; the CRF path never uses it)."""
import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libcrfceilings.so")

# kind -> (name, operations per thread and iteration, unit)
KINDS = {
    0: ("fp32_add", 16, "lane-ops/s"),
    1: ("fp32_fma", 16, "lane-ops/s"),
    2: ("exp2_f32", 8, "lane-ops/s"),
    3: ("log2_f32", 8, "lane-ops/s"),
    4: ("fp64_add", 16, "lane-ops/s"),
    5: ("exp2_with_3_adds", 8, "exp2 lane-ops/s (each beside 3 independent adds)"),
    6: ("lds_read_b32", 8, "lane-reads/s"),
    7: ("barrier_round_trip", 1, "ns per store/barrier/load step"),
}
SIGNATURES = {"crf_ceiling_run": (ctypes.c_int, [ctypes.c_int] * 4 + [ctypes.c_void_p, ctypes.c_void_p])}

_lib = None


def load(path=LIB_PATH):
    global _lib
    if _lib is None:
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is missing: build it with __graft_entry__.build()")
        lib = ctypes.CDLL(path)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def measure(torch, dev, kind, blocks=2048, threads=256, iters=4096, reps=5):
    """Best of `reps` event-timed launches; returns the rate in KINDS' unit."""
    lib = load()
    out = torch.empty(blocks * threads, dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream(dev)
    sp = ctypes.c_void_p(stream.cuda_stream)

    def launch():
        rc = lib.crf_ceiling_run(kind, blocks, threads, iters, ctypes.c_void_p(out.data_ptr()), sp)
        if rc != 0:
            raise RuntimeError(f"crf_ceiling_run({kind}) failed: {rc}")

    launch()
    torch.cuda.synchronize()
    best = None
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        launch()
        b.record(stream)
        torch.cuda.synchronize()
        ms = a.elapsed_time(b)
        best = ms if best is None else min(best, ms)
    name, ops, unit = KINDS[kind]
    if kind == 7:
        return {"name": name, "value": best * 1e6 / iters, "unit": unit, "ms": best,
                "blocks": blocks, "threads": threads, "iters": iters}
    rate = blocks * threads * iters * ops / (best * 1e-3)
    return {"name": name, "value": rate, "unit": unit, "ms": best, "blocks": blocks, "threads": threads,
            "iters": iters}


def measure_all(torch, dev):
    res = [measure(torch, dev, k) for k in range(7)]
    # latency of one sweep step's synchronisation: one workgroup per CU of
    # 512 threads (the CRF kernels' size), many round trips
    res.append(measure(torch, dev, 7, blocks=256, threads=512, iters=20000))
    peak = 256 * 64 * 2.4e9
    by = {r["name"]: r for r in res}
    add = by["fp32_add"]["value"]
    by["exp2_f32"]["slots_vs_fp32_add"] = add / by["exp2_f32"]["value"]
    by["log2_f32"]["slots_vs_fp32_add"] = add / by["log2_f32"]["value"]
    # time of 8 exp + 24 adds vs 24 adds alone, in fp32-add slots per exp
    t_mix = 1.0 / by["exp2_with_3_adds"]["value"]
    by["exp2_with_3_adds"]["slots_per_exp_beside_adds"] = t_mix * add - 3.0
    for r in res:
        if r["unit"] == "lane-ops/s":
            r["frac_of_nominal_lane_slots"] = r["value"] / peak
    return res
