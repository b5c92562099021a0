"""Benchmark of the tiled integer GEMM substrate on one MI355X.

One step = one evaluation of the packed INT16-input / INT32-accumulation GEMM
at M = N = K = 8192 (operands uniform in [-256, 255], seed 7) through a
persistent executor, with inputs resident in HBM.  Prints ONE JSON line.

The timing follows the paper's split (one-time setup / cached steady state /
execute-only): setup = executor creation; cached = host wall time of
back-to-back runs / steps; execute-only = HIP events around each launch on
the executor's stream.  `--all` also measures every other workload and writes
them to --all-out (not to stdout).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HEADLINE = "gemm_i16_8192"
METRIC = "GOPS (2·M·N·K/s) packed INT16/INT32 GEMM; conv & attention-core GOPS"

# MI355X datasheet peaks (dense)
PEAK = {"f16": 2500.0, "i8": 5000.0, "f32": 157.3, "hbm": 8000.0}  # TFLOP/s, TOP/s, GB/s

# HBM bytes per launch of the headline contraction, from two rocprofv3 counter
# passes (FETCH_SIZE, WRITE_SIZE) over this benchmark, each scaled by what the
# counter reads for a 1 GiB device copy (`--copy-calibration`).  Valid only for
# the kernel source they were taken on: the SHA-256 of the contraction
# kernel's text is compared at run time and the figure is dropped (null) if
# the kernel has changed since.
TRAFFIC = {
    "kernel": "gemm_nt_bf16_128x256",
    "kernel_sha256": "0bb74a1223cec68350a328ba966c67024fd244d9e30b741bd6387b409294faca",
    "read_bytes": 2147840000,     # FETCH_SIZE 1048750 KiB x 2.0 (copy: 524304 KiB per GiB read)
    "write_bytes": 268495872,     # WRITE_SIZE 262203 KiB x 1.0 (copy: 1048576 KiB per GiB written)
}
KERNEL_SRC = os.path.join(ROOT, "paper_2606_09905_amd", "csrc", "k_gemm_nt.hip")


def contraction_sha256():
    """SHA-256 of the fp16-exact contraction kernel's source text (its MFMA
    step helper and the k_gemm_nt template, up to the builders)."""
    import hashlib
    try:
        src = open(KERNEL_SRC).read()
        a = src.index("// One 32x32x16 MFMA step of the fp16-exact route")
        src.index("void k_gemm_nt(const GemmParams p)", a)
        b = src.index("// Builders", a)
    except (OSError, ValueError):
        return None
    return hashlib.sha256(src[a:b].encode()).hexdigest()


def traffic_bytes(kernel, launches):
    """Measured HBM bytes per launch (read + written), or None."""
    t = TRAFFIC
    if kernel != t["kernel"] or t["read_bytes"] is None or launches != 1:
        return None
    if t["kernel_sha256"] is None or contraction_sha256() != t["kernel_sha256"]:
        return None
    return t["read_bytes"] + t["write_bytes"]


def copy_calibration(torch):
    n = 1 << 28                      # 2^28 float32 = 1 GiB
    a = torch.ones(n, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    for _ in range(2):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration": "2 x 1 GiB device-to-device copies"}), flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    # the GPU needs a few tens of milliseconds of load to reach its steady
    # clocks: the default warmup covers that
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default=HEADLINE)
    ap.add_argument("--all", action="store_true", help="also measure every workload")
    ap.add_argument("--all-out", default="bench_all.json", help="where --all writes its per-workload results")
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the per-configuration measurements of the other workloads")
    ap.add_argument("--oracle-all", action="store_true",
                    help="time the CPU oracle on every workload (host only) and exit")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run two 1 GiB device-to-device copies (HBM counter calibration)")
    ap.add_argument("--cpu-rows", type=int, default=8192,
                    help="rows of A in the oracle's CPU sample of the headline GEMM")
    return ap.parse_args()


def make_executor(w, qx, route="auto"):
    d = w.dims
    if w.op == "gemm_i16i32":
        return qx.Executor.gemm_i16i32(d["M"], d["N"], d["K"], d["batch"], w.bound, w.bound, route)
    if w.op == "gemm_i32_s24":
        return qx.Executor.gemm_i32_s24(d["M"], d["N"], d["K"], d["batch"], route)
    if w.op == "conv2d":
        return qx.Executor.conv2d(d["N"], d["Ci"], d["H"], d["W"], d["Co"], d["KH"], d["KW"],
                                  d["stride"], d["pad"], w.bound, w.bound)
    if w.op in ("conv2d_f32", "conv2d_i32"):
        return qx.Executor.conv2d_t("f32" if w.op == "conv2d_f32" else "i32", d["N"], d["Ci"], d["H"], d["W"],
                                    d["Co"], d["KH"], d["KW"], d["stride"], d["pad"])
    if w.op == "lenet_i32":
        return qx.Executor.lenet_i32(d["B"])
    if w.op in ("minmax_i32", "minmax_i16"):
        return qx.Executor.minmax(d["n"], w.op[-3:])
    if w.op in ("avgpool_i32", "maxpool_f32"):
        return qx.Executor.pool2x2("avg_i32" if w.op == "avgpool_i32" else "max_f32", d["N"], d["C"], d["H"], d["W"])
    if w.op == "attn_f32":
        return qx.Executor.attn("f32", d["L"], d["d"])
    if w.op == "attn_i32":
        return qx.Executor.attn("i32", d["L"], d["d"], w.bound)
    if w.op == "sdpa_f32":
        return qx.Executor.sdpa_f32(d["BH"], d["L"], d["d"], d["scale"], bool(d["causal"]))
    raise ValueError(w.op)


def measure(w, steps, warmup, torch, qx, route="auto", inputs=None, sustain_ms=0.0):
    """Setup, cached steady state and execute-only time of one workload.
    With sustain_ms > 0 a further back-to-back loop of at least that many
    milliseconds (and 20 runs) gives the sustained-clock step time."""
    if inputs is None:
        inputs = [torch.from_numpy(np.ascontiguousarray(a)).cuda() for a in w.generate()]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ex = make_executor(w, qx, route)
    setup_ms = (time.perf_counter() - t0) * 1e3
    plan = ex.plan()
    out = torch.empty(ex.out_shape, dtype=ex.out_dtype, device="cuda")
    ptrs = [t.data_ptr() for t in inputs]
    stream = torch.cuda.current_stream()
    for _ in range(warmup):
        ex.run_ptrs(ptrs, out.data_ptr(), stream)
    torch.cuda.synchronize()
    # cached steady state: back-to-back runs, one final sync
    t0 = time.perf_counter()
    for _ in range(steps):
        ex.run_ptrs(ptrs, out.data_ptr(), stream)
    torch.cuda.synchronize()
    cached_s = (time.perf_counter() - t0) / steps
    sustained = None
    if sustain_ms > 0:
        # sized from the cached rate with a margin: sustained clocks run faster
        reps = max(20, int(np.ceil(1.3 * sustain_ms / max(cached_s * 1e3, 1e-3))))
        t0 = time.perf_counter()
        for _ in range(reps):
            ex.run_ptrs(ptrs, out.data_ptr(), stream)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        sustained = {"runs": reps, "total_ms": dt * 1e3, "ms_per_step": dt * 1e3 / reps}
    # execute-only: events around each run on the same stream
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    for a, b in evs:
        a.record(stream)
        ex.run_ptrs(ptrs, out.data_ptr(), stream)
        b.record(stream)
    torch.cuda.synchronize()
    exec_ms = [a.elapsed_time(b) for a, b in evs]
    # per-launch execute-only durations (HIP events around each kernel, on
    # the same stream, over `steps` further runs)
    kernels = ex.profile(inputs, out, reps=steps, stream=stream)
    ex.close()
    return {
        "setup_ms": setup_ms,
        "sustained": sustained,
        "cached_ms": cached_s * 1e3,
        "exec_ms_mean": float(np.mean(exec_ms)),
        "exec_ms_median": float(np.median(exec_ms)),
        "kernels": kernels,
        "plan": plan,
        "ops": w.ops,
    }


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, rows):
    """The oracle on a bounded sample of the headline GEMM: `rows` rows of A
    against the full B, on the host cores (OpenMP); then the oracle on one
    thread over the whole of the small GEMM workloads (256^3 INT16, 1024^3
    and 16 x 512^3 smul24)."""
    from oracle import oracle as orc
    from paper_2606_09905_amd.workloads import WORKLOADS
    cores = int(os.environ.get("OMP_NUM_THREADS", 0)) or len(os.sched_getaffinity(0))
    orc.set_threads(cores)
    A, B = w.generate()
    A = np.ascontiguousarray(A[0, :rows])
    orc.gemm_i16i32(A[:2], B[0])          # build/load outside the timed region
    t0 = time.perf_counter()
    orc.gemm_i16i32(A, B[0])
    dt = time.perf_counter() - t0
    d = w.dims
    ops = 2.0 * rows * d["N"] * d["K"]
    one = {}
    for name in ("gemm_i16_256", "gemm_s24_1024", "gemm_s24_16x512"):
        sw = WORKLOADS[name]
        a, b = sw.generate()
        f = orc.gemm_i16i32 if sw.op == "gemm_i16i32" else orc.gemm_i32_s24
        for threads in (1, cores):
            orc.set_threads(threads)
            t1 = time.perf_counter()
            f(a, b)
            t = time.perf_counter() - t1
            one.setdefault(name, {})["threads_1" if threads == 1 else f"threads_{cores}"] = {
                "seconds": round(t, 4), "gops": round(sw.ops / t / 1e9, 3)}
    orc.set_threads(cores)
    return {
        "value": ops / dt / 1e9, "unit": "GOPS", "cores": cores, "kind": "oracle",
        "sample": f"{rows} of {d['M']} rows of A x full B ({ops:.3e} ops, {dt:.1f} s)",
        "cpu_model": cpu_model(),
        "small_gemms_whole": one,
    }


def oracle_timings(workloads):
    """Wall time of the CPU oracle on every workload, on the host cores: the
    whole workload where it finishes in seconds, else a stated sample (rows of
    A, images, heads).  Rates are in the workload's unit (GOPS, or GiB/s of
    input for the memory-bound rows)."""
    from oracle import oracle as orc
    orc.gemm_i16i32(np.zeros((1, 1, 1), np.int16), np.zeros((1, 1, 1), np.int16))   # build/load
    cores = int(os.environ.get("OMP_NUM_THREADS", 0)) or len(os.sched_getaffinity(0))
    out = {}
    for name, w in workloads.items():
        d = w.dims
        inputs = w.generate()
        frac, sample = 1.0, "whole workload"
        if w.op == "gemm_i16i32":
            A, B = inputs
            budget = 1 << 34                      # multiply-adds the sample may take
            per_batch = d["M"] * d["N"] * d["K"]
            nb = max(1, min(d["batch"], budget // per_batch))
            rows = d["M"] if per_batch <= budget else max(1, budget // (d["N"] * d["K"]))
            if rows < d["M"] or nb < d["batch"]:
                sample = f"{rows} of {d['M']} rows of A in {nb} of {d['batch']} batches"
            frac = rows * nb / (d["M"] * d["batch"])
            fn = lambda: orc.gemm_i16i32(np.ascontiguousarray(A[:nb, :rows]), B[:nb])
        elif w.op == "gemm_i32_s24":
            A, B = inputs
            fn = lambda: orc.gemm_i32_s24(A, B)
        elif w.op in ("conv2d", "conv2d_i32", "conv2d_f32"):
            x, wt = inputs
            f = {"conv2d": orc.conv2d_direct, "conv2d_i32": orc.conv2d_s24, "conv2d_f32": orc.conv2d_f64}[w.op]
            fn = lambda: f(x, wt, d["stride"], d["pad"])
        elif w.op == "attn_f32":
            fn = lambda: orc.attn_f64(*inputs)
        elif w.op == "attn_i32":
            fn = lambda: orc.attn_i32(*inputs)
        elif w.op in ("minmax_i32", "minmax_i16"):
            fn = lambda: orc.minmax(inputs[0])
        elif w.op == "avgpool_i32":
            fn = lambda: orc.avgpool2_i32(inputs[0])
        elif w.op == "maxpool_f32":
            fn = lambda: orc.maxpool2_f32(inputs[0])
        elif w.op == "lenet_i32":
            fn = lambda: orc.lenet_i32(*inputs)
        elif w.op == "sdpa_f32":
            Q, K, V = inputs
            frac, sample = 2 / d["BH"], f"2 of {d['BH']} heads"
            fn = lambda: orc.sdpa_f64(Q[:2], K[:2], V[:2], d["scale"], bool(d["causal"]))
        else:
            continue
        t0 = time.perf_counter()
        fn()
        dt = time.perf_counter() - t0
        if w.ops:
            rate, unit = w.ops * frac / dt / 1e9, "GOPS"
        else:
            rate, unit = w.in_bytes * frac / dt / 2 ** 30, "GiB/s"
        out[name] = {"value": rate, "unit": unit, "seconds": dt, "sample": sample, "cores": cores}
        print(f"[oracle] {name}: {rate:.3g} {unit} ({dt:.2f} s, {sample}, {cores} threads)",
              file=sys.stderr, flush=True)
    return out


# Unit and peak of the dominant kernel for each route: the MFMA peak of the
# operand type the matrix cores run, or the vector ALU's integer rate
# (256 CUs x 64 lanes x 2.4 GHz; v_mad_i32_i24 is 2 ops per lane and cycle,
# v_dot2_i32_i16 4).
ROUTE_PEAK = {
    "f16_exact": ("mfma", "f16"), "i8_direct": ("mfma", "i8"), "i8_karatsuba": ("mfma", "i8"),
    "i8_offset4": ("mfma", "i8"), "s24_i8limb": ("mfma", "i8"), "attn_i32_mfma": ("mfma", "i8"),
    "attn_f32_mfma": ("mfma", "f32"), "f32_mfma": ("mfma", "f32"),
    "s24_valu": ("alu", "i32_valu"), "valu_dot2": ("alu", "dot2_valu"), "attn_i32_valu": ("alu", "i32_valu"),
}
PEAK.update({"i32_valu": 78.6, "dot2_valu": 157.3})
PEAK_UNIT = {"f16": "TFLOP/s", "f32": "TFLOP/s", "i8": "TOP/s", "i32_valu": "TOP/s", "dot2_valu": "TOP/s"}

# The configurations the metric is quoted on, by workload, and the forced
# vector-ALU routes measured beside the matrix-core ones.
CONFIGS = [
    ("C1", "gemm_i16_256", "auto"), ("C1_valu", "gemm_i16_256", "valu_dot2"),
    ("C2a", "gemm_s24_1024", "auto"), ("C2a_valu", "gemm_s24_1024", "s24_valu"),
    ("C2b", "gemm_s24_16x512", "auto"), ("C2b_valu", "gemm_s24_16x512", "s24_valu"),
    ("C3", "conv_8x64x56x56_128_3x3", "auto"),
    ("C4f", "attn_f32_4096x64", "auto"), ("C4i", "attn_i32_4096x64", "auto"),
    ("C5a", "gemm_i16_8192", "auto"), ("C5b", "gemm_i16_64x2048", "auto"),
]


def summarize(w, r):
    """Dominant kernel of a measured workload (the one with the most
    execute-only time per step) and its rate against its unit's peak.  A step
    may split it into several launches (column panels or batch groups);
    together they do the whole algorithmic work, so the achieved rate is that
    work over their summed duration."""
    per_name = {}
    for n, v in r["kernels"]:
        c = per_name.setdefault(n, [0.0, 0])
        c[0] += v
        c[1] += 1
    dom_name, (dom_ms, dom_launches) = max(per_name.items(), key=lambda kv: kv[1][0])
    route = r["plan"]["route_name"]
    bound, unit = ROUTE_PEAK.get(route, ("mfma", "f16"))
    achieved = w.ops / (dom_ms / 1e3) / 1e12
    products = 2.0 if route == "attn_i32_mfma" else float(max(r["plan"]["products"], 1))
    return {"route": route, "bound": bound, "peak_name": unit, "peak": PEAK[unit], "peak_unit": PEAK_UNIT[unit],
            "achieved": achieved, "frac": achieved / PEAK[unit],
            "issued_frac": achieved * products / PEAK[unit] if bound == "mfma" and unit == "i8" else None,
            "kernel": dom_name, "kernel_ms": dom_ms, "kernel_launches": dom_launches,
            "kernels_ms": {n: round(v[0], 4) for n, v in per_name.items()},
            "launches": {n: v[1] for n, v in per_name.items()}}


def measure_configs(args, torch, qx, workloads, headline, head_sm, head_gops):
    """Every configuration the metric is quoted on: cached and execute-only
    GOPS and the dominant kernel's fraction of its unit's peak."""
    out = {}
    cache = {}
    for tag, name, route in CONFIGS:
        wl = workloads[name]
        if name == headline and route == "auto":
            sm, gops_c, gops_e = head_sm, head_gops, None
        else:
            if name not in cache:
                cache.clear()
                torch.cuda.empty_cache()
                cache[name] = [torch.from_numpy(np.ascontiguousarray(a)).cuda() for a in wl.generate()]
            m = measure(wl, max(args.steps, 20), max(args.warmup, 5), torch, qx, route=route, inputs=cache[name])
            sm = summarize(wl, m)
            gops_c = wl.ops / (m["cached_ms"] / 1e3) / 1e9
            gops_e = wl.ops / (m["exec_ms_mean"] / 1e3) / 1e9
        e = {"workload": name, "route": sm["route"], "gops_cached": round(gops_c, 1),
             "gops_exec": None if gops_e is None else round(gops_e, 1),
             "kernel": sm["kernel"], "kernel_ms": round(sm["kernel_ms"], 4),
             "bound": sm["bound"], "peak": sm["peak"], "peak_unit": sm["peak_unit"],
             "kernel_frac": round(sm["frac"], 4)}
        if sm["issued_frac"] is not None:
            e["kernel_issued_frac"] = round(sm["issued_frac"], 4)
        out[tag] = e
        print(f"[bench] {tag} {name} ({sm['route']}): {gops_c:.1f} GOPS cached, kernel {sm['kernel']} "
              f"{sm['kernel_ms'] * 1e3:.1f} us = {sm['frac']:.3f} of {sm['peak_name']} peak",
              file=sys.stderr, flush=True)
    cache.clear()
    return out


def main():
    args = parse()
    if args.oracle_all:
        from paper_2606_09905_amd.workloads import WORKLOADS
        res = oracle_timings(WORKLOADS)
        print(json.dumps({"oracle": res}), flush=True)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "the benchmark runs on one GPU only; --gpus must be 1",
                          "n_gpus": args.gpus}), flush=True)
        sys.exit(2)
    import torch
    from paper_2606_09905_amd import qx
    from paper_2606_09905_amd.workloads import WORKLOADS
    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}), flush=True)
        sys.exit(1)
    if args.copy_calibration:
        copy_calibration(torch)
        return
    qx.lib()
    w = WORKLOADS[args.workload]
    r = measure(w, args.steps, args.warmup, torch, qx, sustain_ms=200.0)
    ms = r["cached_ms"]
    gops = w.ops / (ms / 1e3) / 1e9
    sm = summarize(w, r)
    route = sm["route"]
    line = {
        "metric": METRIC,
        "value": round(gops, 1),
        "unit": "GOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        # the arithmetic the contraction runs in: bf16 (bounds <= 256) or fp16
        # products summed exactly in fp32 per chunk, chunks added in int32
        # (the result is the exact int32 GEMM of the int16 inputs)
        "dtype": {"f16_exact": "bf16" if r["plan"].get("operand_format") == 1 else "f16", "s24_i8limb": "i8", "i8_direct": "i8", "i8_karatsuba": "i8",
                  "i8_offset4": "i8", "attn_f32_mfma": "f32", "attn_i32_mfma": "i8",
                  "f32_mfma": "f32", "f32_valu": "f32", "attn_f32_valu": "f32"}.get(route, "i32"),
        "data": "synthetic",
        "config": {"workload": w.name, **w.dims, "operand_range": [w.lo, w.hi], "seed": w.seed,
                   "route": route, "chunk": r["plan"]["chunk"]},
        "roofline": {
            "bound": sm["bound"],
            "achieved": round(sm["achieved"], 1),
            "peak": sm["peak"],
            "unit": sm["peak_unit"],
            "frac": round(sm["frac"], 4),
            "traffic": traffic_bytes(sm["kernel"], sm["kernel_launches"]),
            "kernel": sm["kernel"],
            "kernel_ms": round(sm["kernel_ms"], 4),
            "kernel_launches": sm["kernel_launches"],
            "frac_of_int8_peak": round(sm["achieved"] / PEAK["i8"], 4),
        },
        "timing": {"setup_ms": round(r["setup_ms"], 2), "cached_ms": round(ms, 4),
                   "exec_ms": round(r["exec_ms_mean"], 4),
                   "kernels_ms": sm["kernels_ms"],
                   "launches": sm["launches"],
                   "end_to_end_frac_of_int8_peak": round(gops / 1e3 / PEAK["i8"], 4),
                   # a further >= 200 ms back-to-back loop (sustained clocks),
                   # outside the K timed steps
                   "sustained": {k: round(v, 4) if isinstance(v, float) else v
                                 for k, v in (r["sustained"] or {}).items()}},
    }
    if not args.no_configs:
        line["configs"] = measure_configs(args, torch, qx, WORKLOADS, w.name, sm, gops)
    if not args.no_cpu:
        line["cpu_baseline"] = cpu_baseline(w, args.cpu_rows)
    if args.all:
        res = {}
        for name, wl in WORKLOADS.items():
            m = measure(wl, max(args.steps, 10), args.warmup, torch, qx)
            if wl.ops:
                m["gops_cached"] = wl.ops / (m["cached_ms"] / 1e3) / 1e9
                m["gops_exec"] = wl.ops / (m["exec_ms_mean"] / 1e3) / 1e9
                rate = f"{m['gops_cached']:.1f} GOPS cached, {m['gops_exec']:.1f} GOPS exec-only"
            else:   # HBM-bound rows: input GiB/s (Table 2 footnote)
                m["gibs_cached"] = wl.in_bytes / (m["cached_ms"] / 1e3) / 2 ** 30
                m["gibs_exec"] = wl.in_bytes / (m["exec_ms_mean"] / 1e3) / 2 ** 30
                rate = (f"{m['gibs_cached']:.1f} GiB/s cached, {m['gibs_exec']:.1f} GiB/s exec-only "
                        f"({m['gibs_cached'] * 2 ** 30 / 1e12 / PEAK['hbm'] * 1e3:.2f} of HBM peak)")
            res[name] = m
            print(f"[bench] {name}: {rate}, route {m['plan']['route_name']}", file=sys.stderr, flush=True)
        if os.path.dirname(args.all_out):
            os.makedirs(os.path.dirname(args.all_out), exist_ok=True)
        with open(args.all_out, "w") as f:
            json.dump(res, f, indent=1)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
