#!/usr/bin/env python3
"""Benchmark of the NLR iteration on one MI355X.

A "step" is one full iteration of Algorithm 1 over the whole synthetic
Gaussian-mixture matrix, which is resident in HBM before timing starts.  By
default the split-fp16 products run in the library's default form for the
shape: at the headline shape (97..128 features, 33..64 columns) the one-pass
form (one kernel per iteration does the row work, the primal step and the next
Theta's and s's partials, then a few small control and reduction kernels);
for other shapes with d <= 128, r <= 64 the single-Xhat-pass form (row pass,
fused pass B).  `--gemm fp32` uses the fp32 matrix cores (single-Xhat-pass
form) and `--two-pass` the two-pass form.  A second timed run with the other product form
is reported under "alt".  `value` is points*iterations per second over the
timed run.  `achieved_hbm_gbs` / `hbm_frac` are the bytes the launched row and
pass kernels move (their algorithmic bytes per launch times their launches) over
the timed time: a physical HBM rate.  `effective_two_pass_gbs` divides the fixed
two-pass byte count 4(2nd + 3nr + 2n) per iteration instead, a work-equivalent
rate that counts the bytes a fused form saves as speed.  The `roofline` object
describes the dominant kernel, timed with
HIP events on the library's stream inside the same timed region;
`cpu_baseline` times the fp64 oracle on a bounded sample of the same workload
on the host cores.

Usage: python bench.py [--gpus 1] [--steps 50] [--warmup 3] [--workload gmm10m]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "NLR points·iters/sec + achieved HBM GB/s (n=1e7,d=128,K=64, fp32)"
HBM_PEAK_GBS = 8000.0
FP32_MFMA_PEAK_TFLOPS = 157.3
FP16_MFMA_PEAK_TFLOPS = 2500.0


def eprint(*a):
    print(*a, file=sys.stderr, flush=True)


def algorithmic_bytes(kind: str, n: int, d: int, r: int, dual_frac: float = 0.0) -> float:
    """Bytes each kernel must move per launch (fp32 = 4 B), independent of caching."""
    if kind == "pass_b":      # read Xhat, read U, write W over U, read ytilde
        return 4.0 * (n * d + 2 * n * r + n)
    if kind == "pass_a":      # read Xhat, read U, read ytilde (+ write it on dual steps)
        return 4.0 * (n * d + n * r + n) + 4.0 * n * dual_frac
    if kind == "pass_bf":     # fused pass B: as pass B (the Theta partials stay on chip)
        return 4.0 * (n * d + 2 * n * r + n)
    if kind == "pass_u":      # row pass: read U and ytilde (+ write ytilde on dual steps)
        return 4.0 * (n * r + n) + 4.0 * n * dual_frac
    if kind == "finish":      # read W, write U = c W, read ytilde (+ write it on a pending dual step)
        return 4.0 * (2 * n * r + n) + 4.0 * n * dual_frac
    if kind == "step":        # whole iteration of the two-pass structure: the fixed numerator
        return 4.0 * (2 * n * d + 3 * n * r + 2 * n) + 4.0 * n * dual_frac
    raise ValueError(kind)


def iteration_form(n: int, d: int, r: int, K: int, split: bool, two_pass: bool) -> str:
    """The iteration form the library chooses for the shape (asked of the library itself)."""
    from paper_2609_36074_amd import nlr
    flags = (nlr.NLR_INIT_SPLIT_F16 if split else 0) | (nlr.NLR_INIT_TWO_PASS if two_pass else 0)
    code = nlr.nlr_iteration_form(n, d, r, K, flags)
    if code < 0:
        raise ValueError(f"no iteration form for n={n} d={d} r={r} K={K} flags={flags}")
    return nlr.FORM_NAMES[code]


def iteration_bytes(kinfo: dict, n: int, d: int, r: int, dual_frac: float = 0.0) -> float:
    """Bytes the launched row and pass kernels moved in the timed region: each kernel's
    algorithmic bytes per launch times its launches (the small control and reduction
    kernels move under 0.1% of this)."""
    return sum(algorithmic_bytes(k, n, d, r, dual_frac) * v["launches"] for k, v in kinfo.items()
               if k in ("pass_a", "pass_b", "pass_u", "pass_bf", "finish"))


def kernel_source_hash(kernel: str) -> str:
    """Hash of the sources that define `kernel` (a traffic record is void once they change)."""
    if kernel.startswith("pass_bf"):
        files = ("k_fused.hip",)
    elif kernel.startswith("pass_u"):
        files = ("k_iter.hip",)
    else:  # pass_a / pass_b: generic, resident, split and panel forms
        files = ("k_iter.hip", "k_split.hip", "k_panel.hip")
    h = hashlib.sha256()
    for f in files + ("k_common.hpp", "nlr_internal.hpp"):
        with open(os.path.join(ROOT, "paper_2609_36074_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def load_traffic(kernel: str, workload: str):
    """HBM traffic of `kernel` from the committed rocprofv3 --pmc summary, or None
    when there is none or the kernel source changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.json")
    if not os.path.exists(path):
        return None
    try:
        with open(path) as f:
            t = json.load(f)
        if t.get("kernel_source_hash") != kernel_source_hash(kernel):
            return None
        return float(t["bytes_per_launch"])
    except Exception:
        return None


def cpu_baseline(workload, n_sample: int, iters: int) -> dict:
    """Times the fp64 oracle's iteration loop on a bounded sample of the workload."""
    import numpy as np

    from oracle import nlr as onlr
    from synth import make_workload
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    X, Z, _, wl = make_workload(workload, rows=n_sample)
    Xh, _, _ = onlr.centre_and_normalise(X)
    U0 = onlr.project_omega(Z.astype(np.float64), wl.K)
    alpha = onlr.default_step_size(wl.K)
    t0 = time.perf_counter()
    onlr.run(Xh, U0, wl.K, alpha, 1.0, T=iters, T_min=iters, project_init=False)
    dt = time.perf_counter() - t0
    cpu = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            cpu = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), cpu)
    except OSError:
        pass
    try:
        visible = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        visible = os.cpu_count() or 1
    return {"value": n_sample * iters / dt, "unit": "points*iters/s", "cores": int(threads), "kind": "oracle",
            "sample": f"fp64 oracle loop, {iters} iterations on the first {n_sample} rows of the same "
                      f"seeded {workload} draw (d={wl.d}, K=r={wl.K}; centred and normalised as a matrix "
                      f"of its own); {dt:.1f} s",
            "cpu": cpu, "cores_visible": int(visible)}


def kernel_flops(kind: str, n: int, d: int, r: int) -> float:
    """fp32-equivalent matrix flops of one launch (pass_bf holds both products)."""
    return {"pass_a": 2.0, "pass_b": 2.0, "pass_bf": 4.0}.get(kind, 0.0) * n * d * r


def measure(nlr, torch, np, X_host, Z_host, wl, steps, warm, split, two_pass):
    """Init on fresh device copies of (X_host, U_0 = Z_host), `warm` untimed iterations, then `steps`
    timed ones.  (nlr_init normalises X in place, and the split form also stores it split.)"""
    n, d, r, K = wl.n, wl.d, wl.r, wl.K
    X_dev = torch.from_numpy(X_host).to("cuda:0")
    Ut = torch.from_numpy(Z_host).to(X_dev.device)
    alpha = 1.0 / (2.0 * (2.0 + 1.0 * (6.0 * K + 2.0)))  # half the Prop. 1 step bound at y = 0, beta = 1
    flags = (nlr.NLR_INIT_SPLIT_F16 if split else 0) | (nlr.NLR_INIT_TWO_PASS if two_pass else 0)
    torch.cuda.synchronize()
    ctx = nlr.Context(X_dev, K, Ut, alpha=alpha, beta=1.0, eps_d=1e-4, eps_c=1e-4, T_min=1 << 30, flags=flags)
    if warm > 0:
        ctx.run(warm)
    torch.cuda.synchronize()
    stream = ctx.stream
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    # the timed region: `steps` iterations in one nlr_run, each launch made on its own with the
    # library's HIP events around the row and pass kernels (the roofline's candidates), so the
    # kernel durations come from the same region as the time
    ctx.set_profiling(2)
    rows0 = ctx.inspect("rows_run")
    torch.cuda.synchronize()
    ev0.record(stream)
    done, _ = ctx.run(steps)
    ev1.record(stream)
    torch.cuda.synchronize()
    t_ms = ev0.elapsed_time(ev1)
    kt = ctx.kernel_times()
    ctx.set_profiling(False)
    rows_ran = ctx.inspect("rows_run") - rows0
    assert done == steps, (done, steps)
    hist = ctx.history(steps)
    # the same number of iterations again as a caller's nlr_run makes them without profiling
    # (after its first iteration, graph replays): reported beside the timed figure
    ev0.record(stream)
    done_g, _ = ctx.run(steps)
    ev1.record(stream)
    torch.cuda.synchronize()
    t_graph_ms = ev0.elapsed_time(ev1)
    assert done_g == steps, (done_g, steps)
    # the row-argmax labels of the final factor (not part of the iteration): one call
    # after a warm one, HIP events on the library's stream
    lab = torch.empty(n, dtype=torch.int32, device=X_dev.device)
    ctx.labels(out=lab)
    ev0.record(stream)
    ctx.labels(out=lab)
    ev1.record(stream)
    torch.cuda.synchronize()
    t_lab_ms = ev0.elapsed_time(ev1)
    del lab
    ctx.close()
    del Ut, X_dev
    torch.cuda.empty_cache()
    dual_frac = float(np.mean([h["dual_step"] for h in hist])) if hist else 0.0
    value = n * steps / (t_ms / 1e3)
    # the fixed two-pass numerator 4(2nd + 3nr + 2n) per iteration: a work-equivalent rate
    # (bytes a fused form does not move still count), not a bandwidth
    eff_gbs = algorithmic_bytes("step", n, d, r, dual_frac) * steps / (t_ms / 1e3) / 1e9
    kinfo = {k: {"total_ms": v[0], "launches": v[1], "avg_ms": (v[0] / v[1]) if v[1] else None}
             for k, v in kt.items() if v[1]}
    # the bytes the form actually moved, over the timed region: a physical HBM rate.  The
    # one-pass form launches its row pass every iteration but it runs (and moves U) only
    # where the previous iteration's stop may fire: count those, from the library's counter
    kbytes = {k: dict(v) for k, v in kinfo.items()}
    if "pass_u" in kbytes and split and iteration_form(n, d, r, K, split, two_pass) == "one-pass":
        kbytes["pass_u"]["launches"] = rows_ran
    phys_gbs = iteration_bytes(kbytes, n, d, r, dual_frac) / (t_ms / 1e3) / 1e9
    dom = max(("pass_a", "pass_b", "pass_u", "pass_bf"), key=lambda k: kinfo.get(k, {"total_ms": 0})["total_ms"])
    if rows_ran:
        kinfo["pass_u"]["row_passes_run"] = rows_ran
    dom_ms = kinfo[dom]["avg_ms"]
    dom_bytes = algorithmic_bytes(dom, n, d, r, dual_frac)
    achieved = dom_bytes / (dom_ms / 1e3) / 1e9
    dom_name = dom + ("_split16" if split else "")
    fl = kernel_flops(dom, n, d, r)
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": load_traffic(dom_name, wl.name),
                "kernel": dom_name, "avg_launch_ms": round(dom_ms, 4),
                "algorithmic_bytes_per_launch": dom_bytes}
    if split:  # three fp16 products per fp32 product, against the dense fp16 peak
        roofline["mfma_tflops"] = round(3.0 * fl / (dom_ms / 1e3) / 1e12, 2)
        roofline["mfma_frac"] = round(roofline["mfma_tflops"] / FP16_MFMA_PEAK_TFLOPS, 4)
    else:
        roofline["mfma_tflops"] = round(fl / (dom_ms / 1e3) / 1e12, 2)
        roofline["mfma_frac"] = round(roofline["mfma_tflops"] / FP32_MFMA_PEAK_TFLOPS, 4)
    form = iteration_form(n, d, r, K, split, two_pass)
    label = ("split-fp16 " if split else "fp32 ") + form
    eprint(f"[bench] {label}: {steps} steps in {t_ms:.2f} ms -> {t_ms / steps:.3f} ms/step, {value:.3e} pts*it/s, "
           f"HBM {phys_gbs:.0f} GB/s ({phys_gbs / HBM_PEAK_GBS:.1%} of peak); two-pass work-equivalent "
           f"{eff_gbs:.0f} GB/s; graph replays {t_graph_ms / steps:.3f} ms/step")
    for k, v in kinfo.items():
        eprint(f"[bench]   {k:13s} {v['avg_ms'] * 1e3:9.1f} us x {v['launches']}")
    return {"value": value, "t_ms": t_ms, "t_graph_ms": t_graph_ms, "t_lab_ms": t_lab_ms, "eff_gbs": eff_gbs, "phys_gbs": phys_gbs, "dual_frac": dual_frac,
            "alpha": alpha, "roofline": roofline, "kernels": kinfo, "form": form}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=50,
                    help="untimed iterations first (the clock and caches settle: at the headline shape the timed "
                         "ms per iteration is about 2%% higher after 3 than after 20, and 0.5%% after 50)")
    ap.add_argument("--workload", default="gmm10m")
    ap.add_argument("--gemm", choices=("fp32", "split16"), default="split16",
                    help="split16 (default): two-term fp16 splits of the operands on the fp16 matrix cores "
                         "(NLR_INIT_SPLIT_F16); fp32: both products on the fp32 matrix cores")
    ap.add_argument("--two-pass", action="store_true",
                    help="use the two-pass iteration (NLR_INIT_TWO_PASS) instead of the single-Xhat-pass form")
    ap.add_argument("--no-alt", action="store_true",
                    help="skip the second timed run with the other product form (reported under 'alt')")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample", type=int, default=2_000_000)
    ap.add_argument("--cpu-iters", type=int, default=8)
    ap.add_argument("--pmc-calibrate", action="store_true",
                    help="first run one elementwise copy of 1 GiB (y = x * 1), the reference kernel that scales "
                         "rocprofv3 FETCH_SIZE / WRITE_SIZE readings to bytes")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU (asked for {args.gpus}): the NLR path here is the "
              "single-GPU kernel set; sharding the rows over several GPUs is designed but not built.",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2609_36074_amd import nlr
    from synth import WORKLOADS, make_workload

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    wl = WORKLOADS[args.workload]
    n, d, r, K = wl.n, wl.d, wl.r, wl.K
    eprint(f"[bench] generating {args.workload}: n={n} d={d} K=r={K}")
    t0 = time.perf_counter()
    X, Z, _, _ = make_workload(wl)
    eprint(f"[bench] generated in {time.perf_counter() - t0:.1f} s; uploading")
    dev = torch.device("cuda:0")
    if args.pmc_calibrate:
        src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        del src, dst
    # the split products exist for d <= 128, r <= 64, d % 4 == 0 (and r % 4 == 0 in the two-pass
    # form), and in the two-pass panel form for d % 8 == 0, r % 4 == 0, r <= 256; other shapes run
    # fp32 products
    split_ok = (d <= 128 and r <= 64 and d % 4 == 0 and (r % 4 == 0 or not args.two_pass)) or \
        (d % 8 == 0 and r % 4 == 0 and r <= 256)
    split = args.gemm == "split16" and split_ok
    if args.gemm == "split16" and not split:
        eprint(f"[bench] split-fp16 products are not available for d={d}, r={r}: fp32 products")
    main_run = measure(nlr, torch, np, X, Z, wl, args.steps, args.warmup, split, args.two_pass)
    alt = None
    if not args.no_alt and split_ok:
        # the other product form on the same data and the same start
        a = measure(nlr, torch, np, X, Z, wl, args.steps, args.warmup, not split, args.two_pass)
        alt = {"products": "fp32" if split else "fp16 two-term split, fp32 accumulate",
               "dtype": "f32" if split else "f32 (fp16x3 products)",
               "iteration": a["form"], "value": a["value"], "ms_per_step": a["t_ms"] / args.steps,
               "graph_replay_ms_per_step": a["t_graph_ms"] / args.steps,
               "achieved_hbm_gbs": round(a["phys_gbs"], 1), "hbm_frac": round(a["phys_gbs"] / HBM_PEAK_GBS, 4),
               "effective_two_pass_gbs": round(a["eff_gbs"], 1), "roofline": a["roofline"]}
    del X, Z

    cpu = None
    if not args.no_cpu_baseline:
        eprint("[bench] cpu baseline (fp64 oracle) ...")
        cpu = cpu_baseline(args.workload, min(args.cpu_sample, n), args.cpu_iters)
        eprint(f"[bench] cpu baseline {cpu['value']:.3e} pts*it/s on {cpu['cores']} threads")

    m = main_run
    out = {
        "metric": METRIC,
        "value": m["value"],
        "unit": "points*iters/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": m["t_ms"] / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32 (fp16x3 products)" if split else "f32",
        "data": "synthetic",
        "config": {"workload": args.workload, "n": n, "d": d, "K": K, "r": r, "alpha": m["alpha"], "beta": 1.0,
                   "iteration": m["form"],
                   "products": "fp16 two-term split, fp32 accumulate" if split else "fp32",
                   "eps_d": 1e-4, "eps_c": 1e-4, "dual_step_fraction": m["dual_frac"]},
        "achieved_hbm_gbs": round(m["phys_gbs"], 1),
        "hbm_frac": round(m["phys_gbs"] / HBM_PEAK_GBS, 4),
        "effective_two_pass_gbs": round(m["eff_gbs"], 1),
        "roofline": m["roofline"],
        "labels": {"ms": round(m["t_lab_ms"], 4), "bytes": 4 * n * r + 4 * n,
                   "gbs": round((4 * n * r + 4 * n) / (m["t_lab_ms"] / 1e3) / 1e9, 1),
                   "note": "one nlr_labels call (row argmax) on the final factor, outside the timed region"},
        "graph_replay": {"ms_per_step": m["t_graph_ms"] / args.steps, "value": n * args.steps / (m["t_graph_ms"] / 1e3),
                         "note": "the next `steps` iterations as an unprofiled nlr_run makes them: graph replays "
                                 "after the call's first iteration, no events"},
        "cpu_baseline": cpu,
        "alt": alt,
        "kernels": m["kernels"],
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
