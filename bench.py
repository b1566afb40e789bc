"""Benchmark of the LionMuon optimizer step on one MI355X.

One step = one pass of Algorithm 1 over the whole matrix set (the Lion branch
kernel on Lion steps; preparation, Frobenius norm and five Newton-Schulz
iterations on Muon steps, every P-th step). Reported: amortised ms/step over
K timed steps (K a multiple of P), Lion GB/s (20 bytes per element) and
Newton-Schulz TFLOP/s (symmetric algorithmic flops), with the roofline of the
dominant kernel measured by the library's per-launch HIP events on the launch
stream, and the fp64 CPU oracle timed on a bounded sample as a baseline.

The amortised time is taken over K steps with the library's per-launch events
off (they cost ~6% of a 124M step); the per-kernel times behind the phases,
the roofline and the split come from a second timed region of the same K
steps with the events on.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import workloads  # noqa: E402

HBM_PEAK_GBPS = 8000.0            # MI355X HBM3E
BF16_PEAK_TFLOPS = 2516.6         # dense MFMA: 256 CU x 2.4 GHz x 4096 flop/clk
FP32_MFMA_PEAK_TFLOPS = 157.3
# the kernels, the planner that sets their tiles and grids, and the constants
# both share: traffic per launch depends on all three
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2605_19811_amd", "csrc", f)
                  for f in ("kernels.hip", "plan.cpp", "lm_desc.h")]
TRAFFIC_DIR = os.path.join(ROOT, "profiles")


def kernel_hash():
    """Hash of the kernel, planner and shared-constant sources with comments
    and blank lines removed, so a comment-only edit keeps the counters taken
    with the same code valid."""
    import re
    h = hashlib.sha256()
    for path in KERNEL_SOURCES:
        with open(path) as f:
            src = f.read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        lines = [re.sub(r"//.*$", "", ln).rstrip() for ln in src.splitlines()]
        h.update("\n".join(ln for ln in lines if ln.strip()).encode())
    return h.hexdigest()[:16]


def load_traffic(workload, kernel):
    """HBM traffic (bytes per launch) from the committed rocprofv3 counter
    summary, or None when absent or taken from another kernel source."""
    path = os.path.join(TRAFFIC_DIR, f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)
    if d.get("kernel_source_sha256_16") != kernel_hash():
        return None
    k = d.get("kernels", {}).get(kernel)
    return None if k is None else k.get("bytes_per_launch")


PHASE_OF_KERNEL = (("lion_kernel", "lion"), ("prep_kernel", "prep"), ("norm_kernel", "norm"),
                   ("ns_gram_kernel", "gram"), ("ns_poly_kernel", "poly"),
                   ("ns_apply_", "apply"), ("srank_", "srank"))   # apply: ns_apply_kernel, ns_apply_last_kernel


def phase_of(kernel_name):
    """Phase name of a library kernel from its (mangled or demangled) name."""
    for key, phase in PHASE_OF_KERNEL:
        if key in kernel_name:
            return phase
    return None


def _counter_means(csv_path, counter):
    import collections
    import csv
    vals = collections.defaultdict(list)
    with open(csv_path) as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] == counter:
                vals[r["Kernel_Name"]].append(float(r["Counter_Value"]))
    return vals


def pmc_summary(wl_name, fetch_csv, write_csv, calib_fetch_csv, calib_write_csv, calib_mib,
                commands):
    """Per-launch HBM traffic of each library kernel from rocprofv3 FETCH_SIZE
    and WRITE_SIZE (KiB per dispatch), each scaled by what the same counter
    reads for a plain device copy of a known size."""
    copy_bytes = calib_mib * (1 << 20)
    # only the copy kernel itself (the buffer's initial fill kernel reads nothing)
    cf = [v for k, vs in _counter_means(calib_fetch_csv, "FETCH_SIZE").items() for v in vs
          if "copy" in k.lower()]
    cw = [v for k, vs in _counter_means(calib_write_csv, "WRITE_SIZE").items() for v in vs
          if "copy" in k.lower()]
    f_scale = copy_bytes / (sum(cf) / len(cf) * 1024.0)
    w_scale = copy_bytes / (sum(cw) / len(cw) * 1024.0)
    fetch = _counter_means(fetch_csv, "FETCH_SIZE")
    write = _counter_means(write_csv, "WRITE_SIZE")
    kernels = {}
    # the stable-rank phase is several kernels per step: bytes per step =
    # all of its dispatches / the decide dispatches (one per step)
    steps = [len(v) for k, v in fetch.items() if "srank_decide" in k]
    srank = {"fetch_bytes": 0.0, "write_bytes": 0.0}
    # a Newton-Schulz phase launch is one main-list launch plus, for the
    # apply, an optional launch of its last round as 128-tiles (and the last
    # apply is its own kernel): bytes per launch = all of the phase's
    # dispatches / its 256-tile dispatches (all dispatches where there are none)
    tot = {}
    for name in set(fetch) | set(write):
        ph = phase_of(name)
        if ph is None:
            continue
        fv, wv = fetch.get(name, []), write.get(name, [])
        if ph == "srank":
            srank["fetch_bytes"] += sum(fv) * 1024.0 * f_scale / steps[0]
            srank["write_bytes"] += sum(wv) * 1024.0 * w_scale / steps[0]
            continue
        t = tot.setdefault(ph, {"fetch": 0.0, "write": 0.0, "n_all": 0, "n_256": 0})
        t["fetch"] += sum(fv) * 1024.0 * f_scale
        t["write"] += sum(wv) * 1024.0 * w_scale
        t["n_all"] += len(fv)
        if "Li256" in name:
            t["n_256"] += len(fv)
    for ph, t in tot.items():
        n = t["n_256"] or t["n_all"]
        kernels[ph] = {"fetch_bytes": t["fetch"] / n, "write_bytes": t["write"] / n,
                       "bytes_per_launch": (t["fetch"] + t["write"]) / n}
    if steps:
        srank["bytes_per_launch"] = srank["fetch_bytes"] + srank["write_bytes"]
        kernels["srank"] = srank
    out = {"workload": wl_name, "kernel_source_sha256_16": kernel_hash(),
           "fetch_scale": f_scale, "write_scale": w_scale,
           "calibration": f"plain device copy of {calib_mib} MiB (torch copy_)",
           "commands": commands, "kernels": kernels}
    path = os.path.join(TRAFFIC_DIR, f"traffic_{wl_name}.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    return path


def sq_summary(wl_name, sq_csv, command):
    """MFMA and LDS occupancy of each library kernel from one rocprofv3 SQ
    counter pass (sums over all dispatches of the kernel)."""
    import collections
    import csv
    tot = collections.defaultdict(lambda: collections.defaultdict(float))
    for r in csv.DictReader(open(sq_csv)):
        if phase_of(r["Kernel_Name"]) is None:
            continue
        tot[r["Kernel_Name"]][r["Counter_Name"]] += float(r["Counter_Value"])
    lines = [f"# SQ counters: {wl_name}", "", f"Command: `{command}`", "",
             "MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (4 SIMDs x SQ_BUSY_CU_CYCLES): the fraction of "
             "SIMD cycles, while the CU is busy, in which the matrix core is executing (a "
             "32x32x16 bf16 MFMA occupies its SIMD for 32 cycles; 1024 flop per SIMD-cycle is "
             "the nominal peak). Wait = SQ_WAIT_ANY / SQ_WAVE_CYCLES. LDS conflict = "
             "SQ_LDS_BANK_CONFLICT / SQ_LDS_IDX_ACTIVE.", "",
             "| kernel | phase | MFMA busy | wait | LDS conflict |", "|---|---|---|---|---|"]
    for name, c in sorted(tot.items(), key=lambda kv: phase_of(kv[0])):
        busy = c.get("SQ_BUSY_CU_CYCLES", 0.0)
        mf = c.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) / (4.0 * busy) if busy else 0.0
        wt = c.get("SQ_WAIT_ANY", 0.0) / c["SQ_WAVE_CYCLES"] if c.get("SQ_WAVE_CYCLES") else 0.0
        lc = (c.get("SQ_LDS_BANK_CONFLICT", 0.0) / c["SQ_LDS_IDX_ACTIVE"]
              if c.get("SQ_LDS_IDX_ACTIVE") else 0.0)
        short = name if len(name) < 70 else name[:67] + "..."
        lines.append(f"| `{short}` | {phase_of(name)} | {mf:.3f} | {wt:.3f} | {lc:.3f} |")
    path = os.path.join(TRAFFIC_DIR, f"sq_{wl_name}.md")
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")
    return path


def trace_summary(wl_name, stats_csv, command):
    """Text summary of a rocprofv3 --kernel-trace --stats run."""
    import csv
    rows = list(csv.DictReader(open(stats_csv)))
    lines = [f"# Kernel trace: {wl_name}", "", f"Command: `{command}`", "",
             "| kernel | phase | calls | avg us | total us | % |", "|---|---|---|---|---|---|"]
    for r in rows:
        name = r["Name"]
        ph = phase_of(name) or "-"
        short = name if len(name) < 70 else name[:67] + "..."
        lines.append(f"| `{short}` | {ph} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                     f"{float(r['TotalDurationNs']) / 1e3:.1f} | {float(r['Percentage']):.2f} |")
    # per phase launch, as bench.py times a phase (main list plus the apply's
    # 128-tile tail and last-step kernels; the stable-rank phase per step)
    tot = {}
    for r in rows:
        ph = phase_of(r["Name"])
        if ph is None:
            continue
        t = tot.setdefault(ph, {"ns": 0.0, "n_all": 0, "n_256": 0, "n_decide": 0})
        t["ns"] += float(r["TotalDurationNs"])
        t["n_all"] += int(r["Calls"])
        if "Li256" in r["Name"]:
            t["n_256"] += int(r["Calls"])
        if "srank_decide" in r["Name"]:
            t["n_decide"] += int(r["Calls"])
    lines += ["", "Per phase launch (all of a phase's kernels; launches = its 256-tile dispatches "
              "where there are any, the decide dispatches for srank):", "",
              "| phase | launches | avg us per launch |", "|---|---|---|"]
    for ph, t in sorted(tot.items(), key=lambda kv: -kv[1]["ns"]):
        n = t["n_decide"] if ph == "srank" else (t["n_256"] or t["n_all"])
        lines.append(f"| {ph} | {n} | {t['ns'] / n / 1e3:.1f} |")
    path = os.path.join(TRAFFIC_DIR, f"kernel_trace_{wl_name}.md")
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")
    return path


def ns_flops_per_launch(wl):
    gram = poly = apply = 0.0
    for t in wl.tensors:
        if t.lion_only or t.rows == 1:
            continue
        s, l = min(t.rows, t.cols), max(t.rows, t.cols)
        gram += s * (s + 1) * l
        poly += s * s * (s + 1)
        apply += 2.0 * s * s * l
    return {"gram": gram, "poly": poly, "apply": apply}


def cpu_baseline(wl, P, budget_s=10.0):
    """fp64 oracle on a bounded sample: one Lion step and one Muon step on one
    tensor of every distinct shape, scaled to the whole set by tensor count,
    repeated until about `budget_s` seconds of CPU work (at least once) and
    averaged over the repetitions, amortised over P."""
    import numpy as np
    import oracle
    try:
        from threadpoolctl import threadpool_info
        cores = max([d.get("num_threads", 1) for d in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        cores = len(os.sched_getaffinity(0))
    seen, sample = {}, []
    for i, t in enumerate(wl.tensors):
        key = (t.rows, t.cols, t.lion_only)
        seen[key] = seen.get(key, 0) + 1
        if seen[key] == 1:
            sample.append(i)
    count = {k: v for k, v in seen.items()}
    rng = np.random.default_rng(0)
    inputs = []
    for i in sample:
        t = wl.tensors[i]
        W = rng.standard_normal(t.shape).astype(np.float32) * 0.02
        M = rng.standard_normal(t.shape).astype(np.float32) * wl.grad_std
        G = rng.standard_normal(t.shape).astype(np.float32) * wl.grad_std
        inputs.append((t, W, M, G))
    t_lion = t_muon = 0.0
    rounds = 0
    start = time.perf_counter()
    while rounds == 0 or time.perf_counter() - start < budget_s:
        for t, W, M, G in inputs:
            reps = count[(t.rows, t.cols, t.lion_only)]
            t0 = time.perf_counter()
            oracle.lionmuon_update(W, G, M, 1, P, wl.beta1, wl.beta2, wl.lr_muon, wl.lr_lion,
                                   wl.wd, lion_only=True)
            t1 = time.perf_counter()
            oracle.lionmuon_update(W, G, M, 0, 1, wl.beta1, wl.beta2, wl.lr_muon, wl.lr_lion,
                                   wl.wd, lion_only=t.lion_only)
            t2 = time.perf_counter()
            t_lion += (t1 - t0) * reps
            t_muon += (t2 - t1) * reps
        rounds += 1
    spent = time.perf_counter() - start
    t_lion /= rounds
    t_muon /= rounds
    if P == 0:
        amort = t_lion
    else:
        amort = ((P - 1) * t_lion + t_muon) / P
    return {"value": round(amort * 1e3, 1), "unit": "ms/step", "cores": int(cores),
            "kind": "oracle",
            "sample": (f"one Lion and one Muon fp64 oracle step on one tensor of each of the "
                       f"{len(sample)} distinct shapes of {wl.name}, scaled by tensor count, "
                       f"repeated {rounds}x ({spent:.1f} s of CPU work) and averaged; "
                       f"Lion {t_lion * 1e3:.0f} ms/step, Muon {t_muon * 1e3:.0f} ms/step, "
                       f"amortised over P={P}")}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="gpt2-124m", choices=sorted(workloads.WORKLOADS))
    ap.add_argument("--P", type=int, default=2, help="period; 0 = pure Lion")
    ap.add_argument("--pure-muon", action="store_true", help="P=1 with beta1=beta2=0.9")
    ap.add_argument("--adaptive", type=float, default=0.0, metavar="ALPHA",
                    help="stable-rank rule of Appendix G with this alpha instead of the period")
    ap.add_argument("--power-steps", type=int, default=5, help="power-iteration steps (adaptive)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true",
                    help="time without per-launch events (no roofline object)")
    ap.add_argument("--calib-copy", type=int, default=0, metavar="MIB",
                    help="only run 4 plain device copies of MIB MiB (counter calibration)")
    ap.add_argument("--pmc-summary", nargs=4, metavar=("FETCH_CSV", "WRITE_CSV", "CALIB_FETCH_CSV",
                                                        "CALIB_WRITE_CSV"),
                    help="write profiles/traffic_<workload>.json from rocprofv3 counter CSVs")
    ap.add_argument("--trace-summary", metavar="KERNEL_STATS_CSV",
                    help="write profiles/kernel_trace_<workload>.md from a rocprofv3 stats CSV")
    ap.add_argument("--sq-summary", metavar="SQ_CSV",
                    help="write profiles/sq_<workload>.md from a rocprofv3 SQ counter CSV")
    ap.add_argument("--command", default="", help="profiling command recorded in summaries")
    args = ap.parse_args()
    # profiles of the adaptive variant are kept apart from the periodic step's
    prof_name = args.workload + ("-adaptive" if args.adaptive > 0.0 else "")
    if args.pmc_summary:
        print(pmc_summary(prof_name, *args.pmc_summary, calib_mib=1024,
                          commands=args.command))
        return
    if args.trace_summary:
        print(trace_summary(prof_name, args.trace_summary, args.command))
        return
    if args.sq_summary:
        print(sq_summary(prof_name, args.sq_summary, args.command))
        return
    if args.calib_copy:
        import torch
        n = args.calib_copy * (1 << 20) // 4
        x = torch.ones(n, device="cuda:0")
        y = torch.empty_like(x)
        for _ in range(4):
            y.copy_(x)
        torch.cuda.synchronize()
        print(json.dumps({"calib_copy_bytes_read": 4 * n, "calib_copy_bytes_written": 4 * n,
                          "launches": 4}))
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); the multi-GPU "
              f"layout is a design, not a build.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2605_19811_amd import lionmuon as lm

    wl = workloads.get(args.workload)
    P = 1 if args.pure_muon else args.P
    beta1, beta2 = (0.9, 0.9) if args.pure_muon else (wl.beta1, wl.beta2)
    adaptive = args.adaptive > 0.0
    steps = args.steps
    if P > 1 and steps % P and not adaptive:
        steps += P - steps % P                 # whole periods only
    dev = torch.device("cuda:0")
    params, moms, grad_sets = workloads.device_state(torch, wl, dev, seed=7, warm=True, n_grad=2)
    lion_only = [t.lion_only for t in wl.tensors]
    lists = [lm.TensorList(params, g, moms, lion_only) for g in grad_sets]
    cfg = lm.config(ns_precision=wl.ns_precision, lr_muon=wl.lr_muon, lr_lion=wl.lr_lion,
                    adaptive_alpha=args.adaptive, adaptive_power_steps=args.power_steps)
    cfg_period = lm.config(ns_precision=wl.ns_precision, lr_muon=wl.lr_muon, lr_lion=wl.lr_lion)
    specs = [(t.rows, t.cols, t.lion_only) for t in wl.tensors]
    info_muon = lm.lionmuon_plan_info(specs, 0, 1, cfg_period)
    info_lion = lm.lionmuon_plan_info(specs, 1, 2, cfg_period)
    info_adaptive = lm.lionmuon_plan_info(specs, 0, 0, cfg) if adaptive else None
    stream = torch.cuda.current_stream()

    def run(t0, n):
        for k in range(n):
            t = t0 + k
            lm.lionmuon_step_ex(None, None, None, t, P, beta1, beta2, wl.wd, cfg,
                                stream=stream, tensors=lists[t % 2])

    run(1, args.warmup)
    torch.cuda.synchronize()
    t_start = 1 + args.warmup
    t_start += (-t_start) % max(P, 1)         # timed region starts on a Muon step
    profile = not args.no_profile
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    run(t_start, steps)
    e1.record(stream)
    torch.cuda.synchronize()
    total_ms = e0.elapsed_time(e1)
    ms_step = total_ms / steps
    phases = None
    if profile:
        # per-launch times: a second timed region of the same steps (whole
        # periods, starting on a Muon step) with the library's events on
        lm.lionmuon_profiling_reset()
        lm.lionmuon_profiling_enable(True)
        run(t_start + steps, steps)
        torch.cuda.synchronize()
        phases = lm.lionmuon_profiling_read()
        lm.lionmuon_profiling_enable(False)

    muon_fraction = None
    if adaptive:
        # decisions of one further step (after the timed region)
        dec = torch.zeros(len(wl.tensors), dtype=torch.int32, device=dev)
        t_next = t_start + (2 if profile else 1) * steps
        lm.lionmuon_step_adaptive(None, None, None, t_next, beta1, beta2, wl.wd, cfg,
                                  stream=stream, tensors=lists[0], decisions=dec)
        torch.cuda.synchronize()
        muon_fraction = round(float(dec.sum().item()) / info_adaptive["n_muon"], 4)
        n_muon_steps = 0
    else:
        n_muon_steps = sum(1 for k in range(steps) if P >= 1 and (t_start + k) % P == 0)
    n_lion_steps = steps - n_muon_steps
    out = {
        "metric": "amortised optimizer-step ms per period P (LionMuon step, 1 GPU)",
        "value": round(ms_step, 4),
        "unit": "ms/step",
        "n_gpus": 1,
        "steps": steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.ns_precision == "bf16" else "f32",
        "data": "synthetic (seeded gradients of the workload's shapes; random-init weights)",
        "config": {"workload": wl.name, "P": None if adaptive else P, "beta1": beta1,
                   "beta2": beta2,
                   "n_tensors": len(wl.tensors), "elements": wl.numel,
                   "muon_elements": info_muon["muon_elements"],
                   "ns_precision": wl.ns_precision, "ns_steps": 5,
                   "state": "fp32 W, M, G; bf16 MFMA Newton-Schulz with fp32 accumulation"},
    }
    if adaptive:
        out["metric"] = "optimizer-step ms (adaptive LionMuon step, Appendix G rule, 1 GPU)"
        out["config"].update({"rule": "adaptive stable rank", "alpha": args.adaptive,
                              "power_steps": args.power_steps,
                              "muon_fraction_after_timing": muon_fraction})
    if phases is not None:
        flops = ns_flops_per_launch(wl)
        ph = {}
        for name, v in phases.items():
            if v["launches"] == 0:
                continue
            avg = v["ms"] / v["launches"]
            entry = {"launches": v["launches"], "avg_ms": round(avg, 5)}
            if name in flops and not adaptive:   # adaptive: NS work depends on the decisions
                entry["tflops"] = round(flops[name] / (avg * 1e-3) / 1e12, 1)
                entry["frac_bf16_peak"] = round(entry["tflops"] / BF16_PEAK_TFLOPS, 4)
            if name == "srank":
                entry["gbps"] = round(info_adaptive["srank_bytes"] / (avg * 1e-3) / 1e9, 1)
                entry["frac_hbm_peak"] = round(entry["gbps"] / HBM_PEAK_GBPS, 4)
            if name == "lion" and not adaptive:
                # Lion steps update every tensor; Muon steps only the Lion-only ones
                lion_elems = n_lion_steps * info_lion["lion_elements"]
                if n_muon_steps and info_muon["lion_elements"]:
                    lion_elems += n_muon_steps * info_muon["lion_elements"]
                bytes_launch = 20.0 * lion_elems / v["launches"]
                entry["gbps"] = round(bytes_launch / (avg * 1e-3) / 1e9, 1)
                entry["frac_hbm_peak"] = round(entry["gbps"] / HBM_PEAK_GBPS, 4)
            ph[name] = entry
        out["phases"] = ph
        ns_ms = sum(phases[p]["ms"] for p in ("gram", "poly", "apply"))
        if n_muon_steps:
            out["ns_tflops"] = round(info_muon["ns_flops"] * n_muon_steps / (ns_ms * 1e-3) / 1e12, 1)
            out["ns_frac_bf16_peak"] = round(out["ns_tflops"] / BF16_PEAK_TFLOPS, 4)
            out["ns_tflops_dense_convention"] = round(
                info_muon["ns_flops_dense"] * n_muon_steps / (ns_ms * 1e-3) / 1e12, 1)
            out["ns_ms_per_muon_step"] = round(ns_ms / n_muon_steps, 4)
        if not adaptive:
            # time split of the two step kinds and the amortisation cross-check
            # ((P-1) T_lion + T_muon) / P against the measured ms/step
            lion_ms = phases["lion"]["ms"]
            muon_ms = sum(phases[p]["ms"] for p in ("prep", "norm", "gram", "poly", "apply"))
            split = {}
            if n_lion_steps:
                lion_only_ms = 0.0
                if n_muon_steps and info_muon["lion_elements"] and phases["lion"]["launches"]:
                    # Lion-only tensors on Muon steps: pro rata by element count
                    per_elem = lion_ms / (n_lion_steps * info_lion["lion_elements"]
                                          + n_muon_steps * info_muon["lion_elements"])
                    lion_only_ms = per_elem * n_muon_steps * info_muon["lion_elements"]
                split["t_lion_ms"] = round((lion_ms - lion_only_ms) / n_lion_steps, 4)
                muon_ms += lion_only_ms
            if n_muon_steps:
                split["t_muon_ms"] = round(muon_ms / n_muon_steps, 4)
            if len(split) == 2 or P in (0, 1):
                tl, tm = split.get("t_lion_ms", 0.0), split.get("t_muon_ms", 0.0)
                split["amortised_from_split_ms"] = round(
                    tl if P == 0 else ((P - 1) * tl + tm) / P, 4)
            out["split"] = split
        if "lion" in ph and "gbps" in ph["lion"]:
            out["lion_gbps"] = ph["lion"]["gbps"]
            out["lion_frac_hbm_peak"] = ph["lion"]["frac_hbm_peak"]
        # dominant kernel: most total time in the timed region
        dom = max((p for p in phases if phases[p]["launches"]), key=lambda p: phases[p]["ms"])
        d = ph[dom]
        kernel_names = {"lion": "lion_kernel", "prep": "prep_kernel", "norm": "norm_kernel",
                        "gram": "ns_gram_kernel<bf16>", "poly": "ns_poly_kernel<bf16>",
                        "apply": "ns_apply_kernel<bf16> (+ ns_apply_last_kernel)", "srank": "srank_pass+reduce+decide"}
        if "tflops" in d:
            roof = {"kernel": kernel_names[dom], "bound": "mfma", "achieved": d["tflops"],
                    "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s", "frac": d["frac_bf16_peak"]}
        elif "gbps" in d:
            roof = {"kernel": kernel_names[dom], "bound": "hbm", "achieved": d["gbps"],
                    "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": d["frac_hbm_peak"]}
        else:
            roof = {"kernel": kernel_names[dom], "bound": "hbm", "achieved": None,
                    "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": None}
        roof["avg_launch_ms"] = d["avg_ms"]
        roof["traffic"] = load_traffic(prof_name, dom)
        out["roofline"] = roof
    if not args.no_cpu_baseline and not adaptive:
        out["cpu_baseline"] = cpu_baseline(wl, P)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
