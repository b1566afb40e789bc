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


SIMDS = 1024                      # 256 CUs x 4 SIMDs
XCDS = 8


def sq_summary(wl_name, sq_csvs, command):
    assert len(sq_csvs) == 1, "one counter pass"
    """MFMA issue and utilisation of each Newton-Schulz phase from rocprofv3
    counter passes (one CSV per pass; per-dispatch durations from the CSV's
    timestamps), against the phase's algorithmic flops: issued flops = 512
    SQ_INSTS_VALU_MFMA_MOPS_BF16 (F32 for fp32 products)."""
    import collections
    import csv
    wl = workloads.get(wl_name.replace("-adaptive", ""))
    algo = ns_flops_per_launch(wl)
    fp32 = wl.ns_precision == "fp32"
    peak_tflops = FP32_MFMA_PEAK_TFLOPS if fp32 else BF16_PEAK_TFLOPS
    # per phase: counter sums, per-dispatch durations and dispatch counts
    cnt = collections.defaultdict(lambda: collections.defaultdict(float))
    dur = collections.defaultdict(dict)          # phase -> {(pass, dispatch): ns}
    n256 = collections.defaultdict(set)
    nall = collections.defaultdict(set)
    for k, path in enumerate(sq_csvs):
        for r in csv.DictReader(open(path)):
            ph = phase_of(r["Kernel_Name"])
            if ph is None:
                continue
            key = (k, int(r["Dispatch_Id"]))
            cnt[ph][r["Counter_Name"]] += float(r["Counter_Value"])
            dur[ph][key] = float(r["End_Timestamp"]) - float(r["Start_Timestamp"])
            nall[ph].add(key)
            if "Li256" in r["Kernel_Name"]:
                n256[ph].add(key)
    lines = [f"# MFMA issue and utilisation: {wl_name}", "", f"Command: `{command}`", "",
             "Per Newton-Schulz phase launch (the apply's launch includes its small-tile tail "
             "and last-step kernels), from one counter pass (dispatches serialised; durations "
             "from the pass's own timestamps).", "",
             "- `algorithmic frac`: the phase's symmetric flop count (Gram s(s+1)l, polynomial "
             "s^2(s+1), apply 2 s^2 l per matrix) over the launch duration, against the dense "
             "MFMA peak of the path's type: bf16 2516.6 TFLOP/s (256 CUs x 2.4 GHz x 4096 "
             "flop/clk), fp32 157.3 TFLOP/s" + (" (this workload: fp32)." if fp32 else "."),
             "- `issued frac`: 512 x SQ_INSTS_VALU_MFMA_MOPS_BF16 (+_F32) flops over the same "
             "duration and peak: the MFMA work the kernels actually execute.",
             "- `issued / algorithmic`: MFMA work spent per useful flop. Above 1 where a "
             "symmetric product computes its diagonal tiles in full and where padding to the "
             "tile edge adds rows.",
             "- `MFMA util`: SQ_VALU_MFMA_BUSY_CYCLES / (cycles x 1024 SIMDs), with cycles = "
             "GRBM_GUI_ACTIVE / 8 (the counter is summed over the 8 XCDs and also covers the "
             "collection window around the dispatch). The busy cycles are the issued MOPS / 2 "
             "exactly (one 32x32x16 bf16 MFMA: 64 MOPS, 32 busy cycles), so this is the issued "
             "work in cycles, not a separate measurement; it differs from `issued frac` only "
             "by the clock.",
             "- `clock GHz`: GRBM_GUI_ACTIVE / 8 / duration, an upper bound (collection window).",
             "- `wait`: SQ_WAIT_ANY / SQ_WAVE_CYCLES; `LDS conflict`: SQ_LDS_BANK_CONFLICT / "
             "SQ_LDS_IDX_ACTIVE.", "",
             "| phase | launches | avg us | algorithmic frac | issued frac | issued / algorithmic "
             "| MFMA util | clock GHz | wait | LDS conflict |",
             "|---|---|---|---|---|---|---|---|---|---|"]
    for ph in ("gram", "poly", "apply"):
        if ph not in cnt:
            continue
        c = cnt[ph]
        launches = len(n256[ph]) or len(nall[ph])
        t_ns = sum(dur[ph].values()) / launches
        issued = 512.0 * (c.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0) +
                          c.get("SQ_INSTS_VALU_MFMA_MOPS_F32", 0.0)) / launches
        peak = peak_tflops * 1e12 * t_ns * 1e-9
        cycles = c.get("GRBM_GUI_ACTIVE", 0.0) / XCDS / launches
        util = c.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) / launches / (cycles * SIMDS) if cycles else 0.0
        clock = cycles / t_ns if t_ns else 0.0
        wt = c["SQ_WAIT_ANY"] / c["SQ_WAVE_CYCLES"] if c.get("SQ_WAVE_CYCLES") else float("nan")
        lc = (c["SQ_LDS_BANK_CONFLICT"] / c["SQ_LDS_IDX_ACTIVE"]
              if c.get("SQ_LDS_IDX_ACTIVE") else float("nan"))
        lines.append(
            f"| {ph} | {launches} | {t_ns / 1e3:.1f} | {algo[ph] / peak:.3f} | {issued / peak:.3f} | "
            f"{issued / algo[ph]:.3f} | {util:.3f} | {clock:.2f} | {wt:.3f} | {lc:.3f} |")
    path = os.path.join(TRAFFIC_DIR, f"sq_{wl_name}.md")
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")
    return path


def launch_gaps(trace_csv):
    """Idle time between consecutive library kernels in a rocprofv3 kernel
    trace, over gaps shorter than 50 us (longer ones are host-side pauses
    between timed regions). Gaps under 0.5 us are counted apart: inside one
    call without per-launch events the next kernel's start stamp is the
    previous one's end (the dispatch cost falls inside the kernel durations);
    the others follow the event records of the library (at the end of every
    call, and around every launch while per-launch profiling is on)."""
    import csv
    ev = sorted((int(r["Start_Timestamp"]), int(r["End_Timestamp"]))
                for r in csv.DictReader(open(trace_csv)) if phase_of(r["Kernel_Name"]))
    gaps = [b[0] - a[1] for a, b in zip(ev, ev[1:]) if 0 <= b[0] - a[1] < 50000]
    rest = [x for x in gaps if x >= 500]
    busy = sum(e - s for s, e in ev)
    return {"launches": len(ev), "gaps": len(gaps), "zero": len(gaps) - len(rest),
            "rest": len(rest), "mean_rest_us": sum(rest) / len(rest) / 1e3 if rest else 0.0,
            "gap_share": sum(gaps) / (sum(gaps) + busy) if ev else 0.0}


# order of the phases within one call: a dispatch whose phase comes earlier
# than the previous dispatch's (or repeats a phase launched once per call)
# starts the next call
_CALL_ORDER = {"srank": 0, "lion": 1, "prep": 2, "norm": 3, "gram": 4, "poly": 4, "apply": 4}


def _split_calls(ev, prep_starts):
    calls, prev = [], None
    for s, e, name in ev:
        rank = _CALL_ORDER[phase_of(name)]
        if (prev is None or rank < prev or (rank == prev and rank in (1, 2, 3))
                or (prep_starts and rank == 2)):
            calls.append([])
        calls[-1].append((name, e - s))
        prev = rank
    return calls


def profiled_dispatches(trace_csv, warmup, steps, trailing, lion_in_muon=None):
    """Library dispatches of the profiled steps of one bench run, read from
    its rocprofv3 kernel trace. A `--single` run makes `warmup` calls, `steps`
    timed calls with per-launch events off, `steps` with them on (the
    profiled ones) and `trailing` more. With `warmup` None the run is the
    default one (every configuration, the headline last): its profiled steps
    are its last `steps` calls, and `lion_in_muon` tells whether the headline
    set's Muon calls start with the Lion kernel (a set with Lion-branch
    tensors) or with the preparation kernel. Returns [(kernel name, duration
    ns)], or None when the trace does not split into that many calls."""
    import csv
    ev = sorted((int(r["Start_Timestamp"]), int(r["End_Timestamp"]), r["Kernel_Name"])
                for r in csv.DictReader(open(trace_csv)) if phase_of(r["Kernel_Name"]))
    if warmup is None:
        calls = _split_calls(ev, prep_starts=not lion_in_muon)
        if len(calls) < steps + trailing:
            return None
        return [d for c in calls[len(calls) - trailing - steps:len(calls) - trailing] for d in c]
    # A Muon call starts with the Lion kernel when the list has Lion-branch
    # tensors, else with the preparation kernel: try the second reading when
    # the first does not give the run's number of calls.
    for prep_starts in (False, True):
        calls = _split_calls(ev, prep_starts)
        if len(calls) == warmup + 2 * steps + trailing:
            return [d for c in calls[warmup + steps:warmup + 2 * steps] for d in c]
    return None


def trace_summary(wl_name, stats_csv, command, trace_csv=None, calls=None, file_tag=None):
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
    # the same over the profiled steps only (per-launch events on: the
    # region whose per-launch times bench.py reports), after the clock under
    # load has settled; the whole run includes the first, slower steps
    prof = {}
    for name, ns in ((profiled_dispatches(trace_csv, *calls) if trace_csv and calls else None)
                     or []):
        t = prof.setdefault(phase_of(name), {"ns": 0.0, "n_all": 0, "n_256": 0, "n_decide": 0})
        t["ns"] += ns
        t["n_all"] += 1
        t["n_256"] += "Li256" in name
        t["n_decide"] += "srank_decide" in name

    def per_launch(ph, t):
        n = t["n_decide"] if ph == "srank" else (t["n_256"] or t["n_all"])
        return n, t["ns"] / n / 1e3

    scope = ("over the whole run (every configuration of the default run, so the first "
             "columns mix the sets) and over the headline's profiled steps (its last timed "
             "region, per-launch events on, whose per-launch times the bench line reports)"
             if file_tag == "default_run" else
             "over the whole run and over the profiled steps (the last timed region, "
             "per-launch events on, the one whose per-launch times bench.py reports)")
    lines += ["", "Per phase launch (all of a phase's kernels; launches = its 256-tile dispatches "
              f"where there are any, the decide dispatches for srank), {scope}:", "",
              "| phase | launches | avg us per launch | profiled launches | avg us per launch, "
              "profiled steps |", "|---|---|---|---|---|"]
    for ph, t in sorted(tot.items(), key=lambda kv: -kv[1]["ns"]):
        n, avg = per_launch(ph, t)
        pn, pavg = per_launch(ph, prof[ph]) if ph in prof else (0, float("nan"))
        lines.append(f"| {ph} | {n} | {avg:.1f} | {pn} | {pavg:.1f} |")
    if trace_csv:
        g = launch_gaps(trace_csv)
        lines += ["", f"Between consecutive library kernels (per-dispatch timestamps, {g['launches']} "
                  f"dispatches, {g['gaps']} back-to-back pairs): {g['zero']} pairs with no idle "
                  f"time (within a call, per-launch events off), {g['rest']} pairs with a mean gap of "
                  f"{g['mean_rest_us']:.2f} us (after the end-of-call event records, and around "
                  f"every launch while per-launch events are on); all gaps together "
                  f"{100 * g['gap_share']:.1f}% of the kernels' timeline."]
    path = os.path.join(TRAFFIC_DIR, f"kernel_trace_{file_tag or wl_name}.md")
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


def cpu_oracle_times(wl, budget_s=10.0):
    """fp64 oracle on a bounded sample: one Lion step and one Muon step on one
    tensor of every distinct shape, scaled to the whole set by tensor count,
    repeated until about `budget_s` seconds of CPU work (at least once) and
    averaged over the repetitions. Returns (T_lion, T_muon) in seconds per
    step and a description of the sample."""
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
            oracle.lionmuon_update(W, G, M, 1, 2, wl.beta1, wl.beta2, wl.lr_muon, wl.lr_lion,
                                   wl.wd, lion_only=True)
            t1 = time.perf_counter()
            oracle.lionmuon_update(W, G, M, 0, 1, wl.beta1, wl.beta2, wl.lr_muon, wl.lr_lion,
                                   wl.wd, lion_only=t.lion_only)
            t2 = time.perf_counter()
            t_lion += (t1 - t0) * reps
            t_muon += (t2 - t1) * reps
        rounds += 1
    spent = time.perf_counter() - start
    desc = (f"one Lion and one Muon fp64 oracle step on one tensor of each of the "
            f"{len(sample)} distinct shapes of {wl.name}, scaled by tensor count, "
            f"repeated {rounds}x ({spent:.1f} s of CPU work) and averaged")
    return t_lion / rounds, t_muon / rounds, int(cores), desc


def cpu_baseline_for(times, P):
    """The oracle's amortised ms/step at period P (0 = pure Lion) from the
    sampled step times of cpu_oracle_times."""
    t_lion, t_muon, cores, desc = times
    amort = t_lion if P == 0 else ((P - 1) * t_lion + t_muon) / P
    return {"value": round(amort * 1e3, 1), "unit": "ms/step", "cores": cores, "kind": "oracle",
            "sample": (f"{desc}; Lion {t_lion * 1e3:.0f} ms/step, Muon {t_muon * 1e3:.0f} ms/step, "
                       f"amortised over P={P}")}


KERNEL_NAMES = {"lion": "lion_kernel", "prep": "prep_kernel", "norm": "norm_kernel",
                "gram": "ns_gram_kernel<bf16>", "poly": "ns_poly_kernel<bf16>",
                "apply": "ns_apply_kernel<bf16> (+ ns_apply_last_kernel)",
                "srank": "srank_pass+reduce+decide"}


class Bench:
    """Device state of one workload and timed runs of the step over it."""

    def __init__(self, torch, lm, wl, n_grad=2):
        self.torch, self.lm, self.wl = torch, lm, wl
        self.dev = torch.device("cuda:0")
        self.params, self.moms, self.grad_sets = workloads.device_state(
            torch, wl, self.dev, seed=7, warm=True, n_grad=n_grad)
        lion_only = [t.lion_only for t in wl.tensors]
        self.lists = [lm.TensorList(self.params, g, self.moms, lion_only) for g in self.grad_sets]
        self.specs = [(t.rows, t.cols, t.lion_only) for t in wl.tensors]
        self.stream = torch.cuda.current_stream()

    def close(self, release=True):
        """Free the device state; with `release`, also the library's plans
        and workspaces and torch's cached blocks (the next call rebuilds its
        plan; both take host-side waits during which the GPU idles)."""
        del self.lists, self.params, self.moms, self.grad_sets
        if release:
            self.lm.lionmuon_release()
        self.torch.cuda.synchronize()
        if release:
            self.torch.cuda.empty_cache()

    def run(self, t0, n, P, beta1, beta2, cfg, n_lists=None):
        k_lists = n_lists or len(self.lists)
        for k in range(n):
            t = t0 + k
            self.lm.lionmuon_step_ex(None, None, None, t, P, beta1, beta2, self.wl.wd, cfg,
                                     stream=self.stream, tensors=self.lists[t % k_lists])

    def measure(self, P, steps, warmup, beta1=None, beta2=None, adaptive=0.0, power_steps=5,
                profile=True, n_lists=None):
        """Amortised ms/step over `steps` timed steps (whole periods, the first
        a Muon step) after `warmup` untimed ones, with the library's
        per-launch events off; then, with `profile`, the same number of steps
        again with the events on for the per-phase times, the split and the
        roofline of the dominant kernel."""
        torch, lm, wl = self.torch, self.lm, self.wl
        beta1 = wl.beta1 if beta1 is None else beta1
        beta2 = wl.beta2 if beta2 is None else beta2
        adaptive_on = adaptive > 0.0
        if P > 1 and steps % P and not adaptive_on:
            steps += P - steps % P                 # whole periods only
        cfg = lm.config(ns_precision=wl.ns_precision, lr_muon=wl.lr_muon, lr_lion=wl.lr_lion,
                        adaptive_alpha=adaptive, adaptive_power_steps=power_steps)
        cfg_period = lm.config(ns_precision=wl.ns_precision, lr_muon=wl.lr_muon,
                               lr_lion=wl.lr_lion)
        info_muon = lm.lionmuon_plan_info(self.specs, 0, 1, cfg_period)
        info_lion = lm.lionmuon_plan_info(self.specs, 1, 2, cfg_period)
        info_adaptive = lm.lionmuon_plan_info(self.specs, 0, 0, cfg) if adaptive_on else None
        stream = self.stream
        self.run(1, warmup, P, beta1, beta2, cfg, n_lists)
        torch.cuda.synchronize()
        t_start = 1 + warmup
        t_start += (-t_start) % max(P, 1)         # timed region starts on a Muon step
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        self.run(t_start, steps, P, beta1, beta2, cfg, n_lists)
        e1.record(stream)
        torch.cuda.synchronize()
        ms_step = e0.elapsed_time(e1) / steps
        out = {"ms_per_step": round(ms_step, 4), "steps": steps, "P": None if adaptive_on else P,
               "beta1": beta1, "beta2": beta2}
        if not profile:
            return out
        lm.lionmuon_profiling_reset()
        lm.lionmuon_profiling_enable(True)
        self.run(t_start + steps, steps, P, beta1, beta2, cfg, n_lists)
        torch.cuda.synchronize()
        phases = lm.lionmuon_profiling_read()
        lm.lionmuon_profiling_enable(False)
        if adaptive_on:
            dec = torch.zeros(len(wl.tensors), dtype=torch.int32, device=self.dev)
            lm.lionmuon_step_adaptive(None, None, None, t_start + 2 * steps, beta1, beta2, wl.wd,
                                      cfg, stream=stream, tensors=self.lists[0], decisions=dec)
            torch.cuda.synchronize()
            out["muon_fraction_after_timing"] = round(float(dec.sum().item()) /
                                                      info_adaptive["n_muon"], 4)
            n_muon_steps = 0
        else:
            n_muon_steps = sum(1 for k in range(steps) if P >= 1 and (t_start + k) % P == 0)
        n_lion_steps = steps - n_muon_steps
        flops = ns_flops_per_launch(wl)
        peak_mfma = BF16_PEAK_TFLOPS if wl.ns_precision == "bf16" else FP32_MFMA_PEAK_TFLOPS
        ph = {}
        for name, v in phases.items():
            if v["launches"] == 0:
                continue
            avg = v["ms"] / v["launches"]
            entry = {"launches": v["launches"], "avg_ms": round(avg, 5)}
            if name in flops and not adaptive_on:   # adaptive: NS work depends on the decisions
                entry["tflops"] = round(flops[name] / (avg * 1e-3) / 1e12, 1)
                entry["frac_mfma_peak"] = round(entry["tflops"] / peak_mfma, 4)
            if name == "srank":
                entry["gbps"] = round(info_adaptive["srank_bytes"] / (avg * 1e-3) / 1e9, 1)
                entry["frac_hbm_peak"] = round(entry["gbps"] / HBM_PEAK_GBPS, 4)
            if name == "lion" and not adaptive_on:
                # Lion steps update every tensor; Muon steps only the Lion-only ones
                lion_elems = n_lion_steps * info_lion["lion_elements"]
                if n_muon_steps and info_muon["lion_elements"]:
                    lion_elems += n_muon_steps * info_muon["lion_elements"]
                bytes_launch = 20.0 * lion_elems / v["launches"]
                entry["gbps"] = round(bytes_launch / (avg * 1e-3) / 1e9, 1)
                entry["frac_hbm_peak"] = round(entry["gbps"] / HBM_PEAK_GBPS, 4)
            if name == "prep" and not adaptive_on:
                entry["gbps"] = round(14.0 * info_muon["muon_elements"] / (avg * 1e-3) / 1e9, 1)
                entry["frac_hbm_peak"] = round(entry["gbps"] / HBM_PEAK_GBPS, 4)
            ph[name] = entry
        out["phases"] = ph
        ns_ms = sum(phases[p]["ms"] for p in ("gram", "poly", "apply"))
        if n_muon_steps:
            out["ns_tflops"] = round(info_muon["ns_flops"] * n_muon_steps / (ns_ms * 1e-3) / 1e12, 1)
            out["ns_frac_mfma_peak"] = round(out["ns_tflops"] / peak_mfma, 4)
            out["ns_tflops_dense_convention"] = round(
                info_muon["ns_flops_dense"] * n_muon_steps / (ns_ms * 1e-3) / 1e12, 1)
            out["ns_ms_per_muon_step"] = round(ns_ms / n_muon_steps, 4)
        if not adaptive_on:
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
        kname = KERNEL_NAMES[dom]
        if wl.ns_precision != "bf16":
            kname = kname.replace("<bf16>", "<float>")
        if "tflops" in d:
            roof = {"kernel": kname, "bound": "mfma", "achieved": d["tflops"],
                    "peak": peak_mfma, "unit": "TFLOP/s", "frac": d["frac_mfma_peak"]}
        elif "gbps" in d:
            roof = {"kernel": kname, "bound": "hbm", "achieved": d["gbps"],
                    "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": d["frac_hbm_peak"]}
        else:
            roof = {"kernel": kname, "bound": "hbm", "achieved": None,
                    "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": None}
        roof["avg_launch_ms"] = d["avg_ms"]
        roof["traffic"] = load_traffic(wl.name + ("-adaptive" if adaptive_on else ""), dom)
        out["roofline"] = roof
        return out


def workload_config(wl, info):
    return {"workload": wl.name, "n_tensors": len(wl.tensors), "elements": wl.numel,
            "muon_elements": info["muon_elements"], "ns_precision": wl.ns_precision,
            "ns_steps": 5, "gradients": wl.grad_dist,
            "state": "fp32 W, M, G; " + ("bf16 MFMA Newton-Schulz with fp32 accumulation"
                                         if wl.ns_precision == "bf16"
                                         else "fp32 MFMA Newton-Schulz")}


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
    ap.add_argument("--single", action="store_true",
                    help="only the selected workload and period (no other configurations)")
    ap.add_argument("--grad-sets", type=int, default=2,
                    help="gradient sets the steps rotate through (1 = fixed addresses)")
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
    ap.add_argument("--sq-summary", nargs=1, metavar="SQ_CSV",
                    help="write profiles/sq_<workload>.md from one rocprofv3 SQ counter pass")
    ap.add_argument("--command", default="", help="profiling command recorded in summaries")
    args = ap.parse_args()
    # profiles of the adaptive variant are kept apart from the periodic step's
    prof_name = args.workload + ("-adaptive" if args.adaptive > 0.0 else "")
    if args.pmc_summary:
        print(pmc_summary(prof_name, *args.pmc_summary, calib_mib=1024,
                          commands=args.command))
        return
    if args.trace_summary:
        trace_csv = args.trace_summary.replace("kernel_stats.csv", "kernel_trace.csv")
        # the profiled run's calls: warm-up, timed, profiled (whole periods)
        # and, for the adaptive variant, one more step that reads decisions
        steps = args.steps
        if args.P > 1 and steps % args.P and args.adaptive <= 0.0:
            steps += args.P - steps % args.P
        calls = (args.warmup, steps, 1 if args.adaptive > 0.0 else 0)
        tag = None
        if not args.single and args.adaptive <= 0.0:
            # the default command: the headline's profiled steps end the run
            wl = workloads.get(args.workload)
            lion_in_muon = any(t.lion_only or t.rows == 1 for t in wl.tensors)
            calls = (None, steps, 0, lion_in_muon)
            tag = "default_run"
        print(trace_summary(prof_name, args.trace_summary, args.command,
                            trace_csv if os.path.exists(trace_csv) else None, calls, tag))
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

    def log(msg):
        print(f"[bench] {msg}", file=sys.stderr, flush=True)

    profile = not args.no_profile
    wl = workloads.get(args.workload)
    P = 1 if args.pure_muon else args.P
    beta = (0.9, 0.9) if args.pure_muon else (None, None)
    adaptive = args.adaptive > 0.0
    cpu = not args.no_cpu_baseline and not adaptive
    b = Bench(torch, lm, wl, n_grad=max(1, args.grad_sets))
    configs = None
    if not args.single and not adaptive:
        # The other configurations run first and the headline's steps follow
        # their GPU work at once: after an idle spell (a fresh process, the
        # host-side set-up of a workload, or the allocation of a new plan's
        # workspace) the core clock needs ~20 ms of sustained MFMA load to
        # settle (the first 124M Muon steps take up to ~2.1 ms, the tenth
        # ~1.7; Lion steps, bound by HBM, do not change), which would
        # otherwise fall inside the headline's 20 timed steps.
        configs = other_configs(torch, lm, args, wl.name, P, profile, cpu, log)
    log(f"{wl.name} P={P}{' adaptive' if adaptive else ''}")
    res = b.measure(P, args.steps, args.warmup, beta[0], beta[1], args.adaptive,
                    args.power_steps, profile)
    info = lm.lionmuon_plan_info(b.specs, 0, 1, lm.config(ns_precision=wl.ns_precision))
    b.close()
    out = {
        "metric": "amortised optimizer-step ms per period P (LionMuon step, 1 GPU)",
        "value": res["ms_per_step"],
        "unit": "ms/step",
        "n_gpus": 1,
        "steps": res["steps"],
        "warmup": args.warmup,
        "ms_per_step": res["ms_per_step"],
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.ns_precision == "bf16" else "f32",
        "data": "synthetic (seeded gradients of the workload's shapes; random-init weights)",
        "config": dict(workload_config(wl, info), P=res["P"], beta1=res["beta1"],
                       beta2=res["beta2"], grad_sets=args.grad_sets),
    }
    if adaptive:
        out["metric"] = "optimizer-step ms (adaptive LionMuon step, Appendix G rule, 1 GPU)"
        out["config"].update({"rule": "adaptive stable rank", "alpha": args.adaptive,
                              "power_steps": args.power_steps,
                              "muon_fraction_after_timing": res.get("muon_fraction_after_timing")})
    for k in ("phases", "ns_tflops", "ns_frac_mfma_peak", "ns_tflops_dense_convention",
              "ns_ms_per_muon_step", "split", "lion_gbps", "lion_frac_hbm_peak", "roofline"):
        if k in res:
            out[k] = res[k]
    if cpu:
        log("cpu baseline")
        out["cpu_baseline"] = cpu_baseline_for(cpu_oracle_times(wl, 10.0), P)
    if configs is not None:
        out["configs"] = configs
    print(json.dumps(out), flush=True)


def other_configs(torch, lm, args, main_name, main_P, profile, cpu, log):
    """Every other configuration the metric names, measured with the same
    step counts: the 355M and 720M sets at P = 2, the 768 x 768 fp32 case,
    the 355M period sweep (P = 1, 2, 4, 8, infinity and pure Muon), and the
    headline set with fixed gradient addresses against four rotating sets."""
    keep = ("ms_per_step", "steps", "P", "beta1", "beta2", "ns_tflops", "ns_frac_mfma_peak",
            "ns_tflops_dense_convention", "ns_ms_per_muon_step", "lion_gbps",
            "lion_frac_hbm_peak", "split", "roofline", "phases")
    out = {}

    def pick(res):
        return {k: res[k] for k in keep if k in res}

    for name in ("gpt2-355m", "gpt2-720m", "single768"):
        if name == main_name:
            continue
        wl = workloads.get(name)
        sweep = name == "gpt2-355m"
        log(f"{name}{' + period sweep' if sweep else ''}")
        b = Bench(torch, lm, wl, n_grad=2)
        info = lm.lionmuon_plan_info(b.specs, 0, 1, lm.config(ns_precision=wl.ns_precision))
        entry = dict(config=workload_config(wl, info), **pick(b.measure(wl.P, args.steps,
                                                                        args.warmup,
                                                                        profile=profile)))
        runs = {}
        if sweep:
            for label, Pp, beta in (("P=1", 1, None), ("P=4", 4, None), ("P=8", 8, None),
                                    ("P=inf (pure Lion)", 0, None),
                                    ("pure Muon (P=1, beta1=beta2=0.9)", 1, 0.9)):
                log(f"{name} {label}")
                runs[label] = pick(b.measure(Pp, args.steps, args.warmup, beta, beta,
                                             profile=profile))
        b.close()
        if cpu:
            log(f"{name} cpu baseline")
            times = cpu_oracle_times(wl, 6.0)
            entry["cpu_baseline"] = cpu_baseline_for(times, wl.P)
            for label, r in runs.items():
                r["cpu_baseline"] = cpu_baseline_for(times, r["P"] or 0)
        if sweep:
            runs["P=2"] = {k: entry[k] for k in entry if k != "config"}
            out["period_sweep_gpt2-355m"] = {
                "config": entry["config"],
                "note": "amortised ms/step per period; split = T_lion, T_muon per step kind",
                "runs": {k: runs[k] for k in ("P=1", "P=2", "P=4", "P=8", "P=inf (pure Lion)",
                                              "pure Muon (P=1, beta1=beta2=0.9)")}}
        out[name] = entry
    # gradient addresses: fixed (one set) against four rotating sets, which
    # give the library new addresses on every step
    wl = workloads.get(main_name)
    log(f"{main_name} fixed vs rotating gradient addresses")
    b = Bench(torch, lm, wl, n_grad=4)
    # at least 100 steps per region (a 2% comparison), the two modes
    # alternated twice, the faster region of each mode kept
    n_addr = max(args.steps, 100)
    fixed, rot = [], []
    for _ in range(2):
        fixed.append(b.measure(main_P, n_addr, args.warmup, profile=False, n_lists=1)["ms_per_step"])
        rot.append(b.measure(main_P, n_addr, args.warmup, profile=False, n_lists=4)["ms_per_step"])
    # (the headline set's plans and torch's blocks stay: the headline's steps
    # then follow this GPU work without an idle spell of plan building or of
    # returning memory, during which the clock would drop)
    b.close(release=False)
    out[f"gradient_addresses_{main_name}"] = {
        "fixed_ms_per_step": min(fixed), "rotating4_ms_per_step": min(rot),
        "ratio": round(min(rot) / min(fixed), 4), "steps": n_addr, "regions": {"fixed": fixed,
                                                                           "rotating4": rot},
        "note": "same steps with one gradient set (addresses never change) and with four sets "
                "used in turn (new addresses every step: the library rewrites its per-call "
                "address table on the stream); two regions of each, alternated, the faster kept"}
    return out


if __name__ == "__main__":
    main()
