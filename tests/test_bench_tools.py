"""Host-side tools of bench.py that read rocprofv3 kernel traces: the split of
a traced run into its calls (whose last timed region gives the per-launch
times the bench line reports) and the gap statistics between kernels.
Synthetic traces only; no GPU."""
import csv
import os
import sys

import pytest

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402

LION = "lm::(anonymous namespace)::lion_kernel(lm::(anonymous namespace)::LionArgs)"
PREP = "lm::(anonymous namespace)::prep_kernel(lm::(anonymous namespace)::PrepArgs)"
NORM = "lm::(anonymous namespace)::norm_kernel(lm::(anonymous namespace)::PrepArgs)"
GRAM = "_ZN2lm12_GLOBAL__N_114ns_gram_kernelIDF16bLi256EEEvNS0_8GemmArgsE"
POLY = "_ZN2lm12_GLOBAL__N_114ns_poly_kernelIDF16bLi128EEEvNS0_8GemmArgsE"
APPLY = "_ZN2lm12_GLOBAL__N_120ns_apply_pair_kernelIDF16bLi256ELi64ELb0EEEvN"
LAST = "_ZN2lm12_GLOBAL__N_120ns_apply_pair_kernelIDF16bLi256ELi64ELb1EEEvN"
SRANK = ["lm::(anonymous namespace)::srank_tall_kernel", "lm::(anonymous namespace)::srank_reduce_kernel",
         "lm::(anonymous namespace)::srank_decide_kernel"]
TORCH = "void at::native::vectorized_elementwise_kernel<4>"


def muon_call(lion_first):
    ns = [k for _ in range(4) for k in (GRAM, POLY, APPLY)] + [GRAM, POLY, LAST]
    return ([LION] if lion_first else []) + [PREP, NORM] + ns


def write_trace(path, calls, evented_from, evented_to, foreign_every=0):
    """Kernels of `calls` back to back: no gap inside a call without events,
    8 us after each call, 7.7 us between any two kernels of the calls in
    [evented_from, evented_to). Each kernel's duration encodes its call index
    (1000 + index ns), so a test can tell which calls a selection holds."""
    t, rows, n = 10_000, [], 0
    for ci, call in enumerate(calls):
        evented = evented_from <= ci < evented_to
        for k, name in enumerate(call):
            if k and evented:
                t += 7_700
            rows.append({"Kernel_Name": name, "Start_Timestamp": t, "End_Timestamp": t + 1000 + ci})
            t += 1000 + ci
            n += 1
            if foreign_every and n % foreign_every == 0:   # a torch kernel in between
                rows.append({"Kernel_Name": TORCH, "Start_Timestamp": t, "End_Timestamp": t + 500})
                t += 500
        t += 8_000
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        w.writeheader()
        w.writerows(rows)


def period_calls(n, first_t, P, lion_first):
    return [muon_call(lion_first) if (first_t + i) % P == 0 else [LION] for i in range(n)]


@pytest.mark.parametrize("lion_first", [False, True])
def test_profiled_steps_of_a_periodic_run(tmp_path, lion_first):
    # warm-up t = 1..5, timed t = 6..25, profiled t = 26..45, as bench.py runs them at P = 2
    warmup, steps = 5, 20
    calls = period_calls(warmup + 2 * steps, 1, 2, lion_first)
    path = str(tmp_path / "trace.csv")
    write_trace(path, calls, warmup + steps, warmup + 2 * steps, foreign_every=7)
    got = bench.profiled_dispatches(path, warmup, steps, 0)
    want = [(name, 1000 + ci) for ci in range(warmup + steps, warmup + 2 * steps)
            for name in calls[ci]]
    assert got == want


@pytest.mark.parametrize("lion_first", [False, True])
def test_profiled_steps_of_the_default_run(tmp_path, lion_first):
    # the default run measures the other sets first (Muon calls starting
    # with the preparation kernel, with the Lion kernel, pure Lion calls) and
    # the headline set last; its profiled steps are the run's last 20 calls
    others = (period_calls(45, 1, 2, False) + period_calls(45, 1, 2, True) + [[LION]] * 45
              + period_calls(45, 1, 1, False))
    head = period_calls(45, 1, 2, lion_first)
    calls = others + head
    path = str(tmp_path / "trace.csv")
    write_trace(path, calls, len(calls) - 20, len(calls), foreign_every=11)
    got = bench.profiled_dispatches(path, None, 20, 0, lion_in_muon=lion_first)
    assert got == [(name, 1000 + ci) for ci in range(len(calls) - 20, len(calls))
                   for name in calls[ci]]


def test_profiled_steps_of_an_adaptive_run(tmp_path):
    warmup, steps = 5, 20
    call = SRANK[:2] * 6 + SRANK[2:] + muon_call(True)
    calls = [call] * (warmup + 2 * steps + 1)             # one more step reads the decisions
    path = str(tmp_path / "trace.csv")
    write_trace(path, calls, warmup + steps, warmup + 2 * steps)
    got = bench.profiled_dispatches(path, warmup, steps, 1)
    assert [d for _, d in got] == [1000 + ci for ci in range(warmup + steps, warmup + 2 * steps)
                                   for _ in call]


def test_pure_lion_run_is_one_call_per_kernel(tmp_path):
    calls = [[LION]] * 12
    path = str(tmp_path / "trace.csv")
    write_trace(path, calls, 7, 12)
    got = bench.profiled_dispatches(path, 2, 5, 0)
    assert [d for _, d in got] == [1000 + ci for ci in range(7, 12)]


def test_trace_with_another_number_of_calls_is_rejected(tmp_path):
    calls = period_calls(44, 1, 2, False)                  # one call short of 5 + 2 x 20
    path = str(tmp_path / "trace.csv")
    write_trace(path, calls, 24, 44)
    assert bench.profiled_dispatches(path, 5, 20, 0) is None


def test_launch_gaps_count_back_to_back_pairs_apart(tmp_path):
    warmup, steps = 1, 4
    calls = period_calls(warmup + 2 * steps, 1, 2, False)   # t = 1 (Lion), 2 (Muon), ...
    path = str(tmp_path / "trace.csv")
    write_trace(path, calls, warmup + steps, warmup + 2 * steps)
    g = bench.launch_gaps(path)
    pairs = sum(len(c) for c in calls) - 1
    inside = sum(len(c) - 1 for c in calls)                   # pairs within a call
    inside_evented = sum(len(c) - 1 for c in calls[warmup + steps:])
    assert g["gaps"] == pairs
    assert g["zero"] == inside - inside_evented
    assert g["rest"] == pairs - g["zero"]
    # 8 us after every call but the last, 7.7 us between the kernels of a profiled call
    assert g["mean_rest_us"] == pytest.approx(
        (8.0 * (len(calls) - 1) + 7.7 * inside_evented) / g["rest"])


# --------------------------------------------------------------------------
# Algorithmic units of the bench line's rates and rooflines
# --------------------------------------------------------------------------
# The matrix sets written out from their definitions (per layer: qkv, attention
# projection, MLP in, MLP out), independent of the workload tables.
SETS = {"gpt2-124m": (12, 768), "gpt2-355m": (24, 1024), "gpt2-720m": (36, 1280)}


def _closed_form_ns_flops(layers, d, K=5):
    shapes = [(d, 3 * d), (d, d), (d, 4 * d), (4 * d, d)]
    total = 0
    for m, n in shapes:
        s, l = min(m, n), max(m, n)
        total += s * (s + 1) * l + s * s * (s + 1) + 2 * s * s * l   # Gram, polynomial, apply
    return K * layers * total


@pytest.mark.parametrize("name", sorted(SETS))
def test_ns_flop_counts_agree(name):
    """bench.py's per-launch flops (the roofline's numerator), the planner's
    count and the closed form over the set's shapes are one number; the 124M,
    355M and 720M totals are 1.088, 5.156 and 15.104 TFLOP per Muon step."""
    import workloads
    from paper_2605_19811_amd import lionmuon as lm
    wl = workloads.get(name)
    per_launch = bench.ns_flops_per_launch(wl)
    ours = 5 * sum(per_launch.values())
    closed = _closed_form_ns_flops(*SETS[name])
    specs = [(t.rows, t.cols, t.lion_only) for t in wl.tensors]
    planner = lm.lionmuon_plan_info(specs, t=0, P=1)["ns_flops"]
    assert ours == closed == planner
    assert closed / 1e12 == pytest.approx({"gpt2-124m": 1.088, "gpt2-355m": 5.156,
                                           "gpt2-720m": 15.104}[name], abs=5e-4)


@pytest.mark.parametrize("name,gb", [("gpt2-124m", 1.699), ("gpt2-355m", 6.040),
                                     ("gpt2-720m", 15.454)])
def test_lion_bytes_per_step(name, gb):
    """20 bytes per element on a Lion step (read W, G, M; write W, M), over
    every tensor including the 720M set's Lion-only embedding and vectors."""
    import workloads
    from paper_2605_19811_amd import lionmuon as lm
    wl = workloads.get(name)
    specs = [(t.rows, t.cols, t.lion_only) for t in wl.tensors]
    info = lm.lionmuon_plan_info(specs, t=1, P=2)
    assert info["lion_bytes"] == 20.0 * sum(t.numel for t in wl.tensors)
    assert info["lion_bytes"] / 1e9 == pytest.approx(gb, abs=5e-4)


def test_cpu_baseline_amortisation():
    times = (0.5, 3.5, 16, "sample")
    assert bench.cpu_baseline_for(times, 0)["value"] == 500.0
    assert bench.cpu_baseline_for(times, 1)["value"] == 3500.0
    assert bench.cpu_baseline_for(times, 2)["value"] == 2000.0
    assert bench.cpu_baseline_for(times, 4)["value"] == 1250.0
    b = bench.cpu_baseline_for(times, 2)
    assert b["kind"] == "oracle" and b["cores"] == 16 and b["unit"] == "ms/step"
