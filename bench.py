"""Benchmark: eager composition C = A o B on one MI355X.

One step = one full composition (search, trim, numbering, arc count and the
fill of the output CSR) of the emissions(T=500, C=64) o lexicon(W=10000,
L=3..10) workload, inputs resident in HBM.  Prints one JSON line.

The timed region is K plain steps (no library timing, no statistics read
between them); `value` is E_C / wall time per step, with the per-step device
times (HIP events) as mean / p10 / p50 / p90.  K more steps with the
library's per-kernel HIP events give each kernel group's time, its
algorithmic bytes per launch and the `roofline` of the dominant group; the
group's HBM traffic and occupancy come from the committed rocprofv3 counter
table (profiles/counters_<workload>.txt) while the kernel sources still hash
to the value recorded there.  A timed 256 MiB device-to-device copy gives
the measured copy ceiling beside the 8 TB/s peak.  `cpu_baseline` is the
sequential C oracle on the same inputs in both of its orders (median of
several runs each, single thread), with the host's CPU model and core count.

    python bench.py [--steps K] [--warmup W] [--workload lexicon-T500-W10000] [--seed 0]

``--task score`` measures what a training step runs on the composed graph
instead: one step = forward and backward log-semiring scores of C, the arc
posteriors, and their scatter to the arcs of A and B through provenance (C
is composed once, untimed, from validated inputs; the score calls take it
as the library's own output, with FST_OPT_VALIDATE off).

``--task batch --batch N`` composes N utterances (emissions of T=500 frames,
different seeds) with the one lexicon in a single pass per step.

``--task score_cyclic`` measures the scores of a graph with cycles
(fst_score_cyclic: relaxation sweeps until no value rises): one step = both
scores of a seeded random graph of 10^6 states with 3 out-arcs each (arc
probabilities adding to 1/2 per state), inputs resident in HBM.
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

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, GB/s


def algorithmic_bytes(A, B, st, provenance=False):
    """Bytes the method itself must move per composition (inputs read once,
    one dedupe probe per examined move, each kept key written to and read
    from a frontier once, the output CSR written once)."""
    EA, EB = len(A["src"]), len(B["src"])
    VA, VB = A["num_states"], B["num_states"]
    b_in = 16 * (EA + EB) + 4 * (VA + VB + 2) + 2 * (VA + VB)
    b_search = 4 * st["generated"] + 16 * st["accessible"]
    V, E = st["num_states"], st["num_arcs"]
    b_out = 20 * E + 4 * (V + 1) + 2 * V
    if provenance:
        b_out += 8 * E + 9 * V
    return dict(inputs=b_in, search=b_search, output=b_out, total=b_in + b_search + b_out)


def kernel_bytes(st):
    """Algorithmic bytes per composition of each timed kernel group.
    search (both searches, whose launches the default order shares): 4 B
    probe per move out of an accessible key + 16 B per accessible key
    (frontier write and read), and the same over the predecessor moves of
    the co-accessible keys and those keys; count: 1 B per state of C (its
    count out; keys come from the trim bitmap, 1 bit each) + 4 B per kept
    arc (the probe of its target); fill: the output CSR (20 B per arc, 6 B
    per state + 4 B) and each state's count (1 B)."""
    V, E = st["num_states"], st["num_arcs"]
    return {
        "search": (4 * st["generated"] + 16 * st["accessible"]
                   + 4 * st["generated_backward"] + 16 * st["coaccessible"]),
        "count": V + 4 * E,
        "fill": 20 * E + 4 * (V + 1) + 2 * V + V,
    }


def counters_file(workload, task="compose"):
    stem = workload.replace("-", "_")
    if task == "compose3":
        return os.path.join(ROOT, "profiles", f"counters_compose3_{stem}.txt")
    if task == "score":
        return os.path.join(ROOT, "profiles", f"counters_score_{stem}.txt")
    return os.path.join(ROOT, "profiles", f"counters_{stem}.txt")


def measured_counters(workload, kernel, task="compose"):
    """The committed rocprof counter row of a kernel group for this
    workload ({column: value}), or None if there is none or the kernel
    sources changed since it was taken."""
    from paper_2110_02848_amd import profiling
    t = profiling.read_counters(counters_file(workload, task))
    if t is None:
        return None
    sha, table = t
    if sha != profiling.kernel_source_hash() or kernel not in table:
        return None
    return table[kernel]


def roofline_extras(workload, kernel, achieved, copy_gbs, task="compose"):
    """traffic (HBM bytes per launch from the committed FETCH_SIZE /
    WRITE_SIZE passes, copy-scaled), occupancy figures of the same profile,
    and the fraction of the measured copy ceiling."""
    row = measured_counters(workload, kernel, task)
    out = {"traffic": row["HBM bytes"] if row else None,
           "copy_ceiling_GBs": copy_gbs,
           "frac_of_copy_ceiling": achieved / copy_gbs if copy_gbs else None}
    if row:
        out["counters"] = {"read_bytes_by_request_size": row["read bytes by request size"],
                           "l2_hit_pct": row["L2 hit %"],
                           "waves_per_active_cu": row["waves per active CU"],
                           "occupancy_pct": row["occupancy %"],
                           # OccupancyPercent is of 32 wavefronts per CU
                           "mean_waves_per_cu": row["occupancy %"] * 32 / 100.0,
                           "valu_busy_pct": row["VALUBusy %"],
                           "mem_unit_stalled_pct": row["MemUnitStalled %"]}
    else:
        out["counters"] = None
    return out


def host_info():
    """CPU model and the cores this process may run on (the host of the measured GPU)."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count()
    return {"host_cpu": model, "host_nproc": n}


def percentiles(xs):
    a = np.asarray(xs, dtype=np.float64)
    return {"mean": float(a.mean()), "p10": float(np.percentile(a, 10)),
            "p50": float(np.percentile(a, 50)), "p90": float(np.percentile(a, 90))}


def timed_steps(step, steps):
    """Run `steps` steps between two synchronisations (the timed region).
    Returns (wall ms per step, device ms of each step from HIP events on the
    current stream, the last step's result)."""
    import torch
    stream = torch.cuda.current_stream()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    r = None
    for e0, e1 in evs:
        e0.record(stream)
        r = step()
        e1.record(stream)
    torch.cuda.synchronize()
    wall = 1e3 * (time.perf_counter() - t0) / steps
    return wall, [e0.elapsed_time(e1) for e0, e1 in evs], r


def copy_ceiling(mib=256, reps=10):
    """Device-to-device copy rate on this GPU: (read + write bytes) / time of
    a plain copy of `mib` MiB, best of `reps` (HIP events)."""
    import torch
    n = mib << 20
    src = torch.ones(n, dtype=torch.uint8, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    best = None
    for _ in range(reps):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        dst.copy_(src)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        best = ms if best is None or ms < best else best
    del src, dst
    return 2.0 * n / (best * 1e-3) / 1e9


GATHER_ROWS = 1 << 21


def calibrate_gather():
    """Gathers of known footprint for the counter calibration: 2^21 random
    rows of 32 bytes (float) and of 64 bytes (double) out of 256 MiB tables,
    each row once, by an int64 index (rows x (row + 8) bytes read, rows x
    row bytes written)."""
    import torch
    g = torch.Generator(device="cpu").manual_seed(1)
    for dt, cols in ((torch.float32, 8), (torch.float64, 8)):
        rows_total = (256 << 20) // (cols * torch.empty(0, dtype=dt).element_size())
        table = torch.ones(rows_total, cols, dtype=dt, device="cuda:0")
        idx = torch.randperm(rows_total, generator=g)[:GATHER_ROWS].to("cuda:0")
        out = torch.index_select(table, 0, idx)
        torch.cuda.synchronize()
        del table, idx, out


def score_kernel_bytes(V, E):
    """Algorithmic bytes per score call of each timed kernel group.
    Generations (both directions): every state's value written once (8 B)
    and every arc's term formed from the value at its other end, its weight
    and that end's id (8 + 4 + 4 B), per direction.  In-arc structure: the
    destination of every arc read twice and an owner word stored (12 B), and
    an in-arc reference per state (4 B)."""
    return {"score_gen": 2 * (8 * V + 16 * E), "score_prep": 12 * E + 4 * V}


def _reps_for(first_seconds, budget=8.0):
    return int(min(20, max(3, budget // max(first_seconds, 1e-6))))


def cpu_score_baseline(A, B):
    import oracle
    oracle.build(force=False)
    C = oracle.compose(A, B)

    def once():
        t0 = time.perf_counter()
        r = oracle.score(C)
        post = oracle.posterior(C, r["alpha"], r["beta"], r["total"])
        oracle.scatter(post, C["arc_a"], len(A["src"]))
        oracle.scatter(post, C["arc_b"], len(B["src"]))
        return time.perf_counter() - t0

    ts = [once()]
    ts += [once() for _ in range(_reps_for(ts[0]) - 1)]
    t = float(np.median(ts))
    out = {"value": C["num_arcs"] / t, "unit": "arcs/s", "cores": 1, "kind": "oracle",
           "sample": f"median of {len(ts)} full score steps (forward and backward scores, "
                     "posteriors, both scatters) of the benchmark workload by the C oracle on "
                     "its own composed graph, single thread",
           "seconds_median": round(t, 4), "seconds_runs": [round(x, 4) for x in ts]}
    out.update(host_info())
    return out


def instrumented_kernels(comp, step, steps, kernel_names, times_fn, kb):
    """Per-kernel-group device time (library HIP events on the caller's
    stream) over `steps` extra steps with the library's timing on; these
    steps are not the timed region.  kb: algorithmic bytes per step of each
    group.  Returns {group: launches, ms, average launch, achieved GB/s}."""
    from paper_2110_02848_amd import gpu
    comp.set_option(gpu.FST_OPT_TIMING, 1)
    kern = {k: [0.0, 0] for k in kernel_names}
    for _ in range(steps):
        step()
        for k, (ms_k, n_k) in times_fn().items():
            kern[k][0] += ms_k
            kern[k][1] += n_k
    comp.set_option(gpu.FST_OPT_TIMING, 0)
    # the searches are one group (the default order shares their launches)
    if "search_forward" in kern:
        f, b = kern.pop("search_forward"), kern.pop("search_backward")
        kern["search"] = [f[0] + b[0], f[1] + b[1]]
    out = {}
    for k, (ms_k, n_k) in kern.items():
        if n_k == 0 or ms_k <= 0:
            continue
        per_launch = kb[k] * steps / n_k
        avg_ms = ms_k / n_k
        out[k] = {"launches_per_step": n_k / steps, "ms_per_step": ms_k / steps,
                  "avg_launch_us": 1e3 * avg_ms, "alg_bytes_per_launch": per_launch,
                  "achieved_GBs": per_launch / (avg_ms * 1e-3) / 1e9}
    return out


def roofline_of(kernels, workload, copy_gbs, task="compose"):
    dom = max(kernels, key=lambda k: kernels[k]["ms_per_step"])
    d = kernels[dom]
    r = {"bound": "hbm", "kernel": dom, "achieved": d["achieved_GBs"], "peak": HBM_PEAK_GBS,
         "unit": "GB/s", "frac": d["achieved_GBs"] / HBM_PEAK_GBS}
    r.update(roofline_extras(workload, dom, d["achieved_GBs"], copy_gbs, task))
    r["avg_launch_us"] = d["avg_launch_us"]
    r["alg_bytes_per_launch"] = d["alg_bytes_per_launch"]
    return r


def run_score(args, A, B, comp, dA, dB, copy_gbs):
    import torch
    from paper_2110_02848_amd import gpu, synth
    C = comp.compose(dA, dB, provenance=True, keys=False)
    torch.cuda.synchronize()
    V, E = int(C["num_states"]), int(C["num_arcs"])
    EA, EB = len(A["src"]), len(B["src"])
    # C is the library's own output (A and B were validated by the
    # composition): the score and posterior calls skip its structure checks,
    # as a training loop that scores what it just composed would
    comp.set_option(gpu.FST_OPT_VALIDATE, 0)

    def step():
        sc = comp.score(C)
        post = comp.posterior(C, sc["alpha"], sc["beta"], sc["total"])
        ga = comp.grad_scatter(post, C["arc_a"], EA)
        gb = comp.grad_scatter(post, C["arc_b"], EB)
        return sc, ga, gb

    for _ in range(args.warmup):
        step()
    ms_wall, per_step, (sc, ga, gb) = timed_steps(step, args.steps)
    kernels = instrumented_kernels(comp, step, args.steps, gpu.SCORE_KERNELS,
                                   comp.score_kernel_times, score_kernel_bytes(V, E))
    out = {
        "metric": "scored arcs/sec (scores and operand gradients of emissions o lexicon)",
        "value": E / (ms_wall * 1e-3),
        "unit": "arcs/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_wall,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": synth.WORKLOAD_TITLES[args.workload], "name": args.workload,
                   "seed": args.seed, "task": "score", "validate_C": False, "V_C": V,
                   "E_C": E, "E_A": EA, "E_B": EB,
                   "inputs_sha256": {"A": synth.graph_sha256(A), "B": synth.graph_sha256(B)}},
        "ms_per_step_device": percentiles(per_step),
        "total": float(sc["total"].item()),
        "kernels": kernels,
        "roofline": roofline_of(kernels, args.workload, copy_gbs, "score"),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_score_baseline(A, B)
    return out


def compose3_kernel_bytes(st):
    """Algorithmic bytes per three-input composition of each timed group.
    search3 (both searches): per generated move, the target key probed in
    the hash set (8 B) and the arc recorded (8 B); per accessible key, the
    key stored and read back (16 B) and its frontier entry written and read
    (8 B); backward, per generated arc its source placed and read (8 B)
    and the claim probe of that source (4 B), per co-accessible key its
    frontier entry (8 B).  compact3: the grouping of the arcs by target (8 B
    read twice per arc), the trim keys collected and radix-sorted (8 passes
    of 12 B read and written per key), and count and fill: one hash probe
    per candidate arc in each (16 B per kept arc) plus the output CSR (20 B
    per arc, 6 B per state + 4 B)."""
    V, E = st["num_states"], st["num_arcs"]
    G, acc = st["generated"], st["accessible"]
    return {"search3": 16 * G + 24 * acc + 12 * G + 8 * V,
            "compact3": 16 * G + 8 * 24 * V + 16 * E + 20 * E + 6 * V + 4 * (V + 1)}


def cpu_baseline3(A, B, D, E_C):
    import oracle
    oracle.build(force=False)
    raw = oracle.compose3_raw(A, B, D)
    assert raw["num_arcs"] == E_C, (raw["num_arcs"], E_C)
    ts = [raw["stats"]["compose_seconds"]]
    del raw
    for _ in range(_reps_for(ts[0], 8.0) - 1):
        ts.append(oracle.compose3_raw(A, B, D)["stats"]["compose_seconds"])
    t = float(np.median(ts))
    out = {"value": E_C / t, "unit": "arcs/s", "cores": 1, "kind": "oracle",
           "sample": f"the full three-input composition of the benchmark workload by the "
                     f"sequential C oracle (forward search, then trim), single thread: median "
                     f"of {len(ts)} runs",
           "seconds_median": round(t, 4), "seconds_runs": [round(x, 4) for x in ts]}
    out.update(host_info())
    return out


def run_compose3(args, comp, copy_gbs):
    from paper_2110_02848_amd import gpu, synth
    name = args.workload if args.workload in synth.GRAMMAR_SPECS else "grammar-T100-W1000-G20"
    A, B, D, _ = synth.emissions_lexicon_grammar(name, args.seed)
    dA, dB, dD = gpu.to_device(A), gpu.to_device(B), gpu.to_device(D)

    def step():
        nv, ne = comp.run3(dA, dB, dD)
        C = comp.alloc_output3(nv, ne, provenance=False, keys=False)
        comp.fill3(C)
        return C

    step()  # sizes the hash set once (later runs start at the size found)
    for _ in range(args.warmup):
        step()
    ms_wall, per_step, C = timed_steps(step, args.steps)
    st = comp.stats3()
    kernels = instrumented_kernels(comp, step, args.steps, gpu.KERNELS3, comp.kernel_times3,
                                   compose3_kernel_bytes(st))
    out = {
        "metric": "composed arcs/sec (emissions o lexicon o grammar, three inputs at once)",
        "value": st["num_arcs"] / (ms_wall * 1e-3),
        "unit": "arcs/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_wall,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": synth.GRAMMAR_TITLES[name], "name": name, "seed": args.seed,
                   "task": "compose3", "V_A": A["num_states"], "V_B": B["num_states"],
                   "V_D": D["num_states"], "V_C": st["num_states"], "E_C": st["num_arcs"],
                   "inputs_sha256": {"A": synth.graph_sha256(A), "B": synth.graph_sha256(B),
                                     "D": synth.graph_sha256(D)}},
        "ms_per_composition_device": percentiles(per_step),
        "kernels": kernels,
        "search_stats": st,
        "roofline": roofline_of(kernels, name, copy_gbs, "compose3"),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline3(A, B, D, st["num_arcs"])
    return out


CYCLIC_V, CYCLIC_DEGREE = 1_000_000, 3


def run_score_cyclic(args, comp, copy_gbs):
    import torch
    from paper_2110_02848_amd import gpu, synth
    G = synth.random_cyclic(args.seed, CYCLIC_V, degree=CYCLIC_DEGREE, mass=0.5)
    V, E = int(G["num_states"]), len(G["src"])
    dG = gpu.to_device(G)

    def step():
        return comp.score_cyclic(dG)

    for _ in range(args.warmup):
        step()
    ms_wall, per_step, r = timed_steps(step, args.steps)
    # algorithmic bytes of one sweep: per direction, per arc its neighbour,
    # weight and the neighbour's value (16 B); per state its list bounds and
    # flag, its value read and written (25 B).  Once per call, the in-arc
    # CSR (targets read twice, sources and weights read and written: 24 B
    # per arc, plus the cursors; the counts and offsets, 16 B per state) and
    # the two value buffers set to -inf (16 B per state)
    comp.set_option(gpu.FST_OPT_TIMING, 1)
    step()
    torch.cuda.synchronize()
    runs = comp.score_kernel_times()["score_gen"][1]
    comp.set_option(gpu.FST_OPT_TIMING, 0)
    kb = {"score_gen": runs * 2 * (16 * E + 25 * V), "score_prep": 28 * E + 32 * V}
    kernels = instrumented_kernels(comp, step, args.steps, gpu.SCORE_KERNELS,
                                   comp.score_kernel_times, kb)
    name = f"cyclic-V{V}-d{CYCLIC_DEGREE}"
    return {
        "metric": "scored arcs/sec (both scores of a graph with cycles, relaxation sweeps)",
        "value": E / (ms_wall * 1e-3),
        "unit": "arcs/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_wall,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": f"random graph with cycles, V={V}, {CYCLIC_DEGREE} arcs per state, "
                               "arc probabilities 1/2 per state", "name": name,
                   "seed": args.seed, "task": "score_cyclic", "V": V, "E": E,
                   "sweeps_to_settle": r["sweeps"], "sweeps_run": runs,
                   "inputs_sha256": synth.graph_sha256(G)},
        "ms_per_step_device": percentiles(per_step),
        "total": float(r["total"].item()),
        "kernels": kernels,
        "roofline": roofline_of(kernels, name, copy_gbs, "score_cyclic"),
    }


def run_batch(args, comp):
    import torch
    from paper_2110_02848_amd import gpu, synth
    As, B, _ = synth.lexicon_batch(args.workload, args.batch, args.seed)
    dAs = [gpu.to_device(A) for A in As]
    dB = gpu.to_device(B)

    def step():
        nv, ne, st, ar = comp.run_batch(dAs, dB)
        C = comp.alloc_output(nv, ne, provenance=False, keys=False)
        comp.fill(C)
        return C, st, ar

    for _ in range(args.warmup):
        step()
    ms_wall, per_step, (C, st, ar) = timed_steps(step, args.steps)
    V, E = int(C["num_states"]), int(C["num_arcs"])
    st_moves = comp.stats()
    out = {
        "metric": "composed arcs/sec (batch of emissions o one lexicon)",
        "value": E / (ms_wall * 1e-3),
        "unit": "arcs/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_wall,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"{args.batch} x " + synth.WORKLOAD_TITLES[args.workload],
                   "name": args.workload, "seed": args.seed, "task": "batch",
                   "batch": args.batch, "V_C": V, "E_C": E,
                   "item_states": [int(x) for x in np.diff(st)],
                   "item_arcs": [int(x) for x in np.diff(ar)]},
        "ms_per_step_device": percentiles(per_step),
        "search_stats": {k: st_moves[k] for k in ("key_space", "fwd_levels", "bwd_levels")},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(As[0], B, int(ar[1] - ar[0]))
        out["cpu_baseline"]["sample"] = ("one item of the batch composed by the sequential C "
                                         "oracle, single thread, " +
                                         out["cpu_baseline"]["sample"].split(": ", 1)[1])
    return out


def cpu_baseline(A, B, E_C):
    """The oracle (plain sequential C, one thread) on the same inputs, in
    both of its orders: Algorithm 1's (co-accessible set first) and
    forward-then-trim; the median of several runs of each (compose time
    only, the oracle's own steady clock); the faster order is the value."""
    import oracle
    oracle.build(force=False)
    runs = {}
    for name, order in (("forward", oracle.ORDER_FORWARD), ("paper", oracle.ORDER_PAPER)):
        raw = oracle.compose_raw(A, B, order)
        assert raw["num_arcs"] == E_C, (name, raw["num_arcs"], E_C)
        ts = [raw["stats"]["compose_seconds"]]
        del raw
        for _ in range(_reps_for(ts[0], 6.0) - 1):
            ts.append(oracle.compose_raw(A, B, order)["stats"]["compose_seconds"])
        runs[name] = ts
    med = {k: float(np.median(v)) for k, v in runs.items()}
    best = min(med, key=med.get)
    out = {"value": E_C / med[best], "unit": "arcs/s", "cores": 1, "kind": "oracle",
           "sample": f"the full benchmark composition by the sequential C oracle, single thread: "
                     f"median of {len(runs['forward'])} runs in forward-then-trim order and "
                     f"{len(runs['paper'])} in Algorithm 1's order (co-accessible set first); "
                     f"value = the faster order ({best})",
           "seconds_median": {k: round(v, 4) for k, v in med.items()},
           "seconds_runs": {k: [round(x, 4) for x in v] for k, v in runs.items()}}
    out.update(host_info())
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="lexicon-T500-W10000")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--order", choices=("forward-first", "coaccessible-first", "concurrent"),
                    default="concurrent",
                    help="order of the two searches (Algorithm 1 computes the co-accessible "
                         "set first; concurrent, the default, runs both side by side); the "
                         "result is the same")
    ap.add_argument("--task", choices=("compose", "score", "batch", "compose3", "score_cyclic"),
                    default="compose",
                    help="compose: the composition itself; score: scores and operand "
                         "gradients of the composed graph; batch: --batch utterances "
                         "composed with one lexicon per step; compose3: emissions o lexicon "
                         "o grammar composed at once (three inputs); score_cyclic: scores "
                         "of a random graph with cycles")
    ap.add_argument("--batch", type=int, default=8)
    ap.add_argument("--copy-probe-mb", type=int, default=256,
                    help="size of the device-to-device copy timed for the copy ceiling (and "
                         "counted under rocprofv3 --pmc to calibrate the byte counters)")
    ap.add_argument("--calibrate-gather", action="store_true",
                    help="also run gathers of known footprint (for counter calibration "
                         "under rocprofv3 --pmc)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the composition is a kernel pipeline on one "
              "device and is reported for one GPU; run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2110_02848_amd import gpu, synth

    if args.task in ("compose3", "score_cyclic"):
        comp = gpu.Composer(0)
        copy_gbs = copy_ceiling(args.copy_probe_mb) if args.copy_probe_mb > 0 else None
        if args.calibrate_gather:
            calibrate_gather()
        out = (run_compose3 if args.task == "compose3" else run_score_cyclic)(args, comp,
                                                                               copy_gbs)
        comp.close()
        print(json.dumps(out), flush=True)
        return
    if args.workload not in synth.WORKLOADS:
        ap.error(f"--workload must be one of {', '.join(synth.WORKLOADS)}")
    A, B = synth.workload(args.workload, args.seed)
    dev = "cuda:0"
    dA, dB = gpu.to_device(A, dev), gpu.to_device(B, dev)
    comp = gpu.Composer(0)
    comp.set_option(gpu.FST_OPT_ORDER, {"forward-first": gpu.FST_ORDER_FORWARD_FIRST,
                                        "coaccessible-first": gpu.FST_ORDER_COACCESSIBLE_FIRST,
                                        "concurrent": gpu.FST_ORDER_CONCURRENT}[args.order])

    copy_gbs = copy_ceiling(args.copy_probe_mb) if args.copy_probe_mb > 0 else None
    if args.calibrate_gather:
        calibrate_gather()

    if args.task in ("score", "batch"):
        out = run_score(args, A, B, comp, dA, dB, copy_gbs) if args.task == "score" else \
            run_batch(args, comp)
        comp.close()
        print(json.dumps(out), flush=True)
        return

    def step():
        nv, ne = comp.run(dA, dB)
        C = comp.alloc_output(nv, ne, provenance=False, keys=False)
        comp.fill(C)
        return C

    # one untimed composition that also counts the examined moves (extra
    # passes) for the algorithmic-bytes model
    comp.set_option(gpu.FST_OPT_COUNT_MOVES, 1)
    step()
    torch.cuda.synchronize()
    st_moves = comp.stats()
    comp.set_option(gpu.FST_OPT_COUNT_MOVES, 0)
    for _ in range(args.warmup):
        step()
    # the timed region: K plain compositions (no library timing, no reads
    # of statistics between them)
    ms_wall, per_step, _ = timed_steps(step, args.steps)
    st = comp.stats()
    st["generated"] = st_moves["generated"]
    st["generated_backward"] = st_moves["generated_backward"]
    E_C = st["num_arcs"]

    # per-kernel and per-phase device times from K more steps with the
    # library's timing on (not part of the timed region)
    phases = {k: 0.0 for k in gpu.PHASES}

    def timed_phases():
        for k, v in comp.phase_times().items():
            phases[k] += v
        return comp.kernel_times()

    kernels = instrumented_kernels(comp, step, args.steps, gpu.KERNELS, timed_phases,
                                   kernel_bytes(st))
    phases = {k: round(v / args.steps, 4) for k, v in phases.items()}
    alg = algorithmic_bytes(A, B, st)
    out = {
        "metric": "composed arcs/sec (emissions o lexicon)" if args.workload.startswith("lexicon")
        else "composed arcs/sec (random transducer pair)",
        "value": E_C / (ms_wall * 1e-3),
        "unit": "arcs/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_wall,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": synth.WORKLOAD_TITLES[args.workload], "name": args.workload,
                   "seed": args.seed, "order": args.order,
                   "V_A": A["num_states"], "E_A": len(A["src"]), "V_B": B["num_states"],
                   "E_B": len(B["src"]), "V_C": st["num_states"], "E_C": E_C,
                   "inputs_sha256": {"A": synth.graph_sha256(A), "B": synth.graph_sha256(B)}},
        "ms_per_composition_device": percentiles(per_step),
        "phases_ms": phases,
        "kernels": kernels,
        "search_stats": st,
        "algorithmic_bytes": alg,
        "hbm_roofline_fraction_whole": (alg["total"] / (HBM_PEAK_GBS * 1e9)) / (ms_wall * 1e-3),
        "roofline": roofline_of(kernels, args.workload, copy_gbs),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(A, B, E_C)
    comp.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
