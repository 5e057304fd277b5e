"""Benchmark: eager composition C = A o B on one MI355X.

One step = one full composition (search, trim, numbering, arc count and the
fill of the output CSR) of the emissions(T=500, C=64) o lexicon(W=10000,
L=3..10) workload, inputs resident in HBM.  Prints one JSON line.

    python bench.py [--steps K] [--warmup W] [--workload lexicon-T500-W10000] [--seed 0]

``--task score`` measures what a training step runs on the composed graph
instead: one step = forward and backward log-semiring scores of C, the arc
posteriors, and their scatter to the arcs of A and B through provenance (C
is composed once, untimed).

``--task batch --batch N`` composes N utterances (emissions of T=500 frames,
different seeds) with the one lexicon in a single pass per step.
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
    """Algorithmic bytes per composition of each timed kernel group:
    forward search: 4 B probe per move out of an accessible key + 16 B per
    accessible key (frontier write and read); backward search: the same over
    the predecessor moves and the co-accessible keys; count: 8 B per state of
    C (its key in, its count out) + 4 B per kept arc (the probe of its
    target); fill: the output CSR (20 B per arc, 6 B per state + 4 B)."""
    V, E = st["num_states"], st["num_arcs"]
    return {
        "search_forward": 4 * st["generated"] + 16 * st["accessible"],
        "search_backward": 4 * st["generated_backward"] + 16 * st["coaccessible"],
        "count": 8 * V + 4 * E,
        "fill": 20 * E + 4 * (V + 1) + 2 * V,
    }


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_emissions_lexicon_T500_W10000.txt")
SCORE_TRAFFIC_FILE = os.path.join(ROOT, "profiles",
                                  "traffic_score_emissions_lexicon_T500_W10000.txt")


def measured_traffic(workload, kernel, path=TRAFFIC_FILE):
    """HBM bytes per launch of `kernel` from the committed counter table, or
    None if there is none for this workload or the kernels changed since."""
    if workload != "lexicon-T500-W10000":
        return None
    from paper_2110_02848_amd import profiling
    t = profiling.read_traffic(path)
    if t is None:
        return None
    sha, table = t
    if sha != profiling.kernel_source_hash() or kernel not in table:
        return None
    return table[kernel]


def score_kernel_bytes(V, E):
    """Algorithmic bytes per score call of each timed kernel group.
    Generations (both directions): every state's value written once (8 B)
    and every arc's term formed from the value at its other end, its weight
    and that end's id (8 + 4 + 4 B), per direction.  In-arc structure: the
    destination of every arc read twice and an owner word stored (12 B), and
    an in-arc reference per state (4 B)."""
    return {"score_gen": 2 * (8 * V + 16 * E), "score_prep": 12 * E + 4 * V}


def cpu_score_baseline(A, B):
    import oracle
    oracle.build(force=False)
    C = oracle.compose(A, B)
    t0 = time.perf_counter()
    r = oracle.score(C)
    post = oracle.posterior(C, r["alpha"], r["beta"], r["total"])
    oracle.scatter(post, C["arc_a"], len(A["src"]))
    oracle.scatter(post, C["arc_b"], len(B["src"]))
    t = time.perf_counter() - t0
    return {"value": C["num_arcs"] / t, "unit": "arcs/s", "cores": 1, "kind": "oracle",
            "sample": "one full step (forward and backward scores, posteriors, both "
                      "scatters) of the benchmark workload by the C oracle on its own "
                      "composed graph, single thread",
            "seconds": round(t, 3)}


def run_score(args, A, B, comp, dA, dB):
    import torch
    from paper_2110_02848_amd import gpu, synth
    C = comp.compose(dA, dB, provenance=True, keys=False)
    torch.cuda.synchronize()
    V, E = int(C["num_states"]), int(C["num_arcs"])
    EA, EB = len(A["src"]), len(B["src"])

    def step():
        sc = comp.score(C)
        post = comp.posterior(C, sc["alpha"], sc["beta"], sc["total"])
        ga = comp.grad_scatter(post, C["arc_a"], EA)
        gb = comp.grad_scatter(post, C["arc_b"], EB)
        return sc, ga, gb

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    kern = {k: [0.0, 0] for k in gpu.SCORE_KERNELS}
    stream = torch.cuda.current_stream()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        sc, ga, gb = step()
        for k, (ms_k, n_k) in comp.score_kernel_times().items():
            kern[k][0] += ms_k
            kern[k][1] += n_k
    ev1.record(stream)
    torch.cuda.synchronize()
    ms_wall = 1e3 * (time.perf_counter() - t0) / args.steps
    ms_dev = ev0.elapsed_time(ev1) / args.steps
    kernels = {}
    kb = score_kernel_bytes(V, E)
    for k, (ms_k, n_k) in kern.items():
        per_launch = kb[k] * args.steps / n_k
        avg_ms = ms_k / n_k
        kernels[k] = {"launches_per_step": n_k / args.steps, "ms_per_step": ms_k / args.steps,
                      "avg_launch_us": 1e3 * avg_ms, "alg_bytes_per_launch": per_launch,
                      "achieved_GBs": per_launch / (avg_ms * 1e-3) / 1e9}
    dom = max(kernels, key=lambda k: kernels[k]["ms_per_step"])
    d = kernels[dom]
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
                   "seed": args.seed, "task": "score", "V_C": V, "E_C": E, "E_A": EA,
                   "E_B": EB},
        "ms_per_step_device": ms_dev,
        "total": float(sc["total"].item()),
        "kernels": kernels,
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": d["achieved_GBs"],
                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": d["achieved_GBs"] / HBM_PEAK_GBS,
                     "traffic": measured_traffic(args.workload, dom, SCORE_TRAFFIC_FILE),
                     "avg_launch_us": d["avg_launch_us"],
                     "alg_bytes_per_launch": d["alg_bytes_per_launch"]},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_score_baseline(A, B)
    return out


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
    torch.cuda.synchronize()
    kern = {k: [0.0, 0] for k in gpu.KERNELS}
    t0 = time.perf_counter()
    for _ in range(args.steps):
        C, st, ar = step()
        for k, (ms_k, n_k) in comp.kernel_times().items():
            kern[k][0] += ms_k
            kern[k][1] += n_k
    torch.cuda.synchronize()
    ms_wall = 1e3 * (time.perf_counter() - t0) / args.steps
    V, E = int(C["num_states"]), int(C["num_arcs"])
    st_moves = comp.stats()
    kernels = {k: {"launches_per_step": n / args.steps, "ms_per_step": ms / args.steps,
                   "avg_launch_us": 1e3 * ms / n if n else 0.0}
               for k, (ms, n) in kern.items()}
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
        "kernels": kernels,
        "search_stats": {k: st_moves[k] for k in ("key_space", "fwd_levels", "bwd_levels")},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(As[0], B, int(ar[1] - ar[0]))
        out["cpu_baseline"]["sample"] = ("one item of the batch composed by the sequential C "
                                         "oracle (forward-then-trim order), single thread")
    return out


def cpu_baseline(A, B, E_C):
    import oracle
    oracle.build(force=False)
    t0 = time.perf_counter()
    raw = oracle.compose_raw(A, B, oracle.ORDER_FORWARD)
    wall = time.perf_counter() - t0
    t = raw["stats"]["compose_seconds"]
    assert raw["num_arcs"] == E_C, (raw["num_arcs"], E_C)
    return {"value": E_C / t, "unit": "arcs/s", "cores": 1, "kind": "oracle",
            "sample": "one full composition of the benchmark workload by the sequential "
                      "C oracle (forward-then-trim order), single thread",
            "seconds": round(t, 3), "wall_seconds": round(wall, 3)}


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
    ap.add_argument("--task", choices=("compose", "score", "batch"), default="compose",
                    help="compose: the composition itself; score: scores and operand "
                         "gradients of the composed graph; batch: --batch utterances "
                         "composed with one lexicon per step")
    ap.add_argument("--batch", type=int, default=8)
    ap.add_argument("--copy-probe-mb", type=int, default=0,
                    help="first copy a buffer of this many MiB device to device "
                         "(calibrates HBM byte counters under rocprofv3 --pmc)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the composition is a single-GPU kernel "
              "pipeline on one device; run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2110_02848_amd import gpu, synth

    if args.workload not in synth.WORKLOADS:
        ap.error(f"--workload must be one of {', '.join(synth.WORKLOADS)}")
    A, B = synth.workload(args.workload, args.seed)
    dev = "cuda:0"
    dA, dB = gpu.to_device(A, dev), gpu.to_device(B, dev)
    comp = gpu.Composer(0)
    comp.set_option(gpu.FST_OPT_TIMING, 1)
    comp.set_option(gpu.FST_OPT_ORDER, {"forward-first": gpu.FST_ORDER_FORWARD_FIRST,
                                        "coaccessible-first": gpu.FST_ORDER_COACCESSIBLE_FIRST,
                                        "concurrent": gpu.FST_ORDER_CONCURRENT}[args.order])
    stream = torch.cuda.current_stream()

    if args.copy_probe_mb > 0:
        n = args.copy_probe_mb << 20
        src = torch.ones(n, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    if args.task in ("score", "batch"):
        out = run_score(args, A, B, comp, dA, dB) if args.task == "score" else \
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
    torch.cuda.synchronize()
    phases = {k: 0.0 for k in gpu.PHASES}
    kern = {k: [0.0, 0] for k in gpu.KERNELS}
    t0 = time.perf_counter()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for _ in range(args.steps):
        step()
        for k, v in comp.phase_times().items():
            phases[k] += v
        for k, (ms_k, n_k) in comp.kernel_times().items():
            kern[k][0] += ms_k
            kern[k][1] += n_k
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = ev0.elapsed_time(ev1) / args.steps
    ms_wall = 1e3 * wall / args.steps
    st = comp.stats()
    st["generated"] = st_moves["generated"]
    st["generated_backward"] = st_moves["generated_backward"]
    E_C = st["num_arcs"]
    phases = {k: v / args.steps for k, v in phases.items()}

    alg = algorithmic_bytes(A, B, st)
    kb = kernel_bytes(st)
    if args.order == "concurrent" and kern["search_backward"][1] == 0:
        # the searches ran side by side: one launch advances both
        kb["search_forward"] += kb.pop("search_backward")
    kernels = {}
    for k, (ms_k, n_k) in kern.items():
        if n_k == 0 or ms_k <= 0:
            continue
        per_launch = kb[k] * args.steps / n_k
        avg_ms = ms_k / n_k
        kernels[k] = {"launches_per_step": n_k / args.steps, "ms_per_step": ms_k / args.steps,
                      "avg_launch_us": 1e3 * avg_ms, "alg_bytes_per_launch": per_launch,
                      "achieved_GBs": per_launch / (avg_ms * 1e-3) / 1e9}
    dom = max(kernels, key=lambda k: kernels[k]["ms_per_step"])
    d = kernels[dom]
    roofline = {"bound": "hbm", "kernel": dom, "achieved": d["achieved_GBs"],
                "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": d["achieved_GBs"] / HBM_PEAK_GBS,
                "traffic": measured_traffic(args.workload, dom),
                "avg_launch_us": d["avg_launch_us"],
                "alg_bytes_per_launch": d["alg_bytes_per_launch"]}
    out = {
        "metric": "composed arcs/sec (emissions o lexicon)",
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
                   "E_B": len(B["src"]), "V_C": st["num_states"], "E_C": E_C},
        "ms_per_composition_device": ms,
        "phases_ms": {k: round(v, 4) for k, v in phases.items()},
        "kernels": kernels,
        "search_stats": st,
        "algorithmic_bytes": alg,
        "hbm_roofline_fraction_whole": (alg["total"] / (HBM_PEAK_GBS * 1e9)) / (ms_wall * 1e-3),
        "roofline": roofline,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(A, B, E_C)
    comp.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
