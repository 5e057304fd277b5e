"""Benchmark: eager composition C = A o B on one MI355X.

One step = one full composition (search, trim, numbering, arc count and the
fill of the output CSR) of the emissions(T=500, C=64) o lexicon(W=10000,
L=3..10) workload, inputs resident in HBM.  Prints one JSON line.

    python bench.py [--steps K] [--warmup W] [--config 5] [--seed 0]
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
    """Bytes the method itself must move (inputs read once, one dedupe probe
    per generated move, each accessible key written and read once in the
    frontier, the output CSR written once)."""
    EA, EB = len(A["src"]), len(B["src"])
    VA, VB = A["num_states"], B["num_states"]
    b_in = 16 * (EA + EB) + 4 * (VA + VB + 2) + 2 * (VA + VB)
    b_search = 4 * st["generated"] + 16 * st["accessible"]
    V, E = st["num_states"], st["num_arcs"]
    b_out = 20 * E + 4 * (V + 1) + 2 * V
    if provenance:
        b_out += 8 * E + 9 * V
    return dict(inputs=b_in, search=b_search, output=b_out, total=b_in + b_search + b_out)


def fill_bytes(st):
    """Algorithmic bytes of the fill kernel: the output CSR it writes."""
    V, E = st["num_states"], st["num_arcs"]
    return 20 * E + 4 * (V + 1) + 2 * V


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
    ap.add_argument("--config", type=int, default=5)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the composition is a single-GPU kernel "
              "pipeline (see the sharding notes in DESIGN.md); run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2110_02848_amd import gpu, synth

    A, B = synth.config(args.config, args.seed)
    dev = "cuda:0"
    dA, dB = gpu.to_device(A, dev), gpu.to_device(B, dev)
    comp = gpu.Composer(0)
    comp.set_option(gpu.FST_OPT_TIMING, 1)
    stream = torch.cuda.current_stream()

    def step():
        nv, ne = comp.run(dA, dB)
        C = comp.alloc_output(nv, ne, provenance=False, keys=False)
        comp.fill(C)
        return C

    # one untimed composition that also counts the moves out of accessible
    # keys (an extra pass), for the algorithmic-bytes model
    comp.set_option(gpu.FST_OPT_COUNT_MOVES, 1)
    step()
    torch.cuda.synchronize()
    st_moves = comp.stats()
    comp.set_option(gpu.FST_OPT_COUNT_MOVES, 0)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    phases = {k: 0.0 for k in gpu.PHASES}
    t0 = time.perf_counter()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for _ in range(args.steps):
        step()
        for k, v in comp.phase_times().items():
            phases[k] += v
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = ev0.elapsed_time(ev1) / args.steps
    ms_wall = 1e3 * wall / args.steps
    st = comp.stats()
    st["generated"] = st_moves["generated"]
    E_C = st["num_arcs"]
    phases = {k: v / args.steps for k, v in phases.items()}

    alg = algorithmic_bytes(A, B, st)
    fill_ms = phases["fill"]
    fb = fill_bytes(st)
    achieved = fb / (fill_ms * 1e-3) / 1e9 if fill_ms > 0 else 0.0
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
        "config": {"workload": synth.CONFIG_NAMES[args.config], "seed": args.seed,
                   "V_A": A["num_states"], "E_A": len(A["src"]), "V_B": B["num_states"],
                   "E_B": len(B["src"]), "V_C": st["num_states"], "E_C": E_C},
        "ms_per_composition_device": ms,
        "phases_ms": {k: round(v, 4) for k, v in phases.items()},
        "search_stats": st,
        "algorithmic_bytes": alg,
        "hbm_roofline_fraction_whole": (alg["total"] / (HBM_PEAK_GBS * 1e9)) / (ms_wall * 1e-3),
        "roofline": {"bound": "hbm", "kernel": "fill", "achieved": achieved,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": None},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(A, B, E_C)
    comp.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
