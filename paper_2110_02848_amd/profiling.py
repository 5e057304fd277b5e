"""Short text summaries of rocprofv3 output, and the figures bench.py reads
back from them.

Two summaries are kept with the library's measurements:

* a kernel-time table from ``rocprofv3 --kernel-trace --stats`` (calls,
  total and average duration of every kernel of a run, and per kernel
  group);
* a counter table per kernel group from several ``rocprofv3 --pmc`` passes
  over the same run (one CSV per pass, at most what one pass can hold):
  - HBM bytes: ``FETCH_SIZE`` and ``WRITE_SIZE`` (KiB per dispatch), each
    divided by what the same counter reads for a plain device-to-device copy
    of known size (the run copies ``--copy-bytes`` first);
  - the same read traffic from the L2-to-memory read requests counted by
    size (``TCC_EA0_RDREQ{,_32B,_64B,_128B}_sum``), which needs no factor;
  - a calibration of both methods on gathers of known footprint: random
    rows of 32 and of 64 bytes (the size of the search's scattered record
    reads) gathered by index (bench.py --calibrate-gather), so the copy
    factor can be checked for scattered reads;
  - occupancy and activity: mean resident wavefronts per active CU
    (``MeanOccupancyPerActiveCU``), ``OccupancyPercent``, ``VALUBusy``,
    ``MemUnitStalled``, wavefronts launched (``SQ_WAVES``), L2 hit rate
    (``TCC_HIT_sum``, ``TCC_MISS_sum``).

Usage (on a machine with the GPU, from the repository root)::

    python -m paper_2110_02848_amd.profiling stats STATS_CSV OUT.txt --command "..."
    python -m paper_2110_02848_amd.profiling counters OUT.txt --copy-bytes N \\
        --gather-rows R --command "..." PASS1.csv PASS2.csv ...

``read_counters`` parses a counter table back; bench.py reports its figures
only while the device sources still hash to the value recorded in it.
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import os
import re
from collections import defaultdict

_HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(_HERE, "csrc")

# Kernel groups.  The search groups every launch of a search generation:
# both searches side by side (k_gen2) and either search alone.
FAMILIES = {
    "search": ("k_gen<true>", "k_gen<false>", "k_gen2("),
    "count": ("k_count(", "k_count_heavy("),
    "fill": ("k_fill(", "k_fill_light(", "k_fill_heavy("),
    # scores of the composed graph (bench.py --task score)
    "score_gen": ("k_score_gen<true>", "k_score_gen<false>", "k_score_gen2("),
    "score_structure": ("k_owner(", "k_extra(", "k_merge_index(", "k_merge_place(",
                        "k_score_init<"),
    "posterior": ("k_posterior(",),
    "scatter": ("k_absmax(", "k_bucket_count(", "k_bucket_place(", "k_scatter(",
                "k_scatter_final("),
    # three inputs at once (bench.py --task compose3)
    "search3": ("k3_fwd(", "k3_fwd_chunks(", "k3_bwd(", "k3_bwd_chunks("),
    "compact3": ("k3_arc_keys(", "k3_run_starts(", "k3_run_ends(", "k3_seed_bwd(", "k3_collect(", "k3_ids(",
                 "k3_out_light<", "k3_out_heavy<", "k3_fill_states("),
}

# Counters of each pass (what one rocprofv3 pass can collect on gfx950).
PASSES = (
    ("FETCH_SIZE",),
    ("WRITE_SIZE",),
    ("TCC_EA0_RDREQ_sum", "TCC_EA0_RDREQ_32B_sum", "TCC_EA0_RDREQ_64B_sum",
     "TCC_EA0_RDREQ_128B_sum"),
    ("MeanOccupancyPerActiveCU", "VALUBusy", "SQ_WAVES", "MemUnitStalled"),
    ("OccupancyPercent", "TCC_HIT_sum", "TCC_MISS_sum"),
)


def kernel_source_hash():
    """SHA-256 over the device sources (every file of csrc/, by name)."""
    h = hashlib.sha256()
    for name in sorted(os.listdir(CSRC)):
        if name.endswith((".hip", ".h", ".cpp")):
            h.update(name.encode())
            with open(os.path.join(CSRC, name), "rb") as f:
                h.update(f.read())
    return h.hexdigest()


def short_name(full):
    """'void fstc::(anonymous namespace)::k_gen<true>(fstc::Problem, ...)' -> 'k_gen<true>'."""
    m = re.search(r"([A-Za-z_][A-Za-z0-9_]*(<[^>]*>)?)\(", full)
    return m.group(1) if m else full.strip()


def family_of(full):
    for fam, pats in FAMILIES.items():
        for p in pats:
            if p in full:
                return fam
    return None


def stats_summary(stats_csv, command, top=20):
    rows = list(csv.DictReader(open(stats_csv)))
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    total = sum(float(r["TotalDurationNs"]) for r in rows)
    out = ["# rocprofv3 kernel-time summary", f"command: {command}",
           f"kernel_source_sha256: {kernel_source_hash()}", "",
           "| kernel | calls | total ms | avg us | min us | max us | % |",
           "|---|---|---|---|---|---|---|"]
    for r in rows[:top]:
        out.append("| {} | {} | {:.3f} | {:.2f} | {:.2f} | {:.2f} | {:.1f} |".format(
            short_name(r["Name"]), r["Calls"], float(r["TotalDurationNs"]) / 1e6,
            float(r["AverageNs"]) / 1e3, float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3,
            100.0 * float(r["TotalDurationNs"]) / total))
    fam = defaultdict(lambda: [0, 0.0])
    for r in rows:
        f = family_of(r["Name"])
        if f:
            fam[f][0] += int(r["Calls"])
            fam[f][1] += float(r["TotalDurationNs"])
    out += ["", "| kernel group | launches | total ms | avg us per launch |", "|---|---|---|---|"]
    for f in FAMILIES:
        if f in fam:
            n, t = fam[f]
            out.append(f"| {f} | {n} | {t / 1e6:.3f} | {t / 1e3 / n:.2f} |")
    return "\n".join(out) + "\n"


def _dispatches(csv_paths):
    """{(pass index, dispatch id): {"name", "counters": {counter: value}}},
    values summed over the rows of one dispatch (instances)."""
    d = {}
    for pi, path in enumerate(csv_paths):
        for r in csv.DictReader(open(path)):
            key = (pi, r["Dispatch_Id"])
            e = d.setdefault(key, {"name": r["Kernel_Name"], "counters": defaultdict(float)})
            e["counters"][r["Counter_Name"]] += float(r["Counter_Value"])
    return d


def _read_bytes_by_size(c):
    """Read bytes from the request counts by size; requests counted in
    RDREQ but in none of the sized counters are taken as 64 bytes."""
    n32 = c.get("TCC_EA0_RDREQ_32B_sum", 0.0)
    n64 = c.get("TCC_EA0_RDREQ_64B_sum", 0.0)
    n128 = c.get("TCC_EA0_RDREQ_128B_sum", 0.0)
    other = max(0.0, c.get("TCC_EA0_RDREQ_sum", 0.0) - n32 - n64 - n128)
    return 32 * n32 + 64 * (n64 + other) + 128 * n128


def _mean_by(dd, pred):
    """Mean of every counter over the dispatches whose name satisfies pred
    (each counter averaged over the dispatches of the pass that has it)."""
    sums, counts = defaultdict(float), defaultdict(int)
    for (pi, _), e in dd.items():
        if pred(e["name"]):
            for k, v in e["counters"].items():
                sums[k] += v
                counts[k] += 1
    return {k: sums[k] / counts[k] for k in sums}, max(counts.values()) if counts else 0


def counters_summary(csv_paths, copy_bytes, gather_rows, command):
    dd = _dispatches(csv_paths)
    # the copy: the largest copyBuffer dispatch of each pass
    copy = {}
    for (pi, _), e in dd.items():
        if "copyBuffer" in e["name"]:
            for k, v in e["counters"].items():
                copy[k] = max(copy.get(k, 0.0), v)
    ff = copy.get("FETCH_SIZE", 0.0) * 1024.0 / copy_bytes if copy_bytes else 0.0
    fw = copy.get("WRITE_SIZE", 0.0) * 1024.0 / copy_bytes if copy_bytes else 0.0
    copy_rd = _read_bytes_by_size(copy)
    out = ["# rocprofv3 counters per dispatch, by kernel group", f"command: {command}",
           f"kernel_source_sha256: {kernel_source_hash()}",
           f"copy_bytes: {copy_bytes}",
           f"copy_fetch_factor: {ff:.4f}",
           f"copy_write_factor: {fw:.4f}",
           f"copy_read_bytes_by_request_size: {copy_rd:.0f}", ""]
    # gathers of known footprint: rows of 32 bytes, then of 64 bytes (the
    # first and the second gather dispatch of each pass), each row gathered
    # once by an int64 index, the output written once
    if gather_rows:
        out += ["Gather calibration (random rows read once, int64 index read once, rows written "
                "once):", "",
                "| gather | known read bytes | FETCH_SIZE / copy factor | read bytes by request "
                "size | known write bytes | WRITE_SIZE / copy factor |", "|---|---|---|---|---|---|"]
        by_pass = defaultdict(list)
        for (pi, did), e in dd.items():
            nm = e["name"].lower()
            if "gather" in nm or "index_select" in nm or "indexselect" in nm:
                by_pass[pi].append((int(did), e["counters"]))
        for gi, row in enumerate((32, 64)):
            c = defaultdict(float)
            for pi, lst in by_pass.items():
                lst.sort(key=lambda t: t[0])
                if gi < len(lst):
                    for k, v in lst[gi][1].items():
                        c[k] += v
            if not c:
                continue
            known_rd = gather_rows * (row + 8)
            known_wr = gather_rows * row
            fs = c.get("FETCH_SIZE", 0.0) * 1024.0 / ff if ff else 0.0
            ws = c.get("WRITE_SIZE", 0.0) * 1024.0 / fw if fw else 0.0
            rb = _read_bytes_by_size(c)
            out.append(f"| {row}-byte rows x {gather_rows} | {known_rd} | {fs:.0f} "
                       f"({fs / known_rd:.3f} x) | {rb:.0f} ({rb / known_rd:.3f} x) | "
                       f"{known_wr} | {ws:.0f} ({ws / known_wr:.3f} x) |")
        out.append("")
    out += ["HBM bytes = FETCH_SIZE KiB * 1024 / copy_fetch_factor + WRITE_SIZE KiB * 1024 / "
            "copy_write_factor; read bytes by request size = 32 n32 + 64 n64 + 128 n128 "
            "(L2-to-memory read requests); all per dispatch of the kernel group (mean).", "",
            "| kernel group | dispatches | FETCH_SIZE KiB | WRITE_SIZE KiB | HBM bytes | "
            "read bytes by request size | L2 hit % | waves per active CU | occupancy % | "
            "VALUBusy % | MemUnitStalled % | wavefronts |",
            "|---|---|---|---|---|---|---|---|---|---|---|---|"]
    for fam in FAMILIES:
        c, n = _mean_by(dd, lambda nm, f=fam: family_of(nm) == f)
        if not n:
            continue
        fk, wk = c.get("FETCH_SIZE", 0.0), c.get("WRITE_SIZE", 0.0)
        hbm = (fk * 1024.0 / ff if ff else 0.0) + (wk * 1024.0 / fw if fw else 0.0)
        hit, miss = c.get("TCC_HIT_sum", 0.0), c.get("TCC_MISS_sum", 0.0)
        hr = 100.0 * hit / (hit + miss) if hit + miss else 0.0
        out.append(f"| {fam} | {n} | {fk:.1f} | {wk:.1f} | {hbm:.0f} | "
                   f"{_read_bytes_by_size(c):.0f} | {hr:.1f} | "
                   f"{c.get('MeanOccupancyPerActiveCU', 0.0):.2f} | "
                   f"{c.get('OccupancyPercent', 0.0):.1f} | {c.get('VALUBusy', 0.0):.1f} | "
                   f"{c.get('MemUnitStalled', 0.0):.1f} | {c.get('SQ_WAVES', 0.0):.0f} |")
    return "\n".join(out) + "\n"


COLUMNS = ("dispatches", "FETCH_SIZE KiB", "WRITE_SIZE KiB", "HBM bytes",
           "read bytes by request size", "L2 hit %", "waves per active CU", "occupancy %",
           "VALUBusy %", "MemUnitStalled %", "wavefronts")


def read_counters(path):
    """(kernel_source_sha256, {group: {column: value}}) or None."""
    if not os.path.exists(path):
        return None
    sha, table = None, {}
    for line in open(path):
        if line.startswith("kernel_source_sha256:"):
            sha = line.split(":", 1)[1].strip()
        elif line.startswith("| ") and not line.startswith("| kernel"):
            cells = [c.strip() for c in line.strip().strip("|").split("|")]
            if len(cells) == 1 + len(COLUMNS) and cells[0] in FAMILIES:
                table[cells[0]] = {k: float(v) for k, v in zip(COLUMNS, cells[1:])}
    return sha, table


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    a = sub.add_parser("stats")
    a.add_argument("stats_csv")
    a.add_argument("out")
    a.add_argument("--command", required=True)
    b = sub.add_parser("counters")
    b.add_argument("out")
    b.add_argument("csvs", nargs="+")
    b.add_argument("--copy-bytes", type=int, required=True)
    b.add_argument("--gather-rows", type=int, default=0)
    b.add_argument("--command", required=True)
    args = ap.parse_args()
    if args.cmd == "stats":
        text = stats_summary(args.stats_csv, args.command)
    else:
        text = counters_summary(args.csvs, args.copy_bytes, args.gather_rows, args.command)
    with open(args.out, "w") as f:
        f.write(text)
    print(text)


if __name__ == "__main__":
    main()
