"""Short text summaries of rocprofv3 output, and the HBM traffic they record.

Two summaries are kept with the library's measurements:

* a kernel-time table from ``rocprofv3 --kernel-trace --stats`` (calls,
  total and average duration of every kernel of a run);
* an HBM traffic table from two ``rocprofv3 --pmc`` passes over the same
  run, one collecting ``FETCH_SIZE`` and one ``WRITE_SIZE`` (KiB per
  dispatch).  The run also copies a buffer of known size with a plain
  device-to-device copy, and the counters of that copy give the factor that
  turns counter readings into bytes.

Usage (on a machine with the GPU, from the repository root)::

    python -m paper_2110_02848_amd.profiling stats STATS_CSV OUT.txt --command "..."
    python -m paper_2110_02848_amd.profiling traffic FETCH_CSV WRITE_CSV OUT.txt \\
        --copy-bytes N --command "..."

``read_traffic`` parses a traffic table back (bench.py reports it only while
the kernel sources still hash to the value recorded in the table).
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

# kernel families, as timed by the library (enum fst_kernel) in the default
# (concurrent) search order, where one timer covers every search launch:
# both searches side by side (k_gen2), the forward search alone (its first
# generations) and either search alone once the other has ended
FAMILIES = {
    "search_forward": ("k_gen<true>", "k_gen<false>", "k_gen2("),
    "count": ("k_count(", "k_count_heavy("),
    "fill": ("k_fill(", "k_fill_light(", "k_fill_heavy("),
    # scores of the composed graph (bench.py --task score)
    "score_gen": ("k_score_gen<true>", "k_score_gen<false>", "k_score_gen2("),
    "score_structure": ("k_owner(", "k_extra(", "k_merge_index(", "k_merge_place(",
                        "k_score_init<"),
    "posterior": ("k_posterior(",),
    "scatter": ("k_absmax(", "k_bucket_count(", "k_bucket_place(", "k_scatter(",
                "k_scatter_final("),
}


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
    out = ["# rocprofv3 kernel-time summary", f"command: {command}", "",
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


def _per_dispatch(csv_path, counter):
    """{dispatch id: (kernel name, grid size, value)} for one counter."""
    d = {}
    for r in csv.DictReader(open(csv_path)):
        if r["Counter_Name"] != counter:
            continue
        key = r["Dispatch_Id"]
        v = float(r["Counter_Value"])
        if key in d:
            d[key] = (d[key][0], d[key][1], d[key][2] + v)
        else:
            d[key] = (r["Kernel_Name"], int(r["Grid_Size"]), v)
    return d


def _copy_factor(d, copy_bytes):
    copies = [(g, v) for (n, g, v) in d.values() if "copyBuffer" in n]
    if not copies:
        raise SystemExit("no copy kernel in the counter output")
    g, v = max(copies)
    return v * 1024.0 / copy_bytes


def traffic_summary(fetch_csv, write_csv, copy_bytes, command):
    fe = _per_dispatch(fetch_csv, "FETCH_SIZE")
    wr = _per_dispatch(write_csv, "WRITE_SIZE")
    ff, fw = _copy_factor(fe, copy_bytes), _copy_factor(wr, copy_bytes)
    out = ["# rocprofv3 HBM traffic per dispatch (FETCH_SIZE and WRITE_SIZE passes)",
           f"command: {command}",
           f"kernel_source_sha256: {kernel_source_hash()}",
           f"copy_bytes: {copy_bytes}",
           f"copy_fetch_factor: {ff:.4f}",
           f"copy_write_factor: {fw:.4f}",
           "",
           "Bytes = FETCH_SIZE KiB * 1024 / copy_fetch_factor + WRITE_SIZE KiB * 1024 / "
           "copy_write_factor, per dispatch of the kernel group.",
           "",
           "| kernel group | dispatches | FETCH_SIZE KiB/dispatch | WRITE_SIZE KiB/dispatch | "
           "HBM bytes/dispatch |",
           "|---|---|---|---|---|"]
    for fam in FAMILIES:
        fk = [v for (n, g, v) in fe.values() if family_of(n) == fam]
        wk = [v for (n, g, v) in wr.values() if family_of(n) == fam]
        if not fk or not wk:
            continue
        mf, mw = sum(fk) / len(fk), sum(wk) / len(wk)
        b = mf * 1024.0 / ff + mw * 1024.0 / fw
        out.append(f"| {fam} | {len(fk)} | {mf:.1f} | {mw:.1f} | {b:.0f} |")
    return "\n".join(out) + "\n"


def read_traffic(path):
    """(kernel_source_sha256, {group: HBM bytes per dispatch}) or None."""
    if not os.path.exists(path):
        return None
    sha, table = None, {}
    for line in open(path):
        if line.startswith("kernel_source_sha256:"):
            sha = line.split(":", 1)[1].strip()
        elif line.startswith("| ") and not line.startswith("| kernel"):
            cells = [c.strip() for c in line.strip().strip("|").split("|")]
            if len(cells) == 5 and cells[0] in FAMILIES:
                table[cells[0]] = float(cells[4])
    return sha, table


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    a = sub.add_parser("stats")
    a.add_argument("stats_csv")
    a.add_argument("out")
    a.add_argument("--command", required=True)
    b = sub.add_parser("traffic")
    b.add_argument("fetch_csv")
    b.add_argument("write_csv")
    b.add_argument("out")
    b.add_argument("--copy-bytes", type=int, required=True)
    b.add_argument("--command", required=True)
    args = ap.parse_args()
    if args.cmd == "stats":
        text = stats_summary(args.stats_csv, args.command)
    else:
        text = traffic_summary(args.fetch_csv, args.write_csv, args.copy_bytes, args.command)
    with open(args.out, "w") as f:
        f.write(text)
    print(text)


if __name__ == "__main__":
    main()
