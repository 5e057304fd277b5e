"""Bounded brute-force check of the composition semantics (test infrastructure).

Section 3.1, Eq. (1): C transduces x to z with score
    C(x, z) = log-sum over y of exp(A(x, y) + B(y, z)),
i.e. in the log semiring the score of (x, z) is the log-sum-exp, over all
pairs (pi_A, pi_B) of accepting paths with in(pi_A) = x, out(pi_A) = in(pi_B)
and out(pi_B) = z (epsilon erased), of w(pi_A) + w(pi_B).

This module enumerates accepting paths of A and B up to a length bound, pairs
them by their middle string, and compares against the accepting paths of a
composed graph C, which it projects back to (pi_A, pi_B) through the arc
provenance (arc_a, arc_b) that the oracle records.  Plain Python; tiny graphs
only.
"""
from __future__ import annotations

import math
from collections import defaultdict


def _out_arcs(g):
    off = g["arc_offset"]
    return [list(range(int(off[v]), int(off[v + 1]))) for v in range(g["num_states"])]


def accepting_paths(g, max_len):
    """All paths from a start state to an accepting state with at most
    ``max_len`` arcs, as ``(start state, tuple of arc ids)`` (the start state
    tells apart empty paths).  Cycles are unrolled up to the bound."""
    outs = _out_arcs(g)
    dst, acc = g["dst"], g["accept"]
    res = []

    def walk(s, q, path):
        if acc[q]:
            res.append((s, tuple(path)))
        if len(path) == max_len:
            return
        for e in outs[q]:
            path.append(e)
            walk(s, int(dst[e]), path)
            path.pop()

    for s in range(g["num_states"]):
        if g["start"][s]:
            walk(s, s, [])
    return res


def _strings(g, path, side):
    lab = g["ilabel"] if side == "in" else g["olabel"]
    return tuple(int(lab[e]) for e in path[1] if lab[e] != 0)


def _wsum(g, path):
    return math.fsum(float(g["weight"][e]) for e in path[1])


def path_pairs(A, B, max_len):
    """Map (pi_A, pi_B) -> (x, z, weight) for every pair of accepting paths
    with |pi_A|, |pi_B| <= max_len whose middle strings agree."""
    pa = accepting_paths(A, max_len)
    pb = accepting_paths(B, max_len)
    by_mid = defaultdict(list)
    for p in pb:
        by_mid[_strings(B, p, "in")].append(p)
    out = {}
    for p in pa:
        for q in by_mid.get(_strings(A, p, "out"), ()):
            out[(p, q)] = (_strings(A, p, "in"), _strings(B, q, "out"),
                           _wsum(A, p) + _wsum(B, q))
    return out


def composed_paths(C, max_len, max_proj):
    """Accepting paths of C (length <= max_len) whose projections onto A and B
    both have at most ``max_proj`` arcs.  Returns a list of
    (pi_A, pi_B, x, z, weight) with pi_A, pi_B read from arc provenance and
    the start state of C (its key names the start states of A and B)."""
    outs = _out_arcs(C)
    dst, acc = C["dst"], C["accept"]
    aa, bb = C["arc_a"], C["arc_b"]
    il, ol, w = C["ilabel"], C["olabel"], C["weight"]
    res = []

    def walk(s, q, path, na, nb):
        if acc[q]:
            pa = (int(C["key_a"][s]), tuple(int(aa[e]) for e in path if aa[e] >= 0))
            pb = (int(C["key_b"][s]), tuple(int(bb[e]) for e in path if bb[e] >= 0))
            x = tuple(int(il[e]) for e in path if il[e] != 0)
            z = tuple(int(ol[e]) for e in path if ol[e] != 0)
            res.append((pa, pb, x, z, math.fsum(float(w[e]) for e in path)))
        if len(path) == max_len:
            return
        for e in outs[q]:
            ea, eb = int(aa[e]) >= 0, int(bb[e]) >= 0
            if na + ea > max_proj or nb + eb > max_proj:
                continue
            path.append(e)
            walk(s, int(dst[e]), path, na + ea, nb + eb)
            path.pop()

    for s in range(C["num_states"]):
        if C["start"][s]:
            walk(s, s, [], 0, 0)
    return res


def scores(items):
    """Log-sum-exp per (x, z) of a list of (x, z, weight) triples (float64)."""
    acc = defaultdict(list)
    for x, z, w in items:
        acc[(x, z)].append(w)
    out = {}
    for k, ws in acc.items():
        m = max(ws)
        out[k] = m + math.log(math.fsum(math.exp(v - m) for v in ws))
    return out


def check(A, B, C, max_len):
    """Compare C against brute force.  Returns a list of human-readable
    discrepancies (empty when C is exact up to the bound)."""
    problems = []
    pairs = path_pairs(A, B, max_len)
    cpaths = composed_paths(C, 2 * max_len, max_len)
    seen = defaultdict(int)
    for pa, pb, x, z, w in cpaths:
        seen[(pa, pb)] += 1
        ref = pairs.get((pa, pb))
        if ref is None:
            problems.append(f"C path projects to a non-matching pair {pa} {pb}")
            continue
        if (x, z) != (ref[0], ref[1]):
            problems.append(f"strings differ for {pa} {pb}: {(x, z)} vs {ref[:2]}")
        # each matching arc carries one binary32 add; allow that rounding
        tol = 1e-6 * (1.0 + sum(abs(float(A['weight'][e])) for e in pa[1])
                      + sum(abs(float(B['weight'][e])) for e in pb[1]))
        if abs(w - ref[2]) > tol:
            problems.append(f"weight differs for {pa} {pb}: {w} vs {ref[2]}")
    for k, n in seen.items():
        if n > 1:
            problems.append(f"pair {k} realised by {n} paths of C")
    for k in pairs:
        if k not in seen:
            problems.append(f"pair {k} missing from C")
    # Eq. (1) scores per (x, z)
    s_ref = scores(pairs.values())
    s_c = scores([(x, z, w) for _, _, x, z, w in cpaths])
    for k in set(s_ref) | set(s_c):
        if k not in s_ref or k not in s_c:
            problems.append(f"(x, z) = {k} present on one side only")
        elif abs(s_ref[k] - s_c[k]) > 1e-5 * (1 + abs(s_ref[k])):
            problems.append(f"score of {k}: {s_c[k]} vs {s_ref[k]}")
    return problems


def product_trim_keys(A, B):
    """Independent dense product-space search for the trim key set of an
    epsilon-free pair (every label nonzero): keys are plain pairs (qa, qb),
    with a move for every arc pair whose olabel(ea) = ilabel(eb).  This is the
    textbook product construction, written without the filter machinery."""
    VA, VB = A["num_states"], B["num_states"]
    outA, outB = _out_arcs(A), _out_arcs(B)
    succ = defaultdict(set)
    pred = defaultdict(set)
    for qa in range(VA):
        for qb in range(VB):
            for ea in outA[qa]:
                for eb in outB[qb]:
                    if A["olabel"][ea] == B["ilabel"][eb]:
                        v = (int(A["dst"][ea]), int(B["dst"][eb]))
                        succ[(qa, qb)].add(v)
                        pred[v].add((qa, qb))
    fwd = {(a, b) for a in range(VA) if A["start"][a] for b in range(VB) if B["start"][b]}
    stack = list(fwd)
    while stack:
        u = stack.pop()
        for v in succ[u]:
            if v not in fwd:
                fwd.add(v)
                stack.append(v)
    bwd = {(a, b) for a in range(VA) if A["accept"][a] for b in range(VB) if B["accept"][b]}
    stack = list(bwd)
    while stack:
        v = stack.pop()
        for u in pred[v]:
            if u not in bwd:
                bwd.add(u)
                stack.append(u)
    return fwd & bwd



# --------------------------------------------------------------------------
# three inputs: C = A o B o D (the N-way composition of Section 5)
# --------------------------------------------------------------------------

def path_triples(A, B, D, max_len):
    """Map (pi_A, pi_B, pi_D) -> (x, w, weight) for every triple of
    accepting paths with at most ``max_len`` arcs each whose middle strings
    agree: out(pi_A) = in(pi_B) and out(pi_B) = in(pi_D)."""
    pa = accepting_paths(A, max_len)
    pb = accepting_paths(B, max_len)
    pd = accepting_paths(D, max_len)
    b_by_in = defaultdict(list)
    for p in pb:
        b_by_in[_strings(B, p, "in")].append(p)
    d_by_in = defaultdict(list)
    for p in pd:
        d_by_in[_strings(D, p, "in")].append(p)
    out = {}
    for p in pa:
        for q in b_by_in.get(_strings(A, p, "out"), ()):
            for r in d_by_in.get(_strings(B, q, "out"), ()):
                out[(p, q, r)] = (_strings(A, p, "in"), _strings(D, r, "out"),
                                  _wsum(A, p) + _wsum(B, q) + _wsum(D, r))
    return out


def composed3_paths(C, max_len, max_proj):
    """Accepting paths of a three-input composition C (length <= max_len)
    whose projections onto A, B and D each have at most ``max_proj`` arcs:
    a list of (pi_A, pi_B, pi_D, x, w, weight), the projections read from the
    provenance arc_a, arc_b, arc_d and the keys of C's start state."""
    outs = _out_arcs(C)
    dst, acc = C["dst"], C["accept"]
    prov = (C["arc_a"], C["arc_b"], C["arc_d"])
    keys = (C["key_a"], C["key_b"], C["key_d"])
    il, ol, w = C["ilabel"], C["olabel"], C["weight"]
    res = []

    def walk(s, q, path, n):
        if acc[q]:
            proj = tuple((int(keys[i][s]), tuple(int(prov[i][e]) for e in path if prov[i][e] >= 0))
                         for i in range(3))
            x = tuple(int(il[e]) for e in path if il[e] != 0)
            z = tuple(int(ol[e]) for e in path if ol[e] != 0)
            res.append(proj + (x, z, math.fsum(float(w[e]) for e in path)))
        if len(path) == max_len:
            return
        for e in outs[q]:
            m = [n[i] + (1 if prov[i][e] >= 0 else 0) for i in range(3)]
            if max(m) > max_proj:
                continue
            path.append(e)
            walk(s, int(dst[e]), path, m)
            path.pop()

    for s in range(C["num_states"]):
        if C["start"][s]:
            walk(s, s, [], [0, 0, 0])
    return res


def check3(A, B, D, C, max_len):
    """Compare a three-input composition C against brute force: every
    matching triple of accepting paths (each at most max_len arcs) is
    realised by exactly one accepting path of C, with its strings and
    weight, and nothing else is; and the per-(x, w) log-sum scores agree.
    Returns a list of discrepancies."""
    problems = []
    triples = path_triples(A, B, D, max_len)
    cpaths = composed3_paths(C, 3 * max_len, max_len)
    seen = defaultdict(int)
    for pa, pb, pd, x, z, w in cpaths:
        k = (pa, pb, pd)
        seen[k] += 1
        ref = triples.get(k)
        if ref is None:
            problems.append(f"C path projects to a non-matching triple {k}")
            continue
        if (x, z) != (ref[0], ref[1]):
            problems.append(f"strings differ for {k}: {(x, z)} vs {ref[:2]}")
        tol = 1e-6 * (1.0 + sum(abs(float(A["weight"][e])) for e in pa[1])
                      + sum(abs(float(B["weight"][e])) for e in pb[1])
                      + sum(abs(float(D["weight"][e])) for e in pd[1]))
        if abs(w - ref[2]) > tol:
            problems.append(f"weight differs for {k}: {w} vs {ref[2]}")
    for k, n in seen.items():
        if n > 1:
            problems.append(f"triple {k} realised by {n} paths of C")
    for k in triples:
        if k not in seen:
            problems.append(f"triple {k} missing from C")
    s_ref = scores(triples.values())
    s_c = scores([(x, z, w) for _, _, _, x, z, w in cpaths])
    for k in set(s_ref) | set(s_c):
        if k not in s_ref or k not in s_c:
            problems.append(f"(x, w) = {k} present on one side only")
        elif abs(s_ref[k] - s_c[k]) > 1e-5 * (1 + abs(s_ref[k])):
            problems.append(f"score of {k}: {s_c[k]} vs {s_ref[k]}")
    return problems
