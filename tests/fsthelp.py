"""Test helpers: golden-file parsing, structural invariants of a composed graph,
closed forms for the emissions-lexicon workload, and result comparison.

Everything here reads only the input graphs and a composed graph's arrays; it
does not call the oracle or the GPU library.
"""
from __future__ import annotations

import math
import os
from collections import deque

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")

RESULT_KEYS = ("arc_offset", "src", "dst", "ilabel", "olabel", "weight", "arc_a", "arc_b",
               "start", "accept", "key_a", "key_b", "key_f")


def read_golden(name):
    """Parse ``key: values`` lines (``#`` starts a comment); repeated keys
    accumulate into a list."""
    out = {}
    with open(os.path.join(GOLDEN, name)) as fh:
        for line in fh:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            k, v = line.split(":", 1)
            out.setdefault(k.strip(), []).append(v.split())
    return out


def eps_out(A):
    e = np.zeros(A["num_states"], bool)
    if len(A["src"]):
        e[A["src"][A["olabel"] == 0]] = True
    return e


def _bits(x):
    return np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)


def _padded(g):
    """Arc arrays with one dummy trailing arc, so that masked-out lookups with
    index 0 stay in range for graphs without arcs."""
    out = dict(g)
    for k, dt in (("src", np.int32), ("dst", np.int32), ("ilabel", np.int32),
                  ("olabel", np.int32), ("weight", np.float32)):
        out[k] = np.concatenate([np.asarray(g[k], dtype=dt), np.zeros(1, dt)])
    return out


def check_invariants(A, B, C):
    """Return a list of violated invariants of a canonical composed graph."""
    errs = []
    VA, VB = A["num_states"], B["num_states"]
    V, E = int(C["num_states"]), int(C["num_arcs"])
    ka = C["key_a"].astype(np.int64)
    kb = C["key_b"].astype(np.int64)
    kf = C["key_f"].astype(np.int64)
    epsA = eps_out(A)
    if V == 0:
        if E != 0:
            errs.append("arcs without states")
        return errs
    if ka.min() < 0 or ka.max() >= VA or kb.min() < 0 or kb.max() >= VB:
        return ["key out of range"]
    key = (ka * VB + kb) * 2 + kf
    if np.any(np.diff(key) <= 0):
        errs.append("states not in strictly ascending key order")
    if np.any((kf == 1) & ~epsA[ka]):
        errs.append("filter bit set on a state of A without epsilon output")
    if len(np.unique(ka * VB + kb)) > VA * VB:
        errs.append("more (qa, qb) pairs than VA*VB")
    if V > VB * (VA + int(epsA.sum())):
        errs.append("more states than VB*(VA + #epsOutA)")
    st_exp = ((kf == 0) & (A["start"][ka] == 1) & (B["start"][kb] == 1)).astype(np.uint8)
    ac_exp = ((A["accept"][ka] == 1) & (B["accept"][kb] == 1)).astype(np.uint8)
    if not np.array_equal(st_exp, C["start"]):
        errs.append("start flags differ from keys")
    if not np.array_equal(ac_exp, C["accept"]):
        errs.append("accept flags differ from keys")
    off = C["arc_offset"].astype(np.int64)
    src = C["src"].astype(np.int64)
    dst = C["dst"].astype(np.int64)
    if off[0] != 0 or off[-1] != E or np.any(np.diff(off) < 0):
        errs.append("bad arc_offset")
    elif not np.array_equal(np.repeat(np.arange(V), np.diff(off)), src):
        errs.append("src inconsistent with arc_offset")
    if E:
        if dst.min() < 0 or dst.max() >= V:
            return errs + ["dst out of range"]
        a = C["arc_a"].astype(np.int64)
        b = C["arc_b"].astype(np.int64)
        M = (a >= 0) & (b >= 0)
        EA = (a >= 0) & (b < 0)
        EB = (a < 0) & (b >= 0)
        if np.any(~(M | EA | EB)):
            errs.append("arc without provenance")
        w = _bits(C["weight"])
        aa, bb = np.maximum(a, 0), np.maximum(b, 0)
        A = _padded(A)
        B = _padded(B)
        # matching moves
        m = M
        ok = ((A["olabel"][aa] == B["ilabel"][bb]) & (A["olabel"][aa] != 0)
              & (ka[src] == A["src"][aa]) & (kb[src] == B["src"][bb])
              & (ka[dst] == A["dst"][aa]) & (kb[dst] == B["dst"][bb]) & (kf[dst] == 0)
              & (C["ilabel"] == A["ilabel"][aa]) & (C["olabel"] == B["olabel"][bb])
              & (w == _bits(A["weight"][aa] + B["weight"][bb])))
        if np.any(m & ~ok):
            errs.append("matching arc inconsistent with its provenance")
        ok = ((A["olabel"][aa] == 0) & (kf[src] == 0) & (ka[src] == A["src"][aa])
              & (kb[src] == kb[dst]) & (ka[dst] == A["dst"][aa])
              & (kf[dst] == 0)
              & (C["ilabel"] == A["ilabel"][aa]) & (C["olabel"] == 0)
              & (w == _bits(A["weight"][aa])))
        if np.any(EA & ~ok):
            errs.append("A-epsilon arc inconsistent with its provenance")
        ok = ((B["ilabel"][bb] == 0) & (ka[src] == ka[dst]) & (kb[src] == B["src"][bb])
              & (kb[dst] == B["dst"][bb]) & (kf[dst] == epsA[ka[dst]].astype(np.int64))
              & (C["ilabel"] == 0) & (C["olabel"] == B["olabel"][bb])
              & (w == _bits(B["weight"][bb])))
        if np.any(EB & ~ok):
            errs.append("B-epsilon arc inconsistent with its provenance")
        trip = np.stack([src, a, b], axis=1)
        if len(np.unique(trip, axis=0)) != E:
            errs.append("duplicate (src, arc_a, arc_b)")
        lab = np.where(M, A["olabel"][aa].astype(np.int64), 0)
        big = np.int64(1) << 40
        order = np.lexsort((np.where(b >= 0, b, big), np.where(a >= 0, a, big), lab, src))
        if not np.array_equal(order, np.arange(E)):
            errs.append("arcs not in canonical order")
    # trim: every state reachable from a start state and reaching an accept state
    fwd = _reach(V, src, dst, np.flatnonzero(C["start"]))
    bwd = _reach(V, dst, src, np.flatnonzero(C["accept"]))
    if not fwd.all():
        errs.append("inaccessible state")
    if not bwd.all():
        errs.append("non-coaccessible state")
    return errs


def _reach(V, frm, to, seeds):
    seen = np.zeros(V, bool)
    seen[seeds] = True
    if len(frm) == 0:
        return seen
    order = np.argsort(frm, kind="stable")
    frm_s, to_s = frm[order], to[order]
    off = np.searchsorted(frm_s, np.arange(V + 1))
    frontier = np.asarray(seeds, dtype=np.int64)
    while len(frontier):
        lo, hi = off[frontier], off[frontier + 1]
        cnt = hi - lo
        if cnt.sum() == 0:
            break
        idx = np.repeat(lo - np.concatenate([[0], np.cumsum(cnt)[:-1]]), cnt) + np.arange(cnt.sum())
        nxt = np.unique(to_s[idx])
        nxt = nxt[~seen[nxt]]
        seen[nxt] = True
        frontier = nxt
    return seen


def compare_results(got, ref, keys=RESULT_KEYS):
    """Element-wise, bit-exact comparison; returns a list of mismatches."""
    errs = []
    if int(got["num_states"]) != int(ref["num_states"]):
        errs.append(f"num_states {got['num_states']} != {ref['num_states']}")
    if int(got["num_arcs"]) != int(ref["num_arcs"]):
        errs.append(f"num_arcs {got['num_arcs']} != {ref['num_arcs']}")
    if errs:
        return errs
    for k in keys:
        g, r = np.asarray(got[k]), np.asarray(ref[k])
        if k == "weight":
            g, r = _bits(g), _bits(r)
        else:
            g, r = g.astype(np.int64), r.astype(np.int64)
        if g.shape != r.shape:
            errs.append(f"{k}: shape {g.shape} != {r.shape}")
            continue
        bad = np.flatnonzero(g != r)
        if len(bad):
            i = int(bad[0])
            errs.append(f"{k}: {len(bad)} mismatches, first at {i}: {g[i]} != {r[i]}")
    return errs


# --------------------------------------------------------------------------
# emissions o lexicon closed forms
# --------------------------------------------------------------------------

def lexicon_closed_form(T, spellings):
    """|V_C| and |E_C| of trim(emissions o lexicon) from the word lengths.

    Root keys (t, root) are accessible iff t is a sum of word lengths and
    co-accessible iff T - t is; a word instance starting at frame t0 is in C
    iff (t0, root) is accessible and (t0 + L, root) co-accessible, and then it
    contributes L + 1 states (p_1 .. p_{L+1}) and L + 2 arcs."""
    lens = np.array([len(s) for s in spellings], dtype=np.int64)
    Ls = sorted(set(lens.tolist()))
    acc = np.zeros(T + 1, bool)
    acc[0] = True
    for t in range(1, T + 1):
        acc[t] = any(t - L >= 0 and acc[t - L] for L in Ls)
    co = np.zeros(T + 1, bool)
    co[T] = True
    for t in range(T - 1, -1, -1):
        co[t] = any(t + L <= T and co[t + L] for L in Ls)
    n_by_len = {}
    for L in Ls:
        n_by_len[L] = sum(1 for t0 in range(0, T - L + 1) if acc[t0] and co[t0 + L])
    n = np.array([n_by_len[L] for L in lens], dtype=np.int64)
    V = int(np.sum((lens + 1) * n)) + int(np.sum(acc & co))
    E = int(np.sum((lens + 2) * n))
    return V, E


def lexicon_total_score(table, spellings):
    """Log of the total path sum of emissions o lexicon by a frame recursion
    (float64): alpha(t) = LSE over words w of alpha(t - L_w) + sum_k E[t-L_w+k,
    spell_w[k]]; the answer is alpha(T)."""
    T = table.shape[0]
    tab = table.astype(np.float64)
    alpha = np.full(T + 1, -np.inf)
    alpha[0] = 0.0
    by_len = {}
    for w, s in enumerate(spellings):
        by_len.setdefault(len(s), []).append(np.asarray(s, dtype=np.int64) - 1)
    for t in range(1, T + 1):
        terms = []
        for L, words in by_len.items():
            if L > t or alpha[t - L] == -np.inf:
                continue
            S = np.stack(words)  # [n, L]
            sc = tab[np.arange(t - L, t)[None, :], S].sum(axis=1)
            terms.append(alpha[t - L] + sc)
        if terms:
            x = np.concatenate(terms)
            m = x.max()
            alpha[t] = m + math.log(np.exp(x - m).sum())
    return alpha[T]


def dag_total_score(C):
    """Log of the total weight of all accepting paths of an acyclic composed
    graph (float64 forward recursion in topological order)."""
    V = int(C["num_states"])
    src = C["src"].astype(np.int64)
    dst = C["dst"].astype(np.int64)
    w = C["weight"].astype(np.float64)
    indeg = np.bincount(dst, minlength=V)
    order = np.argsort(src, kind="stable")
    off = np.searchsorted(src[order], np.arange(V + 1))
    alpha = np.full(V, -np.inf)
    alpha[C["start"] == 1] = 0.0
    frontier = np.flatnonzero(indeg == 0)
    done = 0
    while len(frontier):
        done += len(frontier)
        lo, hi = off[frontier], off[frontier + 1]
        cnt = hi - lo
        tot = int(cnt.sum())
        if tot == 0:
            break
        idx = order[np.repeat(lo - np.concatenate([[0], np.cumsum(cnt)[:-1]]), cnt) + np.arange(tot)]
        np.logaddexp.at(alpha, dst[idx], alpha[src[idx]] + w[idx])
        heads, dec = np.unique(dst[idx], return_counts=True)
        indeg[heads] -= dec
        frontier = heads[indeg[heads] == 0]
    if done != V:
        raise ValueError("graph is not acyclic")
    acc = alpha[C["accept"] == 1]
    m = acc.max()
    return m + math.log(np.exp(acc - m).sum())


def trim_graph(g):
    """Trim a single transducer (states reachable from a start state and
    reaching an accept state).  Returns (kept state ids ascending, kept arc ids
    ascending)."""
    V = g["num_states"]
    src = g["src"].astype(np.int64)
    dst = g["dst"].astype(np.int64)
    fwd = _reach(V, src, dst, np.flatnonzero(g["start"]))
    bwd = _reach(V, dst, src, np.flatnonzero(g["accept"]))
    keep = fwd & bwd
    arcs = np.flatnonzero(keep[src] & keep[dst]) if len(src) else np.zeros(0, np.int64)
    return np.flatnonzero(keep), arcs


def bfs_levels(n, adj, seeds):
    """Plain BFS levels (used for small trace checks)."""
    lvl = [-1] * n
    q = deque()
    for s in seeds:
        lvl[s] = 0
        q.append(s)
    while q:
        u = q.popleft()
        for v in adj[u]:
            if lvl[v] < 0:
                lvl[v] = lvl[u] + 1
                q.append(v)
    return lvl


# --------------------------------------------------------------------------
# three inputs: C = A o B o D
# --------------------------------------------------------------------------

def eps_out_t(A, B, qa, qb, fab):
    """Per key: whether the state (qa, qb, fab) of A o B has an arc with
    output epsilon (an A-epsilon move when fab = 0, a B arc eps:eps, or a
    matching pair whose B arc has output epsilon)."""
    epsA = eps_out(A)
    VB = B["num_states"]
    bb_eps = np.zeros(VB, bool)
    b_sets = [set() for _ in range(VB)]
    for s, i, o in zip(B["src"], B["ilabel"], B["olabel"]):
        if o == 0:
            if i == 0:
                bb_eps[s] = True
            else:
                b_sets[s].add(int(i))
    a_sets = [set() for _ in range(A["num_states"])]
    for s, o in zip(A["src"], A["olabel"]):
        if o != 0:
            a_sets[s].add(int(o))
    out = np.zeros(len(qa), bool)
    for i, (a, b, f) in enumerate(zip(qa, qb, fab)):
        out[i] = ((f == 0 and epsA[a]) or bb_eps[b] or bool(a_sets[a] & b_sets[b]))
    return out


def check_invariants3(A, B, D, C):
    """Return a list of violated invariants of a canonical three-input
    composition C = A o B o D (keys (qa, qb, f1, qd, f2), provenance
    arc_a, arc_b, arc_d)."""
    errs = []
    V, E = int(C["num_states"]), int(C["num_arcs"])
    if V == 0:
        return [] if E == 0 else ["arcs without states"]
    ka, kb, kd = (C[k].astype(np.int64) for k in ("key_a", "key_b", "key_d"))
    f1, f2 = C["key_fab"].astype(np.int64), C["key_f"].astype(np.int64)
    VA, VB, VD = A["num_states"], B["num_states"], D["num_states"]
    if min(ka.min(), kb.min(), kd.min()) < 0 or ka.max() >= VA or kb.max() >= VB \
            or kd.max() >= VD:
        return ["key out of range"]
    key = (((ka * VB + kb) * 2 + f1) * VD + kd) * 2 + f2
    if np.any(np.diff(key) <= 0):
        errs.append("states not in strictly ascending key order")
    epsA = eps_out(A)
    epsT = eps_out_t(A, B, ka, kb, f1)
    if np.any((f1 == 1) & ~epsA[ka]):
        errs.append("inner filter bit set where A has no epsilon output")
    if np.any((f2 == 1) & ~epsT):
        errs.append("outer filter bit set where A o B has no epsilon output")
    st = ((f1 == 0) & (f2 == 0) & (A["start"][ka] == 1) & (B["start"][kb] == 1)
          & (D["start"][kd] == 1)).astype(np.uint8)
    ac = ((A["accept"][ka] == 1) & (B["accept"][kb] == 1) & (D["accept"][kd] == 1)).astype(np.uint8)
    if not np.array_equal(st, C["start"]):
        errs.append("start flags differ from keys")
    if not np.array_equal(ac, C["accept"]):
        errs.append("accept flags differ from keys")
    off = C["arc_offset"].astype(np.int64)
    src, dst = C["src"].astype(np.int64), C["dst"].astype(np.int64)
    if off[0] != 0 or off[-1] != E or np.any(np.diff(off) < 0):
        errs.append("bad arc_offset")
    elif not np.array_equal(np.repeat(np.arange(V), np.diff(off)), src):
        errs.append("src inconsistent with arc_offset")
    if E:
        if dst.min() < 0 or dst.max() >= V:
            return errs + ["dst out of range"]
        a, b, d = (C[k].astype(np.int64) for k in ("arc_a", "arc_b", "arc_d"))
        Ap, Bp, Dp = _padded(A), _padded(B), _padded(D)
        aa, bb, dd = np.maximum(a, 0), np.maximum(b, 0), np.maximum(d, 0)
        wA = Ap["weight"][aa].astype(np.float32)
        wB = Bp["weight"][bb].astype(np.float32)
        wD = Dp["weight"][dd].astype(np.float32)
        w = _bits(C["weight"])
        ha, hb, hd = a >= 0, b >= 0, d >= 0
        il, ol = C["ilabel"], C["olabel"]
        same = lambda x: x[src] == x[dst]
        # the T-arc (A o B move) of an arc, when A or B moves
        tm = ha & hb
        t_ok = np.ones(E, bool)
        t_ok &= ~tm | ((Ap["olabel"][aa] == Bp["ilabel"][bb]) & (Ap["olabel"][aa] != 0)
                       & (ka[src] == Ap["src"][aa]) & (kb[src] == Bp["src"][bb])
                       & (ka[dst] == Ap["dst"][aa]) & (kb[dst] == Bp["dst"][bb]) & (f1[dst] == 0))
        ta = ha & ~hb
        t_ok &= ~ta | ((Ap["olabel"][aa] == 0) & (f1[src] == 0) & (ka[src] == Ap["src"][aa])
                       & (ka[dst] == Ap["dst"][aa]) & same(kb) & (f1[dst] == 0))
        tb = ~ha & hb
        t_ok &= ~tb | ((Bp["ilabel"][bb] == 0) & same(ka) & (kb[src] == Bp["src"][bb])
                       & (kb[dst] == Bp["dst"][bb]) & (f1[dst] == epsA[ka[dst]]))
        moves_t = ha | hb
        t_in = np.where(ha, Ap["ilabel"][aa], 0)
        t_out = np.where(hb, Bp["olabel"][bb], 0)
        t_w = np.where(tm, wA + wB, np.where(ha, wA, wB)).astype(np.float32)
        # the move of the key: T-arc with D arc (match), T-arc alone (output
        # epsilon), or D arc alone (input epsilon)
        m = moves_t & hd
        ok = ~m | ((t_out != 0) & (Dp["ilabel"][dd] == t_out) & (kd[src] == Dp["src"][dd])
                   & (kd[dst] == Dp["dst"][dd]) & (f2[dst] == 0) & (il == t_in)
                   & (ol == Dp["olabel"][dd]) & (w == _bits(t_w + wD)))
        te = moves_t & ~hd
        ok &= ~te | ((t_out == 0) & (f2[src] == 0) & same(kd) & (f2[dst] == 0) & (il == t_in)
                     & (ol == 0) & (w == _bits(t_w)))
        de = ~moves_t & hd
        ok &= ~de | ((Dp["ilabel"][dd] == 0) & same(ka) & same(kb) & same(f1)
                     & (kd[src] == Dp["src"][dd]) & (kd[dst] == Dp["dst"][dd])
                     & (f2[dst] == epsT[dst]) & (il == 0) & (ol == Dp["olabel"][dd])
                     & (w == _bits(wD)))
        ok &= ~moves_t | t_ok
        ok &= moves_t | hd
        if not np.all(ok):
            errs.append(f"{int(np.sum(~ok))} arcs inconsistent with their provenance")
        trip = np.stack([src, a, b, d], axis=1)
        if len(np.unique(trip, axis=0)) != E:
            errs.append("duplicate (src, arc_a, arc_b, arc_d)")
        big = np.int64(1) << 40
        lab = np.where(tm, Ap["olabel"][aa].astype(np.int64), 0)
        order = np.lexsort((np.where(hd, d, big), np.where(hb, b, big), np.where(ha, a, big),
                            lab, src))
        if not np.array_equal(order, np.arange(E)):
            errs.append("arcs not in canonical order")
    fwd = _reach(V, src, dst, np.flatnonzero(C["start"]))
    bwd = _reach(V, dst, src, np.flatnonzero(C["accept"]))
    if not fwd.all():
        errs.append("inaccessible state")
    if not bwd.all():
        errs.append("non-coaccessible state")
    return errs


def wide_fanout_pair(rng, fan=(300, 255, 254), n_mid=300, n_gap=5):
    """A pair whose start keys are light states (one work unit) with many
    kept arcs: A's start states (its last states, after n_gap isolated ones)
    have fan[i] arcs with output 1 to the middle states 1..fan[i], each of
    which reaches the accepting state 0 by an arc with output 2; B reads
    1 then 2.  The start key (s, 0) joins its one B arc with A's 1-bucket:
    fan[i] arcs of C from one state (255 and more take the output passes'
    wide-count path).  With n_mid + n_gap + 1 = 306 the start states sit at
    rows 306.. and a batch item's first state follows them in the same
    output chunk of 16 trim words (B has three states: one row per word)."""
    f32 = lambda: float(np.float32(rng.standard_normal()))
    arcs = [(k, 0, 8, 2, f32()) for k in range(1, n_mid + 1)]
    first = n_mid + n_gap + 1
    starts = []
    for i, n in enumerate(fan):
        s = first + i
        starts.append(s)
        arcs += [(s, k, 7, 1, f32()) for k in range(1, n + 1)]
    A = synth_from_arcs(first + len(fan), arcs, start=starts, accept=[0])
    B = synth_from_arcs(3, [(0, 1, 1, 5, f32()), (1, 2, 2, 6, f32())], start=[0], accept=[2])
    return A, B


def synth_from_arcs(V, arcs, start, accept):
    from paper_2110_02848_amd import synth
    return synth.from_arcs(V, arcs, start=start, accept=accept)


def renumber(g, perm):
    """The same graph with state s renamed perm[s] (arcs keep their order
    within a state)."""
    perm = np.asarray(perm, dtype=np.int64)
    arcs = [(int(perm[s]), int(perm[d]), int(i), int(o), float(w))
            for s, d, i, o, w in zip(g["src"], g["dst"], g["ilabel"], g["olabel"], g["weight"])]
    return synth_from_arcs(g["num_states"], arcs,
                           start=[int(perm[v]) for v in np.flatnonzero(g["start"])],
                           accept=[int(perm[v]) for v in np.flatnonzero(g["accept"])])
