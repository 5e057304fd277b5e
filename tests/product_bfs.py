"""Independent check of the trim key set and arc set of C = A o B over the
whole product space (test helper; it uses neither the oracle nor the GPU
library).

Where the oracle runs Algorithm 1 key by key (a queue of keys, each joined
with its arcs), this builds every move of the dense product graph at once,
by a join of all arcs of A with all arcs of B on the matched label, and then
runs two plain breadth-first searches over the keys: forward from the start
keys, backward from the accepting keys.  The trim set is what both reach,
and the arcs of C are the moves between trim keys.  The move rules are the
three of the composition (Section 3.1, Eq. (1), with the epsilon-sequencing
filter read into Algorithm 1):

* matching move: arcs ea, eb with olabel(ea) = ilabel(eb) != 0 lead from
  (src ea, src eb, f), for either filter value f, to (dst ea, dst eb, 0);
* A-epsilon move: an arc ea with olabel(ea) = 0 leads from (src ea, qb, 0)
  to (dst ea, qb, 0), for every state qb of B;
* B-epsilon move: an arc eb with ilabel(eb) = 0 leads from (qa, src eb, f),
  for either f, to (qa, dst eb, epsOutA(qa));

where a key (qa, qb, 1) exists only if qa has an arc with output epsilon
(epsOutA).  Start keys are (sa, sb, 0); accepting keys are the existing keys
whose two states accept.
"""
from __future__ import annotations

import numpy as np


def _eps_out(A):
    e = np.zeros(A["num_states"], bool)
    if len(A["src"]):
        e[A["src"][A["olabel"] == 0]] = True
    return e


def _label_join(la, lb):
    """All index pairs (i, j) with la[i] == lb[j] != 0."""
    la = np.asarray(la, np.int64)
    lb = np.asarray(lb, np.int64)
    ia = np.flatnonzero(la != 0)
    ib = np.flatnonzero(lb != 0)
    ia = ia[np.argsort(la[ia], kind="stable")]
    ib = ib[np.argsort(lb[ib], kind="stable")]
    if len(ia) == 0 or len(ib) == 0:
        return np.zeros(0, np.int64), np.zeros(0, np.int64)
    labs = np.union1d(la[ia], lb[ib])
    a_lo = np.searchsorted(la[ia], labs, "left")
    a_hi = np.searchsorted(la[ia], labs, "right")
    b_lo = np.searchsorted(lb[ib], labs, "left")
    b_hi = np.searchsorted(lb[ib], labs, "right")
    na, nb = a_hi - a_lo, b_hi - b_lo
    npairs = na * nb
    tot = int(npairs.sum())
    if tot == 0:
        return np.zeros(0, np.int64), np.zeros(0, np.int64)
    grp = np.repeat(np.arange(len(labs)), npairs)
    r = np.arange(tot) - np.repeat(np.cumsum(npairs) - npairs, npairs)
    i = ia[a_lo[grp] + r // nb[grp]]
    j = ib[b_lo[grp] + r % nb[grp]]
    return i, j


def product_moves(A, B):
    """Every move of the product graph: (src key, dst key, arc of A or -1,
    arc of B or -1), keys (qa * VB + qb) * 2 + f."""
    VA, VB = int(A["num_states"]), int(B["num_states"])
    eps = _eps_out(A)
    Asrc, Adst = A["src"].astype(np.int64), A["dst"].astype(np.int64)
    Bsrc, Bdst = B["src"].astype(np.int64), B["dst"].astype(np.int64)

    def key(qa, qb, f):
        return (qa * VB + qb) * 2 + f

    parts = []
    # matching moves, from f = 0 and (where epsOutA) from f = 1
    ea, eb = _label_join(A["olabel"], B["ilabel"])
    d = key(Adst[ea], Bdst[eb], 0)
    parts.append((key(Asrc[ea], Bsrc[eb], 0), d, ea, eb))
    one = eps[Asrc[ea]]
    parts.append((key(Asrc[ea][one], Bsrc[eb][one], 1), d[one], ea[one], eb[one]))
    # A-epsilon moves from f = 0, for every state of B
    ae = np.flatnonzero(A["olabel"] == 0)
    qb = np.tile(np.arange(VB, dtype=np.int64), len(ae))
    aer = np.repeat(ae, VB)
    parts.append((key(Asrc[aer], qb, 0), key(Adst[aer], qb, 0), aer,
                  np.full(len(aer), -1, np.int64)))
    # B-epsilon moves from either f, for every state of A
    be = np.flatnonzero(B["ilabel"] == 0)
    qa = np.tile(np.arange(VA, dtype=np.int64), len(be))
    ber = np.repeat(be, VA)
    f_to = eps[qa].astype(np.int64)
    d = key(qa, Bdst[ber], f_to)
    parts.append((key(qa, Bsrc[ber], 0), d, np.full(len(ber), -1, np.int64), ber))
    one = eps[qa]
    parts.append((key(qa[one], Bsrc[ber][one], 1), d[one], np.full(int(one.sum()), -1, np.int64),
                  ber[one]))
    cat = [np.concatenate([p[k] for p in parts]) for k in range(4)]
    return cat[0], cat[1], cat[2], cat[3]


def _reach(n, frm, to, seeds):
    seen = np.zeros(n, bool)
    seeds = np.asarray(seeds, np.int64)
    seen[seeds] = True
    if len(frm) == 0:
        return seen
    order = np.argsort(frm, kind="stable")
    frm_s, to_s = frm[order], to[order]
    frontier = np.unique(seeds)
    while len(frontier):
        lo = np.searchsorted(frm_s, frontier, "left")
        hi = np.searchsorted(frm_s, frontier, "right")
        cnt = hi - lo
        tot = int(cnt.sum())
        if tot == 0:
            break
        idx = np.repeat(lo - np.concatenate([[0], np.cumsum(cnt)[:-1]]), cnt) + np.arange(tot)
        nxt = np.unique(to_s[idx])
        nxt = nxt[~seen[nxt]]
        seen[nxt] = True
        frontier = nxt
    return seen


def trim_product(A, B):
    """dict(keys: sorted trim keys, src, dst: keys of the arcs between trim
    keys, arc_a, arc_b: their provenance, accessible: number of keys the
    forward search reaches), arcs sorted by (src, arc_a, arc_b) with -1
    sorting last."""
    VA, VB = int(A["num_states"]), int(B["num_states"])
    n = 2 * VA * VB
    empty = np.zeros(0, np.int64)
    if n == 0:
        return dict(keys=empty, src=empty, dst=empty, arc_a=empty, arc_b=empty, accessible=0)
    eps = _eps_out(A)
    s, d, ea, eb = product_moves(A, B)
    sa = np.flatnonzero(A["start"])
    sb = np.flatnonzero(B["start"])
    starts = ((sa[:, None] * VB + sb[None, :]) * 2).ravel()
    aa = np.flatnonzero(A["accept"])
    ab = np.flatnonzero(B["accept"])
    acc0 = ((aa[:, None] * VB + ab[None, :]) * 2).ravel()
    aa1 = aa[eps[aa]]
    acc1 = ((aa1[:, None] * VB + ab[None, :]) * 2 + 1).ravel()
    fwd = _reach(n, s, d, starts)
    bwd = _reach(n, d, s, np.concatenate([acc0, acc1]))
    trim = fwd & bwd
    keep = trim[s] & trim[d]
    s, d, ea, eb = s[keep], d[keep], ea[keep], eb[keep]
    big = np.int64(1) << 40
    order = np.lexsort((np.where(eb >= 0, eb, big), np.where(ea >= 0, ea, big), s))
    return dict(keys=np.flatnonzero(trim), src=s[order], dst=d[order], arc_a=ea[order],
                arc_b=eb[order], accessible=int(fwd.sum()))
