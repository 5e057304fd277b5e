"""Seeded synthetic transducers in the structure-of-arrays / CSR layout.

This module only *builds inputs*.  It holds none of the composition's
arithmetic, so both the GPU path and the CPU oracle may consume its arrays.

Graph format (a plain dict of numpy arrays), following the structure-of-arrays
description of Section 3.2 of the paper (start/accept arrays of V booleans,
five E-arrays of arc data, an out-arc offset array of V+1 entries):

    num_states : int                V >= 0
    arc_offset : int32[V+1]         arcs of state v are [arc_offset[v], arc_offset[v+1])
    src, dst   : int32[E]           source / destination state of each arc
    ilabel     : int32[E]           input label, 0 is epsilon, real labels >= 1
    olabel     : int32[E]           output label, 0 is epsilon
    weight     : float32[E]         log-semiring weight
    start      : uint8[V]           1 = start state
    accept     : uint8[V]           1 = accepting state

Arcs are stored grouped by source state ("consecutive by node"); inside a state
they keep the order in which they were generated.

Workloads (Section 4 of the paper; the paper's LibriSpeech lexicon is not
available, so uniform random spellings stand in for it):

* random FST pairs (Section 4.1 recipe, with epsilon labels and several
  accepting states): ``random_pair(name, seed)`` for the names of
  ``RANDOM_SPECS`` ("random-64", "random-1000", "random-5000");
* emissions (A) and lexicon (B) graphs (Section 4.2 recipe):
  ``emissions_lexicon(name, seed)`` for the names of ``LEX_SPECS``
  ("lexicon-T100-W1000", "lexicon-T500-W10000").

``workload(name, seed)`` returns the pair ``(A, B)`` of any of them.
"""
from __future__ import annotations

import hashlib
from dataclasses import dataclass

import numpy as np

EPS = 0

GRAPH_KEYS = ("arc_offset", "src", "dst", "ilabel", "olabel", "weight", "start", "accept")


# --------------------------------------------------------------------------
# construction helpers
# --------------------------------------------------------------------------

def from_arcs(num_states, arcs, start=(0,), accept=()):
    """Build a graph dict from a list of ``(src, dst, ilabel, olabel, weight)``.

    Arcs are grouped by source state with a stable sort, so arcs that share a
    source keep their relative order.  ``start`` and ``accept`` are iterables of
    state ids.
    """
    V = int(num_states)
    arcs = list(arcs)
    E = len(arcs)
    src = np.array([a[0] for a in arcs], dtype=np.int32).reshape(E)
    order = np.argsort(src, kind="stable")
    src = src[order]
    dst = np.array([a[1] for a in arcs], dtype=np.int32).reshape(E)[order]
    il = np.array([a[2] for a in arcs], dtype=np.int32).reshape(E)[order]
    ol = np.array([a[3] for a in arcs], dtype=np.int32).reshape(E)[order]
    w = np.array([a[4] for a in arcs], dtype=np.float32).reshape(E)[order]
    st = np.zeros(V, dtype=np.uint8)
    ac = np.zeros(V, dtype=np.uint8)
    for s in start:
        st[s] = 1
    for s in accept:
        ac[s] = 1
    return _finish(V, src, dst, il, ol, w, st, ac)


def _finish(V, src, dst, il, ol, w, st, ac):
    counts = np.bincount(src, minlength=V).astype(np.int64) if len(src) else np.zeros(V, np.int64)
    off = np.zeros(V + 1, dtype=np.int32)
    if V:
        off[1:] = np.cumsum(counts)
    g = dict(
        num_states=int(V),
        arc_offset=off,
        src=np.ascontiguousarray(src, dtype=np.int32),
        dst=np.ascontiguousarray(dst, dtype=np.int32),
        ilabel=np.ascontiguousarray(il, dtype=np.int32),
        olabel=np.ascontiguousarray(ol, dtype=np.int32),
        weight=np.ascontiguousarray(w, dtype=np.float32),
        start=np.ascontiguousarray(st, dtype=np.uint8),
        accept=np.ascontiguousarray(ac, dtype=np.uint8),
    )
    check_graph(g)
    return g


def check_graph(g):
    """Raise ValueError unless ``g`` is a well-formed graph dict."""
    V = g["num_states"]
    off = g["arc_offset"]
    E = len(g["src"])
    if V < 0 or off.shape != (V + 1,):
        raise ValueError("arc_offset must have V+1 entries")
    if off[0] != 0 or off[-1] != E or np.any(np.diff(off.astype(np.int64)) < 0):
        raise ValueError("arc_offset must be monotone from 0 to E")
    for k in ("dst", "ilabel", "olabel", "weight"):
        if len(g[k]) != E:
            raise ValueError(f"{k} must have E entries")
    if E:
        expect_src = np.repeat(np.arange(V, dtype=np.int32), np.diff(off))
        if not np.array_equal(expect_src, g["src"]):
            raise ValueError("src inconsistent with arc_offset")
        if g["dst"].min() < 0 or g["dst"].max() >= V:
            raise ValueError("dst out of range")
        if g["ilabel"].min() < 0 or g["olabel"].min() < 0:
            raise ValueError("negative label")
    for k in ("start", "accept"):
        if g[k].shape != (V,) or (V and g[k].max() > 1):
            raise ValueError(f"{k} must hold V entries of 0/1")


def graph_sha256(g):
    h = hashlib.sha256()
    h.update(np.int64(g["num_states"]).tobytes())
    for k in GRAPH_KEYS:
        h.update(np.ascontiguousarray(g[k]).tobytes())
    return h.hexdigest()


def num_arcs(g):
    return int(len(g["src"]))


# --------------------------------------------------------------------------
# random transducers (Section 4.1)
# --------------------------------------------------------------------------

def random_fst(rng, V, degree, n_sym, p_eps, p_accept, start=(0,)):
    """Every state gets exactly ``degree`` out-arcs.

    Destinations are uniform over all states (self-loops allowed).  Input and
    output labels are drawn independently: epsilon with probability ``p_eps``,
    otherwise uniform over ``1..n_sym``.  Weights are N(0,1) drawn in float64
    and rounded to float32.  Each state accepts independently with
    probability ``p_accept``.
    """
    E = V * degree
    src = np.repeat(np.arange(V, dtype=np.int32), degree)
    dst = rng.integers(0, V, size=E, dtype=np.int64).astype(np.int32)
    il_eps = rng.random(E) < p_eps
    il_sym = rng.integers(1, n_sym + 1, size=E, dtype=np.int64)
    ol_eps = rng.random(E) < p_eps
    ol_sym = rng.integers(1, n_sym + 1, size=E, dtype=np.int64)
    il = np.where(il_eps, EPS, il_sym).astype(np.int32)
    ol = np.where(ol_eps, EPS, ol_sym).astype(np.int32)
    w = rng.standard_normal(E).astype(np.float32)
    ac = (rng.random(V) < p_accept).astype(np.uint8)
    st = np.zeros(V, dtype=np.uint8)
    for s in start:
        if V:
            st[s] = 1
    return _finish(V, src, dst, il, ol, w, st, ac)


@dataclass(frozen=True)
class RandomSpec:
    V: int
    degree: int
    n_sym: int
    p_eps: float
    p_accept: float


RANDOM_SPECS = {
    "random-64": RandomSpec(64, 4, 16, 0.10, 0.10),
    "random-1000": RandomSpec(1000, 8, 32, 0.05, 0.10),
    "random-5000": RandomSpec(5000, 4, 64, 0.05, 0.05),
}

# Seed stream of each workload: inputs are drawn from
# SeedSequence([stream, seed]).spawn(2), one generator for A and one for B.
_STREAM = {"random-64": 1, "random-1000": 2, "random-5000": 3,
           "lexicon-T100-W1000": 4, "lexicon-T500-W10000": 5}


def _rngs(name, seed):
    ss = np.random.SeedSequence([_STREAM[name], int(seed)])
    return [np.random.default_rng(s) for s in ss.spawn(2)]


def random_pair(name, seed=0):
    spec = RANDOM_SPECS[name]
    ra, rb = _rngs(name, seed)
    A = random_fst(ra, spec.V, spec.degree, spec.n_sym, spec.p_eps, spec.p_accept)
    B = random_fst(rb, spec.V, spec.degree, spec.n_sym, spec.p_eps, spec.p_accept)
    return A, B


# --------------------------------------------------------------------------
# emissions and lexicon (Section 4.2)
# --------------------------------------------------------------------------

def emissions(rng, T, C):
    """Linear acceptor with T frames and C token arcs per frame.

    State t has arcs t -> t+1 labelled c:c for c = 1..C, in label order, with
    weight float32(log_softmax(z_t)[c]) for logits z_t ~ N(0,1)^C drawn in
    float64.  State 0 is the start state and state T the only accepting state.
    Returns the graph and the float32 [T, C] emission table.
    """
    z = rng.standard_normal((T, C))
    m = z.max(axis=1, keepdims=True)
    logp = z - m - np.log(np.exp(z - m).sum(axis=1, keepdims=True))
    table = logp.astype(np.float32)
    V = T + 1
    src = np.repeat(np.arange(T, dtype=np.int32), C)
    dst = src + 1
    lab = np.tile(np.arange(1, C + 1, dtype=np.int32), T)
    st = np.zeros(V, np.uint8)
    st[0] = 1
    ac = np.zeros(V, np.uint8)
    ac[T] = 1
    g = _finish(V, src, dst, lab, lab.copy(), table.reshape(-1).copy(), st, ac)
    return g, table


def lexicon(rng, W, C, len_lo, len_hi):
    """Lexicon transducer over C tokens with W words (word ids 1..W).

    Word lengths are uniform over ``len_lo..len_hi`` and spellings uniform over
    ``1..C``.  Each word w is a path out of the root (state 0): an arc with
    epsilon input and output w into p_1, then token arcs tok_j:epsilon from p_j
    to p_{j+1}, then an epsilon:epsilon arc from p_{L+1} back to the root.  All
    weights are 0.  The root is the start state and the only accepting state.
    Returns the graph and the list of spellings.
    """
    lens = rng.integers(len_lo, len_hi + 1, size=W, dtype=np.int64)
    spell = [rng.integers(1, C + 1, size=int(L), dtype=np.int64).astype(np.int32) for L in lens]
    V = 1 + int(np.sum(lens + 1))
    E = int(np.sum(lens + 2))
    src = np.empty(E, np.int32)
    dst = np.empty(E, np.int32)
    il = np.empty(E, np.int32)
    ol = np.empty(E, np.int32)
    # root arcs first (CSR order): one entry arc per word
    first_state = 1 + np.concatenate([[0], np.cumsum(lens + 1)[:-1]]).astype(np.int64)
    src[:W] = 0
    dst[:W] = first_state
    il[:W] = EPS
    ol[:W] = np.arange(1, W + 1)
    pos = W
    for w in range(W):
        L = int(lens[w])
        p1 = int(first_state[w])
        s = np.arange(p1, p1 + L, dtype=np.int32)
        src[pos:pos + L] = s
        dst[pos:pos + L] = s + 1
        il[pos:pos + L] = spell[w]
        ol[pos:pos + L] = EPS
        pos += L
        src[pos] = p1 + L
        dst[pos] = 0
        il[pos] = EPS
        ol[pos] = EPS
        pos += 1
    order = np.argsort(src, kind="stable")
    w0 = np.zeros(E, np.float32)
    st = np.zeros(V, np.uint8)
    st[0] = 1
    ac = np.zeros(V, np.uint8)
    ac[0] = 1
    g = _finish(V, src[order], dst[order], il[order], ol[order], w0, st, ac)
    return g, spell


@dataclass(frozen=True)
class LexSpec:
    T: int
    C: int
    W: int
    len_lo: int
    len_hi: int


LEX_SPECS = {
    "lexicon-T100-W1000": LexSpec(100, 28, 1000, 3, 8),
    "lexicon-T500-W10000": LexSpec(500, 64, 10000, 3, 10),
}


def emissions_lexicon(name, seed=0, spec=None):
    """A = emissions, B = lexicon (so A o B maps token strings to word
    strings).  ``spec`` overrides the sizes (the seed stream stays that of
    ``name``)."""
    spec = spec or LEX_SPECS[name]
    ra, rb = _rngs(name, seed)
    A, table = emissions(ra, spec.T, spec.C)
    B, spell = lexicon(rb, spec.W, spec.C, spec.len_lo, spec.len_hi)
    return A, B, dict(table=table, spellings=spell, spec=spec)


def lexicon_batch(name, n, seed=0, spec=None, frames=None):
    """A batch of emission graphs with one lexicon: item i is the emissions
    of ``emissions_lexicon(name, seed + i)`` (T frames, or ``frames[i]``),
    and B is the lexicon of ``emissions_lexicon(name, seed)``.  Returns
    (list of A_i, B, meta with the per-item tables and the spellings)."""
    spec = spec or LEX_SPECS[name]
    As, tables = [], []
    for i in range(int(n)):
        ra, _ = _rngs(name, seed + i)
        T = spec.T if frames is None else int(frames[i])
        A, table = emissions(ra, T, spec.C)
        As.append(A)
        tables.append(table)
    _, rb = _rngs(name, seed)
    B, spell = lexicon(rb, spec.W, spec.C, spec.len_lo, spec.len_hi)
    return As, B, dict(tables=tables, spellings=spell, spec=spec)


def word_grammar(rng, G, W, deg, p_backoff, p_accept):
    """Word-level grammar acceptor over word ids 1..W (the third input of an
    emissions o lexicon o grammar composition).  G states, state 0 start and
    accepting, others accepting with probability p_accept.  Each state has
    ``deg`` arcs w:w for distinct words drawn uniformly, to uniform
    destinations; each state other than 0 has, with probability p_backoff,
    an epsilon:epsilon backoff arc to state 0 (listed last).  A state's arc
    weights are a float32 log-softmax of N(0, 1) logits drawn in float64
    (over its word arcs and its backoff arc)."""
    arcs = []
    for s in range(G):
        words = rng.choice(W, size=min(deg, W), replace=False) + 1
        dsts = rng.integers(0, G, size=len(words))
        back = s != 0 and rng.random() < p_backoff
        z = rng.standard_normal(len(words) + (1 if back else 0))
        m = z.max()
        logp = (z - m - np.log(np.exp(z - m).sum())).astype(np.float32)
        for i, (w, d) in enumerate(zip(words, dsts)):
            arcs.append((s, int(d), int(w), int(w), float(logp[i])))
        if back:
            arcs.append((s, 0, EPS, EPS, float(logp[-1])))
    acc = [0] + [s for s in range(1, G) if rng.random() < p_accept]
    return from_arcs(G, arcs, start=[0], accept=acc)


@dataclass(frozen=True)
class GrammarSpec:
    T: int
    C: int
    W: int
    len_lo: int
    len_hi: int
    G: int
    deg: int
    p_backoff: float
    p_accept: float


GRAMMAR_SPECS = {
    "grammar-T40-W300-G6": GrammarSpec(40, 12, 300, 2, 6, 6, 60, 0.5, 0.5),
    "grammar-T100-W1000-G20": GrammarSpec(100, 28, 1000, 3, 8, 20, 200, 0.5, 0.3),
}
_STREAM.update({"grammar-T40-W300-G6": 6, "grammar-T100-W1000-G20": 7})


def emissions_lexicon_grammar(name, seed=0, spec=None):
    """A = emissions, B = lexicon, D = word grammar (so A o B o D maps token
    strings to the word strings the grammar accepts).  Inputs are drawn from
    SeedSequence([stream, seed]).spawn(3), one generator per graph."""
    spec = spec or GRAMMAR_SPECS[name]
    ra, rb, rd = [np.random.default_rng(s)
                  for s in np.random.SeedSequence([_STREAM[name], int(seed)]).spawn(3)]
    A, table = emissions(ra, spec.T, spec.C)
    B, spell = lexicon(rb, spec.W, spec.C, spec.len_lo, spec.len_hi)
    D = word_grammar(rd, spec.G, spec.W, spec.deg, spec.p_backoff, spec.p_accept)
    return A, B, D, dict(table=table, spellings=spell, spec=spec)


def workload(name, seed=0):
    """Inputs ``(A, B)`` of a named workload for a given seed."""
    if name in RANDOM_SPECS:
        return random_pair(name, seed)
    A, B, _ = emissions_lexicon(name, seed)
    return A, B


WORKLOADS = tuple(RANDOM_SPECS) + tuple(LEX_SPECS)

GRAMMAR_TITLES = {
    "grammar-T40-W300-G6": "emissions(T=40,C=12) o lexicon(W=300,L=2..6) o grammar(G=6,deg=60)",
    "grammar-T100-W1000-G20":
        "emissions(T=100,C=28) o lexicon(W=1000,L=3..8) o grammar(G=20,deg=200)",
}

WORKLOAD_TITLES = {
    "random-64": "random pair V=64 d=4 K=16 p_eps=0.1 p_acc=0.1",
    "random-1000": "random pair V=1000 d=8 K=32 p_eps=0.05 p_acc=0.1",
    "random-5000": "random pair V=5000 d=4 K=64 p_eps=0.05 p_acc=0.05",
    "lexicon-T100-W1000": "emissions(T=100,C=28) o lexicon(W=1000,L=3..8)",
    "lexicon-T500-W10000": "emissions(T=500,C=64) o lexicon(W=10000,L=3..10)",
}


# --------------------------------------------------------------------------
# small graphs for tests
# --------------------------------------------------------------------------

def tiny_random(rng, V, max_degree, n_sym, p_eps, p_accept=0.4, n_start=1):
    """Tiny random transducer with variable out-degree (0..max_degree)."""
    arcs = []
    for s in range(V):
        d = int(rng.integers(0, max_degree + 1))
        for _ in range(d):
            t = int(rng.integers(0, V))
            il = 0 if rng.random() < p_eps else int(rng.integers(1, n_sym + 1))
            ol = 0 if rng.random() < p_eps else int(rng.integers(1, n_sym + 1))
            w = float(np.float32(rng.standard_normal()))
            arcs.append((s, t, il, ol, w))
    starts = sorted(set(int(x) for x in rng.integers(0, V, size=n_start)))
    acc = [s for s in range(V) if rng.random() < p_accept]
    return from_arcs(V, arcs, start=starts, accept=acc)


def random_cyclic(seed, V, degree=3, mass=0.5, n_start=2, p_accept=0.2, hubs=0,
                  hub_degree=0):
    """Seeded random graph with cycles whose path sums converge (inputs of
    the cyclic-score tests and benchmark).

    Every state gets ``degree`` (>= 1) out-arcs to uniform destinations
    (self-loops and parallel arcs allowed); ``hubs`` states (drawn at random)
    also get ``hub_degree`` in-arcs from random states.  A state's out-arc
    weights are log(mass * p) for p a softmax of N(0, 1) draws over its
    arcs, rounded to binary32, so the probabilities of a state's arcs add to
    about ``mass`` (< 1: the spectral radius of the arc matrix stays below
    1).  Labels are 1.  ``n_start`` distinct start states; accepting states
    at rate p_accept, at least one."""
    assert degree >= 1
    rng = np.random.default_rng(np.random.SeedSequence([11, int(seed)]))
    src = np.repeat(np.arange(V, dtype=np.int64), degree)
    dst = rng.integers(0, V, size=V * degree)
    if hubs and hub_degree:
        hub = rng.choice(V, size=hubs, replace=False)
        src = np.concatenate([src, rng.integers(0, V, size=hubs * hub_degree)])
        dst = np.concatenate([dst, np.repeat(hub, hub_degree)])
    z = rng.standard_normal(len(src))
    order = np.argsort(src, kind="stable")
    src, dst, z = src[order], dst[order], z[order]
    first = np.searchsorted(src, np.arange(V))  # every state has an arc
    e = np.exp(z - np.maximum.reduceat(z, first)[src])
    w = np.log(mass * e / np.add.reduceat(e, first)[src]).astype(np.float32)
    start = np.zeros(V, np.uint8)
    start[rng.choice(V, size=min(n_start, V), replace=False)] = 1
    accept = (rng.random(V) < p_accept).astype(np.uint8)
    if not accept.any():
        accept[int(rng.integers(0, V))] = 1
    E = len(src)
    off = np.searchsorted(src, np.arange(V + 1)).astype(np.int32)
    return dict(num_states=V, arc_offset=off, src=src.astype(np.int32),
                dst=dst.astype(np.int32), ilabel=np.ones(E, np.int32),
                olabel=np.ones(E, np.int32), weight=w, start=start, accept=accept)


def random_dag(seed, V, mean_out=2.0, window=16, hubs=0, hub_degree=0, p_global=0.1,
               n_start=2, p_accept=0.05, p_parallel=0.05):
    """Seeded random acyclic graph (inputs of the score tests and benchmark).

    States get a random topological rank; each state has Poisson(mean_out)
    out-arcs, each to a later rank, within ``window`` ranks ahead (long
    paths) or, with probability p_global, anywhere later.  ``hubs`` states
    (ranks in the middle) also get ``hub_degree`` in-arcs from earlier ranks
    and as many out-arcs to later ranks.  An arc is duplicated with
    probability p_parallel.  Weights are binary32 N(0, 1) samples; labels
    are 1.  Starts are drawn from the first tenth of the ranks; accepting
    states at rate p_accept, plus the last rank."""
    rng = np.random.default_rng(np.random.SeedSequence([7, int(seed)]))
    V = int(V)
    rank = rng.permutation(V)          # rank[v]: topological position of v
    by_rank = np.argsort(rank)         # by_rank[r]: the state at position r
    src_r, dst_r = [], []
    deg = rng.poisson(mean_out, size=V)
    for r in range(V - 1):
        k = int(deg[r])
        if k == 0:
            continue
        far = rng.random(k) < p_global
        near = r + 1 + rng.integers(0, max(1, min(window, V - 1 - r)), size=k)
        wide = r + 1 + rng.integers(0, V - 1 - r, size=k)
        src_r.append(np.full(k, r))
        dst_r.append(np.where(far, wide, near))
    for _ in range(int(hubs)):
        if V < 3:
            break
        h = int(rng.integers(V // 4, max(V // 4 + 1, 3 * V // 4)))
        if h == 0 or h >= V - 1:
            continue
        src_r.append(rng.integers(0, h, size=hub_degree))
        dst_r.append(np.full(hub_degree, h))
        src_r.append(np.full(hub_degree, h))
        dst_r.append(rng.integers(h + 1, V, size=hub_degree))
    sr = np.concatenate(src_r) if src_r else np.zeros(0, np.int64)
    dr = np.concatenate(dst_r) if dst_r else np.zeros(0, np.int64)
    dup = rng.random(len(sr)) < p_parallel
    sr = np.concatenate([sr, sr[dup]])
    dr = np.concatenate([dr, dr[dup]])
    src = by_rank[sr].astype(np.int32)
    dst = by_rank[dr].astype(np.int32)
    order = np.argsort(src, kind="stable")
    src, dst = src[order], dst[order]
    E = len(src)
    w = rng.standard_normal(E).astype(np.float32)
    lab = np.ones(E, np.int32)
    st = np.zeros(V, np.uint8)
    if V:
        st[by_rank[rng.integers(0, max(1, V // 10), size=n_start)]] = 1
    ac = (rng.random(V) < p_accept).astype(np.uint8)
    if V:
        ac[by_rank[V - 1]] = 1
    return _finish(V, src, dst, lab, lab.copy(), w, st, ac)


def identity_fst(n_sym):
    """One state, start and accepting, with a loop s:s of weight 0 per symbol."""
    return from_arcs(1, [(0, 0, s, s, 0.0) for s in range(1, n_sym + 1)], start=[0], accept=[0])


def empty_graph():
    return from_arcs(0, [], start=[], accept=[])
