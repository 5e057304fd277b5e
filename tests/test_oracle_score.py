"""Pins for the score oracle (forward / backward log-semiring scores,
posteriors, provenance scatter): each is checked against something other
than the oracle itself -- explicit path enumeration, a frame recursion over
word segmentations, finite differences, a library histogram (CPU only)."""
import math

import numpy as np
import pytest

import oracle
from paper_2110_02848_amd import synth

import fsthelp


# --------------------------------------------------------------------------
# tiny acyclic graphs and explicit path enumeration
# --------------------------------------------------------------------------

def tiny_dag(seed, V=None):
    """Random DAG: arcs only go forward in a random permutation of the
    states, parallel arcs allowed, several starts, any accept set."""
    rng = np.random.default_rng(seed)
    V = int(rng.integers(1, 9)) if V is None else V
    rank = rng.permutation(V)  # topological position of each state
    by_rank = np.argsort(rank)
    arcs = []
    for _ in range(int(rng.integers(0, 2 * V + 1))):
        i, j = sorted(rng.integers(0, V, size=2).tolist())
        if i == j:
            continue
        w = float(np.float32(rng.standard_normal()))
        arcs.append((int(by_rank[i]), int(by_rank[j]), 1, 1, w))
    starts = sorted(set(rng.integers(0, V, size=int(rng.integers(1, 3))).tolist()))
    accepts = [v for v in range(V) if rng.random() < 0.4]
    return synth.from_arcs(V, arcs, start=starts, accept=accepts)


def _paths_from(G, v, weights):
    """Every path starting at v: (end state, weight, arcs used)."""
    off, dst = G["arc_offset"], G["dst"]
    out = [(v, 0.0, ())]
    for e in range(off[v], off[v + 1]):
        for end, w, used in _paths_from(G, int(dst[e]), weights):
            out.append((end, weights[e] + w, (e,) + used))
    return out


def _logsum(ws):
    if not ws:
        return -math.inf
    m = max(ws)
    return m + math.log(math.fsum(math.exp(w - m) for w in ws))


def enumerate_scores(G, weights=None):
    """alpha, beta and total by listing every path (float64)."""
    V = int(G["num_states"])
    w = np.asarray(G["weight"], np.float64) if weights is None else weights
    paths = {v: _paths_from(G, v, w) for v in range(V)}
    alpha_terms = [[] for _ in range(V)]
    total_terms = []
    for s in range(V):
        if not G["start"][s]:
            continue
        for end, pw, _ in paths[s]:
            alpha_terms[end].append(pw)
            if G["accept"][end]:
                total_terms.append(pw)
    beta = [_logsum([pw for end, pw, _ in paths[v] if G["accept"][end]]) for v in range(V)]
    return np.array([_logsum(t) for t in alpha_terms]), np.array(beta), _logsum(total_terms)


def _close(a, b, tol=1e-12):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    same_inf = (a == b) & np.isinf(a)
    with np.errstate(invalid="ignore"):
        err = np.abs(np.where(same_inf, 0.0, a - b))
    return bool(np.all(np.isfinite(err) & (err <= tol * (1.0 + np.abs(np.where(same_inf, 0.0, b))))))


@pytest.mark.parametrize("seed", range(60))
def test_score_matches_path_enumeration(seed):
    G = tiny_dag(seed)
    r = oracle.score(G)
    alpha, beta, total = enumerate_scores(G)
    assert _close(r["alpha"], alpha)
    assert _close(r["beta"], beta)
    assert _close([r["total"], r["total_bwd"]], [total, total])


@pytest.mark.parametrize("mutation", [oracle.SMUT_MAX, oracle.SMUT_DROP_WEIGHT,
                                      oracle.SMUT_ALL_ACCEPT, oracle.SMUT_NO_START])
def test_score_mutations_fail_path_enumeration(mutation):
    caught = 0
    for seed in range(40):
        G = tiny_dag(seed)
        r = oracle.score(G, mutation=mutation)
        alpha, beta, total = enumerate_scores(G)
        ok = (_close(r["alpha"], alpha) and _close(r["beta"], beta)
              and _close([r["total"], r["total_bwd"]], [total, total]))
        caught += not ok
    assert caught > 0


def test_score_refuses_cycles():
    # a 2-cycle that no start state reaches still makes the graph cyclic
    G = synth.from_arcs(4, [(0, 1, 1, 1, 0.0), (2, 3, 1, 1, 0.0), (3, 2, 1, 1, 0.0)],
                        start=[0], accept=[1])
    with pytest.raises(oracle.CycleError):
        oracle.score(G)
    loop = synth.from_arcs(1, [(0, 0, 1, 1, -1.0)], start=[0], accept=[0])
    with pytest.raises(oracle.CycleError):
        oracle.score(loop)


def test_score_special_cases():
    empty = synth.empty_graph()
    r = oracle.score(empty)
    assert r["total"] == -math.inf and r["longest"] == 0 and len(r["alpha"]) == 0
    one = synth.from_arcs(1, [], start=[0], accept=[0])
    r = oracle.score(one)
    assert r["alpha"].tolist() == [0.0] and r["beta"].tolist() == [0.0] and r["total"] == 0.0
    # no accepting state: every beta and the total are -inf, alpha is not
    G = synth.from_arcs(3, [(0, 1, 1, 1, -1.0), (1, 2, 1, 1, -2.0)], start=[0], accept=[])
    r = oracle.score(G)
    assert np.all(r["beta"] == -np.inf) and r["total"] == -math.inf
    assert r["alpha"].tolist() == [0.0, -1.0, -3.0]
    # a state no start reaches keeps alpha = -inf; one that reaches no
    # accepting state keeps beta = -inf
    G = synth.from_arcs(4, [(0, 1, 1, 1, 0.5), (2, 1, 1, 1, 0.25), (0, 3, 1, 1, 1.0)],
                        start=[0], accept=[1])
    r = oracle.score(G)
    assert r["alpha"][2] == -math.inf and r["beta"][3] == -math.inf
    assert r["total"] == 0.5 and r["longest"] == 2


def test_score_parallel_arcs_add_up():
    # two parallel arcs of weight log(1/4) and log(3/4): total log(1) = 0
    G = synth.from_arcs(2, [(0, 1, 1, 1, math.log(0.25)), (0, 1, 2, 2, math.log(0.75))],
                        start=[0], accept=[1])
    r = oracle.score(G)
    assert abs(r["total"]) < 1e-7  # the weights are binary32


# --------------------------------------------------------------------------
# emissions o lexicon: the total is a recursion over word segmentations
# --------------------------------------------------------------------------

def _small_lexicon(seed, T=14, C=5, W=12, lo=2, hi=4):
    spec = synth.LexSpec(T, C, W, lo, hi)
    A, B, meta = synth.emissions_lexicon("lexicon-T100-W1000", seed, spec=spec)
    return A, B, meta


def word_arcs(B):
    """For each word (in word-id order): its entry arc, token arcs and exit
    arc in B (followed from the root)."""
    off, dst, ol = B["arc_offset"], B["dst"], B["olabel"]
    words = {}
    for e0 in range(off[0], off[1]):
        chain = [e0]
        s = int(dst[e0])
        while s != 0:
            e = int(off[s])
            chain.append(e)
            s = int(dst[e])
        words[int(ol[e0])] = chain
    return [words[k] for k in sorted(words)]


def segmentation_total(table, spellings, wB, chains):
    """log-sum over segmentations of the T frames into words of
    sum(emission log-probs) + sum(B arc weights of the words), float64."""
    T = table.shape[0]
    F = np.full(T + 1, -np.inf)
    F[0] = 0.0
    for t in range(1, T + 1):
        terms = []
        for s, ch in zip(spellings, chains):
            L = len(s)
            if L > t or F[t - L] == -np.inf:
                continue
            em = sum(float(table[t - L + j, int(s[j]) - 1]) for j in range(L))
            terms.append(F[t - L] + em + math.fsum(float(wB[e]) for e in ch))
        F[t] = _logsum(terms)
    return F[T]


@pytest.mark.parametrize("seed", range(4))
def test_score_lexicon_matches_segmentation_recursion(seed):
    A, B, meta = _small_lexicon(seed)
    C = oracle.compose(A, B)
    r = oracle.score(C)
    ref = segmentation_total(meta["table"].astype(np.float64), meta["spellings"],
                             np.zeros(len(B["src"])), word_arcs(B))
    assert abs(r["total"] - ref) <= 1e-9 * (1 + abs(ref))
    assert abs(r["total_bwd"] - ref) <= 1e-9 * (1 + abs(ref))


def test_score_lexicon_T100_matches_frame_recursion():
    A, B, meta = synth.emissions_lexicon("lexicon-T100-W1000", 0)
    C = oracle.compose(A, B)
    r = oracle.score(C)
    ref = fsthelp.lexicon_total_score(meta["table"], meta["spellings"])
    assert abs(r["total"] - ref) <= 1e-9 * (1 + abs(ref))
    # the longest path: one arc per frame plus an entry and an exit arc per
    # word, so at least T + 1 states
    assert r["longest"] >= meta["spec"].T + 1


# --------------------------------------------------------------------------
# posteriors: the derivative of the total by an arc weight
# --------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(25))
def test_posterior_matches_finite_differences(seed):
    G = tiny_dag(seed + 100)
    if len(G["src"]) == 0:
        return
    r = oracle.score(G)
    post = oracle.posterior(G, r["alpha"], r["beta"], r["total"])
    if r["total"] == -math.inf:
        assert np.all(post == 0)
        return
    w0 = np.asarray(G["weight"], np.float64)
    h = 1e-6
    for e in range(len(w0)):
        wp, wm = w0.copy(), w0.copy()
        wp[e] += h
        wm[e] -= h
        fd = (enumerate_scores(G, wp)[2] - enumerate_scores(G, wm)[2]) / (2 * h)
        assert abs(post[e] - fd) <= 1e-7, (e, post[e], fd)


def test_posterior_flow_is_conserved():
    # posterior mass into a state that is neither start nor accepting equals
    # the mass out of it; the mass out of the start states is 1
    A, B, meta = _small_lexicon(3)
    C = oracle.compose(A, B)
    r = oracle.score(C)
    post = oracle.posterior(C, r["alpha"], r["beta"], r["total"])
    V = C["num_states"]
    inflow = np.bincount(C["dst"], weights=post, minlength=V)
    outflow = np.bincount(C["src"], weights=post, minlength=V)
    mid = (C["start"] == 0) & (C["accept"] == 0)
    assert np.allclose(inflow[mid], outflow[mid], atol=1e-12, rtol=1e-9)
    assert abs(outflow[C["start"] == 1].sum() - 1.0) < 1e-9


# --------------------------------------------------------------------------
# scatter through provenance
# --------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(5))
def test_scatter_matches_bincount(seed):
    rng = np.random.default_rng(seed)
    m = int(rng.integers(1, 50))
    n = int(rng.integers(0, 400))
    idx = rng.integers(-1, m, size=n).astype(np.int32)
    g = rng.standard_normal(n)
    got = oracle.scatter(g, idx, m)
    keep = idx >= 0
    ref = np.bincount(idx[keep], weights=g[keep], minlength=m)
    assert np.allclose(got, ref, rtol=1e-13, atol=1e-13)


def test_scatter_rejects_bad_index():
    with pytest.raises(ValueError):
        oracle.scatter(np.ones(3), np.array([0, 5, 1], np.int32), 3)


@pytest.mark.parametrize("seed", range(3))
def test_operand_gradients_match_finite_differences(seed):
    """d total / d w for every arc of A (the emission table) and of B,
    through posterior + scatter on the oracle's C, against central
    differences of the segmentation recursion (which never builds C)."""
    A, B, meta = _small_lexicon(seed, T=9, C=4, W=6, lo=2, hi=3)
    rng = np.random.default_rng(1000 + seed)
    B = dict(B)
    B["weight"] = (0.5 * rng.standard_normal(len(B["src"]))).astype(np.float32)
    C = oracle.compose(A, B)
    r = oracle.score(C)
    post = oracle.posterior(C, r["alpha"], r["beta"], r["total"])
    gA = oracle.scatter(post, C["arc_a"], len(A["src"]))
    gB = oracle.scatter(post, C["arc_b"], len(B["src"]))
    table = meta["table"].astype(np.float64)
    wB = B["weight"].astype(np.float64)
    chains = word_arcs(B)
    sp = meta["spellings"]
    T, Cn = table.shape
    h = 1e-5
    # A's arc (t, c) is arc t * C + (c - 1) of the emission graph
    for t in range(T):
        for c in range(Cn):
            tp, tm = table.copy(), table.copy()
            tp[t, c] += h
            tm[t, c] -= h
            fd = (segmentation_total(tp, sp, wB, chains) - segmentation_total(tm, sp, wB, chains)) / (2 * h)
            # binary32 arc weights of C move the posteriors by ~1e-6
            assert abs(gA[t * Cn + c] - fd) <= 2e-5, (t, c, gA[t * Cn + c], fd)
    for e in range(len(wB)):
        wp, wm = wB.copy(), wB.copy()
        wp[e] += h
        wm[e] -= h
        fd = (segmentation_total(table, sp, wp, chains) - segmentation_total(table, sp, wm, chains)) / (2 * h)
        assert abs(gB[e] - fd) <= 2e-5, (e, gB[e], fd)


def test_emission_gradients_sum_to_one_per_frame():
    # every accepting path of emissions o lexicon takes exactly one arc of A
    # per frame, so the posteriors of a frame's arcs of A add up to 1
    A, B, meta = synth.emissions_lexicon("lexicon-T100-W1000", 1)
    C = oracle.compose(A, B)
    r = oracle.score(C)
    post = oracle.posterior(C, r["alpha"], r["beta"], r["total"])
    gA = oracle.scatter(post, C["arc_a"], len(A["src"]))
    T, Cn = meta["table"].shape
    assert np.allclose(gA.reshape(T, Cn).sum(axis=1), 1.0, atol=1e-9)
    # and the entry arc, the token arcs and the exit arc of a word are used
    # together, so their gradients agree
    gB = oracle.scatter(post, C["arc_b"], len(B["src"]))
    for ch in word_arcs(B)[:200]:
        assert np.allclose(gB[ch], gB[ch[0]], rtol=1e-9, atol=1e-12)
