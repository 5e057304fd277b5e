"""Pins of the three-input oracle, C = A o B o D composed at once (the
N-way composition the paper names as the next step, Section 5), to things
other than itself:

* bounded brute force (Eq. (1) read for three inputs): every triple of
  accepting paths of A, B and D whose middle strings agree is realised by
  exactly one accepting path of C, with its strings and weight, and the
  per-(x, w) log-sum scores agree; four planted mistakes in the oracle each
  fail it;
* the chained two-input oracle, (A o B) o D: when D has no epsilon input
  the filter bits are never set on the second level, and the two results
  are the same graph, bit for bit (structure, labels, weights, provenance
  through A o B); with epsilon inputs on every side (acyclic inputs, so
  every path can be enumerated) the per-(x, w) scores agree;
* emissions o lexicon o word grammar: the total path score of C equals a
  recursion over the frames and the grammar states that never builds C;
* invariants of every result (trim, flags and labels and weight bits from
  keys and provenance, unique provenance per state, normalised filter
  bits).
"""
import math

import numpy as np
import pytest

import oracle
from oracle import brute
from paper_2110_02848_amd import synth

import fsthelp


def _tiny_triple(seed, fam=808):
    rng = np.random.default_rng([fam, seed])

    def g():
        return synth.tiny_random(rng, int(rng.integers(1, 4)), 4, 2, 0.4, p_accept=0.6,
                                 n_start=1 + seed % 2)
    return g(), g(), g()


@pytest.mark.parametrize("seed", range(60))
def test_brute_force_bijection(seed):
    A, B, D = _tiny_triple(seed)
    C = oracle.compose3(A, B, D)
    assert brute.check3(A, B, D, C, 4) == []
    assert fsthelp.check_invariants3(A, B, D, C) == []


@pytest.mark.parametrize("mutation", [oracle.MUT3_NO_INNER_FILTER, oracle.MUT3_NO_OUTER_FILTER,
                                      oracle.MUT3_DROP_WD, oracle.MUT3_OUTER_LABEL])
def test_planted_mistakes_fail_the_brute_force(mutation):
    for seed in range(60):
        A, B, D = _tiny_triple(seed)
        C = oracle.compose3(A, B, D, mutation=mutation)
        if brute.check3(A, B, D, C, 4):
            return
    pytest.fail(f"mutation {mutation} passes every brute-force case")


def graph_of(C):
    return {k: C[k] for k in ("num_states", "arc_offset", "src", "dst", "ilabel", "olabel",
                              "weight", "start", "accept")}


def chained3(A, B, D):
    """(A o B) o D by the two-input oracle, states and arcs written as those
    of a three-input result (keys through A o B's keys, provenance through
    A o B's provenance), in canonical three-input order."""
    AB = oracle.compose(A, B, oracle.ORDER_FORWARD)
    CD = oracle.compose(graph_of(AB), D, oracle.ORDER_FORWARD)
    ka = CD["key_a"].astype(np.int64)
    aa = CD["arc_a"].astype(np.int64)
    pad = lambda x: np.append(np.asarray(x, np.int32), np.int32(-1))
    raw = dict(num_states=CD["num_states"], num_arcs=CD["num_arcs"],
               key_a=AB["key_a"][ka] if len(ka) else np.zeros(0, np.int32),
               key_b=AB["key_b"][ka] if len(ka) else np.zeros(0, np.int32),
               key_fab=AB["key_f"][ka] if len(ka) else np.zeros(0, np.uint8),
               key_d=CD["key_b"], key_f=CD["key_f"], start=CD["start"], accept=CD["accept"],
               src=CD["src"], dst=CD["dst"], ilabel=CD["ilabel"], olabel=CD["olabel"],
               weight=CD["weight"], arc_a=pad(AB["arc_a"])[aa], arc_b=pad(AB["arc_b"])[aa],
               arc_d=CD["arc_b"], stats={})
    return oracle.canonicalize3(raw, A)


def _no_eps_input(g):
    g = dict(g)
    g["ilabel"] = np.where(g["ilabel"] == 0, 1, g["ilabel"]).astype(np.int32)
    return g


@pytest.mark.parametrize("seed", range(40))
def test_equals_chained_when_d_has_no_epsilon_input(seed):
    A, B, D = _tiny_triple(seed, fam=809)
    D = _no_eps_input(D)
    C3 = oracle.compose3(A, B, D)
    CC = chained3(A, B, D)
    assert not fsthelp.compare_results(C3, CC, oracle.RESULT3_KEYS)


@pytest.mark.parametrize("seed", range(4))
def test_equals_chained_random_transducers(seed):
    rng = np.random.default_rng([810, seed])
    A = synth.random_fst(rng, 30, 3, 4, 0.2, 0.3)
    B = synth.random_fst(rng, 30, 3, 4, 0.2, 0.3)
    D = _no_eps_input(synth.random_fst(rng, 20, 3, 4, 0.2, 0.3))
    C3 = oracle.compose3(A, B, D)
    assert C3["num_arcs"] > 100
    assert not fsthelp.compare_results(C3, chained3(A, B, D), oracle.RESULT3_KEYS)
    assert fsthelp.check_invariants3(A, B, D, C3) == []


def test_equals_chained_lexicon_grammar_without_backoff():
    spec = synth.GrammarSpec(40, 12, 300, 2, 6, 6, 60, 0.0, 0.5)
    A, B, D, _ = synth.emissions_lexicon_grammar("grammar-T40-W300-G6", 0, spec=spec)
    assert not np.any(D["ilabel"] == 0)
    C3 = oracle.compose3(A, B, D)
    assert C3["num_states"] > 10000
    assert not fsthelp.compare_results(C3, chained3(A, B, D), oracle.RESULT3_KEYS)


def _tiny_dag(rng, V, n_sym, p_eps):
    """Acyclic transducer (arcs from lower to higher states), epsilons on
    both sides, several accepting states."""
    arcs = []
    for s in range(V - 1):
        for _ in range(int(rng.integers(1, 4))):
            lab = lambda: 0 if rng.random() < p_eps else int(rng.integers(1, n_sym + 1))
            arcs.append((s, int(rng.integers(s + 1, V)), lab(), lab(),
                         float(np.float32(rng.standard_normal()))))
    acc = [V - 1] + [s for s in range(V - 1) if rng.random() < 0.3]
    return synth.from_arcs(V, arcs, start=[0], accept=sorted(set(acc)))


def _all_path_scores(C):
    """Per-(x, w) log-sum over every accepting path of an acyclic graph."""
    outs = [list(range(int(C["arc_offset"][v]), int(C["arc_offset"][v + 1])))
            for v in range(C["num_states"])]
    items = []

    def walk(q, path):
        if C["accept"][q]:
            x = tuple(int(C["ilabel"][e]) for e in path if C["ilabel"][e] != 0)
            z = tuple(int(C["olabel"][e]) for e in path if C["olabel"][e] != 0)
            items.append((x, z, math.fsum(float(C["weight"][e]) for e in path)))
        for e in outs[q]:
            path.append(e)
            walk(int(C["dst"][e]), path)
            path.pop()

    for s in range(C["num_states"]):
        if C["start"][s]:
            walk(s, [])
    return brute.scores(items)


@pytest.mark.parametrize("seed", range(30))
def test_scores_equal_chained_on_acyclic_inputs(seed):
    rng = np.random.default_rng([811, seed])
    A, B, D = (_tiny_dag(rng, int(rng.integers(3, 6)), 2, 0.35) for _ in range(3))
    C3 = oracle.compose3(A, B, D)
    s3, sc = _all_path_scores(C3), _all_path_scores(chained3(A, B, D))
    assert set(s3) == set(sc)
    for k in s3:
        assert abs(s3[k] - sc[k]) <= 1e-5 * (1 + abs(sc[k])), k
    assert fsthelp.check_invariants3(A, B, D, C3) == []


def lexicon_grammar_total(table, spellings, D):
    """Log of the total path sum of emissions o lexicon o grammar by a
    recursion over frames t and grammar states g (float64): a[t][g] sums the
    prefixes that end a word at frame t in grammar state g, before and after
    the grammar's epsilon arcs (backoffs, which lead to a state without
    epsilon arcs, so at most one is taken between two words)."""
    T = table.shape[0]
    G = D["num_states"]
    tab = table.astype(np.float64)
    eps_arcs = [(int(s), int(d), float(w)) for s, d, i, w in
                zip(D["src"], D["dst"], D["ilabel"], D["weight"]) if i == 0]
    word_arcs = {}
    for s, d, i, w in zip(D["src"], D["dst"], D["ilabel"], D["weight"]):
        if i != 0:
            word_arcs.setdefault(int(i), []).append((int(s), int(d), float(w)))
    for s, d, _ in eps_arcs:
        assert not any(x == d for x, _, _ in eps_arcs), "one epsilon step between words"

    def lse(xs):
        xs = [x for x in xs if x != -math.inf]
        if not xs:
            return -math.inf
        m = max(xs)
        return m + math.log(math.fsum(math.exp(x - m) for x in xs))

    def closure(a):
        b = [[x] for x in a]
        for s, d, w in eps_arcs:
            if a[s] != -math.inf:
                b[d].append(a[s] + w)
        return [lse(x) for x in b]

    alpha = [[-math.inf] * G for _ in range(T + 1)]
    alpha[0][0] = 0.0
    closed = [None] * (T + 1)
    closed[0] = closure(alpha[0])
    for t in range(1, T + 1):
        terms = [[] for _ in range(G)]
        for wid, sp in enumerate(spellings, start=1):
            L = len(sp)
            if L > t or wid not in word_arcs:
                continue
            emit = math.fsum(tab[t - L + k, sp[k] - 1] for k in range(L))
            for s, d, w in word_arcs[wid]:
                if closed[t - L][s] != -math.inf:
                    terms[d].append(closed[t - L][s] + w + emit)
        alpha[t] = [lse(x) for x in terms]
        closed[t] = closure(alpha[t])
    return lse([closed[T][g] for g in range(G) if D["accept"][g]])


@pytest.mark.parametrize("name", ["grammar-T40-W300-G6", "grammar-T100-W1000-G20"])
def test_lexicon_grammar_total_score(name):
    A, B, D, meta = synth.emissions_lexicon_grammar(name, 0)
    C3 = oracle.compose3(A, B, D)
    ref = lexicon_grammar_total(meta["table"], meta["spellings"], D)
    tot = oracle.score(C3)["total"]
    assert abs(tot - ref) <= 1e-9 * (1 + abs(ref)) * C3["num_arcs"] ** 0.5, (tot, ref)
    if name == "grammar-T40-W300-G6":
        assert fsthelp.check_invariants3(A, B, D, C3) == []


def test_degenerate_inputs():
    E0 = synth.empty_graph()
    one = synth.from_arcs(1, [], start=[0], accept=[0])
    C = oracle.compose3(E0, one, one)
    assert C["num_states"] == 0
    C = oracle.compose3(one, one, one)
    assert C["num_states"] == 1 and C["num_arcs"] == 0 and C["start"].tolist() == [1]
    nostart = synth.from_arcs(1, [], start=[], accept=[0])
    assert oracle.compose3(one, nostart, one)["num_states"] == 0
