"""Pins for the CPU oracle: values and facts fixed by the paper and by
mathematics, not by the oracle itself (CPU only)."""
import math

import numpy as np
import pytest

import oracle
from oracle import brute
from paper_2110_02848_amd import synth

import fsthelp


def _fp32(x):
    return np.float32(x)


# --------------------------------------------------------------------------
# Section 3.2: the printed incoming-arc index
# --------------------------------------------------------------------------

def test_in_csr_matches_section_3_2_example():
    g = fsthelp.read_golden("csr_example_section_3_2.txt")
    V = int(g["num_states"][0][0])
    dst = np.array([int(x) for x in g["dst"][0]], np.int32)
    off, arcs = oracle.in_csr(V, dst)
    assert off.tolist() == [int(x) for x in g["inArcOffset"][0]]
    assert arcs.tolist() == [int(x) for x in g["inArcs"][0]]
    node = int(g["lookup_node"][0][0])
    il, ol = g["inLabels"][0], g["outLabels"][0]
    span = arcs[off[node]:off[node + 1]]
    assert [il[i] for i in span] == g["lookup_inLabels"][0]
    assert [ol[i] for i in span] == g["lookup_outLabels"][0]


# --------------------------------------------------------------------------
# hand-worked epsilon example
# --------------------------------------------------------------------------

def _h1_graphs():
    A = synth.from_arcs(3, [(0, 1, 1, 0, 0.5), (1, 2, 2, 3, 0.25)], start=[0], accept=[2])
    B = synth.from_arcs(3, [(0, 1, 0, 4, 1.0), (1, 2, 3, 5, 2.0)], start=[0], accept=[2])
    return A, B


@pytest.mark.parametrize("order", [oracle.ORDER_PAPER, oracle.ORDER_FORWARD])
def test_epsilon_filter_hand_example(order):
    g = fsthelp.read_golden("epsilon_filter_h1.txt")
    A, B = _h1_graphs()
    C = oracle.compose(A, B, order)
    keys = [tuple(int(x) for x in k.split(",")) for k in g["keys"][0]]
    assert list(zip(C["key_a"].tolist(), C["key_b"].tolist(), C["key_f"].tolist())) == keys
    assert C["start"].tolist() == [int(x) for x in g["start"][0]]
    assert C["accept"].tolist() == [int(x) for x in g["accept"][0]]
    arcs = [tuple(float(x) for x in row) for row in g["arc"]]
    got = list(zip(C["src"].tolist(), C["dst"].tolist(), C["ilabel"].tolist(),
                   C["olabel"].tolist(), C["weight"].tolist(), C["arc_a"].tolist(),
                   C["arc_b"].tolist()))
    assert [tuple(float(x) for x in r) for r in got] == arcs
    s = brute.scores([(x, z, w) for _, _, x, z, w in brute.composed_paths(C, 8, 4)])
    key = (tuple(int(x) for x in g["score_in"][0]), tuple(int(x) for x in g["score_out"][0]))
    assert s == {key: float(g["score"][0][0])}


def test_epsilon_filter_off_double_counts():
    A, B = _h1_graphs()
    C = oracle.compose(A, B, oracle.ORDER_FORWARD, oracle.MUT_NO_FILTER)
    s = brute.scores([(x, z, w) for _, _, x, z, w in brute.composed_paths(C, 8, 4)])
    assert len(s) == 1
    (v,) = s.values()
    assert v == pytest.approx(3.75 + math.log(2.0), abs=1e-12)


# --------------------------------------------------------------------------
# binary32 arithmetic of a matching arc: one round-to-nearest-even add
# --------------------------------------------------------------------------

@pytest.mark.parametrize("wa,wb,expect", [
    (1.0, 2.0 ** -24, 1.0),                       # tie rounds to even
    (1.0, 3 * 2.0 ** -25, 1.0 + 2.0 ** -23),      # above the tie rounds up
    (1.0 + 2.0 ** -23, 2.0 ** -24, 1.0 + 2.0 ** -22),  # tie to even, upward
    (2.0 ** -126, -(2.0 ** -127), 2.0 ** -127),   # subnormal result kept
    (2.0 ** -149, 2.0 ** -149, 2.0 ** -148),      # subnormal + subnormal
    (3.0e38, 3.0e38, math.inf),                   # overflow
])
def test_matching_weight_is_one_binary32_add(wa, wb, expect):
    A = synth.from_arcs(2, [(0, 1, 1, 2, wa)], start=[0], accept=[1])
    B = synth.from_arcs(2, [(0, 1, 2, 3, wb)], start=[0], accept=[1])
    C = oracle.compose(A, B)
    assert C["num_arcs"] == 1
    got = C["weight"][0]
    assert np.float32(expect).view(np.uint32) == got.view(np.uint32)


def test_epsilon_arc_copies_weight_bits():
    # -0.0 must survive an epsilon move (no "+ 0.0f")
    A = synth.from_arcs(2, [(0, 1, 1, 0, -0.0)], start=[0], accept=[1])
    B = synth.from_arcs(2, [(0, 1, 0, 7, -0.0)], start=[0], accept=[1])
    C = oracle.compose(A, B)
    assert C["num_arcs"] == 2
    assert all(np.float32(x).view(np.uint32) == np.float32(-0.0).view(np.uint32)
               for x in C["weight"])


# --------------------------------------------------------------------------
# identity transducer: A o Id == trim(A) and Id o B == trim(B), bitwise
# --------------------------------------------------------------------------

def _graph_as_trimmed(g, states, arcs):
    new = -np.ones(g["num_states"], np.int64)
    new[states] = np.arange(len(states))
    return states, arcs, new


@pytest.mark.parametrize("seed", range(6))
def test_identity_right(seed):
    rng = np.random.default_rng(seed)
    A = synth.random_fst(rng, 40, 3, 6, 0.2, 0.15)
    Id = synth.identity_fst(6)
    C = oracle.compose(A, Id)
    states, arcs, new = _graph_as_trimmed(A, *fsthelp.trim_graph(A))
    assert C["num_states"] == len(states)
    assert C["key_a"].tolist() == states.tolist()
    assert not C["key_b"].any() and not C["key_f"].any()
    assert C["num_arcs"] == len(arcs)
    # C arcs correspond one-to-one to A arcs (provenance), same labels, same bits
    assert sorted(C["arc_a"].tolist()) == arcs.tolist()
    a = C["arc_a"]
    assert np.array_equal(C["src"], new[A["src"][a]])
    assert np.array_equal(C["dst"], new[A["dst"][a]])
    assert np.array_equal(C["ilabel"], A["ilabel"][a])
    assert np.array_equal(C["olabel"], A["olabel"][a])
    assert np.array_equal(C["weight"].view(np.uint32), A["weight"][a].view(np.uint32))
    assert np.array_equal(C["start"], A["start"][states])
    assert np.array_equal(C["accept"], A["accept"][states])


@pytest.mark.parametrize("seed", range(6))
def test_identity_left(seed):
    rng = np.random.default_rng(100 + seed)
    B = synth.random_fst(rng, 40, 3, 6, 0.2, 0.15)
    Id = synth.identity_fst(6)
    C = oracle.compose(Id, B)
    states, arcs, new = _graph_as_trimmed(B, *fsthelp.trim_graph(B))
    assert C["key_b"].tolist() == states.tolist()
    assert not C["key_a"].any() and not C["key_f"].any()
    assert sorted(C["arc_b"].tolist()) == arcs.tolist()
    b = C["arc_b"]
    assert np.array_equal(C["src"], new[B["src"][b]])
    assert np.array_equal(C["dst"], new[B["dst"][b]])
    assert np.array_equal(C["ilabel"], B["ilabel"][b])
    assert np.array_equal(C["olabel"], B["olabel"][b])
    assert np.array_equal(C["weight"].view(np.uint32), B["weight"][b].view(np.uint32))


# --------------------------------------------------------------------------
# epsilon-free acceptors: C is the textbook product automaton, trimmed
# --------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(8))
def test_epsilon_free_product(seed):
    rng = np.random.default_rng(200 + seed)
    A = synth.random_fst(rng, 12, 3, 3, 0.0, 0.3)
    B = synth.random_fst(rng, 12, 3, 3, 0.0, 0.3)
    C = oracle.compose(A, B)
    keys = brute.product_trim_keys(A, B)
    assert set(zip(C["key_a"].tolist(), C["key_b"].tolist())) == keys
    # every matching arc pair between kept pairs appears exactly once
    n = 0
    for (qa, qb) in keys:
        for ea in range(A["arc_offset"][qa], A["arc_offset"][qa + 1]):
            for eb in range(B["arc_offset"][qb], B["arc_offset"][qb + 1]):
                if A["olabel"][ea] == B["ilabel"][eb] and \
                        (int(A["dst"][ea]), int(B["dst"][eb])) in keys:
                    n += 1
    assert C["num_arcs"] == n


# --------------------------------------------------------------------------
# Eq. (1) by bounded brute force: a bijection between path pairs and paths of C
# --------------------------------------------------------------------------

def _tiny_pair(seed):
    rng = np.random.default_rng(1000 + seed)
    A = synth.tiny_random(rng, 3, 3, 2, 0.35, p_accept=0.5, n_start=1 + seed % 2)
    B = synth.tiny_random(rng, 3, 3, 2, 0.35, p_accept=0.5, n_start=1 + (seed // 2) % 2)
    return A, B


@pytest.mark.parametrize("order", [oracle.ORDER_PAPER, oracle.ORDER_FORWARD])
def test_brute_force_path_pairs(order):
    nonempty = 0
    for seed in range(80):
        A, B = _tiny_pair(seed)
        C = oracle.compose(A, B, order)
        problems = brute.check(A, B, C, 4)
        assert not problems, (seed, problems[:5])
        assert not fsthelp.check_invariants(A, B, C), seed
        nonempty += C["num_arcs"] > 0
    assert nonempty >= 20


def test_brute_force_epsilon_cycles():
    # epsilon cycles on both sides, self-loops, two start states
    A = synth.from_arcs(2, [(0, 0, 1, 0, 0.5), (0, 1, 0, 0, -0.25), (1, 0, 2, 1, 1.0),
                            (1, 1, 0, 2, 0.125)], start=[0, 1], accept=[1])
    B = synth.from_arcs(2, [(0, 1, 0, 3, 0.5), (1, 0, 0, 0, 0.75), (0, 0, 1, 4, -1.0),
                            (1, 1, 2, 0, 0.25)], start=[0], accept=[0, 1])
    for order in (oracle.ORDER_PAPER, oracle.ORDER_FORWARD):
        C = oracle.compose(A, B, order)
        assert C["num_arcs"] > 0
        assert not brute.check(A, B, C, 5)
        assert not fsthelp.check_invariants(A, B, C)


MUTATIONS = [oracle.MUT_NO_FILTER, oracle.MUT_DROP_WB, oracle.MUT_MIDDLE_LABEL,
             oracle.MUT_ACCEPT_A, oracle.MUT_NO_TRIM, oracle.MUT_EPS_MATCH]


@pytest.mark.parametrize("mutation", MUTATIONS)
def test_pins_detect_planted_mistakes(mutation):
    """Each plausible mistake planted in the oracle is caught by the brute-force
    check or by the structural invariants on some small input."""
    caught = False
    for seed in range(80):
        A, B = _tiny_pair(seed)
        C = oracle.compose(A, B, oracle.ORDER_FORWARD, mutation)
        if brute.check(A, B, C, 4) or fsthelp.check_invariants(A, B, C):
            caught = True
            break
    assert caught


# --------------------------------------------------------------------------
# the two orders agree, and invariants hold, on the benchmark workloads
# --------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(12))
def test_orders_agree_random_small(seed):
    A, B = synth.workload("random-64", seed)
    Cp = oracle.compose(A, B, oracle.ORDER_PAPER)
    Cf = oracle.compose(A, B, oracle.ORDER_FORWARD)
    assert not fsthelp.compare_results(Cp, Cf)
    assert not fsthelp.check_invariants(A, B, Cp)


@pytest.mark.parametrize("name,seed", [("random-1000", 1), ("random-1000", 2),
                                       ("random-5000", 0), ("random-5000", 7)])
def test_orders_agree_random_large(name, seed):
    A, B = synth.workload(name, seed)
    Cp = oracle.compose(A, B, oracle.ORDER_PAPER)
    Cf = oracle.compose(A, B, oracle.ORDER_FORWARD)
    assert not fsthelp.compare_results(Cp, Cf)
    assert not fsthelp.check_invariants(A, B, Cp)


# --------------------------------------------------------------------------
# emissions o lexicon: closed forms at full size
# --------------------------------------------------------------------------

def _lex_check(A, B, meta, C):
    T = meta["spec"].T
    V, E = fsthelp.lexicon_closed_form(T, meta["spellings"])
    assert (C["num_states"], C["num_arcs"]) == (V, E)
    # token arcs carry the emission log-probability bits unchanged
    tok = C["arc_a"] >= 0
    assert np.array_equal(C["weight"][tok].view(np.uint32),
                          A["weight"][C["arc_a"][tok]].view(np.uint32))
    assert not np.any(C["weight"][~tok])
    ref = fsthelp.lexicon_total_score(meta["table"], meta["spellings"])
    got = fsthelp.dag_total_score(C)
    assert got == pytest.approx(ref, rel=1e-9, abs=1e-9)


def test_lexicon_closed_form_small():
    spec = synth.LexSpec(T=30, C=6, W=40, len_lo=2, len_hi=5)
    A, B, meta = synth.emissions_lexicon("lexicon-T100-W1000", 3, spec=spec)
    for order in (oracle.ORDER_PAPER, oracle.ORDER_FORWARD):
        C = oracle.compose(A, B, order)
        assert not fsthelp.check_invariants(A, B, C)
        _lex_check(A, B, meta, C)


def test_lexicon_closed_form_T100_W1000():
    A, B, meta = synth.emissions_lexicon("lexicon-T100-W1000", 0)
    C = oracle.compose(A, B, oracle.ORDER_FORWARD)
    assert not fsthelp.check_invariants(A, B, C)
    _lex_check(A, B, meta, C)
    Cp = oracle.compose(A, B, oracle.ORDER_PAPER)
    assert not fsthelp.compare_results(Cp, C)


@pytest.mark.slow
def test_lexicon_closed_form_T500_W10000():
    A, B, meta = synth.emissions_lexicon("lexicon-T500-W10000", 0)
    C = oracle.compose(A, B, oracle.ORDER_FORWARD)
    _lex_check(A, B, meta, C)


# --------------------------------------------------------------------------
# degenerate inputs
# --------------------------------------------------------------------------

def test_empty_inputs():
    E0 = synth.empty_graph()
    A, _ = synth.workload("random-64", 0)
    for X, Y in ((E0, E0), (E0, A), (A, E0)):
        C = oracle.compose(X, Y)
        assert C["num_states"] == 0 and C["num_arcs"] == 0
        assert C["arc_offset"].tolist() == [0]


def test_no_start_or_dead_start_gives_empty():
    A = synth.from_arcs(2, [(0, 1, 1, 1, 0.0)], start=[], accept=[1])
    B = synth.from_arcs(2, [(0, 1, 1, 1, 0.0)], start=[0], accept=[1])
    assert oracle.compose(A, B)["num_states"] == 0
    A2 = synth.from_arcs(2, [(0, 1, 1, 1, 0.0)], start=[0], accept=[1])
    B2 = synth.from_arcs(2, [(0, 1, 2, 2, 0.0)], start=[0], accept=[1])
    assert oracle.compose(A2, B2)["num_states"] == 0


def test_start_and_accept_single_state():
    A = synth.from_arcs(1, [], start=[0], accept=[0])
    B = synth.from_arcs(1, [], start=[0], accept=[0])
    C = oracle.compose(A, B)
    assert C["num_states"] == 1 and C["num_arcs"] == 0
    assert C["start"].tolist() == [1] and C["accept"].tolist() == [1]


def test_parallel_arcs_are_kept():
    A = synth.from_arcs(2, [(0, 1, 1, 5, 0.5), (0, 1, 2, 5, 0.25)], start=[0], accept=[1])
    B = synth.from_arcs(2, [(0, 1, 5, 7, 1.0), (0, 1, 5, 8, 2.0)], start=[0], accept=[1])
    C = oracle.compose(A, B)
    assert C["num_arcs"] == 4
    assert list(zip(C["arc_a"].tolist(), C["arc_b"].tolist())) == [(0, 0), (0, 1), (1, 0), (1, 1)]


def test_canonical_arc_order():
    # epsilon-A arcs, then epsilon-B arcs, then matching arcs grouped by label
    A = synth.from_arcs(1, [(0, 0, 1, 9, 0.0), (0, 0, 2, 0, 0.0), (0, 0, 3, 4, 0.0)],
                        start=[0], accept=[0])
    B = synth.from_arcs(1, [(0, 0, 4, 1, 0.0), (0, 0, 0, 2, 0.0), (0, 0, 9, 3, 0.0)],
                        start=[0], accept=[0])
    C = oracle.compose(A, B)
    s0 = C["src"] == 0
    got = list(zip(C["arc_a"][s0].tolist(), C["arc_b"][s0].tolist()))
    assert got == [(1, -1), (-1, 1), (2, 0), (0, 2)]


def test_arcless_side_with_epsilon_moves():
    # A has no arcs (start and accepting); only B's epsilon-input arcs move
    A = synth.from_arcs(2, [], start=[0, 1], accept=[0, 1])
    B = synth.from_arcs(3, [(0, 1, 0, 4, 0.5), (1, 2, 0, 0, 0.25), (0, 2, 3, 1, 1.0)],
                        start=[0], accept=[2])
    for order in (oracle.ORDER_PAPER, oracle.ORDER_FORWARD):
        C = oracle.compose(A, B, order)
        assert C["num_states"] == 6 and C["num_arcs"] == 4
        assert not fsthelp.check_invariants(A, B, C)
        assert not brute.check(A, B, C, 3)
