"""The oracle's trim key set and arcs at full size of the random workloads,
checked against an independent construction: the dense product graph of all
moves (a join of all arcs on the matched label) searched forward from the
start keys and backward from the accepting keys (``product_bfs``).  This pins
the oracle where no printed result exists, at the real sizes: 64 states
(many seeds), 1000 states, and 5000 states (the seeds whose composition is
not empty, one that is, and a supercritical variant with 16 symbols)."""
import numpy as np
import pytest

import oracle
from paper_2110_02848_amd import synth

import product_bfs


def _sorted_oracle_arcs(R, VB):
    keys = (R["key_a"].astype(np.int64) * VB + R["key_b"]) * 2 + R["key_f"]
    src = keys[R["src"].astype(np.int64)] if R["num_arcs"] else np.zeros(0, np.int64)
    dst = keys[R["dst"].astype(np.int64)] if R["num_arcs"] else np.zeros(0, np.int64)
    a = R["arc_a"].astype(np.int64)
    b = R["arc_b"].astype(np.int64)
    big = np.int64(1) << 40
    order = np.lexsort((np.where(b >= 0, b, big), np.where(a >= 0, a, big), src))
    return keys, src[order], dst[order], a[order], b[order], R["weight"][order]


def _weights(A, B, a, b):
    """Weight of each arc from its provenance: one binary32 add for a
    matching arc, the single arc's weight copied for an epsilon arc."""
    # one padding entry each, so masked lookups stay in range for a graph
    # without arcs
    wa = np.append(np.asarray(A["weight"], np.float32), np.float32(0))
    wb = np.append(np.asarray(B["weight"], np.float32), np.float32(0))
    both = (a >= 0) & (b >= 0)
    w = np.where(a >= 0, wa[np.maximum(a, 0)], wb[np.maximum(b, 0)]).astype(np.float32)
    w[both] = wa[a[both]] + wb[b[both]]
    return w


def check_against_product(A, B):
    R = oracle.compose(A, B, oracle.ORDER_FORWARD)
    P = product_bfs.trim_product(A, B)
    keys, src, dst, a, b, w = _sorted_oracle_arcs(R, int(B["num_states"]))
    assert np.array_equal(keys, P["keys"])
    assert R["stats"]["accessible"] == P["accessible"]
    for x, y in ((src, P["src"]), (dst, P["dst"]), (a, P["arc_a"]), (b, P["arc_b"])):
        assert np.array_equal(x, y)
    assert np.array_equal(w.view(np.uint32),
                          _weights(A, B, P["arc_a"], P["arc_b"]).view(np.uint32))
    return R


@pytest.mark.parametrize("seed", range(20))
def test_random_64_full_product(seed):
    A, B = synth.workload("random-64", seed)
    check_against_product(A, B)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_random_1000_full_product(seed):
    A, B = synth.workload("random-1000", seed)
    R = check_against_product(A, B)
    assert (R["num_states"] > 0) == (seed > 0)


@pytest.mark.parametrize("seed", [0, 471, 1175, 2216])
def test_random_5000_full_product(seed):
    A, B = synth.workload("random-5000", seed)
    R = check_against_product(A, B)
    assert (R["num_states"] > 0) == (seed != 0)


def test_random_5000_supercritical_full_product():
    ss = np.random.SeedSequence([31, 16, 0])
    ra, rb = [np.random.default_rng(s) for s in ss.spawn(2)]
    A = synth.random_fst(ra, 5000, 4, 16, 0.05, 0.05)
    B = synth.random_fst(rb, 5000, 4, 16, 0.05, 0.05)
    R = check_against_product(A, B)
    assert R["num_states"] > 3000000


@pytest.mark.parametrize("seed", range(30))
def test_tiny_epsilon_full_product(seed):
    rng = np.random.default_rng([606, seed])
    A = synth.tiny_random(rng, int(rng.integers(1, 7)), 4, 3, 0.35, n_start=1 + seed % 2)
    B = synth.tiny_random(rng, int(rng.integers(1, 7)), 4, 3, 0.35, n_start=1 + seed % 3)
    check_against_product(A, B)


def test_product_check_catches_a_planted_mistake():
    """The same comparison fails for an oracle without the epsilon filter
    (a planted mistake): the check is sensitive to the move rules."""
    for seed in range(40):
        rng = np.random.default_rng([607, seed])
        A = synth.tiny_random(rng, 4, 4, 2, 0.4)
        B = synth.tiny_random(rng, 4, 4, 2, 0.4)
        P = product_bfs.trim_product(A, B)
        R = oracle.compose(A, B, oracle.ORDER_FORWARD, mutation=oracle.MUT_NO_FILTER)
        keys = (R["key_a"].astype(np.int64) * B["num_states"] + R["key_b"]) * 2 + R["key_f"]
        if not np.array_equal(keys, P["keys"]) or R["num_arcs"] != len(P["src"]):
            return
    pytest.fail("no seed tells the unfiltered oracle from the product search")
