"""Pins for the cyclic-score oracle (``oracle.cyclic``): each is checked
against something other than the oracle itself -- geometric series in closed
form, explicit enumeration of every path up to a length whose tail is below
rounding, the acyclic score oracle (``score.c``) on graphs without cycles,
and the divergence of sums whose arc mass reaches 1 (CPU only)."""
import math

import numpy as np
import pytest

import oracle
from oracle import cyclic
from paper_2110_02848_amd import synth


def _g(V, arcs, start, accept):
    return synth.from_arcs(V, [(s, d, 1, 1, w) for s, d, w in arcs], start=start, accept=accept)


def _w(x):
    return float(np.float32(x))


@pytest.mark.parametrize("w", [-0.05, -0.7, -3.0, -20.0])
def test_self_loop_is_a_geometric_series(w):
    w = _w(w)
    r = cyclic.score_cyclic(_g(1, [(0, 0, w)], [0], [0]))
    want = -math.log1p(-math.exp(w))  # log of 1 + e^w + e^2w + ...
    assert abs(r["alpha"][0] - want) < 1e-12 * max(1.0, abs(want))
    assert abs(r["beta"][0] - want) < 1e-12 * max(1.0, abs(want))
    assert abs(r["total"] - want) < 1e-12 * max(1.0, abs(want))


def test_two_state_cycle_closed_form():
    w1, w2, w3 = _w(-0.4), _w(-1.1), _w(0.3)
    # 0 -> 1 (w1), 1 -> 0 (w2), 1 -> 2 (w3); start 0, accept 2
    r = cyclic.score_cyclic(_g(3, [(0, 1, w1), (1, 0, w2), (1, 2, w3)], [0], [2]))
    loop = -math.log1p(-math.exp(w1 + w2))  # every number of turns round the cycle
    want_alpha = [loop, w1 + loop, w1 + w3 + loop]
    want_beta = [w1 + w3 + loop, w3 + loop, 0.0]
    assert np.allclose(r["alpha"], want_alpha, rtol=0, atol=1e-12)
    assert np.allclose(r["beta"], want_beta, rtol=0, atol=1e-12)
    assert abs(r["total"] - (w1 + w3 + loop)) < 1e-12


def _tiny_cyclic(seed):
    """A few states, each with up to three arcs of probability <= 0.02, so
    paths longer than L = 10 carry less than 0.061^11 / (1 - 0.061) of any
    sum (< 5e-14)."""
    rng = np.random.default_rng([41, seed])
    V = int(rng.integers(1, 5))
    arcs = []
    for s in range(V):
        for _ in range(int(rng.integers(0, 4))):
            arcs.append((s, int(rng.integers(0, V)), _w(math.log(0.02 * rng.random() + 1e-4))))
    starts = sorted(set(int(x) for x in rng.integers(0, V, size=2)))
    acc = [s for s in range(V) if rng.random() < 0.5] or [V - 1]
    return V, arcs, starts, acc


def _path_sums(V, arcs, starts, acc, L):
    """Every path of at most L arcs, enumerated: probability-domain sums
    from the starts to each state (forward) and from each state to the
    accepting states (backward), each path's probability a product of
    float64 arc probabilities, the sums exact (math.fsum)."""
    out = [[] for _ in range(V)]
    for s, d, w in arcs:
        out[s].append((d, math.exp(w)))
    fwd = [[] for _ in range(V)]
    bwd = [[] for _ in range(V)]

    def walk(first, v, p, k):
        if first in starts:
            fwd[v].append(p)
        if v in acc:
            bwd[first].append(p)
        if k < L:
            for d, q in out[v]:
                walk(first, d, p * q, k + 1)

    for v in range(V):
        walk(v, v, 1.0, 0)
    return (np.array([math.fsum(x) for x in fwd]), np.array([math.fsum(x) for x in bwd]))


@pytest.mark.parametrize("seed", range(24))
def test_explicit_path_enumeration(seed):
    V, arcs, starts, acc = _tiny_cyclic(seed)
    r = cyclic.score_cyclic(synth.from_arcs(V, [(s, d, 1, 1, w) for s, d, w in arcs],
                                            start=starts, accept=acc))
    fwd, bwd = _path_sums(V, arcs, starts, acc, 10)
    with np.errstate(divide="ignore"):
        la, lb = np.log(fwd), np.log(bwd)
    for got, want in ((r["alpha"], la), (r["beta"], lb)):
        assert np.array_equal(np.isneginf(got), np.isneginf(want)), (seed, got, want)
        fin = ~np.isneginf(want)
        assert np.allclose(got[fin], want[fin], rtol=0, atol=1e-12), (seed, got, want)
    tot = math.fsum(fwd[a] for a in acc)
    want_total = math.log(tot) if tot > 0 else -math.inf
    assert (r["total"] == want_total) or abs(r["total"] - want_total) < 1e-12


@pytest.mark.parametrize("seed", range(6))
def test_equals_the_acyclic_oracle_on_dags(seed):
    # arc probabilities below e^-0.7, so that the probability-domain solve
    # is well conditioned (with N(0, 1) weights the sums span e^+-40)
    G = dict(synth.random_dag(seed, 300, hubs=2, hub_degree=40))
    G["weight"] = (0.1 * np.asarray(G["weight"], np.float64) - 1.0).astype(np.float32)
    want = oracle.score(G)
    got = cyclic.score_cyclic(G)
    for k in ("alpha", "beta"):
        a, b = got[k], want[k]
        assert np.array_equal(np.isneginf(a), np.isneginf(b))
        fin = ~np.isneginf(b)
        assert np.allclose(a[fin], b[fin], rtol=1e-12, atol=1e-9), k
    assert abs(got["total"] - want["total"]) < 1e-9 * max(1.0, abs(want["total"]))


@pytest.mark.parametrize("arcs", [
    [(0, 0, 0.0)],                        # probability 1 round the loop
    [(0, 0, _w(math.log(2.0)))],          # more than 1
    [(0, 1, _w(0.5)), (1, 0, _w(-0.2))],  # a cycle of mass e^0.3 > 1
    [(0, 1, -1.0), (1, 1, _w(math.log(1.5))), (1, 2, -1.0)],  # behind an arc
])
def test_divergent_sums_are_refused(arcs):
    V = 1 + max(max(s, d) for s, d, _ in arcs)
    with pytest.raises(cyclic.DivergeError):
        cyclic.score_cyclic(_g(V, arcs, [0], [V - 1]))


def test_parts_no_path_crosses_do_not_count():
    # states 2-3 hold a divergent cycle that no start reaches and that
    # reaches no accepting state: every sum stays finite
    arcs = [(0, 1, -1.0), (2, 3, 0.5), (3, 2, 0.5), (1, 1, _w(-0.5))]
    r = cyclic.score_cyclic(_g(4, arcs, [0], [1]))
    assert np.isneginf(r["alpha"][2:]).all() and np.isneginf(r["beta"][2:]).all()
    loop = -math.log1p(-math.exp(_w(-0.5)))
    assert abs(r["alpha"][1] - (-1.0 + loop)) < 1e-12
    assert abs(r["total"] - (-1.0 + loop)) < 1e-12


def test_no_start_no_accept_and_empty():
    r = cyclic.score_cyclic(_g(2, [(0, 1, -1.0), (1, 0, -1.0)], [], [1]))
    assert np.isneginf(r["alpha"]).all() and r["total"] == -math.inf
    assert np.isfinite(r["beta"]).all()
    r = cyclic.score_cyclic(_g(2, [(0, 1, -1.0), (1, 0, -1.0)], [0], []))
    assert np.isneginf(r["beta"]).all() and r["total"] == -math.inf
    r = cyclic.score_cyclic(synth.from_arcs(0, [], start=[], accept=[]))
    assert len(r["alpha"]) == 0 and r["total"] == -math.inf


def test_generator_sums_converge():
    for seed in range(3):
        G = synth.random_cyclic(seed, 200, hubs=2, hub_degree=60)
        r = cyclic.score_cyclic(G)
        assert math.isfinite(r["total"])


def test_posterior_is_the_gradient_of_the_total():
    """d total / d w(e) = exp(alpha[src e] + w(e) + beta[dst e] - total), the
    expected number of uses of arc e (above 1 on a cycle), against central
    finite differences of the oracle's total in float64 weights."""
    # a random graph, and a cycle of mass 0.9 that paths go round 9 times on
    # average (0 -> 1 -> 0, exit 1 -> 2): arc 0 -> 1 is taken 10 times, the
    # back arc 9 times, the exit once
    cyc = _g(3, [(0, 1, _w(math.log(0.95))), (1, 0, _w(math.log(0.9 / 0.95))),
                 (1, 2, _w(-1.0))], [0], [2])
    for G, most in ((synth.random_cyclic(5, 12, degree=3, mass=0.7, p_accept=0.3), None),
                    (cyc, [10.0, 9.0, 1.0])):
        V, src, dst, w = cyclic._arcs(G)
        start = np.asarray(G["start"]) != 0
        accept = np.asarray(G["accept"]) != 0
        r = cyclic.scores_of(V, src, dst, w, start, accept)
        post = np.exp(r["alpha"][src] + w + r["beta"][dst] - r["total"])
        h = 1e-6
        for e in range(len(w)):
            wp, wm = w.copy(), w.copy()
            wp[e] += h
            wm[e] -= h
            fd = (cyclic.scores_of(V, src, dst, wp, start, accept)["total"]
                  - cyclic.scores_of(V, src, dst, wm, start, accept)["total"]) / (2 * h)
            assert abs(fd - post[e]) < 1e-6 * max(1.0, post[e]), (e, fd, post[e])
        if most is not None:
            assert np.allclose(post, most, rtol=1e-6, atol=0), post
