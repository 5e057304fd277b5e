"""Scores of graphs with cycles on the GPU (fst_score_cyclic through the C
ABI) against the CPU oracle (``oracle.cyclic``: the probability-domain
Neumann series by a float64 solve), and against fst_score bit for bit on
graphs without cycles.

Tolerance: the test graphs keep every state's arc probabilities to a sum of
at most 1/2, so the solve's relative error is a few times cond(I - M) x V x
2^-53 (cond at most a few hundred here) and the sweeps stop within a few
units in the last place of their fixed point; 1e-9 (log domain, absolute,
scaled by 1 + |value|) covers both with a margin of 10^2 or more, while a
dropped arc, cycle or empty path moves a value by far more."""
import math

import numpy as np
import pytest

import oracle
from oracle import cyclic
from paper_2110_02848_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def comp():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2110_02848_amd import gpu
    c = gpu.Composer(0)
    yield c
    c.close()


def _run(comp, G, alpha=True, beta=True, **kw):
    import torch
    from paper_2110_02848_amd import gpu
    r = comp.score_cyclic(gpu.to_device(G), alpha=alpha, beta=beta, **kw)
    torch.cuda.synchronize()
    out = {k: (v.cpu().numpy() if hasattr(v, "cpu") else v) for k, v in r.items()}
    out["total"] = float(out["total"][0])
    return out


def _close(got, want, what):
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    assert np.array_equal(np.isneginf(got), np.isneginf(want)), what
    fin = np.isfinite(want)
    err = np.abs(got[fin] - want[fin]) / (1.0 + np.abs(want[fin]))
    assert err.size == 0 or err.max() < 1e-9, (what, float(err.max()))


def _check(comp, G, tag):
    print(f"[cyclic] {tag}", flush=True)
    want = cyclic.score_cyclic(G)
    got = _run(comp, G)
    _close(got["alpha"], want["alpha"], (tag, "alpha"))
    _close(got["beta"], want["beta"], (tag, "beta"))
    _close([got["total"]], [want["total"]], (tag, "total"))
    assert got["sweeps"] > 0
    return got


@pytest.mark.parametrize("seed", range(6))
def test_random_cyclic_graphs(comp, seed):
    V = [40, 300, 1500][seed % 3]
    G = synth.random_cyclic(seed, V, degree=2 + seed % 3, mass=0.5, hubs=seed % 3,
                            hub_degree=50)
    _check(comp, G, f"random cyclic V={V} seed {seed}")


def test_self_loop_and_two_cycle(comp):
    w = float(np.float32(-0.7))
    got = _check(comp, synth.from_arcs(1, [(0, 0, 1, 1, w)], start=[0], accept=[0]),
                 "self-loop")
    assert abs(got["total"] + math.log1p(-math.exp(w))) < 1e-12
    w1, w2, w3 = (float(np.float32(x)) for x in (-0.4, -1.1, 0.3))
    G = synth.from_arcs(3, [(0, 1, 1, 1, w1), (1, 0, 1, 1, w2), (1, 2, 1, 1, w3)], start=[0],
                        accept=[2])
    got = _check(comp, G, "two-state cycle")
    assert abs(got["total"] - (w1 + w3 - math.log1p(-math.exp(w1 + w2)))) < 1e-12


def test_composed_cyclic_c(comp):
    """C of two random transducers (random-64: cyclic), its arcs given
    probabilities that add to 1/2 per state."""
    import torch
    from paper_2110_02848_amd import gpu
    A, B = synth.workload("random-64", 0)
    C = gpu.to_numpy(comp.compose(gpu.to_device(A), gpu.to_device(B), provenance=False,
                                  keys=False))
    torch.cuda.synchronize()
    V = int(C["num_states"])
    off = np.asarray(C["arc_offset"], np.int64)
    rng = np.random.default_rng(5)
    w = np.empty(len(C["dst"]))
    for v in range(V):
        lo, hi = off[v], off[v + 1]
        if hi > lo:
            z = np.exp(rng.standard_normal(hi - lo))
            w[lo:hi] = np.log(0.5 * z / z.sum())
    G = dict(num_states=V, arc_offset=C["arc_offset"], src=C["src"], dst=C["dst"],
             ilabel=C["ilabel"], olabel=C["olabel"], weight=w.astype(np.float32),
             start=C["start"], accept=C["accept"])
    with pytest.raises(oracle.CycleError):
        oracle.score(G)  # it does have cycles
    _check(comp, G, f"composed random-64, V_C={V}")


@pytest.mark.parametrize("seed", range(3))
def test_equals_fst_score_bitwise_on_dags(comp, seed):
    import torch
    from paper_2110_02848_amd import gpu
    G = synth.random_dag(seed, 3000, hubs=3, hub_degree=300)
    dG = gpu.to_device(G)
    ref = comp.score(dG)
    got = comp.score_cyclic(dG)
    torch.cuda.synchronize()
    for k in ("alpha", "beta", "total"):
        assert torch.equal(got[k], ref[k]), k
    longest = oracle.score(G)["longest"]  # states on the longest path
    assert got["sweeps"] <= longest + 1, (got["sweeps"], longest)


def test_one_direction_and_tolerance(comp):
    G = synth.random_cyclic(7, 400, degree=3, mass=0.5)
    full = _run(comp, G)
    a = _run(comp, G, beta=False)
    b = _run(comp, G, alpha=False)
    assert a["beta"] is None and b["alpha"] is None
    assert np.array_equal(a["alpha"], full["alpha"]) and a["total"] == full["total"]
    assert np.array_equal(b["beta"], full["beta"])
    # with beta alone the total is the log-add of beta over the start states
    assert abs(b["total"] - full["total"]) < 1e-12 * (1 + abs(full["total"]))
    loose = _run(comp, G, tol=1e-6)
    assert loose["sweeps"] < full["sweeps"]
    fin = np.isfinite(full["alpha"])
    assert np.all(loose["alpha"][fin] <= full["alpha"][fin] + 1e-15)
    assert np.all(full["alpha"][fin] - loose["alpha"][fin] < 1e-5)


def test_divergence_and_arguments(comp):
    from paper_2110_02848_amd import gpu
    G = synth.from_arcs(2, [(0, 1, 1, 1, 0.5), (1, 0, 1, 1, -0.2)], start=[0], accept=[1])
    with pytest.raises(gpu.FstError) as e:
        _run(comp, G, max_sweeps=300)
    assert e.value.code == gpu.FST_ERR_NOT_CONVERGED
    with pytest.raises(gpu.FstError) as e:
        _run(comp, G, max_sweeps=0)
    assert e.value.code == gpu.FST_ERR_NOT_CONVERGED
    for kw in (dict(max_sweeps=-1), dict(tol=-1.0)):
        with pytest.raises(gpu.FstError) as e:
            _run(comp, G, **kw)
        assert e.value.code == gpu.FST_ERR_INVALID_ARG
    # the context stays usable
    _check(comp, synth.random_cyclic(3, 60), "after errors")


def test_empty_and_unreachable(comp):
    from paper_2110_02848_amd import gpu
    r = _run(comp, synth.from_arcs(0, [], start=[], accept=[]))
    assert r["total"] == -math.inf
    # a divergent cycle that no path from a start to an accepting state uses
    arcs = [(0, 1, 1, 1, -1.0), (2, 3, 1, 1, 0.5), (3, 2, 1, 1, 0.5), (1, 1, 1, 1, -0.5)]
    G = synth.from_arcs(4, arcs, start=[0], accept=[1])
    _check(comp, G, "unreachable divergent part")
    # once a start reaches it, its forward sums diverge and never settle
    with pytest.raises(gpu.FstError) as e:
        _run(comp, dict(G, start=np.array([1, 0, 1, 0], np.uint8)), max_sweeps=200)
    assert e.value.code == gpu.FST_ERR_NOT_CONVERGED


def test_posteriors_of_a_cyclic_graph(comp):
    """fst_score_posterior with fst_score_cyclic's scores: each arc's
    expected number of uses (above 1 on cycles), the total's gradient
    (pinned by finite differences on the CPU), against the oracle's scores
    (float32 results of float64 arithmetic: 1e-6 relative covers the float32
    rounding and the scores' error passed through exp)."""
    import torch
    from paper_2110_02848_amd import gpu
    G = synth.random_cyclic(9, 500, degree=3, mass=0.6, hubs=2, hub_degree=40)
    dG = gpu.to_device(G)
    r = comp.score_cyclic(dG)
    grad = comp.posterior(dG, r["alpha"], r["beta"], r["total"])
    torch.cuda.synchronize()
    grad = grad.cpu().numpy().astype(np.float64)
    ref = cyclic.score_cyclic(G)
    V, src, dst, w = cyclic._arcs(G)
    want = np.exp(ref["alpha"][src] + w + ref["beta"][dst] - ref["total"])
    assert np.allclose(grad, want, rtol=1e-6, atol=0.0)
    assert want.max() > 0.0


def test_equals_fst_score_bitwise_on_composed_lexicon(comp):
    """C = emissions(T=100) o lexicon(W=1000): 0.59 M states, roots with
    about 10^3 in-arcs (pull lists longer than the register path); the
    sweeps reach fst_score's values bit for bit, with validation off and
    timing on (as a training loop scoring its own output would run)."""
    import torch
    from paper_2110_02848_amd import gpu
    A, B = synth.workload("lexicon-T100-W1000", 0)
    C = comp.compose(gpu.to_device(A), gpu.to_device(B), provenance=False, keys=False)
    torch.cuda.synchronize()
    comp.set_option(gpu.FST_OPT_VALIDATE, 0)
    comp.set_option(gpu.FST_OPT_TIMING, 1)
    try:
        ref = comp.score(C)
        got = comp.score_cyclic(C)
        torch.cuda.synchronize()
        times = comp.score_kernel_times()
    finally:
        comp.set_option(gpu.FST_OPT_VALIDATE, 1)
        comp.set_option(gpu.FST_OPT_TIMING, 0)
    for k in ("alpha", "beta", "total"):
        assert torch.equal(got[k], ref[k]), k
    assert times["score_gen"][1] >= got["sweeps"] > 100
