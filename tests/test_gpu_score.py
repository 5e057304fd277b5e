"""GPU scores, posteriors and provenance scatter versus the CPU oracle,
through the C ABI of libfstcompose.so.

Tolerances (float64 scores): both sides round once per log-add; the oracle
log-adds a state's terms one after another (an error of up to about one
unit in the last place of the running value per term), the GPU forms the
exact sum and rounds once, and errors add up along a path.  So a value
may differ by about (longest path + largest in-degree) units in the last
place of the largest magnitude: the tests allow 8 times that.  Posteriors
and scattered gradients are float32 results of float64 arithmetic: one
float32 rounding (2^-24 relative), plus the score error above passed
through exp, plus (scatter) the oracle's float64 summation error."""
import math

import numpy as np
import pytest

import oracle
from paper_2110_02848_amd import synth

import fsthelp

pytestmark = pytest.mark.gpu

ULP = 2.0 ** -52


@pytest.fixture(scope="module")
def comp():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2110_02848_amd import gpu
    c = gpu.Composer(0)
    yield c
    c.close()


def _dev(G):
    from paper_2110_02848_amd import gpu
    return gpu.to_device(G)


def gpu_score(comp, G, alpha=True, beta=True):
    import torch
    r = comp.score(_dev(G), alpha=alpha, beta=beta)
    torch.cuda.synchronize()
    return {k: (v.cpu().numpy() if v is not None else None) for k, v in r.items()}


def score_tol(G, ref):
    indeg = np.bincount(G["dst"], minlength=G["num_states"]).max() if len(G["dst"]) else 0
    vals = np.concatenate([ref["alpha"], ref["beta"], [ref["total"]]])
    fin = vals[np.isfinite(vals)]
    big = float(np.abs(fin).max()) if len(fin) else 0.0
    return 8.0 * (ref["longest"] + indeg + 2) * ULP * (1.0 + big)


def assert_scores_close(got, ref, tol, what):
    ref = np.asarray(ref, np.float64)
    got = np.asarray(got, np.float64)
    inf_ref, inf_got = np.isinf(ref), np.isinf(got)
    assert np.array_equal(inf_ref, inf_got), (what, np.flatnonzero(inf_ref != inf_got)[:5])
    assert np.array_equal(ref[inf_ref], got[inf_got]), what
    d = np.abs(got[~inf_ref] - ref[~inf_ref])
    assert not np.isnan(d).any(), what
    if len(d):
        i = int(np.argmax(d))
        assert d[i] <= tol, (what, i, float(got[~inf_ref][i]), float(ref[~inf_ref][i]), tol)


def check_scores(comp, G, tag):
    print(f"[score] {tag}", flush=True)
    got = gpu_score(comp, G)
    ref = oracle.score(G)
    tol = score_tol(G, ref)
    assert_scores_close(got["alpha"], ref["alpha"], tol, tag + " alpha")
    assert_scores_close(got["beta"], ref["beta"], tol, tag + " beta")
    assert_scores_close(got["total"], [ref["total"]], tol, tag + " total")
    return got, ref


# --------------------------------------------------------------------------
# scores
# --------------------------------------------------------------------------

DAGS = [
    ("small", dict(V=50, mean_out=1.5, window=4)),
    ("wide", dict(V=3000, mean_out=3.0, window=64, p_global=0.3)),
    ("deep", dict(V=20000, mean_out=1.1, window=2, p_global=0.01)),
    ("hubs", dict(V=6000, mean_out=1.5, window=8, hubs=4, hub_degree=3000)),
    ("dense", dict(V=2000, mean_out=12.0, window=200)),
    ("sparse", dict(V=10000, mean_out=0.7, window=3)),
]


@pytest.mark.parametrize("name,kw", DAGS, ids=[d[0] for d in DAGS])
@pytest.mark.parametrize("seed", range(3))
def test_score_random_dags(comp, name, kw, seed):
    check_scores(comp, synth.random_dag(seed, **kw), f"dag {name} seed {seed}")


def _layered_heavy(seed, width, fan):
    """Start state 0 -> `width` states with `fan` out-arcs each -> `width`
    merges with `fan` in-arcs each -> one accepting state.  Each middle
    layer is `width` heavy states listed in one generation, in either
    direction."""
    rng = np.random.default_rng(seed)
    L1 = [1 + i for i in range(width)]
    L2 = [1 + width + i for i in range(width)]
    F = 1 + 2 * width
    ends = rng.permutation(np.repeat(L2, fan))
    arcs = [(0, a, 1, 1, float(rng.standard_normal())) for a in L1]
    arcs += [(a, int(ends[k * fan + j]), 1, 1, float(rng.standard_normal()))
             for k, a in enumerate(L1) for j in range(fan)]
    arcs += [(b, F, 1, 1, float(rng.standard_normal())) for b in L2]
    return synth.from_arcs(F + 1, arcs, start=[0], accept=[F])


@pytest.mark.parametrize("width", [65, 300])
def test_score_many_heavy_states_in_one_generation(comp, width):
    # more heavy states than one wavefront's lanes in a generation's list
    check_scores(comp, _layered_heavy(width, width, 70), f"{width} heavy states per generation")


@pytest.mark.parametrize("seed", range(40))
def test_score_tiny_dags(comp, seed):
    rng = np.random.default_rng(seed)
    G = synth.random_dag(100 + seed, int(rng.integers(1, 30)), mean_out=float(rng.uniform(0, 3)),
                         window=int(rng.integers(1, 6)), n_start=int(rng.integers(1, 4)),
                         p_accept=0.3)
    check_scores(comp, G, f"tiny dag seed {seed}")


def test_score_special_graphs(comp):
    cases = {
        "empty": synth.empty_graph(),
        "one": synth.from_arcs(1, [], start=[0], accept=[0]),
        "no accept": synth.from_arcs(3, [(0, 1, 1, 1, -1.0), (1, 2, 1, 1, -2.0)],
                                     start=[0], accept=[]),
        "no start": synth.from_arcs(3, [(0, 1, 1, 1, -1.0)], start=[], accept=[1]),
        "unreached": synth.from_arcs(4, [(0, 1, 1, 1, 0.5), (2, 1, 1, 1, 0.25),
                                         (0, 3, 1, 1, 1.0)], start=[0], accept=[1]),
        "parallel": synth.from_arcs(2, [(0, 1, 1, 1, math.log(0.25)),
                                        (0, 1, 2, 2, math.log(0.75))], start=[0], accept=[1]),
        "start accepts mid": synth.from_arcs(3, [(0, 1, 1, 1, -0.5), (1, 2, 1, 1, -0.5)],
                                             start=[0, 1], accept=[1, 2]),
    }
    for tag, G in cases.items():
        check_scores(comp, G, tag)


def test_score_fan_in_and_out_over_many_workgroups(comp):
    # one state with 5000 in-arcs and 3000 out-arcs (heavy both ways), fed
    # and drained by chains longer than a thread's walk budget
    arcs = []
    V = 1 + 5000 + 1 + 3000 + 200
    hub = 5001
    for i in range(5000):
        arcs.append((0, 1 + i, 1, 1, float(np.float32(-0.001 * i))))
        arcs.append((1 + i, hub, 1, 1, float(np.float32(0.5 - 0.0002 * i))))
    for j in range(3000):
        arcs.append((hub, hub + 1 + j, 1, 1, float(np.float32(0.25 * math.sin(j)))))
        arcs.append((hub + 1 + j, hub + 3001, 1, 1, 0.0))
    for k in range(199):
        arcs.append((hub + 3001 + k, hub + 3002 + k, 1, 1, -0.01))
    G = synth.from_arcs(V, arcs, start=[0], accept=[V - 1, hub])
    check_scores(comp, G, "fan in/out")


def test_score_long_chain_and_walk_budget(comp):
    from paper_2110_02848_amd import gpu
    V = 5000
    arcs = [(i, i + 1, 1, 1, float(np.float32(-0.001 * (i % 7)))) for i in range(V - 1)]
    G = synth.from_arcs(V, arcs, start=[0, 2500], accept=[V - 1, 100])
    for depth in (64, 1, 0):
        comp.set_option(gpu.FST_OPT_CHAIN_DEPTH, depth)
        try:
            check_scores(comp, G, f"chain depth {depth}")
        finally:
            comp.set_option(gpu.FST_OPT_CHAIN_DEPTH, 64)


def test_score_one_direction(comp):
    G = synth.random_dag(5, 3000, mean_out=2.0, window=20)
    ref = oracle.score(G)
    tol = score_tol(G, ref)
    a = gpu_score(comp, G, alpha=True, beta=False)
    assert a["beta"] is None
    assert_scores_close(a["alpha"], ref["alpha"], tol, "alpha only")
    assert_scores_close(a["total"], [ref["total"]], tol, "alpha-only total")
    b = gpu_score(comp, G, alpha=False, beta=True)
    assert b["alpha"] is None
    assert_scores_close(b["beta"], ref["beta"], tol, "beta only")
    assert_scores_close(b["total"], [ref["total_bwd"]], tol, "beta-only total")
    t = gpu_score(comp, G, alpha=False, beta=False)
    assert_scores_close(t["total"], [ref["total"]], tol, "total only")


def test_score_is_bitwise_reproducible(comp):
    G = synth.random_dag(11, 8000, mean_out=2.5, window=32, hubs=2, hub_degree=1500)
    r1 = gpu_score(comp, G)
    r2 = gpu_score(comp, G)
    for k in ("alpha", "beta", "total"):
        assert np.array_equal(r1[k].view(np.uint64), r2[k].view(np.uint64)), k


def test_score_refuses_cycles(comp):
    from paper_2110_02848_amd import gpu
    cyc = synth.from_arcs(4, [(0, 1, 1, 1, 0.0), (2, 3, 1, 1, 0.0), (3, 2, 1, 1, 0.0)],
                          start=[0], accept=[1])
    loop = synth.from_arcs(1, [(0, 0, 1, 1, -1.0)], start=[0], accept=[0])
    for G in (cyc, loop):
        with pytest.raises(gpu.FstError) as e:
            gpu_score(comp, G)
        assert e.value.code == gpu.FST_ERR_CYCLIC
    # the context still works afterwards
    check_scores(comp, synth.random_dag(1, 100), "after cycle")


def test_score_rejects_invalid_graph(comp):
    from paper_2110_02848_amd import gpu
    G = synth.random_dag(2, 50)
    G = dict(G)
    G["dst"] = G["dst"].copy()
    G["dst"][3] = 50  # out of range
    with pytest.raises(gpu.FstError) as e:
        gpu_score(comp, G)
    assert e.value.code == gpu.FST_ERR_INVALID_GRAPH


# --------------------------------------------------------------------------
# scores of composed graphs
# --------------------------------------------------------------------------

def _compose(comp, A, B):
    import torch
    from paper_2110_02848_amd import gpu
    C = comp.compose(gpu.to_device(A), gpu.to_device(B))
    torch.cuda.synchronize()
    return C


@pytest.mark.parametrize("seed", range(3))
def test_score_of_composed_lexicon_T100(comp, seed):
    import torch
    from paper_2110_02848_amd import gpu
    A, B, meta = synth.emissions_lexicon("lexicon-T100-W1000", seed)
    Cd = _compose(comp, A, B)
    C = oracle.compose(A, B)  # the GPU's C equals it (composition parity tests)
    assert (C["num_states"], C["num_arcs"]) == (Cd["num_states"], Cd["num_arcs"])
    ref = oracle.score(C)
    tol = score_tol(C, ref)
    got = comp.score(Cd)
    torch.cuda.synchronize()
    assert_scores_close(got["alpha"].cpu().numpy(), ref["alpha"], tol, "alpha")
    assert_scores_close(got["beta"].cpu().numpy(), ref["beta"], tol, "beta")
    closed = fsthelp.lexicon_total_score(meta["table"], meta["spellings"])
    assert abs(float(got["total"].item()) - closed) <= max(tol, 1e-9 * (1 + abs(closed)))


@pytest.mark.parametrize("depth", [3, 1])
def test_score_of_composed_lexicon_short_walks(comp, depth):
    # walks from the heavy root states stop at the depth budget inside the
    # words, so the single-dependency states they stop at are settled (and
    # listed) together with the workgroup's merge arrivals
    import torch
    from paper_2110_02848_amd import gpu
    spec = synth.LexSpec(T=30, C=8, W=400, len_lo=2, len_hi=6)
    A, B, _ = synth.emissions_lexicon("lexicon-T100-W1000", 3, spec=spec)
    Cd = _compose(comp, A, B)
    C = oracle.compose(A, B)
    ref = oracle.score(C)
    tol = score_tol(C, ref)
    comp.set_option(gpu.FST_OPT_CHAIN_DEPTH, depth)
    try:
        got = comp.score(Cd)
        torch.cuda.synchronize()
    finally:
        comp.set_option(gpu.FST_OPT_CHAIN_DEPTH, 64)
    assert_scores_close(got["alpha"].cpu().numpy(), ref["alpha"], tol, f"alpha depth {depth}")
    assert_scores_close(got["beta"].cpu().numpy(), ref["beta"], tol, f"beta depth {depth}")
    assert_scores_close([float(got["total"].item())], [ref["total"]], tol, f"total depth {depth}")


def check_posterior(comp, Cd, C, ref, tag):
    import torch
    print(f"[posterior] {tag}", flush=True)
    sc = comp.score(Cd)
    post = comp.posterior(Cd, sc["alpha"], sc["beta"], sc["total"], scale=1.0)
    torch.cuda.synchronize()
    got = post.cpu().numpy().astype(np.float64)
    want = oracle.posterior(C, ref["alpha"], ref["beta"], ref["total"])
    tol = score_tol(C, ref)
    rel = 2.0 ** -23 + 4 * tol
    err = np.abs(got - want)
    bad = err > rel * np.abs(want) + 1e-37
    assert not bad.any(), (tag, np.flatnonzero(bad)[:5], got[bad][:5], want[bad][:5])
    return sc, post, want


@pytest.mark.parametrize("seed", range(3))
def test_posterior_random_dags(comp, seed):
    G = synth.random_dag(20 + seed, 4000, mean_out=2.0, window=24, hubs=1, hub_degree=500)
    ref = oracle.score(G)
    check_posterior(comp, _dev(G), G, ref, f"dag seed {seed}")


def test_posterior_without_accepting_path(comp):
    import torch
    G = synth.from_arcs(3, [(0, 1, 1, 1, -1.0), (1, 2, 1, 1, -2.0)], start=[0], accept=[])
    Gd = _dev(G)
    sc = comp.score(Gd)
    post = comp.posterior(Gd, sc["alpha"], sc["beta"], sc["total"])
    torch.cuda.synchronize()
    assert float(sc["total"].item()) == -math.inf
    assert np.all(post.cpu().numpy() == 0)


def check_scatter(comp, g, idx, m, tag):
    import torch
    print(f"[scatter] {tag}", flush=True)
    gd = torch.from_numpy(np.ascontiguousarray(g, np.float32)).cuda()
    idd = torch.from_numpy(np.ascontiguousarray(idx, np.int32)).cuda()
    out = comp.grad_scatter(gd, idd, m)
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    want = oracle.scatter(np.asarray(g, np.float32).astype(np.float64), idx, m)
    n = len(g)
    M = float(np.abs(np.asarray(g, np.float32)).max(initial=0.0))
    per = np.bincount(idx[idx >= 0], minlength=m) if m else np.zeros(0)
    atol = per * M * 2.0 ** -50 + 1e-38
    err = np.abs(got - want)
    bad = err > 2.0 ** -23 * np.abs(want) + atol
    assert not bad.any(), (tag, np.flatnonzero(bad)[:5], got[bad][:5], want[bad][:5])
    return got


@pytest.mark.parametrize("seed", range(6))
def test_scatter_random(comp, seed):
    rng = np.random.default_rng(seed)
    m = int(rng.integers(1, 3000))
    n = int(rng.integers(0, 200000))
    idx = rng.integers(-1, m, size=n).astype(np.int32)
    scale = [1.0, 1e-30, 1e30, 3.0, 1e-3, 1.0][seed]
    g = (scale * rng.standard_normal(n)).astype(np.float32)
    check_scatter(comp, g, idx, m, f"random seed {seed}")


@pytest.mark.parametrize("m,pattern", [(5000, "random"), (100000, "random"),
                                       (100000, "runs"), (1 << 21, "random"),
                                       ((1 << 21) + 1, "random")])
def test_scatter_wide_targets(comp, m, pattern):
    """Targets spread wider than one chunk's LDS table: the terms are grouped
    by target range first (up to 2^21 targets), else added with global
    atomics; both give the oracle's sums."""
    rng = np.random.default_rng(m + len(pattern))
    n = 300000
    if pattern == "random":
        idx = rng.integers(-1, m, size=n).astype(np.int32)
    else:
        # ascending runs over the whole range, like the provenance of the
        # arcs of one frame after another
        idx = (np.arange(n) * 7 % m).astype(np.int32)
        idx[rng.random(n) < 0.05] = -1
    g = rng.standard_normal(n).astype(np.float32)
    check_scatter(comp, g, idx, m, f"wide targets m={m} {pattern}")


def test_scatter_wide_targets_bad_index(comp):
    import torch
    from paper_2110_02848_amd import gpu
    n, m = 100000, 10000
    idx = np.random.default_rng(5).integers(0, m, size=n).astype(np.int32)
    idx[77777] = m
    with pytest.raises(gpu.FstError) as e:
        comp.grad_scatter(torch.ones(n, device="cuda"), torch.from_numpy(idx).cuda(), m)
    assert e.value.code == gpu.FST_ERR_INVALID_ARG
    # the context still works
    check_scatter(comp, np.ones(n, np.float32), np.minimum(idx, m - 1), m, "after a bad index")


def test_scatter_edge_cases(comp):
    from paper_2110_02848_amd import gpu
    check_scatter(comp, np.zeros(0, np.float32), np.zeros(0, np.int32), 5, "empty input")
    check_scatter(comp, np.zeros(10, np.float32), np.arange(10, dtype=np.int32) % 3, 3, "zeros")
    check_scatter(comp, np.ones(5, np.float32), np.full(5, -1, np.int32), 4, "all skipped")
    # cancellation: +x and -x into one target sum to exactly 0
    g = np.array([1.5, -1.5, 2.0 ** -20, -(2.0 ** -20)], np.float32)
    got = check_scatter(comp, g, np.array([0, 0, 1, 1], np.int32), 2, "cancel")
    assert got.tolist() == [0.0, 0.0]
    # one hot target with many terms (lanes grouped in a wavefront)
    n = 100000
    g = np.full(n, 0.1, np.float32)
    check_scatter(comp, g, np.zeros(n, np.int32), 1, "hot target")
    import torch
    with pytest.raises(gpu.FstError) as e:
        comp.grad_scatter(torch.ones(3, device="cuda"),
                          torch.tensor([0, 7, 1], dtype=torch.int32, device="cuda"), 3)
    assert e.value.code == gpu.FST_ERR_INVALID_ARG


def test_operand_gradients_of_lexicon_T100(comp):
    """Gradient of the total score of C = A o B by every arc weight of A and
    B: posterior on the GPU, scattered through the GPU's provenance, against
    the oracle's posterior of its own C scattered through its provenance;
    the emission gradients of each frame add up to one."""
    import torch
    from paper_2110_02848_amd import gpu
    A, B, meta = synth.emissions_lexicon("lexicon-T100-W1000", 2)
    Cd = _compose(comp, A, B)
    gA, gB = comp.operand_grads(Cd, len(A["src"]), len(B["src"]))
    torch.cuda.synchronize()
    C = oracle.compose(A, B)
    ref = oracle.score(C)
    post = oracle.posterior(C, ref["alpha"], ref["beta"], ref["total"])
    wA = oracle.scatter(post, C["arc_a"], len(A["src"]))
    wB = oracle.scatter(post, C["arc_b"], len(B["src"]))
    tol = score_tol(C, ref)
    for got, want, tag in ((gA.cpu().numpy(), wA, "A"), (gB.cpu().numpy(), wB, "B")):
        got = got.astype(np.float64)
        bad = np.abs(got - want) > (2.0 ** -22 + 4 * tol) * np.abs(want) + 1e-30
        assert not bad.any(), (tag, np.flatnonzero(bad)[:5], got[bad][:5], want[bad][:5])
    T, Cn = meta["table"].shape
    sums = gA.cpu().numpy().astype(np.float64).reshape(T, Cn).sum(axis=1)
    assert np.allclose(sums, 1.0, atol=1e-5)


def test_score_and_gradients_full_lexicon(comp):
    """The benchmark workload at full size (36.7M states, 41.6M arcs), by
    properties that hold at any size: the total equals the frame recursion
    over word segmentations (which never builds C); the emission gradients
    of every frame sum to one (each accepting path takes one arc of A per
    frame); the entry, token and exit arcs of a word have equal gradients
    (they are always used together); no state's posterior exceeds one."""
    import torch
    A, B, meta = synth.emissions_lexicon("lexicon-T500-W10000", 0)
    Cd = _compose(comp, A, B)
    print("[score] full lexicon composed", flush=True)
    sc = comp.score(Cd)
    post = comp.posterior(Cd, sc["alpha"], sc["beta"], sc["total"])
    gA = comp.grad_scatter(post, Cd["arc_a"], len(A["src"]))
    gB = comp.grad_scatter(post, Cd["arc_b"], len(B["src"]))
    torch.cuda.synchronize()
    total = float(sc["total"].item())
    closed = fsthelp.lexicon_total_score(meta["table"], meta["spellings"])
    # 833 states on the longest path, 10^4 in-arcs at a root, |values| < 2000
    assert abs(total - closed) <= 1e-8 * (1 + abs(closed)), (total, closed)
    T, Cn = meta["table"].shape
    sums = gA.cpu().numpy().astype(np.float64).reshape(T, Cn).sum(axis=1)
    assert np.allclose(sums, 1.0, atol=1e-5), np.abs(sums - 1).max()
    gb = gB.cpu().numpy().astype(np.float64)
    off, dst = B["arc_offset"], B["dst"]
    for e0 in range(off[0], off[1]):
        chain, st = [e0], int(dst[e0])
        while st != 0:
            chain.append(int(off[st]))
            st = int(dst[off[st]])
        assert np.allclose(gb[chain], gb[e0], rtol=1e-6, atol=1e-30), e0
    state_post = (sc["alpha"] + sc["beta"] - sc["total"]).exp()
    assert float(state_post.max().item()) <= 1.0 + 1e-9
