"""GPU path versus the CPU oracle, element by element and bit-exact
(structure, labels, binary32 weight bits, flags, keys, provenance), through
the C ABI of libfstcompose.so."""
import numpy as np
import pytest

import oracle
from paper_2110_02848_amd import synth

import fsthelp

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def comp():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2110_02848_amd import gpu
    c = gpu.Composer(0)
    c.set_option(gpu.FST_OPT_COUNT_MOVES, 1)  # statistics compared with the oracle's
    yield c
    c.close()


def gpu_compose(comp, A, B):
    import torch
    from paper_2110_02848_amd import gpu
    C = comp.compose(gpu.to_device(A), gpu.to_device(B))
    torch.cuda.synchronize()
    return gpu.to_numpy(C)


def check_stats(comp, A, B, ref, tag):
    """The GPU run's search statistics against the oracle's (ref: forward
    order): accessible keys, trim keys, and, when the context counts them,
    the moves out of the accessible keys.  Under the co-accessible-first
    order the forward search places only co-accessible keys, so it counts
    the trim set and the moves out of it, as the oracle's paper order does."""
    from paper_2110_02848_amd import gpu
    st = comp.stats()
    V = int(ref["num_states"])
    exp_acc, exp_gen = ref["stats"]["accessible"], ref["stats"]["generated"]
    if comp.options.get(gpu.FST_OPT_ORDER) == gpu.FST_ORDER_COACCESSIBLE_FIRST:
        exp_acc = V
        if comp.options.get(gpu.FST_OPT_COUNT_MOVES):
            exp_gen = oracle.compose_raw(A, B, oracle.ORDER_PAPER)["stats"]["generated"]
    assert st["num_states"] == V and st["coaccessible"] == V, (tag, st, V)
    assert st["num_arcs"] == int(ref["num_arcs"]), (tag, st)
    assert st["accessible"] == exp_acc, (tag, st["accessible"], exp_acc)
    if comp.options.get(gpu.FST_OPT_COUNT_MOVES):
        assert st["generated"] == exp_gen, (tag, st, exp_gen)


def check_pair(comp, A, B, tag, order=oracle.ORDER_FORWARD, ref=None):
    print(f"[parity] {tag}", flush=True)
    got = gpu_compose(comp, A, B)
    if ref is None:
        ref = oracle.compose(A, B, order)
        if order != oracle.ORDER_FORWARD:
            ref["stats"] = oracle.compose_raw(A, B, oracle.ORDER_FORWARD)["stats"]
    errs = fsthelp.compare_results(got, ref)
    assert not errs, (tag, errs[:5])
    check_stats(comp, A, B, ref, tag)
    return got, ref


_REF_CACHE = {}


def cached_ref(name, seed, A, B):
    """The oracle's forward-order result of a named workload, computed once
    per test session (several orders and option sets compare with it)."""
    k = (name, seed)
    if k not in _REF_CACHE:
        _REF_CACHE[k] = oracle.compose(A, B, oracle.ORDER_FORWARD)
    return _REF_CACHE[k]


def supercritical_5000(seed):
    """V = 5000 pair of the random-5000 recipe with 16 symbols instead of 64:
    a composite key then has about 1.3 moves (supercritical), so the search,
    count and fill do real work at that size (seed 0: 3.0 M states, 3.8 M
    arcs)."""
    ss = np.random.SeedSequence([31, 16, int(seed)])
    ra, rb = [np.random.default_rng(s) for s in ss.spawn(2)]
    A = synth.random_fst(ra, 5000, 4, 16, 0.05, 0.05)
    B = synth.random_fst(rb, 5000, 4, 16, 0.05, 0.05)
    return A, B


def named_pair(name, seed):
    if name == "random-5000-k16":
        return supercritical_5000(seed)
    return synth.workload(name, seed)


# random-5000 seeds in 0..2999 whose composition is not empty (found by a
# scan with the oracle: the recipe is subcritical, C is empty for ~99 % of
# seeds); the largest has 6 states
NONEMPTY_5000 = (15, 471, 1175, 1183, 1216, 1348, 2216, 2235, 2295, 2404, 2446, 2646, 2647,
                 2666)


@pytest.mark.parametrize("seed", range(100))
def test_random_64(comp, seed):
    A, B = synth.workload("random-64", seed)
    got, _ = check_pair(comp, A, B, f"random-64 seed {seed}")
    if seed < 10:
        assert not fsthelp.check_invariants(A, B, got)


@pytest.mark.parametrize("seed", range(12))
def test_random_1000(comp, seed):
    A, B = synth.workload("random-1000", seed)
    got, _ = check_pair(comp, A, B, f"random-1000 seed {seed}",
                        ref=cached_ref("random-1000", seed, A, B))
    if seed > 0:  # seed 0 composes to nothing; seeds 1..11 to ~850 K states
        assert got["num_states"] > 800000


@pytest.mark.parametrize("seed", list(range(10)) + list(NONEMPTY_5000))
def test_random_5000(comp, seed):
    A, B = synth.workload("random-5000", seed)
    got, _ = check_pair(comp, A, B, f"random-5000 seed {seed}",
                        ref=cached_ref("random-5000", seed, A, B))
    assert (got["num_states"] > 0) == (seed in NONEMPTY_5000)


@pytest.mark.parametrize("seed", range(2))
def test_random_5000_supercritical(comp, seed):
    A, B = supercritical_5000(seed)
    got, _ = check_pair(comp, A, B, f"random-5000-k16 seed {seed}",
                        ref=cached_ref("random-5000-k16", seed, A, B))
    if seed == 0:
        assert got["num_states"] > 3000000 and got["num_arcs"] > 3500000
        assert not fsthelp.check_invariants(A, B, got)


@pytest.mark.parametrize("seed", range(10))
def test_lexicon_T100_W1000(comp, seed):
    A, B, meta = synth.emissions_lexicon("lexicon-T100-W1000", seed)
    got, _ = check_pair(comp, A, B, f"lexicon-T100-W1000 seed {seed}",
                        ref=cached_ref("lexicon-T100-W1000", seed, A, B))
    V, E = fsthelp.lexicon_closed_form(meta["spec"].T, meta["spellings"])
    assert (got["num_states"], got["num_arcs"]) == (V, E)


@pytest.mark.timeout(900)
def test_lexicon_T500_W10000_full(comp):
    """Full-size emissions(T=500, C=64) o lexicon(W=10000): every element."""
    A, B, meta = synth.emissions_lexicon("lexicon-T500-W10000", 0)
    got, _ = check_pair(comp, A, B, "lexicon-T500-W10000 seed 0")
    V, E = fsthelp.lexicon_closed_form(meta["spec"].T, meta["spellings"])
    assert (got["num_states"], got["num_arcs"]) == (V, E)


@pytest.mark.parametrize("seed", range(200))
def test_tiny_random_epsilon(comp, seed):
    rng = np.random.default_rng(5000 + seed)
    V = 2 + seed % 6
    A = synth.tiny_random(rng, V, 4, 3, 0.3, p_accept=0.4, n_start=1 + seed % 3)
    B = synth.tiny_random(rng, V + 1, 4, 3, 0.3, p_accept=0.4, n_start=1 + (seed // 3) % 2)
    check_pair(comp, A, B, f"tiny seed {seed}", order=oracle.ORDER_PAPER)


def _hub_pair():
    # A: state 0 has 600 epsilon-output arcs and 300 arcs with output 5;
    # B: state 0 has 700 epsilon-input arcs and 300 arcs with input 5.
    rng = np.random.default_rng(7)
    arcsA = [(0, int(rng.integers(0, 40)), int(rng.integers(1, 4)), 0, float(rng.standard_normal()))
             for _ in range(600)]
    arcsA += [(0, int(rng.integers(0, 40)), 1, 5, float(rng.standard_normal())) for _ in range(300)]
    arcsA += [(s, int(rng.integers(0, 40)), 2, int(rng.integers(0, 6)), float(rng.standard_normal()))
              for s in range(1, 40) for _ in range(3)]
    arcsB = [(0, int(rng.integers(0, 50)), 0, int(rng.integers(1, 4)), float(rng.standard_normal()))
             for _ in range(700)]
    arcsB += [(0, int(rng.integers(0, 50)), 5, 2, float(rng.standard_normal())) for _ in range(300)]
    arcsB += [(s, int(rng.integers(0, 50)), int(rng.integers(0, 6)), 1, float(rng.standard_normal()))
              for s in range(1, 50) for _ in range(3)]
    A = synth.from_arcs(40, arcsA, start=[0], accept=list(range(0, 40, 3)))
    B = synth.from_arcs(50, arcsB, start=[0], accept=list(range(0, 50, 4)))
    return A, B


def _sparse_chain_graph(rng, V, n_sym, p_eps, p_par):
    """Mostly one arc in and one arc out per state (the shape for which
    searches skip claims), with random extra arcs, parallel same-label arcs,
    epsilon labels, cycles back to start states and accepting states with
    out-arcs, so every condition that disables the shortcut occurs."""
    arcs = []
    lab = lambda: 0 if rng.random() < p_eps else int(rng.integers(1, n_sym + 1))
    for s in range(V):
        d = (s + 1) % V if rng.random() < 0.8 else int(rng.integers(0, V))
        il, ol = lab(), lab()
        arcs.append((s, d, il, ol, float(np.float32(rng.standard_normal()))))
        if rng.random() < p_par:  # parallel arc with the same labels
            arcs.append((s, d, il, ol, float(np.float32(rng.standard_normal()))))
        if rng.random() < 0.2:
            arcs.append((s, int(rng.integers(0, V)), lab(), lab(), 0.5))
    starts = [0] + [int(x) for x in rng.integers(0, V, size=int(rng.integers(0, 3)))]
    accepts = [int(x) for x in rng.integers(0, V, size=int(rng.integers(1, V // 3 + 2)))]
    return synth.from_arcs(V, arcs, start=sorted(set(starts)), accept=sorted(set(accepts)))


@pytest.mark.parametrize("seed", range(60))
def test_unique_move_chains(comp, seed):
    rng = np.random.default_rng([77, seed])
    V = int(rng.integers(3, 40))
    n_sym = 1 + (seed % 4 == 3)
    A = _sparse_chain_graph(rng, V, n_sym, [0.0, 0.2, 0.5][seed % 3], 0.1)
    B = _sparse_chain_graph(rng, int(rng.integers(3, 40)), n_sym, [0.3, 0.0, 0.1][seed % 3], 0.1)
    got, _ = check_pair(comp, A, B, f"unique-move chains seed {seed}")
    assert not fsthelp.check_invariants(A, B, got)


def test_unique_move_corner_cases(comp):
    # a start state that a move also reaches; an accepting state that also
    # has an out-move; an A state whose in-arc comes from a state with an
    # epsilon output (two filter states lead to its key)
    A = synth.from_arcs(4, [(0, 1, 1, 1, 0.5), (1, 2, 2, 2, 0.25), (2, 0, 3, 3, 1.0),
                            (2, 3, 1, 0, 2.0), (3, 1, 1, 1, 0.125)], start=[0], accept=[0, 3])
    B = synth.from_arcs(3, [(0, 1, 1, 5, 0.5), (1, 2, 2, 6, 0.0), (2, 0, 3, 7, 1.5),
                            (0, 0, 0, 8, 0.75)], start=[0], accept=[0, 2])
    for X, Y, tag in ((A, B, "A o B"), (B, A, "B o A"), (A, A, "A o A"), (B, B, "B o B")):
        got, _ = check_pair(comp, X, Y, f"corner {tag}")
        assert not fsthelp.check_invariants(X, Y, got)


def test_accepting_states_with_one_move(comp):
    # keys of C with exactly one move whose target is a dead end: (1, 1) by
    # a matching pair (B's one arc, A's labels distinct), (2, 1) by an A
    # epsilon arc.  Both accept, so they are kept with no kept arc; the
    # keys before them have one kept arc each.
    A = synth.from_arcs(4, [(0, 1, 1, 1, 0.5), (1, 3, 2, 2, 0.25), (1, 2, 3, 3, 1.0),
                            (2, 3, 4, 0, 2.0), (0, 2, 6, 6, 0.75)], start=[0], accept=[1, 2])
    B = synth.from_arcs(3, [(0, 1, 1, 5, 0.5), (1, 2, 2, 6, 0.0), (0, 1, 6, 8, 1.5)],
                        start=[0], accept=[1])
    got, _ = check_pair(comp, A, B, "accepting one-move keys")
    assert (got["num_states"], got["num_arcs"]) == (3, 2)
    assert not fsthelp.check_invariants(A, B, got)


def _sparse_emissions(rng, T, C, p_tok, p_dup, p_acc):
    """Linear acceptor where each frame has a random subset of tokens, some
    tokens twice (buckets of two arcs), and some extra accepting frames."""
    arcs = []
    for t in range(T):
        toks = [c for c in range(1, C + 1) if rng.random() < p_tok] or [1]
        for c in toks:
            w = float(np.float32(rng.standard_normal()))
            arcs.append((t, t + 1, c, c, w))
            if rng.random() < p_dup:
                arcs.append((t, t + 1, c, c, w + 1.0))
    acc = [T] + [t for t in range(T) if rng.random() < p_acc]
    return synth.from_arcs(T + 1, arcs, start=[0], accept=sorted(set(acc)))


def _long_word_lexicon(rng, W, C, lo, hi, p_acc):
    """Lexicon whose words can be longer than a chain record (so chains are
    followed over several records), with some accepting word states."""
    arcs, V, acc = [], 1, [0]
    for w in range(1, W + 1):
        L = int(rng.integers(lo, hi + 1))
        first = V
        arcs.append((0, first, 0, w, 0.0))
        for j in range(L):
            arcs.append((first + j, first + j + 1, int(rng.integers(1, C + 1)), 0, 0.0))
            if rng.random() < p_acc:
                acc.append(first + j + 1)
        arcs.append((first + L, 0, 0, 0, 0.0))
        V = first + L + 1
    return synth.from_arcs(V, arcs, start=[0], accept=sorted(set(acc)))


@pytest.mark.parametrize("seed", range(24))
def test_chain_jump_conditions(comp, seed):
    rng = np.random.default_rng([91, seed])
    C = int(rng.integers(2, 5))
    A = _sparse_emissions(rng, int(rng.integers(10, 40)), C, [1.0, 0.7][seed % 2],
                          [0.0, 0.15][(seed // 2) % 2], [0.0, 0.1][(seed // 4) % 2])
    B = _long_word_lexicon(rng, int(rng.integers(5, 40)), C, 2, 16, [0.0, 0.05][(seed // 8) % 2])
    got, _ = check_pair(comp, A, B, f"chain-jump conditions seed {seed}")
    assert not fsthelp.check_invariants(A, B, got)


@pytest.mark.parametrize("mode", ["A shuffled", "A reversed", "B shuffled", "both shuffled"])
@pytest.mark.parametrize("seed", range(2))
def test_renumbered_states(comp, mode, seed):
    """Emissions and lexicon with their states renumbered: chains whose A
    states are not consecutive (a chain jump's guessed A states miss and
    the jump looks them up again, or ends early) and word states scattered
    over the search bitmaps' diagonals.  Same result as the oracle's on the
    same renumbered inputs."""
    spec = synth.LexSpec(T=60, C=8, W=300, len_lo=2, len_hi=14)
    A, B, _ = synth.emissions_lexicon("lexicon-T100-W1000", seed, spec=spec)
    rng = np.random.default_rng([17, seed])
    if mode in ("A shuffled", "both shuffled"):
        A = fsthelp.renumber(A, rng.permutation(A["num_states"]))
    if mode == "A reversed":
        A = fsthelp.renumber(A, np.arange(A["num_states"])[::-1])
    if mode in ("B shuffled", "both shuffled"):
        B = fsthelp.renumber(B, rng.permutation(B["num_states"]))
    got, _ = check_pair(comp, A, B, f"renumbered states ({mode}) seed {seed}")
    assert got["num_arcs"] > 0
    assert not fsthelp.check_invariants(A, B, got)


@pytest.fixture(scope="module")
def comp_paper_order():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2110_02848_amd import gpu
    c = gpu.Composer(0)
    c.set_option(gpu.FST_OPT_ORDER, gpu.FST_ORDER_COACCESSIBLE_FIRST)
    yield c
    c.close()


def _paper_order_cases():
    cases = [("random-64", s) for s in range(30)] + [("random-1000", s) for s in (1, 2)]
    cases += [("random-5000", s) for s in (0, 3, 471, 1175, 2216, 2404, 2647)]
    cases += [("random-5000-k16", 0), ("lexicon-T100-W1000", 0)]
    return cases


@pytest.mark.parametrize("name,seed", _paper_order_cases())
def test_coaccessible_first_order(comp_paper_order, name, seed):
    A, B = named_pair(name, seed)
    got, _ = check_pair(comp_paper_order, A, B, f"co-accessible first {name} seed {seed}",
                        ref=cached_ref(name, seed, A, B))
    if seed < 3:
        assert not fsthelp.check_invariants(A, B, got)


@pytest.mark.parametrize("seed", range(40))
def test_coaccessible_first_order_small(comp_paper_order, seed):
    rng = np.random.default_rng([123, seed])
    if seed % 2:
        V = int(rng.integers(3, 40))
        A = _sparse_chain_graph(rng, V, 1 + (seed % 4 == 3), 0.2, 0.1)
        B = _sparse_chain_graph(rng, int(rng.integers(3, 40)), 1 + (seed % 4 == 3), 0.1, 0.1)
    else:
        A = synth.tiny_random(rng, int(rng.integers(1, 6)), 3, 3, 0.4)
        B = synth.tiny_random(rng, int(rng.integers(1, 6)), 3, 3, 0.4)
    got, _ = check_pair(comp_paper_order, A, B, f"co-accessible first small seed {seed}")
    assert not fsthelp.check_invariants(A, B, got)


@pytest.fixture(scope="module")
def comp_concurrent():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2110_02848_amd import gpu
    c = gpu.Composer(0)
    c.set_option(gpu.FST_OPT_ORDER, gpu.FST_ORDER_CONCURRENT)
    yield c
    c.close()


@pytest.fixture(scope="module")
def comp_forward_first():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2110_02848_amd import gpu
    c = gpu.Composer(0)
    c.set_option(gpu.FST_OPT_ORDER, gpu.FST_ORDER_FORWARD_FIRST)
    yield c
    c.close()


@pytest.mark.parametrize("name,seed", _paper_order_cases() + [("lexicon-T100-W1000", 2)])
def test_forward_first_order(comp_forward_first, name, seed):
    A, B = named_pair(name, seed)
    got, _ = check_pair(comp_forward_first, A, B, f"forward first {name} seed {seed}",
                        ref=cached_ref(name, seed, A, B))
    if seed < 3:
        assert not fsthelp.check_invariants(A, B, got)


@pytest.mark.parametrize("seed", range(40))
def test_forward_first_order_small(comp_forward_first, seed):
    rng = np.random.default_rng([987, seed])
    A = synth.tiny_random(rng, int(rng.integers(1, 6)), 3, 3, 0.4)
    B = synth.tiny_random(rng, int(rng.integers(1, 6)), 3, 3, 0.4)
    got, _ = check_pair(comp_forward_first, A, B, f"forward first small seed {seed}")
    assert not fsthelp.check_invariants(A, B, got)


@pytest.mark.parametrize("name,seed", _paper_order_cases() + [("lexicon-T100-W1000", 2)])
def test_concurrent_order(comp_concurrent, name, seed):
    A, B = named_pair(name, seed)
    got, _ = check_pair(comp_concurrent, A, B, f"concurrent {name} seed {seed}",
                        ref=cached_ref(name, seed, A, B))
    if seed < 3:
        assert not fsthelp.check_invariants(A, B, got)


@pytest.mark.parametrize("seed", range(40))
def test_concurrent_order_small(comp_concurrent, seed):
    rng = np.random.default_rng([321, seed])
    if seed % 2:
        A = _sparse_chain_graph(rng, int(rng.integers(3, 40)), 1 + (seed % 4 == 3), 0.2, 0.1)
        B = _sparse_chain_graph(rng, int(rng.integers(3, 40)), 1 + (seed % 4 == 3), 0.1, 0.1)
    else:
        A = synth.tiny_random(rng, int(rng.integers(1, 6)), 3, 3, 0.4)
        B = synth.tiny_random(rng, int(rng.integers(1, 6)), 3, 3, 0.4)
    got, _ = check_pair(comp_concurrent, A, B, f"concurrent small seed {seed}")
    assert not fsthelp.check_invariants(A, B, got)


def test_concurrent_order_hubs_and_full_lexicon(comp_concurrent):
    A, B = _hub_pair()
    check_pair(comp_concurrent, A, B, "concurrent hub states")
    A, B, meta = synth.emissions_lexicon("lexicon-T500-W10000", 0)
    C = gpu_compose(comp_concurrent, A, B)
    V, E = fsthelp.lexicon_closed_form(meta["spec"].T, meta["spellings"])
    assert (C["num_states"], C["num_arcs"]) == (V, E)
    st = comp_concurrent.stats()
    assert st["fwd_levels"] > 0 and st["bwd_levels"] > 0


def test_heavy_states(comp):
    A, B = _hub_pair()
    got, _ = check_pair(comp, A, B, "hub states")
    assert got["num_arcs"] > 90000
    assert comp.stats()["heavy_states"] > 0


def test_many_heavy_keys_in_one_generation(comp):
    # the forward search lists 300 keys of 70 units each in one generation,
    # more than the heavy list a workgroup keeps in LDS
    rng = np.random.default_rng(5)
    n, fan = 300, 70
    arcsA = [(0, 1 + i, 1, 1, float(rng.standard_normal())) for i in range(n)]
    arcsA += [(1 + i, n + 1, 1, 1 + lab, float(rng.standard_normal()))
              for i in range(n) for lab in range(fan)]
    arcsB = [(0, 0, 1 + lab, 1 + lab, float(rng.standard_normal())) for lab in range(fan)]
    A = synth.from_arcs(n + 2, arcsA, start=[0], accept=[n + 1])
    B = synth.from_arcs(1, arcsB, start=[0], accept=[0])
    got, _ = check_pair(comp, A, B, "300 heavy keys in one generation")
    assert got["num_arcs"] == n + n * fan
    assert comp.stats()["heavy_states"] > n


def test_lexicon_small_many_words(comp):
    spec = synth.LexSpec(T=40, C=8, W=3000, len_lo=1, len_hi=4)
    A, B, meta = synth.emissions_lexicon("lexicon-T100-W1000", 11, spec=spec)
    got, _ = check_pair(comp, A, B, "lexicon W=3000")
    assert comp.stats()["heavy_states"] > 0
    V, E = fsthelp.lexicon_closed_form(spec.T, meta["spellings"])
    assert (got["num_states"], got["num_arcs"]) == (V, E)


def test_identity_compositions(comp):
    rng = np.random.default_rng(3)
    A = synth.random_fst(rng, 300, 4, 8, 0.2, 0.1)
    Id = synth.identity_fst(8)
    check_pair(comp, A, Id, "A o Id")
    check_pair(comp, Id, A, "Id o A")


def test_epsilon_cycles_and_self_loops(comp):
    A = synth.from_arcs(2, [(0, 0, 1, 0, 0.5), (0, 1, 0, 0, -0.25), (1, 0, 2, 1, 1.0),
                            (1, 1, 0, 2, 0.125)], start=[0, 1], accept=[1])
    B = synth.from_arcs(2, [(0, 1, 0, 3, 0.5), (1, 0, 0, 0, 0.75), (0, 0, 1, 4, -1.0),
                            (1, 1, 2, 0, 0.25)], start=[0], accept=[0, 1])
    got, _ = check_pair(comp, A, B, "epsilon cycles")
    assert got["num_arcs"] > 0


def test_rounding_cases(comp):
    for wa, wb in [(1.0, 2.0 ** -24), (1.0, 3 * 2.0 ** -25), (2.0 ** -126, -(2.0 ** -127)),
                   (2.0 ** -149, 2.0 ** -149), (3.0e38, 3.0e38), (-0.0, -0.0)]:
        A = synth.from_arcs(2, [(0, 1, 1, 2, wa), (0, 1, 3, 0, -0.0)], start=[0], accept=[1])
        B = synth.from_arcs(2, [(0, 1, 2, 3, wb), (0, 1, 0, 4, -0.0)], start=[0], accept=[1])
        check_pair(comp, A, B, f"rounding {wa} {wb}")


def test_light_states_with_wide_fanout(comp):
    """Start keys with one work unit each and 300, 255 and 254 kept arcs:
    the counts of 255 and more take the wide-count path of count and fill,
    and the offsets of every later state include them."""
    A, B = fsthelp.wide_fanout_pair(np.random.default_rng(31))
    got, _ = check_pair(comp, A, B, "wide fan-out of light states")
    deg = np.diff(got["arc_offset"].astype(np.int64))
    assert sorted(deg.tolist())[-3:] == [254, 255, 300]


def test_degenerate_inputs(comp):
    E0 = synth.empty_graph()
    A, B = synth.workload("random-64", 0)
    # a composition with states first: the empty runs after it must not
    # reuse its output layout (their fill writes arc_offset[0] only)
    got, _ = check_pair(comp, A, B, "non-empty before empty inputs")
    assert got["num_states"] > 0
    for X, Y, tag in ((E0, E0, "empty/empty"), (E0, A, "empty/A"), (A, E0, "A/empty")):
        got, _ = check_pair(comp, X, Y, tag)
        assert got["num_states"] == 0 and got["arc_offset"].tolist() == [0]
    nostart = synth.from_arcs(2, [(0, 1, 1, 1, 0.0)], start=[], accept=[1])
    dead = synth.from_arcs(2, [(0, 1, 2, 2, 0.0)], start=[0], accept=[1])
    one = synth.from_arcs(2, [(0, 1, 1, 1, 0.0)], start=[0], accept=[1])
    for X, Y, tag in ((nostart, one, "no start"), (one, dead, "dead start")):
        got, _ = check_pair(comp, X, Y, tag)
        assert got["num_states"] == 0
    single = synth.from_arcs(1, [], start=[0], accept=[0])
    got, _ = check_pair(comp, single, single, "single state")
    assert got["num_states"] == 1 and got["start"].tolist() == [1]


def test_deterministic_and_context_reuse(comp):
    A2, B2 = synth.workload("random-1000", 1)
    A1, B1 = synth.workload("random-64", 3)
    r1 = gpu_compose(comp, A2, B2)
    gpu_compose(comp, A1, B1)
    r2 = gpu_compose(comp, A2, B2)
    assert not fsthelp.compare_results(r1, r2)


def test_errors(comp):
    import torch
    from paper_2110_02848_amd import gpu
    A, B = synth.workload("random-64", 0)
    bad = {k: (v.copy() if hasattr(v, "copy") else v) for k, v in A.items()}
    bad["dst"][3] = A["num_states"]  # out of range
    with pytest.raises(gpu.FstError) as ei:
        comp.run(gpu.to_device(bad), gpu.to_device(B))
    assert ei.value.code == gpu.FST_ERR_INVALID_GRAPH
    bad = {k: (v.copy() if hasattr(v, "copy") else v) for k, v in A.items()}
    bad["arc_offset"][5] += 1  # offsets disagree with src
    with pytest.raises(gpu.FstError) as ei:
        comp.run(gpu.to_device(bad), gpu.to_device(B))
    assert ei.value.code == gpu.FST_ERR_INVALID_GRAPH
    # fill after a failed run
    with pytest.raises(gpu.FstError) as ei:
        comp.fill(comp.alloc_output(0, 0))
    assert ei.value.code == gpu.FST_ERR_STATE
    # key space beyond 2^32 keys
    big = synth.from_arcs(70000, [(0, 1, 1, 1, 0.0)], start=[0], accept=[1])
    with pytest.raises(gpu.FstError) as ei:
        comp.run(gpu.to_device(big), gpu.to_device(big))
    assert ei.value.code == gpu.FST_ERR_TOO_LARGE
    # workspace cap
    small = gpu.Composer(0)
    small.set_option(gpu.FST_OPT_MAX_WORKSPACE, 4096)
    with pytest.raises(gpu.FstError) as ei:
        small.run(gpu.to_device(A), gpu.to_device(B))
    assert ei.value.code == gpu.FST_ERR_NOMEM
    small.close()
    torch.cuda.synchronize()
    # the context still works after errors
    check_pair(comp, A, B, "after errors")
