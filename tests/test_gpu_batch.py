"""Batched and chained composition on the GPU versus the CPU oracle.

A batch composes the disjoint union of its A_i with one B; each item's slice
of the result (ids rebased) must equal the oracle's A_i o B bit for bit.  A
chain composes the GPU's C with a third graph; it must equal the oracle's
composition of its own C with that graph."""
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
    yield c
    c.close()


def gpu_batch(comp, As, B):
    import torch
    from paper_2110_02848_amd import gpu
    C, st, ar = comp.compose_batch([gpu.to_device(A) for A in As], gpu.to_device(B))
    torch.cuda.synchronize()
    return gpu.to_numpy(C), st, ar


def item_slice(C, st, ar, i, As):
    """Item i of a batch result with item-local ids."""
    s0, s1, a0, a1 = int(st[i]), int(st[i + 1]), int(ar[i]), int(ar[i + 1])
    vbase = sum(int(A["num_states"]) for A in As[:i])
    ebase = sum(len(A["src"]) for A in As[:i])
    arc_a = C["arc_a"][a0:a1].astype(np.int64)
    return dict(
        num_states=s1 - s0, num_arcs=a1 - a0,
        arc_offset=(C["arc_offset"][s0:s1 + 1].astype(np.int64) - a0).astype(np.int32),
        src=(C["src"][a0:a1].astype(np.int64) - s0).astype(np.int32),
        dst=(C["dst"][a0:a1].astype(np.int64) - s0).astype(np.int32),
        ilabel=C["ilabel"][a0:a1], olabel=C["olabel"][a0:a1], weight=C["weight"][a0:a1],
        arc_a=np.where(arc_a >= 0, arc_a - ebase, -1).astype(np.int32),
        arc_b=C["arc_b"][a0:a1],
        start=C["start"][s0:s1], accept=C["accept"][s0:s1],
        key_a=(C["key_a"][s0:s1].astype(np.int64) - vbase).astype(np.int32),
        key_b=C["key_b"][s0:s1], key_f=C["key_f"][s0:s1])


def check_batch(comp, As, B, tag, ref_B=None):
    """ref_B: the B the oracle composes each item with (default B)."""
    print(f"[batch] {tag}", flush=True)
    C, st, ar = gpu_batch(comp, As, B)
    assert st[0] == 0 and ar[0] == 0
    assert st[-1] == C["num_states"] and ar[-1] == C["num_arcs"]
    assert np.all(np.diff(st) >= 0) and np.all(np.diff(ar) >= 0)
    for i, A in enumerate(As):
        ref = oracle.compose(A, B if ref_B is None else ref_B)
        got = item_slice(C, st, ar, i, As)
        errs = fsthelp.compare_results(got, ref)
        assert not errs, (tag, i, errs[:5])
    return C, st, ar


@pytest.mark.parametrize("seed", range(3))
def test_batch_of_lexicon_items(comp, seed):
    spec = synth.LexSpec(60, 8, 40, 2, 5)
    frames = [30, 45, 0, 60, 17][: 3 + seed]
    As, B, _ = synth.lexicon_batch("lexicon-T100-W1000", len(frames), seed, spec=spec,
                                   frames=frames)
    check_batch(comp, As, B, f"lexicon items {frames} seed {seed}")


@pytest.mark.parametrize("seed", range(4))
def test_batch_of_random_items(comp, seed):
    rng = np.random.default_rng(100 + seed)
    B = synth.tiny_random(rng, 12, 3, 4, 0.2, p_accept=0.5)
    As = [synth.tiny_random(rng, int(rng.integers(1, 15)), 3, 4, 0.2, p_accept=0.5,
                            n_start=int(rng.integers(1, 3))) for _ in range(6)]
    As.insert(2, synth.empty_graph())
    check_batch(comp, As, B, f"random items seed {seed}")


def test_batch_random_1000_items(comp):
    As = [synth.workload("random-1000", s)[0] for s in range(3)]
    B = synth.workload("random-1000", 0)[1]
    check_batch(comp, As, B, "random-1000 items")


def test_batch_of_one_equals_plain_composition(comp):
    import torch
    from paper_2110_02848_amd import gpu
    A, B = synth.workload("lexicon-T100-W1000", 1)
    C, st, ar = gpu_batch(comp, [A], B)
    plain = gpu.to_numpy(comp.compose(gpu.to_device(A), gpu.to_device(B)))
    torch.cuda.synchronize()
    assert list(st) == [0, plain["num_states"]] and list(ar) == [0, plain["num_arcs"]]
    for k in ("arc_offset", "src", "dst", "ilabel", "olabel", "arc_a", "arc_b", "start",
              "accept", "key_a", "key_b", "key_f"):
        assert np.array_equal(C[k], plain[k]), k
    assert np.array_equal(C["weight"].view(np.uint32), plain["weight"].view(np.uint32))


def test_batch_edge_cases(comp):
    from paper_2110_02848_amd import gpu
    B = synth.workload("random-64", 0)[1]
    nv, ne, st, ar = comp.run_batch([], gpu.to_device(B))
    assert (nv, ne) == (0, 0) and list(st) == [0] and list(ar) == [0]
    e = synth.empty_graph()
    nv, ne, st, ar = comp.run_batch([gpu.to_device(e), gpu.to_device(e)], gpu.to_device(B))
    assert (nv, ne) == (0, 0) and list(st) == [0, 0, 0]
    # an arc of one item naming a state of the next is an invalid item, not
    # a valid arc of the union
    A0 = synth.from_arcs(2, [(0, 1, 1, 1, 0.0)], start=[0], accept=[1])
    A0 = dict(A0)
    A0["dst"] = np.array([2], np.int32)
    A1 = synth.from_arcs(2, [(0, 1, 1, 1, 0.0)], start=[0], accept=[1])
    with pytest.raises(gpu.FstError) as err:
        comp.run_batch([gpu.to_device(A0), gpu.to_device(A1)], gpu.to_device(B))
    assert err.value.code == gpu.FST_ERR_INVALID_GRAPH
    # the context still works
    check_batch(comp, [synth.workload("random-64", 3)[0]], B, "after error")


def test_batch_scores_per_item(comp):
    """Per-item forward scores of a batch: scores of the union C, then the
    log-sum of alpha over each item's accepting states, against the frame
    recursion over word segmentations of each item."""
    import torch
    from paper_2110_02848_amd import gpu
    frames = [100, 40, 77, 3, 0]
    As, B, meta = synth.lexicon_batch("lexicon-T100-W1000", len(frames), 5, frames=frames)
    Cd, st, ar = comp.compose_batch([gpu.to_device(A) for A in As], gpu.to_device(B))
    sc = comp.score(Cd, beta=False)
    tot = comp.segment_logsum(sc["alpha"], Cd["accept"], st)
    torch.cuda.synchronize()
    tot = tot.cpu().numpy()
    for i, T in enumerate(frames):
        if T == 0:
            ref = 0.0  # the empty word sequence: the root starts and accepts
        else:
            ref = fsthelp.lexicon_total_score(meta["tables"][i], meta["spellings"])
        if np.isinf(ref):
            assert tot[i] == ref, (i, tot[i], ref)
        else:
            assert abs(tot[i] - ref) <= 1e-9 * (1 + abs(ref)), (i, tot[i], ref)


def test_segment_logsum_cases(comp):
    import torch
    rng = np.random.default_rng(3)
    val = rng.standard_normal(1000) * 50
    val[::7] = -np.inf
    flag = (rng.random(1000) < 0.6).astype(np.uint8)
    bounds = [0, 0, 1, 10, 500, 500, 1000]
    got = comp.segment_logsum(torch.from_numpy(val).cuda(), torch.from_numpy(flag).cuda(),
                              bounds).cpu().numpy()
    for i in range(len(bounds) - 1):
        x = val[bounds[i]:bounds[i + 1]][flag[bounds[i]:bounds[i + 1]] == 1]
        x = x[np.isfinite(x)]
        if len(x) == 0:
            assert got[i] == -np.inf
        else:
            m = x.max()
            ref = m + np.log(np.exp(x - m).sum())
            assert abs(got[i] - ref) <= 1e-13 * (1 + abs(ref)) * len(x), (i, got[i], ref)


@pytest.mark.parametrize("seed", range(4))
def test_chain_of_three(comp, seed):
    """A o B o D as two calls: the GPU's C composed with D equals the
    oracle's C composed with D."""
    import torch
    from paper_2110_02848_amd import gpu
    rng = np.random.default_rng(500 + seed)
    A = synth.tiny_random(rng, 10, 3, 4, 0.2, p_accept=0.5)
    B = synth.tiny_random(rng, 8, 3, 4, 0.2, p_accept=0.5)
    D = synth.tiny_random(rng, 8, 3, 4, 0.2, p_accept=0.5)
    C1 = comp.compose(gpu.to_device(A), gpu.to_device(B), provenance=False, keys=False)
    C2 = gpu.to_numpy(comp.compose(C1, gpu.to_device(D)))
    torch.cuda.synchronize()
    R1 = oracle.compose(A, B)
    R2 = oracle.compose({k: R1[k] for k in synth.GRAPH_KEYS} | {"num_states": R1["num_states"]},
                        D)
    errs = fsthelp.compare_results(C2, R2)
    assert not errs, errs[:5]


def test_batch_item_after_wide_states(comp):
    """Items whose first state follows, in the same output chunk, the
    previous item's start states of 300, 255 and 254 arcs: each item's first
    arc counts them (wide counts) and every item equals the oracle's."""
    rng = np.random.default_rng(32)
    As, B = [], None
    for _ in range(3):
        A, B0 = fsthelp.wide_fanout_pair(rng)
        As.append(A)
        B = B if B is not None else B0
    C, st, ar = check_batch(comp, As, B, "items after wide states")
    assert int(ar[1]) == 1109 and int(ar[2]) == 2 * 1109


def padded(B, extra):
    """B with `extra` isolated states appended (no arcs, neither start nor
    accepting): the same compositions over a larger key space."""
    g = dict(B)
    g["num_states"] = int(B["num_states"]) + extra
    g["arc_offset"] = np.concatenate(
        [B["arc_offset"], np.full(extra, B["arc_offset"][-1], np.int32)])
    g["start"] = np.concatenate([B["start"], np.zeros(extra, np.uint8)])
    g["accept"] = np.concatenate([B["accept"], np.zeros(extra, np.uint8)])
    return g


def test_batch_in_parts(comp):
    """A batch whose union needs more than 2^32 keys: B padded with 2^21
    isolated states has 2^23 keys per A state, so at most 448 A states fit
    one search and the five items (151 + 201, 121 + 251, 91 A states) are
    composed in three parts.  Every item equals the oracle's A_i o B (the
    oracle composes with B without the padding, which no key reaches: the
    same states, keys and arcs), with the ids, key_a and arc_a of the whole
    batch; a second fill writes the same C; the statistics are the sums."""
    import torch
    from paper_2110_02848_amd import gpu
    spec = synth.LexSpec(T=0, C=6, W=40, len_lo=2, len_hi=5)
    As, B, _ = synth.lexicon_batch("lexicon-T100-W1000", 5, 0, spec=spec,
                                   frames=[150, 200, 120, 250, 90])
    Bbig = padded(B, 1 << 21)
    C, st, ar = check_batch(comp, As, Bbig, "batch in three parts", ref_B=B)
    assert C["num_states"] > 0 and int(st[-1]) == C["num_states"]
    stats = comp.stats()
    assert stats["num_states"] == C["num_states"] and stats["num_arcs"] == C["num_arcs"]
    # the inputs stay allocated until the fills are done: the fill of a batch
    # in parts searches its parts again
    dAs, dB = [gpu.to_device(A) for A in As], gpu.to_device(Bbig)
    nv, ne, st2, ar2 = comp.run_batch(dAs, dB)
    assert (list(st2), list(ar2)) == (list(st), list(ar))
    C1 = comp.fill(comp.alloc_output(nv, ne))
    C2 = comp.fill(comp.alloc_output(nv, ne))
    torch.cuda.synchronize()
    g1, g2 = gpu.to_numpy(C1), gpu.to_numpy(C2)
    assert not fsthelp.compare_results(g1, g2)
    assert not fsthelp.compare_results(g1, C)
    del dAs, dB
    # a plain composition after it is a plain composition again
    check_batch(comp, [As[0]], B, "one part after parts")


def test_batch_full_size_lexicon(comp):
    """Four full-size utterances (T = 500, 10,000-word lexicon) in one pass:
    every item's state and arc counts equal the closed form from the word
    lengths, and its forward score the frame recursion."""
    import torch
    from paper_2110_02848_amd import gpu
    As, B, meta = synth.lexicon_batch("lexicon-T500-W10000", 4, 0)
    Cd, st, ar = comp.compose_batch([gpu.to_device(A) for A in As], gpu.to_device(B),
                                    provenance=False, keys=False)
    print("[batch] full size composed", flush=True)
    sc = comp.score(Cd, beta=False)
    tot = comp.segment_logsum(sc["alpha"], Cd["accept"], st).cpu().numpy()
    torch.cuda.synchronize()
    T = meta["spec"].T
    V, E = fsthelp.lexicon_closed_form(T, meta["spellings"])
    for i in range(4):
        assert (st[i + 1] - st[i], ar[i + 1] - ar[i]) == (V, E), i
        ref = fsthelp.lexicon_total_score(meta["tables"][i], meta["spellings"])
        assert abs(tot[i] - ref) <= 1e-8 * (1 + abs(ref)), (i, tot[i], ref)
