"""Options that must never change the result (label bucket tables, the
depth-first budget of a search thread) in every search order: each option
set composes the same inputs and is compared with the oracle element by
element, with its search statistics.  Without bucket tables every label
lookup is a binary search in the label-sorted arcs and no chain jump runs;
with a budget of 0 the search goes frontier by frontier, with 1 a thread
expands one extra key."""
import itertools

import numpy as np
import pytest

from paper_2110_02848_amd import synth

import fsthelp
from test_gpu_parity import (_hub_pair, _long_word_lexicon, _sparse_emissions, cached_ref,
                             check_pair, named_pair)

pytestmark = pytest.mark.gpu

ORDERS = ("forward-first", "coaccessible-first", "concurrent")
OPTION_SETS = list(itertools.product(ORDERS, (0, 1), (0, 1, 64)))

_COMPOSERS = {}


@pytest.fixture(scope="module")
def composers():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    yield _COMPOSERS
    for c in _COMPOSERS.values():
        c.close()
    _COMPOSERS.clear()


def composer(pool, order, buckets, depth):
    from paper_2110_02848_amd import gpu
    k = (order, buckets, depth)
    if k not in pool:
        c = gpu.Composer(0)
        c.set_option(gpu.FST_OPT_ORDER, {"forward-first": gpu.FST_ORDER_FORWARD_FIRST,
                                         "coaccessible-first": gpu.FST_ORDER_COACCESSIBLE_FIRST,
                                         "concurrent": gpu.FST_ORDER_CONCURRENT}[order])
        c.set_option(gpu.FST_OPT_LABEL_BUCKETS, buckets)
        c.set_option(gpu.FST_OPT_CHAIN_DEPTH, depth)
        c.set_option(gpu.FST_OPT_COUNT_MOVES, 1)
        pool[k] = c
    return pool[k]


def _inputs(case):
    kind, seed = case
    if kind in ("random-64", "random-1000", "random-5000", "lexicon-T100-W1000"):
        A, B = named_pair(kind, seed)
        return A, B, cached_ref(kind, seed, A, B)
    if kind == "hubs":
        A, B = _hub_pair()
        return A, B, cached_ref("hubs", 0, A, B)
    if kind == "tiny":
        rng = np.random.default_rng([4040, seed])
        V = 2 + seed % 5
        A = synth.tiny_random(rng, V, 4, 3, 0.35, p_accept=0.4, n_start=1 + seed % 2)
        B = synth.tiny_random(rng, V + 1, 4, 3, 0.35, p_accept=0.4, n_start=1)
        return A, B, cached_ref("tiny-options", seed, A, B)
    if kind == "long-words":
        rng = np.random.default_rng([92, seed])
        A = _sparse_emissions(rng, 30, 3, 1.0, 0.1, 0.05)
        B = _long_word_lexicon(rng, 25, 3, 2, 16, 0.05)
        return A, B, cached_ref("long-words", seed, A, B)
    raise KeyError(kind)


CASES = ([("random-64", s) for s in range(3)] + [("random-1000", 1), ("random-5000", 471),
         ("lexicon-T100-W1000", 0), ("hubs", 0), ("long-words", 0), ("long-words", 1)]
         + [("tiny", s) for s in range(6)])


@pytest.mark.parametrize("order,buckets,depth", OPTION_SETS)
def test_options_never_change_the_result(composers, order, buckets, depth):
    comp = composer(composers, order, buckets, depth)
    for case in CASES:
        A, B, ref = _inputs(case)
        tag = f"{case[0]} seed {case[1]} order={order} buckets={buckets} depth={depth}"
        got, _ = check_pair(comp, A, B, tag, ref=ref)
        if case[0] in ("hubs", "long-words", "random-64"):
            assert not fsthelp.check_invariants(A, B, got), tag


def test_validation_off_same_result(composers):
    """FST_OPT_VALIDATE = 0 (the caller vouches for its graphs): the same
    result on valid inputs, compositions and scores."""
    from paper_2110_02848_amd import gpu
    import torch
    c = gpu.Composer(0)
    c.set_option(gpu.FST_OPT_VALIDATE, 0)
    try:
        for case in [("random-64", 0), ("random-1000", 1), ("lexicon-T100-W1000", 0),
                     ("hubs", 0)] + [("tiny", s) for s in range(4)]:
            A, B, ref = _inputs(case)
            check_pair(c, A, B, f"{case} validation off", ref=ref)
        A, B, ref = _inputs(("lexicon-T100-W1000", 0))
        C = c.compose(gpu.to_device(A), gpu.to_device(B))
        s_off = c.score(C)["total"].item()
        c.set_option(gpu.FST_OPT_VALIDATE, 1)
        s_on = c.score(C)["total"].item()
        torch.cuda.synchronize()
        assert s_off == s_on
    finally:
        c.close()


@pytest.mark.parametrize("order", ORDERS)
def test_search_lists_grow(composers, order):
    """Search lists far too small at first (FST_OPT_LIST_CAPACITY = 256):
    every search overflows them, grows them four-fold and runs again, with
    the same result; the next call starts at the size that sufficed."""
    from paper_2110_02848_amd import gpu
    c = gpu.Composer(0)
    try:
        c.set_option(gpu.FST_OPT_ORDER, {"forward-first": gpu.FST_ORDER_FORWARD_FIRST,
                                         "coaccessible-first": gpu.FST_ORDER_COACCESSIBLE_FIRST,
                                         "concurrent": gpu.FST_ORDER_CONCURRENT}[order])
        c.set_option(gpu.FST_OPT_COUNT_MOVES, 1)
        for case in [("random-1000", 1), ("lexicon-T100-W1000", 0), ("hubs", 0),
                     ("random-64", 1)]:
            c.set_option(gpu.FST_OPT_LIST_CAPACITY, 256)
            A, B, ref = _inputs(case)
            check_pair(c, A, B, f"{case} lists from 256 entries, {order}", ref=ref)
            check_pair(c, A, B, f"{case} again, {order}", ref=ref)
    finally:
        c.close()
