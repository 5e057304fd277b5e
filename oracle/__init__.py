"""CPU oracle for eager transducer composition (test infrastructure only).

Only ``tests/``, the smoke check in ``__graft_entry__`` and the CPU-baseline
leg of ``bench.py`` may import this package.  It shares no code with the GPU
library: it reads the same seeded input arrays and nothing else.

``compose(A, B)`` runs the sequential C implementation of the paper's
Algorithm 1 (Section 3.1) with the epsilon-sequencing filter described in
``oracle.c`` and returns the composed graph in canonical form:

* states are numbered in ascending key order (qa, qb, f);
* the arcs of a state are ordered by (l, a, b), where l is the label the two
  arcs were matched on (0 for the two epsilon moves), a is the arc of A and b
  the arc of B that the arc came from, and a missing arc (-1) sorts last.
  So a state lists its A-side epsilon arcs, then its B-side epsilon arcs, then
  its matching arcs grouped by middle label, each group in (a, b) order.

Parity with the GPU path is checked on this canonical form.

``compose3(A, B, D)`` (``compose3.c``) is the simultaneous composition of
three transducers, C = A o B o D (the N-way composition the paper names as
the next step), canonical in the same way: states by key (qa, qb, f1, qd,
f2), arcs of a state by (l, a, b, d), where l is the label the arcs of A
and B were matched on (0 when A or B did not move, or moved alone) and a,
b, d are the arcs of A, B and D the arc came from, a missing arc (-1)
sorting last.

``score(G)``, ``posterior(G, ...)`` and ``scatter(...)`` (``score.c``) give
the log-semiring forward and backward scores of an acyclic graph, the arc
posteriors that are the total score's gradient, and the scatter of per-arc
gradients of a composed graph to its operands through provenance.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRCS = [os.path.join(_HERE, n) for n in ("oracle.c", "score.c", "compose3.c")]
_DEPS = _SRCS + [os.path.join(_HERE, "og.h")]
# FSTC_ORACLE_LIB names another build of the same sources (the sanitizer
# build of the tests); build() then leaves it alone.
_LIB = os.environ.get("FSTC_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")


def sources():
    """The oracle's C sources (for other builds of the same code)."""
    return list(_SRCS)

ORDER_PAPER = 0
ORDER_FORWARD = 1

MUT_NONE = 0
MUT_NO_FILTER = 1
MUT_DROP_WB = 2
MUT_MIDDLE_LABEL = 3
MUT_ACCEPT_A = 4
MUT_NO_TRIM = 5
MUT_EPS_MATCH = 6

# deliberate mistakes of the score oracle (tests of the pins only)
SMUT_NONE = 0
SMUT_MAX = 1
SMUT_DROP_WEIGHT = 2
SMUT_ALL_ACCEPT = 3
SMUT_NO_START = 4

# deliberate mistakes of the three-input oracle (tests of the pins only)
MUT3_NONE = 0
MUT3_NO_INNER_FILTER = 1
MUT3_NO_OUTER_FILTER = 2
MUT3_DROP_WD = 3
MUT3_OUTER_LABEL = 4

_ERRORS = {1: "invalid argument", 2: "out of memory", 3: "key space too large",
           4: "graph has a cycle"}


class CycleError(ValueError):
    """The graph has a cycle, so its path sums are not defined here."""


def build(force=True):
    """Compile the oracle with gcc (IEEE binary32 adds: no fast-math)."""
    if os.environ.get("FSTC_ORACLE_LIB"):
        return _LIB
    if not force and os.path.exists(_LIB) and all(
            os.path.getmtime(_LIB) >= os.path.getmtime(f) for f in _DEPS):
        return _LIB
    tmp = _LIB + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-std=gnu11", "-fPIC", "-shared", "-fno-fast-math",
           "-ffp-contract=off", "-Wall", "-Wextra", "-Wno-unused-parameter",
           "-o", tmp, *_SRCS, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB)
    return _LIB


class _Graph(ctypes.Structure):
    _fields_ = [("num_states", ctypes.c_int32), ("num_arcs", ctypes.c_int32),
                ("arc_offset", ctypes.c_void_p), ("src", ctypes.c_void_p),
                ("dst", ctypes.c_void_p), ("ilabel", ctypes.c_void_p),
                ("olabel", ctypes.c_void_p), ("weight", ctypes.c_void_p),
                ("start", ctypes.c_void_p), ("accept", ctypes.c_void_p)]


class _Result(ctypes.Structure):
    _fields_ = [("num_states", ctypes.c_int64), ("num_arcs", ctypes.c_int64),
                ("key_a", ctypes.c_void_p), ("key_b", ctypes.c_void_p),
                ("key_f", ctypes.c_void_p), ("start", ctypes.c_void_p),
                ("accept", ctypes.c_void_p), ("arc_src", ctypes.c_void_p),
                ("arc_dst", ctypes.c_void_p), ("arc_ilabel", ctypes.c_void_p),
                ("arc_olabel", ctypes.c_void_p), ("arc_weight", ctypes.c_void_p),
                ("arc_a", ctypes.c_void_p), ("arc_b", ctypes.c_void_p),
                ("accessible", ctypes.c_int64), ("coaccessible", ctypes.c_int64),
                ("generated", ctypes.c_int64), ("pairs_examined", ctypes.c_int64),
                ("compose_seconds", ctypes.c_double)]


class _Result3(ctypes.Structure):
    _fields_ = [("num_states", ctypes.c_int64), ("num_arcs", ctypes.c_int64),
                ("key_a", ctypes.c_void_p), ("key_b", ctypes.c_void_p),
                ("key_d", ctypes.c_void_p), ("key_fab", ctypes.c_void_p),
                ("key_f", ctypes.c_void_p), ("start", ctypes.c_void_p),
                ("accept", ctypes.c_void_p), ("arc_src", ctypes.c_void_p),
                ("arc_dst", ctypes.c_void_p), ("arc_ilabel", ctypes.c_void_p),
                ("arc_olabel", ctypes.c_void_p), ("arc_weight", ctypes.c_void_p),
                ("arc_a", ctypes.c_void_p), ("arc_b", ctypes.c_void_p),
                ("arc_d", ctypes.c_void_p), ("accessible", ctypes.c_int64),
                ("generated", ctypes.c_int64), ("compose_seconds", ctypes.c_double)]


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        lib.oracle_compose.argtypes = [ctypes.POINTER(_Graph), ctypes.POINTER(_Graph),
                                       ctypes.c_int, ctypes.c_int, ctypes.POINTER(_Result)]
        lib.oracle_compose.restype = ctypes.c_int
        lib.oracle_free.argtypes = [ctypes.POINTER(_Result)]
        lib.oracle_free.restype = None
        lib.oracle_compose3.argtypes = [ctypes.POINTER(_Graph), ctypes.POINTER(_Graph),
                                        ctypes.POINTER(_Graph), ctypes.c_int,
                                        ctypes.POINTER(_Result3)]
        lib.oracle_compose3.restype = ctypes.c_int
        lib.oracle_free3.argtypes = [ctypes.POINTER(_Result3)]
        lib.oracle_free3.restype = None
        lib.oracle_in_csr.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                      ctypes.c_void_p, ctypes.c_void_p]
        lib.oracle_in_csr.restype = ctypes.c_int
        lib.oracle_score.argtypes = [ctypes.POINTER(_Graph), ctypes.c_int, ctypes.c_void_p,
                                     ctypes.c_void_p, ctypes.POINTER(ctypes.c_double),
                                     ctypes.POINTER(ctypes.c_double),
                                     ctypes.POINTER(ctypes.c_int32)]
        lib.oracle_score.restype = ctypes.c_int
        lib.oracle_posterior.argtypes = [ctypes.POINTER(_Graph), ctypes.c_void_p,
                                         ctypes.c_void_p, ctypes.c_double, ctypes.c_void_p]
        lib.oracle_posterior.restype = ctypes.c_int
        lib.oracle_scatter.argtypes = [ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                       ctypes.c_int32, ctypes.c_void_p]
        lib.oracle_scatter.restype = ctypes.c_int
        _lib = lib
    return _lib


def _as_struct(g, keep):
    def p(name, dtype):
        a = np.ascontiguousarray(g[name], dtype=dtype)
        keep.append(a)
        return a.ctypes.data
    s = _Graph()
    s.num_states = int(g["num_states"])
    s.num_arcs = int(len(g["src"]))
    s.arc_offset = p("arc_offset", np.int32)
    s.src = p("src", np.int32)
    s.dst = p("dst", np.int32)
    s.ilabel = p("ilabel", np.int32)
    s.olabel = p("olabel", np.int32)
    s.weight = p("weight", np.float32)
    s.start = p("start", np.uint8)
    s.accept = p("accept", np.uint8)
    return s


def _copy(ptr, n, dtype):
    if n == 0 or not ptr:
        return np.zeros(0, dtype=dtype)
    ct = np.ctypeslib.as_ctypes_type(np.dtype(dtype))
    buf = (ct * n).from_address(ptr)
    return np.array(np.ctypeslib.as_array(buf), dtype=dtype, copy=True)


def in_csr(num_states, dst):
    """Incoming-arc index of Section 3.2: (inArcOffset[V+1], inArcs[E])."""
    lib = _load()
    dst = np.ascontiguousarray(dst, dtype=np.int32)
    off = np.zeros(num_states + 1, np.int32)
    arcs = np.zeros(len(dst), np.int32)
    rc = lib.oracle_in_csr(num_states, len(dst), dst.ctypes.data, off.ctypes.data,
                           arcs.ctypes.data)
    if rc:
        raise ValueError("oracle_in_csr: " + _ERRORS.get(rc, str(rc)))
    return off, arcs


def compose_raw(A, B, order=ORDER_PAPER, mutation=MUT_NONE):
    """Run the C oracle; states and arcs in discovery order."""
    lib = _load()
    keep = []
    ga, gb = _as_struct(A, keep), _as_struct(B, keep)
    res = _Result()
    rc = lib.oracle_compose(ctypes.byref(ga), ctypes.byref(gb), order, mutation, ctypes.byref(res))
    if rc:
        raise ValueError("oracle_compose: " + _ERRORS.get(rc, str(rc)))
    try:
        V, E = int(res.num_states), int(res.num_arcs)
        out = dict(
            num_states=V, num_arcs=E,
            key_a=_copy(res.key_a, V, np.int32), key_b=_copy(res.key_b, V, np.int32),
            key_f=_copy(res.key_f, V, np.uint8), start=_copy(res.start, V, np.uint8),
            accept=_copy(res.accept, V, np.uint8),
            src=_copy(res.arc_src, E, np.int32), dst=_copy(res.arc_dst, E, np.int32),
            ilabel=_copy(res.arc_ilabel, E, np.int32), olabel=_copy(res.arc_olabel, E, np.int32),
            weight=_copy(res.arc_weight, E, np.float32),
            arc_a=_copy(res.arc_a, E, np.int32), arc_b=_copy(res.arc_b, E, np.int32),
            stats=dict(accessible=int(res.accessible), coaccessible=int(res.coaccessible),
                       generated=int(res.generated), pairs_examined=int(res.pairs_examined),
                       compose_seconds=float(res.compose_seconds)),
        )
    finally:
        lib.oracle_free(ctypes.byref(res))
    return out


def canonicalize(raw, A):
    """Renumber states by key (qa, qb, f) and sort arcs by (src, l, a, b)."""
    V, E = raw["num_states"], raw["num_arcs"]
    order = np.lexsort((raw["key_f"], raw["key_b"], raw["key_a"]))
    new_id = np.empty(V, np.int64)
    new_id[order] = np.arange(V)
    src = new_id[raw["src"]] if E else np.zeros(0, np.int64)
    dst = new_id[raw["dst"]] if E else np.zeros(0, np.int64)
    a, b = raw["arc_a"].astype(np.int64), raw["arc_b"].astype(np.int64)
    big = np.int64(1) << 40
    olA = np.asarray(A["olabel"], dtype=np.int64)
    match = (a >= 0) & (b >= 0)
    lab = np.zeros(E, np.int64)
    lab[match] = olA[a[match]]
    ak = np.where(a >= 0, a, big)
    bk = np.where(b >= 0, b, big)
    aorder = np.lexsort((bk, ak, lab, src))
    off = np.zeros(V + 1, np.int32)
    if V:
        off[1:] = np.cumsum(np.bincount(src, minlength=V))
    return dict(
        num_states=V, num_arcs=E, arc_offset=off,
        src=src[aorder].astype(np.int32), dst=dst[aorder].astype(np.int32),
        ilabel=raw["ilabel"][aorder], olabel=raw["olabel"][aorder],
        weight=raw["weight"][aorder], arc_a=raw["arc_a"][aorder], arc_b=raw["arc_b"][aorder],
        start=raw["start"][order], accept=raw["accept"][order],
        key_a=raw["key_a"][order], key_b=raw["key_b"][order], key_f=raw["key_f"][order],
        stats=raw["stats"],
    )


def compose(A, B, order=ORDER_PAPER, mutation=MUT_NONE):
    """Canonical composed graph C = A o B (see module docstring)."""
    return canonicalize(compose_raw(A, B, order, mutation), A)


RESULT_KEYS = ("arc_offset", "src", "dst", "ilabel", "olabel", "weight", "arc_a", "arc_b",
               "start", "accept", "key_a", "key_b", "key_f")


def compose3_raw(A, B, D, mutation=MUT3_NONE):
    """Run the three-input C oracle; states and arcs in discovery order."""
    lib = _load()
    keep = []
    ga, gb, gd = _as_struct(A, keep), _as_struct(B, keep), _as_struct(D, keep)
    res = _Result3()
    rc = lib.oracle_compose3(ctypes.byref(ga), ctypes.byref(gb), ctypes.byref(gd), mutation,
                             ctypes.byref(res))
    if rc:
        raise ValueError("oracle_compose3: " + _ERRORS.get(rc, str(rc)))
    try:
        V, E = int(res.num_states), int(res.num_arcs)
        out = dict(
            num_states=V, num_arcs=E,
            key_a=_copy(res.key_a, V, np.int32), key_b=_copy(res.key_b, V, np.int32),
            key_d=_copy(res.key_d, V, np.int32), key_fab=_copy(res.key_fab, V, np.uint8),
            key_f=_copy(res.key_f, V, np.uint8), start=_copy(res.start, V, np.uint8),
            accept=_copy(res.accept, V, np.uint8),
            src=_copy(res.arc_src, E, np.int32), dst=_copy(res.arc_dst, E, np.int32),
            ilabel=_copy(res.arc_ilabel, E, np.int32), olabel=_copy(res.arc_olabel, E, np.int32),
            weight=_copy(res.arc_weight, E, np.float32),
            arc_a=_copy(res.arc_a, E, np.int32), arc_b=_copy(res.arc_b, E, np.int32),
            arc_d=_copy(res.arc_d, E, np.int32),
            stats=dict(accessible=int(res.accessible), generated=int(res.generated),
                       compose_seconds=float(res.compose_seconds)),
        )
    finally:
        lib.oracle_free3(ctypes.byref(res))
    return out


def canonicalize3(raw, A):
    """Renumber states by key (qa, qb, f1, qd, f2) and sort the arcs of each
    state by (l, a, b, d): l = olabel of the arc of A when arcs of A and B
    were matched, else 0; a missing arc (-1) last."""
    V, E = raw["num_states"], raw["num_arcs"]
    order = np.lexsort((raw["key_f"], raw["key_d"], raw["key_fab"], raw["key_b"], raw["key_a"]))
    new_id = np.empty(V, np.int64)
    new_id[order] = np.arange(V)
    src = new_id[raw["src"]] if E else np.zeros(0, np.int64)
    dst = new_id[raw["dst"]] if E else np.zeros(0, np.int64)
    big = np.int64(1) << 40

    def k(x):
        x = x.astype(np.int64)
        return np.where(x >= 0, x, big)

    a, b = raw["arc_a"].astype(np.int64), raw["arc_b"].astype(np.int64)
    match = (a >= 0) & (b >= 0)
    lab = np.zeros(E, np.int64)
    lab[match] = np.asarray(A["olabel"], dtype=np.int64)[a[match]]
    aorder = np.lexsort((k(raw["arc_d"]), k(raw["arc_b"]), k(raw["arc_a"]), lab, src))
    off = np.zeros(V + 1, np.int32)
    if V:
        off[1:] = np.cumsum(np.bincount(src, minlength=V))
    out = dict(num_states=V, num_arcs=E, arc_offset=off,
               src=src[aorder].astype(np.int32), dst=dst[aorder].astype(np.int32),
               start=raw["start"][order], accept=raw["accept"][order], stats=raw["stats"])
    for name in ("ilabel", "olabel", "weight", "arc_a", "arc_b", "arc_d"):
        out[name] = raw[name][aorder]
    for name in ("key_a", "key_b", "key_fab", "key_d", "key_f"):
        out[name] = raw[name][order]
    return out


def compose3(A, B, D, mutation=MUT3_NONE):
    """Canonical C = A o B o D, composed simultaneously (see compose3.c)."""
    return canonicalize3(compose3_raw(A, B, D, mutation), A)


RESULT3_KEYS = ("arc_offset", "src", "dst", "ilabel", "olabel", "weight", "arc_a", "arc_b",
                "arc_d", "start", "accept", "key_a", "key_b", "key_fab", "key_d", "key_f")


def _graph_of(G, keep):
    """A graph dict without labels (a score needs none) gets zero labels."""
    g = dict(G)
    E = len(g["src"])
    for k in ("ilabel", "olabel"):
        if k not in g:
            g[k] = np.zeros(E, np.int32)
    return _as_struct(g, keep)


def score(G, mutation=SMUT_NONE):
    """Forward and backward log-semiring scores of an acyclic graph.

    Returns dict(alpha[V], beta[V], total, total_bwd, longest): ``total`` is
    the log-add of alpha over accepting states, ``total_bwd`` that of beta
    over start states (equal up to rounding), ``longest`` the number of
    states on the longest path.  Raises CycleError for a cyclic graph."""
    lib = _load()
    keep = []
    g = _graph_of(G, keep)
    V = int(G["num_states"])
    alpha = np.zeros(V, np.float64)
    beta = np.zeros(V, np.float64)
    tf, tb = ctypes.c_double(), ctypes.c_double()
    longest = ctypes.c_int32()
    rc = lib.oracle_score(ctypes.byref(g), mutation, alpha.ctypes.data, beta.ctypes.data,
                          ctypes.byref(tf), ctypes.byref(tb), ctypes.byref(longest))
    if rc == 4:
        raise CycleError("oracle_score: graph has a cycle")
    if rc:
        raise ValueError("oracle_score: " + _ERRORS.get(rc, str(rc)))
    return dict(alpha=alpha, beta=beta, total=tf.value, total_bwd=tb.value,
                longest=int(longest.value))


def posterior(G, alpha, beta, total):
    """Arc posteriors exp(alpha[src] + w + beta[dst] - total) (float64)."""
    lib = _load()
    keep = []
    g = _graph_of(G, keep)
    alpha = np.ascontiguousarray(alpha, np.float64)
    beta = np.ascontiguousarray(beta, np.float64)
    out = np.zeros(len(G["src"]), np.float64)
    rc = lib.oracle_posterior(ctypes.byref(g), alpha.ctypes.data, beta.ctypes.data,
                              float(total), out.ctypes.data)
    if rc:
        raise ValueError("oracle_posterior: " + _ERRORS.get(rc, str(rc)))
    return out


def scatter(grad, idx, m):
    """out[i] = sum of grad[e] over e with idx[e] = i (idx -1 is skipped),
    summed in index order in float64."""
    lib = _load()
    grad = np.ascontiguousarray(grad, np.float64)
    idx = np.ascontiguousarray(idx, np.int32)
    out = np.zeros(int(m), np.float64)
    rc = lib.oracle_scatter(len(grad), grad.ctypes.data, idx.ctypes.data, int(m),
                            out.ctypes.data)
    if rc:
        raise ValueError("oracle_scatter: " + _ERRORS.get(rc, str(rc)))
    return out
