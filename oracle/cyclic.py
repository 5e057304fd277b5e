"""Log-semiring scores of a graph that may have cycles (test infrastructure
only: only ``tests/`` may import it; it shares nothing with the GPU library).

The scores are those of ``oracle.score`` (``score.c``), the sums over all
paths of the log semiring of Eq. (1), now over graphs with cycles, where a
state can have infinitely many paths:

* alpha[v] = log-sum over the paths from any start state to v of their
  weight (a start state's empty path weighs 0);
* beta[v]  = log-sum over the paths from v to any accepting state (an
  accepting state's empty path weighs 0);
* total    = log-sum over the paths from a start state to an accepting state;
* an empty sum is -inf.

Written out in the probability domain with M[u, v] = sum of exp(w(e)) over
the arcs e from u to v, s the start indicator and f the accepting one, the
sums over paths of every length k are the Neumann series

    a = sum_k s M^k = s (I - M)^-1,      b = sum_k M^k f = (I - M)^-1 f,

and alpha = log a, beta = log b, total = log(a . f).  Only states that a
start state reaches have paths from one (the others' alpha is -inf), so a is
solved over those states alone, and b over the states that reach an
accepting state.  The series converge exactly when the spectral radius of
that part of M is below 1; for a nonnegative M that is when I - M is
invertible with a nonnegative inverse, so a solve that is singular or has a
component that is not positive means the sums diverge (DivergeError): over
states that s reaches, a positive a with a (I - M) = s >= 0 bounds the
spectral radius of every strongly connected part below 1, since each such
part takes flow from s or from an earlier part.
The solves are float64 LU (numpy), dense: for graphs of a few thousand
states.
"""
from __future__ import annotations

import numpy as np


class DivergeError(ValueError):
    """The path sums of the graph do not converge."""


def _reach(V, frm, to, seeds):
    seen = np.zeros(V, bool)
    adj = [[] for _ in range(V)]
    for u, v in zip(frm, to):
        adj[int(u)].append(int(v))
    stack = [int(s) for s in np.flatnonzero(seeds)]
    for s in stack:
        seen[s] = True
    while stack:
        u = stack.pop()
        for v in adj[u]:
            if not seen[v]:
                seen[v] = True
                stack.append(v)
    return seen


def _arcs(G):
    V = int(G["num_states"])
    off = np.asarray(G["arc_offset"], np.int64)
    src = np.repeat(np.arange(V), np.diff(off))
    dst = np.asarray(G["dst"], np.int64)
    w = np.asarray(G["weight"], np.float32).astype(np.float64)
    return V, src, dst, w


def _solve(M, rhs, transpose):
    """x with x (I - M) = rhs (transpose) or (I - M) x = rhs."""
    n = M.shape[0]
    A = np.eye(n) - M
    try:
        x = np.linalg.solve(A.T if transpose else A, rhs)
    except np.linalg.LinAlgError as e:
        raise DivergeError("path sums diverge: I - M is singular") from e
    if not np.all(np.isfinite(x)) or np.any(x <= 0.0):
        raise DivergeError("path sums diverge: spectral radius of M is at least 1")
    return x


def score_cyclic(G):
    """dict(alpha[V], beta[V], total) of a graph that may have cycles;
    raises DivergeError when its path sums do not converge."""
    V, src, dst, w = _arcs(G)
    return scores_of(V, src, dst, w, np.asarray(G["start"], np.uint8) != 0,
                     np.asarray(G["accept"], np.uint8) != 0)


def scores_of(V, src, dst, w, start, accept):
    """The same from arc arrays with float64 weights w (arc e from src[e]
    to dst[e]) and boolean start / accept arrays."""
    alpha = np.full(V, -np.inf)
    beta = np.full(V, -np.inf)
    acc = _reach(V, src, dst, start)
    coacc = _reach(V, dst, src, accept)
    ia = np.flatnonzero(acc)
    if len(ia):
        pos = -np.ones(V, np.int64)
        pos[ia] = np.arange(len(ia))
        M = np.zeros((len(ia), len(ia)))
        keep = acc[src]  # an arc out of a reached state reaches a reached state
        np.add.at(M, (pos[src[keep]], pos[dst[keep]]), np.exp(w[keep]))
        alpha[ia] = np.log(_solve(M, start[ia].astype(np.float64), transpose=True))
    ic = np.flatnonzero(coacc)
    if len(ic):
        pos = -np.ones(V, np.int64)
        pos[ic] = np.arange(len(ic))
        M = np.zeros((len(ic), len(ic)))
        keep = coacc[dst]  # an arc into a co-accessible state leaves one
        np.add.at(M, (pos[src[keep]], pos[dst[keep]]), np.exp(w[keep]))
        beta[ic] = np.log(_solve(M, accept[ic].astype(np.float64), transpose=False))
    fin = accept & acc
    total = -np.inf
    if fin.any():
        m = float(np.max(alpha[fin]))
        total = m + float(np.log(np.sum(np.exp(alpha[fin] - m))))
    return dict(alpha=alpha, beta=beta, total=total)
