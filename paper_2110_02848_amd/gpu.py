"""Python binding of libfstcompose.so (argument marshalling only).

Every step of the composition runs in the library's HIP kernels; this module
only passes device pointers and the current HIP stream across the C ABI
declared in ``include/fst_compose.h``.  PyTorch supplies device memory and
streams.  There is no fallback: if the library is missing or cannot be loaded
the calls raise.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfstcompose.so")

FST_OK = 0
FST_ERR_INVALID_ARG = 1
FST_ERR_INVALID_GRAPH = 2
FST_ERR_TOO_LARGE = 3
FST_ERR_NOMEM = 4
FST_ERR_HIP = 5
FST_ERR_STATE = 6
FST_ERR_CYCLIC = 7
FST_ERR_NOT_CONVERGED = 8

FST_OPT_MAX_WORKSPACE = 1
FST_OPT_TIMING = 2
FST_OPT_LABEL_BUCKETS = 3
FST_OPT_CHAIN_DEPTH = 4
FST_OPT_COUNT_MOVES = 5
FST_OPT_ORDER = 6
FST_OPT_VALIDATE = 7
FST_OPT_LIST_CAPACITY = 8

FST_SCATTER_NOALLOC_MAX_TARGETS = 1 << 20

FST_ORDER_FORWARD_FIRST = 0
FST_ORDER_COACCESSIBLE_FIRST = 1
FST_ORDER_CONCURRENT = 2

PHASES = ("preprocess", "forward", "backward", "count", "fill")

# kernels timed one by one (enum fst_kernel): a composition's, then a score's
KERNELS = ("search_forward", "search_backward", "count", "fill")
SCORE_KERNELS = ("score_gen", "score_prep")
KERNELS3 = ("search3", "compact3")


class FstError(RuntimeError):
    def __init__(self, code, where):
        self.code = code
        super().__init__(f"{where}: {_strerror(code)} (code {code})")


class _Graph(ctypes.Structure):
    _fields_ = [("num_states", ctypes.c_int32), ("num_arcs", ctypes.c_int32),
                ("arc_offset", ctypes.c_void_p), ("src", ctypes.c_void_p),
                ("dst", ctypes.c_void_p), ("ilabel", ctypes.c_void_p),
                ("olabel", ctypes.c_void_p), ("weight", ctypes.c_void_p),
                ("start", ctypes.c_void_p), ("accept", ctypes.c_void_p)]


class _GraphOut(ctypes.Structure):
    _fields_ = [("arc_offset", ctypes.c_void_p), ("src", ctypes.c_void_p),
                ("dst", ctypes.c_void_p), ("ilabel", ctypes.c_void_p),
                ("olabel", ctypes.c_void_p), ("weight", ctypes.c_void_p),
                ("start", ctypes.c_void_p), ("accept", ctypes.c_void_p),
                ("key_a", ctypes.c_void_p), ("key_b", ctypes.c_void_p),
                ("key_f", ctypes.c_void_p), ("arc_a", ctypes.c_void_p),
                ("arc_b", ctypes.c_void_p)]


class _GraphOut3(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in (
        "arc_offset", "src", "dst", "ilabel", "olabel", "weight", "start", "accept", "key_a",
        "key_b", "key_fab", "key_d", "key_f", "arc_a", "arc_b", "arc_d")]


class _Stats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in (
        "key_space", "accessible", "coaccessible", "generated", "fwd_levels",
        "bwd_levels", "heavy_states", "num_states", "num_arcs", "generated_backward")]


_lib = None


def load():
    """Load the HIP library (raises if it was not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                           "or python -m paper_2110_02848_amd.build")
    lib = ctypes.CDLL(LIB_PATH)
    lib.fst_ctx_create.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_void_p)]
    lib.fst_ctx_create.restype = ctypes.c_int
    lib.fst_ctx_destroy.argtypes = [ctypes.c_void_p]
    lib.fst_ctx_destroy.restype = None
    lib.fst_ctx_set_option.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int64]
    lib.fst_ctx_set_option.restype = ctypes.c_int
    lib.fst_compose_run.argtypes = [ctypes.c_void_p, ctypes.POINTER(_Graph),
                                    ctypes.POINTER(_Graph), ctypes.c_void_p,
                                    ctypes.POINTER(ctypes.c_int64),
                                    ctypes.POINTER(ctypes.c_int64)]
    lib.fst_compose_run.restype = ctypes.c_int
    lib.fst_compose_fill.argtypes = [ctypes.c_void_p, ctypes.POINTER(_GraphOut), ctypes.c_void_p]
    lib.fst_compose_fill.restype = ctypes.c_int
    lib.fst_compose_stats.argtypes = [ctypes.c_void_p, ctypes.POINTER(_Stats)]
    lib.fst_compose_stats.restype = ctypes.c_int
    lib.fst_compose_phase_times.argtypes = [ctypes.c_void_p, ctypes.POINTER(ctypes.c_float),
                                            ctypes.c_int]
    lib.fst_compose_phase_times.restype = ctypes.c_int
    lib.fst_compose_kernel_time.argtypes = [ctypes.c_void_p, ctypes.c_int,
                                            ctypes.POINTER(ctypes.c_float),
                                            ctypes.POINTER(ctypes.c_int64)]
    lib.fst_compose_kernel_time.restype = ctypes.c_int
    lib.fst_score.argtypes = [ctypes.c_void_p, ctypes.POINTER(_Graph), ctypes.c_void_p,
                              ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    lib.fst_score.restype = ctypes.c_int
    lib.fst_score_cyclic.argtypes = [ctypes.c_void_p, ctypes.POINTER(_Graph), ctypes.c_void_p,
                                     ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                     ctypes.c_double, ctypes.POINTER(ctypes.c_int32),
                                     ctypes.c_void_p]
    lib.fst_score_cyclic.restype = ctypes.c_int
    lib.fst_score_posterior.argtypes = [ctypes.c_void_p, ctypes.POINTER(_Graph),
                                        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p]
    lib.fst_score_posterior.restype = ctypes.c_int
    lib.fst_grad_scatter.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                     ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
                                     ctypes.c_void_p]
    lib.fst_grad_scatter.restype = ctypes.c_int
    lib.fst_grad_scatter_noalloc.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                             ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
                                             ctypes.c_void_p]
    lib.fst_grad_scatter_noalloc.restype = ctypes.c_int
    lib.fst_compose_batch_run.argtypes = [ctypes.c_void_p, ctypes.POINTER(_Graph), ctypes.c_int32,
                                          ctypes.POINTER(_Graph), ctypes.c_void_p,
                                          ctypes.POINTER(ctypes.c_int64),
                                          ctypes.POINTER(ctypes.c_int64), ctypes.c_void_p,
                                          ctypes.c_void_p]
    lib.fst_compose_batch_run.restype = ctypes.c_int
    lib.fst_segment_logsum.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                       ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                       ctypes.c_void_p]
    lib.fst_segment_logsum.restype = ctypes.c_int
    lib.fst_compose3_run.argtypes = [ctypes.c_void_p, ctypes.POINTER(_Graph),
                                     ctypes.POINTER(_Graph), ctypes.POINTER(_Graph),
                                     ctypes.c_void_p, ctypes.POINTER(ctypes.c_int64),
                                     ctypes.POINTER(ctypes.c_int64)]
    lib.fst_compose3_run.restype = ctypes.c_int
    lib.fst_compose3_fill.argtypes = [ctypes.c_void_p, ctypes.POINTER(_GraphOut3),
                                      ctypes.c_void_p]
    lib.fst_compose3_fill.restype = ctypes.c_int
    lib.fst_compose3_stats.argtypes = [ctypes.c_void_p, ctypes.POINTER(_Stats)]
    lib.fst_compose3_stats.restype = ctypes.c_int
    lib.fst_strerror.argtypes = [ctypes.c_int]
    lib.fst_strerror.restype = ctypes.c_char_p
    _lib = lib
    return lib


def _strerror(code):
    try:
        return load().fst_strerror(code).decode()
    except Exception:  # pragma: no cover - message only
        return "error"


def _check(rc, where):
    if rc != FST_OK:
        raise FstError(rc, where)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr() if t is not None and t.numel() else None)


def _stream_handle(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


GRAPH_DTYPES = dict(arc_offset=np.int32, src=np.int32, dst=np.int32, ilabel=np.int32,
                    olabel=np.int32, weight=np.float32, start=np.uint8, accept=np.uint8)


def to_device(g, device="cuda:0"):
    """Copy a numpy graph dict to device tensors (dict with the same keys)."""
    import torch
    out = {"num_states": int(g["num_states"])}
    for k, dt in GRAPH_DTYPES.items():
        out[k] = torch.from_numpy(np.ascontiguousarray(g[k], dtype=dt)).to(device)
    return out


def _graph_struct(g):
    s = _Graph()
    s.num_states = int(g["num_states"])
    s.num_arcs = int(g["src"].numel())
    for k in GRAPH_DTYPES:
        setattr(s, k, _ptr(g[k]))
    return s


class Composer:
    """Owns one library context on one device (reuse it across calls)."""

    def __init__(self, device=0):
        self._lib = load()
        self.device = int(device)
        h = ctypes.c_void_p()
        _check(self._lib.fst_ctx_create(self.device, ctypes.byref(h)), "fst_ctx_create")
        self._h = h
        self.options = {}  # options set on this context (option -> value)

    def close(self):
        if getattr(self, "_h", None):
            self._lib.fst_ctx_destroy(self._h)
            self._h = None

    def __del__(self):  # pragma: no cover - interpreter shutdown order
        try:
            self.close()
        except Exception:
            pass

    def set_option(self, option, value):
        _check(self._lib.fst_ctx_set_option(self._h, option, int(value)), "fst_ctx_set_option")
        self.options[option] = int(value)

    def run(self, A, B, stream=None):
        """Phase 1: search, trim, number and count.  Returns (V_C, E_C)."""
        ga, gb = _graph_struct(A), _graph_struct(B)
        nv, ne = ctypes.c_int64(), ctypes.c_int64()
        rc = self._lib.fst_compose_run(self._h, ctypes.byref(ga), ctypes.byref(gb),
                                       _stream_handle(stream), ctypes.byref(nv), ctypes.byref(ne))
        _check(rc, "fst_compose_run")
        return int(nv.value), int(ne.value)

    def alloc_output(self, nv, ne, provenance=True, keys=True):
        import torch
        dev = f"cuda:{self.device}"
        i32 = dict(dtype=torch.int32, device=dev)
        u8 = dict(dtype=torch.uint8, device=dev)
        C = dict(num_states=nv, num_arcs=ne,
                 arc_offset=torch.empty(nv + 1, **i32),
                 src=torch.empty(ne, **i32), dst=torch.empty(ne, **i32),
                 ilabel=torch.empty(ne, **i32), olabel=torch.empty(ne, **i32),
                 weight=torch.empty(ne, dtype=torch.float32, device=dev),
                 start=torch.empty(nv, **u8), accept=torch.empty(nv, **u8))
        if keys:
            C.update(key_a=torch.empty(nv, **i32), key_b=torch.empty(nv, **i32),
                     key_f=torch.empty(nv, **u8))
        if provenance:
            C.update(arc_a=torch.empty(ne, **i32), arc_b=torch.empty(ne, **i32))
        return C

    def fill(self, C, stream=None):
        """Phase 2: write C into the tensors of ``alloc_output`` (async)."""
        o = _GraphOut()
        o.arc_offset = ctypes.c_void_p(C["arc_offset"].data_ptr())
        for k in ("src", "dst", "ilabel", "olabel", "weight", "start", "accept",
                  "key_a", "key_b", "key_f", "arc_a", "arc_b"):
            setattr(o, k, _ptr(C.get(k)))
        _check(self._lib.fst_compose_fill(self._h, ctypes.byref(o), _stream_handle(stream)),
               "fst_compose_fill")
        return C

    def compose(self, A, B, provenance=True, keys=True, stream=None):
        """C = A o B as a dict of device tensors (asynchronous fill)."""
        nv, ne = self.run(A, B, stream)
        C = self.alloc_output(nv, ne, provenance, keys)
        return self.fill(C, stream)

    def run_batch(self, As, B, stream=None):
        """Phase 1 of C_i = A_i o B for every A_i of the list, in one pass.
        Returns (V_C, E_C, item_states, item_arcs): the sizes of the one C
        (the union of the C_i) and the numpy int64 [n + 1] ranges of each
        item's states and arcs in it."""
        n = len(As)
        arr = (_Graph * max(n, 1))()
        for i, A in enumerate(As):
            arr[i] = _graph_struct(A)
        gb = _graph_struct(B)
        nv, ne = ctypes.c_int64(), ctypes.c_int64()
        st = np.zeros(n + 1, np.int64)
        ar = np.zeros(n + 1, np.int64)
        rc = self._lib.fst_compose_batch_run(self._h, arr, n, ctypes.byref(gb),
                                             _stream_handle(stream), ctypes.byref(nv),
                                             ctypes.byref(ne), st.ctypes.data, ar.ctypes.data)
        _check(rc, "fst_compose_batch_run")
        return int(nv.value), int(ne.value), st, ar

    def compose_batch(self, As, B, provenance=True, keys=True, stream=None):
        """C = union of A_i o B as one dict of device tensors (ids of the
        union), with the per-item ranges: (C, item_states, item_arcs)."""
        nv, ne, st, ar = self.run_batch(As, B, stream)
        C = self.alloc_output(nv, ne, provenance, keys)
        return self.fill(C, stream), st, ar

    def segment_logsum(self, val, flag, bounds, stream=None):
        """totals[i] = log-sum of exp(val[v]) over flagged v in
        [bounds[i], bounds[i + 1]) (float64 [n] tensor)."""
        import torch
        b = np.ascontiguousarray(bounds, dtype=np.int64)
        n = len(b) - 1
        out = torch.empty(max(n, 0), dtype=torch.float64, device=f"cuda:{self.device}")
        rc = self._lib.fst_segment_logsum(self._h, _ptr(val), _ptr(flag), n, b.ctypes.data,
                                          _ptr(out), _stream_handle(stream))
        _check(rc, "fst_segment_logsum")
        return out

    def stats(self):
        st = _Stats()
        _check(self._lib.fst_compose_stats(self._h, ctypes.byref(st)), "fst_compose_stats")
        return {n: int(getattr(st, n)) for n, _ in _Stats._fields_}

    def phase_times(self):
        buf = (ctypes.c_float * len(PHASES))()
        _check(self._lib.fst_compose_phase_times(self._h, buf, len(PHASES)),
               "fst_compose_phase_times")
        return dict(zip(PHASES, [float(x) for x in buf]))

    def kernel_times(self):
        """{kernel: (ms, launches)} of the last timed run + fill."""
        out = {}
        for i, name in enumerate(KERNELS):
            ms, n = ctypes.c_float(), ctypes.c_int64()
            _check(self._lib.fst_compose_kernel_time(self._h, i, ctypes.byref(ms), ctypes.byref(n)),
                   "fst_compose_kernel_time")
            out[name] = (float(ms.value), int(n.value))
        return out


    # ---- three inputs at once: C = A o B o D ----

    def run3(self, A, B, D, stream=None):
        """Phase 1 of C = A o B o D.  Returns (V_C, E_C)."""
        ga, gb, gd = _graph_struct(A), _graph_struct(B), _graph_struct(D)
        nv, ne = ctypes.c_int64(), ctypes.c_int64()
        rc = self._lib.fst_compose3_run(self._h, ctypes.byref(ga), ctypes.byref(gb),
                                        ctypes.byref(gd), _stream_handle(stream),
                                        ctypes.byref(nv), ctypes.byref(ne))
        _check(rc, "fst_compose3_run")
        return int(nv.value), int(ne.value)

    def alloc_output3(self, nv, ne, provenance=True, keys=True):
        import torch
        C = self.alloc_output(nv, ne, provenance=provenance, keys=keys)
        dev = f"cuda:{self.device}"
        if keys:
            C.update(key_fab=torch.empty(nv, dtype=torch.uint8, device=dev),
                     key_d=torch.empty(nv, dtype=torch.int32, device=dev))
        if provenance:
            C["arc_d"] = torch.empty(ne, dtype=torch.int32, device=dev)
        return C

    def fill3(self, C, stream=None):
        o = _GraphOut3()
        for k, _ in _GraphOut3._fields_:
            setattr(o, k, _ptr(C.get(k)))
        o.arc_offset = ctypes.c_void_p(C["arc_offset"].data_ptr())
        _check(self._lib.fst_compose3_fill(self._h, ctypes.byref(o), _stream_handle(stream)),
               "fst_compose3_fill")
        return C

    def compose3(self, A, B, D, provenance=True, keys=True, stream=None):
        """C = A o B o D (composed at once) as a dict of device tensors."""
        nv, ne = self.run3(A, B, D, stream)
        C = self.alloc_output3(nv, ne, provenance, keys)
        return self.fill3(C, stream)

    def stats3(self):
        st = _Stats()
        _check(self._lib.fst_compose3_stats(self._h, ctypes.byref(st)), "fst_compose3_stats")
        return {n: int(getattr(st, n)) for n, _ in _Stats._fields_}

    def kernel_times3(self):
        """{kernel: (ms, launches)} of the last timed fst_compose3_run + fill."""
        out = {}
        for i, name in enumerate(KERNELS3):
            ms, n = ctypes.c_float(), ctypes.c_int64()
            _check(self._lib.fst_compose_kernel_time(self._h, 6 + i, ctypes.byref(ms),
                                                     ctypes.byref(n)),
                   "fst_compose_kernel_time")
            out[name] = (float(ms.value), int(n.value))
        return out

    # ---- scores of an acyclic graph and their gradient ----

    def score(self, G, alpha=True, beta=True, stream=None):
        """Forward / backward log-semiring scores of an acyclic graph of
        device tensors: dict(alpha, beta: float64 [V] tensors or None, total:
        float64 [1] tensor).  Raises FstError(FST_ERR_CYCLIC) on a cycle."""
        import torch
        dev = f"cuda:{self.device}"
        V = int(G["num_states"])
        a = torch.empty(V, dtype=torch.float64, device=dev) if alpha else None
        b = torch.empty(V, dtype=torch.float64, device=dev) if beta else None
        total = torch.empty(1, dtype=torch.float64, device=dev)
        g = _graph_struct(G)
        rc = self._lib.fst_score(self._h, ctypes.byref(g), _ptr(a), _ptr(b),
                                 ctypes.c_void_p(total.data_ptr()), _stream_handle(stream))
        _check(rc, "fst_score")
        return dict(alpha=a, beta=b, total=total)

    def score_cyclic(self, G, alpha=True, beta=True, max_sweeps=10000, tol=0.0, stream=None):
        """The same scores of a graph that may have cycles, by relaxation
        sweeps: dict(alpha, beta, total as in ``score``, sweeps: the number
        of sweeps until none raised a value by more than ``tol``).  Raises
        FstError(FST_ERR_NOT_CONVERGED) if that took more than max_sweeps."""
        import torch
        dev = f"cuda:{self.device}"
        V = int(G["num_states"])
        a = torch.empty(V, dtype=torch.float64, device=dev) if alpha else None
        b = torch.empty(V, dtype=torch.float64, device=dev) if beta else None
        total = torch.empty(1, dtype=torch.float64, device=dev)
        n = ctypes.c_int32(0)
        g = _graph_struct(G)
        rc = self._lib.fst_score_cyclic(self._h, ctypes.byref(g), _ptr(a), _ptr(b),
                                        ctypes.c_void_p(total.data_ptr()), int(max_sweeps),
                                        float(tol), ctypes.byref(n), _stream_handle(stream))
        _check(rc, "fst_score_cyclic")
        return dict(alpha=a, beta=b, total=total, sweeps=int(n.value))

    def posterior(self, G, alpha, beta, total, scale=1.0, stream=None):
        """scale * d total / d w for every arc (float32 [E] tensor)."""
        import torch
        grad = torch.empty(int(G["src"].numel()), dtype=torch.float32,
                           device=f"cuda:{self.device}")
        g = _graph_struct(G)
        rc = self._lib.fst_score_posterior(self._h, ctypes.byref(g), _ptr(alpha), _ptr(beta),
                                           ctypes.c_void_p(total.data_ptr()), float(scale),
                                           _ptr(grad), _stream_handle(stream))
        _check(rc, "fst_score_posterior")
        return grad

    def grad_scatter(self, grad, idx, m, stream=None):
        """out[i] = sum of grad[e] over idx[e] = i (float32 [m] tensor)."""
        import torch
        out = torch.empty(int(m), dtype=torch.float32, device=f"cuda:{self.device}")
        rc = self._lib.fst_grad_scatter(self._h, int(grad.numel()), _ptr(grad), _ptr(idx),
                                        int(m), _ptr(out), _stream_handle(stream))
        _check(rc, "fst_grad_scatter")
        return out

    def grad_scatter_noalloc(self, grad, idx, m, out=None, stream=None):
        """grad_scatter through the entry point that allocates no device
        memory (m <= FST_SCATTER_NOALLOC_MAX_TARGETS); ``out`` (float32 [m])
        may be passed in, so that the call itself allocates nothing."""
        import torch
        if out is None:
            out = torch.empty(int(m), dtype=torch.float32, device=f"cuda:{self.device}")
        rc = self._lib.fst_grad_scatter_noalloc(self._h, int(grad.numel()), _ptr(grad), _ptr(idx),
                                                int(m), _ptr(out), _stream_handle(stream))
        _check(rc, "fst_grad_scatter_noalloc")
        return out

    def operand_grads(self, C, A_arcs, B_arcs, scale=1.0, stream=None):
        """Gradient of scale * total(C) by the arc weights of A and B (C
        filled with provenance): (grad_A [A_arcs], grad_B [B_arcs])."""
        sc = self.score(C, stream=stream)
        post = self.posterior(C, sc["alpha"], sc["beta"], sc["total"], scale, stream)
        return (self.grad_scatter(post, C["arc_a"], A_arcs, stream),
                self.grad_scatter(post, C["arc_b"], B_arcs, stream))

    def score_kernel_times(self):
        """{kernel: (ms, launches)} of the last timed fst_score."""
        out = {}
        for i, name in enumerate(SCORE_KERNELS):
            ms, n = ctypes.c_float(), ctypes.c_int64()
            _check(self._lib.fst_compose_kernel_time(self._h, len(KERNELS) + i, ctypes.byref(ms),
                                                     ctypes.byref(n)),
                   "fst_compose_kernel_time")
            out[name] = (float(ms.value), int(n.value))
        return out


def to_numpy(C):
    """Device result dict -> numpy dict (synchronises)."""
    out = {}
    for k, v in C.items():
        out[k] = v.cpu().numpy() if hasattr(v, "cpu") else v
    return out


def compose_numpy(A, B, device=0, composer=None):
    """Convenience: numpy graphs in, numpy canonical C out (via the GPU)."""
    comp = composer or Composer(device)
    dev = f"cuda:{comp.device}"
    C = comp.compose(to_device(A, dev), to_device(B, dev))
    return to_numpy(C)
