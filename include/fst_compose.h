/*
 * fst_compose.h -- C ABI of the MI355X (gfx950) eager transducer composition
 * library, libfstcompose.so.
 *
 * Operation (paper "Parallel Composition of Weighted Finite-State
 * Transducers", Section 3.1, Eq. (1) and Algorithm 1): given weighted
 * transducers A and B in the log semiring, build the trim composed transducer
 * C = A o B, which maps an input string x to an output string z with score
 * log-sum over y of exp(A(x, y) + B(y, z)).  Arcs of A are matched on their
 * output label and arcs of B on their input label.  Label 0 is epsilon.
 *
 * States of C are keys (qa, qb, f): a state of A, a state of B and one filter
 * bit.  From (qa, qb, f) there are three moves:
 *   matching move : arcs ea of qa, eb of qb with olabel(ea) = ilabel(eb) != 0
 *                   -> (dst(ea), dst(eb), 0); label ilabel(ea):olabel(eb);
 *                   weight = w(ea) + w(eb), one IEEE binary32 add (RNE)
 *   A-epsilon move: only when f = 0; arc ea with olabel(ea) = 0
 *                   -> (dst(ea), qb, 0); label ilabel(ea):0; weight w(ea)
 *   B-epsilon move: arc eb with ilabel(eb) = 0
 *                   -> (qa, dst(eb), epsOutA(qa)); label 0:olabel(eb); weight w(eb)
 * where epsOutA(q) says whether q has an out-arc with output label 0.  (The
 * filter bit keeps A's epsilon moves ahead of B's between two matching moves,
 * so each pair of paths of A and B maps to exactly one path of C.)  Start
 * keys are (sa, sb, 0) over start states of A and B.  A key accepts iff both
 * of its states accept.  C keeps only keys reachable from a start key that
 * can reach an accepting key (Section 3.1: the composed graph is trim).
 * Parallel arcs are kept; no weights are summed.
 *
 * Output is canonical and deterministic: states are numbered in ascending
 * key order (qa, qb, f); the arcs of a state are ordered by (l, a, b), where
 * l is the matched label (0 for epsilon moves), a and b are the arcs of A and
 * B the arc came from, and a missing arc sorts last.
 *
 * Graph layout (Section 3.2: structure of arrays, arcs consecutive by node,
 * offsets with V+1 entries).  All pointers passed to the library are DEVICE
 * pointers (hipMalloc or torch CUDA/HIP tensors) on the context's device.
 *
 * Errors: every entry point returns an int status (FST_OK = 0).  Nothing
 * aborts or throws across this interface.
 */
#ifndef FST_COMPOSE_H
#define FST_COMPOSE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__) || defined(__clang__)
#define FST_API __attribute__((visibility("default")))
#else
#define FST_API
#endif

#define FST_EPS 0

enum fst_status {
  FST_OK = 0,
  FST_ERR_INVALID_ARG = 1,   /* null pointer, negative size, bad option      */
  FST_ERR_INVALID_GRAPH = 2, /* input failed validation (see fst_graph)      */
  FST_ERR_TOO_LARGE = 3,     /* key space > 2^32 keys, or |C| > INT32_MAX    */
  FST_ERR_NOMEM = 4,         /* device allocation failed or over the cap     */
  FST_ERR_HIP = 5,           /* a HIP runtime call failed                    */
  FST_ERR_STATE = 6,         /* fill without a successful run               */
  FST_ERR_CYCLIC = 7,        /* fst_score on a graph with a cycle            */
  FST_ERR_NOT_CONVERGED = 8  /* fst_score_cyclic: sweeps did not settle      */
};

/* Read-only transducer view (device memory, caller-owned).
 *   num_states V >= 0, num_arcs E >= 0
 *   arc_offset[V+1]  arcs of state v are [arc_offset[v], arc_offset[v+1]);
 *                    arc_offset[0] = 0, arc_offset[V] = E, non-decreasing
 *   src[E], dst[E]   source / destination state; src consistent with offsets
 *   ilabel[E], olabel[E]  labels >= 0, 0 = epsilon
 *   weight[E]        binary32 log weights (any value, not checked)
 *   start[V], accept[V]   0 or 1; any number of start states
 * Every run validates these rules (unless FST_OPT_VALIDATE is 0) and
 * returns FST_ERR_INVALID_GRAPH on a violation.  Pointers may be NULL only
 * when the array is empty. */
typedef struct {
  int32_t num_states, num_arcs;
  const int32_t *arc_offset;
  const int32_t *src, *dst;
  const int32_t *ilabel, *olabel;
  const float *weight;
  const uint8_t *start, *accept;
} fst_graph;

/* Caller-allocated output arrays (device memory), sized from the V_C and
 * E_C that fst_compose_run reported.
 *   arc_offset[V_C+1]; src, dst, ilabel, olabel, weight [E_C];
 *   start, accept [V_C];
 *   key_a, key_b, key_f [V_C]  optional (NULL skips): the key of each state;
 *   arc_a, arc_b [E_C]         optional (NULL skips): provenance, the arc of
 *                              A / of B each arc of C came from, -1 if none. */
typedef struct {
  int32_t *arc_offset;
  int32_t *src, *dst, *ilabel, *olabel;
  float *weight;
  uint8_t *start, *accept;
  int32_t *key_a, *key_b;
  uint8_t *key_f;
  int32_t *arc_a, *arc_b;
} fst_graph_out;

/* Statistics of the last successful run. */
typedef struct {
  int64_t key_space;     /* key slots: V_A x 2^(b+1), b = max(4, bits(V_B-1)) */
  int64_t accessible;    /* keys reached from the start keys                 */
  int64_t coaccessible;  /* accessible keys that reach an accepting key = V_C */
  int64_t generated;     /* moves out of accessible keys; -1 unless
                            FST_OPT_COUNT_MOVES was set                      */
  int64_t fwd_levels;    /* frontier generations of the forward search       */
  int64_t bwd_levels;    /* frontier generations of the backward search      */
  int64_t heavy_states;  /* states of C handled one workgroup per state      */
  int64_t num_states;    /* V_C                                              */
  int64_t num_arcs;      /* E_C                                              */
  int64_t generated_backward; /* predecessor moves of the co-accessible keys
                            (each probed once by the backward search); -1
                            unless FST_OPT_COUNT_MOVES was set               */
} fst_stats;

typedef struct fst_ctx fst_ctx;

/* Create a context on HIP device `device`.  The context owns a device
 * workspace that grows on demand and is reused across calls.  A context is
 * not thread-safe: use one per host thread / stream.  *ctx is set on success. */
FST_API int fst_ctx_create(int device, fst_ctx **ctx);

/* Release the context and its workspace (NULL is allowed). */
FST_API void fst_ctx_destroy(fst_ctx *ctx);

/* Options: FST_OPT_MAX_WORKSPACE caps the workspace in bytes (0 = no cap;
 * exceeding it gives FST_ERR_NOMEM); FST_OPT_TIMING = 1 records per-phase
 * HIP events (read with fst_compose_phase_times).  Tuning knobs that never
 * change the result: FST_OPT_LABEL_BUCKETS (1 = default: per-state label
 * bucket tables for a graph whose table fits in 256 MiB and in 64 times its
 * arc records (8 bytes per arc); 0 = binary search only) and
 * FST_OPT_CHAIN_DEPTH (default 64: how many newly found keys one search
 * thread may expand depth-first before handing keys to the next frontier;
 * 0 = plain frontier-by-frontier search).  FST_OPT_COUNT_MOVES = 1 makes
 * each run also count the moves out of all accessible keys and the
 * predecessor moves of all co-accessible keys (extra passes, reported in
 * fst_stats.generated and fst_stats.generated_backward).
 * FST_OPT_ORDER picks the order of the two searches (the result is the same):
 * FST_ORDER_FORWARD_FIRST searches forward from the start keys,
 * then backward from the accepting keys it reached, inside the accessible
 * set; FST_ORDER_COACCESSIBLE_FIRST is Algorithm 1's order: the co-accessible
 * set over all key pairs first (backward from every accepting pair), then the
 * forward search inside it (fst_stats.accessible then counts only keys that
 * are also co-accessible); FST_ORDER_CONCURRENT (default) runs the forward
 * search's first generations alone, then, unless it has ended (then it goes
 * on as forward-first), a backward search from every accepting pair beside
 * the rest of it in the same kernels, restricted to accessible keys once
 * the forward search has ended and held back while its frontier is far
 * wider than the forward one (kernel FST_KERNEL_SEARCH_FORWARD then times
 * the launches that advance either search, and FST_KERNEL_SEARCH_BACKWARD
 * has none).  FST_OPT_VALIDATE (default 1) checks every input graph's
 * structure as described at fst_graph; 0 is for callers that vouch for
 * their graphs: the checks are skipped (the composition still reads the
 * largest label, the label order and the accepting states; a score reads
 * nothing before it starts), and a graph that breaks the rules then gives
 * unspecified results, which may include reads outside its arrays.
 * FST_OPT_LIST_CAPACITY (entries, 0 = default 2^22) is the first size of
 * the search's work lists (frontier, heavy and accepting keys); a search
 * that overflows them runs again with four times the size (never more than
 * 2 V_A V_B), and the context keeps the size that sufficed for later calls;
 * the result is the same. */
enum fst_option {
  FST_OPT_MAX_WORKSPACE = 1,
  FST_OPT_TIMING = 2,
  FST_OPT_LABEL_BUCKETS = 3,
  FST_OPT_CHAIN_DEPTH = 4,
  FST_OPT_COUNT_MOVES = 5,
  FST_OPT_ORDER = 6,
  FST_OPT_VALIDATE = 7,
  FST_OPT_LIST_CAPACITY = 8
};
enum fst_order {
  FST_ORDER_FORWARD_FIRST = 0,
  FST_ORDER_COACCESSIBLE_FIRST = 1,
  FST_ORDER_CONCURRENT = 2
};
FST_API int fst_ctx_set_option(fst_ctx *ctx, int option, int64_t value);

/* Phase 1 (Algorithm 1 up to the size of C): validate A and B, search the
 * state pairs reachable from the start keys, prune to co-accessible ones,
 * number the kept states and count their arcs.  Work is queued on `stream`
 * (a hipStream_t; NULL = default stream); the call blocks until the sizes are
 * known and stores them in *num_states (V_C) and *num_arcs (E_C).  A and B
 * must stay valid and unchanged until fst_compose_fill's work has completed.
 * An empty C (V_C = 0) is a valid result. */
FST_API int fst_compose_run(fst_ctx *ctx, const fst_graph *A, const fst_graph *B, void *stream,
                    int64_t *num_states, int64_t *num_arcs);

/* Phase 2 (Section 3.3, second pass): write C into caller-allocated arrays.
 * Asynchronous on `stream`; the caller synchronises before reading C. */
FST_API int fst_compose_fill(fst_ctx *ctx, const fst_graph_out *C, void *stream);

/* Statistics of the last successful fst_compose_run. */
FST_API int fst_compose_stats(const fst_ctx *ctx, fst_stats *out);

/* With FST_OPT_TIMING on, the device time in ms of each phase of the last
 * run + fill: [0] validate+preprocess, [1] forward search, [2] backward
 * search, [3] numbering + arc count, [4] fill.  Writes min(n, 5) values;
 * returns FST_ERR_STATE if timing was off. */
FST_API int fst_compose_phase_times(const fst_ctx *ctx, float *ms, int n);

/* Kernels timed with FST_OPT_TIMING on: every launch of the forward search
 * kernel; every launch of the backward search kernel; the arc-count kernels
 * (states with few moves, then states with many: 2 launches, 1 if C is
 * empty); the fill kernels (every state's offset and flags with the arcs of
 * light states, then heavy states' arcs if any). */
enum fst_kernel {
  FST_KERNEL_SEARCH_FORWARD = 0,
  FST_KERNEL_SEARCH_BACKWARD = 1,
  FST_KERNEL_COUNT = 2,
  FST_KERNEL_FILL = 3,
  FST_KERNEL_SCORE_GEN = 4,   /* fst_score: generation kernels (one launch
                                 advances every direction asked for)       */
  FST_KERNEL_SCORE_PREP = 5,  /* fst_score: in-arc structure of the graph   */
  FST_KERNEL_SEARCH3 = 6,     /* fst_compose3_run: the level launches of the
                                 forward and backward searches             */
  FST_KERNEL_COMPACT3 = 7     /* fst_compose3_run + fill: in-arc grouping,
                                 trim keys, sort and numbering, arc count,
                                 fill                                      */
};

/* With FST_OPT_TIMING on: *ms = summed device time of the launches of
 * `kernel` in the last run + fill (kernels 0-3), the last fst_score
 * (kernels 4-5) or the last fst_compose3_run + fst_compose3_fill (kernels
 * 6-7), each bracketed by HIP events on the caller's stream, and
 * *launches = how many there were.  Returns FST_ERR_STATE if timing was off
 * or no such call was timed, FST_ERR_INVALID_ARG for an unknown kernel. */
FST_API int fst_compose_kernel_time(const fst_ctx *ctx, int kernel, float *ms, int64_t *launches);

/* ---- Scores of C and their gradient ------------------------------------
 * The log-semiring weight of C's paths (Eq. (1)) is what a training user
 * differentiates through (the introduction motivates eager composition by
 * automatic differentiation).  For an acyclic graph G (any fst_graph, e.g.
 * a composed C):
 *   alpha[v] = log-sum over paths from a start state to v of exp(weight),
 *              0 for a start state's empty path;
 *   beta[v]  = log-sum over paths from v to an accepting state;
 *   total    = log-sum over all paths from a start state to an accepting
 *              state (-inf if there is none); the weight of a path is the
 *              sum of its arc weights, and sums are float64.
 * Every log-sum is exact up to its final rounding and independent of the
 * order of its terms, so results are bitwise reproducible. */

/* Forward and backward scores of G (device arrays of V doubles; either may
 * be NULL to skip that direction) and the total (one device double, the
 * log-sum of alpha over accepting states when alpha is computed, else of
 * beta over start states).  G's structure is validated as in
 * fst_compose_run (labels are not read: scores do not depend on them).  Queued on
 * `stream`; blocks on small readbacks as the recursion advances.  Returns
 * FST_ERR_CYCLIC (outputs undefined) if G has a cycle (fst_score_cyclic
 * below takes such graphs).  Weights must be
 * finite (an infinite or NaN weight gives unspecified values, never a
 * fault).  G must stay valid until the work has completed. */
FST_API int fst_score(fst_ctx *ctx, const fst_graph *G, double *alpha, double *beta,
                      double *total, void *stream);

/* The same scores (alpha, beta, total: the sums over all paths) of a graph
 * that may have cycles, where a state can have infinitely many paths; the
 * sums are finite when the spectral radius of the matrix of arc
 * probabilities, M[u][v] = sum of exp(w(e)) over the arcs from u to v, is
 * below 1 over the states that lie on such paths (the Neumann series
 * sum_k M^k of the probability domain).  Shortest distance is among the
 * operations the paper leaves to future work (Section 5); here it is
 * relaxed by Jacobi sweeps of both recursions from every value at -inf:
 * sweep k gives each state the exact log-add of fst_score over the
 * previous sweep's values (its pull list's terms and its empty path), so
 * after k sweeps the values are the sums over the paths of at most k - 1
 * arcs, rising monotonically.  The sweeps stop at the first sweep in which
 * no value rose by more than `tol` (log domain, >= 0; 0 waits for a sweep
 * that changes no value upwards); *sweeps (if not NULL) receives its
 * number.  On a graph without cycles the sweeps reach fst_score's values
 * bit for bit after at most (longest path + 2) sweeps.  Each sweep reads
 * every state's in-arcs and out-arcs once (one thread per state, so a state
 * with many arcs is summed by one thread), in batches of 8 to 64 sweeps
 * between read-backs (a quarter of the sweeps so far).  Arguments, validation and outputs as in fst_score;
 * returns FST_ERR_NOT_CONVERGED (outputs: the last sweep's values) if no
 * sweep settled within max_sweeps (>= 0) sweeps, as when the sums diverge;
 * FST_ERR_INVALID_ARG for a negative max_sweeps or tol. */
FST_API int fst_score_cyclic(fst_ctx *ctx, const fst_graph *G, double *alpha, double *beta,
                             double *total, int32_t max_sweeps, double tol, int32_t *sweeps,
                             void *stream);

/* Arc posteriors times `scale`: grad[e] = scale * exp(alpha[src e] + w(e) +
 * beta[dst e] - *total), the derivative of scale * total by w(e) (0 for every
 * arc when *total is -inf).  alpha, beta, total come from fst_score or
 * fst_score_cyclic on the same G (with cycles, an arc's posterior is its
 * expected number of uses and can exceed 1); grad has E floats (device).
 * G is validated.  Asynchronous after the validation readback. */
FST_API int fst_score_posterior(fst_ctx *ctx, const fst_graph *G, const double *alpha,
                                const double *beta, const double *total, float scale,
                                float *grad, void *stream);

/* Gradient scatter through provenance: out[i] = sum of grad[e] over the
 * e < n with idx[e] = i (idx[e] = -1 is skipped), for i < m.  With idx =
 * C's arc_a (arc_b) and grad = the gradient of a loss by C's arc weights,
 * out is its gradient by the weights of A's (B's) arcs, since an arc of C
 * weighs w(a) + w(b).  Sums are exact to 2^-64 of the largest |grad| per
 * term, rounded once to float, so they do not depend on the order of
 * accumulation.  grad, idx: n entries; out: m floats (device).  Blocks until
 * done; returns FST_ERR_INVALID_ARG if an index lies outside [-1, m). */
FST_API int fst_grad_scatter(fst_ctx *ctx, int64_t n, const float *grad, const int32_t *idx,
                             int32_t m, float *out, void *stream);

/* Largest m (number of targets) that fst_grad_scatter_noalloc accepts. */
#define FST_SCATTER_NOALLOC_MAX_TARGETS (1 << 20)

/* fst_grad_scatter for callers that cannot allocate device memory (code
 * under HIP graph capture, serving loops that must not call hipMalloc,
 * harnesses that forbid it): same arguments and the same result, bit for
 * bit, but the call allocates nothing.  Its accumulators live in a fixed
 * device array of the library (32 bytes per target, for at most
 * FST_SCATTER_NOALLOC_MAX_TARGETS targets: 32 MiB plus a small header),
 * which every device the library runs on holds until the process ends; its
 * address is looked up once per device by fst_ctx_create.  The call clears
 * the part it uses before summing; the array keeps the last call's sums
 * afterwards.  All calls on one device share that one array, so calls that
 * overlap on a device (different streams or host threads without ordering)
 * race and give wrong sums: order them.  Returns FST_ERR_TOO_LARGE if m
 * exceeds the maximum, FST_ERR_INVALID_ARG for an index outside [-1, m) or
 * bad arguments.  Blocks until done (it reads back the bad-index flag into
 * the context's host memory, set up by fst_ctx_create). */
FST_API int fst_grad_scatter_noalloc(fst_ctx *ctx, int64_t n, const float *grad,
                                     const int32_t *idx, int32_t m, float *out, void *stream);

/* ---- Batches and chains ------------------------------------------------
 * Batch (the realistic workload of Section 4.2: the emission graphs of many
 * utterances composed with one lexicon): C_i = A_i o B for i < n in one
 * pass.  The A_i (host array of n device graphs) are composed as their
 * disjoint union; keys of different items never meet, and in the canonical
 * order (qa first) item i's states and arcs are the contiguous ranges
 * [item_states[i], item_states[i+1]) and [item_arcs[i], item_arcs[i+1]) of
 * the one C that fst_compose_fill then writes.  Ids in that C are those of
 * the union: subtract item_states[i] from src, dst (and item_arcs[i] from
 * arc_offset) for item-local values; key_a and arc_a index the union of the
 * A_i (subtract the states / arcs of the items before i).  item_states and
 * item_arcs are host arrays of n + 1 entries, filled on success (the last
 * entries are V_C and E_C).  Items are composed in parts: consecutive
 * items whose union fits the key space of one composition (an item that
 * does not fit alone gives FST_ERR_TOO_LARGE); most batches are one part,
 * one search.  With several parts the run searches each part in turn, and
 * fst_compose_fill searches every part but the last again before writing
 * it, so that fill blocks until done; the A_i and B must stay valid and
 * unchanged until the fill has completed (a part that comes out with other
 * sizes gives FST_ERR_STATE).  fst_compose_stats then reports sums over the
 * parts (levels: the largest).  V_C and E_C are at most INT32_MAX.
 * Chains (N-way composition): C has the input layout, so A o B o D is two
 * calls (compose, then compose C with D). */
FST_API int fst_compose_batch_run(fst_ctx *ctx, const fst_graph *A, int32_t n,
                                  const fst_graph *B, void *stream, int64_t *num_states,
                                  int64_t *num_arcs, int64_t *item_states,
                                  int64_t *item_arcs);

/* Per-item totals of a batch: totals[i] = log-sum of exp(val[v]) over the
 * v in [bounds[i], bounds[i+1]) with flag[v] != 0, for i < n (exact as in
 * fst_score; -inf for an empty set).  With val = alpha of the batch's C,
 * flag = its accept array and bounds = item_states, totals are the items'
 * forward scores.  val, flag, totals: device; bounds: host, n + 1
 * non-decreasing entries within the arrays.  Blocks until done. */
FST_API int fst_segment_logsum(fst_ctx *ctx, const double *val, const uint8_t *flag, int32_t n,
                               const int64_t *bounds, double *totals, void *stream);

/* ---- Three inputs at once ----------------------------------------------
 * N-way composition (Section 5 names composing N inputs at once, instead
 * of two, as the next step): C = A o B o D in one search, without building
 * A o B.  Eq. (1) read for three inputs: C maps x to w with score log-sum,
 * over all y and z, of exp(A(x, y) + B(y, z) + D(z, w)).  States of C are
 * keys (qa, qb, f1, qd, f2): (qa, qb, f1) is a state of T = A o B whose
 * arcs are the three moves of two-input composition (header comment above,
 * filter bit f1), and the key composes T with D by the same three rules,
 * filter bit f2:
 *   match  : a T-arc t with output z != 0, an arc ed of qd with ilabel z
 *            -> (dst t, dst ed, 0); label in(t):olabel(ed);
 *            weight w(t) + w(ed) (a T-match weighs w(ea) + w(eb), so the
 *            adds are (w(ea) + w(eb)) + w(ed), binary32, in that order)
 *   T alone: only when f2 = 0; a T-arc t with output 0 -> (dst t, qd, 0);
 *            label in(t):0; weight w(t)
 *   D alone: an arc ed of qd with ilabel 0 -> ((qa, qb, f1), dst ed,
 *            epsOutT(qa, qb, f1)); label 0:olabel(ed); weight w(ed)
 * where epsOutT says whether the T-state has a T-arc with output 0.  Start
 * keys are (sa, sb, 0, sd, 0); a key accepts iff its three states accept;
 * C is trim.  Output is canonical: states in ascending key order (qa, qb,
 * f1, qd, f2); the arcs of a state by (l, a, b, d), where l is the label
 * the arcs of A and B were matched on (0 when they were not both used) and
 * a, b, d are the arcs of A, B and D the arc came from, a missing arc
 * sorting last.  Key bits: bits(V_A - 1) +
 * bits(V_B - 1) + bits(V_D - 1) + 2 <= 62 (each at least 1), else
 * FST_ERR_TOO_LARGE.  The workspace grows with the number of keys reached
 * (a hash set of 8 bytes per slot, at most half full, grown and searched
 * again when it fills). */
typedef struct {
  int32_t *arc_offset;
  int32_t *src, *dst, *ilabel, *olabel;
  float *weight;
  uint8_t *start, *accept;
  int32_t *key_a, *key_b;   /* optional [V_C] (NULL skips): the key of     */
  uint8_t *key_fab;         /* each state, (key_a, key_b, key_fab, key_d,  */
  int32_t *key_d;           /* key_f) = (qa, qb, f1, qd, f2)               */
  uint8_t *key_f;
  int32_t *arc_a, *arc_b, *arc_d; /* optional [E_C] provenance, -1 = none  */
} fst_graph3_out;

/* Phase 1 of C = A o B o D: validate the three graphs, search forward from
 * the start keys and backward over the generated arcs, number the trim
 * keys and count their arcs.  Blocks until *num_states and *num_arcs are
 * known.  A, B and D must stay valid and unchanged until
 * fst_compose3_fill's work has completed. */
FST_API int fst_compose3_run(fst_ctx *ctx, const fst_graph *A, const fst_graph *B,
                             const fst_graph *D, void *stream, int64_t *num_states,
                             int64_t *num_arcs);

/* Phase 2: write C into caller-allocated arrays sized from phase 1
 * (asynchronous on `stream`). */
FST_API int fst_compose3_fill(fst_ctx *ctx, const fst_graph3_out *C, void *stream);

/* Statistics of the last successful fst_compose3_run: key_space = 2^(key
 * bits), accessible = keys reached, coaccessible = num_states = V_C,
 * generated = moves out of the accessible keys, fwd_levels and bwd_levels
 * = levels of the two searches, num_arcs = E_C, heavy_states = states of
 * C with more work units than one thread takes (one workgroup each in the
 * count and the fill), generated_backward -1. */
FST_API int fst_compose3_stats(const fst_ctx *ctx, fst_stats *out);

/* Static string for a status code. */
FST_API const char *fst_strerror(int code);

#ifdef __cplusplus
}
#endif

#endif /* FST_COMPOSE_H */
