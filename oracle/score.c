/*
 * Log-semiring scores of an acyclic weighted graph, the arc posteriors that
 * are their gradient, and the scatter of per-arc gradients of a composed
 * graph back to the arcs of its operands through provenance.
 *
 * TEST INFRASTRUCTURE ONLY, like oracle.c: only the test-suite, the smoke
 * check and the benchmark's CPU-baseline leg may load this code, and it
 * shares nothing with the GPU library.
 *
 * Definitions (fp64 throughout; arc weights are binary32, widened exactly):
 *   the weight of a path is the sum of its arc weights, and log-add is
 *   x (+) y = log(exp x + exp y), the addition of the log semiring whose
 *   multiplication is + (Eq. (1) reads the composed weight in this
 *   semiring);
 *   alpha[v] = log-sum over paths from any start state to v of their weight
 *              (a start state's empty path has weight 0);
 *   beta[v]  = log-sum over paths from v to any accepting state;
 *   total    = log-sum over paths from a start state to an accepting state;
 *   an empty sum is -inf.
 * total is the forward score a training user reads off the composed graph
 * (the introduction motivates eager composition by differentiation through
 * such scores); alpha and beta are the forward and backward
 * shortest distances of the log semiring.  They are computed the textbook
 * way: states in a topological order (Kahn's algorithm), alpha by log-adding
 * each finished state's value plus the arc weight into its successors, beta
 * by log-adding over each state's out-arcs in reverse order.  A graph with a
 * cycle is refused (its sums need not be finite).
 *
 * The derivative of total by the weight of arc e is its posterior
 *   p[e] = exp(alpha[src e] + w(e) + beta[dst e] - total),
 * the share of the total path mass that passes through e (0 when total is
 * -inf).  For C = A o B, an arc of C built from arc a of A (and arc b of B)
 * has weight w(a) + w(b), so the gradient of anything by w(a) is the sum of
 * the gradients of the C arcs whose provenance names a:
 *   grad_A[a] = sum over arcs e of C with arc_a[e] = a of g[e]
 * (the same for B), summed in arc order.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>

#include "og.h"

/* Deliberate mistakes, used only by tests that show the pins detect them. */
enum {
  SMUT_NONE = 0,
  SMUT_MAX = 1,         /* (+) is max: the Viterbi score                */
  SMUT_DROP_WEIGHT = 2, /* alpha ignores the arc weight                 */
  SMUT_ALL_ACCEPT = 3,  /* beta treats every state as accepting          */
  SMUT_NO_START = 4     /* alpha forgets the start states' empty path    */
};

static double log_add(double x, double y, int mut) {
  if (x == -INFINITY) return y;
  if (y == -INFINITY) return x;
  const double hi = x > y ? x : y, lo = x > y ? y : x;
  if (mut == SMUT_MAX) return hi;
  return hi + log1p(exp(lo - hi));
}

/* Topological order by Kahn's algorithm: order[0..n) with n = V iff the
 * graph has no cycle; depth[v] = number of states on the longest path that
 * ends in v. */
static int topo_order(const og_graph *g, int32_t *order, int32_t *n_out, int32_t *depth) {
  const int32_t V = g->num_states, E = g->num_arcs;
  int32_t *indeg = (int32_t *)calloc((size_t)V + 1, sizeof(int32_t));
  if (!indeg) return OG_ERR_NOMEM;
  for (int32_t e = 0; e < E; e++) indeg[g->dst[e]]++;
  int32_t head = 0, tail = 0;
  for (int32_t v = 0; v < V; v++) {
    depth[v] = 1;
    if (indeg[v] == 0) order[tail++] = v;
  }
  while (head < tail) {
    const int32_t u = order[head++];
    for (int32_t e = g->arc_offset[u]; e < g->arc_offset[u + 1]; e++) {
      const int32_t v = g->dst[e];
      if (depth[u] + 1 > depth[v]) depth[v] = depth[u] + 1;
      if (--indeg[v] == 0) order[tail++] = v;
    }
  }
  free(indeg);
  *n_out = tail;
  return OG_OK;
}

int oracle_score(const og_graph *g, int mut, double *alpha, double *beta, double *total_fwd,
                 double *total_bwd, int32_t *longest) {
  int rc = og_check_graph(g);
  if (rc) return rc;
  const int32_t V = g->num_states;
  *total_fwd = -INFINITY;
  *total_bwd = -INFINITY;
  *longest = 0;
  if (V == 0) return OG_OK;
  int32_t *order = (int32_t *)malloc(sizeof(int32_t) * (size_t)V);
  int32_t *depth = (int32_t *)malloc(sizeof(int32_t) * (size_t)V);
  if (!order || !depth) {
    free(order);
    free(depth);
    return OG_ERR_NOMEM;
  }
  int32_t n = 0;
  rc = topo_order(g, order, &n, depth);
  if (rc == OG_OK && n < V) rc = OG_ERR_CYCLE;
  if (rc == OG_OK) {
    for (int32_t v = 0; v < V; v++) {
      alpha[v] = (g->start[v] && mut != SMUT_NO_START) ? 0.0 : -INFINITY;
      if (depth[v] > *longest) *longest = depth[v];
    }
    /* forward: a state's value is final when it is taken from the order */
    for (int32_t i = 0; i < V; i++) {
      const int32_t u = order[i];
      if (alpha[u] == -INFINITY) continue;
      for (int32_t e = g->arc_offset[u]; e < g->arc_offset[u + 1]; e++) {
        const double w = mut == SMUT_DROP_WEIGHT ? 0.0 : (double)g->weight[e];
        alpha[g->dst[e]] = log_add(alpha[g->dst[e]], alpha[u] + w, mut);
      }
    }
    /* backward: successors come later in the order */
    for (int32_t i = V - 1; i >= 0; i--) {
      const int32_t u = order[i];
      double b = (g->accept[u] || mut == SMUT_ALL_ACCEPT) ? 0.0 : -INFINITY;
      for (int32_t e = g->arc_offset[u]; e < g->arc_offset[u + 1]; e++)
        b = log_add(b, (double)g->weight[e] + beta[g->dst[e]], mut);
      beta[u] = b;
    }
    for (int32_t v = 0; v < V; v++) {
      if (g->accept[v]) *total_fwd = log_add(*total_fwd, alpha[v], mut);
      if (g->start[v]) *total_bwd = log_add(*total_bwd, beta[v], mut);
    }
  }
  free(order);
  free(depth);
  return rc;
}

int oracle_posterior(const og_graph *g, const double *alpha, const double *beta, double total,
                     double *post) {
  int rc = og_check_graph(g);
  if (rc) return rc;
  for (int32_t e = 0; e < g->num_arcs; e++) {
    if (total == -INFINITY) {
      post[e] = 0.0;
      continue;
    }
    post[e] = exp(alpha[g->src[e]] + (double)g->weight[e] + beta[g->dst[e]] - total);
  }
  return OG_OK;
}

int oracle_scatter(int64_t n, const double *grad, const int32_t *idx, int32_t m, double *out) {
  if (n < 0 || m < 0) return OG_ERR_ARG;
  for (int32_t i = 0; i < m; i++) out[i] = 0.0;
  for (int64_t e = 0; e < n; e++) {
    if (idx[e] < -1 || idx[e] >= m) return OG_ERR_ARG;
    if (idx[e] >= 0) out[idx[e]] += grad[e];
  }
  return OG_OK;
}
