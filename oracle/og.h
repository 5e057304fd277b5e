/* Graph layout and error codes shared by the oracle's C files (test
 * infrastructure only; nothing here is used by the GPU library). */
#ifndef OG_H
#define OG_H
#include <stdint.h>

enum { OG_OK = 0, OG_ERR_ARG = 1, OG_ERR_NOMEM = 2, OG_ERR_TOO_LARGE = 3, OG_ERR_CYCLE = 4 };

typedef struct {
  int32_t num_states, num_arcs;
  const int32_t *arc_offset, *src, *dst, *ilabel, *olabel;
  const float *weight;
  const uint8_t *start, *accept;
} og_graph;

/* 0 if the graph is a well-formed CSR (offsets, src, dst in range, labels
 * not negative), else OG_ERR_ARG. */
int og_check_graph(const og_graph *g);

#endif
