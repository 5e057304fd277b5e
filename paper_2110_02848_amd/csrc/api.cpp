// Host orchestration and the C ABI of libfstcompose.so (include/fst_compose.h).
//
// fst_compose_run drives the phases of the parallel composition (paper
// Section 3.3) on one HIP stream:
//   1. validate A and B, build label-sorted out- and in-views;
//   2. forward frontier search from the start keys (accessible keys);
//   3. backward frontier search from the accessible accepting keys over the
//      in-arcs (co-accessible keys); the trim set is what both reach;
//   4. number the trim keys in key order and count each state's kept arcs
//      (the paper's first pass), scan the counts into arc offsets;
// fst_compose_fill then writes the arcs (the paper's second pass).
//
// fst_score, fst_score_posterior and fst_grad_scatter compute the
// log-semiring scores of an acyclic graph (such as C), their gradient, and
// its scatter to the operands through provenance (score.hip).
#include <stdlib.h>
#include <string.h>

#include <initializer_list>
#include <new>
#include <vector>

#include "internal.h"

using namespace fstc;

namespace {

struct DevBuf {
  void *p = nullptr;
  size_t cap = 0;
};

constexpr int NEV = 10;  // a begin and an end event per phase (enum in fst_compose_phase_times)
constexpr int NKERNELS = 8;  // enum fst_kernel
constexpr int NCOMPOSE_KERNELS = 4;  // kernels 0-3 time a composition, 4-5 a score,
                                     // 6-7 a three-input composition

// Per-direction working arrays of the score recursion.
struct ScoreBufs {
  DevBuf sc, rec, term, mkey, pend, q, h, hoff;
  ScoreScalars *host = nullptr;  // pinned mirror of sc
};

}  // namespace

struct fst_ctx {
  int device = 0;
  int64_t max_ws = 0;
  size_t ws_total = 0;
  bool timing = false;
  bool buckets = true;
  bool count_moves = false;
  bool validate = true;
  int order = FST_ORDER_CONCURRENT;
  int chain_depth = CHAIN_MAX;
  bool have_times = false;
  bool timed_run = false;

  DevBuf scal, lists;
  DevBuf k0, k1, v0, v1, sort_tmp, scan_tmp;
  DevBuf aOutPerm, aOutArc, aOutRec, aOutLut, bOutPerm, bOutArc, bOutRec, bOutLut;
  DevBuf aOutLab, aOutW, bOutLab, bOutW, bOutChain, bInChain;
  DevBuf aInOff, aInPerm, aInArc, aInRec, aInLut, bInOff, bInPerm, bInArc, bInRec, bInLut;
  DevBuf vis, coacc, trim, wbase, fq, bq, heavy, hoff, heavy2, hoff2, cnt, btot;
  // score workspace
  DevBuf s_pg, s_pidx, s_bcnt, s_bscan, s_btotal;  // grouped scatter
  DevBuf s_sc, s_owner, s_extra, s_inref, s_mbeg, s_mlen, s_mcur, s_marc, s_val, s_acc,
      s_mpos, s_sweep, s_ioff, s_isrc, s_iw;
  // batches: the union of the A graphs, item tables, segment sums
  DevBuf u_off, u_src, u_dst, u_il, u_ol, u_w, u_start, u_accept, u_items, seg;
  // three-input composition
  DevBuf t_scal, t_aPerm, t_aArc, t_aRec, t_bPerm, t_bArc, t_bRec, t_bLab, t_bW, t_dPerm,
      t_dArc, t_dRec, t_dLab, t_dW, t_bflags, t_lists, t_tab, t_F, t_chunks, t_arcs, t_inoff,
      t_first, t_coacc, t_keys0, t_keys1, t_slots0, t_slots1, t_idof, t_units, t_ucnt,
      t_aLab, t_aW, t_heavy, t_aLut, t_bLut, t_dLut, t_bChain, t_segs, t_segof;
  Scal3 *h_s3 = nullptr;
  uint32_t h3_hint = 0;  // hash capacity the last three-input search needed
  int lv3_hint[2] = {0, 0};  // levels the last three-input searches took (bwd, fwd)
  unsigned long long list_hint = 0;  // search list capacity the last run needed
  int gen_hint = 0;  // launches the last concurrent search took
  unsigned long long list_start = 1ull << 22;  // FST_OPT_LIST_CAPACITY
  struct {
    bool ready = false;
    Problem3 P = {};
    const unsigned long long *keys = nullptr;
    const uint32_t *ustart = nullptr, *uoff = nullptr, *heavy = nullptr, *nheavy = nullptr;
    uint32_t n = 0, U = 0, narcs = 0;
    fst_stats stats = {};
    bool timed = false;
  } c3;
  bool have_times3 = false;
  Scalars *h_sc = nullptr;
  ScoreScalars *h_ssc = nullptr;
  ScoreBufs score_f, score_b;  // forward / backward recursion
  bool have_score_times = false;
  hipEvent_t ev[NEV] = {};
  hipEvent_t kev[2 * NKERNELS] = {};  // per timed kernel: before, after
  float kms[NKERNELS] = {};
  int64_t klaunches[NKERNELS] = {};

  bool ready = false;
  Problem P = {};
  uint32_t nstates = 0, narcs = 0, nheavy = 0;
  unsigned long long nkeys = 0;
  size_t out_words = 0;  // trim words the output passes cover
  fst_stats stats = {};

  // A batch composed in parts: consecutive items whose key space fits 32
  // bits each; the context holds the search state of part cur_part, and the
  // fill searches every other part again.  Empty for a plain composition or
  // a batch of one part.
  struct BatchPart {
    int32_t i0, i1;                  // items [i0, i1)
    long long vbase, ebase;          // first state and arc of the part in C
    long long abase, aebase;         // first state and arc of its items in the union of A
    long long V, E;                  // its states and arcs
  };
  std::vector<BatchPart> parts;
  std::vector<fst_graph> batch_A;
  fst_graph batch_B = {};
  int cur_part = -1;
  fst_stats batch_stats = {};
};

namespace {

struct DeviceGuard {
  int prev = -1;
  bool ok = false;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) prev = -1;
    ok = hipSetDevice(dev) == hipSuccess;
  }
  ~DeviceGuard() {
    if (prev >= 0) (void)hipSetDevice(prev);
  }
};

#define HIP_TRY(expr)                        \
  do {                                       \
    if ((expr) != hipSuccess) return FST_ERR_HIP; \
  } while (0)

#define FST_TRY(expr)             \
  do {                            \
    int rc_ = (expr);             \
    if (rc_ != FST_OK) return rc_; \
  } while (0)

size_t round_up(size_t x) { return (x + 255) & ~(size_t)255; }

int ensure(fst_ctx *c, DevBuf &b, size_t bytes) {
  bytes = round_up(bytes ? bytes : 1);
  if (b.cap >= bytes) return FST_OK;
  size_t next = c->ws_total - b.cap + bytes;
  if (c->max_ws > 0 && next > (size_t)c->max_ws) return FST_ERR_NOMEM;
  if (b.p) {
    // earlier queued work may still read the old buffer
    if (hipDeviceSynchronize() != hipSuccess) return FST_ERR_HIP;
    (void)hipFree(b.p);
    c->ws_total -= b.cap;
    b.p = nullptr;
    b.cap = 0;
  }
  if (hipMalloc(&b.p, bytes) != hipSuccess) {
    (void)hipGetLastError();
    b.p = nullptr;
    return FST_ERR_NOMEM;
  }
  b.cap = bytes;
  c->ws_total += bytes;
  return FST_OK;
}

void release(DevBuf &b) {
  if (b.p) (void)hipFree(b.p);
  b.p = nullptr;
  b.cap = 0;
}

template <typename T>
T *as(DevBuf &b) {
  return reinterpret_cast<T *>(b.p);
}

int readback(fst_ctx *c, hipStream_t s) {
  HIP_TRY(hipMemcpyAsync(c->h_sc, c->scal.p, sizeof(Scalars), hipMemcpyDeviceToHost, s));
  HIP_TRY(hipStreamSynchronize(s));
  return FST_OK;
}

int bitlen(unsigned long long x) { return x ? 64 - __builtin_clzll(x) : 0; }

int check_graph_args(const fst_graph *g) {
  if (g->num_states < 0 || g->num_arcs < 0) return FST_ERR_INVALID_ARG;
  if (g->num_states == 0) return g->num_arcs == 0 ? FST_OK : FST_ERR_INVALID_GRAPH;
  if (!g->arc_offset || !g->start || !g->accept) return FST_ERR_INVALID_ARG;
  if (g->num_arcs > 0 &&
      (!g->src || !g->dst || !g->ilabel || !g->olabel || !g->weight))
    return FST_ERR_INVALID_ARG;
  return FST_OK;
}

DevGraph dev_graph(const fst_graph *g) {
  DevGraph d;
  d.V = g->num_states;
  d.E = g->num_arcs;
  d.off = g->arc_offset;
  d.src = g->src;
  d.dst = g->dst;
  d.il = g->ilabel;
  d.ol = g->olabel;
  d.w = g->weight;
  d.start = g->start;
  d.accept = g->accept;
  return d;
}

enum { PH_PRE = 0, PH_FWD = 1, PH_BWD = 2, PH_COUNT = 3, PH_FILL = 4 };
void phase_begin(fst_ctx *c, int ph, hipStream_t s) {
  if (c->timing) (void)hipEventRecord(c->ev[2 * ph], s);
}
void phase_end(fst_ctx *c, int ph, hipStream_t s) {
  if (c->timing) (void)hipEventRecord(c->ev[2 * ph + 1], s);
}

int finish_empty(fst_ctx *c, int64_t *V_C, int64_t *E_C) {
  c->P = Problem{};  // no trim bitmap: the fill must not read one
  c->out_words = 0;
  c->nstates = 0;
  c->narcs = 0;
  c->nheavy = 0;
  c->ready = true;
  *V_C = 0;
  *E_C = 0;
  return FST_OK;
}

KernelTimer timer(const fst_ctx *c, int kernel) {
  KernelTimer t;
  if (c->timing) {
    t.ev0 = c->kev[2 * kernel];
    t.ev1 = c->kev[2 * kernel + 1];
  }
  return t;
}

// Adds the time between a timer's events (both complete) to kernel's total.
int add_time(fst_ctx *c, int kernel, int64_t launches) {
  if (!c->timing) return FST_OK;
  float t = 0.f;
  HIP_TRY(hipEventElapsedTime(&t, c->kev[2 * kernel], c->kev[2 * kernel + 1]));
  c->kms[kernel] += t;
  c->klaunches[kernel] += launches;
  return FST_OK;
}

// Generations are queued in batches (4, 16, 32, 64, 64, ...) with no host
// round trip; after each batch the host checks whether the next generation
// has any work (generations queued after the search has ended do nothing).
int search(fst_ctx *c, const SearchArgs &S, bool forward, int64_t *levels, hipStream_t s) {
  const int kernel = forward ? FST_KERNEL_SEARCH_FORWARD : FST_KERNEL_SEARCH_BACKWARD;
  const KernelTimer t = timer(c, kernel);
  int g = 0, batch = 4;
  for (;;) {
    t.begin(s);
    for (int b = 0; b < batch; ++b, ++g) HIP_TRY(launch_generation(c->P, S, forward, g, s));
    t.end(s);
    FST_TRY(readback(c, s));
    FST_TRY(add_time(c, kernel, batch));
    if (c->h_sc->overflow) return FST_ERR_TOO_LARGE;
    const GenSlot &nx = c->h_sc->G[g % 3];
    if (nx.qcount == 0 && (uint32_t)nx.hpack == 0) break;
    batch = batch == 4 ? 16 : (batch < 64 ? 2 * batch : 64);
  }
  *levels = c->h_sc->gens;
  return FST_OK;
}

// ---------------------------------------------------------------------------
// scores
// ---------------------------------------------------------------------------

int score_readback(fst_ctx *c, hipStream_t s) {
  HIP_TRY(hipMemcpyAsync(c->h_ssc, c->s_sc.p, sizeof(ScoreScalars), hipMemcpyDeviceToHost, s));
  HIP_TRY(hipStreamSynchronize(s));
  return FST_OK;
}

// Validates G (one readback): FST_ERR_INVALID_GRAPH on a violation.
int score_validate(fst_ctx *c, const DevGraph &d, hipStream_t s) {
  ScoreScalars *dsc = as<ScoreScalars>(c->s_sc);
  HIP_TRY(hipMemsetAsync(dsc, 0, sizeof(ScoreScalars), s));
  // scores read no label: the structure alone is checked (or nothing, for
  // a caller that vouches for it)
  if (!c->validate) return FST_OK;
  if (d.V > 0) HIP_TRY(launch_validate(d, 2, &dsc->err, &dsc->maxlab, s));
  FST_TRY(score_readback(c, s));
  return c->h_ssc->err ? FST_ERR_INVALID_GRAPH : FST_OK;
}

int score_bufs(fst_ctx *c, ScoreBufs &b, int32_t V, size_t E) {
  FST_TRY(ensure(c, b.sc, sizeof(ScoreScalars)));
  FST_TRY(ensure(c, b.rec, (size_t)V * sizeof(int4)));
  FST_TRY(ensure(c, b.term, 2 * E * sizeof(double)));
  FST_TRY(ensure(c, b.mkey, (size_t)V * 8));
  FST_TRY(ensure(c, b.pend, (size_t)V * 4));
  FST_TRY(ensure(c, b.q, (size_t)V * 4));
  FST_TRY(ensure(c, b.h, (size_t)V * 4));
  FST_TRY(ensure(c, b.hoff, (size_t)V * 4));
  return FST_OK;
}

ScoreArgs score_args(fst_ctx *c, ScoreBufs &b, const ScoreGraph &SG, double *val) {
  ScoreArgs S = {};
  S.G = SG;
  S.rec = as<int4>(b.rec);
  S.term = as<double>(b.term);
  S.mpos = as<int32_t>(c->s_mpos);
  S.mkey = as<unsigned long long>(b.mkey);
  S.val = val;
  S.pend = as<int32_t>(b.pend);
  S.Q = as<int32_t>(b.q);
  S.H = as<int32_t>(b.h);
  S.hoff = as<uint32_t>(b.hoff);
  S.cap = (uint32_t)SG.V;
  S.chain = c->chain_depth;
  S.sc = as<ScoreScalars>(b.sc);
  return S;
}

// The recursions asked for (F forward, B backward, either may be null),
// generation after generation, both in the same kernels (batches as in
// search()); FST_ERR_CYCLIC if some state never became ready.
int score_generations(fst_ctx *c, const ScoreArgs *F, const ScoreArgs *B, ScoreBufs *bf,
                      ScoreBufs *bb, hipStream_t s) {
  const ScoreArgs *dirs[2] = {F, B};
  ScoreBufs *bufs[2] = {bf, bb};
  for (int i = 0; i < 2; ++i) {
    if (!dirs[i]) continue;
    HIP_TRY(hipMemsetAsync(dirs[i]->sc, 0, sizeof(ScoreScalars), s));
    HIP_TRY(launch_score_seed(*dirs[i], i == 0, s));
  }
  const KernelTimer t = timer(c, FST_KERNEL_SCORE_GEN);
  int g = 0, batch = 4;
  for (;;) {
    t.begin(s);
    for (int b = 0; b < batch; ++b, ++g) HIP_TRY(launch_score_generation(F, B, g, s));
    t.end(s);
    for (int i = 0; i < 2; ++i)
      if (dirs[i])
        HIP_TRY(hipMemcpyAsync(bufs[i]->host, dirs[i]->sc, sizeof(ScoreScalars),
                               hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    FST_TRY(add_time(c, FST_KERNEL_SCORE_GEN, batch));
    bool more = false;
    for (int i = 0; i < 2; ++i) {
      if (!dirs[i]) continue;
      // cannot happen: each state is listed at most once
      if (bufs[i]->host->overflow) return FST_ERR_TOO_LARGE;
      const GenSlot &nx = bufs[i]->host->G[g % 3];
      more = more || nx.qcount != 0 || (uint32_t)nx.hpack != 0;
    }
    if (!more) break;
    batch = batch == 4 ? 16 : (batch < 64 ? 2 * batch : 64);
  }
  for (int i = 0; i < 2; ++i)
    if (dirs[i] && bufs[i]->host->finished != (unsigned long long)dirs[i]->G.V)
      return FST_ERR_CYCLIC;
  return FST_OK;
}

int score_total(fst_ctx *c, const double *val, const uint8_t *flag, int32_t V, double *total,
                hipStream_t s) {
  ScoreScalars *dsc = as<ScoreScalars>(c->s_sc);
  HIP_TRY(hipMemsetAsync(&dsc->zmax, 0, 3 * sizeof(unsigned long long), s));
  HIP_TRY(launch_score_total(val, flag, V, dsc, total, s));
  return FST_OK;
}

// G with its in-arc structure (single in-arcs, and the in-arc lists of
// merges), built into the context's buffers.
int score_structure(fst_ctx *c, const DevGraph &d, ScoreGraph &SG, hipStream_t s) {
  const int32_t V = d.V;
  const size_t E = (size_t)d.E;
  FST_TRY(ensure(c, c->s_owner, (size_t)V * 4));
  FST_TRY(ensure(c, c->s_extra, (size_t)V * 4));
  FST_TRY(ensure(c, c->s_inref, (size_t)V * 4));
  FST_TRY(ensure(c, c->s_mbeg, (size_t)V * 4));
  FST_TRY(ensure(c, c->s_mlen, (size_t)V * 4));
  FST_TRY(ensure(c, c->s_mcur, (size_t)V * 4));
  FST_TRY(ensure(c, c->s_marc, E * 4));
  FST_TRY(ensure(c, c->s_mpos, E * 4));
  SG = ScoreGraph{};
  SG.V = V;
  SG.E = (long long)E;
  SG.off = d.off;
  SG.src = d.src;
  SG.dst = d.dst;
  SG.w = d.w;
  SG.start = d.start;
  SG.accept = d.accept;
  SG.inref = as<int32_t>(c->s_inref);
  SG.mbeg = as<int32_t>(c->s_mbeg);
  SG.mlen = as<int32_t>(c->s_mlen);
  SG.marc = as<int32_t>(c->s_marc);
  HIP_TRY(hipMemsetAsync(c->s_owner.p, 0xff, (size_t)V * 4, s));
  HIP_TRY(hipMemsetAsync(c->s_extra.p, 0, (size_t)V * 4, s));
  HIP_TRY(launch_score_structure(SG, as<int32_t>(c->s_owner), as<int32_t>(c->s_extra),
                                 as<int32_t>(c->s_inref), as<int32_t>(c->s_mbeg),
                                 as<int32_t>(c->s_mlen), as<int32_t>(c->s_mcur),
                                 as<int32_t>(c->s_marc), as<int32_t>(c->s_mpos),
                                 as<ScoreScalars>(c->s_sc), s));
  return FST_OK;
}

int score_impl(fst_ctx *c, const fst_graph *G, double *alpha, double *beta, double *total,
               hipStream_t s) {
  FST_TRY(check_graph_args(G));
  const DevGraph d = dev_graph(G);
  FST_TRY(ensure(c, c->s_sc, sizeof(ScoreScalars)));
  for (int k = NCOMPOSE_KERNELS; k < NKERNELS; ++k) {
    c->kms[k] = 0.f;
    c->klaunches[k] = 0;
  }
  FST_TRY(score_validate(c, d, s));
  const int32_t V = d.V;
  const size_t E = (size_t)d.E;
  ScoreScalars *dsc = as<ScoreScalars>(c->s_sc);
  const bool fwd = alpha != nullptr || beta == nullptr;
  if (V == 0) {
    // no path at all: total = log 0
    HIP_TRY(hipMemsetAsync(&dsc->zmax, 0, 3 * sizeof(unsigned long long), s));
    HIP_TRY(launch_score_total(nullptr, nullptr, 0, dsc, total, s));
    return FST_OK;
  }
  const KernelTimer tp = timer(c, FST_KERNEL_SCORE_PREP);
  tp.begin(s);
  if (fwd && !alpha) FST_TRY(ensure(c, c->s_val, (size_t)V * 8));
  if (fwd) FST_TRY(score_bufs(c, c->score_f, V, E));
  if (beta) FST_TRY(score_bufs(c, c->score_b, V, E));
  ScoreGraph SG = {};
  FST_TRY(score_structure(c, d, SG, s));
  tp.end(s);
  ScoreArgs SF = {}, SB = {};
  if (fwd) SF = score_args(c, c->score_f, SG, alpha ? alpha : as<double>(c->s_val));
  if (beta) SB = score_args(c, c->score_b, SG, beta);
  FST_TRY(score_generations(c, fwd ? &SF : nullptr, beta ? &SB : nullptr, &c->score_f,
                            &c->score_b, s));
  FST_TRY(add_time(c, FST_KERNEL_SCORE_PREP, 1));
  if (fwd) FST_TRY(score_total(c, SF.val, d.accept, V, total, s));
  else FST_TRY(score_total(c, beta, d.start, V, total, s));
  c->have_score_times = c->timing;
  return FST_OK;
}

// Relaxation sweeps of both recursions (graphs with cycles), from every
// value at -inf, in batches with one read-back of the batch's rises each,
// until a sweep in which no value rose by more than tol.  A batch is a
// quarter of the sweeps done so far (8 to SWEEP_BATCH), so the sweeps run
// past the one that settled stay within about a quarter of the total.  The
// values after the batch's last sweep are returned (later sweeps of a
// batch rise no more than tol either, up to rounding).
ScoreGraph plain_score_graph(const DevGraph &d);

int score_cyclic_impl(fst_ctx *c, const fst_graph *G, double *alpha, double *beta,
                      double *total, int32_t max_sweeps, double tol, int32_t *sweeps,
                      hipStream_t s) {
  FST_TRY(check_graph_args(G));
  if (max_sweeps < 0 || !(tol >= 0.0)) return FST_ERR_INVALID_ARG;
  const DevGraph d = dev_graph(G);
  FST_TRY(ensure(c, c->s_sc, sizeof(ScoreScalars)));
  for (int k = NCOMPOSE_KERNELS; k < NKERNELS; ++k) {
    c->kms[k] = 0.f;
    c->klaunches[k] = 0;
  }
  if (sweeps) *sweeps = 0;
  FST_TRY(score_validate(c, d, s));
  const int32_t V = d.V;
  ScoreScalars *dsc = as<ScoreScalars>(c->s_sc);
  const bool fwd = alpha != nullptr || beta == nullptr, bwd = beta != nullptr;
  if (V == 0) {
    HIP_TRY(hipMemsetAsync(&dsc->zmax, 0, 3 * sizeof(unsigned long long), s));
    HIP_TRY(launch_score_total(nullptr, nullptr, 0, dsc, total, s));
    return FST_OK;
  }
  const KernelTimer tp = timer(c, FST_KERNEL_SCORE_PREP);
  tp.begin(s);
  ScoreGraph SG = plain_score_graph(d);
  FST_TRY(ensure(c, c->s_ioff, ((size_t)V + 1) * 4));
  FST_TRY(ensure(c, c->s_isrc, (size_t)d.E * 4));
  FST_TRY(ensure(c, c->s_iw, (size_t)d.E * 4));
  FST_TRY(ensure(c, c->s_inref, (size_t)V * 4));  // the placing cursors
  FST_TRY(ensure(c, c->scan_tmp, scan_temp_bytes((size_t)V + 1)));
  SG.ioff = as<int32_t>(c->s_ioff);
  SG.isrc = as<int32_t>(c->s_isrc);
  SG.iw = as<float>(c->s_iw);
  HIP_TRY(launch_in_csr(SG, as<int32_t>(c->s_ioff), as<int32_t>(c->s_isrc), as<float>(c->s_iw),
                        as<int32_t>(c->s_inref), c->scan_tmp.p, &dsc->mtotal, s));
  FST_TRY(ensure(c, c->s_sweep, (size_t)V * 4 * sizeof(double)));
  double *a[2] = {as<double>(c->s_sweep), as<double>(c->s_sweep) + V};
  double *b[2] = {a[1] + V, a[1] + 2 * (size_t)V};
  if (fwd) HIP_TRY(launch_fill_f64(a[0], V, -INFINITY, s));
  if (bwd) HIP_TRY(launch_fill_f64(b[0], V, -INFINITY, s));
  tp.end(s);
  const KernelTimer t = timer(c, FST_KERNEL_SCORE_GEN);
  int k = 0;
  bool done = false;
  while (!done && k < max_sweeps) {
    const int batch = k / 4 < 8 ? 8 : (k / 4 > SWEEP_BATCH ? SWEEP_BATCH : k / 4);
    const int n = batch < max_sweeps - k ? batch : max_sweeps - k;
    HIP_TRY(hipMemsetAsync(dsc->rise, 0, (size_t)n * sizeof(unsigned long long), s));
    t.begin(s);
    for (int j = 0; j < n; ++j) {
      const int x = (k + j) & 1, y = x ^ 1;
      HIP_TRY(launch_sweep(SG, a[x], fwd ? a[y] : nullptr, b[x], bwd ? b[y] : nullptr,
                           &dsc->rise[j], s));
    }
    t.end(s);
    HIP_TRY(hipMemcpyAsync(c->h_ssc->rise, dsc->rise, (size_t)n * sizeof(unsigned long long),
                           hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    FST_TRY(add_time(c, FST_KERNEL_SCORE_GEN, n));
    for (int j = 0; j < n && !done; ++j) {
      // the order key of a rise >= +0.0 is its bit pattern with the top bit set
      const unsigned long long key = c->h_ssc->rise[j] & ~(1ull << 63);
      double r;
      memcpy(&r, &key, sizeof r);
      if (r <= tol) {
        done = true;
        if (sweeps) *sweeps = k + j + 1;
      }
    }
    k += n;
  }
  if (c->timing) {
    HIP_TRY(hipStreamSynchronize(s));  // the structure's events (no sweep may have run)
    FST_TRY(add_time(c, FST_KERNEL_SCORE_PREP, 1));
  }
  // the last sweep wrote buffer k mod 2 (the values so far when none ran)
  const double *fa = a[k & 1], *fb = b[k & 1];
  if (alpha) HIP_TRY(hipMemcpyAsync(alpha, fa, (size_t)V * 8, hipMemcpyDeviceToDevice, s));
  if (beta) HIP_TRY(hipMemcpyAsync(beta, fb, (size_t)V * 8, hipMemcpyDeviceToDevice, s));
  if (fwd) FST_TRY(score_total(c, fa, d.accept, V, total, s));
  else FST_TRY(score_total(c, fb, d.start, V, total, s));
  c->have_score_times = c->timing;
  return done ? FST_OK : FST_ERR_NOT_CONVERGED;
}

ScoreGraph plain_score_graph(const DevGraph &d) {
  ScoreGraph SG = {};
  SG.V = d.V;
  SG.E = d.E;
  SG.off = d.off;
  SG.src = d.src;
  SG.dst = d.dst;
  SG.w = d.w;
  SG.start = d.start;
  SG.accept = d.accept;
  return SG;
}

// The forward search (generations from g0 on) and an unrestricted backward
// search (from every accepting key pair, seeded by the caller) side by side,
// both advanced by the same kernels; once the forward search has ended, the
// remaining backward generations expand only accessible keys and run alone.
// The trim set is the keys both reached.
// Accepting pairs up to which the concurrent order starts both searches at
// once.
constexpr unsigned long long FEW_ACCEPTING_PAIRS = 1024;

int search_concurrent(fst_ctx *c, Problem P, const SearchArgs &SF, const SearchArgs &SB, int g0,
                      hipStream_t s) {
  const KernelTimer t = timer(c, FST_KERNEL_SEARCH_FORWARD);
  int gf = g0, gb = 0;  // each search numbers its own generations
  bool fdone = false, bdone = false, pause = false, first = true;
  for (;;) {
    // the one search left after the other ends is usually near its end too;
    // the first batch covers as many launches as the last search took
    int batch = fdone || bdone ? 8 : 16;
    if (first && c->gen_hint > batch) batch = c->gen_hint < 256 ? c->gen_hint : 256;
    first = false;
    t.begin(s);
    for (int b = 0; b < batch; ++b) {
      if (!fdone && !bdone && !pause) HIP_TRY(launch_generation2(P, SF, SB, gf++, gb++, s));
      else if (!fdone) HIP_TRY(launch_generation(P, SF, true, gf++, s));
      else HIP_TRY(launch_generation(P, SB, false, gb++, s));
    }
    t.end(s);
    FST_TRY(readback(c, s));
    FST_TRY(add_time(c, FST_KERNEL_SEARCH_FORWARD, batch));
    if (c->h_sc->overflow) return FST_ERR_TOO_LARGE;
    const GenSlot &nf = c->h_sc->G[gf % 3], &nb = c->h_sc->G2[gb % 3];
    fdone = fdone || (nf.qcount == 0 && (uint32_t)nf.hpack == 0);
    bdone = bdone || (nb.qcount == 0 && (uint32_t)nb.hpack == 0);
    if (fdone) P.restrict_bwd = 1;  // the accessible set is complete
    // an unrestricted backward frontier far wider than the forward one is
    // mostly keys that are not accessible: the backward search waits (its
    // frontier stays in its slot) until the forward search has ended
    const unsigned long long wf = nf.qcount + (nf.hpack >> 32), wb = nb.qcount + (nb.hpack >> 32);
    pause = pause || (!fdone && wb > 4 * wf + 65536);
    if (fdone && bdone) break;
    // (no growth: a read-back every 16 generations costs less than the
    // empty launches a larger batch leaves after the searches end)
  }
  c->stats.fwd_levels = c->h_sc->gens;
  c->stats.bwd_levels = c->h_sc->gens2;
  // launches that found work (both searches side by side from g0 on)
  const int fl = (int)c->h_sc->gens - g0, bl = (int)c->h_sc->gens2;
  c->gen_hint = fl > bl ? fl : bl;
  return FST_OK;
}

// Label buckets are kept when the table is at most this large, and at most
// LUT_PER_ARC times the size of the graph's arc records (a graph with few
// arcs per state finds a label in its short groups about as fast, and its
// table would cost more to build than it saves); chain records of each view
// of B are kept up to CHAIN_BUDGET.
constexpr size_t LUT_BUDGET = (size_t)256 << 20;
constexpr size_t LUT_PER_ARC = 64;
constexpr size_t CHAIN_BUDGET = (size_t)256 << 20;

size_t lut_bytes(int32_t V, uint32_t lab_max) {
  return (size_t)V * ((size_t)lab_max + 1) * sizeof(int4);
}

bool want_lut(const fst_ctx *c, int32_t V, int32_t E, uint32_t lab_max) {
  const size_t b = lut_bytes(V, lab_max);
  return c->buckets && b <= LUT_BUDGET && b <= LUT_PER_ARC * (size_t)E * sizeof(int2);
}

int run_impl(fst_ctx *c, const fst_graph *A, const fst_graph *B, hipStream_t s, int64_t *V_C,
             int64_t *E_C) {
  FST_TRY(check_graph_args(A));
  FST_TRY(check_graph_args(B));
  const DevGraph dA = dev_graph(A), dB = dev_graph(B);
  const int32_t VA = dA.V, VB = dB.V, EA = dA.E, EB = dB.E;

  FST_TRY(ensure(c, c->scal, sizeof(Scalars)));
  Scalars *d_sc = as<Scalars>(c->scal);
  for (int k = 0; k < NKERNELS; ++k) {
    c->kms[k] = 0.f;
    c->klaunches[k] = 0;
  }
  phase_begin(c, PH_PRE, s);
  HIP_TRY(hipMemsetAsync(d_sc, 0, sizeof(Scalars), s));
  if (VA)
    HIP_TRY(launch_validate(dA, 0, &d_sc->errA, &d_sc->maxLabA, s, &d_sc->naccA, c->validate));
  if (VB)
    HIP_TRY(launch_validate(dB, 1, &d_sc->errB, &d_sc->maxLabB, s, &d_sc->naccB, c->validate));
  FST_TRY(readback(c, s));
  const uint32_t info_bits = 1u << 16;  // validation's "not in label order" note
  if ((c->h_sc->errA & ~info_bits) || (c->h_sc->errB & ~info_bits)) return FST_ERR_INVALID_GRAPH;
  const bool presortedA = !(c->h_sc->errA & info_bits), presortedB = !(c->h_sc->errB & info_bits);
  c->stats = fst_stats{};
  if (VA == 0 || VB == 0) return finish_empty(c, V_C, E_C);

  // state ids share their arc-record word with two flag bits
  if (VA > NBR_MASK || VB > NBR_MASK) return FST_ERR_TOO_LARGE;
  // at least 4 bits, so that a key-order bitmap word holds keys of one A state
  const int bitsB = bitlen((unsigned long long)(VB - 1));
  const uint32_t shiftB = (uint32_t)(bitsB > 4 ? bitsB : 4);
  const unsigned long long nkeys = (unsigned long long)VA << (shiftB + 1);
  // the search bitmaps' diagonal layout: rows of A states rounded up to 64
  const unsigned long long rowA = ((unsigned long long)VA + 63) / 64 * 64;
  const unsigned long long nsbits = rowA << (shiftB + 1);
  if (nkeys >= (1ull << 32) || nsbits >= (1ull << 32)) return FST_ERR_TOO_LARGE;
  c->stats.key_space = (int64_t)nkeys;
  c->nkeys = nkeys;
  const int labA = bitlen(c->h_sc->maxLabA), labB = bitlen(c->h_sc->maxLabB);

  // ---- label-sorted views ----
  const size_t Emax = (size_t)(EA > EB ? EA : EB);
  FST_TRY(ensure(c, c->k0, Emax * 8));
  FST_TRY(ensure(c, c->k1, Emax * 8));
  FST_TRY(ensure(c, c->v0, Emax * 4));
  FST_TRY(ensure(c, c->v1, Emax * 4));
  FST_TRY(ensure(c, c->sort_tmp, sort_temp_bytes(Emax)));
  const uint32_t maxA = c->h_sc->maxLabA, maxB = c->h_sc->maxLabB;
  const bool lutA = want_lut(c, (int32_t)VA, (int32_t)EA, maxA);
  const bool lutB = want_lut(c, (int32_t)VB, (int32_t)EB, maxB);
  struct ViewBufs {
    DevBuf *perm, *arc, *rec, *lut, *off, *lab, *w;
  };
  // built in this order: A's in-view needs A's out-view records
  const ViewBufs vb[4] = {
      {&c->aOutPerm, &c->aOutArc, &c->aOutRec, &c->aOutLut, nullptr, &c->aOutLab, &c->aOutW},
      {&c->bOutPerm, &c->bOutArc, &c->bOutRec, &c->bOutLut, nullptr, &c->bOutLab, &c->bOutW},
      {&c->aInPerm, &c->aInArc, &c->aInRec, &c->aInLut, &c->aInOff, nullptr, nullptr},
      {&c->bInPerm, &c->bInArc, &c->bInRec, &c->bInLut, &c->bInOff, nullptr, nullptr}};
  unsigned long long *k0 = as<unsigned long long>(c->k0), *k1 = as<unsigned long long>(c->k1);
  int32_t *v0 = as<int32_t>(c->v0), *v1 = as<int32_t>(c->v1);
  int4 *rec[4], *lutp[4];
  int2 *arc[4];
  int32_t *perm[4], *olab[4];
  float *wv[4];
  for (int i = 0; i < 4; ++i) {
    const bool isA = (i % 2) == 0, in = i >= 2;
    const DevGraph &g = isA ? dA : dB;
    const bool lut = isA ? lutA : lutB;
    FST_TRY(ensure(c, *vb[i].perm, (size_t)g.E * sizeof(int32_t)));
    FST_TRY(ensure(c, *vb[i].arc, (size_t)g.E * sizeof(int2)));
    FST_TRY(ensure(c, *vb[i].rec, (size_t)g.V * 2 * sizeof(int4)));
    if (lut) FST_TRY(ensure(c, *vb[i].lut, lut_bytes(g.V, isA ? maxA : maxB)));
    if (in) FST_TRY(ensure(c, *vb[i].off, ((size_t)g.V + 1) * sizeof(int32_t)));
    olab[i] = nullptr;
    wv[i] = nullptr;
    if (!in) {
      FST_TRY(ensure(c, *vb[i].lab, (size_t)g.E * sizeof(int32_t)));
      FST_TRY(ensure(c, *vb[i].w, (size_t)g.E * sizeof(float)));
      olab[i] = as<int32_t>(*vb[i].lab);
      wv[i] = as<float>(*vb[i].w);
    }
    rec[i] = as<int4>(*vb[i].rec);
    arc[i] = as<int2>(*vb[i].arc);
    perm[i] = as<int32_t>(*vb[i].perm);
    lutp[i] = lut ? as<int4>(*vb[i].lut) : nullptr;
  }
  for (int i = 0; i < 4; ++i) {
    const bool isA = (i % 2) == 0, in = i >= 2;
    HIP_TRY(sort_view(isA ? dA : dB, isA ? 0 : 1, in, isA ? presortedA : presortedB,
                      isA ? labA : labB, rec[i], arc[i], perm[i], olab[i], wv[i],
                      in ? as<int32_t>(*vb[i].off) : nullptr, i == 2 ? rec[0] : nullptr, k0, v0,
                      k1, v1, c->sort_tmp.p, nullptr, s));
  }
  // a view's FLAG_UNIQ comes from the opposite view (i ^ 2) of the same graph
  ViewJobs J = {};
  View views[4];
  for (int i = 0; i < 4; ++i) {
    const bool isA = (i % 2) == 0, in = i >= 2;
    const DevGraph &g = isA ? dA : dB;
    const uint32_t lmax = isA ? maxA : maxB;
    // chain records for B's views, when they fit the budget
    int4 *chain = nullptr;
    if (!isA && (size_t)g.V * CHAIN_INT4 * sizeof(int4) <= CHAIN_BUDGET) {
      FST_TRY(ensure(c, in ? c->bInChain : c->bOutChain, (size_t)g.V * CHAIN_INT4 * sizeof(int4)));
      chain = as<int4>(in ? c->bInChain : c->bOutChain);
    }
    J.j[i] = ViewJob{rec[i], arc[i], lutp[i], rec[i ^ 2], arc[i ^ 2], in ? g.accept : g.start,
                     isA ? 0 : 1, in ? 0 : 1, (int32_t)lmax + 1, chain};
    J.vbegin[i + 1] = J.vbegin[i] + g.V;
    J.ebegin[i + 1] = J.ebegin[i] + g.E;
    J.lbegin[i + 1] = J.lbegin[i] + (lutp[i] ? (long long)g.V * ((long long)lmax + 1) : 0);
    views[i] = View{rec[i], arc[i], perm[i], lutp[i], (int32_t)lmax + 1, olab[i], wv[i], chain};
  }
  HIP_TRY(finish_views(J, s));

  // ---- search state ----
  const size_t nwords = (size_t)((nkeys + 31) / 32);  // key-order bitmaps
  const size_t snwords = (size_t)(nsbits / 32);          // search bitmaps
  // Every list holds at most one entry per key, so 2 V_A V_B (f = 1 only
  // where epsOutA) bounds them; what a search pushes (frontier and heavy
  // keys, the accepting keys it meets) is far less when its threads follow
  // keys depth-first.  The lists start at FST_OPT_LIST_CAPACITY entries
  // (2^22 by default), or the size the last call needed, and the searches
  // run again with four times as much when one overflows.
  const unsigned long long capll = 2ull * (unsigned long long)VA * (unsigned long long)VB;
  const unsigned long long cap_full = capll < nkeys ? capll : nkeys;  // <= nkeys < 2^32
  unsigned long long cap_try = c->list_hint ? c->list_hint : c->list_start;
  uint32_t *wbase = nullptr;
  for (;;) {
    const uint32_t cap = (uint32_t)(cap_try < cap_full ? cap_try : cap_full);
    auto searches = [&]() -> int {
    FST_TRY(ensure(c, c->vis, snwords * 4));
    FST_TRY(ensure(c, c->coacc, snwords * 4));
    FST_TRY(ensure(c, c->trim, nwords * 4));
    FST_TRY(ensure(c, c->wbase, nwords * 4));
    FST_TRY(ensure(c, c->fq, (size_t)cap * 4));
    FST_TRY(ensure(c, c->bq, (size_t)cap * 4));
    FST_TRY(ensure(c, c->heavy, (size_t)cap * 4));
    FST_TRY(ensure(c, c->hoff, (size_t)cap * 4));
    if (c->order == FST_ORDER_CONCURRENT) {
      FST_TRY(ensure(c, c->heavy2, (size_t)cap * 4));
      FST_TRY(ensure(c, c->hoff2, (size_t)cap * 4));
    }
    FST_TRY(ensure(c, c->lists, ((size_t)VA + VB + 2) * 4));
    size_t scan_n = nwords > (size_t)cap + 1 ? nwords : (size_t)cap + 1;
    FST_TRY(ensure(c, c->scan_tmp, scan_temp_bytes(scan_n)));
    HIP_TRY(hipMemsetAsync(c->vis.p, 0, snwords * 4, s));
    HIP_TRY(hipMemsetAsync(c->coacc.p, 0, snwords * 4, s));

    Problem &P = c->P;
    P = Problem{};
    P.A = dA;
    P.B = dB;
    P.aOut = views[0];
    P.bOut = views[1];
    P.aIn = views[2];
    P.bIn = views[3];
    P.shiftB = shiftB;
    P.maskB = (1u << shiftB) - 1u;
    P.rowA = (uint32_t)rowA;
    P.chain_max = c->chain_depth;
    P.mark_accept = 1;
    P.vis = as<uint32_t>(c->vis);
    P.coacc = as<uint32_t>(c->coacc);
    P.trim = as<uint32_t>(c->trim);
    P.wbase = as<uint32_t>(c->wbase);

    // ---- the two searches ----
    int32_t *la = as<int32_t>(c->lists), *lb = la + VA;
    uint32_t *cnts = reinterpret_cast<uint32_t *>(lb + VB);
    uint32_t *fq = as<uint32_t>(c->fq), *bq = as<uint32_t>(c->bq);
    SearchArgs S;
    S.Q = fq;
    S.heavy = as<uint32_t>(c->heavy);
    S.hoff = as<uint32_t>(c->hoff);
    S.acc = bq;
    S.cap = cap;
    S.sc = d_sc;
    S.G = d_sc->G;
    S.gens = &d_sc->gens;
    wbase = as<uint32_t>(c->wbase);
    phase_end(c, PH_PRE, s);
    if (c->order == FST_ORDER_CONCURRENT) {
      // The forward search's first generations run alone (listing accepting
      // keys as in the forward-first order).  If it has ended by then, the
      // backward search follows as in that order; otherwise a backward search
      // from every accepting pair runs beside the rest of it.
      // With few accepting pairs the backward search starts at once (its
      // seeds cannot outnumber much of the forward work).
      const int FIRST =
          (unsigned long long)c->h_sc->naccA * c->h_sc->naccB <= FEW_ACCEPTING_PAIRS ? 0 : 4;
      P.restrict_fwd = 0;
      P.restrict_bwd = 0;
      phase_begin(c, PH_FWD, s);
      // the generation slots are still zero from the run's first memset
      HIP_TRY(hipMemsetAsync(cnts, 0, 8, s));
      HIP_TRY(launch_seed_forward(P, S, la, cnts, lb, cnts + 1, s));
      const KernelTimer tf = timer(c, FST_KERNEL_SEARCH_FORWARD);
      tf.begin(s);
      for (int g = 0; g < FIRST; ++g) HIP_TRY(launch_generation(P, S, true, g, s));
      tf.end(s);
      // with no generation run alone there is nothing to read back yet (an
      // empty forward search ends in the concurrent loop as well)
      bool fwd_over = false;
      if (FIRST > 0) {
        FST_TRY(readback(c, s));
        FST_TRY(add_time(c, FST_KERNEL_SEARCH_FORWARD, FIRST));
        if (c->h_sc->overflow) return FST_ERR_TOO_LARGE;
        const GenSlot &nf = c->h_sc->G[FIRST % 3];
        fwd_over = nf.qcount == 0 && (uint32_t)nf.hpack == 0;
      }
      if (fwd_over) {
        c->stats.fwd_levels = c->h_sc->gens;
        HIP_TRY(launch_popcount(P.vis, snwords, &d_sc->naccessible, s));
        if (c->count_moves) HIP_TRY(launch_count_moves(P, snwords, true, &d_sc->generated, s));
        phase_end(c, PH_FWD, s);
        phase_begin(c, PH_BWD, s);
        P.restrict_bwd = 1;
        HIP_TRY(hipMemsetAsync(d_sc->G, 0, sizeof(d_sc->G), s));
        HIP_TRY(launch_seed_backward(P, S, bq, s));
        FST_TRY(search(c, S, false, &c->stats.bwd_levels, s));
        HIP_TRY(launch_trim(P, (uint32_t)VA, as<uint32_t>(c->trim), wbase, s));
        phase_end(c, PH_BWD, s);
      } else {
        P.mark_accept = 0;  // the backward seeds below are every accepting pair
        SearchArgs SB = S;
        SB.Q = bq;  // the forward search's list of accepting keys is not needed
        SB.heavy = as<uint32_t>(c->heavy2);
        SB.hoff = as<uint32_t>(c->hoff2);
        SB.acc = nullptr;
        SB.G = d_sc->G2;
        SB.gens = &d_sc->gens2;
        HIP_TRY(hipMemsetAsync(cnts, 0, 8, s));
        HIP_TRY(launch_seed_backward_all(P, SB, la, cnts, lb, cnts + 1, s));
        FST_TRY(search_concurrent(c, P, S, SB, FIRST, s));
        HIP_TRY(launch_popcount(P.vis, snwords, &d_sc->naccessible, s));
        if (c->count_moves) HIP_TRY(launch_count_moves(P, snwords, true, &d_sc->generated, s));
        phase_end(c, PH_FWD, s);
        // the backward phase is the final intersection only
        phase_begin(c, PH_BWD, s);
        HIP_TRY(launch_trim(P, (uint32_t)VA, as<uint32_t>(c->trim), wbase, s));
        phase_end(c, PH_BWD, s);
      }
    } else if (c->order == FST_ORDER_COACCESSIBLE_FIRST) {
      // Algorithm 1's order: the co-accessible set over all key pairs first,
      // from every accepting pair, then the forward search inside it
      P.restrict_fwd = 1;
      P.restrict_bwd = 0;
      phase_begin(c, PH_BWD, s);
      HIP_TRY(hipMemsetAsync(cnts, 0, 8, s));
      HIP_TRY(hipMemsetAsync(d_sc->G, 0, sizeof(d_sc->G), s));
      HIP_TRY(launch_seed_backward_all(P, S, la, cnts, lb, cnts + 1, s));
      FST_TRY(search(c, S, false, &c->stats.bwd_levels, s));
      phase_end(c, PH_BWD, s);
      phase_begin(c, PH_FWD, s);
      HIP_TRY(hipMemsetAsync(cnts, 0, 8, s));
      HIP_TRY(hipMemsetAsync(d_sc->G, 0, sizeof(d_sc->G), s));
      HIP_TRY(launch_seed_forward(P, S, la, cnts, lb, cnts + 1, s));
      FST_TRY(search(c, S, true, &c->stats.fwd_levels, s));
      HIP_TRY(launch_popcount(P.vis, snwords, &d_sc->naccessible, s));
      if (c->count_moves) HIP_TRY(launch_count_moves(P, snwords, true, &d_sc->generated, s));
      HIP_TRY(launch_trim(P, (uint32_t)VA, as<uint32_t>(c->trim), wbase, s));
      phase_end(c, PH_FWD, s);
    } else {
      P.restrict_fwd = 0;
      P.restrict_bwd = 1;
      phase_begin(c, PH_FWD, s);
      HIP_TRY(hipMemsetAsync(cnts, 0, 8, s));
      HIP_TRY(hipMemsetAsync(d_sc->G, 0, sizeof(d_sc->G), s));
      HIP_TRY(launch_seed_forward(P, S, la, cnts, lb, cnts + 1, s));
      FST_TRY(search(c, S, true, &c->stats.fwd_levels, s));
      HIP_TRY(launch_popcount(P.vis, snwords, &d_sc->naccessible, s));
      if (c->count_moves) HIP_TRY(launch_count_moves(P, snwords, true, &d_sc->generated, s));
      phase_end(c, PH_FWD, s);

      // backward search, seeded by the accepting keys listed in bq
      phase_begin(c, PH_BWD, s);
      HIP_TRY(hipMemsetAsync(d_sc->G, 0, sizeof(d_sc->G), s));
      HIP_TRY(launch_seed_backward(P, S, bq, s));
      FST_TRY(search(c, S, false, &c->stats.bwd_levels, s));
      // the backward search may set co-accessible bits of keys it never
      // expands (not accessible); the trim set is what remains after masking
      // them, and the same pass counts the trim keys of every bitmap word
      HIP_TRY(launch_trim(P, (uint32_t)VA, as<uint32_t>(c->trim), wbase, s));
      phase_end(c, PH_BWD, s);
    }
    if (c->count_moves) HIP_TRY(launch_count_moves(P, nwords, false, &d_sc->generated_bwd, s));

      return FST_OK;
    };
    const int rc = searches();
    if (rc == FST_ERR_TOO_LARGE && c->h_sc->overflow && (unsigned long long)cap < cap_full) {
      cap_try = 4ull * cap;
      // the search scalars start again from zero (validation's stay)
      HIP_TRY(hipMemsetAsync(&d_sc->tail2, 0, sizeof(uint32_t), s));
      HIP_TRY(hipMemsetAsync(&d_sc->heavy, 0,
                             offsetof(Scalars, gens2) + sizeof(uint32_t) -
                                 offsetof(Scalars, heavy), s));
      continue;
    }
    FST_TRY(rc);
    c->list_hint = cap;
    break;
  }
  if (!wbase) return FST_ERR_HIP;  // the searches set it; never launch on a null buffer

  // ---- numbering and arc counts ----
  phase_begin(c, PH_COUNT, s);
  HIP_TRY(scan_u32(wbase, wbase, nwords, false, &d_sc->total, c->scan_tmp.p, s));
  FST_TRY(readback(c, s));
  const unsigned long long nst = c->h_sc->total;
  if (nst > (unsigned long long)INT32_MAX) return FST_ERR_TOO_LARGE;
  const uint32_t nstates = (uint32_t)nst;
  // the search lists are free now: the forward queue takes the counts of
  // 255 arcs or more, the backward queue the heavy states (id, key)
  FST_TRY(ensure(c, c->fq, ((size_t)nstates + 1) * 4));
  FST_TRY(ensure(c, c->bq, ((size_t)nstates + 1) * 8));
  uint32_t *cnt32 = as<uint32_t>(c->fq);
  uint2 *heavy = as<uint2>(c->bq);
  const Problem &P = c->P;
  const size_t nchunks = out_chunks(nwords);
  FST_TRY(ensure(c, c->cnt, (size_t)nstates + 1));
  FST_TRY(ensure(c, c->btot, (nchunks + 1) * 4));
  FST_TRY(ensure(c, c->scan_tmp, scan_temp_bytes(nchunks + 1)));
  uint8_t *cnt8 = as<uint8_t>(c->cnt);
  uint32_t *btot = as<uint32_t>(c->btot);
  HIP_TRY(hipMemsetAsync(&d_sc->heavy, 0, sizeof(uint32_t), s));
  HIP_TRY(hipMemsetAsync(&d_sc->total, 0, sizeof(unsigned long long), s));
  const KernelTimer tc = timer(c, FST_KERNEL_COUNT);
  tc.begin(s);
  if (nstates) {
    HIP_TRY(launch_count(P, nwords, cnt8, cnt32, btot, heavy, d_sc, s));
    HIP_TRY(launch_count_heavy(P, heavy, &d_sc->heavy, cnt8, cnt32, btot, s));
  }
  tc.end(s);
  // exclusive arc offset of every chunk; the total is E_C
  if (nstates)
    HIP_TRY(scan_u32(btot, btot, nchunks, false, &d_sc->total, c->scan_tmp.p, s));
  phase_end(c, PH_COUNT, s);
  FST_TRY(readback(c, s));
  const unsigned long long narcs = c->h_sc->total;
  if (narcs > (unsigned long long)INT32_MAX) return FST_ERR_TOO_LARGE;
  FST_TRY(add_time(c, FST_KERNEL_COUNT, nstates ? 2 : 1));

  c->nstates = nstates;
  c->out_words = nwords;
  c->narcs = (uint32_t)narcs;
  c->nheavy = c->h_sc->heavy;
  c->stats.accessible = (int64_t)c->h_sc->naccessible;
  c->stats.generated = c->count_moves ? (int64_t)c->h_sc->generated : -1;
  c->stats.generated_backward = c->count_moves ? (int64_t)c->h_sc->generated_bwd : -1;
  c->stats.coaccessible = nstates;
  c->stats.heavy_states = c->nheavy;
  c->stats.num_states = nstates;
  c->stats.num_arcs = (int64_t)narcs;
  c->timed_run = c->timing;
  c->ready = true;
  *V_C = nstates;
  *E_C = (int64_t)narcs;
  return FST_OK;
}

// ---------------------------------------------------------------------------
// three inputs
// ---------------------------------------------------------------------------

int readback3(fst_ctx *c, hipStream_t s) {
  HIP_TRY(hipMemcpyAsync(c->h_s3, c->t_scal.p, sizeof(Scal3), hipMemcpyDeviceToHost, s));
  HIP_TRY(hipStreamSynchronize(s));
  return FST_OK;
}

// One label-sorted out-view of g (side 0: by olabel, 1: by ilabel) into the
// given buffers; lab/w (the other side's label and the weight in sorted
// order) only when lab is given.
int view3(fst_ctx *c, const DevGraph &g, int side, bool presorted, uint32_t maxlab, DevBuf &perm,
          DevBuf &arc, DevBuf &rec, DevBuf *lab, DevBuf *w, DevBuf &lut, View &v, hipStream_t s) {
  FST_TRY(ensure(c, perm, (size_t)g.E * 4));
  FST_TRY(ensure(c, arc, (size_t)g.E * 8));
  FST_TRY(ensure(c, rec, (size_t)g.V * 2 * sizeof(int4)));
  int32_t *olab = nullptr;
  float *wv = nullptr;
  if (lab) {
    FST_TRY(ensure(c, *lab, (size_t)g.E * 4));
    FST_TRY(ensure(c, *w, (size_t)g.E * 4));
    olab = as<int32_t>(*lab);
    wv = as<float>(*w);
  }
  HIP_TRY(sort_view(g, side, false, presorted, bitlen(maxlab), as<int4>(rec), as<int2>(arc),
                    as<int32_t>(perm), olab, wv, nullptr, nullptr, as<unsigned long long>(c->k0),
                    as<int32_t>(c->v0), as<unsigned long long>(c->k1), as<int32_t>(c->v1),
                    c->sort_tmp.p, nullptr, s));
  v = View{as<int4>(rec), as<int2>(arc), as<int32_t>(perm), nullptr, 0, olab, wv, nullptr};
  // bucket table under the same budget as the two-input views
  if (want_lut(c, g.V, g.E, maxlab)) {
    FST_TRY(ensure(c, lut, lut_bytes(g.V, maxlab)));
    v.lut = as<int4>(lut);
    v.lstride = (int32_t)maxlab + 1;
    HIP_TRY(launch3_lut(v, g.V, s));
  }
  return FST_OK;
}

// Levels of a three-input search in batches with one read-back after each
// batch; *done tells whether it ended (false: a capacity was exceeded).
// The first batch is as many levels as the last search in this direction
// took (at least 4), then 16, 32, 64, 64, ...
int levels3(fst_ctx *c, const Problem3 &P, const Search3 &S, bool forward, uint32_t grow_at,
            bool *done, hipStream_t s) {
  const KernelTimer t = timer(c, FST_KERNEL_SEARCH3);
  int &hint = c->lv3_hint[forward ? 1 : 0];
  int g = 0, batch = hint > 4 ? (hint < 256 ? hint : 256) : 4;
  *done = false;
  for (;;) {
    t.begin(s);
    for (int b = 0; b < batch; ++b, ++g) HIP_TRY(launch3_level(P, S, forward, g, s));
    t.end(s);
    FST_TRY(readback3(c, s));
    FST_TRY(add_time(c, FST_KERNEL_SEARCH3, 2 * batch));
    const Lvl3 &nx = c->h_s3->ring[g % 3];
    // keys in the set: those of the frontiers and those walks went on to
    if (c->h_s3->overflow ||
        (unsigned long long)nx.fbase + nx.fcount + c->h_s3->ncont > grow_at)
      return FST_OK;
    // walks that reach a heavy key leave it as a chunk of the next level:
    // a level can hold chunks and no frontier
    if (nx.fcount == 0 && nx.ccount == 0) break;
    batch = batch < 16 ? 16 : (batch < 64 ? 2 * batch : 64);
  }
  hint = (int)c->h_s3->levels;
  *done = true;
  return FST_OK;
}

int compose3_impl(fst_ctx *c, const fst_graph *A, const fst_graph *B, const fst_graph *D,
                  hipStream_t s, int64_t *V_C, int64_t *E_C) {
  FST_TRY(check_graph_args(A));
  FST_TRY(check_graph_args(B));
  FST_TRY(check_graph_args(D));
  const DevGraph dA = dev_graph(A), dB = dev_graph(B), dD = dev_graph(D);
  FST_TRY(ensure(c, c->t_scal, sizeof(Scal3)));
  Scal3 *d3 = as<Scal3>(c->t_scal);
  for (int k = 6; k < NKERNELS; ++k) {
    c->kms[k] = 0.f;
    c->klaunches[k] = 0;
  }
  HIP_TRY(hipMemsetAsync(d3, 0, sizeof(Scal3), s));
  if (dA.V) HIP_TRY(launch_validate(dA, 0, &d3->errA, &d3->maxA, s, nullptr, c->validate));
  if (dB.V) HIP_TRY(launch_validate(dB, 1, &d3->errB, &d3->maxB, s, nullptr, c->validate));
  if (dD.V) HIP_TRY(launch_validate(dD, 1, &d3->errD, &d3->maxD, s, nullptr, c->validate));
  FST_TRY(readback3(c, s));
  const uint32_t info = 1u << 16;  // validation's "not in label order" note
  const Scal3 v = *c->h_s3;
  if ((v.errA & ~info) || (v.errB & ~info) || (v.errD & ~info)) return FST_ERR_INVALID_GRAPH;
  c->c3.stats = fst_stats{};
  if (dA.V == 0 || dB.V == 0 || dD.V == 0) {
    c->c3.n = c->c3.U = c->c3.narcs = 0;
    c->c3.ready = true;
    return FST_OK;
  }
  if (dA.V > NBR_MASK || dB.V > NBR_MASK || dD.V > NBR_MASK) return FST_ERR_TOO_LARGE;
  const int bA = bitlen((unsigned long long)(dA.V - 1)) > 0 ? bitlen((unsigned long long)(dA.V - 1)) : 1;
  const int bB = bitlen((unsigned long long)(dB.V - 1)) > 0 ? bitlen((unsigned long long)(dB.V - 1)) : 1;
  const int bD = bitlen((unsigned long long)(dD.V - 1)) > 0 ? bitlen((unsigned long long)(dD.V - 1)) : 1;
  const int kbits = bA + bB + bD + 2;
  if (kbits > 62) return FST_ERR_TOO_LARGE;
  c->c3.stats.key_space = (int64_t)1 << kbits;

  // label-sorted views
  int32_t EA = dA.E, EB = dB.E, ED = dD.E;
  const size_t Emax = (size_t)(EA > EB ? (EA > ED ? EA : ED) : (EB > ED ? EB : ED));
  FST_TRY(ensure(c, c->k0, Emax * 8));
  FST_TRY(ensure(c, c->k1, Emax * 8));
  FST_TRY(ensure(c, c->v0, Emax * 4));
  FST_TRY(ensure(c, c->v1, Emax * 4));
  FST_TRY(ensure(c, c->sort_tmp, sort_temp_bytes(Emax)));
  Problem3 P = {};
  P.A = dA;
  P.B = dB;
  P.D = dD;
  FST_TRY(view3(c, dA, 0, !(v.errA & info), v.maxA, c->t_aPerm, c->t_aArc, c->t_aRec,
                &c->t_aLab, &c->t_aW, c->t_aLut, P.aOut, s));
  FST_TRY(view3(c, dB, 1, !(v.errB & info), v.maxB, c->t_bPerm, c->t_bArc, c->t_bRec,
                &c->t_bLab, &c->t_bW, c->t_bLut, P.bOut, s));
  FST_TRY(view3(c, dD, 1, !(v.errD & info), v.maxD, c->t_dPerm, c->t_dArc, c->t_dRec,
                &c->t_dLab, &c->t_dW, c->t_dLut, P.dOut, s));
  // chain records of B for the search's chain jumps (which look up A's
  // buckets: only with A's bucket table)
  if (P.aOut.lut) {
    FST_TRY(ensure(c, c->t_bChain, (size_t)dB.V * CHAIN_INT4 * sizeof(int4)));
    P.bOut.chain = as<int4>(c->t_bChain);
    HIP_TRY(launch3_chains(P.bOut, dB.V, as<int4>(c->t_bChain), s));
  }
  FST_TRY(ensure(c, c->t_bflags, (size_t)dB.V * 4));
  HIP_TRY(hipMemsetAsync(c->t_bflags.p, 0, (size_t)dB.V * 4, s));
  HIP_TRY(launch3_bflags(dB, as<uint32_t>(c->t_bflags), s));
  P.bflags = as<uint32_t>(c->t_bflags);
  P.shB = (uint32_t)bB;
  P.shD = (uint32_t)bD;
  FST_TRY(ensure(c, c->t_lists, ((size_t)dA.V + dB.V + dD.V) * 4 + 16));
  int32_t *lists = as<int32_t>(c->t_lists);
  uint32_t *counts = reinterpret_cast<uint32_t *>(lists + dA.V + dB.V + dD.V);

  // forward search; a table that fills up (or lists that overflow) is
  // grown two-fold and the search starts again (the later passes scan the
  // whole table: a smaller one pays off more than the longer first call)
  const KernelTimer tout = timer(c, FST_KERNEL_COMPACT3);
  unsigned long long H = c->h3_hint ? c->h3_hint : (1ull << 20);
  Search3 S = {};
  for (;;) {
    if (H > (1ull << 31)) return FST_ERR_TOO_LARGE;
    const unsigned long long acap = 4 * H;
    FST_TRY(ensure(c, c->t_tab, H * 8));
    FST_TRY(ensure(c, c->t_F, H * 4));
    FST_TRY(ensure(c, c->t_chunks, 2 * H * 8));
    FST_TRY(ensure(c, c->t_arcs, acap * 8));
    HIP_TRY(hipMemsetAsync(c->t_tab.p, 0xff, H * 8, s));
    HIP_TRY(hipMemsetAsync(&d3->overflow, 0, offsetof(Scal3, ring) - offsetof(Scal3, overflow) +
                                                 sizeof(d3->ring), s));
    HIP_TRY(hipMemsetAsync(counts, 0, 3 * 4, s));
    P.tab = as<unsigned long long>(c->t_tab);
    P.hmask = (uint32_t)(H - 1);
    S.F = as<uint32_t>(c->t_F);
    S.fcap = (uint32_t)H;
    S.chunks = as<uint2>(c->t_chunks);
    S.ccap = (uint32_t)H;
    S.arcs = as<uint2>(c->t_arcs);
    S.acap = acap;
    S.ring = d3->ring;
    // chain segments of the jumps for the backward search (a quarter of the
    // table's size, below 2^28 so that seg_of packs the index with the
    // length; jumps past that record none)
    if (P.bOut.chain) {
      const unsigned long long scap = H / 4 < (1ull << 28) ? H / 4 : (1ull << 28) - 1;
      FST_TRY(ensure(c, c->t_segof, H * 4));
      FST_TRY(ensure(c, c->t_segs, scap * 32));
      HIP_TRY(hipMemsetAsync(c->t_segof.p, 0xff, H * 4, s));
      S.segs = as<uint32_t>(c->t_segs);
      S.seg_of = as<uint32_t>(c->t_segof);
      S.scap = (uint32_t)scap;
    }
    S.sc = d3;
    HIP_TRY(launch3_starts(dA, dB, dD, lists, counts, s));
    HIP_TRY(launch3_seed(P, S, lists, counts, s));
    bool done = false;
    // a table at most half full keeps probe sequences short (most keys sit
    // in the first group of four slots they probe)
    FST_TRY(levels3(c, P, S, true, (uint32_t)(H / 2), &done, s));
    if (done) break;
    H *= 2;
  }
  c->h3_hint = (uint32_t)H;
  const Scal3 f = *c->h_s3;
  c->c3.stats.fwd_levels = f.levels;
  const unsigned long long nacc = (f.ring[0].fbase > f.ring[1].fbase
                                       ? (f.ring[0].fbase > f.ring[2].fbase ? f.ring[0].fbase
                                                                            : f.ring[2].fbase)
                                       : (f.ring[1].fbase > f.ring[2].fbase ? f.ring[1].fbase
                                                                            : f.ring[2].fbase)) +
                                  (unsigned long long)f.ncont;
  c->c3.stats.accessible = (int64_t)nacc;
  const unsigned long long narcs = f.narcs;
  c->c3.stats.generated = (int64_t)narcs;

  // backward search over the generated arcs, grouped by target (sorted)
  tout.begin(s);
  FST_TRY(ensure(c, c->t_inoff, (H + 1) * 4));
  FST_TRY(ensure(c, c->t_first, H * 4));
  FST_TRY(ensure(c, c->k0, (narcs + 1) * 8));
  FST_TRY(ensure(c, c->k1, (narcs + 1) * 8));
  FST_TRY(ensure(c, c->v0, (narcs + 1) * 4));
  FST_TRY(ensure(c, c->v1, (narcs + 1) * 4));
  FST_TRY(ensure(c, c->sort_tmp, sort_temp_bytes(narcs + 1)));
  FST_TRY(ensure(c, c->t_coacc, (H / 32 + 1) * 4));
  FST_TRY(ensure(c, c->scan_tmp, scan_temp_bytes(H + 1)));
  // chunks of CHUNK3 in-arcs: a key is chunked at most once
  const unsigned long long ccap = H + narcs / CHUNK3 + 1;
  if (ccap > 0xffffffffull) return FST_ERR_TOO_LARGE;
  FST_TRY(ensure(c, c->t_chunks, 2 * ccap * 8));
  uint32_t *inoff = as<uint32_t>(c->t_inoff);
  HIP_TRY(hipMemsetAsync(inoff, 0, (H + 1) * 4, s));
  bool in_second = false;
  HIP_TRY(launch3_arc_keys(S.arcs, narcs, as<unsigned long long>(c->k0), as<int32_t>(c->v0), s));
  if (narcs)
    HIP_TRY(radix_sort(as<unsigned long long>(c->k0), as<int32_t>(c->v0),
                       as<unsigned long long>(c->k1), as<int32_t>(c->v1), narcs,
                       bitlen(H - 1) > 0 ? bitlen(H - 1) : 1, c->sort_tmp.p, s, &in_second));
  const unsigned long long *tkey = as<unsigned long long>(in_second ? c->k1 : c->k0);
  HIP_TRY(launch3_in_degrees(tkey, narcs, as<uint32_t>(c->t_first), inoff, s));
  HIP_TRY(scan_u32(inoff, inoff, H, true, &d3->total, c->scan_tmp.p, s));
  HIP_TRY(hipMemsetAsync(c->t_coacc.p, 0, (H / 32 + 1) * 4, s));
  HIP_TRY(hipMemsetAsync(&d3->overflow, 0, offsetof(Scal3, ring) - offsetof(Scal3, overflow) +
                                               sizeof(d3->ring), s));
  P.coacc = as<uint32_t>(c->t_coacc);
  P.in_off = inoff;
  // the sorted sources are the in-arc lists
  P.in_src = reinterpret_cast<const uint32_t *>(as<int32_t>(in_second ? c->v1 : c->v0));
  S.chunks = as<uint2>(c->t_chunks);
  S.ccap = (uint32_t)ccap;
  tout.end(s);
  HIP_TRY(launch3_seed_bwd(P, S, s));
  bool done = false;
  FST_TRY(levels3(c, P, S, false, 0xffffffffu, &done, s));
  if (!done) return FST_ERR_TOO_LARGE;  // every list holds each slot at most once
  c->c3.stats.bwd_levels = c->h_s3->levels;
  FST_TRY(add_time(c, FST_KERNEL_COMPACT3, 1));

  // trim keys, sorted: a state's id is its rank
  tout.begin(s);
  FST_TRY(ensure(c, c->t_keys0, (nacc + 1) * 8));
  FST_TRY(ensure(c, c->t_keys1, (nacc + 1) * 8));
  FST_TRY(ensure(c, c->t_slots0, (nacc + 1) * 4));
  FST_TRY(ensure(c, c->t_slots1, (nacc + 1) * 4));
  FST_TRY(ensure(c, c->sort_tmp, sort_temp_bytes(nacc + 1)));
  HIP_TRY(hipMemsetAsync(&d3->ntrim, 0, 4, s));
  HIP_TRY(launch3_collect(P, as<unsigned long long>(c->t_keys0), as<int32_t>(c->t_slots0),
                          &d3->ntrim, (uint32_t)nacc, &d3->overflow, s));
  tout.end(s);
  FST_TRY(readback3(c, s));
  FST_TRY(add_time(c, FST_KERNEL_COMPACT3, 1));
  if (c->h_s3->overflow) return FST_ERR_TOO_LARGE;
  const uint32_t n = c->h_s3->ntrim;
  c->c3.stats.coaccessible = n;
  c->c3.stats.num_states = n;
  c->c3.stats.generated_backward = -1;
  if (n == 0) {
    c->c3.n = c->c3.U = c->c3.narcs = 0;
    c->c3.ready = true;
    return FST_OK;
  }
  tout.begin(s);
  bool second = false;
  HIP_TRY(radix_sort(as<unsigned long long>(c->t_keys0), as<int32_t>(c->t_slots0),
                     as<unsigned long long>(c->t_keys1), as<int32_t>(c->t_slots1), n, kbits,
                     c->sort_tmp.p, s, &second));
  const unsigned long long *keys = as<unsigned long long>(second ? c->t_keys1 : c->t_keys0);
  const int32_t *slots = as<int32_t>(second ? c->t_slots1 : c->t_slots0);
  FST_TRY(ensure(c, c->t_idof, H * 4));
  FST_TRY(ensure(c, c->t_units, ((size_t)n + 1) * 4));
  FST_TRY(ensure(c, c->t_heavy, (size_t)n * 4));
  FST_TRY(ensure(c, c->scan_tmp, scan_temp_bytes((size_t)n + 1)));
  HIP_TRY(hipMemsetAsync(c->t_idof.p, 0xff, H * 4, s));
  HIP_TRY(hipMemsetAsync(d3->nheavy, 0, sizeof(d3->nheavy), s));
  uint32_t *units = as<uint32_t>(c->t_units);
  HIP_TRY(launch3_ids(P, keys, slots, n, as<int32_t>(c->t_idof), units, as<uint32_t>(c->t_heavy),
                      d3->nheavy, s));
  P.id_of = as<int32_t>(c->t_idof);
  HIP_TRY(scan_u32(units, units, n, true, &d3->total, c->scan_tmp.p, s));
  tout.end(s);
  FST_TRY(readback3(c, s));
  FST_TRY(add_time(c, FST_KERNEL_COMPACT3, 1));
  const unsigned long long U = c->h_s3->total;
  if (U >= 0xffffffffull) return FST_ERR_TOO_LARGE;

  // arcs kept by every work unit, scanned into positions
  tout.begin(s);
  FST_TRY(ensure(c, c->t_ucnt, (U + 1) * 4));
  FST_TRY(ensure(c, c->scan_tmp, scan_temp_bytes(U + 1)));
  uint32_t *ucnt = as<uint32_t>(c->t_ucnt);
  HIP_TRY(launch3_count(P, keys, units, n, as<uint32_t>(c->t_heavy), d3->nheavy, ucnt, s));
  HIP_TRY(scan_u32(ucnt, ucnt, U, true, &d3->total, c->scan_tmp.p, s));
  tout.end(s);
  FST_TRY(readback3(c, s));
  FST_TRY(add_time(c, FST_KERNEL_COMPACT3, 1));
  const unsigned long long E = c->h_s3->total;
  if (E > (unsigned long long)INT32_MAX) return FST_ERR_TOO_LARGE;
  c->c3.P = P;
  c->c3.keys = keys;
  c->c3.ustart = units;
  c->c3.uoff = ucnt;
  c->c3.heavy = as<uint32_t>(c->t_heavy);
  c->c3.nheavy = d3->nheavy;
  c->c3.stats.heavy_states = c->h_s3->nheavy[0];
  c->c3.n = n;
  c->c3.U = (uint32_t)U;
  c->c3.narcs = (uint32_t)E;
  c->c3.stats.num_arcs = (int64_t)E;
  c->c3.timed = c->timing;
  c->have_times3 = c->timing;
  c->c3.ready = true;
  *V_C = n;
  *E_C = (int64_t)E;
  return FST_OK;
}

// Batch: validate every item, lay the items out as one disjoint union (state
// and arc offsets shifted), compose the union with B, then find each item's
// state and arc range in C.
// The disjoint union of items A[0 .. n) in the context's union arrays, as
// one graph U (state and arc ids of item i shifted by the items before it).
int build_union(fst_ctx *c, const fst_graph *A, int32_t n, hipStream_t s, fst_graph *U) {
  long long VA = 0, EA = 0;
  for (int32_t i = 0; i < n; ++i) {
    VA += A[i].num_states;
    EA += A[i].num_arcs;
  }
  FST_TRY(ensure(c, c->u_off, ((size_t)VA + 1) * 4));
  FST_TRY(ensure(c, c->u_src, (size_t)EA * 4));
  FST_TRY(ensure(c, c->u_dst, (size_t)EA * 4));
  FST_TRY(ensure(c, c->u_il, (size_t)EA * 4));
  FST_TRY(ensure(c, c->u_ol, (size_t)EA * 4));
  FST_TRY(ensure(c, c->u_w, (size_t)EA * 4));
  FST_TRY(ensure(c, c->u_start, (size_t)VA));
  FST_TRY(ensure(c, c->u_accept, (size_t)VA));
  int32_t *off = as<int32_t>(c->u_off);
  HIP_TRY(hipMemsetAsync(off, 0, 4, s));  // the offsets of an empty union
  long long vb = 0, eb = 0;
  for (int32_t i = 0; i < n; ++i) {
    const DevGraph a = dev_graph(&A[i]);
    if (a.V > 0) {
      HIP_TRY(launch_union_copy(a, vb, eb, off, as<int32_t>(c->u_src), as<int32_t>(c->u_dst), s));
      HIP_TRY(hipMemcpyAsync(as<uint8_t>(c->u_start) + vb, a.start, (size_t)a.V,
                             hipMemcpyDeviceToDevice, s));
      HIP_TRY(hipMemcpyAsync(as<uint8_t>(c->u_accept) + vb, a.accept, (size_t)a.V,
                             hipMemcpyDeviceToDevice, s));
    }
    if (a.E > 0) {
      HIP_TRY(hipMemcpyAsync(as<int32_t>(c->u_il) + eb, a.il, (size_t)a.E * 4,
                             hipMemcpyDeviceToDevice, s));
      HIP_TRY(hipMemcpyAsync(as<int32_t>(c->u_ol) + eb, a.ol, (size_t)a.E * 4,
                             hipMemcpyDeviceToDevice, s));
      HIP_TRY(hipMemcpyAsync(as<float>(c->u_w) + eb, a.w, (size_t)a.E * 4,
                             hipMemcpyDeviceToDevice, s));
    }
    vb += a.V;
    eb += a.E;
  }
  *U = fst_graph{};
  U->num_states = (int32_t)VA;
  U->num_arcs = (int32_t)EA;
  U->arc_offset = off;
  U->src = as<int32_t>(c->u_src);
  U->dst = as<int32_t>(c->u_dst);
  U->ilabel = as<int32_t>(c->u_il);
  U->olabel = as<int32_t>(c->u_ol);
  U->weight = as<float>(c->u_w);
  U->start = as<uint8_t>(c->u_start);
  U->accept = as<uint8_t>(c->u_accept);
  return FST_OK;
}

// Items [i0, i1) composed with B as one union: run, then the first state and
// arc of every item in that run's C (st[i - i0], ar[i - i0]; the last
// entries are the run's V_C and E_C).
int run_items(fst_ctx *c, const fst_graph *A, int32_t i0, int32_t i1, const fst_graph *B,
              hipStream_t s, int64_t *V_C, int64_t *E_C, long long *st, long long *ar) {
  const int32_t n = i1 - i0;
  fst_graph U;
  FST_TRY(build_union(c, A + i0, n, s, &U));
  FST_TRY(run_impl(c, &U, B, s, V_C, E_C));
  if (c->nstates == 0) {
    for (int32_t i = 0; i <= n; ++i) st[i] = ar[i] = 0;
    return FST_OK;
  }
  // qa_base[0..n] (first state of A of each item, then the union's V_A)
  std::vector<long long> h(3 * ((size_t)n + 1), 0);
  long long acc = 0;
  for (int32_t i = 0; i < n; ++i) {
    h[i] = acc;
    acc += A[i0 + i].num_states;
  }
  h[n] = acc;
  FST_TRY(ensure(c, c->u_items, ((size_t)n + 1) * 3 * sizeof(long long)));
  long long *dq = as<long long>(c->u_items), *dout = dq + (n + 1);
  HIP_TRY(hipMemcpyAsync(dq, h.data(), ((size_t)n + 1) * sizeof(long long),
                         hipMemcpyHostToDevice, s));
  HIP_TRY(launch_item_ranges(c->P, c->nkeys, n, dq, as<uint8_t>(c->cnt), as<uint32_t>(c->fq),
                             as<uint32_t>(c->btot), c->nstates, c->narcs, dout, s));
  HIP_TRY(hipMemcpyAsync(h.data() + (n + 1), dout, 2 * ((size_t)n + 1) * sizeof(long long),
                         hipMemcpyDeviceToHost, s));
  HIP_TRY(hipStreamSynchronize(s));
  for (int32_t i = 0; i <= n; ++i) {
    st[i] = h[(n + 1) + i];
    ar[i] = h[2 * (n + 1) + i];
  }
  return FST_OK;
}

void add_stats(fst_stats &t, const fst_stats &p) {
  t.key_space += p.key_space;
  t.accessible += p.accessible;
  t.coaccessible += p.coaccessible;
  t.generated = t.generated < 0 || p.generated < 0 ? -1 : t.generated + p.generated;
  t.generated_backward = t.generated_backward < 0 || p.generated_backward < 0
                             ? -1
                             : t.generated_backward + p.generated_backward;
  t.fwd_levels = t.fwd_levels > p.fwd_levels ? t.fwd_levels : p.fwd_levels;
  t.bwd_levels = t.bwd_levels > p.bwd_levels ? t.bwd_levels : p.bwd_levels;
  t.heavy_states += p.heavy_states;
  t.num_states += p.num_states;
  t.num_arcs += p.num_arcs;
}

int batch_impl(fst_ctx *c, const fst_graph *A, int32_t n, const fst_graph *B, hipStream_t s,
               int64_t *V_C, int64_t *E_C, int64_t *item_states, int64_t *item_arcs) {
  c->parts.clear();
  c->batch_A.clear();
  c->cur_part = -1;
  long long VA = 0, EA = 0;
  for (int32_t i = 0; i < n; ++i) {
    FST_TRY(check_graph_args(&A[i]));
    VA += A[i].num_states;
    EA += A[i].num_arcs;
  }
  FST_TRY(check_graph_args(B));
  if (EA > INT32_MAX) return FST_ERR_TOO_LARGE;
  // each item on its own first: an arc of one item must not name a state
  // of another once the union shifts its ids
  FST_TRY(ensure(c, c->scal, sizeof(Scalars)));
  Scalars *d_sc = as<Scalars>(c->scal);
  HIP_TRY(hipMemsetAsync(d_sc, 0, sizeof(Scalars), s));
  for (int32_t i = 0; i < n; ++i)
    if (A[i].num_states > 0)
      HIP_TRY(launch_validate(dev_graph(&A[i]), 0, &d_sc->errA, &d_sc->maxLabA, s, nullptr,
                              c->validate));
  FST_TRY(readback(c, s));
  if (c->h_sc->errA & ~(1u << 16)) return FST_ERR_INVALID_GRAPH;

  // Parts: consecutive items whose union has a key space below 2^32 (with
  // its A states rounded up to 64 for the search layout, as the run checks)
  unsigned long long max_rows = ~0ull;
  if (B->num_states > 0) {
    const int bitsB = bitlen((unsigned long long)(B->num_states - 1));
    const uint32_t shiftB = (uint32_t)(bitsB > 4 ? bitsB : 4);
    max_rows = (((1ull << 32) - 1) >> (shiftB + 1)) / 64 * 64;
    if (max_rows > NBR_MASK) max_rows = NBR_MASK;
  }
  std::vector<std::pair<int32_t, int32_t>> ranges;
  {
    int32_t i0 = 0;
    unsigned long long rows = 0;
    for (int32_t i = 0; i < n; ++i) {
      const unsigned long long v = (unsigned long long)A[i].num_states;
      if (v > max_rows) return FST_ERR_TOO_LARGE;  // one item alone is too large
      if (rows + v > max_rows && i > i0) {
        ranges.emplace_back(i0, i);
        i0 = i;
        rows = 0;
      }
      rows += v;
    }
    ranges.emplace_back(i0, n);
  }

  std::vector<long long> st((size_t)n + 1), ar((size_t)n + 1);
  if (ranges.size() == 1) {
    if (VA > NBR_MASK) return FST_ERR_TOO_LARGE;
    FST_TRY(run_items(c, A, 0, n, B, s, V_C, E_C, st.data(), ar.data()));
    for (int32_t i = 0; i <= n; ++i) {
      item_states[i] = st[i];
      item_arcs[i] = ar[i];
    }
    return FST_OK;
  }

  // several parts: each run in turn; C is the parts' results one after the
  // other (item order), ids shifted by the parts before
  fst_stats total = {};
  total.generated = total.generated_backward = 0;
  long long vbase = 0, ebase = 0, abase = 0, aebase = 0;
  for (size_t p = 0; p < ranges.size(); ++p) {
    const int32_t i0 = ranges[p].first, i1 = ranges[p].second;
    int64_t Vp = 0, Ep = 0;
    FST_TRY(run_items(c, A, i0, i1, B, s, &Vp, &Ep, st.data(), ar.data()));
    for (int32_t i = i0; i < i1; ++i) {
      item_states[i] = vbase + st[i - i0];
      item_arcs[i] = ebase + ar[i - i0];
    }
    long long va = 0, ea = 0;
    for (int32_t i = i0; i < i1; ++i) {
      va += A[i].num_states;
      ea += A[i].num_arcs;
    }
    c->parts.push_back(fst_ctx::BatchPart{i0, i1, vbase, ebase, abase, aebase, Vp, Ep});
    add_stats(total, c->stats);
    vbase += Vp;
    ebase += Ep;
    abase += va;
    aebase += ea;
    if (vbase > INT32_MAX || ebase > INT32_MAX) {
      c->parts.clear();
      return FST_ERR_TOO_LARGE;
    }
  }
  item_states[n] = vbase;
  item_arcs[n] = ebase;
  *V_C = vbase;
  *E_C = ebase;
  c->batch_A.assign(A, A + n);
  c->batch_B = *B;
  c->cur_part = (int)ranges.size() - 1;
  c->batch_stats = total;
  c->stats = total;
  c->timed_run = false;
  return FST_OK;
}

// The fill of a batch in parts: the part whose search state the context
// holds first, then every other part searched again (same sizes, or the
// inputs changed: FST_ERR_STATE), each written at its place in C.
int fill_parts(fst_ctx *c, const fst_graph_out *C, hipStream_t s) {
  std::vector<int> order;
  order.push_back(c->cur_part);
  for (int p = 0; p < (int)c->parts.size(); ++p)
    if (p != c->cur_part) order.push_back(p);
  for (int p : order) {
    const fst_ctx::BatchPart &part = c->parts[(size_t)p];
    if (p != c->cur_part) {
      int64_t Vp = 0, Ep = 0;
      std::vector<long long> st((size_t)(part.i1 - part.i0) + 1), ar(st.size());
      c->cur_part = -1;
      FST_TRY(run_items(c, c->batch_A.data(), part.i0, part.i1, &c->batch_B, s, &Vp, &Ep,
                        st.data(), ar.data()));
      c->cur_part = p;
      if (Vp != part.V || Ep != part.E) return FST_ERR_STATE;
    }
    const long long vb = part.vbase, eb = part.ebase;
    OutGraph O = {};
    O.arc_offset = C->arc_offset + vb;
    O.src = C->src ? C->src + eb : nullptr;
    O.dst = C->dst ? C->dst + eb : nullptr;
    O.il = C->ilabel ? C->ilabel + eb : nullptr;
    O.ol = C->olabel ? C->olabel + eb : nullptr;
    O.w = C->weight ? C->weight + eb : nullptr;
    O.start = C->start ? C->start + vb : nullptr;
    O.accept = C->accept ? C->accept + vb : nullptr;
    O.key_a = C->key_a ? C->key_a + vb : nullptr;
    O.key_b = C->key_b ? C->key_b + vb : nullptr;
    O.key_f = C->key_f ? C->key_f + vb : nullptr;
    O.arc_a = C->arc_a ? C->arc_a + eb : nullptr;
    O.arc_b = C->arc_b ? C->arc_b + eb : nullptr;
    O.vbase = (int32_t)vb;
    O.ebase = (int32_t)eb;
    O.abase = (int32_t)part.abase;
    O.aebase = (int32_t)part.aebase;
    HIP_TRY(launch_fill(c->P, c->nstates ? c->out_words : 0, as<uint8_t>(c->cnt),
                        as<uint32_t>(c->fq), as<uint32_t>(c->btot), as<uint2>(c->bq), c->nheavy,
                        c->nstates, c->narcs, O, s));
  }
  c->stats = c->batch_stats;
  c->timed_run = false;
  return FST_OK;
}

}  // namespace

extern "C" {

int fst_ctx_create(int device, fst_ctx **ctx) {
  if (!ctx) return FST_ERR_INVALID_ARG;
  *ctx = nullptr;
  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || device < 0 || device >= ndev) {
    (void)hipGetLastError();
    return FST_ERR_INVALID_ARG;
  }
  fst_ctx *c = new (std::nothrow) fst_ctx();
  if (!c) return FST_ERR_NOMEM;
  c->device = device;
  DeviceGuard g(device);
  if (!g.ok) {
    delete c;
    return FST_ERR_HIP;
  }
  if (hipHostMalloc(reinterpret_cast<void **>(&c->h_sc), sizeof(Scalars), 0) != hipSuccess) {
    delete c;
    return FST_ERR_NOMEM;
  }
  memset(c->h_sc, 0, sizeof(Scalars));
  if (hipHostMalloc(reinterpret_cast<void **>(&c->h_ssc), sizeof(ScoreScalars), 0) !=
      hipSuccess) {
    fst_ctx_destroy(c);
    return FST_ERR_NOMEM;
  }
  memset(c->h_ssc, 0, sizeof(ScoreScalars));
  if (hipHostMalloc(reinterpret_cast<void **>(&c->h_s3), sizeof(Scal3), 0) != hipSuccess) {
    fst_ctx_destroy(c);
    return FST_ERR_NOMEM;
  }
  memset(c->h_s3, 0, sizeof(Scal3));
  for (ScoreBufs *b : {&c->score_f, &c->score_b}) {
    if (hipHostMalloc(reinterpret_cast<void **>(&b->host), sizeof(ScoreScalars), 0) !=
        hipSuccess) {
      fst_ctx_destroy(c);
      return FST_ERR_NOMEM;
    }
    memset(b->host, 0, sizeof(ScoreScalars));
  }
  // the device array of fst_grad_scatter_noalloc: its address on this device
  void *scr = nullptr;
  if (scatter_scratch(device, &scr) != hipSuccess) {
    (void)hipGetLastError();
    fst_ctx_destroy(c);
    return FST_ERR_HIP;
  }
  for (int i = 0; i < NEV; ++i) {
    if (hipEventCreate(&c->ev[i]) != hipSuccess) {
      fst_ctx_destroy(c);
      return FST_ERR_HIP;
    }
  }
  for (int i = 0; i < 2 * NKERNELS; ++i) {
    if (hipEventCreate(&c->kev[i]) != hipSuccess) {
      fst_ctx_destroy(c);
      return FST_ERR_HIP;
    }
  }
  *ctx = c;
  return FST_OK;
}

void fst_ctx_destroy(fst_ctx *c) {
  if (!c) return;
  DeviceGuard g(c->device);
  (void)hipDeviceSynchronize();
  DevBuf *bufs[] = {&c->scal,     &c->lists,    &c->k0,      &c->k1,      &c->v0,
                    &c->v1,       &c->sort_tmp, &c->scan_tmp, &c->aOutPerm, &c->aOutArc,
                    &c->aOutRec,  &c->aOutLut,  &c->bOutPerm, &c->bOutArc, &c->bOutRec,
                    &c->bOutLut,  &c->aInOff,   &c->aInPerm, &c->aInArc,  &c->aInRec,
                    &c->aInLut,   &c->bInOff,   &c->bInPerm, &c->bInArc,  &c->bInRec,
                    &c->bInLut,   &c->vis,      &c->coacc,   &c->trim,    &c->wbase,   &c->heavy2,
                    &c->hoff2,    &c->fq,
                    &c->bq,       &c->heavy,    &c->hoff,    &c->cnt,     &c->aOutLab,
                    &c->aOutW,    &c->bOutLab,  &c->bOutW,   &c->btot,    &c->bOutChain,
                    &c->bInChain, &c->s_sc,     &c->s_owner, &c->s_extra, &c->s_inref,
                    &c->s_mbeg,   &c->s_mlen,   &c->s_mcur,  &c->s_marc,  &c->s_val,
                    &c->s_acc,    &c->s_pg,     &c->s_pidx,  &c->s_bcnt,  &c->s_bscan,
                    &c->s_btotal, &c->s_mpos,   &c->s_sweep, &c->s_ioff, &c->s_isrc, &c->s_iw, &c->u_off,   &c->u_src,   &c->u_dst,
                    &c->u_il,     &c->u_ol,     &c->u_w,     &c->u_start, &c->u_accept,
                    &c->u_items,  &c->seg,    &c->t_scal,  &c->t_aPerm, &c->t_aArc,
                    &c->t_aRec,   &c->t_bPerm,  &c->t_bArc,  &c->t_bRec,  &c->t_bLab,
                    &c->t_bW,     &c->t_dPerm,  &c->t_dArc,  &c->t_dRec,  &c->t_dLab,
                    &c->t_dW,     &c->t_bflags, &c->t_lists, &c->t_tab,   &c->t_F,
                    &c->t_chunks, &c->t_arcs,   &c->t_inoff, &c->t_first,
                    &c->t_coacc,  &c->t_keys0,  &c->t_keys1, &c->t_slots0, &c->t_slots1,
                    &c->t_idof,   &c->t_units,  &c->t_ucnt,  &c->t_aLab,  &c->t_aW,
                    &c->t_heavy,  &c->t_aLut,   &c->t_bLut,  &c->t_dLut, &c->t_bChain,
                    &c->t_segs,   &c->t_segof};
  for (DevBuf *b : bufs) release(*b);
  for (ScoreBufs *sb : {&c->score_f, &c->score_b}) {
    for (DevBuf *b : {&sb->sc, &sb->rec, &sb->term, &sb->mkey, &sb->pend, &sb->q, &sb->h,
                      &sb->hoff})
      release(*b);
    if (sb->host) (void)hipHostFree(sb->host);
  }
  for (int i = 0; i < NEV; ++i)
    if (c->ev[i]) (void)hipEventDestroy(c->ev[i]);
  for (int i = 0; i < 2 * NKERNELS; ++i)
    if (c->kev[i]) (void)hipEventDestroy(c->kev[i]);
  if (c->h_sc) (void)hipHostFree(c->h_sc);
  if (c->h_ssc) (void)hipHostFree(c->h_ssc);
  if (c->h_s3) (void)hipHostFree(c->h_s3);
  delete c;
}

int fst_ctx_set_option(fst_ctx *c, int option, int64_t value) {
  if (!c) return FST_ERR_INVALID_ARG;
  switch (option) {
    case FST_OPT_MAX_WORKSPACE:
      if (value < 0) return FST_ERR_INVALID_ARG;
      c->max_ws = value;
      return FST_OK;
    case FST_OPT_TIMING:
      c->timing = value != 0;
      c->have_times = false;
      return FST_OK;
    case FST_OPT_LABEL_BUCKETS:
      c->buckets = value != 0;
      return FST_OK;
    case FST_OPT_COUNT_MOVES:
      c->count_moves = value != 0;
      return FST_OK;
    case FST_OPT_ORDER:
      if (value != FST_ORDER_FORWARD_FIRST && value != FST_ORDER_COACCESSIBLE_FIRST &&
          value != FST_ORDER_CONCURRENT)
        return FST_ERR_INVALID_ARG;
      c->order = (int)value;
      return FST_OK;
    case FST_OPT_LIST_CAPACITY:
      if (value < 0 || value > (1ll << 32)) return FST_ERR_INVALID_ARG;
      c->list_start = value ? (unsigned long long)value : (1ull << 22);
      c->list_hint = 0;
      return FST_OK;
    case FST_OPT_VALIDATE:
      c->validate = value != 0;
      return FST_OK;
    case FST_OPT_CHAIN_DEPTH:
      if (value < 0 || value > (1 << 20)) return FST_ERR_INVALID_ARG;
      c->chain_depth = (int)value;
      return FST_OK;
    default:
      return FST_ERR_INVALID_ARG;
  }
}

int fst_compose_run(fst_ctx *c, const fst_graph *A, const fst_graph *B, void *stream,
                    int64_t *num_states, int64_t *num_arcs) {
  if (!c || !A || !B || !num_states || !num_arcs) return FST_ERR_INVALID_ARG;
  DeviceGuard g(c->device);
  if (!g.ok) return FST_ERR_HIP;
  c->ready = false;
  c->have_times = false;
  c->timed_run = false;
  c->parts.clear();
  *num_states = 0;
  *num_arcs = 0;
  int rc = run_impl(c, A, B, reinterpret_cast<hipStream_t>(stream), num_states, num_arcs);
  if (rc != FST_OK) {
    c->ready = false;
    *num_states = 0;
    *num_arcs = 0;
    (void)hipGetLastError();
  }
  return rc;
}

int fst_compose_batch_run(fst_ctx *c, const fst_graph *A, int32_t n, const fst_graph *B,
                          void *stream, int64_t *num_states, int64_t *num_arcs,
                          int64_t *item_states, int64_t *item_arcs) {
  if (!c || n < 0 || (n > 0 && !A) || !B || !num_states || !num_arcs || !item_states ||
      !item_arcs)
    return FST_ERR_INVALID_ARG;
  DeviceGuard g(c->device);
  if (!g.ok) return FST_ERR_HIP;
  c->ready = false;
  c->have_times = false;
  c->timed_run = false;
  *num_states = 0;
  *num_arcs = 0;
  int rc = FST_OK;
  try {
    rc = batch_impl(c, A, n, B, reinterpret_cast<hipStream_t>(stream), num_states, num_arcs,
                    item_states, item_arcs);
  } catch (const std::bad_alloc &) {
    rc = FST_ERR_NOMEM;
  }
  if (rc != FST_OK) {
    c->ready = false;
    c->parts.clear();
    *num_states = 0;
    *num_arcs = 0;
    for (int32_t i = 0; i <= n; ++i) item_states[i] = item_arcs[i] = 0;
    (void)hipGetLastError();
  }
  return rc;
}

int fst_compose_fill(fst_ctx *c, const fst_graph_out *C, void *stream) {
  if (!c || !C) return FST_ERR_INVALID_ARG;
  if (!c->ready) return FST_ERR_STATE;
  const bool parts = !c->parts.empty();
  const long long nst = parts ? c->batch_stats.num_states : c->nstates;
  const long long nar = parts ? c->batch_stats.num_arcs : c->narcs;
  if (!C->arc_offset) return FST_ERR_INVALID_ARG;
  if (nst && (!C->start || !C->accept)) return FST_ERR_INVALID_ARG;
  if (nar && (!C->src || !C->dst || !C->ilabel || !C->olabel || !C->weight))
    return FST_ERR_INVALID_ARG;
  DeviceGuard g(c->device);
  if (!g.ok) return FST_ERR_HIP;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (parts) {
    int rc = FST_OK;
    try {
      rc = fill_parts(c, C, s);
    } catch (const std::bad_alloc &) {
      rc = FST_ERR_NOMEM;
    }
    if (rc != FST_OK) {
      c->ready = false;
      c->parts.clear();
      (void)hipGetLastError();
    }
    c->have_times = false;
    return rc;
  }
  OutGraph O = {};
  O.arc_offset = C->arc_offset;
  O.src = C->src;
  O.dst = C->dst;
  O.il = C->ilabel;
  O.ol = C->olabel;
  O.w = C->weight;
  O.start = C->start;
  O.accept = C->accept;
  O.key_a = C->key_a;
  O.key_b = C->key_b;
  O.key_f = C->key_f;
  O.arc_a = C->arc_a;
  O.arc_b = C->arc_b;
  phase_begin(c, PH_FILL, s);
  const KernelTimer tf = c->timed_run ? timer(c, FST_KERNEL_FILL) : KernelTimer{};
  tf.begin(s);
  // with no states the fill only writes arc_offset[0] (and reads no bitmap)
  hipError_t e = launch_fill(c->P, c->nstates ? c->out_words : 0, as<uint8_t>(c->cnt),
                             as<uint32_t>(c->fq),
                             as<uint32_t>(c->btot), as<uint2>(c->bq), c->nheavy, c->nstates,
                             c->narcs, O, s);
  tf.end(s);
  // one launch: offsets, flags and arcs of every state
  c->klaunches[FST_KERNEL_FILL] = c->timed_run ? 1 : 0;
  c->kms[FST_KERNEL_FILL] = 0.f;
  phase_end(c, PH_FILL, s);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return FST_ERR_HIP;
  }
  c->have_times = c->timed_run;
  return FST_OK;
}

int fst_compose3_run(fst_ctx *c, const fst_graph *A, const fst_graph *B, const fst_graph *D,
                     void *stream, int64_t *num_states, int64_t *num_arcs) {
  if (!c || !A || !B || !D || !num_states || !num_arcs) return FST_ERR_INVALID_ARG;
  DeviceGuard g(c->device);
  if (!g.ok) return FST_ERR_HIP;
  c->c3.ready = false;
  c->have_times3 = false;
  *num_states = 0;
  *num_arcs = 0;
  int rc = compose3_impl(c, A, B, D, reinterpret_cast<hipStream_t>(stream), num_states,
                         num_arcs);
  if (rc != FST_OK) {
    c->c3.ready = false;
    *num_states = 0;
    *num_arcs = 0;
    (void)hipGetLastError();
  }
  return rc;
}

int fst_compose3_fill(fst_ctx *c, const fst_graph3_out *C, void *stream) {
  if (!c || !C) return FST_ERR_INVALID_ARG;
  if (!c->c3.ready) return FST_ERR_STATE;
  if (!C->arc_offset) return FST_ERR_INVALID_ARG;
  if (c->c3.n && (!C->start || !C->accept)) return FST_ERR_INVALID_ARG;
  if (c->c3.narcs && (!C->src || !C->dst || !C->ilabel || !C->olabel || !C->weight))
    return FST_ERR_INVALID_ARG;
  DeviceGuard g(c->device);
  if (!g.ok) return FST_ERR_HIP;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (c->c3.n == 0) {
    HIP_TRY(hipMemsetAsync(C->arc_offset, 0, sizeof(int32_t), s));
    return FST_OK;
  }
  OutGraph3 O;
  O.arc_offset = C->arc_offset;
  O.src = C->src;
  O.dst = C->dst;
  O.il = C->ilabel;
  O.ol = C->olabel;
  O.w = C->weight;
  O.start = C->start;
  O.accept = C->accept;
  O.key_a = C->key_a;
  O.key_b = C->key_b;
  O.key_fab = C->key_fab;
  O.key_d = C->key_d;
  O.key_f = C->key_f;
  O.arc_a = C->arc_a;
  O.arc_b = C->arc_b;
  O.arc_d = C->arc_d;
  const KernelTimer t = c->c3.timed ? timer(c, FST_KERNEL_COMPACT3) : KernelTimer{};
  t.begin(s);
  hipError_t e = launch3_fill(c->c3.P, c->c3.keys, c->c3.ustart, c->c3.n, c->c3.heavy,
                              c->c3.nheavy, c->c3.uoff, c->c3.narcs, O, s);
  t.end(s);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return FST_ERR_HIP;
  }
  if (c->c3.timed) {
    // the fill's launches join the time of the compaction kernels
    HIP_TRY(hipEventSynchronize(c->kev[2 * FST_KERNEL_COMPACT3 + 1]));
    FST_TRY(add_time(c, FST_KERNEL_COMPACT3, 2));
  }
  return FST_OK;
}

int fst_compose3_stats(const fst_ctx *c, fst_stats *out) {
  if (!c || !out) return FST_ERR_INVALID_ARG;
  if (!c->c3.ready) return FST_ERR_STATE;
  *out = c->c3.stats;
  return FST_OK;
}

int fst_compose_stats(const fst_ctx *c, fst_stats *out) {
  if (!c || !out) return FST_ERR_INVALID_ARG;
  if (!c->ready) return FST_ERR_STATE;
  *out = c->stats;
  return FST_OK;
}

int fst_compose_phase_times(const fst_ctx *c, float *ms, int n) {
  if (!c || !ms || n < 0) return FST_ERR_INVALID_ARG;
  if (!c->have_times) return FST_ERR_STATE;
  DeviceGuard g(c->device);
  if (hipEventSynchronize(c->ev[2 * PH_FILL + 1]) != hipSuccess) return FST_ERR_HIP;
  for (int i = 0; i < n && i < 5; ++i) {
    float t = 0.f;
    if (hipEventElapsedTime(&t, c->ev[2 * i], c->ev[2 * i + 1]) != hipSuccess)
      return FST_ERR_HIP;
    ms[i] = t;
  }
  return FST_OK;
}

int fst_compose_kernel_time(const fst_ctx *c, int kernel, float *ms, int64_t *launches) {
  if (!c || !ms || !launches || kernel < 0 || kernel >= NKERNELS) return FST_ERR_INVALID_ARG;
  const bool have = kernel < NCOMPOSE_KERNELS ? c->have_times
                    : kernel < 6                ? c->have_score_times
                                                : c->have_times3;
  if (!have) return FST_ERR_STATE;
  float t = c->kms[kernel];
  if (kernel == FST_KERNEL_FILL) {
    // the fill is asynchronous: its events are read here
    DeviceGuard g(c->device);
    if (hipEventSynchronize(c->kev[2 * kernel + 1]) != hipSuccess) return FST_ERR_HIP;
    if (hipEventElapsedTime(&t, c->kev[2 * kernel], c->kev[2 * kernel + 1]) != hipSuccess)
      return FST_ERR_HIP;
  }
  *ms = t;
  *launches = c->klaunches[kernel];
  return FST_OK;
}

int fst_score(fst_ctx *c, const fst_graph *G, double *alpha, double *beta, double *total,
              void *stream) {
  if (!c || !G || !total) return FST_ERR_INVALID_ARG;
  DeviceGuard g(c->device);
  if (!g.ok) return FST_ERR_HIP;
  c->have_score_times = false;
  int rc = score_impl(c, G, alpha, beta, total, reinterpret_cast<hipStream_t>(stream));
  if (rc != FST_OK) (void)hipGetLastError();
  return rc;
}

int fst_score_cyclic(fst_ctx *c, const fst_graph *G, double *alpha, double *beta,
                     double *total, int32_t max_sweeps, double tol, int32_t *sweeps,
                     void *stream) {
  if (!c || !G || !total) return FST_ERR_INVALID_ARG;
  DeviceGuard g(c->device);
  if (!g.ok) return FST_ERR_HIP;
  c->have_score_times = false;
  int rc = score_cyclic_impl(c, G, alpha, beta, total, max_sweeps, tol, sweeps,
                             reinterpret_cast<hipStream_t>(stream));
  if (rc != FST_OK && rc != FST_ERR_NOT_CONVERGED) (void)hipGetLastError();
  return rc;
}

int fst_score_posterior(fst_ctx *c, const fst_graph *G, const double *alpha, const double *beta,
                        const double *total, float scale, float *grad, void *stream) {
  if (!c || !G || !total) return FST_ERR_INVALID_ARG;
  FST_TRY(check_graph_args(G));
  if (G->num_arcs > 0 && (!alpha || !beta || !grad)) return FST_ERR_INVALID_ARG;
  DeviceGuard g(c->device);
  if (!g.ok) return FST_ERR_HIP;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const DevGraph d = dev_graph(G);
  FST_TRY(ensure(c, c->s_sc, sizeof(ScoreScalars)));
  FST_TRY(score_validate(c, d, s));
  if (launch_posterior(plain_score_graph(d), alpha, beta, total, scale, grad, s) != hipSuccess) {
    (void)hipGetLastError();
    return FST_ERR_HIP;
  }
  return FST_OK;
}

int fst_grad_scatter(fst_ctx *c, int64_t n, const float *grad, const int32_t *idx, int32_t m,
                     float *out, void *stream) {
  if (!c || n < 0 || m < 0) return FST_ERR_INVALID_ARG;
  if ((n > 0 && (!grad || !idx)) || (m > 0 && !out)) return FST_ERR_INVALID_ARG;
  DeviceGuard g(c->device);
  if (!g.ok) return FST_ERR_HIP;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  FST_TRY(ensure(c, c->s_sc, sizeof(ScoreScalars)));
  FST_TRY(ensure(c, c->s_acc, (size_t)m * 4 * sizeof(unsigned long long)));
  ScoreScalars *dsc = as<ScoreScalars>(c->s_sc);
  HIP_TRY(hipMemsetAsync(dsc, 0, sizeof(ScoreScalars), s));
  if (m > 0) HIP_TRY(hipMemsetAsync(c->s_acc.p, 0, (size_t)m * 4 * sizeof(unsigned long long), s));
  // grouping the terms by target range needs 8 bytes per term of workspace;
  // without it (workspace cap) every term goes to the plain scatter
  ScatterTemp tmp{}, *tp = nullptr;
  if (scatter_grouped((long long)n, m)) {
    const size_t words = scatter_count_words((long long)n, m);
    if (ensure(c, c->s_pg, (size_t)n * sizeof(float)) == FST_OK &&
        ensure(c, c->s_pidx, (size_t)n * sizeof(int32_t)) == FST_OK &&
        ensure(c, c->s_bcnt, words * sizeof(uint32_t)) == FST_OK &&
        ensure(c, c->s_bscan, scan_temp_bytes(words)) == FST_OK &&
        ensure(c, c->s_btotal, sizeof(unsigned long long)) == FST_OK) {
      tmp = ScatterTemp{as<float>(c->s_pg), as<int32_t>(c->s_pidx), as<uint32_t>(c->s_bcnt),
                        c->s_bscan.p, as<unsigned long long>(c->s_btotal)};
      tp = &tmp;
    }
  }
  if (launch_scatter(grad, idx, (long long)n, m, as<unsigned long long>(c->s_acc), &dsc->absmax,
                     &dsc->bad, out, tp, s) != hipSuccess) {
    (void)hipGetLastError();
    return FST_ERR_HIP;
  }
  FST_TRY(score_readback(c, s));
  return c->h_ssc->bad ? FST_ERR_INVALID_ARG : FST_OK;
}

int fst_grad_scatter_noalloc(fst_ctx *c, int64_t n, const float *grad, const int32_t *idx,
                             int32_t m, float *out, void *stream) {
  if (!c || n < 0 || m < 0) return FST_ERR_INVALID_ARG;
  if ((n > 0 && (!grad || !idx)) || (m > 0 && !out)) return FST_ERR_INVALID_ARG;
  if (m > FST_SCATTER_NOALLOC_MAX_TARGETS) return FST_ERR_TOO_LARGE;
  DeviceGuard g(c->device);
  if (!g.ok) return FST_ERR_HIP;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  void *scr = nullptr;
  if (scatter_scratch(c->device, &scr) != hipSuccess ||
      launch_scatter_noalloc(grad, idx, (long long)n, m, scr, out, s) != hipSuccess) {
    (void)hipGetLastError();
    return FST_ERR_HIP;
  }
  // the bad-index flag (32-bit word 1 of the array) into pinned host memory
  // the context allocated at creation
  HIP_TRY(hipMemcpyAsync(&c->h_ssc->bad, static_cast<uint32_t *>(scr) + 1, sizeof(uint32_t),
                         hipMemcpyDeviceToHost, s));
  HIP_TRY(hipStreamSynchronize(s));
  return c->h_ssc->bad ? FST_ERR_INVALID_ARG : FST_OK;
}

int fst_segment_logsum(fst_ctx *c, const double *val, const uint8_t *flag, int32_t n,
                       const int64_t *bounds, double *totals, void *stream) {
  if (!c || n < 0 || !bounds) return FST_ERR_INVALID_ARG;
  if (n > 0 && !totals) return FST_ERR_INVALID_ARG;
  long long max_len = 0;
  for (int32_t i = 0; i < n; ++i) {
    if (bounds[i] < 0 || bounds[i + 1] < bounds[i]) return FST_ERR_INVALID_ARG;
    if (bounds[i + 1] - bounds[i] > max_len) max_len = bounds[i + 1] - bounds[i];
  }
  if (max_len > 0 && (!val || !flag)) return FST_ERR_INVALID_ARG;
  if (n == 0) return FST_OK;
  DeviceGuard g(c->device);
  if (!g.ok) return FST_ERR_HIP;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  FST_TRY(ensure(c, c->seg, ((size_t)n + 1) * sizeof(long long) +
                                3 * (size_t)n * sizeof(unsigned long long)));
  long long *db = as<long long>(c->seg);
  unsigned long long *z = reinterpret_cast<unsigned long long *>(db + n + 1);
  HIP_TRY(hipMemcpyAsync(db, bounds, ((size_t)n + 1) * sizeof(long long), hipMemcpyHostToDevice,
                         s));
  HIP_TRY(hipMemsetAsync(z, 0, 3 * (size_t)n * sizeof(unsigned long long), s));
  if (launch_segment_logsum(val, flag, n, db, max_len, z, totals, s) != hipSuccess) {
    (void)hipGetLastError();
    return FST_ERR_HIP;
  }
  // the host bounds were read by the copy above; nothing else is pending on
  // host memory
  HIP_TRY(hipStreamSynchronize(s));
  return FST_OK;
}

const char *fst_strerror(int code) {
  switch (code) {
    case FST_OK: return "ok";
    case FST_ERR_INVALID_ARG: return "invalid argument";
    case FST_ERR_INVALID_GRAPH: return "invalid graph";
    case FST_ERR_TOO_LARGE: return "problem too large (key space or output size)";
    case FST_ERR_NOMEM: return "out of device memory or over the workspace cap";
    case FST_ERR_HIP: return "HIP runtime error";
    case FST_ERR_STATE: return "no successful fst_compose_run to fill from";
    case FST_ERR_CYCLIC: return "graph has a cycle (scores need an acyclic graph)";
    case FST_ERR_NOT_CONVERGED: return "relaxation sweeps did not converge (path sums may diverge)";
    default: return "unknown error";
  }
}

}  // extern "C"
