// Log-semiring scores of an acyclic graph, their gradient (the arc
// posteriors), and the scatter of per-arc gradients of a composed graph back
// to the arcs of its operands through provenance, for gfx950.
//
// Scores.  alpha[v] is the log-sum over the paths from a start state to v of
// exp(path weight), beta[v] the log-sum over the paths from v to an accepting
// state, and the total the log-sum over accepting paths: the forward and
// backward shortest distances of the log semiring in which Eq. (1) reads the
// composed weight.  A state's value is final once the values it pulls from
// are (its in-arcs' sources for alpha, its out-arcs' targets for beta), so
// states are finished in topological generations, one kernel each, and a
// kernel boundary separates every value from its reads by other threads:
//   * In-degrees are classified without atomics: every arc stores its id in
//     owner[dst] (one store wins), then every arc that does not find its own
//     id there counts itself as an extra in-arc of dst.  A state with no extra
//     in-arc has at most one in-arc (owner, or none).  Only the states with
//     several in-arcs ("merges") get an in-arc list, built with atomics; in a
//     composed speech graph almost every state has exactly one in-arc.
//   * A thread that finishes a state walks on, in the same kernel, to a
//     successor whose only dependency that state was: the successor's value
//     follows from the thread's registers.  Other ready successors go to the
//     next generation's lists; a successor with several dependencies counts
//     an atomic pending counter down, and the thread that takes it to zero
//     lists it.  Every dependency a listed state still has to pull is left
//     as a term (value + arc weight) in a slot indexed by the arc, so a pull
//     reads slots (contiguous ones backward) instead of chasing sources.
//   * A 16-byte record per state packs what a walk needs: its flags and, for
//     a state with one arc to notify, that arc's other end, weight and id; a
//     walk along a chain takes one dependent load per state.
//   * A state with more than SCORE_LIGHT arcs to pull from or to notify is
//     heavy: the next generation gives every NT of its notified arcs a
//     workgroup, which pulls the value cooperatively; then each thread walks
//     on from one successor.
//   * A walk settles the state it stops at only once every lane of its
//     wavefront has stopped (walks differ in length), and in the workgroups
//     of heavy states the arrivals at each merge are first gathered in LDS,
//     so a merge is counted down once per workgroup.
// Log-add is exact up to its final rounding and does not depend on the order
// of its terms: the maximum m first, then every exp(x - m), which lies in
// (0, 1], truncated to a multiple of 2^-64 and added as a 128-bit integer.
// In-arc lists may therefore be in any order, and every thread, workgroup
// and run returns the same bits.
//
// Provenance scatter.  out[i] = sum of g[e] over the arcs e with idx[e] = i.
// Each g[e] is turned into a 64-bit fixed-point magnitude relative to the
// largest |g| and added into a positive or negative pair of 64-bit words as
// two 32-bit digits (lazy carries), so the sums are exact integers and the
// result does not depend on the order of the atomics.
#include <math.h>

#include <mutex>

#include "internal.h"

namespace fstc {
namespace {

typedef unsigned long long ull;

constexpr int32_t SCORE_LIGHT = 64;  // arcs a single thread pulls or notifies
constexpr unsigned SCORE_GRID = 1024;
// Workgroups of a relaxation sweep at most (each ends with one atomic on the
// sweep's rise word).
constexpr long long SWEEP_GRID = 512;
// Pull lists of at most this many terms are loaded once into registers.
constexpr int SWEEP_REGS = 8;
// Structure passes take ST_ITEMS items per thread and round, their loads
// issued before any store or atomic (which would otherwise make every load
// wait for the previous item's store).
constexpr int ST_ITEMS = 8;

// ---------------------------------------------------------------------------
// exact log-add
// ---------------------------------------------------------------------------

// Adds exp-term y in [0, 1] as y * 2^64 truncated: (hi, lo) is a 128-bit sum.
__device__ __forceinline__ void acc_add(ull &lo, ull &hi, double y) {
  if (!(y > 0.0)) return;  // zero (or a term made of non-finite weights)
  if (y >= 1.0) {
    hi += 1ull;
    return;
  }
  const ull t = (ull)(y * 18446744073709551616.0);  // < 2^64
  lo += t;
  hi += lo < t ? 1ull : 0ull;
}

__device__ __forceinline__ double acc_finish(double m, ull lo, ull hi) {
  if (m == -INFINITY || m == INFINITY) return m;
  const double s = (double)hi + (double)lo * 0x1p-64;  // >= 1: the maximum adds 1
  return m + log(s);
}

__device__ __forceinline__ void add128(ull &lo, ull &hi, ull olo, ull ohi) {
  const ull n = lo + olo;
  hi += ohi + (n < lo ? 1ull : 0ull);
  lo = n;
}

__device__ __forceinline__ double wave_fmax(double x) {
#pragma unroll
  for (int o = WAVE / 2; o > 0; o >>= 1) x = fmax(x, __shfl_xor(x, o));
  return x;
}

__device__ __forceinline__ void wave_sum128(ull &lo, ull &hi) {
#pragma unroll
  for (int o = WAVE / 2; o > 0; o >>= 1) {
    const ull olo = __shfl_xor(lo, o), ohi = __shfl_xor(hi, o);
    add128(lo, hi, olo, ohi);
  }
}

// Workgroup reductions (every thread gets the result; all must call).
__device__ __forceinline__ double block_fmax(double x) {
  __shared__ double s_m[NWAVES];
  x = wave_fmax(x);
  __syncthreads();
  if (__lane_id() == 0) s_m[threadIdx.x / WAVE] = x;
  __syncthreads();
  double r = s_m[0];
#pragma unroll
  for (int w = 1; w < NWAVES; ++w) r = fmax(r, s_m[w]);
  return r;
}

__device__ __forceinline__ void block_sum128(ull &lo, ull &hi) {
  __shared__ ull s_lo[NWAVES], s_hi[NWAVES];
  wave_sum128(lo, hi);
  __syncthreads();
  if (__lane_id() == 0) {
    s_lo[threadIdx.x / WAVE] = lo;
    s_hi[threadIdx.x / WAVE] = hi;
  }
  __syncthreads();
  lo = s_lo[0];
  hi = s_hi[0];
#pragma unroll
  for (int w = 1; w < NWAVES; ++w) add128(lo, hi, s_lo[w], s_hi[w]);
}

// Order-preserving integer key of a double (a larger double has a larger key;
// key 0 is below every double).
__device__ __forceinline__ ull order_key(double d) {
  const ull b = (ull)__double_as_longlong(d);
  return (b >> 63) ? ~b : (b | (1ull << 63));
}
__device__ __forceinline__ double from_order_key(ull k) {
  const ull b = (k >> 63) ? (k & ~(1ull << 63)) : ~k;
  return __longlong_as_double((long long)b);
}

// ---------------------------------------------------------------------------
// arc lists of a state
// ---------------------------------------------------------------------------

// Arcs beg .. beg + n - 1, or (ind) marc[beg .. beg + n - 1].
struct AList {
  int32_t beg, n;
  bool ind;
};

__device__ __forceinline__ AList in_list(const ScoreGraph &G, int32_t v) {
  const int32_t r = G.inref[v];
  if (r >= 0) return AList{r, 1, false};
  if (r == -1) return AList{0, 0, false};
  const int32_t m = -2 - r;
  return AList{G.mbeg[m], G.mlen[m], true};
}

__device__ __forceinline__ AList out_list(const ScoreGraph &G, int32_t v) {
  const int32_t b = G.off[v];
  return AList{b, G.off[v + 1] - b, false};
}

__device__ __forceinline__ int32_t arc_at(const ScoreGraph &G, const AList &l, int32_t j) {
  return l.ind ? G.marc[l.beg + j] : l.beg + j;
}

// Forward: pull over in-arcs (value at the source), notify over out-arcs.
// Backward: pull over out-arcs (value at the target), notify over in-arcs.
template <bool FWD>
__device__ __forceinline__ AList pull_list(const ScoreGraph &G, int32_t v) {
  return FWD ? in_list(G, v) : out_list(G, v);
}
template <bool FWD>
__device__ __forceinline__ AList notify_list(const ScoreGraph &G, int32_t v) {
  return FWD ? out_list(G, v) : in_list(G, v);
}
// Per-state record of one direction (built by k_score_init):
//   x: with one notified arc, the state it reaches; else the first entry of
//      the notify list (an arc id, or a marc position when REC_IND)
//   y: flags << 28 | number of notified arcs (saturated at 2^28 - 1)
//   z: with one notified arc, its weight (binary32 bits)
//   w: with one notified arc, the slot its term goes to when the state it
//      reaches is not walked to (see pull_slots); else -1
// so a walk takes one dependent load per state.
constexpr uint32_t REC_INIT = 1u << 28;    // start (forward) / accepting (backward)
constexpr uint32_t REC_SINGLE = 1u << 29;  // exactly one arc to pull from
constexpr uint32_t REC_HEAVY = 1u << 30;   // more than SCORE_LIGHT arcs to pull or notify
constexpr uint32_t REC_IND = 1u << 31;     // notify list is marc[x ...]
constexpr uint32_t REC_COUNT = (1u << 28) - 1u;

__device__ __forceinline__ uint32_t rec_flags(const int4 &r) { return (uint32_t)r.y; }
__device__ __forceinline__ int32_t rec_count(const int4 &r) {
  return (int32_t)((uint32_t)r.y & REC_COUNT);
}

// Value of a state from the term slots of its pull list, by one thread.
// Terms were stored by the states it depends on: term[e] = value + w(e).
// Slots of a pull list: the terms of a merge's in-arcs (forward) sit at
// E + their position in marc, every other term at its arc id, so the slots
// of a pull list are contiguous except for one forward in-arc.
__device__ __forceinline__ const double *pull_slots(const ScoreArgs &S, const AList &l) {
  return S.term + (l.ind ? S.G.E : 0) + l.beg;
}

// The largest term of a state with two or more, kept by its notifiers.
__device__ __forceinline__ double pull_max(const ScoreArgs &S, int32_t v, bool init) {
  const ull k = S.mkey[v];
  const double m = k ? from_order_key(k) : -INFINITY;
  return init ? fmax(m, 0.0) : m;
}

template <bool FWD>
__device__ double thread_pull(const ScoreArgs &S, int32_t v, const AList &l, bool init) {
  const double *t = pull_slots(S, l);
  if (l.n == 1 && !init) return t[0];
  double m;
  if (l.n >= 2) {
    m = pull_max(S, v, init);
  } else {
    m = init ? 0.0 : -INFINITY;
    if (l.n == 1) m = fmax(m, t[0]);
  }
  if (m == -INFINITY || m == INFINITY) return m;
  ull lo = 0, hi = 0;
  if (init) acc_add(lo, hi, exp(0.0 - m));
#pragma unroll 4
  for (int32_t j = 0; j < l.n; ++j) acc_add(lo, hi, exp(t[j] - m));
  return acc_finish(m, lo, hi);
}

// The same value, formed by a whole workgroup (identical bits), from the n
// term slots at t whose largest term (with the empty path's 0 when init) is
// m.
constexpr int PULL_BATCH = 20;
__device__ __forceinline__ double block_logsum(const double *t, int32_t n, double m, bool init) {
  if (m == -INFINITY || m == INFINITY) return m;
  ull lo = 0, hi = 0;
  if (threadIdx.x == 0 && init) acc_add(lo, hi, exp(0.0 - m));
  // PULL_BATCH terms per thread are loaded before any is used (one round
  // trip per batch; the sum is exact, so the grouping changes no bit)
  for (int32_t j0 = 0; j0 < n; j0 += PULL_BATCH * NT) {
    double x[PULL_BATCH];
#pragma unroll
    for (int k = 0; k < PULL_BATCH; ++k) {
      const int32_t j = j0 + k * NT + (int32_t)threadIdx.x;
      x[k] = j < n ? t[j] : 0.0;
    }
#pragma unroll
    for (int k = 0; k < PULL_BATCH; ++k)
      if (j0 + k * NT + (int32_t)threadIdx.x < n) acc_add(lo, hi, exp(x[k] - m));
  }
  block_sum128(lo, hi);
  return acc_finish(m, lo, hi);
}

// Value of a state whose one dependency contributes x (and its own empty
// path when init): the same arithmetic as thread_pull over that one term.
__device__ __forceinline__ double one_term(double x, bool init) {
  if (!init) return x;
  const double m = fmax(0.0, x);
  if (m == INFINITY) return m;
  ull lo = 0, hi = 0;
  acc_add(lo, hi, exp(0.0 - m));
  acc_add(lo, hi, exp(x - m));
  return acc_finish(m, lo, hi);
}

// ---------------------------------------------------------------------------
// generation lists
// ---------------------------------------------------------------------------

struct ScoreNext {
  GenSlot *slot;
  uint32_t qbase, hbase;
};

// Appends ready state y (record ry) to the next generation: light states to
// the light list (one atomic per wavefront), heavy ones with a workgroup per
// NT notified arcs.
template <bool FWD>
__device__ void list_ready(const ScoreArgs &S, const ScoreNext &nx, bool want, int32_t y,
                           const int4 &ry) {
  const bool heavy = want && (rec_flags(ry) & REC_HEAVY);
  const bool light = want && !heavy;
  const ull m = __ballot(light);
  if (m) {
    const int leader = __ffsll((long long)m) - 1;
    uint32_t base = 0;
    if ((int)__lane_id() == leader) base = atomicAdd(&nx.slot->qcount, (uint32_t)__popcll(m));
    base = __shfl(base, leader);
    if (light) {
      const uint32_t pos = nx.qbase + base + (uint32_t)__popcll(m & __lanemask_lt());
      if (pos < S.cap) S.Q[pos] = y;
      else S.sc->overflow = 1u;
    }
  }
  if (heavy) {
    const int32_t nd = notify_list<FWD>(S.G, y).n;
    const uint32_t blocks = nd > 0 ? (uint32_t)((nd + NT - 1) / NT) : 1u;
    const ull old = atomicAdd(&nx.slot->hpack, ((ull)blocks << 32) | 1ull);
    const uint32_t pos = nx.hbase + (uint32_t)(old & 0xffffffffull);
    if (pos < S.cap) {
      S.H[pos] = y;
      S.hoff[pos] = (uint32_t)(old >> 32);
    } else {
      S.sc->overflow = 1u;
    }
  }
}

// The finished state's value x reaches y over arc e of weight w.  If y
// depends on nothing else it is ready: the caller walks on to it (the first
// such light y, within the depth budget) or it is listed with its term.
// Otherwise the term goes to its slot and y's pending counter counts down;
// the thread that takes it to zero lists y.
// slot >= 0 is the precomputed slot of arc e's term; -1 derives it from e.
// ry is y's record.
template <bool FWD>
__device__ __forceinline__ void settle(const ScoreArgs &S, const ScoreNext &nx, int32_t y,
                                       const int4 &ry, float w, int32_t e, long long slot,
                                       double x, int depth, int32_t &next, double &next_val,
                                       int4 &next_rec) {
  const uint32_t fy = rec_flags(ry);
  const double t = x + (double)w;
  bool ready, walk = false;
  if (fy & REC_SINGLE) {
    ready = true;
    walk = next < 0 && depth + 1 < S.chain && !(fy & REC_HEAVY);
    if (!walk) S.term[e] = t;
  } else {
    // a forward merge's term goes to its in-list position (contiguous pull)
    if (slot < 0) slot = FWD ? S.G.E + S.mpos[e] : (long long)e;
    S.term[slot] = t;
    // the lanes of the wavefront here that reach the same state count its
    // pending counter down with one atomic (the lane that takes it to zero
    // lists it) and raise its largest term with one atomic; one round per
    // distinct state
    const ull key = order_key(t);
    ull rem = __ballot(true);
    ready = false;
    while (rem) {
      const int leader = __ffsll((long long)rem) - 1;
      const ull gm = __ballot(y == __shfl(y, leader));
      ull kmax = 0;
      for (ull b = gm; b; b &= b - 1) {
        const ull o = __shfl(key, __ffsll((long long)b) - 1);
        kmax = o > kmax ? o : kmax;
      }
      if ((int)__lane_id() == leader) {
        atomicMax(S.mkey + y, kmax);
        const int32_t k = (int32_t)__popcll(gm);
        ready = atomicSub(S.pend + y, k) == k;
      }
      rem &= ~gm;
    }
  }
  if (walk) {
    next = y;
    next_val = one_term(t, (fy & REC_INIT) != 0);
    next_rec = ry;
  }
  list_ready<FWD>(S, nx, ready && !walk, y, ry);
}

// Notified arc j of a state's notify list: arc id, other end, weight.
template <bool FWD>
__device__ __forceinline__ void notified(const ScoreGraph &G, const int4 &rv, int32_t j,
                                         int32_t &e, int32_t &y, float &w) {
  e = (rec_flags(rv) & REC_IND) ? G.marc[rv.x + j] : rv.x + j;
  y = FWD ? G.dst[e] : G.src[e];
  w = G.w[e];
}

// A settle left for later: state y (record ry) gets the term x + w over arc
// e (slot as in settle).  y < 0: none.
struct Pending {
  int32_t y, e;
  int4 ry;
  float w;
  long long slot;
  double x;
};

// Finishes state v (record rv) with value x, then walks on depth-first.
// A walk along single arcs stops at the first state it may not walk to.
// That last settle is left in *defer when given (the caller settles it
// together with the workgroup's others), else it is done after the loop,
// when every lane of the wavefront has stopped: walks have different
// lengths, and the atomics of lanes that stop early would otherwise hold up
// the lanes still walking.
template <bool FWD>
__device__ __forceinline__ void walk_from(const ScoreArgs &S, const ScoreNext &nx, int32_t v, int4 rv, double x,
                          int depth, uint32_t &fin, Pending *defer) {
  Pending p;
  p.y = -1;
  for (;;) {
    const int32_t nd = rec_count(rv);
    if (nd == 1) {
      const int32_t y = rv.x;
      const int4 ry = S.rec[y];
      // v's value is stored after the load of y's record is issued (a wait
      // for a load also waits for every store issued before it)
      S.val[v] = x;
      ++fin;
      const float w = __int_as_float(rv.z);
      const uint32_t fy = rec_flags(ry);
      if ((fy & REC_SINGLE) && !(fy & REC_HEAVY) && depth + 1 < S.chain) {
        // v was y's only dependency: y's value follows here
        x = one_term(x + (double)w, (fy & REC_INIT) != 0);
        v = y;
        rv = ry;
        ++depth;
        continue;
      }
      // the slot is the arc id unless it leads to a forward merge, where the
      // arc id is not needed (a merge's terms go to their precomputed slots)
      p.slot = (long long)(uint32_t)rv.w;
      p.e = p.slot < S.G.E ? (int32_t)p.slot : -1;
      p.y = y;
      p.ry = ry;
      p.w = w;
      p.x = x;
      break;
    }
    S.val[v] = x;
    ++fin;
    int32_t next = -1;
    double next_val = 0.0;
    int4 next_rec = rv;
    for (int32_t j = 0; j < nd; ++j) {
      int32_t e, y;
      float w;
      notified<FWD>(S.G, rv, j, e, y, w);
      settle<FWD>(S, nx, y, S.rec[y], w, e, -1, x, depth, next, next_val, next_rec);
    }
    if (next < 0) break;
    v = next;
    x = next_val;
    rv = next_rec;
    ++depth;
  }
  if (defer) {
    *defer = p;
  } else if (p.y >= 0) {
    int32_t none = 0;  // >= 0: no walk from here
    double nv;
    int4 nr;
    settle<FWD>(S, nx, p.y, p.ry, p.w, p.e, p.slot, p.x, depth, none, nv, nr);
  }
}

// The pending settles of a workgroup (every thread calls; p.y < 0: none).
// Terms go to their slots; the arrivals at each merge are first gathered in
// an LDS table keyed by the merge, so that one atomic per distinct merge
// and workgroup counts its pending counter down and raises its largest
// term.  Many walks of a generation end at the same few merges, where
// atomics of single wavefronts would queue up behind each other.
template <bool FWD>
__device__ void settle_block(const ScoreArgs &S, const ScoreNext &nx, const Pending &p) {
  __shared__ int32_t s_y[NT];
  __shared__ uint32_t s_n[NT];
  __shared__ ull s_k[NT];
  __shared__ uint32_t s_f[NT];
  const unsigned tid = threadIdx.x;
  __syncthreads();  // the previous use of the table is over
  s_y[tid] = -1;
  s_n[tid] = 0;
  s_k[tid] = 0;
  __syncthreads();
  const uint32_t fy = rec_flags(p.ry);
  const bool single = p.y >= 0 && (fy & REC_SINGLE);
  const bool merge = p.y >= 0 && !(fy & REC_SINGLE);
  if (p.y >= 0) {
    const double t = p.x + (double)p.w;
    long long slot = p.slot;
    if (single) slot = p.e;
    else if (slot < 0) slot = FWD ? S.G.E + S.mpos[p.e] : (long long)p.e;
    S.term[slot] = t;
    if (merge) {
      static_assert(NT == 256, "the table hash yields 8 bits");
      uint32_t h = ((uint32_t)p.y * 2654435761u) >> 24;  // one of NT buckets
      for (;;) {
        const int32_t old = atomicCAS(&s_y[h], -1, p.y);
        if (old == -1 || old == p.y) break;
        h = (h + 1) & (NT - 1);
      }
      atomicAdd(&s_n[h], 1u);
      atomicMax(&s_k[h], order_key(t));
      s_f[h] = fy;  // the same flags from every lane that reaches p.y
    }
  }
  __syncthreads();
  // a single-dependency state not walked to is ready
  list_ready<FWD>(S, nx, single, p.y, p.ry);
  const int32_t y = s_y[tid];
  bool ready = false;
  int4 ry = make_int4(0, 0, 0, 0);
  if (y >= 0) {
    const int32_t k = (int32_t)s_n[tid];
    atomicMax(S.mkey + y, s_k[tid]);
    ready = atomicSub(S.pend + y, k) == k;
    ry.y = (int32_t)s_f[tid];
  }
  list_ready<FWD>(S, nx, ready, y, ry);
}

// Generation g of one direction on workgroups bid = 0 .. nb - 1: workgroups
// of heavy states, then one thread per light state.
template <bool FWD>
__device__ void gen_body(const ScoreArgs &S, int g, unsigned bid, unsigned nb) {
  ScoreScalars *sc = S.sc;
  const uint32_t ovf = sc->overflow;
  const GenSlot cur = sc->G[g % 3];
  if (ovf) return;
  const uint32_t hcount = (uint32_t)(cur.hpack & 0xffffffffull);
  const ull HB = cur.hpack >> 32;
  ScoreNext nx;
  nx.slot = &sc->G[(g + 1) % 3];
  nx.qbase = cur.qbase + cur.qcount;
  nx.hbase = cur.hbase + hcount;
  if (bid == 0 && threadIdx.x == 0) {
    nx.slot->qbase = nx.qbase;  // read by generation g + 1 only
    nx.slot->hbase = nx.hbase;
    GenSlot *done = &sc->G[(g + 2) % 3];  // generation g - 1: free
    done->qcount = 0;
    done->hpack = 0;
    if (HB + cur.qcount) sc->gens = (uint32_t)g + 1;
  }
  uint32_t fin = 0;
  const uint32_t *ho = S.hoff + cur.hbase;
  for (ull ub = bid; ub < HB; ub += nb) {
    // the heavy state of unit ub: entry a, the last one with ho[a] <= ub
    int32_t v;
    uint32_t hoa;
    if (hcount <= (uint32_t)WAVE) {
      const uint32_t l = __lane_id();
      const bool in = l < hcount;
      const uint32_t hl = in ? ho[l] : 0u;
      const int32_t vl = in ? S.H[cur.hbase + l] : 0;
      const int a = __popcll(__ballot(in && (ull)hl <= ub)) - 1;  // ho[0] = 0
      v = __shfl(vl, a);
      hoa = __shfl(hl, a);
    } else {
      uint32_t a = 0, b = hcount - 1;
      while (a < b) {
        const uint32_t mid = (a + b + 1) >> 1;
        if (ho[mid] <= ub) a = mid; else b = mid - 1;
      }
      v = S.H[cur.hbase + a];
      hoa = ho[a];
    }
    const uint32_t part = (uint32_t)(ub - hoa);
    const long long j = (long long)part * NT + threadIdx.x;
    // The loads of the pull and of this thread's notified arc are issued
    // round by round together: neither needs the other's values, and only
    // the settle at the end needs the pulled value.
    const int32_t r_in = S.G.inref[v];
    const int32_t o0 = S.G.off[v], o1 = S.G.off[v + 1];
    const ull mk = S.mkey[v];
    const int4 rv = S.rec[v];
    const AList out = AList{o0, o1 - o0, false};
    int32_t e = -1, y = -1;
    float w = 0.0f;
    if (FWD && j < out.n) {
      e = o0 + (int32_t)j;
      y = S.G.dst[e];
      w = S.G.w[e];
    }
    AList in = AList{r_in >= 0 ? r_in : 0, r_in >= 0 ? 1 : 0, false};
    if (r_in <= -2) in = AList{S.G.mbeg[-2 - r_in], S.G.mlen[-2 - r_in], true};
    if (!FWD && j < in.n) {
      e = arc_at(S.G, in, (int32_t)j);
      y = S.G.src[e];
      w = S.G.w[e];
    }
    const AList nl = FWD ? out : in, pl = FWD ? in : out;
    int4 ry = make_int4(0, 0, 0, 0);
    if (j < nl.n) ry = S.rec[y];
    const bool init = (rec_flags(rv) & REC_INIT) != 0;
    const double *t = pull_slots(S, pl);
    double m;
    if (pl.n >= 2) {
      m = mk ? from_order_key(mk) : -INFINITY;
      if (init) m = fmax(m, 0.0);
    } else {
      m = init ? 0.0 : -INFINITY;
      if (pl.n == 1) m = fmax(m, t[0]);
    }
    const double x = block_logsum(t, pl.n, m, init);
    if (part == 0 && threadIdx.x == 0) {
      S.val[v] = x;
      ++fin;
    }
    int32_t next = -1;
    double next_val = 0.0;
    int4 next_rec = rv;
    if (j < nl.n) settle<FWD>(S, nx, y, ry, w, e, -1, x, 0, next, next_val, next_rec);
    Pending pd;
    pd.y = -1;
    if (next >= 0) walk_from<FWD>(S, nx, next, next_rec, next_val, 1, fin, &pd);
    settle_block<FWD>(S, nx, pd);
  }
  // light states start at the workgroups with the fewest heavy units (the
  // heavy units went to workgroups 0, 1, ... in turn), so walks cut short
  // by the depth budget resume beside the heavy work, not behind it
  const ull n = cur.qcount;
  const unsigned hrem = (unsigned)(HB % nb);
  const unsigned lb = bid >= hrem ? bid - hrem : bid + nb - hrem;
  for (ull i = (ull)lb * NT + threadIdx.x; i < n; i += (ull)nb * NT) {
    const int32_t v = S.Q[cur.qbase + (uint32_t)i];
    const int4 rv = S.rec[v];
    const double x =
        thread_pull<FWD>(S, v, pull_list<FWD>(S.G, v), (rec_flags(rv) & REC_INIT) != 0);
    walk_from<FWD>(S, nx, v, rv, x, 0, fin, nullptr);
  }
  // one atomic per wavefront
#pragma unroll
  for (int o = WAVE / 2; o > 0; o >>= 1) fin += __shfl_xor(fin, o);
  if (__lane_id() == 0 && fin) atomicAdd(&sc->finished, (ull)fin);
}

template <bool FWD>
__global__ __launch_bounds__(NT) void k_score_gen(ScoreArgs S, int g) {
  gen_body<FWD>(S, g, blockIdx.x, gridDim.x);
}

// Both directions at once (they are independent): the first half of the
// workgroups advances the forward recursion, the second half the backward.
__global__ __launch_bounds__(NT) void k_score_gen2(ScoreArgs F, ScoreArgs B, int g) {
  const unsigned half = gridDim.x / 2;
  if (blockIdx.x < half) gen_body<true>(F, g, blockIdx.x, half);
  else gen_body<false>(B, g, blockIdx.x - half, half);
}

// Every state of one direction in one pass: its record (see REC_*), its
// pending counter (the number of arcs it pulls from) and no largest term
// yet, both only for states with two or more (no other state's are read),
// and, for a state that depends on nothing (forward: no in-arc; backward:
// no out-arc), its place in generation 0.  ST_ITEMS states per thread and
// round, each round's loads issued level by level before the stores; the
// rounds run in whole wavefronts (list_ready uses ballots).
template <bool FWD>
__global__ __launch_bounds__(NT) void k_score_init(ScoreArgs S) {
  const ScoreGraph &G = S.G;
  ScoreNext nx;
  nx.slot = &S.sc->G[0];
  nx.qbase = 0;
  nx.hbase = 0;
  const long long V = G.V, stride = (long long)gridDim.x * NT * ST_ITEMS;
  for (long long base = (long long)blockIdx.x * NT * ST_ITEMS; base < V; base += stride) {
    int32_t o0[ST_ITEMS], o1[ST_ITEMS], ir[ST_ITEMS];
    uint8_t fl[ST_ITEMS];
#pragma unroll
    for (int k = 0; k < ST_ITEMS; ++k) {
      const long long v = base + (long long)k * NT + threadIdx.x;
      o0[k] = o1[k] = 0;
      ir[k] = -1;
      fl[k] = 0;
      if (v < V) {
        o0[k] = G.off[v];
        o1[k] = G.off[v + 1];
        ir[k] = G.inref[v];
        fl[k] = FWD ? G.start[v] : G.accept[v];
      }
    }
    AList pl[ST_ITEMS], nl[ST_ITEMS];
#pragma unroll
    for (int k = 0; k < ST_ITEMS; ++k) {
      AList in = AList{ir[k] >= 0 ? ir[k] : 0, ir[k] >= 0 ? 1 : 0, false};
      if (ir[k] <= -2) in = AList{G.mbeg[-2 - ir[k]], G.mlen[-2 - ir[k]], true};
      const AList out = AList{o0[k], o1[k] - o0[k], false};
      pl[k] = FWD ? in : out;
      nl[k] = FWD ? out : in;
    }
    // the one notified arc (if so): its id, other end, weight and slot
    int32_t e[ST_ITEMS], x[ST_ITEMS], wz[ST_ITEMS], mp[ST_ITEMS];
#pragma unroll
    for (int k = 0; k < ST_ITEMS; ++k) {
      e[k] = -1;
      if (nl[k].n == 1) e[k] = nl[k].ind ? G.marc[nl[k].beg] : nl[k].beg;
    }
#pragma unroll
    for (int k = 0; k < ST_ITEMS; ++k) {
      x[k] = wz[k] = mp[k] = 0;
      if (e[k] >= 0) {
        x[k] = FWD ? G.dst[e[k]] : G.src[e[k]];
        wz[k] = __float_as_int(G.w[e[k]]);
        if (FWD) mp[k] = S.mpos[e[k]];
      }
    }
    bool to_merge[ST_ITEMS];
#pragma unroll
    for (int k = 0; k < ST_ITEMS; ++k) to_merge[k] = FWD && e[k] >= 0 && G.inref[x[k]] <= -2;
#pragma unroll
    for (int k = 0; k < ST_ITEMS; ++k) {
      const long long v = base + (long long)k * NT + threadIdx.x;
      bool want = false;
      int4 r = make_int4(0, 0, 0, 0);
      if (v < V) {
        uint32_t f = fl[k] ? REC_INIT : 0u;
        if (pl[k].n == 1) f |= REC_SINGLE;
        if (pl[k].n > SCORE_LIGHT || nl[k].n > SCORE_LIGHT) f |= REC_HEAVY;
        if (nl[k].ind) f |= REC_IND;
        const int32_t cnt = nl[k].n < (int32_t)REC_COUNT ? nl[k].n : (int32_t)REC_COUNT;
        r.y = (int32_t)(f | (uint32_t)cnt);
        if (e[k] >= 0) {
          r.x = x[k];
          r.z = wz[k];
          // slot of the term (see pull_slots); < 2^32 since E < 2^31
          r.w = (int32_t)(uint32_t)(to_merge[k] ? (ull)G.E + (uint32_t)mp[k] : (ull)e[k]);
        } else {
          r.x = nl[k].beg;
          r.z = 0;
          r.w = -1;
        }
        S.rec[v] = r;
        if (pl[k].n >= 2) {
          S.pend[v] = pl[k].n;
          S.mkey[v] = 0ull;
        }
        want = pl[k].n == 0;
      }
      list_ready<FWD>(S, nx, want, (int32_t)v, r);
    }
  }
}

// ---------------------------------------------------------------------------
// relaxation sweeps (graphs with cycles)
// ---------------------------------------------------------------------------

// The value of state v from the values x of the previous sweep: the exact
// log-add of thread_pull over the terms x[other end] + w(e) of v's pull list
// and, for a start (forward) or accepting (backward) state, its empty
// path's 0.  The terms are formed twice (their maximum first).  Since every
// step is the recursion's own, the sweeps reach on a graph without cycles
// the recursion's values bit for bit.
template <bool FWD>
__device__ double sweep_value(const ScoreGraph &G, const double *x, int32_t v, bool init) {
  // forward: the in-arc CSR; backward: the out-arcs
  const int32_t b = FWD ? G.ioff[v] : G.off[v];
  const AList l = AList{b, (FWD ? G.ioff[v + 1] : G.off[v + 1]) - b, false};
  auto term = [&](int32_t j) -> double {
    const int32_t p = l.beg + j;
    return FWD ? x[G.isrc[p]] + (double)G.iw[p] : x[G.dst[p]] + (double)G.w[p];
  };
  if (l.n == 1 && !init) return term(0);
  double m = init ? 0.0 : -INFINITY;
  ull lo = 0, hi = 0;
  if (l.n <= SWEEP_REGS) {
    // few terms: each loaded once, kept in registers
    double t[SWEEP_REGS];
#pragma unroll
    for (int j = 0; j < SWEEP_REGS; ++j) {
      t[j] = j < l.n ? term(j) : -INFINITY;
      m = fmax(m, t[j]);
    }
    if (m == -INFINITY || m == INFINITY) return m;
    if (init) acc_add(lo, hi, exp(0.0 - m));
#pragma unroll
    for (int j = 0; j < SWEEP_REGS; ++j)
      if (j < l.n) acc_add(lo, hi, exp(t[j] - m));
    return acc_finish(m, lo, hi);
  }
  for (int32_t j = 0; j < l.n; ++j) m = fmax(m, term(j));
  if (m == -INFINITY || m == INFINITY) return m;
  if (init) acc_add(lo, hi, exp(0.0 - m));
  for (int32_t j = 0; j < l.n; ++j) acc_add(lo, hi, exp(term(j) - m));
  return acc_finish(m, lo, hi);
}

// How much a value rose in a sweep (0 if it did not; a value that leaves
// -inf rises by +inf).
__device__ __forceinline__ double rise(double before, double after) {
  if (!(after > before)) return 0.0;
  return before == -INFINITY ? INFINITY : after - before;
}

// One Jacobi sweep of both recursions over every state: ya = sweep of xa
// (forward), yb = sweep of xb (backward); a direction whose output is null
// is skipped.  *incr = max(*incr, order key of the largest rise), one
// atomic per workgroup.
__global__ __launch_bounds__(NT) void k_sweep(ScoreGraph G, const double *xa, double *ya,
                                              const double *xb, double *yb, ull *incr) {
  __shared__ ull s_m[NWAVES];
  ull mk = 0;
  for (long long v = (long long)blockIdx.x * NT + threadIdx.x; v < G.V;
       v += (long long)gridDim.x * NT) {
    double r = 0.0;
    if (ya) {
      const double a = sweep_value<true>(G, xa, (int32_t)v, G.start[v] != 0);
      r = fmax(r, rise(xa[v], a));
      ya[v] = a;
    }
    if (yb) {
      const double b = sweep_value<false>(G, xb, (int32_t)v, G.accept[v] != 0);
      r = fmax(r, rise(xb[v], b));
      yb[v] = b;
    }
    const ull k = order_key(r);
    mk = k > mk ? k : mk;
  }
#pragma unroll
  for (int o = WAVE / 2; o > 0; o >>= 1) {
    const ull t = __shfl_xor(mk, o);
    mk = t > mk ? t : mk;
  }
  if (__lane_id() == 0) s_m[threadIdx.x / WAVE] = mk;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < NWAVES; ++w) mk = s_m[w] > mk ? s_m[w] : mk;
    atomicMax(incr, mk);
  }
}

// In-arc CSR: the in-degrees (one atomic per arc), then, after a scan,
// every arc placed at its target's cursor.
__global__ __launch_bounds__(NT) void k_in_count(ScoreGraph G, int32_t *cnt) {
  for (long long e = (long long)blockIdx.x * NT + threadIdx.x; e < G.E;
       e += (long long)gridDim.x * NT)
    atomicAdd(cnt + G.dst[e], 1);
}

__global__ __launch_bounds__(NT) void k_in_place(ScoreGraph G, const int32_t *ioff,
                                                 int32_t *cur, int32_t *isrc, float *iw) {
  for (long long e = (long long)blockIdx.x * NT + threadIdx.x; e < G.E;
       e += (long long)gridDim.x * NT) {
    const int32_t d = G.dst[e];
    const int32_t p = ioff[d] + atomicAdd(cur + d, 1);
    isrc[p] = G.src[e];
    iw[p] = G.w[e];
  }
}

__global__ __launch_bounds__(NT) void k_fill_f64(double *p, long long n, double x) {
  for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < n;
       i += (long long)gridDim.x * NT)
    p[i] = x;
}

// ---------------------------------------------------------------------------
// in-arc structure
// ---------------------------------------------------------------------------

// owner[v] = the id of one in-arc of v (whichever store lands last).  Plain
// aligned 32-bit stores: concurrent ones to one address leave one of the
// stored values, and the next kernel (after the kernel boundary's release
// and acquire) reads that one value everywhere.  Device-scope atomic stores
// and loads would write through and read past the L2 at every access.
__global__ __launch_bounds__(NT) void k_owner(ScoreGraph G, int32_t *owner) {
  const long long stride = (long long)gridDim.x * NT * ST_ITEMS;
  for (long long e0 = (long long)blockIdx.x * NT * ST_ITEMS + threadIdx.x; e0 < G.E;
       e0 += stride) {
    int32_t d[ST_ITEMS];
#pragma unroll
    for (int k = 0; k < ST_ITEMS; ++k) {
      const long long e = e0 + (long long)k * NT;
      d[k] = e < G.E ? G.dst[e] : -1;
    }
#pragma unroll
    for (int k = 0; k < ST_ITEMS; ++k)
      if (d[k] >= 0) owner[d[k]] = (int32_t)(e0 + (long long)k * NT);
  }
}

// Lanes of a wavefront that add to the same counter as the first needy lane
// add together (the targets of a merge's in-arcs are often adjacent).
__device__ __forceinline__ uint32_t wave_group(bool need, int32_t key, bool &grouped,
                                               int &leader) {
  const ull m = __ballot(need);
  grouped = false;
  leader = 0;
  if (!m) return 0;
  leader = __ffsll((long long)m) - 1;
  const int32_t lk = __shfl(key, leader);
  grouped = need && key == lk;
  const ull g = __ballot(grouped);
  return (uint32_t)__popcll(g);
}

__global__ __launch_bounds__(NT) void k_extra(ScoreGraph G, const int32_t *owner,
                                              int32_t *extra) {
  const long long stride = (long long)gridDim.x * NT * ST_ITEMS;
  for (long long base = (long long)blockIdx.x * NT * ST_ITEMS; base < G.E; base += stride) {
    int32_t xs[ST_ITEMS], ow[ST_ITEMS];
#pragma unroll
    for (int k = 0; k < ST_ITEMS; ++k) {
      const long long e = base + (long long)k * NT + threadIdx.x;
      xs[k] = e < G.E ? G.dst[e] : -1;
    }
#pragma unroll
    for (int k = 0; k < ST_ITEMS; ++k) ow[k] = xs[k] >= 0 ? owner[xs[k]] : 0;
#pragma unroll
    for (int k = 0; k < ST_ITEMS; ++k) {
      const long long e = base + (long long)k * NT + threadIdx.x;
      const int32_t x = xs[k];
      const bool need = x >= 0 && ow[k] != (int32_t)e;  // owner: k_owner, an earlier kernel
      bool grouped;
      int leader;
      const uint32_t cnt = wave_group(need, x, grouped, leader);
      if (grouped) {
        if ((int)__lane_id() == leader) atomicAdd(extra + x, (int32_t)cnt);
      } else if (need) {
        atomicAdd(extra + x, 1);
      }
    }
  }
}

// Numbers the merges (any order), gives each an in-arc list range, and sets
// inref for every state.
__global__ __launch_bounds__(NT) void k_merge_index(ScoreGraph G, const int32_t *owner,
                                                    const int32_t *extra, int32_t *inref,
                                                    int32_t *mbeg, int32_t *mlen, int32_t *mcur,
                                                    ScoreScalars *sc) {
  const long long stride = (long long)gridDim.x * NT;
  for (long long base = (long long)blockIdx.x * NT; base < G.V; base += stride) {
    const long long v = base + threadIdx.x;
    int32_t len = 0;
    if (v < G.V) {
      const int32_t ex = extra[v];
      len = ex > 0 ? ex + 1 : 0;
      if (!len) inref[v] = owner[v];
    }
    const bool want = len > 0;
    const ull m = __ballot(want);
    if (!m) continue;
    // inclusive prefix of the lengths over the wavefront
    int32_t pre = len;
#pragma unroll
    for (int o = 1; o < WAVE; o <<= 1) {
      const int32_t t = __shfl_up(pre, o);
      if ((int)__lane_id() >= o) pre += t;
    }
    const int32_t total = __shfl(pre, WAVE - 1);
    uint32_t mb = 0, lb = 0;
    if (__lane_id() == 0) {
      mb = atomicAdd(&sc->nmerge, (uint32_t)__popcll(m));
      lb = (uint32_t)atomicAdd(&sc->mtotal, (ull)total);
    }
    mb = __shfl(mb, 0);
    lb = __shfl(lb, 0);
    if (want) {
      const int32_t mi = (int32_t)(mb + (uint32_t)__popcll(m & __lanemask_lt()));
      const int32_t beg = (int32_t)lb + pre - len;
      inref[v] = -2 - mi;
      mbeg[mi] = beg;
      mlen[mi] = len;
      mcur[mi] = beg;
    }
  }
}

// In-arc lists of the merges, in any order.  Each workgroup takes chunks of
// MP_ITEMS * NT arcs and counts, in an LDS hash table, how many of them go
// into each merge; one global atomic per (chunk, merge) then reserves their
// positions (the in-arcs of a merge in a composed speech graph come from
// runs of neighbouring arcs, so a chunk meets few merges).  Arcs whose merge
// finds no table slot take their position with their own atomic.
constexpr int MP_ITEMS = 16;
constexpr int MP_TABLE = 512;

__device__ __forceinline__ int mp_slot(int32_t *keys, int32_t m, bool insert) {
  int h = (int)(((uint32_t)m * 2654435761u) >> 23) & (MP_TABLE - 1);
  for (int probe = 0; probe < 32; ++probe) {
    const int32_t k = insert ? atomicCAS(keys + h, -1, m) : keys[h];
    if (k == m || (insert && k == -1)) return h;
    if (!insert && k == -1) return -1;
    h = (h + 1) & (MP_TABLE - 1);
  }
  return -1;
}

__global__ __launch_bounds__(NT) void k_merge_place(ScoreGraph G, const int32_t *inref,
                                                    int32_t *mcur, int32_t *marc,
                                                    int32_t *mpos) {
  __shared__ int32_t s_key[MP_TABLE], s_cnt[MP_TABLE], s_base[MP_TABLE];
  const long long chunk = (long long)MP_ITEMS * NT;
  for (long long base = (long long)blockIdx.x * chunk; base < G.E;
       base += (long long)gridDim.x * chunk) {
    for (int i = threadIdx.x; i < MP_TABLE; i += NT) {
      s_key[i] = -1;
      s_cnt[i] = 0;
    }
    __syncthreads();
    int32_t mi[MP_ITEMS];
    int slot[MP_ITEMS];
    // the loads of all items first (targets, then their inref)
#pragma unroll
    for (int j = 0; j < MP_ITEMS; ++j) {
      const long long e = base + (long long)j * NT + threadIdx.x;
      mi[j] = e < G.E ? G.dst[e] : -1;
    }
#pragma unroll
    for (int j = 0; j < MP_ITEMS; ++j) {
      const int32_t r = mi[j] >= 0 ? inref[mi[j]] : -1;
      mi[j] = r <= -2 ? -2 - r : -1;
    }
#pragma unroll
    for (int j = 0; j < MP_ITEMS; ++j) {
      slot[j] = -1;
      if (mi[j] >= 0) {
        slot[j] = mp_slot(s_key, mi[j], true);
        if (slot[j] >= 0) atomicAdd(s_cnt + slot[j], 1);
      }
    }
    __syncthreads();
    for (int i = threadIdx.x; i < MP_TABLE; i += NT)
      if (s_key[i] >= 0) {
        s_base[i] = atomicAdd(mcur + s_key[i], s_cnt[i]);
        s_cnt[i] = 0;  // now the cursor inside the reservation
      }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < MP_ITEMS; ++j) {
      if (mi[j] < 0) continue;
      const long long e = base + (long long)j * NT + threadIdx.x;
      const int32_t pos = slot[j] >= 0 ? s_base[slot[j]] + atomicAdd(s_cnt + slot[j], 1)
                                       : atomicAdd(mcur + mi[j], 1);
      marc[pos] = (int32_t)e;
      mpos[e] = pos;
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// total: log-add of val over the flagged states (same exact log-add)
// ---------------------------------------------------------------------------


// Calls f(v) for every v < V with flag[v] set: sixteen flags per load when
// the flags are 16-byte aligned (flagged states are few: accepting or start
// states), one byte per load for the rest.
template <class F>
__device__ __forceinline__ void for_flagged(const uint8_t *flag, int32_t V, F &&f) {
  const long long stride = (long long)gridDim.x * NT;
  const long long n16 = ((uintptr_t)flag & 15) ? 0 : (long long)V / 16;
  const uint4 *f16 = reinterpret_cast<const uint4 *>(flag);
  for (long long w = (long long)blockIdx.x * NT + threadIdx.x; w < n16; w += stride) {
    const uint4 q = f16[w];
    if (!(q.x | q.y | q.z | q.w)) continue;
    const uint32_t word[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int j = 0; j < 16; ++j)
      if ((word[j >> 2] >> (8 * (j & 3))) & 0xffu) f(16 * w + j);
  }
  for (long long v = 16 * n16 + (long long)blockIdx.x * NT + threadIdx.x; v < V; v += stride)
    if (flag[v]) f(v);
}

__global__ __launch_bounds__(NT) void k_total_max(const double *val, const uint8_t *flag,
                                                  int32_t V, ScoreScalars *sc) {
  double m = -INFINITY;
  for_flagged(flag, V, [&](long long v) { m = fmax(m, val[v]); });
  m = block_fmax(m);
  if (threadIdx.x == 0 && m != -INFINITY) atomicMax(&sc->zmax, order_key(m));
}

__global__ __launch_bounds__(NT) void k_total_sum(const double *val, const uint8_t *flag,
                                                  int32_t V, ScoreScalars *sc) {
  if (sc->zmax == 0) return;  // nothing flagged is finite
  const double M = from_order_key(sc->zmax);
  if (M == INFINITY) return;
  ull lo = 0, hi = 0;
  for_flagged(flag, V, [&](long long v) { acc_add(lo, hi, exp(val[v] - M)); });
  block_sum128(lo, hi);
  if (threadIdx.x == 0 && (lo | hi)) {
    const ull old = atomicAdd(&sc->zlo, lo);
    const ull carry = old + lo < old ? 1ull : 0ull;
    atomicAdd(&sc->zhi, hi + carry);
  }
}

__global__ void k_total_final(ScoreScalars *sc, double *total) {
  if (sc->zmax == 0) {
    *total = -INFINITY;
    return;
  }
  *total = acc_finish(from_order_key(sc->zmax), sc->zlo, sc->zhi);
}

// Segments (blockIdx.y = segment i, states [bounds[i], bounds[i + 1])):
// the same exact log-add per segment; z holds 3 words per segment (order
// key of the maximum, 128-bit sum).
__global__ __launch_bounds__(NT) void k_seg_max(const double *val, const uint8_t *flag,
                                                const long long *bounds, ull *z) {
  const int i = blockIdx.y;
  const long long lo = bounds[i], hi = bounds[i + 1];
  double m = -INFINITY;
  for (long long v = lo + (long long)blockIdx.x * NT + threadIdx.x; v < hi;
       v += (long long)gridDim.x * NT)
    if (flag[v]) m = fmax(m, val[v]);
  m = block_fmax(m);
  if (threadIdx.x == 0 && m != -INFINITY) atomicMax(z + 3 * i, order_key(m));
}

__global__ __launch_bounds__(NT) void k_seg_sum(const double *val, const uint8_t *flag,
                                                const long long *bounds, ull *z) {
  const int i = blockIdx.y;
  if (z[3 * i] == 0) return;  // nothing flagged is finite
  const double M = from_order_key(z[3 * i]);
  if (M == INFINITY) return;
  const long long lo = bounds[i], hi = bounds[i + 1];
  ull slo = 0, shi = 0;
  for (long long v = lo + (long long)blockIdx.x * NT + threadIdx.x; v < hi;
       v += (long long)gridDim.x * NT)
    if (flag[v]) acc_add(slo, shi, exp(val[v] - M));
  block_sum128(slo, shi);
  if (threadIdx.x == 0 && (slo | shi)) {
    const ull old = atomicAdd(z + 3 * i + 1, slo);
    const ull carry = old + slo < old ? 1ull : 0ull;
    atomicAdd(z + 3 * i + 2, shi + carry);
  }
}

__global__ __launch_bounds__(NT) void k_seg_final(int32_t n, const ull *z, double *totals) {
  for (int i = blockIdx.x * NT + threadIdx.x; i < n; i += gridDim.x * NT)
    totals[i] = z[3 * i] == 0 ? -INFINITY : acc_finish(from_order_key(z[3 * i]), z[3 * i + 1],
                                                       z[3 * i + 2]);
}

// ---------------------------------------------------------------------------
// posteriors and the provenance scatter
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(NT) void k_posterior(ScoreGraph G, const double *alpha,
                                                  const double *beta, const double *total,
                                                  float scale, float *grad) {
  const double Z = *total;
  for (long long e = (long long)blockIdx.x * NT + threadIdx.x; e < G.E;
       e += (long long)gridDim.x * NT) {
    double p = 0.0;
    if (Z != -INFINITY) p = exp(alpha[G.src[e]] + (double)G.w[e] + beta[G.dst[e]] - Z);
    grad[e] = (float)((double)scale * p);
  }
}

__global__ __launch_bounds__(NT) void k_absmax(const float *g, long long n, uint32_t *mx) {
  uint32_t m = 0;  // |g| orders as its bits
  const long long n4 = ((uintptr_t)g & 15) ? 0 : n / 4;
  const float4 *g4 = reinterpret_cast<const float4 *>(g);
#pragma unroll 4
  for (long long e = (long long)blockIdx.x * NT + threadIdx.x; e < n4;
       e += (long long)gridDim.x * NT) {
    const float4 q = g4[e];
    m = max(m, __float_as_uint(q.x) & 0x7fffffffu);
    m = max(m, __float_as_uint(q.y) & 0x7fffffffu);
    m = max(m, __float_as_uint(q.z) & 0x7fffffffu);
    m = max(m, __float_as_uint(q.w) & 0x7fffffffu);
  }
  for (long long e = 4 * n4 + (long long)blockIdx.x * NT + threadIdx.x; e < n;
       e += (long long)gridDim.x * NT)
    m = max(m, __float_as_uint(g[e]) & 0x7fffffffu);
#pragma unroll
  for (int o = WAVE / 2; o > 0; o >>= 1) m = max(m, (uint32_t)__shfl_xor(m, o));
  // one atomic per workgroup (same-address atomics serialize)
  __shared__ uint32_t s_m[NWAVES];
  if (__lane_id() == 0) s_m[threadIdx.x / WAVE] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < NWAVES; ++w) m = max(m, s_m[w]);
    if (m) atomicMax(mx, m);
  }
}

// Scale exponent: every |g| < 2^ex, so |g| * 2^(64 - ex) < 2^64.
__device__ __forceinline__ int scale_exp(uint32_t mbits) {
  int ex = 0;
  (void)frexpf(__uint_as_float(mbits), &ex);
  return ex;
}

// acc[4 i + 0, 1]: digits of the positive terms of target i, [2, 3] of the
// negative ones (low 32 bits, high 32 bits of each 64-bit magnitude).
//
// Each workgroup takes chunks of SC_CHUNK terms.  When a chunk's targets
// span at most SC_BINS indices (provenance of consecutive arcs of C often
// does: they come from a few states of A), the chunk is added up in LDS with
// LDS atomics and only its nonzero words go to global atomics; otherwise
// every term goes to global atomics, lanes of a wavefront that share the
// first lane's target adding together.  Integer sums: the order is free.
constexpr int SC_CHUNK = NT * 32;
constexpr int SC_BINS = 2048;
constexpr long long SC_BLOCKS = 2048;  // workgroups of the grouping passes
constexpr int SC_ITEMS = 8;  // terms per thread whose loads are issued together

// Fixed-point digits of one term (target i, gradient x); i = -1: no term
// (also the lanes of a batch past the end of the terms).
__device__ __forceinline__ bool term_digits(int32_t i, float x, int32_t m, int ex, int32_t &key,
                                            ull &d0, ull &d1, uint32_t *bad) {
  key = -1;
  d0 = d1 = 0;
  if (i < -1 || i >= m) {
    atomicOr(bad, 1u);
    return false;
  }
  if (i < 0) return false;
  const ull T = (ull)ldexp(fabs((double)x), 64 - ex);
  if (!T) return false;
  key = 2 * i + (x < 0.f ? 1 : 0);
  d0 = T & 0xffffffffull;
  d1 = T >> 32;
  return true;
}

__device__ __forceinline__ bool scatter_digits(const float *g, const int32_t *idx, long long e,
                                               int32_t m, int ex, int32_t &key, ull &d0,
                                               ull &d1, uint32_t *bad) {
  const int32_t i = idx[e];
  return term_digits(i, (i >= 0 && i < m) ? g[e] : 0.f, m, ex, key, d0, d1, bad);
}

// n_dev, when given, holds the number of terms instead of n.
__global__ __launch_bounds__(NT) void k_scatter(const float *g, const int32_t *idx, long long n,
                                                int32_t m, const uint32_t *mx, ull *acc,
                                                uint32_t *bad, const ull *n_dev) {
  __shared__ ull s_acc[4 * SC_BINS];
  __shared__ int32_t s_lo[NWAVES], s_hi[NWAVES];
  if (n_dev) n = (long long)*n_dev;
  const uint32_t mbits = *mx;
  if (mbits == 0 || mbits >= 0x7f800000u) return;  // all zero, or not finite
  const int ex = scale_exp(mbits);
  for (long long base = (long long)blockIdx.x * SC_CHUNK; base < n;
       base += (long long)gridDim.x * SC_CHUNK) {
    const long long end = base + SC_CHUNK < n ? base + SC_CHUNK : n;
    // index range of the chunk
    int32_t lo = 0x7fffffff, hi = -1;
    for (long long e0 = base + threadIdx.x; e0 < end; e0 += (long long)NT * SC_ITEMS) {
      int32_t iv[SC_ITEMS];
#pragma unroll
      for (int k = 0; k < SC_ITEMS; ++k) {
        const long long e = e0 + (long long)k * NT;
        iv[k] = e < end ? idx[e] : -1;
      }
#pragma unroll
      for (int k = 0; k < SC_ITEMS; ++k)
        if (iv[k] >= 0 && iv[k] < m) {
          lo = min(lo, iv[k]);
          hi = max(hi, iv[k]);
        }
    }
#pragma unroll
    for (int o = WAVE / 2; o > 0; o >>= 1) {
      lo = min(lo, __shfl_xor(lo, o));
      hi = max(hi, __shfl_xor(hi, o));
    }
    __syncthreads();  // s_acc / s_lo of the previous chunk are no longer read
    if (__lane_id() == 0) {
      s_lo[threadIdx.x / WAVE] = lo;
      s_hi[threadIdx.x / WAVE] = hi;
    }
    __syncthreads();
    lo = s_lo[0];
    hi = s_hi[0];
#pragma unroll
    for (int w = 1; w < NWAVES; ++w) {
      lo = min(lo, s_lo[w]);
      hi = max(hi, s_hi[w]);
    }
    if (hi < 0) {
      // nothing to add; still report bad indices
      for (long long e = base + threadIdx.x; e < end; e += NT) {
        const int32_t i = idx[e];
        if (i < -1 || i >= m) atomicOr(bad, 1u);
      }
      continue;
    }
    if (hi - lo < SC_BINS) {
      const int words = 4 * (hi - lo + 1);
      for (int b = threadIdx.x; b < words; b += NT) s_acc[b] = 0ull;
      __syncthreads();
      for (long long e0 = base + threadIdx.x; e0 < end; e0 += (long long)NT * SC_ITEMS) {
        int32_t iv[SC_ITEMS];
        float gv[SC_ITEMS];
#pragma unroll
        for (int k = 0; k < SC_ITEMS; ++k) {
          const long long e = e0 + (long long)k * NT;
          iv[k] = e < end ? idx[e] : -1;
          gv[k] = e < end ? g[e] : 0.f;
        }
#pragma unroll
        for (int k = 0; k < SC_ITEMS; ++k) {
          int32_t key;
          ull d0, d1;
          if (term_digits(iv[k], gv[k], m, ex, key, d0, d1, bad)) {
            ull *a = s_acc + 2 * (key - 2 * lo);
            if (d0) atomicAdd(a, d0);
            if (d1) atomicAdd(a + 1, d1);
          }
        }
      }
      __syncthreads();
      ull *ga = acc + 4 * (size_t)lo;
      for (int b = threadIdx.x; b < words; b += NT)
        if (s_acc[b]) atomicAdd(ga + b, s_acc[b]);
    } else {
      // whole wavefronts per iteration (the grouping reads every lane)
      for (long long off = 0; off < end - base; off += NT) {
        const long long e = base + off + threadIdx.x;
        int32_t key = -1;
        ull d0 = 0, d1 = 0;
        const bool need = e < end && scatter_digits(g, idx, e, m, ex, key, d0, d1, bad);
        bool grouped;
        int leader;
        (void)wave_group(need, key, grouped, leader);
        ull s0 = grouped ? d0 : 0ull, s1 = grouped ? d1 : 0ull;
#pragma unroll
        for (int o = WAVE / 2; o > 0; o >>= 1) {
          s0 += __shfl_xor(s0, o);
          s1 += __shfl_xor(s1, o);
        }
        if (grouped && (int)__lane_id() == leader) {
          ull *a = acc + 2 * (size_t)key;
          if (s0) atomicAdd(a, s0);
          if (s1) atomicAdd(a + 1, s1);
        } else if (need && !grouped) {
          ull *a = acc + 2 * (size_t)key;
          if (d0) atomicAdd(a, d0);
          if (d1) atomicAdd(a + 1, d1);
        }
      }
    }
  }
}

// Terms whose targets are spread wider than SC_BINS within a chunk are first
// grouped by target range (bucket = target / SC_BINS): a counting pass and a
// placing pass, each workgroup over one contiguous share of the terms, with
// the wavefront's lanes of one bucket taking their places with one LDS
// atomic.  k_scatter then adds every chunk of the grouped terms in LDS.
constexpr int SC_BUCKETS = 1024;  // at most this many buckets (m <= 2^21)

// The lanes of a wavefront with want set and the same bucket b: one of them
// adds their count to h[b] (LDS); each gets the old value plus its rank.
__device__ __forceinline__ uint32_t wave_bucket_add(uint32_t *h, bool want, int32_t b) {
  uint32_t pos = 0;
  ull rem = __ballot(want);
  while (rem) {
    const int leader = __ffsll((long long)rem) - 1;
    const int32_t lb = __shfl(b, leader);
    const ull same = __ballot(want && b == lb);
    uint32_t base = 0;
    if ((int)__lane_id() == leader) base = atomicAdd(h + lb, (uint32_t)__popcll(same));
    base = __shfl(base, leader);
    if (want && b == lb) pos = base + (uint32_t)__popcll(same & __lanemask_lt());
    rem &= ~same;
  }
  return pos;
}

// cnt[b * gridDim.x + block] = terms of the block's share with a target in
// bucket b (valid targets only).
__global__ __launch_bounds__(NT) void k_bucket_count(const int32_t *idx, long long n, int32_t m,
                                                     int32_t nbk, long long per,
                                                     uint32_t *__restrict__ cnt) {
  __shared__ uint32_t h[SC_BUCKETS];
  for (int b = threadIdx.x; b < nbk; b += NT) h[b] = 0;
  __syncthreads();
  const long long e0 = (long long)blockIdx.x * per, e1 = e0 + per < n ? e0 + per : n;
  for (long long base = e0; base < e1; base += (long long)NT * SC_ITEMS) {
    int32_t iv[SC_ITEMS];
#pragma unroll
    for (int k = 0; k < SC_ITEMS; ++k) {
      const long long e = base + (long long)k * NT + threadIdx.x;
      iv[k] = e < e1 ? idx[e] : -1;
    }
#pragma unroll
    for (int k = 0; k < SC_ITEMS; ++k) {
      const bool want = iv[k] >= 0 && iv[k] < m;
      (void)wave_bucket_add(h, want, want ? iv[k] / SC_BINS : 0);
    }
  }
  __syncthreads();
  for (int b = threadIdx.x; b < nbk; b += NT) cnt[(size_t)b * gridDim.x + blockIdx.x] = h[b];
}

// Places every valid term of the block's share at off[bucket * gridDim.x +
// block] + its rank: pidx / pg grouped by bucket.  Out-of-range targets set
// *bad.
__global__ __launch_bounds__(NT) void k_bucket_place(const float *g, const int32_t *idx,
                                                     long long n, int32_t m, int32_t nbk,
                                                     long long per, const uint32_t *off,
                                                     float *__restrict__ pg,
                                                     int32_t *__restrict__ pidx, uint32_t *bad) {
  __shared__ uint32_t h[SC_BUCKETS];
  for (int b = threadIdx.x; b < nbk; b += NT) h[b] = off[(size_t)b * gridDim.x + blockIdx.x];
  __syncthreads();
  const long long e0 = (long long)blockIdx.x * per, e1 = e0 + per < n ? e0 + per : n;
  for (long long base = e0; base < e1; base += (long long)NT * SC_ITEMS) {
    int32_t iv[SC_ITEMS];
    float gv[SC_ITEMS];
#pragma unroll
    for (int k = 0; k < SC_ITEMS; ++k) {
      const long long e = base + (long long)k * NT + threadIdx.x;
      iv[k] = e < e1 ? idx[e] : -1;
      gv[k] = e < e1 ? g[e] : 0.f;
    }
#pragma unroll
    for (int k = 0; k < SC_ITEMS; ++k) {
      const int32_t i = iv[k];
      if (i < -1 || i >= m) atomicOr(bad, 1u);
      const bool want = i >= 0 && i < m;
      const uint32_t p = wave_bucket_add(h, want, want ? i / SC_BINS : 0);
      if (want) {
        pidx[p] = i;
        pg[p] = gv[k];
      }
    }
  }
}

// 128-bit (hi, lo) of d1 * 2^32 + d0.
__device__ __forceinline__ void digits128(ull d0, ull d1, ull &lo, ull &hi) {
  lo = d0 + (d1 << 32);
  hi = (d1 >> 32) + (lo < d0 ? 1ull : 0ull);
}

__global__ __launch_bounds__(NT) void k_scatter_final(const ull *acc, int32_t m,
                                                      const uint32_t *mx, float *out) {
  const uint32_t mbits = *mx;
  const int ex = (mbits == 0 || mbits >= 0x7f800000u) ? 0 : scale_exp(mbits);
  for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < m;
       i += (long long)gridDim.x * NT) {
    if (mbits == 0) {
      out[i] = 0.f;
      continue;
    }
    if (mbits >= 0x7f800000u) {
      out[i] = __uint_as_float(0x7fc00000u);  // NaN in, NaN out
      continue;
    }
    ull plo, phi, nlo, nhi;
    digits128(acc[4 * i], acc[4 * i + 1], plo, phi);
    digits128(acc[4 * i + 2], acc[4 * i + 3], nlo, nhi);
    // difference of the two 128-bit magnitudes, then one conversion
    bool neg = nhi > phi || (nhi == phi && nlo > plo);
    ull dlo, dhi;
    if (!neg) {
      dlo = plo - nlo;
      dhi = phi - nhi - (plo < nlo ? 1ull : 0ull);
    } else {
      dlo = nlo - plo;
      dhi = nhi - phi - (nlo < plo ? 1ull : 0ull);
    }
    double d = (double)dhi * 0x1p64 + (double)dlo;
    d = ldexp(d, ex - 64);
    out[i] = (float)(neg ? -d : d);
  }
}

// Zeroes words [0, n) (a kernel rather than a memset, so that the call
// that uses it records no memset node when captured in a graph).
__global__ __launch_bounds__(NT) void k_clear(ull *w, long long n) {
  for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < n;
       i += (long long)gridDim.x * NT)
    w[i] = 0ull;
}

// Device memory of fst_grad_scatter_noalloc, which allocates nothing: a
// header of SCRATCH_HEAD words (32-bit word 0: bits of the largest
// |gradient|, word 1: the bad-index flag), then the four accumulator words
// of each of up to FST_SCATTER_NOALLOC_MAX_TARGETS targets.  Each device
// holds its own copy for the life of the process; host code reaches it only
// through the address hipGetSymbolAddress gives on that device
// (scatter_scratch below).
constexpr long long SCRATCH_HEAD = 4;
constexpr long long SCRATCH_WORDS = SCRATCH_HEAD + 4ll * FST_SCATTER_NOALLOC_MAX_TARGETS;
static __device__ __align__(256) ull scratch[SCRATCH_WORDS];

int grid_for(long long n) {
  long long b = (n + NT - 1) / NT;
  if (b < 1) b = 1;
  if (b > 4096) b = 4096;
  return (int)b;
}

}  // namespace

// ---------------------------------------------------------------------------
// host-side launchers
// ---------------------------------------------------------------------------

hipError_t launch_score_structure(const ScoreGraph &G, int32_t *owner, int32_t *extra,
                                  int32_t *inref, int32_t *mbeg, int32_t *mlen, int32_t *mcur,
                                  int32_t *marc, int32_t *mpos, ScoreScalars *sc,
                                  hipStream_t s) {
  if (G.E > 0) {
    k_owner<<<grid_for(G.E), NT, 0, s>>>(G, owner);
    k_extra<<<grid_for(G.E), NT, 0, s>>>(G, owner, extra);
  }
  k_merge_index<<<grid_for(G.V), NT, 0, s>>>(G, owner, extra, inref, mbeg, mlen, mcur, sc);
  if (G.E > 0) {
    const long long chunks = (G.E + (long long)MP_ITEMS * NT - 1) / ((long long)MP_ITEMS * NT);
    k_merge_place<<<(unsigned)(chunks < 4096 ? chunks : 4096), NT, 0, s>>>(G, inref, mcur, marc,
                                                                          mpos);
  }
  return hipGetLastError();
}

hipError_t launch_score_seed(const ScoreArgs &S, bool forward, hipStream_t s) {
  if (forward) k_score_init<true><<<grid_for(S.G.V), NT, 0, s>>>(S);
  else k_score_init<false><<<grid_for(S.G.V), NT, 0, s>>>(S);
  return hipGetLastError();
}

hipError_t launch_score_generation(const ScoreArgs *F, const ScoreArgs *B, int g,
                                   hipStream_t s) {
  if (F && B) k_score_gen2<<<2 * SCORE_GRID, NT, 0, s>>>(*F, *B, g);
  else if (F) k_score_gen<true><<<SCORE_GRID, NT, 0, s>>>(*F, g);
  else if (B) k_score_gen<false><<<SCORE_GRID, NT, 0, s>>>(*B, g);
  return hipGetLastError();
}

hipError_t launch_sweep(const ScoreGraph &G, const double *xa, double *ya, const double *xb,
                        double *yb, unsigned long long *incr, hipStream_t s) {
  if (G.V == 0) return hipSuccess;
  const long long b = ((long long)G.V + NT - 1) / NT;
  k_sweep<<<(unsigned)(b < SWEEP_GRID ? b : SWEEP_GRID), NT, 0, s>>>(G, xa, ya, xb, yb, incr);
  return hipGetLastError();
}

hipError_t launch_in_csr(const ScoreGraph &G, int32_t *ioff, int32_t *isrc, float *iw,
                         int32_t *cur, void *scan_temp, unsigned long long *total_dev,
                         hipStream_t s) {
  hipError_t e = hipMemsetAsync(ioff, 0, ((size_t)G.V + 1) * 4, s);
  if (e != hipSuccess) return e;
  if ((e = hipMemsetAsync(cur, 0, (size_t)G.V * 4, s)) != hipSuccess) return e;
  if (G.E) {
    k_in_count<<<grid_for(G.E), NT, 0, s>>>(G, ioff);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  // ioff[v] = in-arcs of the states before v; ioff[V] = E
  e = scan_u32(reinterpret_cast<const uint32_t *>(ioff), reinterpret_cast<uint32_t *>(ioff),
               (size_t)G.V, true, total_dev, scan_temp, s);
  if (e != hipSuccess || G.E == 0) return e;
  k_in_place<<<grid_for(G.E), NT, 0, s>>>(G, ioff, cur, isrc, iw);
  return hipGetLastError();
}

hipError_t launch_fill_f64(double *p, long long n, double x, hipStream_t s) {
  if (n == 0) return hipSuccess;
  k_fill_f64<<<grid_for(n), NT, 0, s>>>(p, n, x);
  return hipGetLastError();
}

hipError_t launch_score_total(const double *val, const uint8_t *flag, int32_t V,
                              ScoreScalars *sc, double *total, hipStream_t s) {
  k_total_max<<<grid_for((long long)V / 16 + 1), NT, 0, s>>>(val, flag, V, sc);
  k_total_sum<<<grid_for((long long)V / 16 + 1), NT, 0, s>>>(val, flag, V, sc);
  k_total_final<<<1, 1, 0, s>>>(sc, total);
  return hipGetLastError();
}

hipError_t launch_segment_logsum(const double *val, const uint8_t *flag, int32_t n,
                                 const long long *bounds, long long max_len, ull *z,
                                 double *totals, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (max_len > 0) {
    long long bx = (max_len + NT - 1) / NT;
    if (bx > 1024) bx = 1024;
    const dim3 grid((unsigned)bx, (unsigned)n);
    k_seg_max<<<grid, NT, 0, s>>>(val, flag, bounds, z);
    k_seg_sum<<<grid, NT, 0, s>>>(val, flag, bounds, z);
  }
  k_seg_final<<<grid_for(n), NT, 0, s>>>(n, z, totals);
  return hipGetLastError();
}

hipError_t launch_posterior(const ScoreGraph &G, const double *alpha, const double *beta,
                            const double *total, float scale, float *grad, hipStream_t s) {
  if (G.E > 0) k_posterior<<<grid_for(G.E), NT, 0, s>>>(G, alpha, beta, total, scale, grad);
  return hipGetLastError();
}

hipError_t launch_scatter(const float *g, const int32_t *idx, long long n, int32_t m, ull *acc,
                          uint32_t *mx, uint32_t *bad, float *out, const ScatterTemp *tmp,
                          hipStream_t s) {
  if (n > 0) {
    // few workgroups: each ends with one atomic on the same word
    k_absmax<<<grid_for(n / 4 + 1) < 512 ? grid_for(n / 4 + 1) : 512, NT, 0, s>>>(g, n, mx);
    const int32_t nbk = (int32_t)((m + SC_BINS - 1) / SC_BINS);
    if (tmp && scatter_grouped(n, m)) {
      const long long nblk = (n + 8 * NT - 1) / (8 * NT) < SC_BLOCKS ? (n + 8 * NT - 1) / (8 * NT)
                                                                     : SC_BLOCKS;
      const long long per = (n + nblk - 1) / nblk;
      k_bucket_count<<<(unsigned)nblk, NT, 0, s>>>(idx, n, m, nbk, per, tmp->cnt);
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
      e = scan_u32(tmp->cnt, tmp->cnt, (size_t)nbk * nblk, false, tmp->total, tmp->scan, s);
      if (e != hipSuccess) return e;
      k_bucket_place<<<(unsigned)nblk, NT, 0, s>>>(g, idx, n, m, nbk, per, tmp->cnt, tmp->pg,
                                                   tmp->pidx, bad);
      const long long chunks = (n + SC_CHUNK - 1) / SC_CHUNK;
      k_scatter<<<(unsigned)(chunks < 2048 ? chunks : 2048), NT, 0, s>>>(
          tmp->pg, tmp->pidx, n, m, mx, acc, bad, tmp->total);
    } else {
      const long long chunks = (n + SC_CHUNK - 1) / SC_CHUNK;
      k_scatter<<<(unsigned)(chunks < 2048 ? chunks : 2048), NT, 0, s>>>(g, idx, n, m, mx, acc,
                                                                        bad, nullptr);
    }
  }
  if (m > 0) k_scatter_final<<<grid_for(m), NT, 0, s>>>(acc, m, mx, out);
  return hipGetLastError();
}

bool scatter_grouped(long long n, int32_t m) {
  return m > SC_BINS && (long long)m <= (long long)SC_BUCKETS * SC_BINS && n >= 4 * SC_CHUNK;
}

namespace {
constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void *g_scratch[MAX_DEVICES] = {};
}  // namespace

hipError_t scatter_scratch(int device, void **out) {
  *out = nullptr;
  if (device < 0 || device >= MAX_DEVICES) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[device]) {
    // the symbol's address on the current device, which must be `device`
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return e;
    if (cur != device) return hipErrorInvalidDevice;
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch[device] = p;
  }
  *out = g_scratch[device];
  return hipSuccess;
}

hipError_t launch_scatter_noalloc(const float *g, const int32_t *idx, long long n, int32_t m,
                                  void *scr, float *out, hipStream_t s) {
  if (m < 0 || m > FST_SCATTER_NOALLOC_MAX_TARGETS) return hipErrorInvalidValue;
  ull *w = static_cast<ull *>(scr);
  uint32_t *head = static_cast<uint32_t *>(scr);
  // the header and the accumulators of this call's targets start at zero
  // (an earlier call leaves its sums behind)
  const long long words = SCRATCH_HEAD + 4ll * m;
  k_clear<<<grid_for(words), NT, 0, s>>>(w, words);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_scatter(g, idx, n, m, w + SCRATCH_HEAD, head, head + 1, out, nullptr, s);
}

size_t scatter_count_words(long long n, int32_t m) {
  const long long nblk = (n + 8 * NT - 1) / (8 * NT) < SC_BLOCKS ? (n + 8 * NT - 1) / (8 * NT)
                                                                 : SC_BLOCKS;
  return (size_t)((m + SC_BINS - 1) / SC_BINS) * (size_t)nblk;
}

}  // namespace fstc
