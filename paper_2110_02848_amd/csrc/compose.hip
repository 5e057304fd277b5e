// Kernels of the eager composition C = A o B (paper Section 3.3) for gfx950.
//
//  * validation of the input layout (Section 3.2);
//  * label-sorted arc views, the per-state "label buckets" used to join A's
//    output labels with B's input labels in O(deg) instead of O(deg^2);
//  * frontier expansion: one workgroup takes 256 frontier keys, a workgroup
//    prefix sum spreads their (very uneven) work units over its threads, and
//    new keys are claimed in a bitmap and appended with one atomic per
//    wavefront (ballot + popcount);
//  * the same expansion run backwards over in-arcs for co-accessibility;
//  * compaction: a popcount prefix over the trim bitmap numbers the states in
//    key order; arcs are counted, scanned and written in canonical order.
#include "internal.h"

namespace fstc {

namespace {

typedef unsigned long long ull;

enum : uint32_t { ERR_OFFSETS = 1, ERR_SRC = 2, ERR_DST = 4, ERR_LABEL = 8, ERR_FLAG = 16 };

unsigned grid_for(size_t n, unsigned cap = 4096) {
  size_t g = (n + NT - 1) / NT;
  if (g < 1) g = 1;
  if (g > cap) g = cap;
  return (unsigned)g;
}

__device__ __forceinline__ uint32_t wave_or(uint32_t x) {
#pragma unroll
  for (int o = WAVE / 2; o > 0; o >>= 1) x |= __shfl_xor(x, o, WAVE);
  return x;
}
__device__ __forceinline__ uint32_t wave_max(uint32_t x) {
#pragma unroll
  for (int o = WAVE / 2; o > 0; o >>= 1) {
    uint32_t y = __shfl_xor(x, o, WAVE);
    x = y > x ? y : x;
  }
  return x;
}

// ---------------------------------------------------------------------------
// validation
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(NT) void k_validate(DevGraph g, int side, uint32_t *err,
                                                 uint32_t *maxlab) {
  uint32_t bits = 0, mx = 0;
  const long long V = g.V, E = g.E;
  const long long n = (V + 1 > E) ? V + 1 : E;
  for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < n;
       i += (long long)gridDim.x * NT) {
    if (i <= V) {
      if (i == 0 && g.off[0] != 0) bits |= ERR_OFFSETS;
      if (i == V && g.off[V] != E) bits |= ERR_OFFSETS;
      if (i < V) {
        if (g.off[i + 1] < g.off[i]) bits |= ERR_OFFSETS;
        if (g.start[i] > 1 || g.accept[i] > 1) bits |= ERR_FLAG;
      }
    }
    if (i < E) {
      int32_t s = g.src[i], d = g.dst[i], il = g.il[i], ol = g.ol[i];
      if (d < 0 || d >= V) bits |= ERR_DST;
      if (il < 0 || ol < 0) bits |= ERR_LABEL;
      if (s < 0 || s >= V) {
        bits |= ERR_SRC;
      } else if (!(g.off[s] <= i && i < g.off[s + 1])) {
        bits |= ERR_SRC;
      }
      int32_t lab = side == 0 ? ol : il;
      if (lab > 0 && (uint32_t)lab > mx) mx = (uint32_t)lab;
    }
  }
  bits = wave_or(bits);
  mx = wave_max(mx);
  if (__lane_id() == 0) {
    if (bits) atomicOr(err, bits);
    if (mx) atomicMax(maxlab, mx);
  }
}

// ---------------------------------------------------------------------------
// label-sorted views
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(NT) void k_make_keys(DevGraph g, int side, int by_dst, int lab_bits,
                                                  ull *__restrict__ k, int32_t *__restrict__ v) {
  for (long long e = (long long)blockIdx.x * NT + threadIdx.x; e < g.E;
       e += (long long)gridDim.x * NT) {
    ull grp = (ull)(uint32_t)(by_dst ? g.dst[e] : g.src[e]);
    ull lab = (ull)(uint32_t)(side == 0 ? g.ol[e] : g.il[e]);
    k[e] = (grp << lab_bits) | lab;
    v[e] = (int32_t)e;
  }
}

__global__ __launch_bounds__(NT) void k_split(DevGraph g, int by_dst, const ull *__restrict__ k,
                                              const int32_t *__restrict__ v, long long n,
                                              int lab_bits, int32_t *__restrict__ perm,
                                              int32_t *__restrict__ lab,
                                              int32_t *__restrict__ nbr) {
  const ull mask = (lab_bits >= 64) ? ~0ull : ((1ull << lab_bits) - 1ull);
  for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < n;
       i += (long long)gridDim.x * NT) {
    const int32_t e = v[i];
    perm[i] = e;
    lab[i] = (int32_t)(k[i] & mask);
    nbr[i] = by_dst ? g.src[e] : g.dst[e];
  }
}

// Label buckets: lut[v * S + l] = first position of label >= l in group v.
__global__ __launch_bounds__(NT) void k_build_lut(const int32_t *__restrict__ off,
                                                  const int32_t *__restrict__ lab, int V, int S,
                                                  int32_t *__restrict__ lut) {
  const long long n = (long long)V * S;
  for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < n;
       i += (long long)gridDim.x * NT) {
    const int32_t v = (int32_t)(i / S), l = (int32_t)(i % S);
    lut[i] = lower_bound_i32(lab, off[v], off[v + 1], l);
  }
}

// off[v] = first sorted position whose group is >= v (v = 0..V).
__global__ __launch_bounds__(NT) void k_group_offsets(const ull *__restrict__ k, long long n,
                                                      int V, int lab_bits,
                                                      int32_t *__restrict__ off) {
  for (long long v = (long long)blockIdx.x * NT + threadIdx.x; v <= V;
       v += (long long)gridDim.x * NT) {
    ull x = (ull)v << lab_bits;
    long long lo = 0, hi = n;
    while (lo < hi) {
      long long mid = lo + ((hi - lo) >> 1);
      if (k[mid] < x) lo = mid + 1; else hi = mid;
    }
    off[v] = (int32_t)lo;
  }
}

__global__ __launch_bounds__(NT) void k_neps(const int32_t *__restrict__ off,
                                             const int32_t *__restrict__ lab, int V,
                                             int32_t *__restrict__ neps,
                                             uint32_t *eps_states) {
  for (long long v = (long long)blockIdx.x * NT + threadIdx.x; v < V;
       v += (long long)gridDim.x * NT) {
    int32_t s0 = off[v], s1 = off[v + 1];
    int32_t n = lower_bound_i32(lab, s0, s1, 1) - s0;
    neps[v] = n;
    if (eps_states) {
      unsigned long long m = __ballot(n > 0);
      if (m && __lane_id() == (unsigned)(__ffsll(m) - 1))
        atomicAdd(eps_states, (uint32_t)__popcll(m));
    }
  }
}

// ---------------------------------------------------------------------------
// search helpers
// ---------------------------------------------------------------------------

// Positions of label `lab` inside group q of a view, whose non-epsilon part
// is [lo, hi): one bucket lookup when the view has buckets, else a binary
// search.
__device__ __forceinline__ void label_range(const View &v, uint32_t q, int32_t lo, int32_t hi,
                                            int32_t lab, int32_t &r0, int32_t &r1) {
  if (v.lut) {
    if ((uint32_t)lab < (uint32_t)(v.lstride - 1)) {
      const int32_t *b = v.lut + (size_t)q * (uint32_t)v.lstride + lab;
      r0 = b[0];
      r1 = b[1];
    } else {
      r0 = r1 = hi;
    }
    return;
  }
  r0 = lower_bound_i32(v.lab, lo, hi, lab);
  r1 = upper_bound_i32(v.lab, r0, hi, lab);
}

// Claim key k in bitmap bm; true for exactly one caller per key.
__device__ __forceinline__ bool claim(uint32_t *bm, uint32_t k) {
  const uint32_t bit = 1u << (k & 31u);
  uint32_t *w = bm + (k >> 5);
  if (*w & bit) return false;  // already set (a stale zero falls through)
  return (atomicOr(w, bit) & bit) == 0;
}

// An append-only key list with a device counter.
struct Pusher {
  uint32_t *Q;
  uint32_t cap;
  uint32_t *count;
  Scalars *sc;
};

// Append `key` for every lane with `want`, one atomic per wavefront.
__device__ __forceinline__ void wave_push(bool want, uint32_t key, const Pusher &pu) {
  unsigned long long m = __ballot(want);
  if (m == 0) return;
  const int leader = __ffsll(m) - 1;
  uint32_t base = 0;
  if ((int)__lane_id() == leader) base = atomicAdd(pu.count, (uint32_t)__popcll(m));
  base = __shfl(base, leader, WAVE);
  if (want) {
    uint32_t pos = base + (uint32_t)__popcll(m & __lanemask_lt());
    if (pos < pu.cap) pu.Q[pos] = key;
    else atomicOr(&pu.sc->overflow, 1u);
  }
}

// A key the forward search reached for the first time: count it, and if it
// accepts, mark it co-accessible and list it as a seed of the backward search.
__device__ __forceinline__ void note_accessible(const Problem &P, bool fresh, uint32_t v,
                                                const Pusher &acc, uint32_t &nacc) {
  bool accepting = false;
  if (fresh) {
    ++nacc;
    accepting = P.A.accept[key_qa(v, P.shiftB)] && P.B.accept[key_qb(v, P.shiftB)];
    if (accepting) atomicOr(P.coacc + (v >> 5), 1u << (v & 31u));
  }
  wave_push(accepting, v, acc);
}

// Move structure of a key (forward direction; also used by compaction).
struct Fwd {
  uint32_t qa, qb, f;
  int32_t aS, ae, aE, bS, be, bE;
  uint32_t eA, nA, nB, mU;
};

__device__ __forceinline__ Fwd fwd_info(const Problem &P, uint32_t key) {
  Fwd s;
  s.f = key_f(key);
  s.qb = key_qb(key, P.shiftB);
  s.qa = key_qa(key, P.shiftB);
  s.aS = P.aOut.off[s.qa];
  s.aE = P.aOut.off[s.qa + 1];
  s.ae = P.aOut.neps[s.qa];
  s.bS = P.bOut.off[s.qb];
  s.bE = P.bOut.off[s.qb + 1];
  s.be = P.bOut.neps[s.qb];
  s.eA = s.f ? 0u : (uint32_t)s.ae;
  s.nA = (uint32_t)(s.aE - s.aS - s.ae);
  s.nB = (uint32_t)(s.bE - s.bS - s.be);
  s.mU = (s.nA && s.nB) ? (s.nA < s.nB ? s.nA : s.nB) : 0u;
  return s;
}

// Work units of a key: its A-epsilon arcs, its B-epsilon arcs, and the
// non-epsilon arcs of the smaller side (each joined with the other side's
// bucket of its label).
__device__ __forceinline__ uint32_t fwd_units(const Fwd &s) { return s.eA + (uint32_t)s.be + s.mU; }

// Calls f(dst key) for the moves of unit `u` of key s.
template <class F>
__device__ __forceinline__ void fwd_unit(const Problem &P, const Fwd &s, uint32_t u, F &&f) {
  const uint32_t sh = P.shiftB;
  if (u < s.eA) {
    f(make_key((uint32_t)P.aOut.nbr[s.aS + (int32_t)u], s.qb, 0u, sh));
  } else if (u < s.eA + (uint32_t)s.be) {
    f(make_key(s.qa, (uint32_t)P.bOut.nbr[s.bS + (int32_t)(u - s.eA)], s.ae > 0 ? 1u : 0u, sh));
  } else {
    const uint32_t j = u - s.eA - (uint32_t)s.be;
    int32_t lo, hi;
    if (s.nA <= s.nB) {
      const int32_t pa = s.aS + s.ae + (int32_t)j;
      const uint32_t da = (uint32_t)P.aOut.nbr[pa];
      label_range(P.bOut, s.qb, s.bS + s.be, s.bE, P.aOut.lab[pa], lo, hi);
      for (int32_t p = lo; p < hi; ++p) f(make_key(da, (uint32_t)P.bOut.nbr[p], 0u, sh));
    } else {
      const int32_t pb = s.bS + s.be + (int32_t)j;
      const uint32_t db = (uint32_t)P.bOut.nbr[pb];
      label_range(P.aOut, s.qa, s.aS + s.ae, s.aE, P.bOut.lab[pb], lo, hi);
      for (int32_t p = lo; p < hi; ++p) f(make_key((uint32_t)P.aOut.nbr[p], db, 0u, sh));
    }
  }
}

// Backward structure of key v = (va, vb, g): the predecessors are the exact
// inverse of the three forward moves.
struct Bwd {
  uint32_t va, vb, g, epsV;
  int32_t aS, ae, aE, bS, be, bE;
  uint32_t eA, eB, nA, nB, mU;
};

__device__ __forceinline__ Bwd bwd_info(const Problem &P, uint32_t key) {
  Bwd s;
  s.g = key_f(key);
  s.vb = key_qb(key, P.shiftB);
  s.va = key_qa(key, P.shiftB);
  s.aS = P.aIn.off[s.va];
  s.aE = P.aIn.off[s.va + 1];
  s.ae = P.aIn.neps[s.va];
  s.bS = P.bIn.off[s.vb];
  s.bE = P.bIn.off[s.vb + 1];
  s.be = P.bIn.neps[s.vb];
  s.epsV = P.aOut.neps[s.va] > 0 ? 1u : 0u;
  s.eA = (s.g == 0) ? (uint32_t)s.ae : 0u;          // A-epsilon moves land on f = 0
  s.eB = (s.g == s.epsV) ? (uint32_t)s.be : 0u;     // B-epsilon moves land on f = epsOutA
  s.nA = (uint32_t)(s.aE - s.aS - s.ae);
  s.nB = (uint32_t)(s.bE - s.bS - s.be);
  s.mU = (s.g == 0 && s.nA && s.nB) ? (s.nA < s.nB ? s.nA : s.nB) : 0u;
  return s;
}

__device__ __forceinline__ uint32_t bwd_units(const Bwd &s) { return s.eA + s.eB + s.mU; }

// Calls f(predecessor key) for the predecessors of unit `u` of key s.
template <class F>
__device__ __forceinline__ void bwd_unit(const Problem &P, const Bwd &s, uint32_t u, F &&f) {
  const uint32_t sh = P.shiftB;
  if (u < s.eA) {
    f(make_key((uint32_t)P.aIn.nbr[s.aS + (int32_t)u], s.vb, 0u, sh));
  } else if (u < s.eA + s.eB) {
    const uint32_t ub = (uint32_t)P.bIn.nbr[s.bS + (int32_t)(u - s.eA)];
    f(make_key(s.va, ub, 0u, sh));
    if (s.epsV) f(make_key(s.va, ub, 1u, sh));
  } else {
    const uint32_t j = u - s.eA - s.eB;
    int32_t lo, hi;
    if (s.nA <= s.nB) {
      const int32_t pa = s.aS + s.ae + (int32_t)j;
      const uint32_t ua = (uint32_t)P.aIn.nbr[pa];
      const bool fa = P.aOut.neps[ua] > 0;
      label_range(P.bIn, s.vb, s.bS + s.be, s.bE, P.aIn.lab[pa], lo, hi);
      for (int32_t p = lo; p < hi; ++p) {
        const uint32_t ub = (uint32_t)P.bIn.nbr[p];
        f(make_key(ua, ub, 0u, sh));
        if (fa) f(make_key(ua, ub, 1u, sh));
      }
    } else {
      const int32_t pb = s.bS + s.be + (int32_t)j;
      const uint32_t ub = (uint32_t)P.bIn.nbr[pb];
      label_range(P.aIn, s.va, s.aS + s.ae, s.aE, P.bIn.lab[pb], lo, hi);
      for (int32_t p = lo; p < hi; ++p) {
        const uint32_t ua = (uint32_t)P.aIn.nbr[p];
        f(make_key(ua, ub, 0u, sh));
        if (P.aOut.neps[ua] > 0) f(make_key(ua, ub, 1u, sh));
      }
    }
  }
}

template <bool FWD>
__device__ __forceinline__ uint32_t units_of(const Problem &P, uint32_t key) {
  if (FWD) return fwd_units(fwd_info(P, key));
  return bwd_units(bwd_info(P, key));
}

// A key reached for the first time: forward = newly accessible; backward =
// accessible and newly co-accessible.
template <bool FWD>
__device__ __forceinline__ bool first_visit(const Problem &P, uint32_t k) {
  if (FWD) return claim(P.vis, k);
  return test_bit(P.vis, k) && claim(P.coacc, k);
}

// A newly claimed key either becomes this thread's next key (depth-first
// continuation, only for light keys) or is appended to the next frontier.
template <bool FWD>
__device__ __forceinline__ void offer(const Problem &P, bool fresh, uint32_t v, uint32_t &cont,
                                      int depth, const Pusher &pu) {
  bool take = false;
  if (fresh && cont == NO_KEY && depth < P.chain_max) take = units_of<FWD>(P, v) <= LIGHT_SEARCH;
  if (take) cont = v;
  wave_push(fresh && !take, v, pu);
}

// Per-thread search counters, summed per wavefront at kernel end.
struct Tally {
  ull gen = 0;        // moves generated (forward)
  uint32_t nacc = 0;  // keys reached for the first time (forward)
};

__device__ __forceinline__ void flush_tally(Tally &t, Scalars *sc) {
  const ull gen = wave_sum(t.gen);
  const uint32_t nacc = wave_sum(t.nacc);
  if (__lane_id() == 0) {
    if (gen) atomicAdd(&sc->generated, gen);
    if (nacc) atomicAdd(&sc->naccessible, nacc);
  }
}

// Visit one move target (forward) or predecessor (backward) v.
template <bool FWD>
__device__ __forceinline__ void visit(const Problem &P, uint32_t v, uint32_t &cont, int depth,
                                      const Pusher &pu, const Pusher &acc, Tally &t) {
  const bool fresh = first_visit<FWD>(P, v);
  if (FWD) {
    ++t.gen;
    note_accessible(P, fresh, v, acc, t.nacc);
  }
  offer<FWD>(P, fresh, v, cont, depth, pu);
}

// Expand `key` and then, depth-first, the light keys it discovers, until a
// key discovers nothing new or the depth budget is spent.
template <bool FWD>
__device__ void run_chain(const Problem &P, uint32_t key, int depth, const Pusher &pu,
                          const Pusher &acc, Tally &t) {
  while (key != NO_KEY) {
    uint32_t cont = NO_KEY;
    auto f = [&](uint32_t v) { visit<FWD>(P, v, cont, depth, pu, acc, t); };
    if (FWD) {
      const Fwd s = fwd_info(P, key);
      const uint32_t n = fwd_units(s);
      for (uint32_t u = 0; u < n; ++u) fwd_unit(P, s, u, f);
    } else {
      const Bwd s = bwd_info(P, key);
      const uint32_t n = bwd_units(s);
      for (uint32_t u = 0; u < n; ++u) bwd_unit(P, s, u, f);
    }
    key = cont;
    ++depth;
  }
}

// Generation step 1: every frontier key Q[qlo, qhi).  Light keys are expanded
// by their thread (with continuation); heavy keys are listed with the prefix
// of their unit counts (one packed 64-bit atomic per wavefront keeps list
// positions and unit offsets consistent) for step 2.
template <bool FWD>
__global__ __launch_bounds__(NT) void k_gen_expand(Problem P, Pusher pu, Pusher acc,
                                                   uint32_t *heavy, uint32_t *hoff, int g) {
  Scalars *sc = pu.sc;
  if (sc->overflow) return;
  const GenDesc d = sc->D[g & 1];
  Tally t;
  for (ull i0 = (ull)d.qlo + (ull)blockIdx.x * NT; i0 < d.qhi; i0 += (ull)gridDim.x * NT) {
    const ull i = i0 + threadIdx.x;
    const bool valid = i < d.qhi;
    const uint32_t key = valid ? pu.Q[i] : 0u;
    const uint32_t units = valid ? units_of<FWD>(P, key) : 0u;
    const bool hv = valid && units > LIGHT_SEARCH;
    const unsigned long long m = __ballot(hv);
    if (m) {
      const ull mine = hv ? (ull)units : 0ull;
      const ull incl = wave_incl_scan(mine);
      const ull tot = __shfl(incl, WAVE - 1, WAVE);
      const int leader = __ffsll(m) - 1;
      ull old = 0;
      if ((int)__lane_id() == leader) old = atomicAdd(&sc->hpack, (tot << 32) | (ull)__popcll(m));
      old = __shfl(old, leader, WAVE);
      if (hv) {
        const ull pos = (ull)d.hlo + (old & 0xffffffffull) + (ull)__popcll(m & __lanemask_lt());
        const ull off = (old >> 32) + incl - mine;
        if (pos < pu.cap && (old >> 32) + tot < (1ull << 32)) {
          heavy[pos] = key;
          hoff[pos] = (uint32_t)off;
        } else {
          atomicOr(&sc->overflow, 2u);
        }
      }
    }
    if (valid && !hv) run_chain<FWD>(P, key, 0, pu, acc, t);
  }
  if (FWD) flush_tally(t, sc);
}

// Generation step 2: one thread per unit of this generation's heavy keys.
template <bool FWD>
__global__ __launch_bounds__(NT) void k_gen_units(Problem P, Pusher pu, Pusher acc,
                                                  const uint32_t *__restrict__ heavy,
                                                  const uint32_t *__restrict__ hoff, int g) {
  Scalars *sc = pu.sc;
  if (sc->overflow) return;  // the heavy list may be incomplete
  const GenDesc d = sc->D[g & 1];
  const ull hp = sc->hpack;
  const ull U = hp >> 32;
  const uint32_t n = (uint32_t)(hp & 0xffffffffull);
  const uint32_t *hk = heavy + d.hlo;
  const uint32_t *ho = hoff + d.hlo;
  Tally t;
  for (ull u = (ull)blockIdx.x * NT + threadIdx.x; u < U; u += (ull)gridDim.x * NT) {
    uint32_t a = 0, b = n - 1;  // largest i with ho[i] <= u
    while (a < b) {
      const uint32_t mid = (a + b + 1) >> 1;
      if (ho[mid] <= u) a = mid; else b = mid - 1;
    }
    const uint32_t key = hk[a];
    const uint32_t local = (uint32_t)(u - ho[a]);
    uint32_t cont = NO_KEY;
    auto f = [&](uint32_t v) { visit<FWD>(P, v, cont, 0, pu, acc, t); };
    if (FWD) fwd_unit(P, fwd_info(P, key), local, f);
    else bwd_unit(P, bwd_info(P, key), local, f);
    if (cont != NO_KEY) run_chain<FWD>(P, cont, 1, pu, acc, t);
  }
  if (FWD) flush_tally(t, sc);
}

// Generation step 3: the keys appended during this generation form the next
// frontier.
__global__ void k_gen_advance(Scalars *sc, int g, uint32_t cap) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  const GenDesc d = sc->D[g & 1];
  GenDesc nd;
  nd.qlo = d.qhi;
  nd.qhi = sc->tail < cap ? sc->tail : cap;
  nd.hlo = d.hlo + (uint32_t)(sc->hpack & 0xffffffffull);
  nd.pad = 0;
  sc->D[(g + 1) & 1] = nd;
  sc->hpack = 0;
  if (d.qlo < d.qhi) sc->gens = (uint32_t)g + 1;
}

__global__ void k_gen_init(Scalars *sc, uint32_t cap) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  GenDesc d;
  d.qlo = 0;
  d.qhi = sc->tail < cap ? sc->tail : cap;
  d.hlo = 0;
  d.pad = 0;
  sc->D[0] = d;
  sc->D[1] = d;
  sc->hpack = 0;
  sc->gens = 0;
}

__global__ __launch_bounds__(NT) void k_collect(const uint8_t *__restrict__ flags, int V,
                                                int32_t *__restrict__ list,
                                                uint32_t *__restrict__ count) {
  for (long long v = (long long)blockIdx.x * NT + threadIdx.x; v < V;
       v += (long long)gridDim.x * NT) {
    bool want = flags[v] != 0;
    unsigned long long m = __ballot(want);
    if (!m) continue;
    const int leader = __ffsll(m) - 1;
    uint32_t base = 0;
    if ((int)__lane_id() == leader) base = atomicAdd(count, (uint32_t)__popcll(m));
    base = __shfl(base, leader, WAVE);
    if (want) list[base + __popcll(m & __lanemask_lt())] = (int32_t)v;
  }
}

// Start keys (sa, sb, 0) for every pair of start states (Algorithm 1).
__global__ __launch_bounds__(NT) void k_seed(Problem P, const int32_t *__restrict__ la,
                                             const uint32_t *__restrict__ na_p,
                                             const int32_t *__restrict__ lb,
                                             const uint32_t *__restrict__ nb_p, Pusher pu,
                                             Pusher acc) {
  const ull na = *na_p, nb = *nb_p, n = na * nb;
  Tally t;
  for (ull i0 = (ull)blockIdx.x * NT; i0 < n; i0 += (ull)gridDim.x * NT) {
    const ull i = i0 + threadIdx.x;
    bool fresh = false;
    uint32_t k = 0;
    if (i < n) {
      k = make_key((uint32_t)la[i / nb], (uint32_t)lb[i % nb], 0u, P.shiftB);
      fresh = claim(P.vis, k);
    }
    note_accessible(P, fresh, k, acc, t.nacc);
    wave_push(fresh, k, pu);
  }
  flush_tally(t, pu.sc);
}

// ---------------------------------------------------------------------------
// compaction
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(NT) void k_popc_words(const uint32_t *__restrict__ bm,
                                                   uint32_t *__restrict__ cnt, ull nwords) {
  for (ull w = (ull)blockIdx.x * NT + threadIdx.x; w < nwords; w += (ull)gridDim.x * NT)
    cnt[w] = (uint32_t)__popc(bm[w]);
}

__global__ __launch_bounds__(NT) void k_key_of_id(const uint32_t *__restrict__ bm,
                                                  const uint32_t *__restrict__ wbase,
                                                  ull nwords, uint32_t *__restrict__ key_of) {
  for (ull w = (ull)blockIdx.x * NT + threadIdx.x; w < nwords; w += (ull)gridDim.x * NT) {
    uint32_t m = bm[w];
    uint32_t id = wbase[w];
    while (m) {
      uint32_t b = (uint32_t)(__ffs(m) - 1);
      key_of[id++] = (uint32_t)(w * 32u + b);
      m &= m - 1u;
    }
  }
}

__device__ __forceinline__ uint32_t new_id(const Problem &P, uint32_t k) {
  const uint32_t w = k >> 5;
  return P.wbase[w] + (uint32_t)__popc(P.coacc[w] & ((1u << (k & 31u)) - 1u));
}

__device__ __forceinline__ uint32_t out_units(const Fwd &s) { return s.eA + (uint32_t)s.be + s.mU; }

// Sequential enumeration of a state's moves in canonical order: A-epsilon
// arcs, B-epsilon arcs, then matching arcs by (label, a, b).  The join walks
// the label groups of the side with fewer non-epsilon arcs and looks up the
// other side's bucket; each group is emitted row-major (a outer, b inner).
template <class Visit>
__device__ __forceinline__ void enum_light(const Problem &P, const Fwd &s, Visit &&vis) {
  const uint32_t sh = P.shiftB;
  for (int32_t p = s.aS; p < s.aS + (int32_t)s.eA; ++p) {
    int32_t ea = P.aOut.perm[p];
    vis(make_key((uint32_t)P.aOut.nbr[p], s.qb, 0u, sh), P.A.il[ea], 0, P.A.w[ea], ea, -1);
  }
  const uint32_t f2 = s.ae > 0 ? 1u : 0u;
  for (int32_t p = s.bS; p < s.bS + s.be; ++p) {
    int32_t eb = P.bOut.perm[p];
    vis(make_key(s.qa, (uint32_t)P.bOut.nbr[p], f2, sh), 0, P.B.ol[eb], P.B.w[eb], -1, eb);
  }
  if (!s.mU) return;
  if (s.nA <= s.nB) {
    int32_t p = s.aS + s.ae, bl = s.bS + s.be;
    while (p < s.aE) {
      const int32_t lab = P.aOut.lab[p];
      int32_t pend = p + 1;
      while (pend < s.aE && P.aOut.lab[pend] == lab) ++pend;
      int32_t lo, hi;
      label_range(P.bOut, s.qb, bl, s.bE, lab, lo, hi);
      if (lo < hi) bl = hi;
      for (int32_t pa = p; pa < pend && lo < hi; ++pa) {
        const int32_t ea = P.aOut.perm[pa];
        const uint32_t da = (uint32_t)P.aOut.nbr[pa];
        const int32_t ia = P.A.il[ea];
        const float wa = P.A.w[ea];
        for (int32_t pb = lo; pb < hi; ++pb) {
          const int32_t eb = P.bOut.perm[pb];
          vis(make_key(da, (uint32_t)P.bOut.nbr[pb], 0u, sh), ia, P.B.ol[eb], wa + P.B.w[eb], ea,
              eb);
        }
      }
      p = pend;
    }
  } else {
    int32_t p = s.bS + s.be, al = s.aS + s.ae;
    while (p < s.bE) {
      const int32_t lab = P.bOut.lab[p];
      int32_t pend = p + 1;
      while (pend < s.bE && P.bOut.lab[pend] == lab) ++pend;
      int32_t lo, hi;
      label_range(P.aOut, s.qa, al, s.aE, lab, lo, hi);
      if (lo < hi) al = hi;
      for (int32_t pa = lo; pa < hi; ++pa) {
        const int32_t ea = P.aOut.perm[pa];
        const uint32_t da = (uint32_t)P.aOut.nbr[pa];
        const int32_t ia = P.A.il[ea];
        const float wa = P.A.w[ea];
        for (int32_t pb = p; pb < pend; ++pb) {
          const int32_t eb = P.bOut.perm[pb];
          vis(make_key(da, (uint32_t)P.bOut.nbr[pb], 0u, sh), ia, P.B.ol[eb], wa + P.B.w[eb], ea,
              eb);
        }
      }
      p = pend;
    }
  }
}

__device__ __forceinline__ void put_arc(const OutGraph &O, const Problem &P, uint32_t pos,
                                        uint32_t id, uint32_t dk, int32_t il, int32_t ol,
                                        float w, int32_t ea, int32_t eb) {
  O.src[pos] = (int32_t)id;
  O.dst[pos] = (int32_t)new_id(P, dk);
  O.il[pos] = il;
  O.ol[pos] = ol;
  O.w[pos] = w;
  if (O.arc_a) O.arc_a[pos] = ea;
  if (O.arc_b) O.arc_b[pos] = eb;
}

// Workgroup-cooperative canonical enumeration of one heavy state.  Every
// thread of the workgroup must call it.  Returns the number of kept arcs;
// with FILL it also writes them from arc position `pos0` on.
template <bool FILL>
__device__ uint32_t heavy_state(const Problem &P, uint32_t id, uint32_t key, uint32_t pos0,
                                const OutGraph &O, uint32_t *s_w) {
  const Fwd s = fwd_info(P, key);
  const uint32_t sh = P.shiftB;
  const unsigned t = threadIdx.x;
  uint32_t run = 0;
  for (uint32_t c = 0; c < s.eA; c += NT) {
    const uint32_t i = c + t;
    bool keep = false;
    int32_t ea = 0;
    uint32_t d = 0;
    if (i < s.eA) {
      ea = P.aOut.perm[s.aS + (int32_t)i];
      d = make_key((uint32_t)P.aOut.nbr[s.aS + (int32_t)i], s.qb, 0u, sh);
      keep = test_bit(P.coacc, d);
    }
    uint32_t tot;
    uint32_t ex = block_excl_scan<uint32_t>(keep ? 1u : 0u, s_w, tot);
    if (FILL && keep) put_arc(O, P, pos0 + run + ex, id, d, P.A.il[ea], 0, P.A.w[ea], ea, -1);
    run += tot;
  }
  const uint32_t f2 = s.ae > 0 ? 1u : 0u;
  for (uint32_t c = 0; c < (uint32_t)s.be; c += NT) {
    const uint32_t i = c + t;
    bool keep = false;
    int32_t eb = 0;
    uint32_t d = 0;
    if (i < (uint32_t)s.be) {
      eb = P.bOut.perm[s.bS + (int32_t)i];
      d = make_key(s.qa, (uint32_t)P.bOut.nbr[s.bS + (int32_t)i], f2, sh);
      keep = test_bit(P.coacc, d);
    }
    uint32_t tot;
    uint32_t ex = block_excl_scan<uint32_t>(keep ? 1u : 0u, s_w, tot);
    if (FILL && keep) put_arc(O, P, pos0 + run + ex, id, d, 0, P.B.ol[eb], P.B.w[eb], -1, eb);
    run += tot;
  }
  if (s.mU) {
    // A-driven: A's non-epsilon arcs in (label, a) order, each joined with
    // B's bucket of its label, gives (label, a, b) order.
    for (uint32_t c = 0; c < s.nA; c += NT) {
      const uint32_t i = c + t;
      int32_t lo = 0, hi = 0, ea = 0;
      uint32_t kept = 0, da = 0;
      if (i < s.nA) {
        const int32_t pa = s.aS + s.ae + (int32_t)i;
        ea = P.aOut.perm[pa];
        da = (uint32_t)P.aOut.nbr[pa];
        label_range(P.bOut, s.qb, s.bS + s.be, s.bE, P.aOut.lab[pa], lo, hi);
        for (int32_t pb = lo; pb < hi; ++pb)
          kept += test_bit(P.coacc, make_key(da, (uint32_t)P.bOut.nbr[pb], 0u, sh));
      }
      uint32_t tot;
      uint32_t ex = block_excl_scan<uint32_t>(kept, s_w, tot);
      if (FILL && kept) {
        const int32_t ia = P.A.il[ea];
        const float wa = P.A.w[ea];
        uint32_t pos = pos0 + run + ex;
        for (int32_t pb = lo; pb < hi; ++pb) {
          const int32_t eb = P.bOut.perm[pb];
          const uint32_t d = make_key(da, (uint32_t)P.bOut.nbr[pb], 0u, sh);
          if (test_bit(P.coacc, d)) put_arc(O, P, pos++, id, d, ia, P.B.ol[eb], wa + P.B.w[eb], ea, eb);
        }
      }
      run += tot;
    }
  }
  return run;
}

__global__ __launch_bounds__(NT) void k_count(Problem P, const uint32_t *__restrict__ key_of,
                                              uint32_t n, uint32_t *__restrict__ cnt,
                                              uint32_t *__restrict__ heavy, Scalars *sc) {
  for (ull i0 = (ull)blockIdx.x * NT; i0 < n; i0 += (ull)gridDim.x * NT) {
    const ull id = i0 + threadIdx.x;
    bool hv = false;
    if (id < n) {
      const Fwd s = fwd_info(P, key_of[id]);
      uint32_t c = 0;
      if (out_units(s) > LIGHT_UNITS) {
        hv = true;
      } else {
        enum_light(P, s, [&](uint32_t d, int32_t, int32_t, float, int32_t, int32_t) {
          c += test_bit(P.coacc, d) ? 1u : 0u;
        });
      }
      cnt[id] = c;
    }
    unsigned long long m = __ballot(hv);
    if (m) {
      const int leader = __ffsll(m) - 1;
      uint32_t base = 0;
      if ((int)__lane_id() == leader) base = atomicAdd(&sc->heavy, (uint32_t)__popcll(m));
      base = __shfl(base, leader, WAVE);
      if (hv) heavy[base + __popcll(m & __lanemask_lt())] = (uint32_t)id;
    }
  }
}

__global__ __launch_bounds__(NT) void k_count_heavy(Problem P, const uint32_t *__restrict__ key_of,
                                                    const uint32_t *__restrict__ heavy,
                                                    const uint32_t *__restrict__ nheavy_p,
                                                    uint32_t *__restrict__ cnt) {
  __shared__ uint32_t s_w[NWAVES];
  const uint32_t nheavy = *nheavy_p;
  OutGraph none = {};
  for (uint32_t h = blockIdx.x; h < nheavy; h += gridDim.x) {
    const uint32_t id = heavy[h];
    uint32_t c = heavy_state<false>(P, id, key_of[id], 0, none, s_w);
    if (threadIdx.x == 0) cnt[id] = c;
  }
}

__global__ __launch_bounds__(NT) void k_fill_light(Problem P, const uint32_t *__restrict__ key_of,
                                                   uint32_t n, const uint32_t *__restrict__ arc_off,
                                                   OutGraph O) {
  for (ull id = (ull)blockIdx.x * NT + threadIdx.x; id < n; id += (ull)gridDim.x * NT) {
    const Fwd s = fwd_info(P, key_of[id]);
    if (out_units(s) > LIGHT_UNITS) continue;
    uint32_t pos = arc_off[id];
    const uint32_t sid = (uint32_t)id;
    enum_light(P, s, [&](uint32_t d, int32_t il, int32_t ol, float w, int32_t ea, int32_t eb) {
      if (test_bit(P.coacc, d)) put_arc(O, P, pos++, sid, d, il, ol, w, ea, eb);
    });
  }
}

__global__ __launch_bounds__(NT) void k_fill_heavy(Problem P, const uint32_t *__restrict__ key_of,
                                                   const uint32_t *__restrict__ heavy,
                                                   uint32_t nheavy,
                                                   const uint32_t *__restrict__ arc_off,
                                                   OutGraph O) {
  __shared__ uint32_t s_w[NWAVES];
  for (uint32_t h = blockIdx.x; h < nheavy; h += gridDim.x) {
    const uint32_t id = heavy[h];
    heavy_state<true>(P, id, key_of[id], arc_off[id], O, s_w);
  }
}

__global__ __launch_bounds__(NT) void k_state_flags(Problem P, const uint32_t *__restrict__ key_of,
                                                    uint32_t n, const uint32_t *__restrict__ arc_off,
                                                    uint32_t narcs, OutGraph O) {
  for (ull id = (ull)blockIdx.x * NT + threadIdx.x; id <= n; id += (ull)gridDim.x * NT) {
    if (id == n) {
      O.arc_offset[n] = (int32_t)narcs;
      continue;
    }
    const uint32_t k = key_of[id];
    const uint32_t qa = key_qa(k, P.shiftB), qb = key_qb(k, P.shiftB), f = key_f(k);
    O.arc_offset[id] = (int32_t)arc_off[id];
    O.accept[id] = (P.A.accept[qa] && P.B.accept[qb]) ? 1 : 0;
    O.start[id] = (f == 0 && P.A.start[qa] && P.B.start[qb]) ? 1 : 0;
    if (O.key_a) O.key_a[id] = (int32_t)qa;
    if (O.key_b) O.key_b[id] = (int32_t)qb;
    if (O.key_f) O.key_f[id] = (uint8_t)f;
  }
}

int bitlen(unsigned long long x) { return x ? 64 - __builtin_clzll(x) : 0; }

}  // namespace

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
hipError_t launch_validate(const DevGraph &g, int side, uint32_t *err, uint32_t *maxlab,
                           hipStream_t s) {
  size_t n = (size_t)(g.V + 1 > g.E ? g.V + 1 : g.E);
  k_validate<<<grid_for(n, 1024), NT, 0, s>>>(g, side, err, maxlab);
  return hipGetLastError();
}

hipError_t build_view(const DevGraph &g, int side, bool by_dst, int lab_bits, int32_t lab_max,
                      int32_t *perm, int32_t *lab, int32_t *nbr, int32_t *neps, int32_t *lut,
                      int32_t *off_out, unsigned long long *k0, int32_t *v0,
                      unsigned long long *k1, int32_t *v1, void *sort_temp, uint32_t *eps_states,
                      hipStream_t s) {
  const size_t E = (size_t)g.E;
  hipError_t e;
  if (E) {
    k_make_keys<<<grid_for(E), NT, 0, s>>>(g, side, by_dst ? 1 : 0, lab_bits, k0, v0);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    int bits = bitlen((unsigned long long)(g.V > 0 ? g.V - 1 : 0)) + lab_bits;
    if ((e = radix_sort(k0, v0, k1, v1, E, bits, sort_temp, s)) != hipSuccess) return e;
    k_split<<<grid_for(E), NT, 0, s>>>(g, by_dst ? 1 : 0, k0, v0, (long long)E, lab_bits, perm,
                                       lab, nbr);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  const int32_t *off = g.off;
  if (by_dst) {
    k_group_offsets<<<grid_for((size_t)g.V + 1), NT, 0, s>>>(k0, (long long)E, g.V, lab_bits,
                                                            off_out);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    off = off_out;
  }
  if (g.V) {
    k_neps<<<grid_for((size_t)g.V), NT, 0, s>>>(off, lab, g.V, neps, eps_states);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (lut) {
      const size_t n = (size_t)g.V * (size_t)(lab_max + 2);
      k_build_lut<<<grid_for(n, 8192), NT, 0, s>>>(off, lab, g.V, lab_max + 2, lut);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
  }
  return hipSuccess;
}

hipError_t launch_seed_lists(const Problem &P, int32_t *la, uint32_t *na, int32_t *lb,
                             uint32_t *nb, uint32_t *queue, uint32_t *acc_list, uint32_t cap,
                             Scalars *sc, hipStream_t s) {
  k_collect<<<grid_for((size_t)P.A.V, 1024), NT, 0, s>>>(P.A.start, P.A.V, la, na);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  k_collect<<<grid_for((size_t)P.B.V, 1024), NT, 0, s>>>(P.B.start, P.B.V, lb, nb);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const Pusher pu{queue, cap, &sc->tail, sc}, acc{acc_list, cap, &sc->tail2, sc};
  k_seed<<<64, NT, 0, s>>>(P, la, na, lb, nb, pu, acc);
  return hipGetLastError();
}

hipError_t launch_gen_init(Scalars *sc, uint32_t cap, hipStream_t s) {
  k_gen_init<<<1, 64, 0, s>>>(sc, cap);
  return hipGetLastError();
}

hipError_t launch_generation(const Problem &P, bool forward, uint32_t *Q, uint32_t *acc_list,
                             uint32_t cap, uint32_t *heavy, uint32_t *hoff, int g, Scalars *sc,
                             hipStream_t s) {
  const Pusher pu{Q, cap, &sc->tail, sc}, acc{acc_list, cap, &sc->tail2, sc};
  constexpr unsigned GRID = 1024;
  if (forward) {
    k_gen_expand<true><<<GRID, NT, 0, s>>>(P, pu, acc, heavy, hoff, g);
    k_gen_units<true><<<GRID, NT, 0, s>>>(P, pu, acc, heavy, hoff, g);
  } else {
    k_gen_expand<false><<<GRID, NT, 0, s>>>(P, pu, acc, heavy, hoff, g);
    k_gen_units<false><<<GRID, NT, 0, s>>>(P, pu, acc, heavy, hoff, g);
  }
  k_gen_advance<<<1, 64, 0, s>>>(sc, g, cap);
  return hipGetLastError();
}

hipError_t launch_popc_words(const uint32_t *bm, uint32_t *cnt, size_t nwords, hipStream_t s) {
  if (!nwords) return hipSuccess;
  k_popc_words<<<grid_for(nwords, 8192), NT, 0, s>>>(bm, cnt, nwords);
  return hipGetLastError();
}

hipError_t launch_key_of_id(const uint32_t *bm, const uint32_t *wbase, size_t nwords,
                            uint32_t *key_of, hipStream_t s) {
  if (!nwords) return hipSuccess;
  k_key_of_id<<<grid_for(nwords, 8192), NT, 0, s>>>(bm, wbase, nwords, key_of);
  return hipGetLastError();
}

hipError_t launch_count(const Problem &P, const uint32_t *key_of, uint32_t nstates,
                        uint32_t *cnt, uint32_t *heavy, Scalars *sc, hipStream_t s) {
  if (!nstates) return hipSuccess;
  k_count<<<grid_for(nstates, 8192), NT, 0, s>>>(P, key_of, nstates, cnt, heavy, sc);
  return hipGetLastError();
}

hipError_t launch_count_heavy(const Problem &P, const uint32_t *key_of, const uint32_t *heavy,
                              const uint32_t *nheavy_dev, uint32_t *cnt, hipStream_t s) {
  k_count_heavy<<<1024, NT, 0, s>>>(P, key_of, heavy, nheavy_dev, cnt);
  return hipGetLastError();
}

hipError_t launch_fill(const Problem &P, const uint32_t *key_of, uint32_t nstates,
                       const uint32_t *arc_off, const uint32_t *heavy, uint32_t nheavy,
                       uint32_t narcs, const OutGraph &O, hipStream_t s) {
  hipError_t e;
  if (nstates) {
    k_fill_light<<<grid_for(nstates, 8192), NT, 0, s>>>(P, key_of, nstates, arc_off, O);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (nheavy) {
    unsigned g = nheavy < 4096 ? nheavy : 4096;
    k_fill_heavy<<<g, NT, 0, s>>>(P, key_of, heavy, nheavy, arc_off, O);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  k_state_flags<<<grid_for((size_t)nstates + 1, 8192), NT, 0, s>>>(P, key_of, nstates, arc_off,
                                                                   narcs, O);
  return hipGetLastError();
}

}  // namespace fstc
