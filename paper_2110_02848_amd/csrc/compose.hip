// Kernels of the eager composition C = A o B (paper Section 3.3) for gfx950.
//
//  * validation of the input layout (Section 3.2);
//  * label-sorted arc views with packed per-state and per-arc records and
//    per-state label buckets, so that joining A's output labels with B's
//    input labels costs one bucket lookup per arc instead of a scan of the
//    arc-pair cross product;
//  * the search over composite keys in generations: a light key is expanded
//    by one thread, which then follows the light keys it reaches first
//    depth-first; heavy keys (many epsilon arcs, large label joins) are cut
//    into work units spread over the whole grid; new keys are claimed in a
//    bitmap and appended with one atomic per wavefront (ballot + popcount);
//  * the same search run backwards over in-arcs for co-accessibility;
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

int bitlen(unsigned long long x) { return x ? 64 - __builtin_clzll(x) : 0; }

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

// First index in [lo, hi) whose label (.x) is >= x.
__device__ __forceinline__ int32_t lb_label(const int2 *a, int32_t lo, int32_t hi, int32_t x) {
  while (lo < hi) {
    int32_t mid = lo + ((hi - lo) >> 1);
    if (a[mid].x < x) lo = mid + 1; else hi = mid;
  }
  return lo;
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
  // one atomic per workgroup: same-address atomics serialize
  __shared__ uint32_t s_bits[NWAVES], s_mx[NWAVES];
  bits = wave_or(bits);
  mx = wave_max(mx);
  if (__lane_id() == 0) {
    s_bits[threadIdx.x / WAVE] = bits;
    s_mx[threadIdx.x / WAVE] = mx;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < NWAVES; ++w) {
      bits |= s_bits[w];
      mx = s_mx[w] > mx ? s_mx[w] : mx;
    }
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

// Sorted (key, arc) pairs -> arc records {label, other end} and arc ids.
__global__ __launch_bounds__(NT) void k_split(DevGraph g, int by_dst, const ull *__restrict__ k,
                                              const int32_t *__restrict__ v, long long n,
                                              int lab_bits, const int4 *__restrict__ eps_rec,
                                              int32_t *__restrict__ perm,
                                              int2 *__restrict__ arec) {
  const ull mask = (lab_bits >= 64) ? ~0ull : ((1ull << lab_bits) - 1ull);
  for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < n;
       i += (long long)gridDim.x * NT) {
    const int32_t e = v[i];
    perm[i] = e;
    int32_t nb = by_dst ? g.src[e] : g.dst[e];
    if (eps_rec && eps_rec[nb].y > 0) nb |= (int32_t)0x80000000;
    arec[i] = make_int2((int32_t)(k[i] & mask), nb);
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

// State records.  eps_mode: 0 = no epsOutA flag (views of B), 1 = A's
// out-view (flag from its own epsilon count), 2 = A's in-view (flag from
// A's out-view records in eps_rec).
__global__ __launch_bounds__(NT) void k_state_rec(const int32_t *__restrict__ off,
                                                  const int2 *__restrict__ arec, int V,
                                                  const uint8_t *__restrict__ accept,
                                                  int eps_mode, const int4 *__restrict__ eps_rec,
                                                  int4 *__restrict__ srec,
                                                  uint32_t *eps_states) {
  __shared__ uint32_t s_w[NWAVES];
  uint32_t neps_states = 0;
  for (long long v = (long long)blockIdx.x * NT + threadIdx.x; v < V;
       v += (long long)gridDim.x * NT) {
    const int32_t s0 = off[v], s1 = off[v + 1];
    const int32_t n = lb_label(arec, s0, s1, 1) - s0;
    int32_t flags = accept[v] ? (int32_t)FLAG_ACCEPT : 0;
    if ((eps_mode == 1 && n > 0) || (eps_mode == 2 && eps_rec[v].y > 0))
      flags |= (int32_t)FLAG_EPS_OUT;
    srec[v] = make_int4(s0, n, s1, flags);
    neps_states += n > 0 ? 1u : 0u;
  }
  if (eps_states) {
    const uint32_t tot = block_sum(neps_states, s_w);
    if (threadIdx.x == 0 && tot) atomicAdd(eps_states, tot);
  }
}

// Label buckets: lut[v * S + l] = {first position of label l, first > l,
// neighbour of the first arc (or -1), 0}.
__global__ __launch_bounds__(NT) void k_build_lut(const int4 *__restrict__ srec,
                                                  const int2 *__restrict__ arec, int V, int S,
                                                  int4 *__restrict__ lut) {
  const long long n = (long long)V * S;
  for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < n;
       i += (long long)gridDim.x * NT) {
    const int32_t v = (int32_t)(i / S), l = (int32_t)(i % S);
    const int4 r = srec[v];
    const int32_t lo = lb_label(arec, r.x, r.z, l);
    const int32_t hi = lb_label(arec, lo, r.z, l + 1);
    lut[i] = make_int4(lo, hi, lo < hi ? arec[lo].y : -1, 0);
  }
}

// ---------------------------------------------------------------------------
// search helpers
// ---------------------------------------------------------------------------

// Positions [r0, r1) of label `lab` inside group q of a view, whose
// non-epsilon part is [lo, hi), and the neighbour of the first of them: one
// bucket lookup when the view has buckets, else a binary search.
__device__ __forceinline__ void label_range(const View &v, uint32_t q, int32_t lo, int32_t hi,
                                            int32_t lab, int32_t &r0, int32_t &r1,
                                            int32_t &nb0) {
  if (v.lut) {
    if ((uint32_t)lab < (uint32_t)v.lstride) {
      const int4 b = v.lut[(size_t)q * (uint32_t)v.lstride + (uint32_t)lab];
      r0 = b.x;
      r1 = b.y;
      nb0 = b.z;
    } else {
      r0 = r1 = hi;
      nb0 = -1;
    }
    return;
  }
  r0 = lb_label(v.arec, lo, hi, lab);
  r1 = lb_label(v.arec, r0, hi, lab + 1);
  nb0 = r0 < r1 ? v.arec[r0].y : -1;
}

__device__ __forceinline__ void label_range(const View &v, uint32_t q, int32_t lo, int32_t hi,
                                            int32_t lab, int32_t &r0, int32_t &r1) {
  int32_t nb0;
  label_range(v, q, lo, hi, lab, r0, r1, nb0);
}

// Claim a key that few threads are expected to reach at once.
__device__ __forceinline__ bool claim_cold(uint32_t *bm, uint32_t k) {
  const uint32_t bit = 1u << (k & 31u);
  return (atomicOr(bm + (k >> 5), bit) & bit) == 0;
}

// Claim key k in bitmap bm; true for exactly one caller per key.  The plain
// load first matters: keys such as a lexicon root are reached by thousands
// of threads at once, and only the first few should reach the atomic.
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

// Move structure of a key in the forward direction (also used to write C).
struct Fwd {
  uint32_t qa, qb, f;
  int32_t aS, ae, aE, bS, be, bE;
  uint32_t eA, nA, nB, mU;
  uint32_t epsA;    // epsOutA(qa)
  uint32_t accept;  // accept(qa) and accept(qb)
};

__device__ __forceinline__ Fwd fwd_info(const Problem &P, uint32_t key) {
  Fwd s;
  s.f = key_f(key);
  s.qb = key_qb(key, P.shiftB);
  s.qa = key_qa(key, P.shiftB);
  const int4 ra = P.aOut.srec[s.qa];
  const int4 rb = P.bOut.srec[s.qb];
  s.aS = ra.x;
  s.ae = ra.y;
  s.aE = ra.z;
  s.bS = rb.x;
  s.be = rb.y;
  s.bE = rb.z;
  s.epsA = ra.y > 0 ? 1u : 0u;
  s.accept = (uint32_t)(ra.w & rb.w) & FLAG_ACCEPT;
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

// The keys a work unit reaches: for p in [lo, hi), with nb_p the neighbour
// field of arcs[p] (nb_lo given), the key (A state, B state, f) where the
// side named by varyA takes nb_p and the other side is fixed.  In the
// backward direction a key is also visited with f = 1 when `dual` holds or,
// with dual_from_nb, when bit 31 of nb_p (epsOutA of an A-side neighbour)
// is set.  One shape for all move kinds keeps a single visit site per kernel.
struct UnitRange {
  const int2 *arcs;
  int32_t lo, hi, nb0;
  uint32_t fa, fb, f;
  bool varyA, dual, dual_from_nb;
  bool hot;  // the keys may be reached by many threads at once
};

__device__ __forceinline__ UnitRange fwd_range(const Problem &P, const Fwd &s, uint32_t u) {
  UnitRange r;
  r.f = 0;
  r.fa = r.fb = 0;
  r.dual = r.dual_from_nb = false;
  r.hot = true;
  if (u < s.eA) {  // A-epsilon move
    r.arcs = P.aOut.arec;
    r.lo = s.aS + (int32_t)u;
    r.varyA = true;
    r.fb = s.qb;
  } else if (u < s.eA + (uint32_t)s.be) {  // B-epsilon move
    r.arcs = P.bOut.arec;
    r.lo = s.bS + (int32_t)(u - s.eA);
    r.varyA = false;
    r.fa = s.qa;
    r.f = s.epsA;
  } else {  // matching moves of one arc of the smaller side
    r.hot = false;
    const uint32_t j = u - s.eA - (uint32_t)s.be;
    if (s.nA <= s.nB) {
      const int2 ar = P.aOut.arec[s.aS + s.ae + (int32_t)j];
      label_range(P.bOut, s.qb, s.bS + s.be, s.bE, ar.x, r.lo, r.hi, r.nb0);
      r.arcs = P.bOut.arec;
      r.varyA = false;
      r.fa = (uint32_t)ar.y;
    } else {
      const int2 br = P.bOut.arec[s.bS + s.be + (int32_t)j];
      label_range(P.aOut, s.qa, s.aS + s.ae, s.aE, br.x, r.lo, r.hi, r.nb0);
      r.arcs = P.aOut.arec;
      r.varyA = true;
      r.fb = (uint32_t)br.y;
    }
    return r;
  }
  r.hi = r.lo + 1;
  r.nb0 = r.arcs[r.lo].y;
  return r;
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
  const int4 ra = P.aIn.srec[s.va];
  const int4 rb = P.bIn.srec[s.vb];
  s.aS = ra.x;
  s.ae = ra.y;
  s.aE = ra.z;
  s.bS = rb.x;
  s.be = rb.y;
  s.bE = rb.z;
  s.epsV = (ra.w & (int32_t)FLAG_EPS_OUT) ? 1u : 0u;
  s.eA = (s.g == 0) ? (uint32_t)s.ae : 0u;          // A-epsilon moves land on f = 0
  s.eB = (s.g == s.epsV) ? (uint32_t)s.be : 0u;     // B-epsilon moves land on f = epsOutA
  s.nA = (uint32_t)(s.aE - s.aS - s.ae);
  s.nB = (uint32_t)(s.bE - s.bS - s.be);
  s.mU = (s.g == 0 && s.nA && s.nB) ? (s.nA < s.nB ? s.nA : s.nB) : 0u;
  return s;
}

__device__ __forceinline__ uint32_t bwd_units(const Bwd &s) { return s.eA + s.eB + s.mU; }

__device__ __forceinline__ UnitRange bwd_range(const Problem &P, const Bwd &s, uint32_t u) {
  UnitRange r;
  r.f = 0;
  r.fa = r.fb = 0;
  r.dual = r.dual_from_nb = false;
  r.hot = true;
  if (u < s.eA) {  // predecessor by an A-epsilon move: (ua, vb, 0)
    r.arcs = P.aIn.arec;
    r.lo = s.aS + (int32_t)u;
    r.varyA = true;
    r.fb = s.vb;
  } else if (u < s.eA + s.eB) {  // by a B-epsilon move: (va, ub, 0 and 1)
    r.arcs = P.bIn.arec;
    r.lo = s.bS + (int32_t)(u - s.eA);
    r.varyA = false;
    r.fa = s.va;
    r.dual = s.epsV != 0;
  } else {  // by matching moves: (ua, ub, 0 and, if epsOutA(ua), 1)
    r.hot = false;
    const uint32_t j = u - s.eA - s.eB;
    if (s.nA <= s.nB) {
      const int2 ar = P.aIn.arec[s.aS + s.ae + (int32_t)j];
      label_range(P.bIn, s.vb, s.bS + s.be, s.bE, ar.x, r.lo, r.hi, r.nb0);
      r.arcs = P.bIn.arec;
      r.varyA = false;
      r.fa = (uint32_t)(ar.y & NBR_MASK);
      r.dual = ar.y < 0;
    } else {
      const int2 br = P.bIn.arec[s.bS + s.be + (int32_t)j];
      label_range(P.aIn, s.va, s.aS + s.ae, s.aE, br.x, r.lo, r.hi, r.nb0);
      r.arcs = P.aIn.arec;
      r.varyA = true;
      r.fb = (uint32_t)br.y;
      r.dual_from_nb = true;
    }
    return r;
  }
  r.hi = r.lo + 1;
  r.nb0 = r.arcs[r.lo].y;
  return r;
}

// Calls f(key) for every key of unit `u` of a key with structure s.
template <bool FWD, class Info, class F>
__device__ __forceinline__ void for_unit(const Problem &P, const Info &s, uint32_t u, F &&f) {
  UnitRange r;
  if constexpr (FWD) r = fwd_range(P, s, u);
  else r = bwd_range(P, s, u);
  const uint32_t sh = P.shiftB;
  for (int32_t p = r.lo; p < r.hi; ++p) {
    const int32_t y = p == r.lo ? r.nb0 : r.arcs[p].y;
    const uint32_t nb = (uint32_t)(y & NBR_MASK);
    const uint32_t qa = r.varyA ? nb : r.fa, qb = r.varyA ? r.fb : nb;
    const uint32_t nf = (r.dual || (r.dual_from_nb && y < 0)) ? 2u : 1u;
    for (uint32_t ff = 0; ff < nf; ++ff) f(make_key(qa, qb, FWD ? r.f : ff, sh), r.hot);
  }
}

// Direction traits: move structure, unit count and unit expansion.
template <bool FWD>
struct Dir;
template <>
struct Dir<true> {
  typedef Fwd Info;
  static __device__ __forceinline__ Fwd info(const Problem &P, uint32_t k) { return fwd_info(P, k); }
  static __device__ __forceinline__ uint32_t units(const Fwd &s) { return fwd_units(s); }
  template <class F>
  static __device__ __forceinline__ void unit(const Problem &P, const Fwd &s, uint32_t u, F &&f) {
    for_unit<true>(P, s, u, f);
  }
};
template <>
struct Dir<false> {
  typedef Bwd Info;
  static __device__ __forceinline__ Bwd info(const Problem &P, uint32_t k) { return bwd_info(P, k); }
  static __device__ __forceinline__ uint32_t units(const Bwd &s) { return bwd_units(s); }
  template <class F>
  static __device__ __forceinline__ void unit(const Problem &P, const Bwd &s, uint32_t u, F &&f) {
    for_unit<false>(P, s, u, f);
  }
};

// Where the next generation's work goes.
struct NextGen {
  GenSlot *slot;
  uint32_t qbase, hbase;
};

// List a heavy key for the next generation: one packed atomic gives its
// position and the offset of its first unit, consistently.
__device__ __forceinline__ void list_heavy(const SearchArgs &S, const NextGen &nx, uint32_t v,
                                           uint32_t units) {
  const ull old = atomicAdd(&nx.slot->hpack, ((ull)units << 32) | 1ull);
  const ull pos = (ull)nx.hbase + (old & 0xffffffffull);
  if (pos < S.cap && (old >> 32) + units < (1ull << 32)) {
    S.heavy[pos] = v;
    S.hoff[pos] = (uint32_t)(old >> 32);
  } else {
    atomicOr(&S.sc->overflow, 2u);
  }
}

// A key reached for the first time (`fresh`).  Forward: it is counted, and if
// it accepts it is marked co-accessible and listed as a seed of the backward
// search.  Then: heavy keys go to the next generation's heavy list; a light
// key becomes this thread's next key (depth-first continuation) if it has none
// yet and the depth budget allows, else it joins the next frontier.  The
// continuation's move structure is kept in `ci`.
template <bool FWD>
__device__ __forceinline__ void place(const Problem &P, const SearchArgs &S, const NextGen &nx,
                                      bool fresh, uint32_t v, const typename Dir<FWD>::Info &vi,
                                      uint32_t &cont, typename Dir<FWD>::Info &ci, int depth) {
  bool push = false, seed = false;
  if (fresh) {
    const uint32_t u = Dir<FWD>::units(vi);
    if constexpr (FWD) {
      seed = vi.accept != 0;
      if (seed) atomicOr(P.coacc + (v >> 5), 1u << (v & 31u));
    }
    if (u > LIGHT_SEARCH) {
      list_heavy(S, nx, v, u);
    } else if (cont == NO_KEY && depth < P.chain_max) {
      cont = v;
      ci = vi;
    } else {
      push = true;
    }
  }
  if (FWD) wave_push(seed, v, Pusher{S.acc, S.cap, &S.sc->tail2, S.sc});
  wave_push(push, v, Pusher{S.Q + nx.qbase, S.cap - nx.qbase, &nx.slot->qcount, S.sc});
}

// Visit a move target (forward) or a predecessor (backward, where only
// accessible keys are claimed).  The key's state records are loaded before
// the claim is resolved, so both memory round trips overlap.
template <bool FWD>
__device__ __forceinline__ void visit(const Problem &P, const SearchArgs &S, const NextGen &nx,
                                      uint32_t v, bool hot, uint32_t &cont,
                                      typename Dir<FWD>::Info &ci, int depth) {
  const typename Dir<FWD>::Info vi = Dir<FWD>::info(P, v);
  bool fresh;
  if (FWD) {
    fresh = hot ? claim(P.vis, v) : claim_cold(P.vis, v);
  } else {
    const uint32_t bit = 1u << (v & 31u), w = v >> 5;
    const uint32_t wv = P.vis[w], wc = P.coacc[w];  // one round trip for both
    fresh = (wv & bit) && !(wc & bit) && (atomicOr(P.coacc + w, bit) & bit) == 0;
  }
  place<FWD>(P, S, nx, fresh, v, vi, cont, ci, depth);
}

// Generation g (one kernel): one thread per unit of the generation's heavy
// keys, then one thread per light frontier key.  A thread expands its units,
// then, depth-first, the light keys it reached first (one loop, so the visit
// code exists once).  New work goes to the slot of generation g + 1.
template <bool FWD>
__global__ __launch_bounds__(NT) void k_gen(Problem P, SearchArgs S, int g) {
  typedef typename Dir<FWD>::Info Info;
  Scalars *sc = S.sc;
  if (sc->overflow) return;
  const GenSlot cur = sc->G[g % 3];
  const uint32_t hcount = (uint32_t)(cur.hpack & 0xffffffffull);
  const ull U = cur.hpack >> 32;
  NextGen nx;
  nx.slot = &sc->G[(g + 1) % 3];
  nx.qbase = cur.qbase + cur.qcount;
  nx.hbase = cur.hbase + hcount;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    nx.slot->qbase = nx.qbase;  // read by generation g + 1 only
    nx.slot->hbase = nx.hbase;
    GenSlot *done = &sc->G[(g + 2) % 3];  // generation g - 1: free
    done->qcount = 0;
    done->hpack = 0;
    if (U + cur.qcount) sc->gens = (uint32_t)g + 1;
  }
  const uint32_t *hk = S.heavy + cur.hbase;
  const uint32_t *ho = S.hoff + cur.hbase;
  const ull n = U + cur.qcount;
  for (ull i = (ull)blockIdx.x * NT + threadIdx.x; i < n; i += (ull)gridDim.x * NT) {
    uint32_t key, u0 = 0, u1 = 0;
    bool one_unit = false;
    if (i < U) {
      uint32_t a = 0, b = hcount - 1;  // largest a with ho[a] <= i
      while (a < b) {
        const uint32_t mid = (a + b + 1) >> 1;
        if (ho[mid] <= i) a = mid; else b = mid - 1;
      }
      key = hk[a];
      u0 = (uint32_t)(i - ho[a]);
      one_unit = true;
    } else {
      key = S.Q[cur.qbase + (uint32_t)(i - U)];
    }
    Info info = Dir<FWD>::info(P, key);
    u1 = one_unit ? u0 + 1 : Dir<FWD>::units(info);
    for (int depth = 0;; ++depth) {
      uint32_t cont = NO_KEY;
      Info ci = info;
      for (uint32_t u = u0; u < u1; ++u)
        Dir<FWD>::unit(P, info, u,
                       [&](uint32_t v, bool hot) { visit<FWD>(P, S, nx, v, hot, cont, ci, depth); });
      if (cont == NO_KEY) break;
      info = ci;
      u0 = 0;
      u1 = Dir<FWD>::units(ci);
    }
  }
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

// Start keys (sa, sb, 0) for every pair of start states (Algorithm 1) form
// generation 0 of the forward search.
__global__ __launch_bounds__(NT) void k_seed_forward(Problem P, SearchArgs S,
                                                     const int32_t *__restrict__ la,
                                                     const uint32_t *__restrict__ na_p,
                                                     const int32_t *__restrict__ lb,
                                                     const uint32_t *__restrict__ nb_p) {
  const ull na = *na_p, nb = *nb_p, n = na * nb;
  const NextGen nx{&S.sc->G[0], 0u, 0u};
  for (ull i0 = (ull)blockIdx.x * NT; i0 < n; i0 += (ull)gridDim.x * NT) {
    const ull i = i0 + threadIdx.x;
    uint32_t cont = NO_KEY, k = 0;
    bool fresh = false;
    Fwd ci;
    if (i < n) {
      k = make_key((uint32_t)la[i / nb], (uint32_t)lb[i % nb], 0u, P.shiftB);
      fresh = claim(P.vis, k);
      ci = fwd_info(P, k);
    }
    // depth = chain_max: every light start key joins the frontier
    place<true>(P, S, nx, fresh, k, ci, cont, ci, P.chain_max);
  }
}

// The accepting keys listed by the forward search (already co-accessible)
// form generation 0 of the backward search.
__global__ __launch_bounds__(NT) void k_seed_backward(Problem P, SearchArgs S,
                                                      const uint32_t *__restrict__ list) {
  const uint32_t n = S.sc->tail2;
  const NextGen nx{&S.sc->G[0], 0u, 0u};
  for (ull i0 = (ull)blockIdx.x * NT; i0 < n; i0 += (ull)gridDim.x * NT) {
    const ull i = i0 + threadIdx.x;
    uint32_t cont = NO_KEY;
    const bool valid = i < n;
    const uint32_t k = valid ? list[i] : 0u;
    Bwd ci;
    if (valid) ci = bwd_info(P, k);
    place<false>(P, S, nx, valid, k, ci, cont, ci, P.chain_max);
  }
}

// Number of moves the search examines (a statistic, on request): forward,
// the moves out of the accessible keys; backward, the predecessor moves of
// the co-accessible keys.
template <bool FWD>
__global__ __launch_bounds__(NT) void k_count_moves(Problem P, ull nwords,
                                                    unsigned long long *__restrict__ out) {
  __shared__ ull s_w[NWAVES];
  const uint32_t *bm = FWD ? P.vis : P.coacc;
  ull c = 0;
  const ull nkeys = nwords * 32u;
  for (ull k = (ull)blockIdx.x * NT + threadIdx.x; k < nkeys; k += (ull)gridDim.x * NT) {
    if (!test_bit(bm, (uint32_t)k)) continue;
    const typename Dir<FWD>::Info s = Dir<FWD>::info(P, (uint32_t)k);
    const uint32_t nu = Dir<FWD>::units(s);
    for (uint32_t u = 0; u < nu; ++u) Dir<FWD>::unit(P, s, u, [&](uint32_t, bool) { ++c; });
  }
  const ull tot = block_sum(c, s_w);
  if (threadIdx.x == 0 && tot) atomicAdd(out, tot);
}

// Number of set bits of a bitmap (one atomic per workgroup).
__global__ __launch_bounds__(NT) void k_popcount(const uint32_t *__restrict__ bm, ull nwords,
                                                 unsigned long long *__restrict__ out) {
  __shared__ ull s_w[NWAVES];
  ull c = 0;
  for (ull w = (ull)blockIdx.x * NT + threadIdx.x; w < nwords; w += (ull)gridDim.x * NT)
    c += (ull)__popc(bm[w]);
  const ull tot = block_sum(c, s_w);
  if (threadIdx.x == 0 && tot) atomicAdd(out, tot);
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
    const int32_t ea = P.aOut.perm[p];
    vis(make_key((uint32_t)P.aOut.arec[p].y, s.qb, 0u, sh), P.A.il[ea], 0, P.A.w[ea], ea, -1);
  }
  for (int32_t p = s.bS; p < s.bS + s.be; ++p) {
    const int32_t eb = P.bOut.perm[p];
    vis(make_key(s.qa, (uint32_t)P.bOut.arec[p].y, s.epsA, sh), 0, P.B.ol[eb], P.B.w[eb], -1, eb);
  }
  if (!s.mU) return;
  if (s.nA <= s.nB) {
    int32_t p = s.aS + s.ae, bl = s.bS + s.be;
    while (p < s.aE) {
      const int32_t lab = P.aOut.arec[p].x;
      int32_t pend = p + 1;
      while (pend < s.aE && P.aOut.arec[pend].x == lab) ++pend;
      int32_t lo, hi;
      label_range(P.bOut, s.qb, bl, s.bE, lab, lo, hi);
      if (lo < hi) bl = hi;
      for (int32_t pa = p; pa < pend && lo < hi; ++pa) {
        const int32_t ea = P.aOut.perm[pa];
        const uint32_t da = (uint32_t)P.aOut.arec[pa].y;
        const int32_t ia = P.A.il[ea];
        const float wa = P.A.w[ea];
        for (int32_t pb = lo; pb < hi; ++pb) {
          const int32_t eb = P.bOut.perm[pb];
          vis(make_key(da, (uint32_t)P.bOut.arec[pb].y, 0u, sh), ia, P.B.ol[eb], wa + P.B.w[eb],
              ea, eb);
        }
      }
      p = pend;
    }
  } else {
    int32_t p = s.bS + s.be, al = s.aS + s.ae;
    while (p < s.bE) {
      const int32_t lab = P.bOut.arec[p].x;
      int32_t pend = p + 1;
      while (pend < s.bE && P.bOut.arec[pend].x == lab) ++pend;
      int32_t lo, hi;
      label_range(P.aOut, s.qa, al, s.aE, lab, lo, hi);
      if (lo < hi) al = hi;
      for (int32_t pa = lo; pa < hi; ++pa) {
        const int32_t ea = P.aOut.perm[pa];
        const uint32_t da = (uint32_t)P.aOut.arec[pa].y;
        const int32_t ia = P.A.il[ea];
        const float wa = P.A.w[ea];
        for (int32_t pb = p; pb < pend; ++pb) {
          const int32_t eb = P.bOut.perm[pb];
          vis(make_key(da, (uint32_t)P.bOut.arec[pb].y, 0u, sh), ia, P.B.ol[eb], wa + P.B.w[eb],
              ea, eb);
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
      d = make_key((uint32_t)P.aOut.arec[s.aS + (int32_t)i].y, s.qb, 0u, sh);
      keep = test_bit(P.coacc, d);
    }
    uint32_t tot;
    uint32_t ex = block_excl_scan<uint32_t>(keep ? 1u : 0u, s_w, tot);
    if (FILL && keep) put_arc(O, P, pos0 + run + ex, id, d, P.A.il[ea], 0, P.A.w[ea], ea, -1);
    run += tot;
  }
  for (uint32_t c = 0; c < (uint32_t)s.be; c += NT) {
    const uint32_t i = c + t;
    bool keep = false;
    int32_t eb = 0;
    uint32_t d = 0;
    if (i < (uint32_t)s.be) {
      eb = P.bOut.perm[s.bS + (int32_t)i];
      d = make_key(s.qa, (uint32_t)P.bOut.arec[s.bS + (int32_t)i].y, s.epsA, sh);
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
        const int2 ar = P.aOut.arec[pa];
        ea = P.aOut.perm[pa];
        da = (uint32_t)ar.y;
        label_range(P.bOut, s.qb, s.bS + s.be, s.bE, ar.x, lo, hi);
        for (int32_t pb = lo; pb < hi; ++pb)
          kept += test_bit(P.coacc, make_key(da, (uint32_t)P.bOut.arec[pb].y, 0u, sh));
      }
      uint32_t tot;
      uint32_t ex = block_excl_scan<uint32_t>(kept, s_w, tot);
      if (FILL && kept) {
        const int32_t ia = P.A.il[ea];
        const float wa = P.A.w[ea];
        uint32_t pos = pos0 + run + ex;
        for (int32_t pb = lo; pb < hi; ++pb) {
          const int32_t eb = P.bOut.perm[pb];
          const uint32_t d = make_key(da, (uint32_t)P.bOut.arec[pb].y, 0u, sh);
          if (test_bit(P.coacc, d))
            put_arc(O, P, pos++, id, d, ia, P.B.ol[eb], wa + P.B.w[eb], ea, eb);
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

}  // namespace

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
hipError_t launch_validate(const DevGraph &g, int side, uint32_t *err, uint32_t *maxlab,
                           hipStream_t s) {
  size_t n = (size_t)(g.V + 1 > g.E ? g.V + 1 : g.E);
  k_validate<<<grid_for(n, 64), NT, 0, s>>>(g, side, err, maxlab);
  return hipGetLastError();
}

hipError_t build_view(const DevGraph &g, int side, bool by_dst, int lab_bits, int32_t lab_max,
                      int4 *srec, int2 *arec, int32_t *perm, int4 *lut, int32_t *off_tmp,
                      const int4 *eps_rec, unsigned long long *k0, int32_t *v0,
                      unsigned long long *k1, int32_t *v1, void *sort_temp, uint32_t *eps_states,
                      hipStream_t s) {
  const size_t E = (size_t)g.E;
  hipError_t e;
  if (E) {
    k_make_keys<<<grid_for(E), NT, 0, s>>>(g, side, by_dst ? 1 : 0, lab_bits, k0, v0);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    int bits = bitlen((unsigned long long)(g.V > 0 ? g.V - 1 : 0)) + lab_bits;
    if ((e = radix_sort(k0, v0, k1, v1, E, bits, sort_temp, s)) != hipSuccess) return e;
    k_split<<<grid_for(E), NT, 0, s>>>(g, by_dst ? 1 : 0, k0, v0, (long long)E, lab_bits,
                                       eps_rec, perm, arec);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  const int32_t *off = g.off;
  if (by_dst) {
    k_group_offsets<<<grid_for((size_t)g.V + 1), NT, 0, s>>>(k0, (long long)E, g.V, lab_bits,
                                                            off_tmp);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    off = off_tmp;
  }
  if (g.V) {
    const int eps_mode = side == 1 ? 0 : (by_dst ? 2 : 1);
    k_state_rec<<<grid_for((size_t)g.V, 256), NT, 0, s>>>(off, arec, g.V, g.accept, eps_mode,
                                                          eps_rec, srec, eps_states);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (lut) {
      const size_t n = (size_t)g.V * (size_t)(lab_max + 1);
      k_build_lut<<<grid_for(n, 8192), NT, 0, s>>>(srec, arec, g.V, lab_max + 1, lut);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
  }
  return hipSuccess;
}

hipError_t launch_seed_forward(const Problem &P, const SearchArgs &S, int32_t *la, uint32_t *na,
                               int32_t *lb, uint32_t *nb, hipStream_t s) {
  k_collect<<<grid_for((size_t)P.A.V, 1024), NT, 0, s>>>(P.A.start, P.A.V, la, na);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  k_collect<<<grid_for((size_t)P.B.V, 1024), NT, 0, s>>>(P.B.start, P.B.V, lb, nb);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  k_seed_forward<<<64, NT, 0, s>>>(P, S, la, na, lb, nb);
  return hipGetLastError();
}

hipError_t launch_seed_backward(const Problem &P, const SearchArgs &S, const uint32_t *acc_list,
                                hipStream_t s) {
  k_seed_backward<<<1024, NT, 0, s>>>(P, S, acc_list);
  return hipGetLastError();
}

hipError_t launch_generation(const Problem &P, const SearchArgs &S, bool forward, int g,
                             hipStream_t s) {
  constexpr unsigned GRID = 1024;
  if (forward) k_gen<true><<<GRID, NT, 0, s>>>(P, S, g);
  else k_gen<false><<<GRID, NT, 0, s>>>(P, S, g);
  return hipGetLastError();
}

hipError_t launch_count_moves(const Problem &P, size_t nwords, bool forward,
                              unsigned long long *out, hipStream_t s) {
  if (!nwords) return hipSuccess;
  if (forward) k_count_moves<true><<<grid_for(nwords * 32, 8192), NT, 0, s>>>(P, nwords, out);
  else k_count_moves<false><<<grid_for(nwords * 32, 8192), NT, 0, s>>>(P, nwords, out);
  return hipGetLastError();
}

hipError_t launch_popcount(const uint32_t *bm, size_t nwords, unsigned long long *out,
                           hipStream_t s) {
  if (!nwords) return hipSuccess;
  k_popcount<<<grid_for(nwords, 256), NT, 0, s>>>(bm, nwords, out);
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
